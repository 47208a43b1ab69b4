/*
 * cdb_oracle.c -- plain, slow CPU oracle for continuous depth batching (CDB).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or calls
 * this file; only the tests, the smoke check and the CPU-baseline leg of the
 * benchmark do.  It shares no code, header, table or helper with the HIP path.
 *
 * What it computes (paper, Section 2, Eq. 1): a looped decoder-only LM split
 * into a prelude P, a shared recurrent core R iterated r_t <= r_max times and a
 * coda C:
 *     h^(0)_t = P(x_t),  h^(r+1)_t = R(h^(r)_t, K^(r)_{<t}),
 *     p(x_{t+1}) = softmax(C(h^(r_t)_t)).
 * Depth-indexed KV with the last-exited rule (Section 4.2, Fig. 2 right): the
 * core keeps one KV plane per loop index; when a token exits after d loops,
 * planes d+1..r_max receive a copy of plane d, so a later token at loop r reads
 * the state of loop min(r, d_s) of every earlier token s.
 *
 * Arithmetic is fp64.  Weights arrive as bf16 bit patterns and are widened
 * exactly.  With desc->bf16_storage set, the values the model keeps in bf16
 * (normalised activations that feed a matrix product, the attention output, the
 * SwiGLU product, the adapter input, and every K/V entry) are rounded to bf16
 * at the point they are produced; with it clear, nothing is rounded.
 *
 * Model details the paper leaves open (the readings are listed with the design
 * notes): pre-RMSNorm layers with unit gains and no biases; multi-head
 * attention (kv heads == heads); rotate-half RoPE on q and k at the absolute
 * position; SwiGLU MLP; untied LM head after a final RMSNorm; greedy argmax
 * with the lowest index winning ties; the optional input-injection adapter maps
 * [h; e] (2d) to d before every core pass; exit score sigmoid(w_exit . RMSNorm(h))
 * or, for the convergence criterion (App. C.2), the L2 distance between the
 * states before and after the loop.
 *
 * Other core KV layouts (Section 4.2; App. C.1, Table 1): with a single shared
 * slot per layer, every loop overwrites the token's one K/V entry, so a later
 * token reads each earlier token's most recent state -- that of its final loop
 * d_s -- at every loop; with first-then-shared, loop 1 keeps a private slot and
 * loops 2..r_max share a second one, so loop 1 reads loop 1 and later loops
 * read loop d_s (a token that exits after loop 1 has its loop-1 state copied
 * into the shared slot by the same last-exited rule).
 *
 * Three independent executors are provided:
 *   orc_brute_force   -- no cache at all: every position is recomputed from the
 *                        token sequence, reading earlier tokens' K/V of loop
 *                        min(r, d_s) explicitly (no copies).
 *   orc_ref_sequence  -- one sequence with a dense per-position cache and
 *                        copy-on-exit.
 *   orc_prelude / orc_loop_step / orc_coda -- the batched stage operators over a
 *                        paged pool addressed through a page table, driven by a
 *                        scheduler in oracle/executor.py.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "cdb_oracle.h"

/* Accumulator type.  The oracle is fp64 (ORC_ACC = double).  Built with
 * -DORC_ACC=float it performs the same steps with every sum and product rounded
 * to fp32; the tests use that build only to measure how far an fp32
 * implementation of the same arithmetic drifts from fp64 on a given input. */
#ifndef ORC_ACC
#define ORC_ACC double
#endif
typedef ORC_ACC acc_t;
/* Summation order of the projections' dot products: 0 in index order (the
 * oracle), 1 in reverse index order, 2 in blocks of 32 terms whose partial sums
 * are then added in order.  Orders 1 and 2 are built only with fp32
 * accumulators, as further samples of how far an fp32 implementation that sums
 * in another order drifts from fp64. */
#ifndef ORC_SUM_ORDER
#define ORC_SUM_ORDER 0
#endif

/* ------------------------------------------------------------------ layouts */

/* The loop of an earlier token s (exit depth ds) whose K/V a token at loop r
 * attends to, by definition of the layout. */
static int read_loop(int layout, int r, int ds) {
    if (layout == ORC_KV_SHARED) return ds;
    if (layout == ORC_KV_FIRST_THEN_SHARED) return r == 1 ? 1 : ds;
    return r < ds ? r : ds;
}

/* The physical slot (0-based) that loop r writes in a dense per-token cache. */
static int write_slot(int layout, int r) {
    if (layout == ORC_KV_SHARED) return 0;
    if (layout == ORC_KV_FIRST_THEN_SHARED) return r == 1 ? 0 : 1;
    return r - 1;
}

/* ------------------------------------------------------------------ scalars */

static double bf(uint16_t bits) {
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

/* Round a value to bf16 (round to nearest, ties to even), going through fp32
 * first, as a device that computes in fp32 and stores bf16 does. */
static double to_bf16(double x) {
    float f = (float)x;
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7f800000u) == 0x7f800000u) return (double)f; /* inf / nan */
    uint32_t lsb = (u >> 16) & 1u;
    u = (u + 0x7fffu + lsb) & 0xffff0000u;
    memcpy(&f, &u, 4);
    return (double)f;
}

static double store(const orc_desc* m, double x) { return m->bf16_storage ? to_bf16(x) : x; }

static double silu(double x) { return x / (1.0 + exp(-x)); }
static double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

/* ------------------------------------------------------------------ vectors */

/* y = x / sqrt(mean(x^2) + eps); unit gains. */
static void rmsnorm(const double* x, int n, double eps, double* y) {
    acc_t ss = 0.0;
    for (int i = 0; i < n; ++i) ss += (acc_t)x[i] * (acc_t)x[i];
    acc_t inv = (acc_t)1.0 / (acc_t)sqrt((double)(ss / (acc_t)n + (acc_t)eps));
    for (int i = 0; i < n; ++i) y[i] = (acc_t)x[i] * inv;
}

/* y[o] = sum_i W[o][i] x[i] for a row-major bf16 matrix W [n_out][n_in]. */
static void matvec(const uint16_t* W, int n_out, int n_in, const double* x, double* y) {
    /* outputs are independent: for a large product called outside a parallel region (calls
     * with fewer rows than threads), they are shared among the threads; each output's sum is
     * the same either way */
#pragma omp parallel for schedule(static) if (!omp_in_parallel() && (long)n_out * n_in >= (1L << 20))
    for (int o = 0; o < n_out; ++o) {
        const uint16_t* w = W + (size_t)o * n_in;
        acc_t acc = 0.0;
#if ORC_SUM_ORDER == 1
        for (int i = n_in - 1; i >= 0; --i) acc += (acc_t)bf(w[i]) * (acc_t)x[i];
#elif ORC_SUM_ORDER == 2
        for (int b = 0; b < n_in; b += 32) {
            acc_t part = 0.0;
            for (int i = b; i < n_in && i < b + 32; ++i) part += (acc_t)bf(w[i]) * (acc_t)x[i];
            acc += part;
        }
#else
        for (int i = 0; i < n_in; ++i) acc += (acc_t)bf(w[i]) * (acc_t)x[i];
#endif
        y[o] = acc;
    }
}

/* Rotate-half RoPE applied to every head of v [n_heads * hd] at position pos:
 * pair (j, j + hd/2) is rotated by angle pos * base^(-2j/hd). */
static void rope(double* v, int n_heads, int hd, int pos, double base) {
    int half = hd / 2;
    for (int h = 0; h < n_heads; ++h) {
        double* x = v + (size_t)h * hd;
        for (int j = 0; j < half; ++j) {
            double ang = (double)pos * pow(base, -2.0 * j / hd);
            double c = cos(ang), s = sin(ang);
            double a = x[j], b = x[j + half];
            x[j] = a * c - b * s;
            x[j + half] = b * c + a * s;
        }
    }
}

/* One head: out = sum_s softmax_s(q . k_s / sqrt(hd)) v_s over n context rows.
 * kctx[s] / vctx[s] point at the head's hd values of position s. */
static void attend(const double* q, const double* const* kctx, const double* const* vctx, int n,
                   int hd, double* out) {
    acc_t* sc = (acc_t*)malloc(sizeof(acc_t) * (size_t)n);
    acc_t* o = (acc_t*)malloc(sizeof(acc_t) * (size_t)hd);
    acc_t scale = (acc_t)(1.0 / sqrt((double)hd));
    acc_t mx = -INFINITY;
    for (int s = 0; s < n; ++s) {
        acc_t dot = 0.0;
        for (int j = 0; j < hd; ++j) dot += (acc_t)q[j] * (acc_t)kctx[s][j];
        sc[s] = dot * scale;
        if (sc[s] > mx) mx = sc[s];
    }
    acc_t den = 0.0;
    for (int s = 0; s < n; ++s) {
        sc[s] = (acc_t)exp((double)(sc[s] - mx));
        den += sc[s];
    }
    for (int j = 0; j < hd; ++j) o[j] = 0.0;
    for (int s = 0; s < n; ++s) {
        acc_t p = sc[s] / den;
        for (int j = 0; j < hd; ++j) o[j] += p * (acc_t)vctx[s][j];
    }
    for (int j = 0; j < hd; ++j) out[j] = o[j];
    free(sc);
    free(o);
}

static const uint16_t* wt(const orc_weights* w, int layer, int which) {
    return w->layer[7 * layer + which];
}
enum { WQ = 0, WK, WV, WO, WG, WU, WD };

/* --------------------------------------------------------------- one layer */

/* First half of a pre-norm layer for one token: n = RMSNorm(h); q, k, v = W n;
 * RoPE(q, k; pos).  k and v are what the KV cache stores. */
static void layer_qkv(const orc_desc* m, const orc_weights* w, int layer, const double* h, int pos,
                      double* q, double* k, double* v) {
    int d = m->d;
    double* n = (double*)malloc(sizeof(double) * (size_t)d);
    rmsnorm(h, d, m->rms_eps, n);
    for (int i = 0; i < d; ++i) n[i] = store(m, n[i]);
    matvec(wt(w, layer, WQ), d, d, n, q);
    matvec(wt(w, layer, WK), d, d, n, k);
    matvec(wt(w, layer, WV), d, d, n, v);
    rope(q, m->n_heads, m->head_dim, pos, m->rope_base);
    rope(k, m->n_heads, m->head_dim, pos, m->rope_base);
    for (int i = 0; i < d; ++i) {
        k[i] = store(m, k[i]);
        v[i] = store(m, v[i]);
    }
    free(n);
}

/* Second half: attention of q over the n context rows (each row holds all
 * heads' K or V, d values), h += W_o o, then h += W_d (silu(W_g n') * W_u n')
 * with n' = RMSNorm(h). */
static void layer_rest(const orc_desc* m, const orc_weights* w, int layer, double* h, const double* q,
                       const double* const* krows, const double* const* vrows, int n) {
    int d = m->d, F = m->d_ff, H = m->n_heads, hd = m->head_dim;
    double* o = (double*)malloc(sizeof(double) * (size_t)d);
    double* t = (double*)malloc(sizeof(double) * (size_t)d);
    const double** kh = (const double**)malloc(sizeof(double*) * (size_t)n);
    const double** vh = (const double**)malloc(sizeof(double*) * (size_t)n);
    for (int hh = 0; hh < H; ++hh) {
        for (int s = 0; s < n; ++s) {
            kh[s] = krows[s] + (size_t)hh * hd;
            vh[s] = vrows[s] + (size_t)hh * hd;
        }
        attend(q + (size_t)hh * hd, kh, vh, n, hd, o + (size_t)hh * hd);
    }
    for (int i = 0; i < d; ++i) o[i] = store(m, o[i]);
    matvec(wt(w, layer, WO), d, d, o, t);
    for (int i = 0; i < d; ++i) h[i] = (acc_t)h[i] + (acc_t)t[i];

    double* g = (double*)malloc(sizeof(double) * (size_t)F);
    double* u = (double*)malloc(sizeof(double) * (size_t)F);
    rmsnorm(h, d, m->rms_eps, o);
    for (int i = 0; i < d; ++i) o[i] = store(m, o[i]);
    matvec(wt(w, layer, WG), F, d, o, g);
    matvec(wt(w, layer, WU), F, d, o, u);
    for (int i = 0; i < F; ++i) g[i] = store(m, (acc_t)silu(g[i]) * (acc_t)u[i]);
    matvec(wt(w, layer, WD), d, F, g, t);
    for (int i = 0; i < d; ++i) h[i] = (acc_t)h[i] + (acc_t)t[i];
    free(g);
    free(u);
    free(kh);
    free(vh);
    free(o);
    free(t);
}

/* Core input: the identity, or the adapter W_a [h; e] for input injection. */
static void core_input(const orc_desc* m, const orc_weights* w, const double* h, const double* e,
                       double* out) {
    int d = m->d;
    if (!m->injection) {
        memcpy(out, h, sizeof(double) * (size_t)d);
        return;
    }
    double* cat = (double*)malloc(sizeof(double) * 2 * (size_t)d);
    for (int i = 0; i < d; ++i) {
        cat[i] = store(m, h[i]);
        cat[d + i] = store(m, e[i]);
    }
    matvec(w->adapter, d, 2 * d, cat, out);
    free(cat);
}

/* Exit signal after a loop: sigmoid(w_exit . RMSNorm(h_new)) or ||h_new - h_old||_2. */
static double exit_score(const orc_desc* m, const orc_weights* w, const double* h_new,
                         const double* h_old) {
    int d = m->d;
    if (m->exit_kind == 1) {
        acc_t ss = 0.0;
        for (int i = 0; i < d; ++i) ss += ((acc_t)h_new[i] - (acc_t)h_old[i]) * ((acc_t)h_new[i] - (acc_t)h_old[i]);
        return sqrt((double)ss);
    }
    double* n = (double*)malloc(sizeof(double) * (size_t)d);
    rmsnorm(h_new, d, m->rms_eps, n);
    acc_t z = 0.0;
    for (int i = 0; i < d; ++i) z += (acc_t)bf(w->w_exit[i]) * (acc_t)n[i];
    free(n);
    return sigmoid(z);
}

/* logits = W_out RMSNorm(h); returns the argmax (lowest index on ties). */
static int32_t lm_head(const orc_desc* m, const orc_weights* w, const double* h, double* logits) {
    int d = m->d, V = m->vocab;
    double* n = (double*)malloc(sizeof(double) * (size_t)d);
    rmsnorm(h, d, m->rms_eps, n);
    for (int i = 0; i < d; ++i) n[i] = store(m, n[i]);
    matvec(w->lm_head, V, d, n, logits);
    free(n);
    int32_t best = 0;
    for (int i = 1; i < V; ++i)
        if (logits[i] > logits[best]) best = i;
    return best;
}

static void embed(const orc_desc* m, const orc_weights* w, int32_t tok, double* h) {
    for (int i = 0; i < m->d; ++i) h[i] = bf(w->embed[(size_t)tok * m->d + i]);
}

/* ======================================================== dense references */

/* Per-sequence KV store: prelude [T][P][2][d], core [T][r_max][C][2][d],
 * coda [T][Cd][2][d]. */
typedef struct {
    int T, d, P, C, Cd, R;
    double *pre, *core, *coda;
} dense_kv;

static double* dk_pre(dense_kv* kv, int t, int l, int kvi) {
    return kv->pre + ((((size_t)t * kv->P + l) * 2 + kvi) * kv->d);
}
static double* dk_core(dense_kv* kv, int t, int plane, int l, int kvi) {
    return kv->core + (((((size_t)t * kv->R + plane) * kv->C + l) * 2 + kvi) * kv->d);
}
static double* dk_coda(dense_kv* kv, int t, int l, int kvi) {
    return kv->coda + ((((size_t)t * kv->Cd + l) * 2 + kvi) * kv->d);
}

static void dense_alloc(dense_kv* kv, const orc_desc* m, int T) {
    kv->T = T;
    kv->d = m->d;
    kv->P = m->n_prelude;
    kv->C = m->n_core;
    kv->Cd = m->n_coda;
    kv->R = m->r_max;
    kv->pre = (double*)calloc((size_t)T * (kv->P ? kv->P : 1) * 2 * m->d, sizeof(double));
    kv->core = (double*)calloc((size_t)T * m->r_max * m->n_core * 2 * m->d, sizeof(double));
    kv->coda = (double*)calloc((size_t)T * (kv->Cd ? kv->Cd : 1) * 2 * m->d, sizeof(double));
}
static void dense_free(dense_kv* kv) {
    free(kv->pre);
    free(kv->core);
    free(kv->coda);
}

/* Run layer `layer` for token t whose context rows are given by pointer arrays
 * of length t+1 (the last entry is the token's own slot, written here). */
static void run_layer(const orc_desc* m, const orc_weights* w, int layer, double* h, int t, double* kslot,
                      double* vslot, const double** kr, const double** vr) {
    double* q = (double*)malloc(sizeof(double) * (size_t)m->d);
    layer_qkv(m, w, layer, h, t, q, kslot, vslot);
    kr[t] = kslot;
    vr[t] = vslot;
    layer_rest(m, w, layer, h, q, kr, vr, t + 1);
    free(q);
}

/* Tokens are processed in blocks: the first n_prefill tokens form one prefill
 * block, run loop by loop over the whole block (every block token finishes
 * loop r before any starts loop r + 1); each later token is a block of its
 * own.  Under the full layout the blocking changes nothing; under the shared
 * layouts it decides which state of an earlier token is the most recent one
 * when it is read (within a block: the loop being run). */
/* Threshold exit rule (Section 4.3; App. C.2): whether the score after loop r
 * meets the model's criterion -- gate score >= threshold, or for the
 * convergence criterion a distance below threshold from loop 2 on (the distance
 * after loop 1 compares the recurrent state with the prelude output). */
static int gate_meets(const orc_desc* m, int r, double score, double threshold) {
    if (m->exit_kind == 1) return r >= 2 && score < threshold;
    return score >= threshold;
}

/* depth: the exit depth of every token, or NULL for threshold exits (gate) of
 * the decode tokens t >= n_prefill; prefill tokens then run r_max loops. */
typedef struct {
    double threshold;
    int lookahead;
    int32_t* depth_out;
} gate_args;

static int ref_sequence(const orc_desc* m, const orc_weights* w, int32_t T, int32_t* tokens, int32_t n_given,
                        int32_t n_prefill, const int32_t* depth, const gate_args* gate, double* logits_out,
                        double* h_out, double* scores_out, double* core_kv_out) {
    int d = m->d, R = m->r_max;
    if (n_prefill < 0 || n_prefill > n_given || n_prefill > T) return ORC_ERR_ARG;
    if (depth)
        for (int t = 0; t < T; ++t)
            if (depth[t] < 1 || depth[t] > R) return ORC_ERR_ARG;
    dense_kv kv;
    dense_alloc(&kv, m, T);
    const int maxb = n_prefill > 1 ? n_prefill : 1;
    double* hb = (double*)malloc(sizeof(double) * (size_t)maxb * d); /* per block token: h */
    double* eb = (double*)malloc(sizeof(double) * (size_t)maxb * d); /* per block token: e */
    double* hp = (double*)malloc(sizeof(double) * (size_t)d);
    double* logits = (double*)malloc(sizeof(double) * (size_t)m->vocab);
    const double** kr = (const double**)malloc(sizeof(double*) * (size_t)T);
    const double** vr = (const double**)malloc(sizeof(double*) * (size_t)T);
    int32_t* dep = (int32_t*)malloc(sizeof(int32_t) * (size_t)(T > 0 ? T : 1)); /* exit depth, 0 while running */
    int* pending = (int*)calloc((size_t)(T > 0 ? T : 1), sizeof(int));       /* lookahead: exits after next loop */

    for (int b0 = 0; b0 < T;) {
        const int b1 = b0 < n_prefill ? n_prefill : b0 + 1; /* block [b0, b1) */
        for (int t = b0; t < b1; ++t) {
            double* h = hb + (size_t)(t - b0) * d;
            embed(m, w, tokens[t], h);
            for (int l = 0; l < m->n_prelude; ++l) {
                for (int s = 0; s < t; ++s) {
                    kr[s] = dk_pre(&kv, s, l, 0);
                    vr[s] = dk_pre(&kv, s, l, 1);
                }
                run_layer(m, w, l, h, t, dk_pre(&kv, t, l, 0), dk_pre(&kv, t, l, 1), kr, vr);
            }
            memcpy(eb + (size_t)(t - b0) * d, h, sizeof(double) * (size_t)d);
        }
        for (int t = b0; t < b1; ++t) dep[t] = 0;
        for (int r = 1; r <= R; ++r) {
            const int slot = write_slot(m->kv_layout, r);
            for (int t = b0; t < b1; ++t) {
                if (dep[t]) continue; /* exited */
                double* h = hb + (size_t)(t - b0) * d;
                memcpy(hp, h, sizeof(double) * (size_t)d);
                core_input(m, w, hp, eb + (size_t)(t - b0) * d, h);
                for (int l = 0; l < m->n_core; ++l) {
                    for (int s = 0; s < t; ++s) {
                        kr[s] = dk_core(&kv, s, slot, l, 0);
                        vr[s] = dk_core(&kv, s, slot, l, 1);
                    }
                    run_layer(m, w, m->n_prelude + l, h, t, dk_core(&kv, t, slot, l, 0),
                              dk_core(&kv, t, slot, l, 1), kr, vr);
                }
                const double sc = exit_score(m, w, h, hp);
                if (scores_out) scores_out[(size_t)t * R + (r - 1)] = sc;
                /* is loop r the token's last? */
                int last;
                if (depth) {
                    last = r == depth[t];
                } else if (t < n_prefill) {
                    last = r == R;
                } else if (gate->lookahead) {
                    last = r == R || pending[t];
                    pending[t] = !last && gate_meets(m, r, sc, gate->threshold);
                } else {
                    last = r == R || gate_meets(m, r, sc, gate->threshold);
                }
                if (last) dep[t] = r;
            }
            /* last-exited cache: a token that exits after loop r gets the slots
             * of loops r+1..R filled with a copy of the slot of loop r (nothing
             * to do where they are the same slot) */
            for (int t = b0; t < b1; ++t) {
                if (dep[t] != r) continue;
                for (int r2 = r + 1; r2 <= R; ++r2) {
                    const int dst = write_slot(m->kv_layout, r2);
                    if (dst == slot) continue;
                    for (int l = 0; l < m->n_core; ++l)
                        for (int kvi = 0; kvi < 2; ++kvi)
                            memcpy(dk_core(&kv, t, dst, l, kvi), dk_core(&kv, t, slot, l, kvi),
                                   sizeof(double) * (size_t)d);
                }
            }
        }
        for (int t = b0; t < b1; ++t) {
            double* h = hb + (size_t)(t - b0) * d;
            if (scores_out)
                for (int r = dep[t] + 1; r <= R; ++r) scores_out[(size_t)t * R + (r - 1)] = NAN;
            if (gate && gate->depth_out) gate->depth_out[t] = dep[t];
            if (h_out) memcpy(h_out + (size_t)t * d, h, sizeof(double) * (size_t)d);
            for (int l = 0; l < m->n_coda; ++l) {
                for (int s = 0; s < t; ++s) {
                    kr[s] = dk_coda(&kv, s, l, 0);
                    vr[s] = dk_coda(&kv, s, l, 1);
                }
                run_layer(m, w, m->n_prelude + m->n_core + l, h, t, dk_coda(&kv, t, l, 0), dk_coda(&kv, t, l, 1),
                          kr, vr);
            }
            int32_t nxt = lm_head(m, w, h, logits);
            if (logits_out) memcpy(logits_out + (size_t)t * m->vocab, logits, sizeof(double) * (size_t)m->vocab);
            if (t + 1 < T && t + 1 >= n_given) tokens[t + 1] = nxt;
        }
        b0 = b1;
    }
    if (core_kv_out)
        memcpy(core_kv_out, kv.core, sizeof(double) * (size_t)T * R * m->n_core * 2 * d);
    free(kr);
    free(vr);
    free(hb);
    free(eb);
    free(hp);
    free(logits);
    free(dep);
    free(pending);
    dense_free(&kv);
    return ORC_OK;
}

int orc_ref_sequence(const orc_desc* m, const orc_weights* w, int32_t T, int32_t* tokens, int32_t n_given,
                     int32_t n_prefill, const int32_t* depth, double* logits_out, double* h_out, double* scores_out,
                     double* core_kv_out) {
    if (!depth) return ORC_ERR_ARG;
    return ref_sequence(m, w, T, tokens, n_given, n_prefill, depth, NULL, logits_out, h_out, scores_out,
                        core_kv_out);
}

/* One loop step's threshold decisions for n rows at loop index c[i] with exit
 * score score[i] (the state after loop c[i] + 1): exit_mask[i] = this loop is
 * the token's last; exit_next[i] = a continuing token's next loop will be its
 * last.  pending[i] (in/out) carries the lookahead decision of the row's token
 * between steps. */
int orc_gate_decide(const orc_desc* m, int32_t n, const int32_t* c, const double* score, double threshold,
                    int32_t lookahead, uint8_t* pending, uint8_t* exit_mask, uint8_t* exit_next) {
    const int R = m->r_max;
    for (int i = 0; i < n; ++i) {
        if (c[i] < 0 || c[i] >= R) return ORC_ERR_ARG;
        const int r = c[i] + 1;
        const int meets = gate_meets(m, r, score[i], threshold);
        int last, next;
        if (lookahead) {
            last = r == R || pending[i];
            next = !last && (meets || r + 1 == R);
            pending[i] = (uint8_t)next;
        } else {
            last = r == R || meets;
            next = !last && r + 1 == R;
        }
        exit_mask[i] = (uint8_t)last;
        exit_next[i] = (uint8_t)next;
    }
    return ORC_OK;
}

int orc_ref_sequence_gated(const orc_desc* m, const orc_weights* w, int32_t T, int32_t* tokens, int32_t n_given,
                           int32_t n_prefill, double threshold, int32_t lookahead, int32_t* depth_out,
                           double* logits_out, double* h_out, double* scores_out) {
    gate_args g = {threshold, lookahead != 0, depth_out};
    return ref_sequence(m, w, T, tokens, n_given, n_prefill, NULL, &g, logits_out, h_out, scores_out, NULL);
}

/* No cache: for every position t the whole prefix 0..t is recomputed from the
 * tokens; a token at loop r reads earlier token s's K/V of loop
 * read_loop(layout, r, d_s) -- min(r, d_s) for the full layout -- indexed
 * directly by loop (no copy-on-exit, no slot sharing).  Within the prefill
 * block (both tokens below n_prefill) s's most recent state at loop r is that
 * of loop min(r, d_s) under every layout. */
int orc_brute_force(const orc_desc* m, const orc_weights* w, int32_t T, const int32_t* tokens, int32_t n_prefill,
                    const int32_t* depth, double* logits_out, double* h_out, double* scores_out) {
    int d = m->d, R = m->r_max;
    if (n_prefill < 0 || n_prefill > T) return ORC_ERR_ARG;
    for (int t = 0; t < T; ++t)
        if (depth[t] < 1 || depth[t] > R) return ORC_ERR_ARG;
    double* h = (double*)malloc(sizeof(double) * (size_t)d);
    double* e = (double*)malloc(sizeof(double) * (size_t)d);
    double* hp = (double*)malloc(sizeof(double) * (size_t)d);
    double* logits = (double*)malloc(sizeof(double) * (size_t)m->vocab);
    const double** kr = (const double**)malloc(sizeof(double*) * (size_t)T);
    const double** vr = (const double**)malloc(sizeof(double*) * (size_t)T);

    for (int last = 0; last < T; ++last) {
        dense_kv kv; /* written only at planes r-1 < depth[s]; never copied */
        dense_alloc(&kv, m, last + 1);
        for (int t = 0; t <= last; ++t) {
            embed(m, w, tokens[t], h);
            for (int l = 0; l < m->n_prelude; ++l) {
                for (int s = 0; s < t; ++s) {
                    kr[s] = dk_pre(&kv, s, l, 0);
                    vr[s] = dk_pre(&kv, s, l, 1);
                }
                run_layer(m, w, l, h, t, dk_pre(&kv, t, l, 0), dk_pre(&kv, t, l, 1), kr, vr);
            }
            memcpy(e, h, sizeof(double) * (size_t)d);
            for (int r = 1; r <= depth[t]; ++r) {
                memcpy(hp, h, sizeof(double) * (size_t)d);
                core_input(m, w, hp, e, h);
                for (int l = 0; l < m->n_core; ++l) {
                    for (int s = 0; s < t; ++s) {
                        const int rs = t < n_prefill ? (r < depth[s] ? r : depth[s])
                                                     : read_loop(m->kv_layout, r, depth[s]);
                        kr[s] = dk_core(&kv, s, rs - 1, l, 0);
                        vr[s] = dk_core(&kv, s, rs - 1, l, 1);
                    }
                    run_layer(m, w, m->n_prelude + l, h, t, dk_core(&kv, t, r - 1, l, 0),
                              dk_core(&kv, t, r - 1, l, 1), kr, vr);
                }
                if (t == last && scores_out) scores_out[(size_t)t * R + (r - 1)] = exit_score(m, w, h, hp);
            }
            if (t == last && scores_out)
                for (int r = depth[t] + 1; r <= R; ++r) scores_out[(size_t)t * R + (r - 1)] = NAN;
            if (t == last && h_out) memcpy(h_out + (size_t)t * d, h, sizeof(double) * (size_t)d);
            for (int l = 0; l < m->n_coda; ++l) {
                for (int s = 0; s < t; ++s) {
                    kr[s] = dk_coda(&kv, s, l, 0);
                    vr[s] = dk_coda(&kv, s, l, 1);
                }
                run_layer(m, w, m->n_prelude + m->n_core + l, h, t, dk_coda(&kv, t, l, 0),
                          dk_coda(&kv, t, l, 1), kr, vr);
            }
            if (t == last) {
                lm_head(m, w, h, logits);
                if (logits_out)
                    memcpy(logits_out + (size_t)t * m->vocab, logits, sizeof(double) * (size_t)m->vocab);
            }
        }
        dense_free(&kv);
    }
    free(kr);
    free(vr);
    free(h);
    free(e);
    free(hp);
    free(logits);
    return ORC_OK;
}

/* ==================================================== paged stage operators */

/* Page table: [max_seqs][r_max + 2][max_pages] int32.  Plane 0 addresses the
 * prelude pool, planes 1..r_max the core pool (core loop index c uses plane
 * c + 1), plane r_max + 1 the coda pool; -1 is unmapped.  A page holds 16
 * tokens of every layer of its stage: [layer][K,V][head][token][head_dim]. */
#define ORC_PAGE 16

static int32_t pt_get(const orc_paged* p, int seq, int plane, int page) {
    if (seq < 0 || seq >= p->max_seqs || page < 0 || page >= p->max_pages) return -1;
    return p->page_table[((size_t)seq * (p->r_max + 2) + plane) * p->max_pages + page];
}

/* Address of the K (kvi = 0) or V (kvi = 1) entry of head hh, token pos, layer
 * `l` (index inside the stage) for sequence seq in a plane; NULL if unmapped. */
static double* kv_at(const orc_paged* p, const orc_desc* m, int plane, int seq, int pos, int l, int kvi,
                     int hh) {
    int32_t pg = pt_get(p, seq, plane, pos / ORC_PAGE);
    if (pg < 0) return NULL;
    double* pool;
    int nl, npages;
    if (plane == 0) {
        pool = p->pre_pool;
        nl = m->n_prelude;
        npages = p->pre_pages;
    } else if (plane == m->r_max + 1) {
        pool = p->coda_pool;
        nl = m->n_coda;
        npages = p->coda_pages;
    } else {
        pool = p->core_pool;
        nl = m->n_core;
        npages = p->core_pages;
    }
    if (pg >= npages) return NULL;
    int H = m->n_heads, hd = m->head_dim;
    size_t page_elems = (size_t)nl * 2 * H * ORC_PAGE * hd;
    size_t off = (size_t)pg * page_elems + ((((size_t)l * 2 + kvi) * H + hh) * ORC_PAGE + (pos % ORC_PAGE)) * hd;
    return pool + off;
}

/* Run stage layers [first, first + nl) for all rows, layer by layer: every row
 * writes its K/V for a layer before any row attends at that layer, so rows of
 * one sequence at consecutive positions see each other causally.  Rows run in
 * parallel when there are at least as many as threads; fewer run one after the
 * other, with each product's outputs shared among the threads (matvec). */
static int stage_layers(const orc_desc* m, const orc_weights* w, const orc_paged* p, int plane, int first,
                        int nl, int n, const int32_t* seq, const int32_t* pos, double* hs) {
    int d = m->d, H = m->n_heads, hd = m->head_dim;
    double* q = (double*)malloc(sizeof(double) * (size_t)n * d);
    int err = ORC_OK;
    for (int l = 0; l < nl && err == ORC_OK; ++l) {
        /* each row writes only its own K/V slot, so rows run independently */
#pragma omp parallel for schedule(dynamic, 1) if (n >= omp_get_max_threads())
        for (int i = 0; i < n; ++i) {
            double* k = (double*)malloc(sizeof(double) * (size_t)d);
            double* v = (double*)malloc(sizeof(double) * (size_t)d);
            layer_qkv(m, w, first + l, hs + (size_t)i * d, pos[i], q + (size_t)i * d, k, v);
            int bad = 0;
            for (int hh = 0; hh < H && !bad; ++hh) {
                double* ks = kv_at(p, m, plane, seq[i], pos[i], l, 0, hh);
                double* vs = kv_at(p, m, plane, seq[i], pos[i], l, 1, hh);
                if (!ks || !vs) {
                    bad = 1;
                } else {
                    memcpy(ks, k + (size_t)hh * hd, sizeof(double) * (size_t)hd);
                    memcpy(vs, v + (size_t)hh * hd, sizeof(double) * (size_t)hd);
                }
            }
            if (bad) {
#pragma omp critical
                err = ORC_ERR_UNMAPPED;
            }
            free(k);
            free(v);
        }
        if (err != ORC_OK) break;
#pragma omp parallel for schedule(dynamic, 1) if (n >= omp_get_max_threads())
        for (int i = 0; i < n; ++i) {
            int ctx = pos[i] + 1;
            double* kbuf = (double*)malloc(sizeof(double) * (size_t)ctx * d);
            double* vbuf = (double*)malloc(sizeof(double) * (size_t)ctx * d);
            const double** kr = (const double**)malloc(sizeof(double*) * (size_t)ctx);
            const double** vr = (const double**)malloc(sizeof(double*) * (size_t)ctx);
            int bad = 0;
            for (int s = 0; s < ctx && !bad; ++s) {
                for (int hh = 0; hh < H; ++hh) {
                    double* ks = kv_at(p, m, plane, seq[i], s, l, 0, hh);
                    double* vs = kv_at(p, m, plane, seq[i], s, l, 1, hh);
                    if (!ks || !vs) {
                        bad = 1;
                        break;
                    }
                    memcpy(kbuf + (size_t)s * d + (size_t)hh * hd, ks, sizeof(double) * (size_t)hd);
                    memcpy(vbuf + (size_t)s * d + (size_t)hh * hd, vs, sizeof(double) * (size_t)hd);
                }
                kr[s] = kbuf + (size_t)s * d;
                vr[s] = vbuf + (size_t)s * d;
            }
            if (bad) {
#pragma omp critical
                err = ORC_ERR_UNMAPPED;
            } else {
                layer_rest(m, w, first + l, hs + (size_t)i * d, q + (size_t)i * d, kr, vr, ctx);
            }
            free(kbuf);
            free(vbuf);
            free(kr);
            free(vr);
        }
    }
    free(q);
    return err;
}

int orc_prelude(const orc_desc* m, const orc_weights* w, const orc_paged* p, double* state_h, double* state_e,
                int32_t n_slots, int32_t n, const int32_t* slot, const int32_t* seq, const int32_t* pos,
                const int32_t* tokens) {
    int d = m->d;
    for (int i = 0; i < n; ++i)
        if (slot[i] < 0 || slot[i] >= n_slots || tokens[i] < 0 || tokens[i] >= m->vocab || pos[i] < 0)
            return ORC_ERR_ARG;
    double* hs = (double*)malloc(sizeof(double) * (size_t)(n ? n : 1) * d);
    for (int i = 0; i < n; ++i) embed(m, w, tokens[i], hs + (size_t)i * d);
    int err = stage_layers(m, w, p, 0, 0, m->n_prelude, n, seq, pos, hs);
    if (err == ORC_OK)
        for (int i = 0; i < n; ++i) {
            memcpy(state_h + (size_t)slot[i] * d, hs + (size_t)i * d, sizeof(double) * (size_t)d);
            if (m->injection && state_e)
                memcpy(state_e + (size_t)slot[i] * d, hs + (size_t)i * d, sizeof(double) * (size_t)d);
        }
    free(hs);
    return err;
}

int orc_exit_compact(int32_t n, const int32_t* c, const int32_t* depth, int32_t r_max, uint8_t* exit_mask,
                     int32_t* cont, int32_t* exited, int32_t* counts) {
    int nc = 0, ne = 0;
    for (int i = 0; i < n; ++i)
        if (depth[i] < 1 || depth[i] > r_max || c[i] < 0 || c[i] >= depth[i]) return ORC_ERR_ARG;
    for (int i = 0; i < n; ++i) {
        int ex = (c[i] + 1 == depth[i]);
        exit_mask[i] = (uint8_t)ex;
        if (ex)
            exited[ne++] = i;
        else
            cont[nc++] = i;
    }
    counts[0] = nc;
    counts[1] = ne;
    return ORC_OK;
}

int orc_loop_step(const orc_desc* m, const orc_weights* w, const orc_paged* p, double* state_h,
                  const double* state_e, int32_t n_slots, int32_t n, const int32_t* slot, const int32_t* seq,
                  const int32_t* pos, const int32_t* c, const int32_t* depth, double* score, uint8_t* exit_mask,
                  int32_t* cont, int32_t* exited, int32_t* counts) {
    int d = m->d, H = m->n_heads, hd = m->head_dim;
    for (int i = 0; i < n; ++i)
        if (slot[i] < 0 || slot[i] >= n_slots || pos[i] < 0) return ORC_ERR_ARG;
    int err = orc_exit_compact(n, c, depth, m->r_max, exit_mask, cont, exited, counts);
    if (err != ORC_OK) return err;
    /* rows of one loop step may sit at different loop indices; each row's own
     * plane is c + 1, so the layers run per distinct plane */
    double* hs = (double*)malloc(sizeof(double) * (size_t)(n ? n : 1) * d);
    double* h0 = (double*)malloc(sizeof(double) * (size_t)(n ? n : 1) * d);
    for (int i = 0; i < n; ++i) {
        memcpy(h0 + (size_t)i * d, state_h + (size_t)slot[i] * d, sizeof(double) * (size_t)d);
        core_input(m, w, h0 + (size_t)i * d, m->injection ? state_e + (size_t)slot[i] * d : NULL,
                   hs + (size_t)i * d);
    }
    int32_t* sub_seq = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n ? n : 1));
    int32_t* sub_pos = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n ? n : 1));
    int32_t* sub_idx = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n ? n : 1));
    double* sub_h = (double*)malloc(sizeof(double) * (size_t)(n ? n : 1) * d);
    for (int cc = 0; cc < m->r_max && err == ORC_OK; ++cc) {
        int k = 0;
        for (int i = 0; i < n; ++i)
            if (c[i] == cc) {
                sub_idx[k] = i;
                sub_seq[k] = seq[i];
                sub_pos[k] = pos[i];
                memcpy(sub_h + (size_t)k * d, hs + (size_t)i * d, sizeof(double) * (size_t)d);
                ++k;
            }
        if (!k) continue;
        err = stage_layers(m, w, p, cc + 1, m->n_prelude, m->n_core, k, sub_seq, sub_pos, sub_h);
        for (int j = 0; j < k; ++j)
            memcpy(hs + (size_t)sub_idx[j] * d, sub_h + (size_t)j * d, sizeof(double) * (size_t)d);
    }
    if (err == ORC_OK) {
        for (int i = 0; i < n; ++i) {
            score[i] = exit_score(m, w, hs + (size_t)i * d, h0 + (size_t)i * d);
            memcpy(state_h + (size_t)slot[i] * d, hs + (size_t)i * d, sizeof(double) * (size_t)d);
        }
        /* copy-on-exit: an exiting row's K/V of its last plane fills the
         * deeper planes at its position, every core layer and head */
        for (int j = 0; j < counts[1] && err == ORC_OK; ++j) {
            int i = exited[j];
            for (int pl = depth[i] + 1; pl <= m->r_max; ++pl)
                for (int l = 0; l < m->n_core; ++l)
                    for (int kvi = 0; kvi < 2; ++kvi)
                        for (int hh = 0; hh < H; ++hh) {
                            double* src = kv_at(p, m, depth[i], seq[i], pos[i], l, kvi, hh);
                            double* dst = kv_at(p, m, pl, seq[i], pos[i], l, kvi, hh);
                            if (!src || !dst) {
                                err = ORC_ERR_UNMAPPED;
                                break;
                            }
                            if (dst != src) memcpy(dst, src, sizeof(double) * (size_t)hd);
                        }
        }
    }
    free(sub_seq);
    free(sub_pos);
    free(sub_idx);
    free(sub_h);
    free(hs);
    free(h0);
    return err;
}

int orc_coda(const orc_desc* m, const orc_weights* w, const orc_paged* p, const double* state_h,
             int32_t n_slots, int32_t n, const int32_t* slot, const int32_t* seq, const int32_t* pos,
             double* logits, int32_t* next_ids) {
    int d = m->d;
    for (int i = 0; i < n; ++i)
        if (slot[i] < 0 || slot[i] >= n_slots || pos[i] < 0) return ORC_ERR_ARG;
    double* hs = (double*)malloc(sizeof(double) * (size_t)(n ? n : 1) * d);
    for (int i = 0; i < n; ++i)
        memcpy(hs + (size_t)i * d, state_h + (size_t)slot[i] * d, sizeof(double) * (size_t)d);
    int err = stage_layers(m, w, p, m->r_max + 1, m->n_prelude + m->n_core, m->n_coda, n, seq, pos, hs);
    if (err == ORC_OK) {
#pragma omp parallel for schedule(dynamic, 1) if (n >= omp_get_max_threads())
        for (int i = 0; i < n; ++i)
            next_ids[i] = lm_head(m, w, hs + (size_t)i * d, logits + (size_t)i * m->vocab);
    }
    free(hs);
    return err;
}

/* Small exported pieces, so tests can pin them against closed forms. */
void orc_rmsnorm(const double* x, int32_t n, double eps, double* y) { rmsnorm(x, n, eps, y); }
void orc_rope(double* v, int32_t n_heads, int32_t hd, int32_t pos, double base) { rope(v, n_heads, hd, pos, base); }
void orc_attend(const double* q, const double* k, const double* v, int32_t n, int32_t hd, double* out) {
    const double** kr = (const double**)malloc(sizeof(double*) * (size_t)(n ? n : 1));
    const double** vr = (const double**)malloc(sizeof(double*) * (size_t)(n ? n : 1));
    for (int s = 0; s < n; ++s) {
        kr[s] = k + (size_t)s * hd;
        vr[s] = v + (size_t)s * hd;
    }
    attend(q, kr, vr, n, hd, out);
    free(kr);
    free(vr);
}
double orc_silu(double x) { return silu(x); }
double orc_to_bf16(double x) { return to_bf16(x); }

/* Threads of the OpenMP loops over independent rows (timing runs only). */
int orc_set_threads(int n) {
    if (n > 0) omp_set_num_threads(n);
    return omp_get_max_threads();
}
