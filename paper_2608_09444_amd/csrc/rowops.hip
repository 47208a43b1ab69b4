// Row-wise kernels of the stage calls: gather and validation, RMSNorm, embedding,
// state write-back, exit score and decision, stable compaction, copy-on-exit,
// argmax, weight packing and workspace initialisation.  All are bandwidth- or
// latency-bound; accesses are 16-byte coalesced where the data allows.
#include "cdb_internal.h"

namespace cdb {

// Block-wide fp32 sum (blockDim.x a multiple of 64, at most 1024); result
// broadcast to all threads, summed in wave order.
__device__ __forceinline__ float block_sum(float v, float* red) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[w] = v;
    __syncthreads();
    float t = 0.f;
    for (int i = 0; i < nw; ++i) t += red[i];
    return t;
}

// RoPE table of one row: (cos, sin) of pos * base^(-2j/hd) for j < hd/2, fp64 angles.
__device__ __forceinline__ void rope_row(int pos, int hd, float base, float2* out) {
    for (int j = threadIdx.x; j < hd / 2; j += blockDim.x) {
        const double ang = (double)pos * pow((double)base, -2.0 * j / hd);
        double sn, cs;
        sincos(ang, &sn, &cs);
        out[j] = make_float2((float)cs, (float)sn);
    }
}

// ------------------------------------------------------------------ row order
// order[rank] = row, ranked by descending position (ties by row index), for
// the paged attention's row pairing.  Run by every thread of one workgroup;
// M <= kMaxRows.  The stage calls run it in the first workgroup of their
// row-entry kernel instead of a launch of its own.
__device__ __forceinline__ void row_order_block(const int32_t* __restrict__ pos, int M, int32_t* __restrict__ order) {
    __shared__ int s_pos[kMaxRows];
    for (int i = threadIdx.x; i < M; i += blockDim.x) s_pos[i] = pos[i];
    __syncthreads();
    for (int i = threadIdx.x; i < M; i += blockDim.x) {
        const int pi = s_pos[i];
        int rank = 0;
        for (int j = 0; j < M; ++j) {
            const int pj = s_pos[j];
            rank += (pj > pi) || (pj == pi && j < i);
        }
        order[rank] = i;
    }
}

// ------------------------------------------------------------------ gather
// h[i] = state.h[slot[i]] (zeros with the adapter); h_in[i] = state.h[slot[i]]
// (exit score of the L2 criterion); xcat[i] = bf16([h; e]) for the
// input-injection adapter.  Validates the row.
// kvpid[i]: the page of the stage pool that receives row i's K/V (plane c+1 of
// the core, or the stage's fixed plane); -1 when the stage has no layers.
__device__ __forceinline__ void write_page(const KvTarget& kt, int i, int sq, int ps, const int32_t* c_row,
                                           int32_t* kvpid, int* err) {
    int pid = -1;
    if (kt.n_layers > 0) {
        // a row's own loop index selects a core plane, 1..r_max; a c outside
        // [0, r_max) must not resolve the prelude or coda plane's page
        const int plane = c_row ? c_row[i] + 1 : kt.plane_fixed;
        const bool plane_ok = c_row ? (plane >= 1 && plane <= kt.n_planes - 2) : (plane >= 0 && plane < kt.n_planes);
        const int pg = ps >= 0 ? ps / kPage : -1;
        if (sq >= 0 && sq < kt.max_seqs && pg >= 0 && pg < kt.max_pages && plane_ok)
            pid = kt.page_table[((size_t)sq * kt.n_planes + plane) * kt.max_pages + pg];
        if (pid < 0 || pid >= kt.n_pages) {
            set_err(err, CDB_DEV_UNMAPPED_PAGE);
            pid = -1;
        }
    }
    kvpid[i] = pid;
}

__global__ __launch_bounds__(256) void k_gather(int d, int r_max, int n_slots, int max_seqs, int max_pos, int hd,
                                                float base, const int32_t* __restrict__ slot,
                                                const int32_t* __restrict__ seq, const int32_t* __restrict__ pos,
                                                const int32_t* __restrict__ c, const int32_t* __restrict__ depth,
                                                const float* __restrict__ sh, const float* __restrict__ se,
                                                float* __restrict__ h, float* __restrict__ h_in,
                                                uint16_t* __restrict__ xcat, float2* __restrict__ rope, KvTarget kt,
                                                int32_t* __restrict__ kvpid, int32_t* __restrict__ order, float eps,
                                                uint16_t* __restrict__ xn, int* err, const int32_t* __restrict__ dn) {
    __shared__ float red[4];
    const int i = blockIdx.x;
    const int n = live_rows(dn, gridDim.x);
    if (order && i == 0 && gridDim.x <= kMaxRows) row_order_block(pos, n, order);
    if (i >= n) return;
    const int sl = slot[i];
    rope_row(pos[i], hd, base, rope + (size_t)i * (hd / 2));
    if (threadIdx.x == 0) {
        if (depth ? (depth[i] < 1 || depth[i] > r_max || c[i] < 0 || c[i] >= depth[i]) : (c[i] < 0 || c[i] >= r_max))
            set_err(err, CDB_DEV_BAD_DEPTH);
        if (sl < 0 || sl >= n_slots || seq[i] < 0 || seq[i] >= max_seqs || pos[i] < 0 || pos[i] >= max_pos)
            set_err(err, CDB_DEV_BAD_INDEX);
        write_page(kt, i, seq[i], pos[i], c, kvpid, err);
    }
    const bool ok = sl >= 0 && sl < n_slots;
    for (int k = threadIdx.x * 4; k < d; k += 256 * 4) {
        float4 v = ok ? *reinterpret_cast<const float4*>(sh + (size_t)sl * d + k) : make_float4(0.f, 0.f, 0.f, 0.f);
        // with the adapter, h starts at zero: the adapter's split-K partials are added to it
        *reinterpret_cast<float4*>(h + (size_t)i * d + k) = xcat ? make_float4(0.f, 0.f, 0.f, 0.f) : v;
        *reinterpret_cast<float4*>(h_in + (size_t)i * d + k) = v;
        if (xcat) {  // adapter input [h; e], fragment layout with K = 2d
            float4 e = ok ? *reinterpret_cast<const float4*>(se + (size_t)sl * d + k) : make_float4(0.f, 0.f, 0.f, 0.f);
            uint2 ph, pe;
            ph.x = pack_bf16(v.x, v.y);
            ph.y = pack_bf16(v.z, v.w);
            pe.x = pack_bf16(e.x, e.y);
            pe.y = pack_bf16(e.z, e.w);
            *reinterpret_cast<uint2*>(xcat + frag_index(i, k, 2 * d)) = ph;
            *reinterpret_cast<uint2*>(xcat + frag_index(i, d + k, 2 * d)) = pe;
        }
    }
    if (xn) {  // no adapter: the first core layer's input bf16(RMSNorm(h)), fragment layout
        float ss = 0.f;
        for (int k = threadIdx.x * 4; k < d; k += 256 * 4) {
            const float4 v = *reinterpret_cast<const float4*>(h + (size_t)i * d + k);
            ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
        }
        ss = block_sum(ss, red);
        const float inv = 1.0f / sqrtf(ss / d + eps);
        for (int k = threadIdx.x * 4; k < d; k += 256 * 4) {
            const float4 v = *reinterpret_cast<const float4*>(h + (size_t)i * d + k);
            uint2 pk;
            pk.x = pack_bf16(v.x * inv, v.y * inv);
            pk.y = pack_bf16(v.z * inv, v.w * inv);
            *reinterpret_cast<uint2*>(xn + frag_index(i, k, d)) = pk;
        }
    }
}

// h[i] = state.h[slot[i]] (coda input)
__global__ __launch_bounds__(256) void k_load_state(int d, int n_slots, int hd, float base,
                                                    const int32_t* __restrict__ slot, const int32_t* __restrict__ seq,
                                                    const int32_t* __restrict__ pos, KvTarget kt,
                                                    const float* __restrict__ sh, float* __restrict__ h,
                                                    float2* __restrict__ rope, int32_t* __restrict__ kvpid,
                                                    int32_t* __restrict__ order, int* err,
                                                    const int32_t* __restrict__ dn) {
    const int i = blockIdx.x;
    const int n = live_rows(dn, gridDim.x);
    if (order && i == 0 && gridDim.x <= kMaxRows) row_order_block(pos, n, order);
    if (i >= n) return;
    const int sl = slot[i];
    rope_row(pos[i], hd, base, rope + (size_t)i * (hd / 2));
    const bool ok = sl >= 0 && sl < n_slots;
    if (threadIdx.x == 0) {
        if (!ok) set_err(err, CDB_DEV_BAD_INDEX);
        write_page(kt, i, seq[i], pos[i], nullptr, kvpid, err);
    }
    for (int k = threadIdx.x * 4; k < d; k += 1024)
        *reinterpret_cast<float4*>(h + (size_t)i * d + k) =
            ok ? *reinterpret_cast<const float4*>(sh + (size_t)sl * d + k) : make_float4(0.f, 0.f, 0.f, 0.f);
}

// ------------------------------------------------------------------ residual + RMSNorm
// h[i] += sum_s part[s][i] (split order 0..S-1); out[i] = bf16(h[i] / sqrt(mean(h[i]^2) + eps)),
// unit gains.  Row i is one workgroup; each thread keeps its NV runs of 4
// values in registers between the sum and the normalisation, and issues the
// partial loads of up to 4 splits at once.
template <int NV>
__global__ __launch_bounds__(1024) void k_resid_norm(float* __restrict__ h, const float* __restrict__ part, int S, int M,
                                                     int d, float eps, uint16_t* __restrict__ out,
                                                     const int32_t* __restrict__ dn) {
    __shared__ float red[16];
    const int i = blockIdx.x;
    if (i >= live_rows(dn, M)) return;
    float* x = h + (size_t)i * d;
    float4 v[NV];
    float ss = 0.f;
#pragma unroll
    for (int u = 0; u < NV; ++u) {
        const int k = (threadIdx.x + u * blockDim.x) * 4;
        if (k >= d) continue;
        v[u] = *reinterpret_cast<const float4*>(x + k);
        for (int s0 = 0; s0 < S; s0 += 4) {
            float4 p[4];
#pragma unroll
            for (int t = 0; t < 4; ++t)
                if (s0 + t < S) p[t] = *reinterpret_cast<const float4*>(part + ((size_t)(s0 + t) * M + i) * d + k);
#pragma unroll
            for (int t = 0; t < 4; ++t)
                if (s0 + t < S) {
                    v[u].x += p[t].x;
                    v[u].y += p[t].y;
                    v[u].z += p[t].z;
                    v[u].w += p[t].w;
                }
        }
        if (S > 0) *reinterpret_cast<float4*>(x + k) = v[u];
        ss += v[u].x * v[u].x + v[u].y * v[u].y + v[u].z * v[u].z + v[u].w * v[u].w;
    }
    if (!out) return;
    ss = block_sum(ss, red);
    const float inv = 1.0f / sqrtf(ss / d + eps);
#pragma unroll
    for (int u = 0; u < NV; ++u) {
        const int k = (threadIdx.x + u * blockDim.x) * 4;
        if (k >= d) continue;
        uint2 pk;
        pk.x = pack_bf16(v[u].x * inv, v[u].y * inv);
        pk.y = pack_bf16(v[u].z * inv, v[u].w * inv);
        *reinterpret_cast<uint2*>(out + frag_index(i, k, d)) = pk;  // 4 consecutive k share one 8-slot run
    }
}

// ------------------------------------------------------------------ embedding
__global__ __launch_bounds__(256) void k_embed(int d, int vocab, int n_slots, int max_seqs, int max_pos, int hd,
                                               float base, const uint16_t* __restrict__ E,
                                               const int32_t* __restrict__ tok, const int32_t* __restrict__ slot,
                                               const int32_t* __restrict__ seq, const int32_t* __restrict__ pos,
                                               float* __restrict__ h, float2* __restrict__ rope, KvTarget kt,
                                               int32_t* __restrict__ kvpid, int32_t* __restrict__ order, int* err,
                                               const int32_t* __restrict__ dn) {
    const int i = blockIdx.x;
    const int n = live_rows(dn, gridDim.x);
    if (order && i == 0 && gridDim.x <= kMaxRows) row_order_block(pos, n, order);
    if (i >= n) return;
    rope_row(pos[i], hd, base, rope + (size_t)i * (hd / 2));
    const int t = tok[i];
    const bool ok = t >= 0 && t < vocab;
    if (threadIdx.x == 0) {
        if (!ok || slot[i] < 0 || slot[i] >= n_slots || seq[i] < 0 || seq[i] >= max_seqs || pos[i] < 0 ||
            pos[i] >= max_pos)
            set_err(err, CDB_DEV_BAD_INDEX);
        write_page(kt, i, seq[i], pos[i], nullptr, kvpid, err);
    }
    for (int k = threadIdx.x * 4; k < d; k += 1024) {
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (ok) {
            const uint2 w = *reinterpret_cast<const uint2*>(E + (size_t)t * d + k);
            v = make_float4(bflo(w.x), bfhi(w.x), bflo(w.y), bfhi(w.y));
        }
        *reinterpret_cast<float4*>(h + (size_t)i * d + k) = v;
    }
}

__global__ __launch_bounds__(256) void k_store_state(int d, int n_slots, const int32_t* __restrict__ slot,
                                                     const float* __restrict__ h, float* __restrict__ sh,
                                                     float* __restrict__ se, const int32_t* __restrict__ dn) {
    const int i = blockIdx.x;
    if (i >= live_rows(dn, gridDim.x)) return;
    const int sl = slot[i];
    if (sl < 0 || sl >= n_slots) return;
    for (int k = threadIdx.x * 4; k < d; k += 1024) {
        const float4 v = *reinterpret_cast<const float4*>(h + (size_t)i * d + k);
        *reinterpret_cast<float4*>(sh + (size_t)sl * d + k) = v;
        if (se) *reinterpret_cast<float4*>(se + (size_t)sl * d + k) = v;
    }
}

// ------------------------------------------------------------------ exit
// h += sum_s part[s] (the last down projection's split-K partials, split order
// 0..S-1, as the residual + norm kernel adds them); score: sigmoid(w_exit .
// RMSNorm(h)) or ||h - h_in||_2; exit = (c + 1 == depth); state.h[slot] = h.
// Exit score and decision of every row.  Replayed depths (gated == 0):
// exit = (c + 1 == depth).  Threshold gate (gated == 1, Section 4.3; App. C.2):
// the criterion (score >= threshold, or for convergence distance < threshold
// from loop 2 on) ends the token after this loop, or with lookahead after the
// next one, carried in pending[slot]; loop r_max always ends it.  deff[i] is
// the exiting row's depth (c + 1), 0 for continuing rows.
__global__ __launch_bounds__(256) void k_exit(int d, float eps, int exit_kind, int r_max, int n_slots,
                                              const int32_t* __restrict__ slot, const int32_t* __restrict__ c,
                                              const int32_t* __restrict__ depth, float* __restrict__ h,
                                              const float* __restrict__ part, int S, int M,
                                              const float* __restrict__ h_in, const uint16_t* __restrict__ w_exit,
                                              float* __restrict__ sh, float* __restrict__ score,
                                              uint8_t* __restrict__ mask, uint8_t* __restrict__ exit_next,
                                              int32_t* __restrict__ deff, int gated, float threshold, int lookahead,
                                              uint8_t* __restrict__ pending, const int32_t* __restrict__ dn) {
    __shared__ float red[4];
    const int i = blockIdx.x;
    if (i >= live_rows(dn, M)) return;
    float* x = h + (size_t)i * d;
    const float* x0 = h_in + (size_t)i * d;
    float a = 0.f, b = 0.f;
    for (int k = threadIdx.x * 4; k < d; k += 1024) {
        float4 v = *reinterpret_cast<const float4*>(x + k);
        if (S > 0) {
            for (int s0 = 0; s0 < S; ++s0) {
                const float4 p = *reinterpret_cast<const float4*>(part + ((size_t)s0 * M + i) * d + k);
                v.x += p.x;
                v.y += p.y;
                v.z += p.z;
                v.w += p.w;
            }
            *reinterpret_cast<float4*>(x + k) = v;
        }
        if (exit_kind == 1) {
            const float4 u = *reinterpret_cast<const float4*>(x0 + k);
            const float dx = v.x - u.x, dy = v.y - u.y, dz = v.z - u.z, dw = v.w - u.w;
            a += dx * dx + dy * dy + dz * dz + dw * dw;
        } else {
            const uint2 w = *reinterpret_cast<const uint2*>(w_exit + k);
            a += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
            b += v.x * bflo(w.x) + v.y * bfhi(w.x) + v.z * bflo(w.y) + v.w * bfhi(w.y);
        }
    }
    a = block_sum(a, red);
    b = block_sum(b, red);
    const int sl = slot[i];
    const bool slot_ok = sl >= 0 && sl < n_slots;
    if (threadIdx.x == 0) {
        float sc;
        if (exit_kind == 1) {
            sc = sqrtf(a);
        } else {
            const float z = b / sqrtf(a / d + eps);
            sc = 1.0f / (1.0f + __expf(-z));
        }
        score[i] = sc;
        const int r = c[i] + 1;  // loops done after this step
        bool ex, nxt;
        if (!gated) {
            const bool valid = depth[i] >= 1 && depth[i] <= r_max && c[i] >= 0 && c[i] < depth[i];
            ex = valid && r == depth[i];
            nxt = valid && r + 1 == depth[i];
        } else {
            const bool valid = c[i] >= 0 && c[i] < r_max && slot_ok;
            const bool meets = r >= (exit_kind == 1 ? 2 : 1) && (exit_kind == 1 ? sc < threshold : sc >= threshold);
            if (lookahead) {
                ex = valid && (r == r_max || pending[sl] != 0);
                nxt = valid && !ex && (meets || r + 1 == r_max);
                if (valid) pending[sl] = nxt ? 1 : 0;
            } else {
                ex = valid && (r == r_max || meets);
                nxt = valid && !ex && r + 1 == r_max;
            }
        }
        mask[i] = (uint8_t)ex;
        if (exit_next) exit_next[i] = (uint8_t)nxt;
        deff[i] = ex ? r : 0;
    }
    if (slot_ok)
        for (int k = threadIdx.x * 4; k < d; k += 1024)
            *reinterpret_cast<float4*>(sh + (size_t)sl * d + k) = *reinterpret_cast<const float4*>(x + k);
}
// Stable compaction of one step's rows: cont / exited list the continuing and
// exiting rows in batch order, counts = {continuing, exiting}.  Run by every
// thread of one 256-thread workgroup.
__device__ __forceinline__ void compact_block(int M, const uint8_t* __restrict__ mask, int32_t* __restrict__ cont,
                                              int32_t* __restrict__ exited, int32_t* __restrict__ counts) {
    __shared__ int s_scan[256];
    __shared__ int s_base;
    if (threadIdx.x == 0) s_base = 0;
    __syncthreads();
    for (int b0 = 0; b0 < M; b0 += 256) {
        const int i = b0 + threadIdx.x;
        const int e = i < M ? (int)mask[i] : 0;
        s_scan[threadIdx.x] = e;
        __syncthreads();
        for (int o = 1; o < 256; o <<= 1) {
            const int v = threadIdx.x >= o ? s_scan[threadIdx.x - o] : 0;
            __syncthreads();
            s_scan[threadIdx.x] += v;
            __syncthreads();
        }
        const int incl = s_scan[threadIdx.x];
        const int base = s_base;
        if (i < M) {
            const int ex_before = base + incl - e;  // exits before row i
            if (e)
                exited[ex_before] = i;
            else
                cont[i - ex_before] = i;
        }
        __syncthreads();
        if (threadIdx.x == 255) s_base = base + incl;
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        counts[0] = M - s_base;
        counts[1] = s_base;
    }
}

__global__ __launch_bounds__(256) void k_compact(int M, const uint8_t* __restrict__ mask, int32_t* __restrict__ cont,
                                                 int32_t* __restrict__ exited, int32_t* __restrict__ counts) {
    compact_block(M, mask, cont, exited, counts);
}

// Last-exited cache: for each exiting row (depth < r_max), copy its K/V at pos
// from plane depth to planes depth+1..r_max.  blockIdx.y = core layer * parts +
// part: a workgroup takes the destination planes depth+1+4*part .. +3 of one
// layer, so deep loops (31 destinations at r_max 32) spread over several
// workgroups.  depth is the row's exit depth, 0 for a continuing row.
// Workgroup (0, 0) also runs the step's stable compaction (the copy needs none
// of its output).  The destination page ids are read into LDS first and each
// chunk of the source entry (up to 8 16-byte vectors per thread) is loaded
// once, before any store: source and destinations share the pool, so a load
// left after a store would wait for it, one round trip per vector and plane.
// Planes that share a page (shared layouts) are written once, by the lowest
// plane that maps to it, and not at all when it is the source page.
constexpr int kCopyPlanesPerWg = 4;

__global__ __launch_bounds__(256) void k_copy_on_exit(int H, int hd, int r_max, KvTarget kv,
                                                      const int32_t* __restrict__ seq, const int32_t* __restrict__ pos,
                                                      const int32_t* __restrict__ depth,
                                                      const uint8_t* __restrict__ mask, int32_t* __restrict__ cont,
                                                      int32_t* __restrict__ exited, int32_t* __restrict__ counts,
                                                      int* err, const int32_t* __restrict__ dn) {
    __shared__ int s_dst[64];  // destination page of plane dep + 1 + k, -1 if unmapped (r_max <= 64)
    const int n = live_rows(dn, gridDim.x);
    if (blockIdx.x == 0 && blockIdx.y == 0) compact_block(n, mask, cont, exited, counts);
    const int i = blockIdx.x;
    if (i >= n) return;
    const int dep = depth[i];
    if (dep >= r_max || dep < 1) return;
    const int parts = max(1, (r_max - 1 + kCopyPlanesPerWg - 1) / kCopyPlanesPerWg);
    const int l = blockIdx.y / parts, part = blockIdx.y - l * parts;
    const int n_dst = r_max - dep;
    const int k0 = part * kCopyPlanesPerWg, k1 = min(n_dst, k0 + kCopyPlanesPerWg);
    if (k0 >= k1) return;
    const int sq = seq[i], ps = pos[i], pg = ps / kPage;
    if (sq < 0 || sq >= kv.max_seqs || pg < 0 || pg >= kv.max_pages) {
        if (threadIdx.x == 0 && part == 0) set_err(err, CDB_DEV_BAD_INDEX);
        return;
    }
    const int32_t* pt = kv.page_table + (size_t)sq * kv.n_planes * kv.max_pages;
    const int src = pt[(size_t)dep * kv.max_pages + pg];
    if (src < 0 || src >= kv.n_pages) {
        if (threadIdx.x == 0 && part == 0) set_err(err, CDB_DEV_UNMAPPED_PAGE);
        return;
    }
    if (threadIdx.x < n_dst) {
        const int dst = pt[(size_t)(dep + 1 + threadIdx.x) * kv.max_pages + pg];
        const bool ok = dst >= 0 && dst < kv.n_pages;
        if (!ok && threadIdx.x >= k0 && threadIdx.x < k1) set_err(err, CDB_DEV_UNMAPPED_PAGE);
        s_dst[threadIdx.x] = ok ? dst : -1;
    }
    __syncthreads();
    const int vec_per_head = hd / 8;  // 16-byte vectors per (kv, head) entry
    const int nvec = 2 * H * vec_per_head;
    const int tok = ps % kPage;
    // vector v = (kv * H + head, 8-element run e) of the entry: its offset from
    // kv_offset(l, page, ..., kv 0, head 0, tok 0) is the same on every page
    auto in_page = [&](int v) {
        const int kvh = v / vec_per_head, e = v - kvh * vec_per_head;
        return ((size_t)kvh * kPage + tok) * hd + e * 8;
    };
    // this workgroup's planes that receive a copy
    auto writes = [&](int k) {
        const int dst = s_dst[k];
        if (dst < 0 || dst == src) return false;
        for (int j = 0; j < k; ++j)
            if (s_dst[j] == dst) return false;
        return true;
    };
    const uint16_t* src_base = kv.pool + kv_offset(l, src, kv.n_pages, 0, 0, H, 0, hd);
    constexpr int VPT = 8;  // vectors per thread per chunk
    for (int base = 0; base < nvec; base += VPT * 256) {
        uint4 buf[VPT];
        size_t off[VPT];
#pragma unroll
        for (int u = 0; u < VPT; ++u) {
            const int v = base + threadIdx.x + u * 256;
            off[u] = v < nvec ? in_page(v) : 0;
            if (v < nvec) buf[u] = *reinterpret_cast<const uint4*>(src_base + off[u]);
        }
        for (int k = k0; k < k1; ++k) {
            if (!writes(k)) continue;
            uint16_t* dst_base = kv.pool + kv_offset(l, s_dst[k], kv.n_pages, 0, 0, H, 0, hd);
#pragma unroll
            for (int u = 0; u < VPT; ++u) {
                const int v = base + threadIdx.x + u * 256;
                if (v < nvec) *reinterpret_cast<uint4*>(dst_base + off[u]) = buf[u];
            }
        }
    }
}

// ------------------------------------------------------------------ argmax
__global__ __launch_bounds__(256) void k_argmax(int V, const float* __restrict__ logits, int32_t* __restrict__ ids,
                                                const int32_t* __restrict__ dn) {
    __shared__ float sv[256];
    __shared__ int si[256];
    const int i = blockIdx.x;
    if (i >= live_rows(dn, gridDim.x)) return;
    const float* x = logits + (size_t)i * V;
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    // each thread visits its values in increasing k, so a strict > keeps the
    // lower index on ties; 16-byte loads where the row allows them
    if ((V & 3) == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0) {
        const float4* x4 = reinterpret_cast<const float4*>(x);
        for (int k4 = threadIdx.x; k4 < (V >> 2); k4 += 256) {
            const float4 v = x4[k4];
            const int k = k4 * 4;
            if (v.x > bv) { bv = v.x; bi = k; }
            if (v.y > bv) { bv = v.y; bi = k + 1; }
            if (v.z > bv) { bv = v.z; bi = k + 2; }
            if (v.w > bv) { bv = v.w; bi = k + 3; }
        }
    } else {
        for (int k = threadIdx.x; k < V; k += 256) {
            const float v = x[k];
            if (v > bv) {
                bv = v;
                bi = k;
            }
        }
    }
    sv[threadIdx.x] = bv;
    si[threadIdx.x] = bi;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (threadIdx.x < o) {
            const float v2 = sv[threadIdx.x + o];
            const int i2 = si[threadIdx.x + o];
            if (v2 > sv[threadIdx.x] || (v2 == sv[threadIdx.x] && i2 < si[threadIdx.x])) {
                sv[threadIdx.x] = v2;
                si[threadIdx.x] = i2;
            }
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) ids[i] = si[0] == 0x7fffffff ? 0 : si[0];
}

// ------------------------------------------------------------------ packing
// dst tile (nt, ks), lane l, element e  <-  row r(nt*32 + l%32), column ks*16 + 8*(l/32) + e
// (A operand of v_mfma_f32_32x32x16_bf16, tiles of a 32-column stripe contiguous along K)
__global__ __launch_bounds__(256) void k_pack(int kind, const uint16_t* __restrict__ A, const uint16_t* __restrict__ B,
                                              const uint16_t* __restrict__ Cm, int N, int K, int hd, int H,
                                              uint16_t* __restrict__ dst) {
    const size_t KS = K / 16;
    const size_t total = (size_t)(N / 32) * KS * 64;
    for (size_t t = (size_t)blockIdx.x * 256 + threadIdx.x; t < total; t += (size_t)gridDim.x * 256) {
        const int lane = (int)(t & 63);
        const size_t tile = t >> 6;
        const int nt = (int)(tile / KS), ks = (int)(tile % KS);
        const int p = nt * 32 + (lane & 31);
        const int k = ks * 16 + 8 * (lane >> 5);
        const uint16_t* src;
        int row;
        if (kind == PACK_QKV) {
            const int g = p >> 5, w = p & 31, half = w >> 4, jj = w & 15;
            const int gph = hd >> 5, hg = H * gph;
            const int part = g / hg, rem = g - part * hg;
            const int head = rem / gph, gi = rem - head * gph;
            row = head * hd + gi * 16 + jj + half * (hd >> 1);
            src = part == 0 ? A : (part == 1 ? B : Cm);
        } else if (kind == PACK_GU) {
            const int g = p >> 5, half = (p >> 4) & 1;
            row = g * 16 + (p & 15);
            src = half ? B : A;
        } else {
            row = p;
            src = A;
        }
        *reinterpret_cast<uint4*>(dst + t * 8) = *reinterpret_cast<const uint4*>(src + (size_t)row * K + k);
    }
}

__global__ void k_copy16(const uint16_t* __restrict__ s, size_t n, uint16_t* __restrict__ d) {
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) d[i] = s[i];
}

__global__ void k_ws_init(int* err) {
    if (threadIdx.x == 0) *err = 0;
}

// ------------------------------------------------------------------ launchers
static int page_cap(const cdb_kv& kv) { return kv.max_pages * kPage; }

hipError_t launch_gather(const cdb_model_desc& md, const cdb_state& s, const cdb_rows& r, const cdb_kv& kv,
                         const KvTarget& kt, float* h, float* h_in, uint16_t* xcat, float2* rope, int32_t* kvpid,
                         int32_t* order, uint16_t* xn, int* err, hipStream_t st) {
    if (r.n_rows <= 0) return hipSuccess;
    if (order && r.n_rows > kMaxRows) return hipErrorInvalidValue;
    if (xcat && xn) return hipErrorInvalidValue;
    k_gather<<<r.n_rows, 256, 0, st>>>(md.d, md.r_max, s.n_slots, kv.max_seqs, page_cap(kv), md.head_dim, md.rope_base,
                                        r.slot, r.seq, r.pos, r.c, r.depth, s.h, s.e, h, h_in, xcat, rope, kt, kvpid,
                                        order, md.rms_eps, xn, err, r.d_n_rows);
    return hipGetLastError();
}

hipError_t launch_load_state(const cdb_model_desc& md, int M, const int32_t* slot, const int32_t* seq,
                             const int32_t* pos, const KvTarget& kt, const float* state_h, int n_slots, float* h,
                             float2* rope, int32_t* kvpid, int32_t* order, int* err, hipStream_t st,
                             const int32_t* dn) {
    if (M <= 0) return hipSuccess;
    if (order && M > kMaxRows) return hipErrorInvalidValue;
    k_load_state<<<M, 256, 0, st>>>(md.d, n_slots, md.head_dim, md.rope_base, slot, seq, pos, kt, state_h, h, rope,
                                    kvpid, order, err, dn);
    return hipGetLastError();
}

hipError_t launch_resid_norm(float* h, const float* part, int S, int M, int d, float eps, uint16_t* out,
                             hipStream_t st, const int32_t* dn) {
    if (M <= 0) return hipSuccess;
    // one workgroup per row, runs of 4 elements, at most 4 runs per thread
    if (d % 4 || d > 16384) return hipErrorInvalidValue;
    int threads = 64;
    while (threads < 1024 && threads * 4 < d) threads *= 2;
    const int nv = (d / 4 + threads - 1) / threads;
    if (nv == 1)
        k_resid_norm<1><<<M, threads, 0, st>>>(h, part, S, M, d, eps, out, dn);
    else if (nv == 2)
        k_resid_norm<2><<<M, threads, 0, st>>>(h, part, S, M, d, eps, out, dn);
    else
        k_resid_norm<4><<<M, threads, 0, st>>>(h, part, S, M, d, eps, out, dn);
    return hipGetLastError();
}

hipError_t launch_embed(const cdb_model_desc& md, const uint16_t* embed, const int32_t* tokens, const cdb_rows& r,
                        const cdb_kv& kv, const KvTarget& kt, int n_slots, float* h, float2* rope, int32_t* kvpid,
                        int32_t* order, int* err, hipStream_t st) {
    if (r.n_rows <= 0) return hipSuccess;
    if (order && r.n_rows > kMaxRows) return hipErrorInvalidValue;
    k_embed<<<r.n_rows, 256, 0, st>>>(md.d, md.vocab, n_slots, kv.max_seqs, page_cap(kv), md.head_dim, md.rope_base,
                                       embed, tokens, r.slot, r.seq, r.pos, h, rope, kt, kvpid, order, err,
                                       r.d_n_rows);
    return hipGetLastError();
}

hipError_t launch_store_state(int M, int d, int n_slots, const int32_t* slot, const float* h, float* state_h,
                              float* state_e, hipStream_t st, const int32_t* dn) {
    // out-of-range slots were reported by the embed kernel and are skipped here
    if (M <= 0) return hipSuccess;
    k_store_state<<<M, 256, 0, st>>>(d, n_slots, slot, h, state_h, state_e, dn);
    return hipGetLastError();
}

hipError_t launch_exit(const cdb_model_desc& md, const cdb_rows& r, float* h, const float* part, int S,
                       const float* h_in, const uint16_t* w_exit, float* state_h, int n_slots, const cdb_step_out& o,
                       const cdb_gate* gate, int32_t* deff, hipStream_t st) {
    if (r.n_rows <= 0) return hipSuccess;
    if (S < 0 || (S > 0 && !part)) return hipErrorInvalidValue;
    k_exit<<<r.n_rows, 256, 0, st>>>(md.d, md.rms_eps, md.exit_kind, md.r_max, n_slots, r.slot, r.c, r.depth, h,
                                      part, S, r.n_rows, h_in, w_exit, state_h, o.exit_score, o.exit_mask, o.exit_next, deff,
                                      gate ? 1 : 0, gate ? gate->threshold : 0.f, gate ? gate->lookahead : 0,
                                      gate ? gate->pending : nullptr, r.d_n_rows);
    return hipGetLastError();
}

hipError_t launch_compact(int M, const uint8_t* mask, int32_t* cont, int32_t* exited, int32_t* counts, hipStream_t st) {
    k_compact<<<1, 256, 0, st>>>(M, mask, cont, exited, counts);
    return hipGetLastError();
}

hipError_t launch_copy_on_exit(const cdb_model_desc& md, const cdb_kv& kv, const cdb_rows& r, const int32_t* deff,
                               const uint8_t* mask, int32_t* cont, int32_t* exited, int32_t* counts, int* err,
                               hipStream_t st) {
    if (r.n_rows <= 0 || md.n_core <= 0) return launch_compact(r.n_rows > 0 ? r.n_rows : 0, mask, cont, exited, counts, st);
    KvTarget t{};
    t.pool = static_cast<uint16_t*>(kv.core_pool);
    t.n_pages = kv.core_pages;
    t.n_layers = md.n_core;
    t.page_table = kv.page_table;
    t.max_seqs = kv.max_seqs;
    t.max_pages = kv.max_pages;
    t.n_planes = md.r_max + 2;
    const int parts = (md.r_max - 1 + kCopyPlanesPerWg - 1) / kCopyPlanesPerWg;
    dim3 grid(r.n_rows, md.n_core * std::max(parts, 1));
    k_copy_on_exit<<<grid, 256, 0, st>>>(md.n_heads, md.head_dim, md.r_max, t, r.seq, r.pos, deff, mask, cont, exited,
                                         counts, err, r.d_n_rows);
    return hipGetLastError();
}

// out[seq[i] * stride + index[i]] = ids[i]: files a coda batch's greedy ids
// under their sequence and decode index (rows outside the table are skipped).
__global__ __launch_bounds__(256) void k_scatter_ids(int M, const int32_t* __restrict__ ids,
                                                     const int32_t* __restrict__ seq,
                                                     const int32_t* __restrict__ index, int max_seqs, int stride,
                                                     int32_t* __restrict__ out) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= M) return;
    const int q = seq[i], k = index[i];
    if (q < 0 || q >= max_seqs || k < 0 || k >= stride) return;
    out[(size_t)q * stride + k] = ids[i];
}

hipError_t launch_scatter_ids(int M, const int32_t* ids, const int32_t* seq, const int32_t* index, int max_seqs,
                              int stride, int32_t* out, hipStream_t st) {
    if (M <= 0) return hipSuccess;
    k_scatter_ids<<<(M + 255) / 256, 256, 0, st>>>(M, ids, seq, index, max_seqs, stride, out);
    return hipGetLastError();
}

// dst[i] = src[seq[i]]: a batch's first decode inputs from the per-sequence
// entries the prefill wrote (out-of-range sequences read 0; the row-entry
// kernels report them).
__global__ __launch_bounds__(256) void k_gather_ids(int M, const int32_t* __restrict__ seq,
                                                    const int32_t* __restrict__ src, int max_seqs,
                                                    int32_t* __restrict__ dst) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= M) return;
    const int q = seq[i];
    dst[i] = q >= 0 && q < max_seqs ? src[q] : 0;
}

hipError_t launch_gather_ids(int M, const int32_t* seq, const int32_t* src, int max_seqs, int32_t* dst,
                             hipStream_t st) {
    if (M <= 0) return hipSuccess;
    k_gather_ids<<<(M + 255) / 256, 256, 0, st>>>(M, seq, src, max_seqs, dst);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void k_prefill_rows(int seq, int pos0, int M, int32_t* __restrict__ rows) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= M) return;
    rows[i] = i;
    rows[M + i] = seq;
    rows[2 * M + i] = pos0 + i;
}

hipError_t launch_prefill_rows(int seq, int pos0, int M, int32_t* rows, hipStream_t st) {
    if (M <= 0) return hipSuccess;
    k_prefill_rows<<<(M + 255) / 256, 256, 0, st>>>(seq, pos0, M, rows);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void k_kv_pages(KvTarget kt, int M, const int32_t* __restrict__ seq,
                                                  const int32_t* __restrict__ pos, int32_t* __restrict__ kvpid,
                                                  int* err) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < M) write_page(kt, i, seq[i], pos[i], nullptr, kvpid, err);
}

hipError_t launch_kv_pages(const KvTarget& kt, const cdb_rows& r, int32_t* kvpid, int* err, hipStream_t st) {
    if (r.n_rows <= 0) return hipSuccess;
    k_kv_pages<<<(r.n_rows + 255) / 256, 256, 0, st>>>(kt, r.n_rows, r.seq, r.pos, kvpid, err);
    return hipGetLastError();
}

// xcat[m] = bf16([h[m]; e[m]]) in fragment layout with K = 2d
__global__ __launch_bounds__(256) void k_concat_frag(int d, const float* __restrict__ h, const float* __restrict__ e,
                                                     uint16_t* __restrict__ xcat) {
    const int m = blockIdx.x;
    for (int k = threadIdx.x * 4; k < d; k += 1024) {
        const float4 a = *reinterpret_cast<const float4*>(h + (size_t)m * d + k);
        const float4 b = *reinterpret_cast<const float4*>(e + (size_t)m * d + k);
        uint2 pa, pb;
        pa.x = pack_bf16(a.x, a.y);
        pa.y = pack_bf16(a.z, a.w);
        pb.x = pack_bf16(b.x, b.y);
        pb.y = pack_bf16(b.z, b.w);
        *reinterpret_cast<uint2*>(xcat + frag_index(m, k, 2 * d)) = pa;
        *reinterpret_cast<uint2*>(xcat + frag_index(m, d + k, 2 * d)) = pb;
    }
}

hipError_t launch_concat_frag(int M, int d, const float* h, const float* e, uint16_t* xcat, hipStream_t st) {
    if (M <= 0) return hipSuccess;
    k_concat_frag<<<M, 256, 0, st>>>(d, h, e, xcat);
    return hipGetLastError();
}

hipError_t launch_argmax(int M, int V, const float* logits, int32_t* ids, hipStream_t st, const int32_t* dn) {
    if (M <= 0) return hipSuccess;
    k_argmax<<<M, 256, 0, st>>>(V, logits, ids, dn);
    return hipGetLastError();
}

hipError_t launch_pack(int kind, const uint16_t* a, const uint16_t* b, const uint16_t* c, int N, int K, int hd,
                       uint16_t* dst, hipStream_t st) {
    const int H = hd > 0 ? (N / 3) / hd : 0;
    k_pack<<<2048, 256, 0, st>>>(kind, a, b, c, N, K, hd, H, dst);
    return hipGetLastError();
}

hipError_t launch_copy_bf16(const uint16_t* src, size_t n, uint16_t* dst, hipStream_t st) {
    k_copy16<<<1024, 256, 0, st>>>(src, n, dst);
    return hipGetLastError();
}

hipError_t launch_ws_init(int* err, hipStream_t st) {
    k_ws_init<<<1, 64, 0, st>>>(err);
    return hipGetLastError();
}

}  // namespace cdb
