// Skinny bf16 GEMM for the block projections: Y[M][N] = X[M][K] . W[N][K]^T
// with M = rows of one stage call (ragged, <= 256) and the weight streamed from
// HBM exactly once per call.
//
// Design (gfx950):
//  * W is pre-packed into 32x16 operand tiles of v_mfma_f32_32x32x16_bf16 in
//    lane order (1 KiB each), so one 16-byte load per lane fetches a whole A
//    operand, coalesced; the tiles of one 32-column stripe are contiguous
//    along K.  A 32-wide stripe halves the activation (B operand) traffic per
//    weight byte compared with a 16-wide one.
//  * A workgroup owns NS (1 or 2) 32-column stripes and one K split; its KW
//    waves split that K range further.  Each wave streams its weight tiles and the matching
//    activation fragments (L2-resident) in batches, double-buffered in
//    registers so one batch is in flight while the previous one feeds the
//    MFMAs.  The KW partial tiles are summed in LDS in wave order.
//  * No reduction crosses workgroups inside the kernel.  Stripes whose K is
//    split over S workgroups write fp32 partial tiles; the row kernel that
//    runs next (residual add + RMSNorm) adds them in split order.  Every
//    reduction order depends on (N, K) only, so a row's result does not depend
//    on which other rows share the batch.
//  * Epilogues: q/k/v with RoPE and the K/V page write (a 32-column group is
//    16 first-half and the 16 matching second-half dims of one head), SwiGLU (a
//    group is 16 gate and the 16 matching up columns), plain fp32 store, and
//    the split-K partial store.
#include "cdb_internal.h"

namespace cdb {

constexpr int kMaxKw = 8;     // waves per workgroup (2 per SIMD, so 256 registers each)

struct GemmArgs {
    const uint16_t* X;  // fragment layout, gemm_rows(M) rows (rows >= M are never read back), K columns
    const uint16_t* Wp;
    int M, N, K, S, KW;
    float* part;  // EPI_PARTIAL: [S][M][N]
    const int32_t* dn;  // optional device row count (<= M): rows at or past it are not stored
};

// Inputs of the q/k/v epilogue, staged in LDS: the RoPE factors of the
// stripe's 16 rotary pairs for every row, and each row's K/V write page and
// slot within it.
struct QkvStage {
    const float2* rope;  // [rows][16]; NULL: read the call's tables in global memory
    const int* pid;      // [rows]
    const int* tok;      // [rows]
};

// split: the workgroup's K split (EPI_PARTIAL writes partial tile `split`)
template <int EPI>
__device__ __forceinline__ void epilogue_elem(float val, float partner, int m, int p, int split, const GemmArgs& ga,
                                              const EpiArgs& ea, const QkvStage& qs) {
    if (EPI == EPI_STORE) {
        ea.out[(size_t)m * ea.ld_out + p] = val;
    } else if (EPI == EPI_PARTIAL) {
        ga.part[((size_t)split * ga.M + m) * ga.N + p] = val;
    } else if (EPI == EPI_SWIGLU) {
        if (p & 16) return;
        const int f = (p >> 5) * 16 + (p & 15);
        const float s = val / (1.0f + __expf(-val));
        ea.act[frag_index(m, f, ea.ld_act)] = f2bf(s * partner);
    } else {  // EPI_QKV
        const int g = p >> 5, w = p & 31, half = w >> 4, jj = w & 15;
        const int gph = ea.hd >> 5;  // groups per head
        const int hg = ea.H * gph;
        const int part = g / hg, rem = g - part * hg;
        const int head = rem / gph, gi = rem - head * gph;
        const int dim = gi * 16 + jj + half * (ea.hd >> 1);
        float outv = val;
        if (part < 2) {
            const float2 cs = qs.rope ? qs.rope[m * 16 + jj] : ea.rope[(size_t)m * (ea.hd >> 1) + gi * 16 + jj];
            const float xf = half ? partner : val, xs = half ? val : partner;
            outv = half ? (xs * cs.x + xf * cs.y) : (xf * cs.x - xs * cs.y);
        }
        if (part == 0) {
            ea.q[(size_t)m * (ea.H * ea.hd) + head * ea.hd + dim] = outv;
            return;
        }
        const int pid = qs.rope ? qs.pid[m] : ea.kvpid[m];  // -1: unmapped (reported by the row-entry kernel)
        if (pid < 0) return;
        const KvTarget& kv = ea.kv;
        const int tok = qs.rope ? qs.tok[m] : ea.pos[m] % kPage;
        kv.pool[kv_offset(kv.layer, pid, kv.n_pages, part - 1, head, ea.H, tok, ea.hd) + dim] = f2bf(outv);
    }
}

// Epilogue of the skinny kernel from the reduced tiles fin[ns][n][m] (row
// pitch fld), with 16-byte stores: each thread takes a run of consecutive
// output columns of one row (4 fp32 values, or 8 bf16 values in the
// fragment or K/V layouts).  Same arithmetic per element as epilogue_elem.
template <int EPI>
__device__ __forceinline__ void stripe_epilogue(const float* fin, int fld, int nt, int NS, int mcap, int split, int tid,
                                                int nthr, const GemmArgs& ga, const EpiArgs& ea, const QkvStage& qs) {
    if (EPI == EPI_PARTIAL || EPI == EPI_STORE) {
        // (ns, m, 4-column run)
        const int per = mcap * 8;
        float* base = EPI == EPI_PARTIAL ? ga.part + (size_t)split * ga.M * ga.N : ea.out;
        const int ld = EPI == EPI_PARTIAL ? ga.N : ea.ld_out;
        for (int e = tid; e < NS * per; e += nthr) {
            const int ns = e / per, r = e - ns * per;
            if (nt + ns >= (ga.N >> 5)) break;
            const int m = r >> 3, c4 = (r & 7) * 4;
            const float* f = fin + ns * 32 * fld + c4 * fld + m;
            const float4 v = make_float4(f[0], f[fld], f[2 * fld], f[3 * fld]);
            float* dst = base + (size_t)m * ld + (nt + ns) * 32 + c4;
            if ((ld & 3) == 0) {
                *reinterpret_cast<float4*>(dst) = v;
            } else {
                dst[0] = v.x;
                dst[1] = v.y;
                dst[2] = v.z;
                dst[3] = v.w;
            }
        }
    } else if (EPI == EPI_SWIGLU) {
        // (ns, m, 8-feature run): gate columns c8 .. c8 + 7, up columns 16 + c8 ..
        const int per = mcap * 2;
        for (int e = tid; e < NS * per; e += nthr) {
            const int ns = e / per, r = e - ns * per;
            if (nt + ns >= (ga.N >> 5)) break;
            const int m = r >> 1, c8 = (r & 1) * 8;
            const float* f = fin + ns * 32 * fld + m;
            uint32_t w[4];
#pragma unroll
            for (int i = 0; i < 8; i += 2) {
                const float g0 = f[(c8 + i) * fld], u0 = f[(16 + c8 + i) * fld];
                const float g1 = f[(c8 + i + 1) * fld], u1 = f[(16 + c8 + i + 1) * fld];
                const float s0 = g0 / (1.0f + __expf(-g0)), s1 = g1 / (1.0f + __expf(-g1));
                w[i / 2] = pack_bf16(s0 * u0, s1 * u1);
            }
            const int feat = (nt + ns) * 16 + c8;
            *reinterpret_cast<u32x4*>(ea.act + frag_index(m, feat, ea.ld_act)) = u32x4{w[0], w[1], w[2], w[3]};
        }
    } else {  // EPI_QKV: a stripe holds 16 rotary pairs (dims gi*16 + jj and + hd/2) of one head
      const int mrows = fld - 1;  // rows of a stripe's staged RoPE table
      for (int ns = 0; ns < NS; ++ns) {
        const int g = nt + ns, gph = ea.hd >> 5, hg = ea.H * gph;
        if (g >= (ga.N >> 5)) break;
        const int part = g / hg, rem = g - part * hg;
        const int head = rem / gph, gi = rem - head * gph;
        const int half_hd = ea.hd >> 1;
        const float* fs = fin + ns * 32 * fld;
        const float2* srope = qs.rope ? qs.rope + (size_t)ns * mrows * 16 : nullptr;
        if (part == 0) {
            // (m, half, 4-pair run) -> 4 consecutive fp32 q values
            for (int e = tid; e < mcap * 8; e += nthr) {
                const int m = e >> 3, half = (e >> 2) & 1, j4 = (e & 3) * 4;
                float o[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int jj = j4 + i;
                    const float val = fs[(half * 16 + jj) * fld + m], partner = fs[((half ^ 1) * 16 + jj) * fld + m];
                    const float2 cs = srope ? srope[m * 16 + jj] : ea.rope[(size_t)m * half_hd + gi * 16 + jj];
                    const float xf = half ? partner : val, xs = half ? val : partner;
                    o[i] = half ? (xs * cs.x + xf * cs.y) : (xf * cs.x - xs * cs.y);
                }
                float* dst = ea.q + (size_t)m * (ea.H * ea.hd) + head * ea.hd + gi * 16 + j4 + half * half_hd;
                *reinterpret_cast<float4*>(dst) = make_float4(o[0], o[1], o[2], o[3]);
            }
        } else {
            // (m, half, 8-pair run) -> 8 consecutive bf16 K or V values
            for (int e = tid; e < mcap * 4; e += nthr) {
                const int m = e >> 2, half = (e >> 1) & 1, j8 = (e & 1) * 8;
                const int pid = qs.rope ? qs.pid[m] : ea.kvpid[m];  // -1: unmapped (reported by the row-entry kernel)
                if (pid < 0) continue;
                const int tok = qs.rope ? qs.tok[m] : ea.pos[m] % kPage;
                uint32_t w[4];
#pragma unroll
                for (int i = 0; i < 8; i += 2) {
                    float o2[2];
#pragma unroll
                    for (int b = 0; b < 2; ++b) {
                        const int jj = j8 + i + b;
                        const float val = fs[(half * 16 + jj) * fld + m];
                        float outv = val;
                        if (part == 1) {
                            const float partner = fs[((half ^ 1) * 16 + jj) * fld + m];
                            const float2 cs =
                                srope ? srope[m * 16 + jj] : ea.rope[(size_t)m * half_hd + gi * 16 + jj];
                            const float xf = half ? partner : val, xs = half ? val : partner;
                            outv = half ? (xs * cs.x + xf * cs.y) : (xf * cs.x - xs * cs.y);
                        }
                        o2[b] = outv;
                    }
                    w[i / 2] = pack_bf16(o2[0], o2[1]);
                }
                const KvTarget& kv = ea.kv;
                uint16_t* dst = kv.pool + kv_offset(kv.layer, pid, kv.n_pages, part - 1, head, ea.H, tok, ea.hd) +
                                gi * 16 + j8 + half * half_hd;
                *reinterpret_cast<u32x4*>(dst) = u32x4{w[0], w[1], w[2], w[3]};
            }
        }
      }
    }
}

// k steps per register load batch of the decode kernel (register budget: two
// batches of NS weight + MT activation operands)
__host__ __device__ constexpr int decode_batch_steps(int MT, int NS) {
    return NS == 1 ? (MT <= 2 ? 8 : (MT == 4 ? 4 : 1)) : (MT <= 2 ? 4 : (MT == 4 ? 2 : 1));
}

// 32x32 tiles the decode kernel's wave reduction sums per round: all NS x MT
// of them when 8 waves' copies, the reduced block and the q/k/v staging fit in
// 160 KB of LDS, else one
__host__ __device__ constexpr int decode_red_tiles(bool qkv, int MT, int NS) {
    return (8 * NS * MT * 1024 + NS * 32 * (MT * 32 + 1) + (qkv ? NS * MT * 32 * 32 + MT * 64 : 0)) * 4 <= 160 * 1024
               ? NS * MT : 1;
}

// MT = 32-row tiles of M covered by one pass (M <= 32 * MT); NS = adjacent
// 32-column stripes per workgroup (they share every activation load); TAIL:
// some wave's K range is not a whole number of load batches (decode_batch_steps).
template <int EPI, int MT, int NS, bool TAIL>
__global__ __launch_bounds__(512) void k_gemm(GemmArgs ga, EpiArgs ea) {
    extern __shared__ __align__(16) float smem[];
    // the wave index as a scalar, so each wave's K range and its batch tests
    // below are wave-uniform branches
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int KW = ga.KW;
    const int KS = ga.K >> 4;  // 16-wide k steps
    const int s = blockIdx.y;
    const int a0 = (int)(((long)s * KS) / ga.S), a1 = (int)(((long)(s + 1) * KS) / ga.S);
    const int ks0 = a0 + (int)(((long)wave * (a1 - a0)) / KW);
    const int ks1 = a0 + (int)(((long)(wave + 1) * (a1 - a0)) / KW);
    const int nt = blockIdx.x * NS;  // first 32-column stripe
    const int M = ga.M;

    floatx16 acc[NS][MT];
#pragma unroll
    for (int ns = 0; ns < NS; ++ns)
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
            for (int j = 0; j < 16; ++j) acc[ns][t][j] = 0.f;

    // a workgroup's last stripes may lie past the matrix (an odd stripe count
    // with NS = 2): they re-read the last stripe and their results are not stored
    const int stripes = ga.N >> 5;
    const u32x4* wsrc[NS];
#pragma unroll
    for (int ns = 0; ns < NS; ++ns)
        wsrc[ns] = reinterpret_cast<const u32x4*>(ga.Wp) + (size_t)min(nt + ns, stripes - 1) * KS * 64 + lane;
    // X is in fragment layout: the operand of m-tile t at k step k is the 1 KiB tile (t, k)
    const u32x4* xsrc = reinterpret_cast<const u32x4*>(ga.X) + lane;
    constexpr int CH = decode_batch_steps(MT, NS);

    // Two register sets: the next batch's loads are in flight while the
    // current batch feeds the MFMAs.
    u32x4 wa[CH][NS], wb[CH][NS];
    u32x4 xa[CH][MT], xb[CH][MT];
    // Loads are unconditional (steps past the wave's range re-read its last
    // step) so that the compiler keeps each batch's loads in flight across the
    // other batch's MFMAs.  With TAIL, the wave's last batch skips the MFMAs of
    // the steps past its range (a wave-uniform branch); without it every batch
    // is whole and no step is tested.
    auto load = [&](u32x4 (&w)[CH][NS], u32x4 (&x)[CH][MT], int c0) {
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            const int ks = min(c0 + i, ks1 - 1);
#pragma unroll
            for (int ns = 0; ns < NS; ++ns) w[i][ns] = wsrc[ns][(size_t)ks * 64];
#pragma unroll
            for (int t = 0; t < MT; ++t) x[i][t] = xsrc[((size_t)t * KS + ks) * 64];
        }
    };
    auto step = [&](const u32x4 (&w)[NS], const u32x4 (&x)[MT]) {
#pragma unroll
        for (int ns = 0; ns < NS; ++ns) {
            const bf16x8 a = __builtin_bit_cast(bf16x8, w[ns]);
#pragma unroll
            for (int t = 0; t < MT; ++t)
                acc[ns][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, __builtin_bit_cast(bf16x8, x[t]), acc[ns][t],
                                                                     0, 0, 0);
        }
    };
    auto compute = [&](const u32x4 (&w)[CH][NS], const u32x4 (&x)[CH][MT], int c0) {
#pragma unroll
        for (int i = 0; i < CH; ++i)
            if (!TAIL || c0 + i < ks1) step(w[i], x[i]);
    };
    if (ks0 < ks1) load(wa, xa, ks0);

    // q/k/v epilogue inputs, loaded while the weight stream is in flight (no
    // wait on them before the main loop ends); above 64 rows the RoPE factors
    // would cost more registers than the loop can spare and are loaded after it
    const int mcap = min(live_rows(ga.dn, M), MT * 32);
    const int nthr = KW * 64;
    constexpr int RP = MT <= 2 ? MT * 2 : 1;  // MT <= 2: >= mcap * 16 / nthr, as nthr >= 256
    float2 pf_rope[RP];
    int pf_pid = -1, pf_tok = 0;
    int q_part = 0, q_gi = 0, q_part_last = 0;
    if constexpr (EPI == EPI_QKV) {
        const int gph = ea.hd >> 5, hg = ea.H * gph;
        q_part = nt / hg;
        q_gi = (nt - q_part * hg) % gph;
        q_part_last = min(nt + NS - 1, stripes - 1) / hg;
        if (MT <= 2 && NS == 1 && q_part < 2) {
#pragma unroll
            for (int r = 0; r < RP; ++r) {
                const int idx = tid + r * nthr;
                if (idx < mcap * 16)
                    pf_rope[r] = ea.rope[(size_t)(idx >> 4) * (ea.hd >> 1) + q_gi * 16 + (idx & 15)];
            }
        }
        if (q_part_last > 0 && tid < mcap) {  // a K or V stripe
            pf_pid = ea.kvpid[tid];
            pf_tok = ea.pos[tid] % kPage;
        }
    }

    for (int c0 = ks0; c0 < ks1; c0 += 2 * CH) {
        if (c0 + CH < ks1) load(wb, xb, c0 + CH);
        compute(wa, xa, c0);
        if (c0 + 2 * CH < ks1) load(wa, xa, c0 + 2 * CH);
        if (c0 + CH < ks1) compute(wb, xb, c0 + CH);
    }

    // Sum the KW wave tiles in wave order: with 8 waves (a grid of one
    // workgroup per CU at most) all NS x MT 32x32 tiles in one round where they
    // fit in LDS (decode_red_tiles), else one tile at a time, which keeps the
    // LDS of wider grids small enough for several workgroups per CU.
    // acc[ns][t][j] holds D[n = (j/4)*8 + (lane/32)*4 + j%4][m = t*32 + lane%32]
    // of stripe nt + ns.
    constexpr int RT = decode_red_tiles(EPI == EPI_QKV, MT, NS);
    const bool one_round = RT > 1 && KW == 8;
    float* red = smem;                                   // [KW][RT or 1][32 n][32 m]
    float* fin = smem + KW * (one_round ? RT : 1) * 1024;  // [NS][32 n][MT*32 m + 1]
    const int fld = MT * 32 + 1;
    QkvStage qs{};
    if constexpr (EPI == EPI_QKV) {
        // per stripe a [MT*32][16] RoPE table; 32 * fld is even
        float2* s_rope = reinterpret_cast<float2*>(fin + NS * 32 * fld);
        int* s_pid = reinterpret_cast<int*>(s_rope + NS * MT * 32 * 16);
        int* s_tok = s_pid + MT * 32;
        if (MT <= 2 && NS == 1) {
            if (q_part < 2) {
#pragma unroll
                for (int r = 0; r < RP; ++r) {
                    const int idx = tid + r * nthr;
                    if (idx < mcap * 16) s_rope[idx] = pf_rope[r];
                }
            }
        } else {
            const int gph = ea.hd >> 5, hg = ea.H * gph;
            for (int ns = 0; ns < NS; ++ns) {
                const int g = min(nt + ns, stripes - 1);
                if (g / hg >= 2) continue;  // V: no rotation
                const int gi = (g % hg) % gph;
                for (int idx = tid; idx < mcap * 16; idx += nthr)
                    s_rope[ns * MT * 32 * 16 + idx] = ea.rope[(size_t)(idx >> 4) * (ea.hd >> 1) + gi * 16 + (idx & 15)];
            }
        }
        if (tid < mcap) {
            s_pid[tid] = pf_pid;
            s_tok[tid] = pf_tok;
        }
        qs = QkvStage{s_rope, s_pid, s_tok};  // visible after the reduction's barriers
    }
    if (RT > 1 && one_round) {
#pragma unroll
        for (int ns = 0; ns < NS; ++ns)
#pragma unroll
            for (int t = 0; t < MT; ++t)
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const int nn = (j >> 2) * 8 + (lane >> 5) * 4 + (j & 3);
                    red[(wave * RT + ns * MT + t) * 1024 + nn * 32 + (lane & 31)] = acc[ns][t][j];
                }
        __syncthreads();
        for (int e = tid; e < RT * 1024; e += nthr) {
            const int tile = e >> 10, r = e & 1023, ns = tile / MT, t = tile - ns * MT;
            float sum = 0.f;
            for (int w = 0; w < KW; ++w) sum += red[(w * RT + tile) * 1024 + r];
            fin[ns * 32 * fld + (r >> 5) * fld + t * 32 + (r & 31)] = sum;
        }
        __syncthreads();
    } else {
#pragma unroll
        for (int ns = 0; ns < NS; ++ns) {
#pragma unroll
            for (int t = 0; t < MT; ++t) {
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const int nn = (j >> 2) * 8 + (lane >> 5) * 4 + (j & 3);
                    red[wave * 1024 + nn * 32 + (lane & 31)] = acc[ns][t][j];
                }
                __syncthreads();
                for (int e = tid; e < 1024; e += nthr) {
                    float sum = 0.f;
                    for (int w = 0; w < KW; ++w) sum += red[w * 1024 + e];
                    fin[ns * 32 * fld + (e >> 5) * fld + t * 32 + (e & 31)] = sum;
                }
                __syncthreads();
            }
        }
    }

    stripe_epilogue<EPI>(fin, fld, nt, NS, mcap, s, tid, nthr, ga, ea, qs);
}

// q/k/v epilogue of a wave's (32 WM)-row x 64-column block (stripes nt0,
// nt0 + 1; rows m0 .. m0 + 32 WM - 1) staged in LDS as fin[n][m - m0] (pitch
// fld): each lane takes a run of consecutive dims of one row, so the stores
// are 16-byte vectors (4 fp32 q values, or 8 bf16 K/V values) instead of one
// column of 32 rows per instruction.  A q stripe gives a lane 4 WM runs (rows
// lane/8 + 8i, 4 dims), a K/V stripe 2 WM runs (rows lane/4 + 16i, 8 dims).  The global loads
// (RoPE factors, page ids, positions; qkv_block_loads) are issued before the
// GEMM's main loop: the stores may alias them, so loads left between stores
// would wait one by one.  Same arithmetic per element as epilogue_elem.
struct QkvBlockInputs {
    float4 rc[2][16];  // (cos, sin) pairs of each run, two per float4
    int pid[2][4], tok[2][4];
};

template <int WM>
__device__ __forceinline__ void qkv_block_loads(QkvBlockInputs& in, int nt0, int stripes, int m0, int M, int lane,
                                                const EpiArgs& ea) {
    const int gph = ea.hd >> 5, hg = ea.H * gph, half_hd = ea.hd >> 1;
    float4 (&rc)[2][16] = in.rc;
    int (&pid)[2][4] = in.pid;
    int (&tok)[2][4] = in.tok;
#pragma unroll
    for (int a = 0; a < 2; ++a) {
        const int g = nt0 + a;
        if (g >= stripes) break;
        const int part = g / hg, gi = (g - part * hg) % gph;
        if (part == 0) {
#pragma unroll
            for (int it = 0; it < 4 * WM; ++it) {
                const int m = min(m0 + (lane >> 3) + 8 * it, M - 1);
                const float4* cs = reinterpret_cast<const float4*>(ea.rope + (size_t)m * half_hd + gi * 16 + (lane & 3) * 4);
                rc[a][2 * it] = cs[0];
                rc[a][2 * it + 1] = cs[1];
            }
        } else {
#pragma unroll
            for (int it = 0; it < 2 * WM; ++it) {
                const int m = min(m0 + (lane >> 2) + 16 * it, M - 1);
                pid[a][it] = ea.kvpid[m];
                tok[a][it] = ea.pos[m] % kPage;
                if (part == 1) {
                    const float4* cs = reinterpret_cast<const float4*>(ea.rope + (size_t)m * half_hd + gi * 16 + (lane & 1) * 8);
#pragma unroll
                    for (int i = 0; i < 4; ++i) rc[a][4 * it + i] = cs[i];
                }
            }
        }
    }
}

template <int WM>
__device__ __forceinline__ void qkv_block_epilogue(const QkvBlockInputs& in, const float* fin, int fld, int nt0,
                                                   int stripes, int m0, int M, int lane, const EpiArgs& ea) {
    const int gph = ea.hd >> 5, hg = ea.H * gph, half_hd = ea.hd >> 1;
    const float4 (&rc)[2][16] = in.rc;
    const int (&pid)[2][4] = in.pid;
    const int (&tok)[2][4] = in.tok;
    // pair t of a run from its float4s
    auto cpair = [](const float4* r, int t) {
        const float4 v = r[t >> 1];
        return (t & 1) ? make_float2(v.z, v.w) : make_float2(v.x, v.y);
    };
#pragma unroll
    for (int a = 0; a < 2; ++a) {
        const int g = nt0 + a;
        if (g >= stripes) break;
        const int part = g / hg, rem = g - part * hg;
        const int head = rem / gph, gi = rem - head * gph;
        const float* f = fin + a * 32 * fld;
        if (part == 0) {
#pragma unroll
            for (int it = 0; it < 4 * WM; ++it) {
                const int ml = (lane >> 3) + 8 * it, half = (lane >> 2) & 1, j4 = (lane & 3) * 4;
                const int m = m0 + ml;
                if (m >= M) continue;
                float o[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int jj = j4 + i;
                    const float val = f[(half * 16 + jj) * fld + ml], partner = f[((half ^ 1) * 16 + jj) * fld + ml];
                    const float2 c = cpair(&rc[a][2 * it], i);
                    const float xf = half ? partner : val, xs = half ? val : partner;
                    o[i] = half ? (xs * c.x + xf * c.y) : (xf * c.x - xs * c.y);
                }
                float* dst = ea.q + (size_t)m * (ea.H * ea.hd) + head * ea.hd + gi * 16 + j4 + half * half_hd;
                *reinterpret_cast<float4*>(dst) = make_float4(o[0], o[1], o[2], o[3]);
            }
        } else {
#pragma unroll
            for (int it = 0; it < 2 * WM; ++it) {
                const int ml = (lane >> 2) + 16 * it, half = (lane >> 1) & 1, j8 = (lane & 1) * 8;
                const int m = m0 + ml;
                // pid -1: unmapped (reported by the row-entry kernel)
                if (m >= M || pid[a][it] < 0) continue;
                uint32_t w[4];
#pragma unroll
                for (int i = 0; i < 8; i += 2) {
                    float o2[2];
#pragma unroll
                    for (int b = 0; b < 2; ++b) {
                        const int jj = j8 + i + b;
                        const float val = f[(half * 16 + jj) * fld + ml];
                        float outv = val;
                        if (part == 1) {
                            const float partner = f[((half ^ 1) * 16 + jj) * fld + ml];
                            const float2 c = cpair(&rc[a][4 * it], i + b);
                            const float xf = half ? partner : val, xs = half ? val : partner;
                            outv = half ? (xs * c.x + xf * c.y) : (xf * c.x - xs * c.y);
                        }
                        o2[b] = outv;
                    }
                    w[i / 2] = pack_bf16(o2[0], o2[1]);
                }
                const KvTarget& kv = ea.kv;
                uint16_t* dst = kv.pool + kv_offset(kv.layer, pid[a][it], kv.n_pages, part - 1, head, ea.H, tok[a][it], ea.hd) +
                                gi * 16 + j8 + half * half_hd;
                *reinterpret_cast<u32x4*>(dst) = u32x4{w[0], w[1], w[2], w[3]};
            }
        }
    }
}

// Large-M GEMM (prefill chunks of up to 512 rows), where the product is
// compute-bound (about M FLOP per weight byte).  A workgroup owns a
// (64 WM)-row x 128-column output tile and one K split: 4 waves in 2 x 2, each
// 32 WM rows x 64 columns (WM m-tiles x 2 stripes, 2 WM MFMAs per 16-wide k
// step), operands read straight from the packed weights and the fragment-
// layout activations (each tile feeds two waves; the second read is served by
// the caches), double-buffered in registers.  Each wave owns its outputs, so
// the epilogue runs from the accumulators: column n's RoPE / SwiGLU partner
// n ^ 16 is element j ^ 8 of the same lane.
//
// Tile order (xcd_order): the grid is one-dimensional, padded to a multiple of
// 8, and the dispatcher hands workgroup b to XCD b % 8.  With xcd_order 0 the
// tasks run column group first (every row tile of a column group lands on a
// different XCD); with 1 each XCD takes a contiguous range of tasks ordered
// row tile first, so the row tiles that read one weight tile run together on
// one XCD and share its L2.
template <int EPI, bool LDS, int WM>
__global__ __launch_bounds__(256) void k_gemm_mn(GemmArgs ga, EpiArgs ea, int xcd_order) {
    static_assert(WM == 1 || WM == 2, "one or two m-tiles per wave");
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int KS = ga.K >> 4;
    const int stripes = ga.N >> 5;
    const int mtiles = (gemm_rows(ga.M) + 31) >> 5;  // m-tiles the activation buffer holds
    const int gx = (stripes + 3) / 4, gy = (ga.M + 64 * WM - 1) / (64 * WM), tasks = gx * gy * ga.S;
    int bx, by, s;
    if (xcd_order) {
        const int per = (tasks + 7) / 8;
        const int t = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
        if (t >= tasks) return;
        by = t % gy;
        s = (t / gy) % ga.S;
        bx = t / (gy * ga.S);
    } else {
        const int t = blockIdx.x;
        if (t >= tasks) return;
        bx = t % gx;
        by = (t / gx) % gy;
        s = t / (gx * gy);
    }
    const int k0 = (int)(((long)s * KS) / ga.S), k1 = (int)(((long)(s + 1) * KS) / ga.S);
    const int nt0 = bx * 4 + (wave & 1) * 2;   // first stripe of this wave
    const int mt0 = by * 2 * WM + (wave >> 1) * WM;  // first m-tile of this wave

    floatx16 acc[2][WM];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < WM; ++b)
#pragma unroll
            for (int j = 0; j < 16; ++j) acc[a][b][j] = 0.f;
    QkvBlockInputs qin;
    if constexpr (EPI == EPI_QKV) qkv_block_loads<WM>(qin, nt0, stripes, mt0 * 32, ga.M, lane, ea);

    if constexpr (!LDS) {
        // tiles past the matrix re-read the last one (their results are not stored)
        const u32x4* wsrc[2];
        const u32x4* xsrc[WM];
    #pragma unroll
        for (int a = 0; a < 2; ++a)
            wsrc[a] = reinterpret_cast<const u32x4*>(ga.Wp) + (size_t)min(nt0 + a, stripes - 1) * KS * 64 + lane;
    #pragma unroll
        for (int b = 0; b < WM; ++b)
            xsrc[b] = reinterpret_cast<const u32x4*>(ga.X) + (size_t)min(mt0 + b, mtiles - 1) * KS * 64 + lane;
        constexpr int CH = 4;
        u32x4 wa[CH][2], wb[CH][2], xa[CH][WM], xb[CH][WM];
        auto load = [&](u32x4 (&w)[CH][2], u32x4 (&x)[CH][WM], int c0) {
    #pragma unroll
            for (int i = 0; i < CH; ++i) {
                const int ks = min(c0 + i, k1 - 1);
    #pragma unroll
                for (int a = 0; a < 2; ++a) w[i][a] = wsrc[a][(size_t)ks * 64];
    #pragma unroll
                for (int b = 0; b < WM; ++b) x[i][b] = xsrc[b][(size_t)ks * 64];
            }
        };
        auto compute = [&](const u32x4 (&w)[CH][2], const u32x4 (&x)[CH][WM], int c0) {
    #pragma unroll
            for (int i = 0; i < CH; ++i) {
                const uint32_t keep = c0 + i < k1 ? 0xffffffffu : 0u;
    #pragma unroll
                for (int a = 0; a < 2; ++a) {
                    const bf16x8 wv = __builtin_bit_cast(bf16x8, w[i][a] & keep);
    #pragma unroll
                    for (int b = 0; b < WM; ++b)
                        acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wv, __builtin_bit_cast(bf16x8, x[i][b]),
                                                                            acc[a][b], 0, 0, 0);
                }
            }
        };
        if (k0 < k1) load(wa, xa, k0);
        for (int c0 = k0; c0 < k1; c0 += 2 * CH) {
            if (c0 + CH < k1) load(wb, xb, c0 + CH);
            compute(wa, xa, c0);
            if (c0 + 2 * CH < k1) load(wa, xa, c0 + 2 * CH);
            if (c0 + CH < k1) compute(wb, xb, c0 + CH);
        }
    } else {
        // LDS ring of 2 stages of 4 k steps: a stage holds the workgroup's 4
        // weight tiles and 2 WM activation tiles of each k step (1 KiB each,
        // lane order), copied global -> LDS by the waves with direct loads (tile
        // i of a stage by wave i % 4); each wave then reads its 2 + WM operands
        // per k step
        constexpr int CH = 4, NBUF = 2;
        constexpr int TPK = 4 + 2 * WM;  // tiles per k step
        constexpr int TPS = CH * TPK;    // tiles per stage
        constexpr int LPW = TPS / 4;     // loads per wave per stage
        static_assert(TPS % 4 == 0, "a stage's tiles split evenly over the 4 waves");
        extern __shared__ __align__(16) unsigned char lds_ring[];
        const int ntb = bx * 4, mtb = by * 2 * WM;
        const u32x4* Wg = reinterpret_cast<const u32x4*>(ga.Wp);
        const u32x4* Xg = reinterpret_cast<const u32x4*>(ga.X);
        const int nst = (k1 - k0 + CH - 1) / CH;
        auto issue = [&](int st) {
            unsigned char* base = lds_ring + (size_t)(st % NBUF) * TPS * 1024;
#pragma unroll
            for (int i = 0; i < LPW; ++i) {
                const int t = wave + 4 * i;  // tile within the stage
                const int kk = t / TPK, slot = t - kk * TPK;
                const int ks = min(k0 + st * CH + kk, k1 - 1);
                const u32x4* src = slot < 4 ? Wg + ((size_t)min(ntb + slot, stripes - 1) * KS + ks) * 64
                                            : Xg + ((size_t)min(mtb + slot - 4, mtiles - 1) * KS + ks) * 64;
                __builtin_amdgcn_global_load_lds(src + lane, (__attribute__((address_space(3))) void*)(base + t * 1024),
                                                 16, 0, 0);
            }
        };
        if (nst > 0) issue(0);
        const int wn = wave & 1, wm = wave >> 1;
        for (int st = 0; st < nst; ++st) {
            // this wave's loads of stage st are done; the barrier covers the
            // other waves' loads and every wave's reads of the stage refilled next
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __builtin_amdgcn_s_barrier();
            if (st + 1 < nst) issue(st + 1);
            const unsigned char* base = lds_ring + (size_t)(st % NBUF) * TPS * 1024 + lane * 16;
#pragma unroll
            for (int i = 0; i < CH; ++i) {
                const uint32_t keep = k0 + st * CH + i < k1 ? 0xffffffffu : 0u;
                u32x4 w[2], x[WM];
#pragma unroll
                for (int a = 0; a < 2; ++a)
                    w[a] = *reinterpret_cast<const u32x4*>(base + (i * TPK + wn * 2 + a) * 1024);
#pragma unroll
                for (int b = 0; b < WM; ++b)
                    x[b] = *reinterpret_cast<const u32x4*>(base + (i * TPK + 4 + wm * WM + b) * 1024);
#pragma unroll
                for (int a = 0; a < 2; ++a) {
                    const bf16x8 wv = __builtin_bit_cast(bf16x8, w[a] & keep);
#pragma unroll
                    for (int b = 0; b < WM; ++b)
                        acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wv, __builtin_bit_cast(bf16x8, x[b]),
                                                                            acc[a][b], 0, 0, 0);
                }
            }
        }
    }
    if constexpr (EPI == EPI_QKV) {
        // the wave's block through its own LDS region (64 columns x (32 WM + 1)-float rows);
        // on the LDS path the region overlaps the ring, which the other waves may still be reading
        if constexpr (LDS) __syncthreads();
        extern __shared__ __align__(16) unsigned char lds_ring[];
        constexpr int fld = 32 * WM + 1;
        float* fin = reinterpret_cast<float*>(lds_ring) + wave * 64 * fld;
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < WM; ++b)
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const int n = a * 32 + (j >> 2) * 8 + (lane >> 5) * 4 + (j & 3);
                    fin[n * fld + b * 32 + (lane & 31)] = acc[a][b][j];
                }
        qkv_block_epilogue<WM>(qin, fin, fld, nt0, stripes, mt0 * 32, ga.M, lane, ea);
        return;
    }
    const QkvStage qs{};
#pragma unroll
    for (int a = 0; a < 2; ++a) {
        if (nt0 + a >= stripes) continue;
#pragma unroll
        for (int b = 0; b < WM; ++b) {
            const int m = (mt0 + b) * 32 + (lane & 31);
            if (m >= ga.M) continue;
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int n = (j >> 2) * 8 + (lane >> 5) * 4 + (j & 3);
                epilogue_elem<EPI>(acc[a][b][j], acc[a][b][j ^ 8], m, (nt0 + a) * 32 + n, s, ga, ea, qs);
            }
        }
    }
}

// Which tile-kernel path a projection takes: the LDS-staged one pays off for
// the wide projections (gate/up and a full-width LM head: 20% faster at 512
// rows) and for split-K projections whose splits run long k loops (Huginn-
// shaped O and down, 165 and 560 k steps per split at 512 rows: 64 -> 52 and
// 218 -> 174 us); q/k/v and the short-split O and down (Ouro-shaped: 32 and 88
// k steps) are faster with direct loads.
static int mn_splits(int N, int K, int M, int rows_per_tile);
static int lds_wave_mtiles(int M) { return ((M + 63) / 64) % 2 ? 1 : 2; }
static bool mn_lds(int epi, int N, int K, int M) {
    if (epi == EPI_SWIGLU || (epi == EPI_STORE && N >= 8192)) return true;
    return epi == EPI_PARTIAL && (K / 16) / mn_splits(N, K, M, 64 * lds_wave_mtiles(M)) >= 128;
}

// m-tiles per wave of the tile kernel: 2 (128-row workgroup tiles) or 1 (64-row
// tiles; the sums are the same either way).  Direct loads: 1 for q/k/v when
// that grid still runs in one round on the 256 CUs; its workgroups take one
// CU each (register bound), so at 257-320 rows of the Ouro-shaped q/k/v the
// 64-row tiles use 240 CUs instead of 144 (29 -> 22 us); above that they would
// take two rounds.  O and down are as fast or faster with 128-row tiles at
// every size from 272 to 512 rows but 480-512.  LDS-staged: 1 when the rows
// span an odd number of 64-row tiles, which 128-row tiles would pad by 64 rows
// (gate/up at 300 rows: 36.0 -> 30.1 us; at 512 rows 64-row tiles gain nothing).
static int mn_wave_mtiles(int epi, int N, int K, int M) {
    if (mn_lds(epi, N, K, M)) return lds_wave_mtiles(M);
    return epi == EPI_QKV && ((M + 63) / 64) * ((N / 32 + 3) / 4) <= 256 ? 1 : 2;
}

// K splits of the split-K partial epilogue: doubled until the grid covers the
// chip, keeping at least 32 k steps per split.
static int mn_splits(int N, int K, int M, int rows_per_tile) {
    const int tiles = ((N / 32 + 3) / 4) * ((M + rows_per_tile - 1) / rows_per_tile);
    const int KS = K / 16;
    int S = 1;
    while (tiles * S < 256 && KS / (S * 2) >= 32) S *= 2;
    return S;
}

// Launch shape for M > kMaxRows rows (k_gemm_mn): K split only for the
// split-K partial epilogue.
GemmShape gemm_shape_mn(int N, int K, int M, int epi) {
    const int S = epi == EPI_PARTIAL ? mn_splits(N, K, M, 64 * mn_wave_mtiles(epi, N, K, M)) : 1;
    return GemmShape{N, K, S, 4, 4};
}

// XCD-aware tile order (see k_gemm_mn) for grids of more than two workgroups
// per CU (LM heads and Huginn-shaped gate/up at 512 rows: 615 -> 485 and
// 325 -> 292 us) and for LDS-staged split-K grids; the others keep the plain
// order, which is as fast or up to 5% faster for them.
static int mn_xcd_order(bool lds, int tasks, int S) { return tasks > 512 || (lds && S > 1) ? 1 : 0; }

GemmShape gemm_shape(int N, int K, int epi, int M) {
    // S and KW fix every wave's K range and so the summation order of each
    // output: they depend on (N, K, epi) only, which keeps a row's result
    // independent of the rows that share its call.  NS (stripes per
    // workgroup) only regroups whole stripes, and follows the row count.
    const int stripes = N / 32;
    const int KS = K / 16;
    const int MT = M <= 32 ? 1 : (M <= 64 ? 2 : (M <= 128 ? 4 : 8));  // 32-row tiles per pass
    // K split until the grid covers the chip, keeping at least 64 k steps per
    // workgroup (a 4-way split of a 2048-long K loses more to each workgroup's
    // fixed costs than its extra workgroups gain: Ouro's O at 64 rows 6.4 ->
    // 5.8 us with 2 ways)
    int S = 1;
    if (epi == EPI_PARTIAL) {
        while (stripes * S < 256 && KS / (S * 2) >= 64) S *= 2;
    }
    // Two stripes per workgroup share every activation load.  Wide projections
    // without a K split (gate/up, LM head) take them at up to 128 rows (a
    // 256-row pass holds one stripe); split-K projections over long K ranges
    // (and q/k/v, whose epilogue handles a pair) take them at 65-128 rows, where
    // each weight byte brings 4 activation bytes from L2 and that stream bounds
    // the kernel: with at least 160 k steps per workgroup (Huginn-shaped O,
    // down and q/k/v: 36 -> 28, 99 -> 69 and 75 -> 54 us), not with 128 or fewer
    // (Ouro-shaped q/k/v: 15 -> 22 us), nor below 65 rows.
    const bool pair_wide = epi != EPI_QKV && epi != EPI_PARTIAL && S == 1 && stripes > 256 && stripes % 2 == 0 &&
                           KS >= 64;
    const bool pair_long = (epi == EPI_PARTIAL || epi == EPI_QKV) && KS / S >= 160;
    const int NS = (pair_wide && MT < 8) || (pair_long && MT == 4) ? 2 : 1;
    // waves per workgroup: 8 (more weight bytes in flight per CU) while the
    // grid fits the chip in one round, counted with the stripe pairs where
    // they may be used, else 4
    const int groups = (pair_wide || pair_long) ? (stripes + 1) / 2 : stripes;
    const int KW = groups * S <= 256 && KS / S >= 32 ? 8 : 4;
    return GemmShape{N, K, S, KW, NS};
}

// Whether some wave's K range in k_gemm (the same proportional split of each
// workgroup's split over its KW waves) is not a whole number of batches.
static bool decode_has_tail(int K, int S, int KW, int ch) {
    const int KS = K / 16;
    for (int s = 0; s < S; ++s) {
        const int a0 = (int)(((long)s * KS) / S), a1 = (int)(((long)(s + 1) * KS) / S);
        for (int w = 0; w < KW; ++w) {
            const int n = (int)(((long)(w + 1) * (a1 - a0)) / KW) - (int)(((long)w * (a1 - a0)) / KW);
            if (n % ch) return true;
        }
    }
    return false;
}

template <int EPI, int MT, int NS, bool TAIL>
static hipError_t launch_tail(const GemmArgs& ga, const EpiArgs& ea, hipStream_t st) {
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemm<EPI, MT, NS, TAIL>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int rt = decode_red_tiles(EPI == EPI_QKV, MT, NS);
    size_t lds = ((size_t)ga.KW * (rt > 1 && ga.KW == 8 ? rt : 1) * 1024 + (size_t)NS * 32 * (MT * 32 + 1)) * 4;
    if (EPI == EPI_QKV) lds += (size_t)NS * MT * 32 * 16 * 8 + (size_t)MT * 32 * 2 * 4;
    dim3 grid((ga.N / 32 + NS - 1) / NS, ga.S);
    k_gemm<EPI, MT, NS, TAIL><<<grid, ga.KW * 64, lds, st>>>(ga, ea);
    return hipGetLastError();
}

template <int EPI, int MT, int NS>
static hipError_t launch_mt(const GemmArgs& ga, const EpiArgs& ea, hipStream_t st) {
    return decode_has_tail(ga.K, ga.S, ga.KW, decode_batch_steps(MT, NS)) ? launch_tail<EPI, MT, NS, true>(ga, ea, st)
                                                                          : launch_tail<EPI, MT, NS, false>(ga, ea, st);
}

template <int EPI, int NS>
static hipError_t launch_ns(const GemmArgs& ga, const EpiArgs& ea, hipStream_t st) {
    if (ga.M <= 32) return launch_mt<EPI, 1, NS>(ga, ea, st);
    if (ga.M <= 64) return launch_mt<EPI, 2, NS>(ga, ea, st);
    if (ga.M <= 128) return launch_mt<EPI, 4, NS>(ga, ea, st);
    return launch_mt<EPI, 8, 1>(ga, ea, st);  // two stripes of 256 rows exceed the register file
}

template <int EPI>
static hipError_t launch_epi(const GemmArgs& ga, const EpiArgs& ea, int ns, hipStream_t st) {
    return ns == 2 ? launch_ns<EPI, 2>(ga, ea, st) : launch_ns<EPI, 1>(ga, ea, st);
}

template <int EPI, bool LDS, int WM>
static hipError_t launch_mn_wm(const GemmArgs& ga, const EpiArgs& ea, hipStream_t st) {
    const int tasks = (ga.N / 32 + 3) / 4 * ((ga.M + 64 * WM - 1) / (64 * WM)) * ga.S;
    const dim3 grid((tasks + 7) / 8 * 8);
    // dynamic LDS: the ring of the LDS path, the q/k/v epilogue's staging blocks
    constexpr size_t ring = LDS ? 2 * 4 * (4 + 2 * WM) * 1024 : 0;
    constexpr size_t stage = EPI == EPI_QKV ? 4 * 64 * (32 * WM + 1) * 4 : 0;
    constexpr size_t smem = ring > stage ? ring : stage;
    if constexpr (smem > 0) {
        static bool attr_set = false;
        if (!attr_set) {
            hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemm_mn<EPI, LDS, WM>),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
            if (e != hipSuccess) return e;
            attr_set = true;
        }
    }
    k_gemm_mn<EPI, LDS, WM><<<grid, 256, smem, st>>>(ga, ea, mn_xcd_order(LDS, tasks, ga.S));
    return hipGetLastError();
}

template <int EPI>
static hipError_t launch_mn(const GemmArgs& ga, const EpiArgs& ea, hipStream_t st) {
    const int wm = mn_wave_mtiles(EPI, ga.N, ga.K, ga.M);
    if (mn_lds(EPI, ga.N, ga.K, ga.M))
        return wm == 1 ? launch_mn_wm<EPI, true, 1>(ga, ea, st) : launch_mn_wm<EPI, true, 2>(ga, ea, st);
    if (wm == 1) return launch_mn_wm<EPI, false, 1>(ga, ea, st);
    return launch_mn_wm<EPI, false, 2>(ga, ea, st);
}

hipError_t launch_gemm(int epi, const uint16_t* X, const uint16_t* Wp, int M, GemmShape g, float* part,
                       const EpiArgs& ea, hipStream_t st, const int32_t* dn) {
    if (M <= 0) return hipSuccess;
    if (g.K % 16 || g.N % 32 || g.S < 1) return hipErrorInvalidValue;
    GemmArgs ga{X, Wp, M, g.N, g.K, g.S, g.KW, part, dn};
    if (M > kMaxRows) {  // prefill chunks: the compute-bound tile kernel (shape from gemm_shape_mn)
        if (M > kMaxPrefillRows || g.NS != 4 || dn) return hipErrorInvalidValue;
        switch (epi) {
            case EPI_QKV: return launch_mn<EPI_QKV>(ga, ea, st);
            case EPI_SWIGLU: return launch_mn<EPI_SWIGLU>(ga, ea, st);
            case EPI_PARTIAL: return launch_mn<EPI_PARTIAL>(ga, ea, st);
            default: return launch_mn<EPI_STORE>(ga, ea, st);
        }
    }
    if (g.KW < 1 || g.KW > kMaxKw || (g.NS != 1 && g.NS != 2)) return hipErrorInvalidValue;
    if (epi == EPI_QKV && g.KW < 4) return hipErrorInvalidValue;  // epilogue staging: >= 256 threads
    switch (epi) {
        case EPI_QKV: return launch_epi<EPI_QKV>(ga, ea, g.NS, st);
        case EPI_SWIGLU: return launch_epi<EPI_SWIGLU>(ga, ea, g.NS, st);
        case EPI_PARTIAL: return launch_epi<EPI_PARTIAL>(ga, ea, g.NS, st);
        default: return launch_epi<EPI_STORE>(ga, ea, g.NS, st);
    }
}

}  // namespace cdb
