// Skinny bf16 GEMM for the block projections: Y[M][N] = X[M][K] . W[N][K]^T
// with M = rows of one stage call (ragged, <= 256) and the weight streamed from
// HBM exactly once per call.
//
// Design (gfx950):
//  * W is pre-packed into 16x32 MFMA operand tiles (1 KiB each) in lane order,
//    so one global_load_dwordx4 per lane fetches a full A operand of
//    v_mfma_f32_16x16x32_bf16, perfectly coalesced.  Tiles of one 16-column
//    stripe are contiguous along K.
//  * A workgroup of 4 waves owns 64 output columns (one 16-column stripe per
//    wave) and one K split.  The wave loads all its W tiles of the split into
//    registers up front (<= 16 tiles in flight), then runs over the rows in
//    chunks of 64: the chunk of X is staged in LDS once and read as the B
//    operand by all four waves.
//  * K splits are combined deterministically: each split writes fp32 partial
//    sums, and the last workgroup of a column tile to arrive (device-scope
//    counter) adds the partials in split order 0..S-1 and runs the fused
//    epilogue.  The split count depends on (N, K) only, so a row's result does
//    not depend on which other rows share the batch.
//  * Epilogues: q/k/v with RoPE and the K/V page write; residual add into the
//    fp32 stream; SwiGLU; plain store (adapter, LM head).
#include "cdb_internal.h"

namespace cdb {

constexpr int kWaves = 4;
constexpr int kTileN = 64;    // output columns per workgroup
constexpr int kChunkM = 64;   // rows per LDS chunk
constexpr int kMaxKt = 16;    // 32-wide K tiles per split held in registers
constexpr int kFtileLd = kTileN + 4;

__device__ __forceinline__ void epilogue(int epi, const float* ft, int m0, int M, int n_base, int N,
                                         const EpiArgs& ea) {
    const int tid = threadIdx.x;
    const int nl = tid & 63;
    const int p = n_base + nl;
    if (p >= N) return;
    for (int r = tid >> 6; r < kChunkM; r += 4) {
        const int m = m0 + r;
        if (m >= M) break;
        const float val = ft[r * kFtileLd + nl];
        if (epi == EPI_RESID) {
            ea.out[(size_t)m * ea.ld_out + p] += val;
        } else if (epi == EPI_STORE) {
            ea.out[(size_t)m * ea.ld_out + p] = val;
        } else if (epi == EPI_SWIGLU) {
            // packed order: groups of 32 columns = 16 gate columns then the 16
            // matching up columns
            if (p & 16) continue;
            const float g = val, u = ft[r * kFtileLd + (nl ^ 16)];
            const int f = (p >> 5) * 16 + (p & 15);
            const float s = g / (1.0f + __expf(-g));
            ea.act[(size_t)m * ea.ld_act + f] = f2bf(s * u);
        } else {  // EPI_QKV
            // packed order: groups of 32 columns per (part, head, 16 pairs):
            // 16 first-half dims j then the 16 second-half dims j + hd/2
            const int g = p >> 5, w = p & 31, half = w >> 4, jj = w & 15;
            const int gph = ea.hd >> 5;  // groups per head
            const int hg = ea.H * gph;
            const int part = g / hg, rem = g - part * hg;
            const int head = rem / gph, gi = rem - head * gph;
            const int j = gi * 16 + jj;
            const int dim = j + half * (ea.hd >> 1);
            float outv = val;
            if (part < 2) {
                const float partner = ft[r * kFtileLd + (nl ^ 16)];
                const double ang = (double)ea.pos[m] * pow((double)ea.rope_base, -2.0 * j / ea.hd);
                double sn, cs;
                sincos(ang, &sn, &cs);
                const float c = (float)cs, s = (float)sn;
                const float xf = half ? partner : val, xs = half ? val : partner;
                outv = half ? (xs * c + xf * s) : (xf * c - xs * s);
            }
            if (part == 0) {
                ea.q[(size_t)m * (ea.H * ea.hd) + head * ea.hd + dim] = outv;
            } else {
                const KvTarget& kv = ea.kv;
                const int sq = ea.seq[m], ps = ea.pos[m];
                const int plane = kv.c_row ? kv.c_row[m] + 1 : kv.plane_fixed;
                const int pg = ps / kPage;
                int pid = -1;
                if (sq >= 0 && sq < kv.max_seqs && pg >= 0 && pg < kv.max_pages && plane >= 0 && plane < kv.n_planes)
                    pid = kv.page_table[((size_t)sq * kv.n_planes + plane) * kv.max_pages + pg];
                if (pid < 0 || pid >= kv.n_pages) {
                    set_err(ea.err, CDB_DEV_UNMAPPED_PAGE);
                    continue;
                }
                const size_t page_elems = (size_t)kv.n_layers * 2 * ea.H * kPage * ea.hd;
                const size_t off = (size_t)pid * page_elems +
                                   ((((size_t)kv.layer * 2 + (part - 1)) * ea.H + head) * kPage + (ps % kPage)) * ea.hd +
                                   dim;
                kv.pool[off] = f2bf(outv);
            }
        }
    }
}

template <int EPI>
__global__ __launch_bounds__(256) void k_gemm(const uint16_t* __restrict__ X, int ldx, const uint16_t* __restrict__ Wp,
                                              int M, int N, int K, int S, float* __restrict__ part,
                                              int* __restrict__ counters, EpiArgs ea) {
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ int s_last;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int KT = K >> 5;
    const int s = blockIdx.y;
    const int kt0 = (int)(((long)s * KT) / S), kt1 = (int)(((long)(s + 1) * KT) / S);
    const int nk = kt1 - kt0;
    const int n_base = blockIdx.x * kTileN;
    const int nt = blockIdx.x * kWaves + wave;  // 16-column stripe of this wave
    const bool wave_ok = nt * 16 < N;

    // all W operand tiles of this split, straight into registers
    u32x4 wf[kMaxKt];
    if (wave_ok) {
        const u32x4* src = reinterpret_cast<const u32x4*>(Wp) + ((size_t)nt * KT + kt0) * 64 + lane;
#pragma unroll
        for (int i = 0; i < kMaxKt; ++i)
            if (i < nk) wf[i] = __builtin_nontemporal_load(src + (size_t)i * 64);
    }

    uint16_t* xs = reinterpret_cast<uint16_t*>(smem);
    float* ft = reinterpret_cast<float*>(smem);
    const int xld = nk * 32 + 8;  // LDS row stride (elements), padded against bank conflicts

    for (int m0 = 0; m0 < M; m0 += kChunkM) {
        __syncthreads();
        // stage X[m0 .. m0+64)[kt0*32 .. kt1*32) in LDS, 16 bytes per thread-step
        const int vec_per_row = nk * 4;
        for (int v = tid; v < kChunkM * vec_per_row; v += 256) {
            const int r = v / vec_per_row, cv = v - r * vec_per_row;
            uint4 val = make_uint4(0, 0, 0, 0);
            if (m0 + r < M) val = *reinterpret_cast<const uint4*>(X + (size_t)(m0 + r) * ldx + kt0 * 32 + cv * 8);
            *reinterpret_cast<uint4*>(xs + r * xld + cv * 8) = val;
        }
        __syncthreads();
        floatx4 acc[4];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) acc[mt] = floatx4{0.f, 0.f, 0.f, 0.f};
        if (wave_ok) {
#pragma unroll
            for (int i = 0; i < kMaxKt; ++i) {
                if (i < nk) {
                    const bf16x8 a = __builtin_bit_cast(bf16x8, wf[i]);
#pragma unroll
                    for (int mt = 0; mt < 4; ++mt) {
                        const uint4 bv = *reinterpret_cast<const uint4*>(xs + (mt * 16 + (lane & 15)) * xld + i * 32 +
                                                                         (lane >> 4) * 8);
                        acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8, bv), acc[mt],
                                                                          0, 0, 0);
                    }
                }
            }
        }
        // lane holds D[n = 4*(lane/16) + j][m = lane%16] of each 16x16 tile
        const int ncol = nt * 16 + 4 * (lane >> 4);
        if (S == 1) {
            __syncthreads();  // xs is about to be overwritten by the output tile
            if (wave_ok) {
#pragma unroll
                for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        ft[(mt * 16 + (lane & 15)) * kFtileLd + wave * 16 + 4 * (lane >> 4) + j] = acc[mt][j];
            }
            __syncthreads();
            epilogue(EPI, ft, m0, M, n_base, N, ea);
        } else if (wave_ok) {
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                const int m = m0 + mt * 16 + (lane & 15);
                if (m < M)
                    *reinterpret_cast<float4*>(part + ((size_t)s * M + m) * N + ncol) =
                        make_float4(acc[mt][0], acc[mt][1], acc[mt][2], acc[mt][3]);
            }
        }
    }
    if (S == 1) return;

    // split-K: the last workgroup of this column tile sums the partials in order
    __threadfence();
    __syncthreads();
    if (tid == 0) {
        const int old = atomicAdd(&counters[blockIdx.x], 1);
        s_last = (old == S - 1);
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    for (int m0 = 0; m0 < M; m0 += kChunkM) {
        __syncthreads();
        for (int v = tid; v < kChunkM * (kTileN / 4); v += 256) {
            const int r = v / (kTileN / 4), c4 = (v - r * (kTileN / 4)) * 4;
            const int m = m0 + r, n = n_base + c4;
            float4 sum = make_float4(0.f, 0.f, 0.f, 0.f);
            if (m < M && n < N) {
                for (int ss = 0; ss < S; ++ss) {
                    const floatx4 pv = __builtin_nontemporal_load(
                        reinterpret_cast<const floatx4*>(part + ((size_t)ss * M + m) * N + n));
                    sum.x += pv[0];
                    sum.y += pv[1];
                    sum.z += pv[2];
                    sum.w += pv[3];
                }
            }
            *reinterpret_cast<float4*>(ft + r * kFtileLd + c4) = sum;
        }
        __syncthreads();
        epilogue(EPI, ft, m0, M, n_base, N, ea);
    }
    if (tid == 0) atomicExch(&counters[blockIdx.x], 0);
}

GemmShape gemm_shape(int N, int K) {
    const int tiles = (N + kTileN - 1) / kTileN;
    const int KT = K / 32;
    int S = (512 + tiles - 1) / tiles;
    if (S > KT / 4) S = KT / 4;
    const int smin = (KT + kMaxKt - 1) / kMaxKt;
    if (S < smin) S = smin;
    if (S < 1) S = 1;
    return GemmShape{N, K, S};
}

template <int EPI>
static hipError_t launch_one(const uint16_t* X, int ldx, const uint16_t* Wp, int M, GemmShape g, float* part,
                             int* counters, const EpiArgs& ea, hipStream_t st) {
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemm<EPI>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 96 * 1024);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int KT = g.K / 32;
    const int nk_max = (KT + g.S - 1) / g.S;
    size_t lds = (size_t)kChunkM * (nk_max * 32 + 8) * 2;
    const size_t lds_ft = (size_t)kChunkM * kFtileLd * 4;
    if (lds < lds_ft) lds = lds_ft;
    dim3 grid((g.N + kTileN - 1) / kTileN, g.S);
    k_gemm<EPI><<<grid, 256, lds, st>>>(X, ldx, Wp, M, g.N, g.K, g.S, part, counters, ea);
    return hipGetLastError();
}

hipError_t launch_gemm(int epi, const uint16_t* X, int ldx, const uint16_t* Wp, int M, GemmShape g, float* part,
                       int* counters, const EpiArgs& ea, hipStream_t st) {
    if (M <= 0) return hipSuccess;
    switch (epi) {
        case EPI_QKV: return launch_one<EPI_QKV>(X, ldx, Wp, M, g, part, counters, ea, st);
        case EPI_RESID: return launch_one<EPI_RESID>(X, ldx, Wp, M, g, part, counters, ea, st);
        case EPI_SWIGLU: return launch_one<EPI_SWIGLU>(X, ldx, Wp, M, g, part, counters, ea, st);
        default: return launch_one<EPI_STORE>(X, ldx, Wp, M, g, part, counters, ea, st);
    }
}

}  // namespace cdb
