// Paged decode attention over the depth-indexed KV cache.
//
// One query per (row, head): the row's q (after RoPE) attends to positions
// 0..pos of its sequence in one KV plane (the row's loop plane for the core,
// the stage plane for prelude/coda).  HBM-bound: every K/V byte is read once
// and used by one query, so the kernel is built for streaming, not MFMA.
//
// Layout of one (layer, page, head): K [16 tokens][hd] then (after H*16*hd
// elements) V [16][hd], bf16; pools are layer-major (kv_offset).  A wave reads a page as four coalesced
// loads for K and four for V: lane l covers token (4*j + l/16) and dims
// [(l%16)*hd/16, +hd/16).  The 16 lanes of a DPP row reduce q.k with row DPP
// (quad_perm, half_mirror, mirror), and each DPP row keeps its own online
// softmax over the tokens it owns, so no cross-row traffic happens per page.
//
// Balance: rows of one batch have different context lengths, and all
// workgroups of a launch are resident at once, so one workgroup per row would
// leave the chip idle while the longest rows finish.  A workgroup therefore
// takes two rows -- the p-th longest and the p-th shortest, from the order
// ranked at the start of the stage call (by the first workgroup of its
// row-entry kernel, or by k_row_order for a standalone attention call) -- and
// deals the pages of both to its 4 waves.  Each wave keeps one softmax state
// per row.  With pairs, mixed and equal context lengths run at the same
// bandwidth.  The partial states are merged through LDS in an order fixed by
// the row alone, so every row's output is bit-identical whatever else shares
// the batch; the output is written in the fragment layout the output
// projection reads.
#include "cdb_internal.h"

namespace cdb {


template <int DPL>
struct RawVec {
    uint32_t w[DPL / 2];
};

// DPL bf16 values (held as DPL/2 dwords) to fp32
template <int DPL>
__device__ __forceinline__ void unpack_vec(const uint32_t* w, float* out) {
#pragma unroll
    for (int e = 0; e < DPL / 2; ++e) {
        out[2 * e] = bflo(w[e]);
        out[2 * e + 1] = bfhi(w[e]);
    }
}

// K and V are read once per launch and never again by it: the loads are
// non-temporal (streamed past the caches' normal allocation), which lifts a
// plain read stream on this part from about 6.3 to 7.1 TB/s.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <int DPL>
__device__ __forceinline__ RawVec<DPL> load_raw(const uint16_t* p) {
    RawVec<DPL> r;
    if constexpr (DPL == 8) {
        const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
        r.w[0] = v[0]; r.w[1] = v[1]; r.w[2] = v[2]; r.w[3] = v[3];
    } else if constexpr (DPL == 4) {
        const u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
        r.w[0] = v[0]; r.w[1] = v[1];
    } else {
        const uint32_t* q = reinterpret_cast<const uint32_t*>(p);
        r.w[0] = __builtin_nontemporal_load(q);
        r.w[1] = __builtin_nontemporal_load(q + 1);
        r.w[2] = __builtin_nontemporal_load(q + 2);
    }
    return r;
}

#define CDB_DPP(v, ctrl) __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, (v)), (ctrl), 0xF, 0xF, true))

// Sum over the 16 lanes of a DPP row; every lane of the row gets the sum.
__device__ __forceinline__ float row_sum16(float v) {
    v += CDB_DPP(v, 0xB1);   // quad_perm [1,0,3,2]
    v += CDB_DPP(v, 0x4E);   // quad_perm [2,3,0,1]
    v += CDB_DPP(v, 0x141);  // row_half_mirror
    v += CDB_DPP(v, 0x140);  // row_mirror
    return v;
}

template <int DPL>
struct PageData {
    RawVec<DPL> k[4], v[4];
};

// Online-softmax update of one row's state with one 16-token page.
template <int DPL>
__device__ __forceinline__ void attend_page(const PageData<DPL>& pd, const float* qr, int first_tok, int n_ctx, int g,
                                            float& m_run, float& l_run, float* acc) {
    float sc[4];
    float mx = m_run;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        float kf[DPL];
        unpack_vec<DPL>(pd.k[j].w, kf);
        float dot = 0.f;
#pragma unroll
        for (int e = 0; e < DPL; ++e) dot += qr[e] * kf[e];
        dot = row_sum16(dot);
        const bool valid = first_tok + j * 4 + g < n_ctx;
        sc[j] = valid ? dot : -1e30f;
        mx = fmaxf(mx, sc[j]);
    }
    const float corr = exp2f(m_run - mx);
    l_run *= corr;
#pragma unroll
    for (int e = 0; e < DPL; ++e) acc[e] *= corr;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const bool valid = first_tok + j * 4 + g < n_ctx;
        const float pj = valid ? exp2f(sc[j] - mx) : 0.f;
        l_run += pj;
        float vf[DPL];
        unpack_vec<DPL>(pd.v[j].w, vf);
#pragma unroll
        for (int e = 0; e < DPL; ++e) acc[e] += valid ? pj * vf[e] : 0.f;
    }
    m_run = mx;
}

constexpr int kAttnWaves = 4;

template <int HD>
__global__ __launch_bounds__(kAttnWaves * 64) void k_attn(const float* __restrict__ q, KvTarget kv,
                                                          const int32_t* __restrict__ seq,
                                                          const int32_t* __restrict__ pos,
                                                          const int32_t* __restrict__ order, int M, int H,
                                                          uint16_t* __restrict__ out, int* err,
                                                          const int32_t* __restrict__ dn) {
    constexpr int DPL = HD / 16;
    constexpr int NP = kAttnWaves * 4;  // partial states per row
    __shared__ float s_m[2][NP], s_l[2][NP];
    __shared__ float s_acc[2][NP][HD];
    const int head = blockIdx.x, pair = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, li = lane & 15;
    const int d = H * HD;
    const float qscale = 1.4426950408889634f / sqrtf((float)HD);  // log2(e) / sqrt(hd)
    const size_t vofs = (size_t)H * kPage * HD;  // V follows K within a (layer, page)

    // the pair: p-th longest and p-th shortest row (one row when they meet);
    // with a device row count the grid covers the capacity M
    const int n = live_rows(dn, M);
    if (2 * pair >= n) return;
    int rows[2];
    rows[0] = order[pair];
    rows[1] = (n - 1 - pair > pair) ? order[n - 1 - pair] : -1;
    int n_ctx[2] = {0, 0}, npg[2] = {0, 0}, valid[2] = {0, 0};
    const int32_t* pt[2] = {kv.page_table, kv.page_table};
    float qr[2][DPL];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
#pragma unroll
        for (int e = 0; e < DPL; ++e) qr[r][e] = 0.f;
        const int m = rows[r];
        if (m < 0) continue;
        const int sq = seq[m];
        // a row's own loop index reads a core plane (1..r_max) only
        const int plane = kv.c_row ? kv.c_row[m] + 1 : kv.plane_fixed;
        const bool plane_ok =
            kv.c_row ? (plane >= 1 && plane <= kv.n_planes - 2) : (plane >= 0 && plane < kv.n_planes);
        const int nc = pos[m] + 1;
        const int np = (nc + kPage - 1) / kPage;
        if (!(sq >= 0 && sq < kv.max_seqs && plane_ok && nc >= 1 && np <= kv.max_pages)) {
            if (tid == 0) set_err(err, CDB_DEV_UNMAPPED_PAGE);
            continue;
        }
        valid[r] = 1;
        n_ctx[r] = nc;
        npg[r] = np;
        pt[r] = kv.page_table + ((size_t)sq * kv.n_planes + plane) * kv.max_pages;
#pragma unroll
        for (int e = 0; e < DPL; ++e) qr[r][e] = q[(size_t)m * d + head * HD + li * DPL + e] * qscale;
    }

    float m_run[2] = {-1e30f, -1e30f}, l_run[2] = {0.f, 0.f};
    float acc0[DPL], acc1[DPL];
#pragma unroll
    for (int e = 0; e < DPL; ++e) {
        acc0[e] = 0.f;
        acc1[e] = 0.f;
    }

    // the concatenated page list of both rows, dealt round-robin to the waves
    const int n0 = npg[0], total = npg[0] + npg[1];
    auto page_ptr = [&](int item) -> const uint16_t* {
        const int r = item < n0 ? 0 : 1;
        const int p = item < n0 ? item : item - n0;
        const int pid = pt[r][p];
        if (pid < 0 || pid >= kv.n_pages) return nullptr;
        return kv.pool + kv_offset(kv.layer, pid, kv.n_pages, 0, head, H, 0, HD);
    };
    auto fetch = [&](const uint16_t* base, PageData<DPL>& pd) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int t = j * 4 + g;
            pd.k[j] = load_raw<DPL>(base + t * HD + li * DPL);
            pd.v[j] = load_raw<DPL>(base + vofs + t * HD + li * DPL);
        }
    };

    // (a one-page register prefetch of the next item measured no faster)
    for (int item = wave; item < total; item += kAttnWaves) {
        const uint16_t* base = page_ptr(item);
        if (!base) {
            if (lane == 0) set_err(err, CDB_DEV_UNMAPPED_PAGE);
            continue;
        }
        PageData<DPL> cur;
        fetch(base, cur);
        if (item < n0)
            attend_page<DPL>(cur, qr[0], item * kPage, n_ctx[0], g, m_run[0], l_run[0], acc0);
        else
            attend_page<DPL>(cur, qr[1], (item - n0) * kPage, n_ctx[1], g, m_run[1], l_run[1], acc1);
    }

    const int part = wave * 4 + g;
    if (li == 0) {
        s_m[0][part] = m_run[0];
        s_l[0][part] = l_run[0];
        s_m[1][part] = m_run[1];
        s_l[1][part] = l_run[1];
    }
#pragma unroll
    for (int e = 0; e < DPL; ++e) {
        s_acc[0][part][li * DPL + e] = acc0[e];
        s_acc[1][part][li * DPL + e] = acc1[e];
    }
    __syncthreads();
    if (tid < 2 * HD) {
        const int r = tid / HD, dim = tid - r * HD;
        const int m = rows[r];
        if (m >= 0 && valid[r]) {
            // merge in the order of the row's own page classes (page p lives in
            // partial (p + first) % waves), so a row's result does not depend on
            // the row it was paired with
            const int first = r == 0 ? 0 : n0 % kAttnWaves;
            float Mx = -1e30f;
            for (int i = 0; i < NP; ++i) Mx = fmaxf(Mx, s_m[r][i]);
            float num = 0.f, den = 0.f;
            for (int i = 0; i < NP; ++i) {
                const int j = ((first + (i >> 2)) % kAttnWaves) * 4 + (i & 3);
                const float w = exp2f(s_m[r][j] - Mx);
                num += w * s_acc[r][j][dim];
                den += w * s_l[r][j];
            }
            out[frag_index(m, head * HD + dim, d)] = f2bf(den > 0.f ? num / den : 0.f);
        }
    }
}

hipError_t launch_attention(const float* q, const KvTarget& kv, const int32_t* seq, const int32_t* pos,
                            const int32_t* order, int M, int H, int hd, uint16_t* out, int* err, hipStream_t st,
                            const int32_t* dn) {
    if (M <= 0) return hipSuccess;
    dim3 grid(H, (M + 1) / 2);
    switch (hd) {
        case 64: k_attn<64><<<grid, kAttnWaves * 64, 0, st>>>(q, kv, seq, pos, order, M, H, out, err, dn); break;
        case 96: k_attn<96><<<grid, kAttnWaves * 64, 0, st>>>(q, kv, seq, pos, order, M, H, out, err, dn); break;
        case 128: k_attn<128><<<grid, kAttnWaves * 64, 0, st>>>(q, kv, seq, pos, order, M, H, out, err, dn); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// order[rank] = row, ranked by descending position (ties by row index).  One
// workgroup; M <= 256.
__global__ __launch_bounds__(256) void k_row_order(const int32_t* __restrict__ pos, int M, int32_t* __restrict__ order,
                                                   const int32_t* __restrict__ dn) {
    M = live_rows(dn, M);
    for (int i = threadIdx.x; i < M; i += blockDim.x) {
        const int pi = pos[i];
        int rank = 0;
        for (int j = 0; j < M; ++j) {
            const int pj = pos[j];
            rank += (pj > pi) || (pj == pi && j < i);
        }
        order[rank] = i;
    }
}

hipError_t launch_row_order(const int32_t* pos, int M, int32_t* order, hipStream_t st, const int32_t* dn) {
    if (M <= 0) return hipSuccess;
    k_row_order<<<1, 256, 0, st>>>(pos, M, order, dn);
    return hipGetLastError();
}

}  // namespace cdb
