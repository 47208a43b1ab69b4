// Paged decode attention over the depth-indexed KV cache.
//
// One query per (row, head): the row's q (after RoPE) attends to positions
// 0..pos of its sequence in one KV plane (the row's loop plane for the core,
// the stage plane for prelude/coda).  HBM-bound: every K/V byte is read once
// and used by one query, so the kernel is built for streaming, not MFMA.
//
// Layout of one page for one (layer, head): K [16 tokens][hd] then (after
// H*16*hd elements) V [16][hd], bf16.  A wave reads a page as four
// coalesced loads for K and four for V: lane l covers token (4*j + l/16) and
// dims [(l%16)*hd/16, +hd/16).  The 16 lanes of a DPP row reduce q.k with row
// DPP (quad_perm, half_mirror, mirror), and each row keeps its own online
// softmax over the tokens it owns, so no cross-row traffic happens per page.
// A workgroup of 4 waves takes one (row, head); wave w takes pages w, w+4, ...
// The 16 partial (max, sum, acc) states are merged through LDS at the end; the
// output is written in the fragment layout the output projection reads.
#include "cdb_internal.h"

namespace cdb {

template <int DPL>
__device__ __forceinline__ void load_vec(const uint16_t* p, float* out) {
    if constexpr (DPL == 8) {
        const uint4 w = *reinterpret_cast<const uint4*>(p);
        out[0] = bflo(w.x); out[1] = bfhi(w.x); out[2] = bflo(w.y); out[3] = bfhi(w.y);
        out[4] = bflo(w.z); out[5] = bfhi(w.z); out[6] = bflo(w.w); out[7] = bfhi(w.w);
    } else if constexpr (DPL == 4) {
        const uint2 w = *reinterpret_cast<const uint2*>(p);
        out[0] = bflo(w.x); out[1] = bfhi(w.x); out[2] = bflo(w.y); out[3] = bfhi(w.y);
    } else {
        const uint32_t* q = reinterpret_cast<const uint32_t*>(p);
        const uint32_t a = q[0], b = q[1], c = q[2];
        out[0] = bflo(a); out[1] = bfhi(a); out[2] = bflo(b); out[3] = bfhi(b); out[4] = bflo(c); out[5] = bfhi(c);
    }
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

template <int HD>
__global__ __launch_bounds__(256) void k_attn(const float* __restrict__ q, KvTarget kv, const int32_t* __restrict__ seq,
                                              const int32_t* __restrict__ pos, int H, uint16_t* __restrict__ out,
                                              int* err) {
    constexpr int DPL = HD / 16;
    __shared__ float s_m[16], s_l[16];
    __shared__ float s_acc[16][HD];
    const int head = blockIdx.x, m = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, li = lane & 15;
    const int d = H * HD;
    const float qscale = 1.4426950408889634f / sqrtf((float)HD);  // log2(e) / sqrt(hd)

    float qr[DPL];
#pragma unroll
    for (int e = 0; e < DPL; ++e) qr[e] = q[(size_t)m * d + head * HD + li * DPL + e] * qscale;

    const int sq = seq[m], ps = pos[m];
    const int plane = kv.c_row ? kv.c_row[m] + 1 : kv.plane_fixed;
    const int n_ctx = ps + 1;
    const int npg = (n_ctx + kPage - 1) / kPage;
    const size_t page_elems = (size_t)kv.n_layers * 2 * H * kPage * HD;
    const size_t kofs = (((size_t)kv.layer * 2) * H + head) * kPage * HD;
    const size_t vofs = kofs + (size_t)H * kPage * HD;
    const bool row_ok = sq >= 0 && sq < kv.max_seqs && plane >= 0 && plane < kv.n_planes && npg <= kv.max_pages;
    const int32_t* pt = kv.page_table + ((size_t)(row_ok ? sq : 0) * kv.n_planes + (row_ok ? plane : 0)) * kv.max_pages;

    float m_run = -1e30f, l_run = 0.f;
    float acc[DPL];
#pragma unroll
    for (int e = 0; e < DPL; ++e) acc[e] = 0.f;

    if (row_ok) {
        for (int p = wave; p < npg; p += 4) {
            const int pid = pt[p];
            if (pid < 0 || pid >= kv.n_pages) {
                if (lane == 0) set_err(err, CDB_DEV_UNMAPPED_PAGE);
                continue;
            }
            const uint16_t* kb = kv.pool + (size_t)pid * page_elems + kofs;
            const uint16_t* vb = kv.pool + (size_t)pid * page_elems + vofs;
            float kf[4][DPL], vf[4][DPL];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int t = j * 4 + g;
                load_vec<DPL>(kb + t * HD + li * DPL, kf[j]);
                load_vec<DPL>(vb + t * HD + li * DPL, vf[j]);
            }
            float sc[4];
            float mx = m_run;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                float dot = 0.f;
#pragma unroll
                for (int e = 0; e < DPL; ++e) dot += qr[e] * kf[j][e];
                dot = row_sum16(dot);
                const bool valid = p * kPage + j * 4 + g < n_ctx;
                sc[j] = valid ? dot : -1e30f;
                mx = fmaxf(mx, sc[j]);
            }
            const float corr = exp2f(m_run - mx);
            l_run *= corr;
#pragma unroll
            for (int e = 0; e < DPL; ++e) acc[e] *= corr;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const bool valid = p * kPage + j * 4 + g < n_ctx;
                const float pj = valid ? exp2f(sc[j] - mx) : 0.f;
                l_run += pj;
#pragma unroll
                for (int e = 0; e < DPL; ++e) acc[e] += valid ? pj * vf[j][e] : 0.f;
            }
            m_run = mx;
        }
    } else if (tid == 0) {
        set_err(err, CDB_DEV_UNMAPPED_PAGE);
    }

    const int part = wave * 4 + g;
    if (li == 0) {
        s_m[part] = m_run;
        s_l[part] = l_run;
    }
#pragma unroll
    for (int e = 0; e < DPL; ++e) s_acc[part][li * DPL + e] = acc[e];
    __syncthreads();
    if (tid < HD) {
        float M = -1e30f;
        for (int i = 0; i < 16; ++i) M = fmaxf(M, s_m[i]);
        float num = 0.f, den = 0.f;
        for (int i = 0; i < 16; ++i) {
            const float w = exp2f(s_m[i] - M);
            num += w * s_acc[i][tid];
            den += w * s_l[i];
        }
        out[frag_index(m, head * HD + tid, d)] = f2bf(den > 0.f ? num / den : 0.f);
    }
}

hipError_t launch_attention(const float* q, const KvTarget& kv, const int32_t* seq, const int32_t* pos, int M, int H,
                            int hd, uint16_t* out, int* err, hipStream_t st) {
    if (M <= 0) return hipSuccess;
    dim3 grid(H, M);
    switch (hd) {
        case 64: k_attn<64><<<grid, 256, 0, st>>>(q, kv, seq, pos, H, out, err); break;
        case 96: k_attn<96><<<grid, 256, 0, st>>>(q, kv, seq, pos, H, out, err); break;
        case 128: k_attn<128><<<grid, 256, 0, st>>>(q, kv, seq, pos, H, out, err); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace cdb
