// Causal prefill attention on MFMA (v_mfma_f32_32x32x16_bf16) for chunked
// prefill: a chunk's rows attend to the stage plane's K/V of all earlier
// positions and of the chunk itself.
#include "cdb_internal.h"

namespace cdb {

// Causal attention of a prefill chunk: rows 0..M-1 are positions pos0..pos0+M-1
// of one sequence; row i attends to positions 0..pos0+i of its plane.  A dense
// contraction, so it runs on MFMA (v_mfma_f32_32x32x16_bf16).
//
// Workgroup = (head, 32 rows), 4 waves splitting the keys: the workgroup
// stages 4 blocks of 32 keys at a time in LDS (K rows as stored, V transposed
// to dims x keys so both operands read as 16-byte vectors) and wave w takes
// block w.  Each wave keeps an online softmax state for the 32 rows; the four
// states are merged through LDS at the end.  Per wave and block:
//   S^T = K Q^T: A = K rows (keys), B = q (queries), 16 dims per MFMA.  q is
//     split into bf16 hi + lo parts (two independent MFMA chains), keeping the
//     scores at about 16 mantissa bits; K is bf16 already.  Lane l ends up
//     with query l % 32 and 16 of its 32 keys; lane l ^ 32 holds the other 16.
//   online softmax per query in the exp2 domain (one lane swap per reduction);
//   O^T += V^T P^T: A = V^T (dims x keys), B = P (keys x queries, regrouped
//     by one lane swap), P split hi + lo as well.
// The output is normalised and written in bf16 fragment layout.
template <int HD>
__global__ __launch_bounds__(256) void k_prefill_attn(const float* __restrict__ q, KvTarget kv, int seq, int pos0,
                                                      int M, int H, uint16_t* __restrict__ out, int* err) {
    constexpr int KB = 32;                         // keys per block
    constexpr int LD = HD + 8;                     // K row pitch (bf16), 16-byte pad
    constexpr int LV = KB + 8;                     // V^T row pitch (bf16)
    constexpr int NDB = HD / 32;                   // 32-dim output blocks
    constexpr int KBYTES = KB * LD * 2, VBYTES = HD * LV * 2;
    constexpr int SLOT = KBYTES + VBYTES;          // one block's staging
    constexpr int PIECES = 4 * 2 * KB * (HD / 8);  // 16-byte pieces of 4 blocks of K and V
    static_assert(4 * HD * 32 * 4 + 4 * 64 * 4 <= 4 * SLOT, "merge buffers fit the staging area");
    __shared__ __align__(16) unsigned char smem[4 * SLOT];
    __shared__ int s_pid[640];                     // page ids of the key range (10240 positions)
    const int head = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int d = H * HD;
    const int row0 = blockIdx.y * 32;
    const int qrow = row0 + (lane & 31);  // this lane's query row
    const bool qvalid = qrow < M;
    const int qpos = pos0 + qrow;
    const int last = pos0 + min(M, row0 + 32) - 1;  // last position any row of the tile needs
    const float qscale = 1.4426950408889634f / sqrtf((float)HD);
    const int32_t* pt = kv.page_table + ((size_t)seq * kv.n_planes + kv.plane_fixed) * kv.max_pages;

    const int n_pg = last / kPage + 1;
    if (n_pg > 640) {  // the launcher bounds the context; kept as a guard
        if (tid == 0) set_err(err, CDB_DEV_BAD_INDEX);
        return;
    }
    for (int i = tid; i < n_pg; i += 256) {
        const int pid = i < kv.max_pages ? pt[i] : -1;
        s_pid[i] = pid >= 0 && pid < kv.n_pages ? pid : -1;
        if (s_pid[i] < 0) set_err(err, CDB_DEV_UNMAPPED_PAGE);
    }

    // q tile (32 rows x HD, fp32) through LDS: coalesced 16-byte loads, then
    // each lane takes its B-operand dims 16t + 8*(lane/32) + e of row lane%32,
    // scaled and split into bf16 hi + lo
    constexpr int QP = HD + 4;  // row pitch (floats)
    static_assert(32 * QP * 4 <= 4 * SLOT, "q tile fits the staging area");
    float* sq = reinterpret_cast<float*>(smem);
    for (int i = tid; i < 32 * (HD / 4); i += 256) {
        const int r = i / (HD / 4), c4 = i - r * (HD / 4);
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (row0 + r < M) v = *reinterpret_cast<const float4*>(q + (size_t)(row0 + r) * d + head * HD + c4 * 4);
        *reinterpret_cast<float4*>(sq + r * QP + c4 * 4) = v;
    }
    __syncthreads();  // q tile and page ids
    bf16x8 qh[HD / 16], ql[HD / 16];
#pragma unroll
    for (int t = 0; t < HD / 16; ++t) {
        const float* src = sq + (lane & 31) * QP + t * 16 + (lane >> 5) * 8;
        const float4 a = *reinterpret_cast<const float4*>(src), b = *reinterpret_cast<const float4*>(src + 4);
        const float x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
        uint32_t hw[4], lw[4];
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
            const float x0 = x[e] * qscale, x1 = x[e + 1] * qscale;
            const uint16_t h0 = f2bf(x0), h1 = f2bf(x1);
            const uint16_t l0 = f2bf(x0 - bf2f(h0)), l1 = f2bf(x1 - bf2f(h1));
            hw[e / 2] = (uint32_t)h0 | ((uint32_t)h1 << 16);
            lw[e / 2] = (uint32_t)l0 | ((uint32_t)l1 << 16);
        }
        qh[t] = __builtin_bit_cast(bf16x8, u32x4{hw[0], hw[1], hw[2], hw[3]});
        ql[t] = __builtin_bit_cast(bf16x8, u32x4{lw[0], lw[1], lw[2], lw[3]});
    }

    floatx16 o[NDB];
#pragma unroll
    for (int b = 0; b < NDB; ++b)
#pragma unroll
        for (int j = 0; j < 16; ++j) o[b][j] = 0.f;
    float m_run = -1e30f, l_run = 0.f;
    uint16_t* sK = reinterpret_cast<uint16_t*>(smem + wave * SLOT);
    uint16_t* sVt = reinterpret_cast<uint16_t*>(smem + wave * SLOT + KBYTES);
    __syncthreads();  // the q tile is read before the staging area is reused

    for (int sb = 0; sb <= last; sb += 4 * KB) {
        // stage keys sb .. sb + 127: block w in slot w; loads in batches of 4
        // per thread, issued before their LDS writes
        constexpr int PPT = PIECES / 256, SB = 4;
        static_assert(PPT % SB == 0, "staging batches");
#pragma unroll
        for (int b0 = 0; b0 < PPT; b0 += SB) {
            u32x4 v[SB];
            int slot_off[SB], which_k[SB];
#pragma unroll
            for (int i = 0; i < SB; ++i) {
                const int p = tid + (b0 + i) * 256;
                const int blk = p / (2 * KB * (HD / 8));
                const int r0 = p - blk * 2 * KB * (HD / 8);
                const int which = r0 / (KB * (HD / 8));
                const int r = r0 - which * KB * (HD / 8);
                const int key = r / (HD / 8), c8 = r - key * (HD / 8);
                const int kp = sb + blk * KB + key;
                v[i] = u32x4{0u, 0u, 0u, 0u};
                if (kp <= last) {
                    const int pid = s_pid[kp / kPage];
                    if (pid >= 0)
                        v[i] = *reinterpret_cast<const u32x4*>(
                            kv.pool + kv_offset(kv.layer, pid, kv.n_pages, which, head, H, kp % kPage, HD) + c8 * 8);
                }
                slot_off[i] = blk * SLOT + (which == 0 ? (key * LD + c8 * 8) * 2 : KBYTES + (c8 * 8 * LV + key) * 2);
                which_k[i] = which;
            }
#pragma unroll
            for (int i = 0; i < SB; ++i) {
                if (which_k[i] == 0) {
                    *reinterpret_cast<u32x4*>(smem + slot_off[i]) = v[i];
                } else {
                    uint16_t* vt = reinterpret_cast<uint16_t*>(smem + slot_off[i]);
                    const uint32_t w[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
#pragma unroll
                    for (int e = 0; e < 8; ++e) vt[e * LV] = (uint16_t)(w[e >> 1] >> ((e & 1) * 16));
                }
            }
        }
        __syncthreads();
        const int kb = sb + wave * KB;
        if (kb <= last) {
            // S^T[key][query] for the 32 queries
            floatx16 sc, sl;
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                sc[j] = 0.f;
                sl[j] = 0.f;
            }
#pragma unroll
            for (int t = 0; t < HD / 16; ++t) {
                const bf16x8 ka = *reinterpret_cast<const bf16x8*>(sK + (lane & 31) * LD + t * 16 + (lane >> 5) * 8);
                sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qh[t], sc, 0, 0, 0);
                sl = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, ql[t], sl, 0, 0, 0);
            }
            // causal mask and online softmax; lane holds keys (j/4)*8 + (lane/32)*4 + j%4
            float mx = -1e30f;
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int kp = kb + (j >> 2) * 8 + (lane >> 5) * 4 + (j & 3);
                const bool ok = qvalid && kp <= qpos;
                sc[j] = ok ? sc[j] + sl[j] : -1e30f;
                mx = fmaxf(mx, sc[j]);
            }
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float m_new = fmaxf(m_run, mx);
            const float corr = exp2f(m_run - m_new);
            float ls = 0.f;
            float p[16];
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                p[j] = sc[j] > -1e29f ? exp2f(sc[j] - m_new) : 0.f;
                ls += p[j];
            }
            ls += __shfl_xor(ls, 32);
            l_run = l_run * corr + ls;
            m_run = m_new;
#pragma unroll
            for (int b = 0; b < NDB; ++b)
#pragma unroll
                for (int j = 0; j < 16; ++j) o[b][j] *= corr;

            // regroup P for the B operand: k step s needs keys 16s + 8*(lane/32) + e
            const bool lo_half = lane < 32;
            float mine[8], theirs[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                mine[e] = lo_half ? p[4 + e] : p[e];  // what the partner lane needs from this lane
                mine[4 + e] = lo_half ? p[12 + e] : p[8 + e];
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) theirs[e] = __shfl_xor(mine[e], 32);
#pragma unroll
            for (int st = 0; st < 2; ++st) {
                float pk[8];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    // lanes < 32: own keys first, then the partner's; lanes >= 32 the reverse
                    pk[e] = lo_half ? p[st * 8 + e] : theirs[st * 4 + e];
                    pk[4 + e] = lo_half ? theirs[st * 4 + e] : p[st * 8 + 4 + e];
                }
                uint32_t hw[4], lw[4];
#pragma unroll
                for (int e = 0; e < 8; e += 2) {
                    const uint16_t h0 = f2bf(pk[e]), h1 = f2bf(pk[e + 1]);
                    const uint16_t l0 = f2bf(pk[e] - bf2f(h0)), l1 = f2bf(pk[e + 1] - bf2f(h1));
                    hw[e / 2] = (uint32_t)h0 | ((uint32_t)h1 << 16);
                    lw[e / 2] = (uint32_t)l0 | ((uint32_t)l1 << 16);
                }
                const bf16x8 ph = __builtin_bit_cast(bf16x8, u32x4{hw[0], hw[1], hw[2], hw[3]});
                const bf16x8 pl = __builtin_bit_cast(bf16x8, u32x4{lw[0], lw[1], lw[2], lw[3]});
                // V^T operand: dims 32b + lane%32, keys 16st + 8*(lane/32) .. + 7
#pragma unroll
                for (int b = 0; b < NDB; ++b) {
                    const bf16x8 va = *reinterpret_cast<const bf16x8*>(sVt + (b * 32 + (lane & 31)) * LV + st * 16 +
                                                                       (lane >> 5) * 8);
                    o[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, ph, o[b], 0, 0, 0);
                    o[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pl, o[b], 0, 0, 0);
                }
            }
        }
        __syncthreads();  // the slots are restaged next
    }

    // merge the four waves' states: O^T[dim][query] with lane holding query
    // lane%32 and dims 32b + (j/4)*8 + (lane/32)*4 + j%4
    float* sO = reinterpret_cast<float*>(smem);          // [4 waves][HD][32]
    float* sM = sO + 4 * HD * 32;                         // [4][32] maxima, then [4][32] sums
    float* sL = sM + 4 * 32;
#pragma unroll
    for (int b = 0; b < NDB; ++b)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int dim = b * 32 + (j >> 2) * 8 + (lane >> 5) * 4 + (j & 3);
            sO[(wave * HD + dim) * 32 + (lane & 31)] = o[b][j];
        }
    if (lane < 32) {
        sM[wave * 32 + lane] = m_run;
        sL[wave * 32 + lane] = l_run;
    }
    __syncthreads();
    // (row, 8-dim run) per item: one 16-byte store in the fragment layout
    for (int e = tid; e < 32 * (HD / 8); e += 256) {
        const int qq = e & 31, c8 = e >> 5;
        const int row = row0 + qq;
        if (row >= M) continue;
        float mx = -1e30f;
#pragma unroll
        for (int w = 0; w < 4; ++w) mx = fmaxf(mx, sM[w * 32 + qq]);
        float f[4], den = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            f[w] = exp2f(sM[w * 32 + qq] - mx);
            den += f[w] * sL[w * 32 + qq];
        }
        uint32_t pk[4];
#pragma unroll
        for (int i = 0; i < 8; i += 2) {
            float num[2] = {0.f, 0.f};
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                num[0] += f[w] * sO[(w * HD + c8 * 8 + i) * 32 + qq];
                num[1] += f[w] * sO[(w * HD + c8 * 8 + i + 1) * 32 + qq];
            }
            pk[i / 2] = (uint32_t)f2bf(den > 0.f ? num[0] / den : 0.f) |
                        ((uint32_t)f2bf(den > 0.f ? num[1] / den : 0.f) << 16);
        }
        *reinterpret_cast<u32x4*>(out + frag_index(row, head * HD + c8 * 8, d)) = u32x4{pk[0], pk[1], pk[2], pk[3]};
    }
}

hipError_t launch_prefill_attention(const float* q, const KvTarget& kv, int seq, int pos0, int M, int H, int hd,
                                    uint16_t* out, int* err, hipStream_t st) {
    if (M <= 0) return hipSuccess;
    if (pos0 + M > 640 * kPage) return hipErrorInvalidValue;  // page ids of the key range must fit in LDS
    dim3 grid(H, (M + 31) / 32);
    switch (hd) {
        case 64: k_prefill_attn<64><<<grid, 256, 0, st>>>(q, kv, seq, pos0, M, H, out, err); break;
        case 96: k_prefill_attn<96><<<grid, 256, 0, st>>>(q, kv, seq, pos0, M, H, out, err); break;
        case 128: k_prefill_attn<128><<<grid, 256, 0, st>>>(q, kv, seq, pos0, M, H, out, err); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace cdb
