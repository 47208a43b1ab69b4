// Causal prefill attention on MFMA (v_mfma_f32_32x32x16_bf16) for chunked
// prefill: a chunk's rows attend to the stage plane's K/V of all earlier
// positions and of the chunk itself.
#include "cdb_internal.h"

namespace cdb {

// LDS reads written as inline assembly: the compiler cannot tell which LDS
// bytes the direct global->LDS loads in flight will write, and would make
// every compiler-visible LDS read wait for all of them.  Each helper issues a
// group of reads and waits for them in the same statement, so its outputs
// hold the data when the statement ends.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}
// N 16-byte reads, v[i] from byte address a[i]
template <int N>
__device__ __forceinline__ void lds_read_b128xN(u32x4 (&v)[N], const uint32_t (&a)[N]) {
    static_assert(N == 2 || N == 4 || N == 6 || N == 8, "read group size");
    if constexpr (N == 2) {
        asm volatile("ds_read_b128 %0, %2\n ds_read_b128 %1, %3\n s_waitcnt lgkmcnt(0)"
                     : "=&v"(v[0]), "=&v"(v[1]) : "v"(a[0]), "v"(a[1]) : "memory");
    } else if constexpr (N == 4) {
        asm volatile("ds_read_b128 %0, %4\n ds_read_b128 %1, %5\n ds_read_b128 %2, %6\n ds_read_b128 %3, %7\n"
                     " s_waitcnt lgkmcnt(0)"
                     : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3])
                     : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]) : "memory");
    } else if constexpr (N == 6) {
        asm volatile("ds_read_b128 %0, %6\n ds_read_b128 %1, %7\n ds_read_b128 %2, %8\n ds_read_b128 %3, %9\n"
                     " ds_read_b128 %4, %10\n ds_read_b128 %5, %11\n s_waitcnt lgkmcnt(0)"
                     : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(v[5])
                     : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]) : "memory");
    } else {
        asm volatile("ds_read_b128 %0, %8\n ds_read_b128 %1, %9\n ds_read_b128 %2, %10\n ds_read_b128 %3, %11\n"
                     " ds_read_b128 %4, %12\n ds_read_b128 %5, %13\n ds_read_b128 %6, %14\n ds_read_b128 %7, %15\n"
                     " s_waitcnt lgkmcnt(0)"
                     : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(v[5]), "=&v"(v[6]), "=&v"(v[7])
                     : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]), "v"(a[7])
                     : "memory");
    }
}
// V^T operands of NB 32-dim blocks: r[8b + e] gets the bf16 value at byte
// address a[e] + 64b (zero-extended; 16-bit loads into half registers do not
// keep the other half here), where a[e] is the lane's column in key row e.
template <int NB>
__device__ __forceinline__ void lds_read_vcols(uint32_t (&r)[32], const uint32_t (&a)[8]) {
    static_assert(NB >= 2 && NB <= 4, "32-dim blocks");
    // outputs are operands 0 .. 8NB-1, the 8 addresses follow
    if constexpr (NB == 2) {
        asm volatile("ds_read_u16 %0, %16 offset:0\n" "ds_read_u16 %1, %17 offset:0\n"
                     "ds_read_u16 %2, %18 offset:0\n" "ds_read_u16 %3, %19 offset:0\n"
                     "ds_read_u16 %4, %20 offset:0\n" "ds_read_u16 %5, %21 offset:0\n"
                     "ds_read_u16 %6, %22 offset:0\n" "ds_read_u16 %7, %23 offset:0\n"
                     "ds_read_u16 %8, %16 offset:64\n" "ds_read_u16 %9, %17 offset:64\n"
                     "ds_read_u16 %10, %18 offset:64\n" "ds_read_u16 %11, %19 offset:64\n"
                     "ds_read_u16 %12, %20 offset:64\n" "ds_read_u16 %13, %21 offset:64\n"
                     "ds_read_u16 %14, %22 offset:64\n" "ds_read_u16 %15, %23 offset:64\n"
                     " s_waitcnt lgkmcnt(0)"
                     : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]), "=&v"(r[6]),
                       "=&v"(r[7]), "=&v"(r[8]), "=&v"(r[9]), "=&v"(r[10]), "=&v"(r[11]), "=&v"(r[12]),
                       "=&v"(r[13]), "=&v"(r[14]), "=&v"(r[15])
                     : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]), "v"(a[7])
                     : "memory");
    } else if constexpr (NB == 3) {
        asm volatile("ds_read_u16 %0, %24 offset:0\n" "ds_read_u16 %1, %25 offset:0\n"
                     "ds_read_u16 %2, %26 offset:0\n" "ds_read_u16 %3, %27 offset:0\n"
                     "ds_read_u16 %4, %28 offset:0\n" "ds_read_u16 %5, %29 offset:0\n"
                     "ds_read_u16 %6, %30 offset:0\n" "ds_read_u16 %7, %31 offset:0\n"
                     "ds_read_u16 %8, %24 offset:64\n" "ds_read_u16 %9, %25 offset:64\n"
                     "ds_read_u16 %10, %26 offset:64\n" "ds_read_u16 %11, %27 offset:64\n"
                     "ds_read_u16 %12, %28 offset:64\n" "ds_read_u16 %13, %29 offset:64\n"
                     "ds_read_u16 %14, %30 offset:64\n" "ds_read_u16 %15, %31 offset:64\n"
                     "ds_read_u16 %16, %24 offset:128\n" "ds_read_u16 %17, %25 offset:128\n"
                     "ds_read_u16 %18, %26 offset:128\n" "ds_read_u16 %19, %27 offset:128\n"
                     "ds_read_u16 %20, %28 offset:128\n" "ds_read_u16 %21, %29 offset:128\n"
                     "ds_read_u16 %22, %30 offset:128\n" "ds_read_u16 %23, %31 offset:128\n"
                     " s_waitcnt lgkmcnt(0)"
                     : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]), "=&v"(r[6]),
                       "=&v"(r[7]), "=&v"(r[8]), "=&v"(r[9]), "=&v"(r[10]), "=&v"(r[11]), "=&v"(r[12]),
                       "=&v"(r[13]), "=&v"(r[14]), "=&v"(r[15]), "=&v"(r[16]), "=&v"(r[17]), "=&v"(r[18]),
                       "=&v"(r[19]), "=&v"(r[20]), "=&v"(r[21]), "=&v"(r[22]), "=&v"(r[23])
                     : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]), "v"(a[7])
                     : "memory");
    } else {
        asm volatile("ds_read_u16 %0, %32 offset:0\n" "ds_read_u16 %1, %33 offset:0\n"
                     "ds_read_u16 %2, %34 offset:0\n" "ds_read_u16 %3, %35 offset:0\n"
                     "ds_read_u16 %4, %36 offset:0\n" "ds_read_u16 %5, %37 offset:0\n"
                     "ds_read_u16 %6, %38 offset:0\n" "ds_read_u16 %7, %39 offset:0\n"
                     "ds_read_u16 %8, %32 offset:64\n" "ds_read_u16 %9, %33 offset:64\n"
                     "ds_read_u16 %10, %34 offset:64\n" "ds_read_u16 %11, %35 offset:64\n"
                     "ds_read_u16 %12, %36 offset:64\n" "ds_read_u16 %13, %37 offset:64\n"
                     "ds_read_u16 %14, %38 offset:64\n" "ds_read_u16 %15, %39 offset:64\n"
                     "ds_read_u16 %16, %32 offset:128\n" "ds_read_u16 %17, %33 offset:128\n"
                     "ds_read_u16 %18, %34 offset:128\n" "ds_read_u16 %19, %35 offset:128\n"
                     "ds_read_u16 %20, %36 offset:128\n" "ds_read_u16 %21, %37 offset:128\n"
                     "ds_read_u16 %22, %38 offset:128\n" "ds_read_u16 %23, %39 offset:128\n"
                     "ds_read_u16 %24, %32 offset:192\n" "ds_read_u16 %25, %33 offset:192\n"
                     "ds_read_u16 %26, %34 offset:192\n" "ds_read_u16 %27, %35 offset:192\n"
                     "ds_read_u16 %28, %36 offset:192\n" "ds_read_u16 %29, %37 offset:192\n"
                     "ds_read_u16 %30, %38 offset:192\n" "ds_read_u16 %31, %39 offset:192\n"
                     " s_waitcnt lgkmcnt(0)"
                     : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]), "=&v"(r[6]),
                       "=&v"(r[7]), "=&v"(r[8]), "=&v"(r[9]), "=&v"(r[10]), "=&v"(r[11]), "=&v"(r[12]),
                       "=&v"(r[13]), "=&v"(r[14]), "=&v"(r[15]), "=&v"(r[16]), "=&v"(r[17]), "=&v"(r[18]),
                       "=&v"(r[19]), "=&v"(r[20]), "=&v"(r[21]), "=&v"(r[22]), "=&v"(r[23]), "=&v"(r[24]),
                       "=&v"(r[25]), "=&v"(r[26]), "=&v"(r[27]), "=&v"(r[28]), "=&v"(r[29]), "=&v"(r[30]),
                       "=&v"(r[31])
                     : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]), "v"(a[7])
                     : "memory");
    }
}

// Causal attention of a prefill chunk: rows 0..M-1 are positions pos0..pos0+M-1
// of one sequence; row i attends to positions 0..pos0+i of its plane.  A dense
// contraction, so it runs on MFMA (v_mfma_f32_32x32x16_bf16).
//
// Workgroup = (head, 32 rows), 4 waves splitting the keys in blocks of 32
// (wave w takes blocks w, w + 4, ...).  Each wave streams its blocks from HBM
// straight into a private double buffer in LDS with direct loads (K rows with
// their 16-byte chunks rotated by the key index, so the operand reads of 32
// rows at one column hit distinct banks; V rows as stored), one block ahead of
// the one it computes, so no barrier sits in the loop.  Each wave keeps an
// online softmax state for the 32 rows; the four states are merged through LDS
// at the end.  Per wave and block:
//   S^T = K Q^T: A = K rows (keys), B = q (queries), 16 dims per MFMA.  q is
//     split into bf16 hi + lo parts (two independent MFMA chains), keeping the
//     scores at about 16 mantissa bits; K is bf16 already.  Lane l ends up
//     with query l % 32 and 16 of its 32 keys; lane l ^ 32 holds the other 16.
//   online softmax per query in the exp2 domain (one lane swap per reduction);
//   O^T += V^T P^T: A = V^T (dims x keys, gathered from the key-major rows
//     with 2-byte LDS reads), B = P (keys x queries, regrouped by one lane
//     swap), P split hi + lo as well.
// The output is normalised and written in bf16 fragment layout.
template <int HD>
__global__ __launch_bounds__(256) void k_prefill_attn(const float* __restrict__ q, KvTarget kv, int seq, int pos0,
                                                      int M, int H, uint16_t* __restrict__ out, int* err) {
    constexpr int KB = 32;              // keys per block
    constexpr int CPK = HD / 8;         // 16-byte chunks per key row
    constexpr int NDB = HD / 32;        // 32-dim output blocks
    constexpr int BLK = KB * HD * 2;    // bytes of one block of K (or of V)
    constexpr int WBUF = 2 * 2 * BLK;   // a wave's two buffers of K and V
    constexpr int NDMA = KB * CPK / 64; // 1 KiB direct loads per block and tensor
    constexpr int QP = HD + 4;          // q tile row pitch (floats)
    static_assert(KB * CPK % 64 == 0, "a block is whole 1 KiB loads");
    static_assert(4 * HD * 32 * 4 + 4 * 64 * 4 <= 4 * WBUF, "merge buffers fit the wave buffers");
    __shared__ __align__(16) unsigned char smem[4 * WBUF + 32 * QP * 4];
    __shared__ int s_pid[kMaxPrefillPos / kPage];  // page ids of the key range
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
    if (n_pg > kMaxPrefillPos / kPage) {  // the launcher bounds the context; kept as a guard
        if (tid == 0) set_err(err, CDB_DEV_BAD_INDEX);
        return;
    }
    for (int i = tid; i < n_pg; i += 256) {
        const int pid = i < kv.max_pages ? pt[i] : -1;
        s_pid[i] = pid >= 0 && pid < kv.n_pages ? pid : -1;
        if (s_pid[i] < 0) set_err(err, CDB_DEV_UNMAPPED_PAGE);
    }
    // q tile (32 rows x HD, fp32), coalesced 16-byte loads
    float* sq = reinterpret_cast<float*>(smem + 4 * WBUF);
    for (int i = tid; i < 32 * (HD / 4); i += 256) {
        const int r = i / (HD / 4), c4 = i - r * (HD / 4);
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (row0 + r < M) v = *reinterpret_cast<const float4*>(q + (size_t)(row0 + r) * d + head * HD + c4 * 4);
        *reinterpret_cast<float4*>(sq + r * QP + c4 * 4) = v;
    }
    __syncthreads();  // q tile and page ids

    // block kb (keys kb .. kb + 31) into buffer b: K row `key` keeps chunk c at
    // position (c + key) % CPK; keys past `last` repeat the last key (masked)
    unsigned char* wbase = smem + wave * WBUF;
    auto issue = [&](int kb, int b) {
        unsigned char* kd = wbase + b * 2 * BLK;
#pragma unroll
        for (int i = 0; i < NDMA; ++i) {
            const int f = i * 64 + lane;  // chunk slot within the block
            const int key = f / CPK, pos = f - key * CPK;
            const int rot = key % CPK;
            const int c = pos >= rot ? pos - rot : pos - rot + CPK;
            const int kp = min(kb + key, last);
            const int pid = max(s_pid[kp / kPage], 0);  // unmapped pages were reported above
            const u32x4* kr = reinterpret_cast<const u32x4*>(
                kv.pool + kv_offset(kv.layer, pid, kv.n_pages, 0, head, H, kp % kPage, HD));
            const u32x4* vr = reinterpret_cast<const u32x4*>(
                kv.pool + kv_offset(kv.layer, pid, kv.n_pages, 1, head, H, kp % kPage, HD));
            __builtin_amdgcn_global_load_lds(kr + c, (__attribute__((address_space(3))) void*)(kd + i * 1024), 16, 0, 0);
            __builtin_amdgcn_global_load_lds(vr + pos, (__attribute__((address_space(3))) void*)(kd + BLK + i * 1024),
                                             16, 0, 0);
        }
    };
    int kb = wave * KB;
    if (kb <= last) issue(kb, 0);

    // q operands: dims 16t + 8*(lane/32) + e of row lane%32, scaled and split into bf16 hi + lo
    bf16x8 qh[HD / 16], ql[HD / 16];
#pragma unroll
    for (int t = 0; t < HD / 16; ++t) {
        const float* src = sq + (lane & 31) * QP + t * 16 + (lane >> 5) * 8;
        u32x4 qv[2];
        const uint32_t qa[2] = {lds_addr(src), lds_addr(src + 4)};
        lds_read_b128xN(qv, qa);
        const float4 a = __builtin_bit_cast(float4, qv[0]), b = __builtin_bit_cast(float4, qv[1]);
        const float x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
        uint32_t hw[4], lw[4];
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
            const float x0 = x[e] * qscale, x1 = x[e + 1] * qscale;
            const uint32_t h = pack_bf16(x0, x1);
            hw[e / 2] = h;
            lw[e / 2] = pack_bf16(x0 - bflo(h), x1 - bfhi(h));
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

    for (int b = 0; kb <= last; kb += 4 * KB, b ^= 1) {
        if (kb + 4 * KB <= last) {
            issue(kb + 4 * KB, b ^ 1);
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * NDMA) : "memory");
        } else {
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        }
        const uint16_t* sK = reinterpret_cast<const uint16_t*>(wbase + b * 2 * BLK);
        const uint16_t* sV = sK + KB * HD;
        // S^T[key][query] for the 32 queries
        floatx16 sc, sl;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            sc[j] = 0.f;
            sl[j] = 0.f;
        }
        const int krow = lane & 31;
        u32x4 ka[HD / 16];
        uint32_t kaddr[HD / 16];
#pragma unroll
        for (int t = 0; t < HD / 16; ++t) {
            const int c = t * 2 + (lane >> 5);
            const int pos = (c + krow) % CPK;
            kaddr[t] = lds_addr(sK + (krow * CPK + pos) * 8);
        }
        lds_read_b128xN(ka, kaddr);
#pragma unroll
        for (int t = 0; t < HD / 16; ++t) {
            const bf16x8 a = __builtin_bit_cast(bf16x8, ka[t]);
            sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qh[t], sc, 0, 0, 0);
            sl = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, ql[t], sl, 0, 0, 0);
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
        for (int b2 = 0; b2 < NDB; ++b2)
#pragma unroll
            for (int j = 0; j < 16; ++j) o[b2][j] *= corr;

        // regroup P for the B operand: k step st needs keys 16st + 8*(lane/32) + e
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
                const uint32_t h = pack_bf16(pk[e], pk[e + 1]);
                hw[e / 2] = h;
                lw[e / 2] = pack_bf16(pk[e] - bflo(h), pk[e + 1] - bfhi(h));
            }
            const bf16x8 ph = __builtin_bit_cast(bf16x8, u32x4{hw[0], hw[1], hw[2], hw[3]});
            const bf16x8 pl = __builtin_bit_cast(bf16x8, u32x4{lw[0], lw[1], lw[2], lw[3]});
            // V^T operand: dim 32b + lane%32, keys 16st + 8*(lane/32) .. + 7
            const uint32_t vcol = lds_addr(sV + (st * 16 + (lane >> 5) * 8) * HD + (lane & 31));
            uint32_t vaddr[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) vaddr[e] = vcol + e * HD * 2;
            uint32_t vr[32];
            lds_read_vcols<NDB>(vr, vaddr);
#pragma unroll
            for (int b2 = 0; b2 < NDB; ++b2) {
                const uint32_t* r8 = vr + 8 * b2;
                const bf16x8 a = __builtin_bit_cast(
                    bf16x8, u32x4{r8[0] | (r8[1] << 16), r8[2] | (r8[3] << 16), r8[4] | (r8[5] << 16), r8[6] | (r8[7] << 16)});
                o[b2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, ph, o[b2], 0, 0, 0);
                o[b2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pl, o[b2], 0, 0, 0);
            }
        }
    }
    __syncthreads();  // every wave is done with its buffers

    // merge the four waves' states: O^T[dim][query] with lane holding query
    // lane%32 and dims 32b + (j/4)*8 + (lane/32)*4 + j%4
    float* sO = reinterpret_cast<float*>(smem);  // [4 waves][HD][32]
    float* sM = sO + 4 * HD * 32;                // [4][32] maxima, then [4][32] sums
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
            pk[i / 2] = pack_bf16(den > 0.f ? num[0] / den : 0.f, den > 0.f ? num[1] / den : 0.f);
        }
        *reinterpret_cast<u32x4*>(out + frag_index(row, head * HD + c8 * 8, d)) = u32x4{pk[0], pk[1], pk[2], pk[3]};
    }
}

hipError_t launch_prefill_attention(const float* q, const KvTarget& kv, int seq, int pos0, int M, int H, int hd,
                                    uint16_t* out, int* err, hipStream_t st) {
    if (M <= 0) return hipSuccess;
    if (pos0 + M > kMaxPrefillPos) return hipErrorInvalidValue;  // page ids of the key range must fit in LDS
    if (kv.n_pages < 1 || !kv.pool) return hipErrorInvalidValue;
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
