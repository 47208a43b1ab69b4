// Internal declarations shared by the libcdb translation units (device helpers,
// packed-weight layout, workspace layout, kernel launchers).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/libcdb.h"

namespace cdb {

constexpr int kPage = 16;       // tokens per KV page
constexpr int kMaxRows = 256;          // rows per stage call
constexpr int kMaxPrefillRows = 512;   // rows per prefill chunk
constexpr int kMaxPrefillPos = 10240;  // positions one prefill call spans (key-range page ids sit in LDS)

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- bf16 helpers
__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }
__device__ __forceinline__ float bflo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bfhi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
// fp32 -> bf16, round to nearest even, by the gfx950 conversion instruction
// (v_cvt_pk_bf16_f32; fp32 denormals are kept, NaN stays NaN).
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
// Two values in one instruction: a in the low half, b in the high half.
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((floatx2){a, b}, bf16x2));
}

// Activations that feed a GEMM are stored in the B-operand fragment order of
// v_mfma_f32_32x32x16_bf16 ("fragment layout"): element (m, k) of an [M][K]
// matrix sits in 1 KiB tile (m/32, k/16), lane m%32 + 32*((k%16)/8), slot k%8,
// tiles ordered row-tile-major.  A wave then fetches one operand with a single
// contiguous 1 KiB load.  Buffers hold a multiple of 32 rows.
__host__ __device__ __forceinline__ size_t frag_index(int m, int k, int K) {
    return ((((size_t)(m >> 5) * (K >> 4) + (k >> 4)) * 64 + (m & 31) + 32 * ((k & 15) >> 3)) << 3) + (k & 7);
}
__host__ __device__ __forceinline__ int round32(int m) { return (m + 31) & ~31; }
// Rows a fragment-layout activation buffer must hold for m rows: every row of
// the tiles the GEMM that reads it covers m with (1, 2, 4 or 8 tiles of 32 rows
// up to 256 rows, whole 128-row tiles above).
__host__ __device__ __forceinline__ int gemm_rows(int m) {
    return m <= 32 ? 32 : m <= 64 ? 64 : m <= 128 ? 128 : ((m + 127) / 128) * 128;
}

// Element offset of (layer, page, K/V, head, token) in a stage pool laid out
// [layers][pages][K, V][heads][16 tokens][hd]: one layer's pages are
// contiguous, so one layer's working set spans few translation fragments.
__host__ __device__ __forceinline__ size_t kv_offset(int layer, int pid, int n_pages, int kv, int head, int H, int tok,
                                                     int hd) {
    return (((((size_t)layer * n_pages + pid) * 2 + kv) * H + head) * 16 + tok) * (size_t)hd;
}

// Rows a call holds: the host count M, or, when the caller passes a device
// count, that count clamped to [0, M] (M is then the launch capacity).
__device__ __forceinline__ int live_rows(const int32_t* dn, int M) {
    if (!dn) return M;
    const int n = *dn;
    return n < 0 ? 0 : (n > M ? M : n);
}

// First sticky error wins.
__device__ __forceinline__ void set_err(int* err, int code) { atomicCAS(err, 0, code); }

// ---------------------------------------------------------------- GEMM epilogues
enum Epi : int { EPI_QKV = 0, EPI_PARTIAL = 1, EPI_SWIGLU = 2, EPI_STORE = 3 };

// Where a stage's K/V lives and which rows write it.
struct KvTarget {
    uint16_t* pool;  // stage pool
    int n_pages;     // pages in that pool
    int layer;       // layer index inside the stage
    int n_layers;    // layers per page of that stage
    const int32_t* page_table;
    int max_seqs, max_pages, n_planes;  // n_planes = r_max + 2
    const int32_t* c_row;               // plane = c_row[m] + 1 when non-null
    int plane_fixed;                    // otherwise this plane
};

struct EpiArgs {
    float* out;     // STORE: destination
    int ld_out;
    uint16_t* act;  // SWIGLU output, fragment layout [M][F]
    int ld_act;     // F
    float* q;       // QKV: q after RoPE [M][d]
    KvTarget kv;
    const int32_t* kvpid;  // QKV: page id of each row's K/V write in this stage's pool, -1 = none
    const int32_t* pos;
    const float2* rope;  // [M][hd/2] (cos, sin) of pos * base^(-2j/hd), one table per stage call
    int H, hd;
    int* err;
};

struct GemmShape {
    int N, K, S, KW;  // packed output columns, reduction length, K splits over workgroups, waves per workgroup
    int NS;           // 32-column stripes per workgroup (1 or 2)
};

// ---------------------------------------------------------------- layouts
struct WeightLayout {
    size_t qkv, o, gu, down;  // byte offsets of layer 0's tensors
    size_t layer_stride;      // bytes per layer
    size_t adapter, lm_head, embed, w_exit, total;
};
bool weight_layout(const cdb_model_desc& d, WeightLayout* out);

struct WsLayout {
    size_t err, h, h_in, q, x, act, part, rope, order, kvpid, deff, prow, lm, total;
};
WsLayout ws_layout(const cdb_model_desc& d, int rows);

GemmShape gemm_shape(int N, int K, int epi, int M);  // M <= kMaxRows
GemmShape gemm_shape_mn(int N, int K, int M, int epi);  // M > kMaxRows
bool desc_supported(const cdb_model_desc& d);

// ---------------------------------------------------------------- launchers
// dn: optional device row count (<= M); rows at or past it are not stored
hipError_t launch_gemm(int epi, const uint16_t* X, const uint16_t* Wp, int M, GemmShape g, float* part,
                       const EpiArgs& ea, hipStream_t st, const int32_t* dn = nullptr);
// order: the call's rows ranked by descending position (by the row-entry
// kernels of a stage call, or by launch_row_order)
hipError_t launch_attention(const float* q, const KvTarget& kv, const int32_t* seq, const int32_t* pos,
                            const int32_t* order, int M, int H, int hd, uint16_t* out, int* err, hipStream_t st,
                            const int32_t* dn = nullptr);
hipError_t launch_row_order(const int32_t* pos, int M, int32_t* order, hipStream_t st, const int32_t* dn = nullptr);
// causal attention of a prefill chunk: rows are positions pos0..pos0+M-1 of one
// sequence in the target's fixed plane
hipError_t launch_prefill_attention(const float* q, const KvTarget& kv, int seq, int pos0, int M, int H, int hd,
                                    uint16_t* out, int* err, hipStream_t st);
// h[i] += sum over s < S of part[s][i] (split order), then, when out is set,
// out = bf16(RMSNorm(h)) in fragment layout.
hipError_t launch_resid_norm(float* h, const float* part, int S, int M, int d, float eps, uint16_t* out,
                             hipStream_t st, const int32_t* dn = nullptr);
// The row-entry kernels of the three stage calls also fill the call's RoPE
// table rope[M][hd/2] = (cos, sin) of pos * base^(-2j/hd), angles in fp64,
// and kvpid[M], the page of the stage's pool that receives each row's K/V
// (the page table looked up once per call; -1 and a device error if unmapped).
// They (gather, embed, state load) also write the attention's row order when
// `order` is non-null (at most kMaxRows rows).  The gather writes either the
// adapter input xcat = [h; e] or, with xn set, the first core layer's input
// xn = bf16(RMSNorm(h)), both in fragment layout.
hipError_t launch_gather(const cdb_model_desc& md, const cdb_state& s, const cdb_rows& r, const cdb_kv& kv,
                         const KvTarget& kt, float* h, float* h_in, uint16_t* xcat, float2* rope, int32_t* kvpid,
                         int32_t* order, uint16_t* xn, int* err, hipStream_t st);
hipError_t launch_embed(const cdb_model_desc& md, const uint16_t* embed, const int32_t* tokens, const cdb_rows& r,
                        const cdb_kv& kv, const KvTarget& kt, int n_slots, float* h, float2* rope, int32_t* kvpid,
                        int32_t* order, int* err, hipStream_t st);
hipError_t launch_store_state(int M, int d, int n_slots, const int32_t* slot, const float* h, float* state_h,
                              float* state_e, hipStream_t st, const int32_t* dn = nullptr);
hipError_t launch_load_state(const cdb_model_desc& md, int M, const int32_t* slot, const int32_t* seq,
                             const int32_t* pos, const KvTarget& kt, const float* state_h, int n_slots, float* h,
                             float2* rope, int32_t* kvpid, int32_t* order, int* err, hipStream_t st,
                             const int32_t* dn = nullptr);
// h += the S split-K partials in part (split order) first; gate: NULL replays
// rows.depth; deff[M] receives each exiting row's depth.
hipError_t launch_exit(const cdb_model_desc& md, const cdb_rows& r, float* h, const float* part, int S,
                       const float* h_in, const uint16_t* w_exit, float* state_h, int n_slots, const cdb_step_out& o,
                       const cdb_gate* gate, int32_t* deff, hipStream_t st);
hipError_t launch_compact(int M, const uint8_t* mask, int32_t* cont, int32_t* exited, int32_t* counts,
                          hipStream_t st);
// copy-on-exit for the rows with deff > 0, and the step's stable compaction
hipError_t launch_copy_on_exit(const cdb_model_desc& md, const cdb_kv& kv, const cdb_rows& r, const int32_t* deff,
                               const uint8_t* mask, int32_t* cont, int32_t* exited, int32_t* counts, int* err,
                               hipStream_t st);
hipError_t launch_argmax(int M, int V, const float* logits, int32_t* ids, hipStream_t st, const int32_t* dn = nullptr);
// prefill: row arrays slot = i, seq, pos = pos0 + i in rows[0..3M); per-row
// write pages of a fixed plane; adapter input [h; e] in fragment layout
hipError_t launch_prefill_rows(int seq, int pos0, int M, int32_t* rows, hipStream_t st);
hipError_t launch_kv_pages(const KvTarget& kt, const cdb_rows& r, int32_t* kvpid, int* err, hipStream_t st);
hipError_t launch_concat_frag(int M, int d, const float* h, const float* e, uint16_t* xcat, hipStream_t st);
hipError_t launch_scatter_ids(int M, const int32_t* ids, const int32_t* seq, const int32_t* index, int max_seqs,
                              int stride, int32_t* out, hipStream_t st);
hipError_t launch_pack(int kind, const uint16_t* a, const uint16_t* b, const uint16_t* c, int N, int K, int hd,
                       uint16_t* dst, hipStream_t st);
hipError_t launch_copy_bf16(const uint16_t* src, size_t n, uint16_t* dst, hipStream_t st);
hipError_t launch_ws_init(int* err, hipStream_t st);

enum PackKind : int { PACK_PLAIN = 0, PACK_QKV = 1, PACK_GU = 2 };

}  // namespace cdb
