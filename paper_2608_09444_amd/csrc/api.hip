// libcdb C ABI: argument validation, packed-weight and workspace layouts, and
// the launch sequences of the three stage calls.
#include <string.h>

#include <algorithm>
#include <mutex>

#include "cdb_internal.h"

namespace cdb {

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

bool desc_supported(const cdb_model_desc& d) {
    if (d.d <= 0 || d.n_heads <= 0 || d.head_dim <= 0 || d.d_ff <= 0 || d.vocab <= 0) return false;
    if (d.n_prelude < 0 || d.n_core < 1 || d.n_coda < 0 || d.r_max < 1 || d.r_max > 64) return false;
    if (d.d % 32 || d.d_ff % 32 || d.vocab % 32 || d.n_heads * d.head_dim != d.d) return false;
    if (d.head_dim != 64 && d.head_dim != 96 && d.head_dim != 128) return false;
    if (d.page_tokens != kPage) return false;
    if (d.injection != 0 && d.injection != 1) return false;
    if (d.exit_kind != 0 && d.exit_kind != 1) return false;
    return true;
}

bool weight_layout(const cdb_model_desc& d, WeightLayout* w) {
    if (!desc_supported(d)) return false;
    const size_t D = d.d, F = d.d_ff, V = d.vocab;
    size_t off = 0;
    w->qkv = off;
    off = align256(off + 3 * D * D * 2);
    w->o = off;
    off = align256(off + D * D * 2);
    w->gu = off;
    off = align256(off + 2 * F * D * 2);
    w->down = off;
    off = align256(off + D * F * 2);
    w->layer_stride = off;
    off = w->layer_stride * (size_t)(d.n_prelude + d.n_core + d.n_coda);
    w->adapter = off;
    if (d.injection) off = align256(off + D * 2 * D * 2);
    w->lm_head = off;
    off = align256(off + V * D * 2);
    w->embed = off;
    off = align256(off + V * D * 2);
    w->w_exit = off;
    off = align256(off + D * 2);
    w->total = off;
    return true;
}

// The four per-layer GEMMs and the adapter / LM head, with their split counts.
// The loop step's adapter writes split-K partials that the first core layer's
// residual + norm sums (adapter_part); the prefill's writes its result (adapter).
struct ModelGemms {
    GemmShape qkv, o, gu, down, adapter, adapter_part, lm;
};
// Launch shapes of the model's projections for calls of M rows: the skinny
// weight-streaming kernel up to kMaxRows rows, the tile kernel above.
static ModelGemms model_gemms(const cdb_model_desc& d, int M = 0) {
    ModelGemms g;
    if (M > kMaxRows) {
        g.qkv = gemm_shape_mn(3 * d.d, d.d, M, EPI_QKV);
        g.o = gemm_shape_mn(d.d, d.d, M, EPI_PARTIAL);
        g.gu = gemm_shape_mn(2 * d.d_ff, d.d, M, EPI_SWIGLU);
        g.down = gemm_shape_mn(d.d, d.d_ff, M, EPI_PARTIAL);
        g.adapter = gemm_shape_mn(d.d, 2 * d.d, M, EPI_STORE);
        g.adapter_part = g.adapter;  // the loop step never has more than kMaxRows rows
        g.lm = gemm_shape_mn(d.vocab, d.d, M, EPI_STORE);
        return g;
    }
    g.qkv = gemm_shape(3 * d.d, d.d, EPI_QKV, M);
    g.o = gemm_shape(d.d, d.d, EPI_PARTIAL, M);
    g.gu = gemm_shape(2 * d.d_ff, d.d, EPI_SWIGLU, M);
    g.down = gemm_shape(d.d, d.d_ff, EPI_PARTIAL, M);
    g.adapter = gemm_shape(d.d, 2 * d.d, EPI_STORE, M);
    g.adapter_part = gemm_shape(d.d, 2 * d.d, EPI_PARTIAL, M);
    g.lm = gemm_shape(d.vocab, d.d, EPI_STORE, M);
    return g;
}

WsLayout ws_layout(const cdb_model_desc& d, int rows) {
    WsLayout L;
    const size_t D = d.d, F = d.d_ff, M = rows, M32 = gemm_rows(rows);
    const ModelGemms g = model_gemms(d, rows);
    // split-K partials of O, down and the loop step's adapter
    const size_t part = (size_t)std::max({g.o.S, g.down.S, d.injection ? g.adapter_part.S : 0}) * D;
    size_t off = 0;
    L.err = off;
    off = 256;
    L.h = off;
    off = align256(off + M * D * 4);
    L.h_in = off;
    off = align256(off + M * D * 4);
    L.q = off;
    off = align256(off + M * D * 4);
    L.x = off;
    off = align256(off + M32 * 2 * D * 2);
    L.act = off;
    off = align256(off + M32 * F * 2);
    L.part = off;
    off = align256(off + part * M * 4);
    L.rope = off;
    off = align256(off + M * (size_t)(d.head_dim / 2) * 8);
    L.order = off;
    off = align256(off + M * 4);
    L.kvpid = off;
    off = align256(off + M * 4);
    L.deff = off;
    off = align256(off + M * 4);
    L.prow = off;  // prefill row arrays: slot, seq, pos
    off = align256(off + 3 * M * 4);
    L.lm = off;  // prefill without logits: the LM head of the last 32-row tile
    off = align256(off + (size_t)32 * d.vocab * 4);
    L.total = off;
    return L;
}

// Everything a stage call needs, resolved once per call.
struct Ctx {
    const cdb_model_desc* md;
    const unsigned char* wb;
    WeightLayout wl;
    ModelGemms gm;
    unsigned char* ws;
    WsLayout L;
    int* err;
    float* h;
    float* h_in;
    float* q;
    uint16_t* x;
    uint16_t* act;
    float* part;
    float2* rope;
    int32_t* order;
    int32_t* kvpid;
    int32_t* deff;
    int32_t* prow;
    float* lm;
};

static Ctx make_ctx(const cdb_model* model, void* ws, int rows) {
    Ctx c;
    c.md = &model->desc;
    c.wb = static_cast<const unsigned char*>(model->packed);
    weight_layout(model->desc, &c.wl);
    c.gm = model_gemms(model->desc, rows);
    c.ws = static_cast<unsigned char*>(ws);
    c.L = ws_layout(model->desc, rows);
    c.err = reinterpret_cast<int*>(c.ws + c.L.err);
    c.h = reinterpret_cast<float*>(c.ws + c.L.h);
    c.h_in = reinterpret_cast<float*>(c.ws + c.L.h_in);
    c.q = reinterpret_cast<float*>(c.ws + c.L.q);
    c.x = reinterpret_cast<uint16_t*>(c.ws + c.L.x);
    c.act = reinterpret_cast<uint16_t*>(c.ws + c.L.act);
    c.part = reinterpret_cast<float*>(c.ws + c.L.part);
    c.rope = reinterpret_cast<float2*>(c.ws + c.L.rope);
    c.order = reinterpret_cast<int32_t*>(c.ws + c.L.order);
    c.kvpid = reinterpret_cast<int32_t*>(c.ws + c.L.kvpid);
    c.deff = reinterpret_cast<int32_t*>(c.ws + c.L.deff);
    c.prow = reinterpret_cast<int32_t*>(c.ws + c.L.prow);
    c.lm = reinterpret_cast<float*>(c.ws + c.L.lm);
    return c;
}

static const uint16_t* wptr(const Ctx& c, size_t off) { return reinterpret_cast<const uint16_t*>(c.wb + off); }

#define HIPCHK(x)                                  \
    do {                                           \
        if ((x) != hipSuccess) return CDB_ERR_HIP; \
    } while (0)

// A prefill chunk: the rows are positions pos0.. of sequence seq.
struct Chunk {
    int seq, pos0;
};

// Run `count` transformer layers (global index first..) of one stage over the
// rows in ctx.h, with K/V in `kv`.  On return ctx.h holds the stage output and
// ctx.x its RMSNorm when `norm_out` is set.  With `chunk` the rows are a
// prefill chunk and attention runs query-tiled on MFMA.
// x_ready: c.x already holds the first layer's input (the loop step's gather
// wrote it), so its residual + norm is skipped.  pending_out: the last down
// projection's partials are left for the caller (the loop step's exit kernel
// adds them) instead of a closing residual kernel; not with norm_out.
static cdb_status run_layers(const Ctx& c, int first, int count, KvTarget kv, const cdb_rows& r, bool norm_out,
                             hipStream_t st, const Chunk* chunk = nullptr, int pending_in = 0, bool x_ready = false,
                             int* pending_out = nullptr) {
    const cdb_model_desc& d = *c.md;
    const int M = r.n_rows;
    const int32_t* dn = r.d_n_rows;  // device row count (M is then the capacity)
    if ((x_ready && pending_in) || (pending_out && norm_out)) return CDB_ERR_INVALID_ARG;
    // split-K partials not yet added to h: the previous down projection's, or at
    // the start those of the loop step's adapter (h then holds zeros)
    int pending = pending_in;
    // the attention's row order (c.order) was written by the call's row-entry
    // kernel (gather, embed or state load); prefill chunks need none
    for (int l = 0; l < count; ++l) {
        const size_t lb = (size_t)(first + l) * c.wl.layer_stride;
        kv.layer = l;
        EpiArgs ea{};
        ea.kvpid = c.kvpid;
        ea.pos = r.pos;
        ea.H = d.n_heads;
        ea.hd = d.head_dim;
        ea.rope = c.rope;
        ea.err = c.err;
        ea.kv = kv;
        ea.q = c.q;
        ea.act = c.act;
        ea.ld_act = d.d_ff;
        // attention half: h += down partials; x = RMSNorm(h); q/k/v + RoPE + K/V write
        if (l > 0 || !x_ready) HIPCHK(launch_resid_norm(c.h, c.part, pending, M, d.d, d.rms_eps, c.x, st, dn));
        HIPCHK(launch_gemm(EPI_QKV, c.x, wptr(c, lb + c.wl.qkv), M, c.gm.qkv, c.part, ea, st, dn));
        if (chunk)
            HIPCHK(launch_prefill_attention(c.q, kv, chunk->seq, chunk->pos0, M, d.n_heads, d.head_dim, c.x, c.err,
                                            st));
        else
            HIPCHK(launch_attention(c.q, kv, r.seq, r.pos, c.order, M, d.n_heads, d.head_dim, c.x, c.err, st, dn));
        HIPCHK(launch_gemm(EPI_PARTIAL, c.x, wptr(c, lb + c.wl.o), M, c.gm.o, c.part, ea, st, dn));
        // MLP half: h += O partials; x = RMSNorm(h); act = SwiGLU; down partials
        HIPCHK(launch_resid_norm(c.h, c.part, c.gm.o.S, M, d.d, d.rms_eps, c.x, st, dn));
        HIPCHK(launch_gemm(EPI_SWIGLU, c.x, wptr(c, lb + c.wl.gu), M, c.gm.gu, c.part, ea, st, dn));
        HIPCHK(launch_gemm(EPI_PARTIAL, c.act, wptr(c, lb + c.wl.down), M, c.gm.down, c.part, ea, st, dn));
        pending = c.gm.down.S;
    }
    if (pending_out)
        *pending_out = pending;
    else if (pending || norm_out)
        HIPCHK(launch_resid_norm(c.h, c.part, pending, M, d.d, d.rms_eps, norm_out ? c.x : nullptr, st, dn));
    return CDB_OK;
}

static KvTarget stage_target(const cdb_model_desc& d, const cdb_kv& kv, int stage) {
    KvTarget t{};
    t.page_table = kv.page_table;
    t.max_seqs = kv.max_seqs;
    t.max_pages = kv.max_pages;
    t.n_planes = d.r_max + 2;
    if (stage == 0) {
        t.pool = static_cast<uint16_t*>(kv.pre_pool);
        t.n_pages = kv.pre_pages;
        t.n_layers = d.n_prelude;
        t.plane_fixed = 0;
    } else if (stage == 1) {
        t.pool = static_cast<uint16_t*>(kv.core_pool);
        t.n_pages = kv.core_pages;
        t.n_layers = d.n_core;
        t.plane_fixed = -1;
    } else {
        t.pool = static_cast<uint16_t*>(kv.coda_pool);
        t.n_pages = kv.coda_pages;
        t.n_layers = d.n_coda;
        t.plane_fixed = d.r_max + 1;
    }
    return t;
}

static cdb_status check_common(const cdb_model* model, const cdb_kv* kv, const cdb_state* state, const cdb_rows* rows,
                               void* ws, size_t ws_bytes, int stage) {
    if (!model || !kv || !state || !rows || !ws || !model->packed || !state->h) return CDB_ERR_INVALID_ARG;
    const cdb_model_desc& d = model->desc;
    if (!desc_supported(d)) return CDB_ERR_UNSUPPORTED;
    if (rows->n_rows < 0 || state->n_slots < 0 || kv->max_seqs < 0 || kv->max_pages < 0) return CDB_ERR_INVALID_ARG;
    if (rows->n_rows > kMaxRows) return CDB_ERR_CAPACITY;
    if (rows->n_rows > 0 && (!rows->slot || !rows->seq || !rows->pos)) return CDB_ERR_INVALID_ARG;
    if (ws_bytes < ws_layout(d, rows->n_rows).total) return CDB_ERR_CAPACITY;
    const int layers = stage == 0 ? d.n_prelude : (stage == 1 ? d.n_core : d.n_coda);
    if (layers > 0) {
        void* pool = stage == 0 ? kv->pre_pool : (stage == 1 ? kv->core_pool : kv->coda_pool);
        const int np = stage == 0 ? kv->pre_pages : (stage == 1 ? kv->core_pages : kv->coda_pages);
        if (!pool || np < 0 || !kv->page_table) return CDB_ERR_INVALID_ARG;
    }
    return CDB_OK;
}

}  // namespace cdb

using namespace cdb;

extern "C" {

size_t cdb_packed_weight_bytes(const cdb_model_desc* desc) {
    WeightLayout w;
    if (!desc || !weight_layout(*desc, &w)) return 0;
    return w.total;
}

cdb_status cdb_pack_weights(const cdb_model_desc* desc, const cdb_plain_weights* w, void* packed, size_t bytes,
                            hipStream_t st) {
    if (!desc || !w || !packed) return CDB_ERR_INVALID_ARG;
    WeightLayout L;
    if (!weight_layout(*desc, &L)) return CDB_ERR_UNSUPPORTED;
    if (bytes < L.total) return CDB_ERR_CAPACITY;
    const cdb_model_desc& d = *desc;
    const int nl = d.n_prelude + d.n_core + d.n_coda;
    if (!w->embed || !w->lm_head || !w->w_exit || (nl > 0 && !w->layer) || (d.injection && !w->adapter))
        return CDB_ERR_INVALID_ARG;
    for (int i = 0; i < 7 * nl; ++i)
        if (!w->layer[i]) return CDB_ERR_INVALID_ARG;
    unsigned char* b = static_cast<unsigned char*>(packed);
    auto P = [&](size_t off) { return reinterpret_cast<uint16_t*>(b + off); };
    auto S = [&](const void* p) { return static_cast<const uint16_t*>(p); };
    for (int l = 0; l < nl; ++l) {
        const void* const* t = w->layer + 7 * l;
        const size_t lb = (size_t)l * L.layer_stride;
        HIPCHK(launch_pack(PACK_QKV, S(t[0]), S(t[1]), S(t[2]), 3 * d.d, d.d, d.head_dim, P(lb + L.qkv), st));
        HIPCHK(launch_pack(PACK_PLAIN, S(t[3]), nullptr, nullptr, d.d, d.d, 0, P(lb + L.o), st));
        HIPCHK(launch_pack(PACK_GU, S(t[4]), S(t[5]), nullptr, 2 * d.d_ff, d.d, 0, P(lb + L.gu), st));
        HIPCHK(launch_pack(PACK_PLAIN, S(t[6]), nullptr, nullptr, d.d, d.d_ff, 0, P(lb + L.down), st));
    }
    if (d.injection) HIPCHK(launch_pack(PACK_PLAIN, S(w->adapter), nullptr, nullptr, d.d, 2 * d.d, 0, P(L.adapter), st));
    HIPCHK(launch_pack(PACK_PLAIN, S(w->lm_head), nullptr, nullptr, d.vocab, d.d, 0, P(L.lm_head), st));
    HIPCHK(launch_copy_bf16(S(w->embed), (size_t)d.vocab * d.d, P(L.embed), st));
    HIPCHK(launch_copy_bf16(S(w->w_exit), (size_t)d.d, P(L.w_exit), st));
    return CDB_OK;
}

size_t cdb_kv_page_bytes(const cdb_model_desc* desc, int32_t stage) {
    if (!desc || !desc_supported(*desc) || stage < 0 || stage > 2) return 0;
    const int layers = stage == 0 ? desc->n_prelude : (stage == 1 ? desc->n_core : desc->n_coda);
    return (size_t)layers * 2 * desc->n_heads * kPage * desc->head_dim * 2;
}

size_t cdb_workspace_bytes(const cdb_model_desc* desc, int32_t max_rows) {
    if (!desc || !desc_supported(*desc) || max_rows < 0 || max_rows > kMaxPrefillRows) return 0;
    // the layout is not monotonic in the row count (the split-K factor of the
    // tile GEMM shrinks as its grid grows): the largest one up to max_rows
    size_t n = ws_layout(*desc, 0).total;
    for (int r = 1; r <= max_rows; ++r) n = std::max(n, ws_layout(*desc, r).total);
    return n;
}

cdb_status cdb_workspace_init(void* ws, size_t ws_bytes, hipStream_t st) {
    if (!ws) return CDB_ERR_INVALID_ARG;
    if (ws_bytes < 256) return CDB_ERR_CAPACITY;
    HIPCHK(launch_ws_init(static_cast<int*>(ws), st));
    return CDB_OK;
}

cdb_status cdb_boundary_prelude(const cdb_model* model, const cdb_kv* kv, const cdb_state* state, const cdb_rows* rows,
                                const int32_t* tokens, void* ws, size_t ws_bytes, hipStream_t st) {
    cdb_status s = check_common(model, kv, state, rows, ws, ws_bytes, 0);
    if (s != CDB_OK) return s;
    const cdb_model_desc& d = model->desc;
    if (rows->n_rows > 0 && !tokens) return CDB_ERR_INVALID_ARG;
    if (d.injection && !state->e) return CDB_ERR_INVALID_ARG;
    if (rows->n_rows == 0) return CDB_OK;
    Ctx c = make_ctx(model, ws, rows->n_rows);
    const KvTarget t = stage_target(d, *kv, 0);
    HIPCHK(launch_embed(d, wptr(c, c.wl.embed), tokens, *rows, *kv, t, state->n_slots, c.h, c.rope, c.kvpid, c.order,
                        c.err,
                        st));
    s = run_layers(c, 0, d.n_prelude, t, *rows, false, st);
    if (s != CDB_OK) return s;
    HIPCHK(launch_store_state(rows->n_rows, d.d, state->n_slots, rows->slot, c.h, state->h,
                              d.injection ? state->e : nullptr, st, rows->d_n_rows));
    return CDB_OK;
}

// err: where device errors go (NULL: the workspace's own error word)
static cdb_status loop_step(const cdb_model* model, const cdb_kv* kv, const cdb_state* state, const cdb_rows* rows,
                            const cdb_gate* gate, const cdb_step_out* out, void* ws, size_t ws_bytes, hipStream_t st,
                            int* err = nullptr) {
    cdb_status s = check_common(model, kv, state, rows, ws, ws_bytes, 1);
    if (s != CDB_OK) return s;
    const cdb_model_desc& d = model->desc;
    if (!out || !out->exit_score || !out->exit_mask || !out->cont || !out->exited || !out->counts)
        return CDB_ERR_INVALID_ARG;
    if (rows->n_rows > 0 && (!rows->c || (!gate && !rows->depth))) return CDB_ERR_INVALID_ARG;
    if (gate && gate->lookahead && !gate->pending) return CDB_ERR_INVALID_ARG;
    if (d.injection && !state->e) return CDB_ERR_INVALID_ARG;
    const int M = rows->n_rows;
    Ctx c = make_ctx(model, ws, M);
    if (err) c.err = err;
    cdb_rows r = *rows;
    if (gate) r.depth = nullptr;
    if (M > 0) {
        KvTarget t = stage_target(d, *kv, 1);
        t.c_row = r.c;
        // the gather also writes the first core layer's input (the adapter's
        // input for injection models)
        HIPCHK(launch_gather(d, *state, r, *kv, t, c.h, c.h_in, d.injection ? c.x : nullptr, c.rope, c.kvpid, c.order,
                             d.injection ? nullptr : c.x, c.err, st));
        // injection models: the gather zeroed h; the adapter's split-K
        // partials become the first layer's input in its residual + norm
        if (d.injection) {
            EpiArgs ea{};
            ea.err = c.err;
            HIPCHK(launch_gemm(EPI_PARTIAL, c.x, wptr(c, c.wl.adapter), M, c.gm.adapter_part, c.part, ea, st,
                               r.d_n_rows));
        }
        int pending = 0;
        s = run_layers(c, d.n_prelude, d.n_core, t, r, false, st, nullptr, d.injection ? c.gm.adapter_part.S : 0,
                       !d.injection, &pending);
        if (s != CDB_OK) return s;
        // the exit kernel adds the last down projection's partials to h first
        HIPCHK(launch_exit(d, r, c.h, c.part, pending, c.h_in, wptr(c, c.wl.w_exit), state->h, state->n_slots, *out,
                           gate, c.deff, st));
    }
    // copy-on-exit, with the stable compaction in its first workgroup
    HIPCHK(launch_copy_on_exit(d, *kv, r, c.deff, out->exit_mask, out->cont, out->exited, out->counts, c.err, st));
    return CDB_OK;
}

cdb_status cdb_loop_step(const cdb_model* model, const cdb_kv* kv, const cdb_state* state, const cdb_rows* rows,
                         const cdb_step_out* out, void* ws, size_t ws_bytes, hipStream_t st) {
    return loop_step(model, kv, state, rows, nullptr, out, ws, ws_bytes, st);
}

cdb_status cdb_loop_step_gated(const cdb_model* model, const cdb_kv* kv, const cdb_state* state,
                               const cdb_rows* rows, const cdb_gate* gate, const cdb_step_out* out, void* ws,
                               size_t ws_bytes, hipStream_t st) {
    if (!gate) return CDB_ERR_INVALID_ARG;
    return loop_step(model, kv, state, rows, gate, out, ws, ws_bytes, st);
}

}  // extern "C"

// Scratch of cdb_loop_step_noalloc: one copy per device, alive until the
// process ends.  Host code never uses this name as an address (on the host it
// is a stand-in symbol); it uses the device address hipGetSymbolAddress gives,
// looked up once per device.
constexpr size_t kNoAllocScratchBytes = (size_t)48 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's scratch address (NULL if the lookup fails).
void* device_scratch() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        g_scratch_ptr[dev] = p;
    }
    return g_scratch_ptr[dev];
}
}  // namespace

extern "C" {

cdb_status cdb_loop_step_noalloc(const cdb_model* model, const cdb_kv* kv, const cdb_state* state,
                                 const cdb_rows* rows, const cdb_step_out* out, int32_t* d_error, hipStream_t st) {
    if (!d_error || !model || !rows) return CDB_ERR_INVALID_ARG;
    if (!desc_supported(model->desc)) return CDB_ERR_UNSUPPORTED;
    if (rows->n_rows < 0) return CDB_ERR_INVALID_ARG;
    if (rows->n_rows > kMaxRows || ws_layout(model->desc, rows->n_rows).total > kNoAllocScratchBytes)
        return CDB_ERR_CAPACITY;
    void* ws = device_scratch();
    if (!ws) return CDB_ERR_HIP;
    return loop_step(model, kv, state, rows, nullptr, out, ws, kNoAllocScratchBytes, st, d_error);
}

cdb_status cdb_boundary_coda(const cdb_model* model, const cdb_kv* kv, const cdb_state* state, const cdb_rows* rows,
                             float* logits, int32_t* next_ids, void* ws, size_t ws_bytes, hipStream_t st) {
    cdb_status s = check_common(model, kv, state, rows, ws, ws_bytes, 2);
    if (s != CDB_OK) return s;
    const cdb_model_desc& d = model->desc;
    if (!logits || !next_ids) return CDB_ERR_INVALID_ARG;
    const int M = rows->n_rows;
    if (M == 0) return CDB_OK;
    Ctx c = make_ctx(model, ws, M);
    const KvTarget t = stage_target(d, *kv, 2);
    HIPCHK(launch_load_state(d, M, rows->slot, rows->seq, rows->pos, t, state->h, state->n_slots, c.h, c.rope, c.kvpid,
                             c.order, c.err, st, rows->d_n_rows));
    s = run_layers(c, d.n_prelude + d.n_core, d.n_coda, t, *rows, true, st);
    if (s != CDB_OK) return s;
    EpiArgs ea{};
    ea.ld_out = d.vocab;
    ea.err = c.err;
    ea.out = logits;
    HIPCHK(launch_gemm(EPI_STORE, c.x, wptr(c, c.wl.lm_head), M, c.gm.lm, c.part, ea, st, rows->d_n_rows));
    HIPCHK(launch_argmax(M, d.vocab, logits, next_ids, st, rows->d_n_rows));
    return CDB_OK;
}

cdb_status cdb_prefill(const cdb_model* model, const cdb_kv* kv, int32_t seq, int32_t pos0, int32_t n_rows,
                       const int32_t* tokens, float* logits, int32_t* next_ids, void* ws, size_t ws_bytes,
                       hipStream_t st) {
    if (!model || !kv || !model->packed || !tokens || !next_ids || !ws) return CDB_ERR_INVALID_ARG;
    const cdb_model_desc& d = model->desc;
    if (!desc_supported(d)) return CDB_ERR_UNSUPPORTED;
    if (n_rows < 1 || n_rows > kMaxPrefillRows) return CDB_ERR_CAPACITY;
    if (seq < 0 || seq >= kv->max_seqs || pos0 < 0 || (size_t)pos0 + n_rows > (size_t)kv->max_pages * kPage)
        return CDB_ERR_INVALID_ARG;
    if (pos0 + n_rows > kMaxPrefillPos) return CDB_ERR_CAPACITY;  // checked before any launch
    if (!kv->page_table) return CDB_ERR_INVALID_ARG;
    for (int stage = 0; stage < 3; ++stage) {
        const int layers = stage == 0 ? d.n_prelude : (stage == 1 ? d.n_core : d.n_coda);
        void* pool = stage == 0 ? kv->pre_pool : (stage == 1 ? kv->core_pool : kv->coda_pool);
        if (layers > 0 && !pool) return CDB_ERR_INVALID_ARG;
    }
    if (ws_bytes < ws_layout(d, n_rows).total) return CDB_ERR_CAPACITY;
    const int M = n_rows;
    Ctx c = make_ctx(model, ws, M);
    const Chunk chunk{seq, pos0};
    cdb_rows r{M, c.prow, c.prow + M, c.prow + 2 * M, nullptr, nullptr, nullptr};
    HIPCHK(launch_prefill_rows(seq, pos0, M, c.prow, st));
    // prelude (plane 0): embedding, RoPE table, write pages
    KvTarget t = stage_target(d, *kv, 0);
    HIPCHK(launch_embed(d, wptr(c, c.wl.embed), tokens, r, *kv, t, M, c.h, c.rope, c.kvpid, nullptr, c.err, st));
    cdb_status s = run_layers(c, 0, d.n_prelude, t, r, false, st, &chunk);
    if (s != CDB_OK) return s;
    if (d.injection) HIPCHK(hipMemcpyAsync(c.h_in, c.h, (size_t)M * d.d * 4, hipMemcpyDeviceToDevice, st));  // e
    // r_max core loops over the whole chunk, loop r in plane r (prompt tokens run every loop)
    for (int loop = 1; loop <= d.r_max; ++loop) {
        t = stage_target(d, *kv, 1);
        t.plane_fixed = loop;
        HIPCHK(launch_kv_pages(t, r, c.kvpid, c.err, st));
        if (d.injection) {
            HIPCHK(launch_concat_frag(M, d.d, c.h, c.h_in, c.x, st));
            EpiArgs ea{};
            ea.out = c.h;
            ea.ld_out = d.d;
            ea.err = c.err;
            HIPCHK(launch_gemm(EPI_STORE, c.x, wptr(c, c.wl.adapter), M, c.gm.adapter, c.part, ea, st));
        }
        s = run_layers(c, d.n_prelude, d.n_core, t, r, false, st, &chunk);
        if (s != CDB_OK) return s;
    }
    // coda (plane r_max + 1), final RMSNorm, LM head, argmax
    t = stage_target(d, *kv, 2);
    HIPCHK(launch_kv_pages(t, r, c.kvpid, c.err, st));
    s = run_layers(c, d.n_prelude + d.n_core, d.n_coda, t, r, true, st, &chunk);
    if (s != CDB_OK) return s;
    EpiArgs ea{};
    ea.ld_out = d.vocab;
    ea.err = c.err;
    if (logits) {
        ea.out = logits;
        HIPCHK(launch_gemm(EPI_STORE, c.x, wptr(c, c.wl.lm_head), M, c.gm.lm, c.part, ea, st));
        HIPCHK(launch_argmax(M, d.vocab, logits, next_ids, st));
        return CDB_OK;
    }
    // only the last row's greedy id: the LM head over the 32-row tile holding it
    const int T = (M - 1) / 32, MT = M - 32 * T;
    const uint16_t* xt = c.x + (size_t)T * (d.d / 16) * 512;  // fragment m-tiles are contiguous
    ea.out = c.lm;
    HIPCHK(launch_gemm(EPI_STORE, xt, wptr(c, c.wl.lm_head), MT, gemm_shape(d.vocab, d.d, EPI_STORE, MT), c.part, ea, st));
    HIPCHK(launch_argmax(1, d.vocab, c.lm + (size_t)(MT - 1) * d.vocab, next_ids, st));
    return CDB_OK;
}

cdb_status cdb_paged_attention(const cdb_model_desc* desc, const cdb_kv* kv, const cdb_rows* rows, int32_t stage,
                               int32_t layer, const float* q, const int32_t* order, void* out, void* ws,
                               size_t ws_bytes, hipStream_t st) {
    if (!desc || !kv || !rows || !q || !out || !ws) return CDB_ERR_INVALID_ARG;
    const cdb_model_desc& d = *desc;
    if (!desc_supported(d)) return CDB_ERR_UNSUPPORTED;
    if (stage < 0 || stage > 2 || rows->n_rows < 0) return CDB_ERR_INVALID_ARG;
    const int layers = stage == 0 ? d.n_prelude : (stage == 1 ? d.n_core : d.n_coda);
    if (layer < 0 || layer >= layers) return CDB_ERR_INVALID_ARG;
    if (rows->n_rows > kMaxRows) return CDB_ERR_CAPACITY;
    if (ws_bytes < 256 + (size_t)kMaxRows * 4) return CDB_ERR_CAPACITY;
    if (rows->n_rows == 0) return CDB_OK;
    if (!rows->seq || !rows->pos || (stage == 1 && !rows->c) || !kv->page_table) return CDB_ERR_INVALID_ARG;
    KvTarget t = stage_target(d, *kv, stage);
    if (!t.pool) return CDB_ERR_INVALID_ARG;
    t.layer = layer;
    if (stage == 1) t.c_row = rows->c;
    if (!order) {
        int32_t* own = reinterpret_cast<int32_t*>(static_cast<unsigned char*>(ws) + 256);
        HIPCHK(launch_row_order(rows->pos, rows->n_rows, own, st, rows->d_n_rows));
        order = own;
    }
    HIPCHK(launch_attention(q, t, rows->seq, rows->pos, order, rows->n_rows, d.n_heads, d.head_dim,
                            static_cast<uint16_t*>(out), static_cast<int*>(ws), st, rows->d_n_rows));
    return CDB_OK;
}

cdb_status cdb_read_device_error(void* ws, hipStream_t st, int32_t* code) {
    if (!ws || !code) return CDB_ERR_INVALID_ARG;
    int32_t v = 0;
    if (hipMemcpyAsync(&v, ws, 4, hipMemcpyDeviceToHost, st) != hipSuccess) return CDB_ERR_HIP;
    if (hipStreamSynchronize(st) != hipSuccess) return CDB_ERR_HIP;
    *code = v;
    if (v != 0) {
        int* err = static_cast<int*>(ws);
        if (launch_ws_init(err, st) != hipSuccess) return CDB_ERR_HIP;
        if (hipStreamSynchronize(st) != hipSuccess) return CDB_ERR_HIP;
    }
    return CDB_OK;
}

const char* cdb_status_str(cdb_status s) {
    switch (s) {
        case CDB_OK: return "ok";
        case CDB_ERR_INVALID_ARG: return "invalid argument";
        case CDB_ERR_CAPACITY: return "capacity exceeded";
        case CDB_ERR_HIP: return "HIP error";
        case CDB_ERR_UNSUPPORTED: return "unsupported shape";
    }
    return "unknown status";
}

}  // extern "C"
