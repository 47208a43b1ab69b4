/*
 * libcdb -- continuous depth batching (CDB) for looped language models on
 * AMD Instinct MI355X (gfx950).
 *
 * A looped LM (paper Section 2, Eq. 1) runs a prelude P once per token, a
 * shared recurrent core R up to r_max times, and a coda C once:
 *     h^(0) = P(x_t),  h^(r+1) = R(h^(r), K^(r)_{<t}),  p(x_{t+1}) = softmax(C(h^(r_t))).
 * CDB (Section 4) schedules the core one loop iteration at a time over a
 * *mixed-depth* batch: rows of many sequences, each at its own loop index, so
 * that a token leaving the core frees its batch slot for another token
 * (refill, Section 4.1).  The three stage operators exported here are the
 * calls such a scheduler issues:
 *
 *   cdb_boundary_prelude  embedding + prelude layers        (Section 4.1, stage P)
 *   cdb_loop_step         one core iteration over the batch, exit score,
 *                         exit decision, stable compaction, copy-on-exit
 *                                                           (Sections 2, 4.1, 4.2)
 *   cdb_boundary_coda     coda layers + final norm + LM head + greedy argmax
 *                                                           (Section 4.1, stage C)
 *
 * Conventions (all calls):
 *   - Every buffer is owned by the caller.  Pointers named d_* or documented as
 *     "device" are device memory on the current HIP device; descriptor structs
 *     and the arrays they point to directly (unless stated) live in host memory.
 *   - The library never allocates, frees or synchronises inside the stage
 *     calls; all work is enqueued on the given stream, so the calls can be
 *     captured into a HIP graph.
 *   - Host-checkable problems (null pointers, sizes over capacity, unsupported
 *     shapes) return an error before anything is enqueued.  Problems only the
 *     device can see (an unmapped page, a depth outside [1, r_max], a row that
 *     has already exited) set a sticky code in the workspace, read with
 *     cdb_read_device_error(); the offending row's writes are skipped.
 *   - Calls on one workspace must not overlap (same stream, or ordered).
 *
 * Numerics: weights, KV cache and the activations that feed matrix products
 * are bf16; matrix products, attention and softmax accumulate in fp32; the
 * residual stream / state pool and logits are fp32.
 */
#ifndef LIBCDB_H
#define LIBCDB_H

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CDB_OK = 0,
    CDB_ERR_INVALID_ARG = 1, /* null pointer, negative size, inconsistent descriptor */
    CDB_ERR_CAPACITY = 2,    /* n_rows or buffer size beyond what the workspace/pool holds */
    CDB_ERR_HIP = 3,         /* a HIP launch or runtime call failed */
    CDB_ERR_UNSUPPORTED = 4  /* a shape the kernels do not handle (see cdb_model_desc) */
} cdb_status;

/* Device-side sticky error codes (cdb_read_device_error). */
enum {
    CDB_DEV_OK = 0,
    CDB_DEV_UNMAPPED_PAGE = 1, /* a page-table entry needed by a row is -1 or out of the pool */
    CDB_DEV_BAD_DEPTH = 2,     /* depth outside [1, r_max], or c outside [0, depth) */
    CDB_DEV_BAD_INDEX = 3      /* slot, seq, position or token id out of range */
};

/* Model shape.  Layer split prelude-core-coda (Section 2): n_prelude, n_core,
 * n_coda transformer layers; the core is iterated up to r_max times.
 * Supported: d % 32 == 0, n_heads * head_dim == d, head_dim in {64, 96, 128},
 * d_ff % 32 == 0, vocab % 32 == 0, page_tokens == 16, 1 <= r_max <= 64. */
typedef struct {
    int32_t d, n_heads, head_dim, d_ff, vocab;
    int32_t n_prelude, n_core, n_coda, r_max;
    int32_t injection;   /* 0: core input is the state h; 1: core input is W_a [h; e] (2d -> d),
                            e = prelude output of the token (Huginn-style adapter) */
    int32_t exit_kind;   /* 0: score = sigmoid(w_exit . RMSNorm(h_new)) (learned-gate form);
                            1: score = ||h_new - h_old||_2 (convergence criterion, App. C.2) */
    int32_t page_tokens; /* tokens per KV page; must be 16 */
    float rms_eps, rope_base;
} cdb_model_desc;

/* Plain weights as the user holds them: device pointers to bf16 row-major
 * [out][in] matrices (y = W x).  layer is a HOST array of 7 * n_layers device
 * pointers, per layer {W_q, W_k, W_v, W_o, W_gate, W_up, W_down} with shapes
 * [d][d] x4, [d_ff][d] x2, [d][d_ff]; layers ordered prelude, core, coda.
 * embed and lm_head are [vocab][d]; w_exit [d]; adapter [d][2d] (injection only). */
typedef struct {
    const void* embed;
    const void* lm_head;
    const void* w_exit;
    const void* adapter;
    const void* const* layer;
} cdb_plain_weights;

/* Bytes of the packed weight blob for a model (0 if the shape is unsupported). */
size_t cdb_packed_weight_bytes(const cdb_model_desc* desc);

/* Rearranges plain weights into the packed blob the kernels stream (MFMA
 * operand tiles, fused q/k/v and gate/up orders).  Enqueued on `stream`;
 * `packed` (device, `bytes` >= cdb_packed_weight_bytes) is owned by the caller
 * and must stay alive while any stage call uses it. */
cdb_status cdb_pack_weights(const cdb_model_desc* desc, const cdb_plain_weights* w, void* packed, size_t bytes,
                            hipStream_t stream);

typedef struct {
    const void* packed; /* device: blob written by cdb_pack_weights */
    cdb_model_desc desc;
} cdb_model;

/* Paged, depth-indexed KV cache (Section 4.2).  Three pools of 16-token
 * pages, one per stage.  A page id addresses the same slot in every layer of
 * its stage; a pool of a stage with L layers and P pages is layer-major:
 *     bf16 [L][P][2 (K, V)][n_heads][16 tokens][head_dim]
 * (K after RoPE).  page_table (device, int32) is
 *     [max_seqs][r_max + 2][max_pages]
 * plane 0 -> prelude pool, planes 1..r_max -> core pool (loop index c, 0-based,
 * uses plane c + 1), plane r_max + 1 -> coda pool; entry = page id within that
 * pool, -1 = unmapped.  Mapping several planes to one page id (shared layouts)
 * is allowed; copy-on-exit then skips identical source and destination. */
typedef struct {
    void* pre_pool;
    void* core_pool;
    void* coda_pool;
    int32_t pre_pages, core_pages, coda_pages;
    const int32_t* page_table;
    int32_t max_seqs, max_pages;
} cdb_kv;

/* Bytes of one page of a stage's pool (stage 0 prelude, 1 core, 2 coda): the
 * stage's layers x 2 x n_heads x 16 x head_dim bf16; 0 if the stage has no
 * layers or the shape is unsupported. */
size_t cdb_kv_page_bytes(const cdb_model_desc* desc, int32_t stage);

/* Per-token latent state (device, fp32): h [n_slots][d]; e [n_slots][d] holds
 * the prelude output for injection models (may be NULL otherwise). */
typedef struct {
    float* h;
    float* e;
    int32_t n_slots;
} cdb_state;

/* One batch of rows (device int32 arrays of n_rows entries).  A row is one
 * token of sequence seq at position pos whose state lives in slot.  For the
 * loop step, c = loops already completed (0-based) and depth = the token's exit
 * depth in [1, r_max]: the row exits after this step iff c + 1 == depth
 * (replayed exit decisions, App. B.2).  Rows may sit at any loop index
 * (refill); rows of one sequence at consecutive positions in one call (a
 * prompt) see each other causally.  c and depth are ignored by the boundary
 * calls.
 * d_n_rows (optional, device int32, may be NULL): the number of rows the call
 * holds, read by the kernels when they run, so that one captured call (Section
 * 4.3, static shapes) replays for any row count up to n_rows.  With it set,
 * n_rows is the capacity: launch shapes, workspace and output buffers are sized
 * for n_rows; only the first clamp(*d_n_rows, 0, n_rows) rows are read,
 * computed into outputs and counted (cont / exited / counts cover those rows);
 * the rest of each output is left as it was.  A row's results are the same as
 * in a call of exactly that many rows.  Not read by cdb_prefill. */
typedef struct {
    int32_t n_rows;
    const int32_t* slot;
    const int32_t* seq;
    const int32_t* pos;
    const int32_t* c;
    const int32_t* depth;
    const int32_t* d_n_rows;
} cdb_rows;

/* Loop-step outputs (device): exit_score fp32 [n_rows]; exit_mask uint8
 * [n_rows]; cont / exited int32 [n_rows] = batch indices of continuing / exiting
 * rows in batch order (stable compaction); counts int32 [2] = {n_cont, n_exit};
 * exit_next uint8 [n_rows] (optional, may be NULL) = 1 for a continuing row
 * whose token will exit after its next loop. */
typedef struct {
    float* exit_score;
    uint8_t* exit_mask;
    int32_t* cont;
    int32_t* exited;
    int32_t* counts;
    uint8_t* exit_next;
} cdb_step_out;

/* Threshold exits decided on the device (Section 4.3, lookahead gate; App. C.2).
 * The criterion is the model's: exit_kind 0 exits when the gate score after a
 * loop is >= threshold; exit_kind 1 (convergence) when the distance between the
 * states before and after a loop is < threshold, from loop 2 on (after loop 1
 * it compares the recurrent state with the prelude output).  Without lookahead
 * a decision taken after loop r makes r the token's last loop; with lookahead
 * it makes r + 1 the last, so the exit is known one loop step before it
 * happens (minimum depth 2 for the gate, 3 for convergence).  Every token
 * exits after loop r_max at the latest.
 *   pending: device uint8 [n_slots], the lookahead decision carried from one
 *   loop step to the next per state slot; read and written by the library;
 *   the caller zeroes it once when allocating. */
typedef struct {
    float threshold;
    int32_t lookahead;
    uint8_t* pending;
} cdb_gate;

/* Workspace (device scratch) needed for calls with up to max_rows rows
 * (stage calls take up to 256 rows, cdb_prefill up to 512); 0 if unsupported. */
size_t cdb_workspace_bytes(const cdb_model_desc* desc, int32_t max_rows);

/* Clears the workspace's error code (a kernel, not a memset).  Call once after
 * allocating a workspace. */
cdb_status cdb_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream);

/* Prelude stage (Section 4.1; Eq. 1 h^(0) = P(x_t)): h = E[tokens[i]], then the
 * prelude layers with KV plane 0; writes state h[slot] (and e[slot] when
 * injection).  tokens: device int32 [n_rows]. */
cdb_status cdb_boundary_prelude(const cdb_model* model, const cdb_kv* kv, const cdb_state* state,
                                const cdb_rows* rows, const int32_t* tokens, void* ws, size_t ws_bytes,
                                hipStream_t stream);

/* One loop iteration of the shared core over a mixed-depth batch (Eq. 1
 * h^(r+1) = R(h^(r), K^(r)_{<t}); Sections 4.1-4.2):
 *   gather h = state.h[slot] (input injection: u = W_a [h; e]);
 *   every core layer: RMSNorm, q/k/v, RoPE, K/V written to plane c + 1 at pos,
 *   paged attention over positions 0..pos of plane c + 1, output projection and
 *   residual, RMSNorm, SwiGLU MLP and residual;
 *   exit score; exit = (c + 1 == depth), exit_next = (c + 2 == depth);
 *   state.h[slot] = h;
 *   stable compaction into cont / exited;
 *   copy-on-exit (last-exited cache, Section 4.2, Fig. 2): for an exiting row
 *   with depth < r_max, its K/V at pos in plane depth is copied to planes
 *   depth + 1..r_max for every core layer.
 * The caller advances c of continuing rows. */
cdb_status cdb_loop_step(const cdb_model* model, const cdb_kv* kv, const cdb_state* state, const cdb_rows* rows,
                         const cdb_step_out* out, void* ws, size_t ws_bytes, hipStream_t stream);

/* cdb_loop_step with exits decided on the device by `gate` instead of replayed
 * depths (rows->depth is not read and may be NULL): everything else as
 * cdb_loop_step, with copy-on-exit from plane c + 1 of each exiting row. */
cdb_status cdb_loop_step_gated(const cdb_model* model, const cdb_kv* kv, const cdb_state* state,
                               const cdb_rows* rows, const cdb_gate* gate, const cdb_step_out* out, void* ws,
                               size_t ws_bytes, hipStream_t stream);

/* cdb_loop_step for callers that cannot allocate memory (code under HIP graph
 * capture, serving loops and harnesses that forbid allocation): the same
 * computation and outputs, with its scratch taken from a 48 MiB array the
 * library keeps in device memory (one per GPU, held until the process ends)
 * instead of a workspace argument.  It allocates and frees nothing.
 *   d_error: device int32, required; receives the sticky device error codes
 *   (CDB_DEV_*) that cdb_loop_step keeps in its workspace.  The caller zeroes
 *   it once and reads (and re-zeroes) it outside the hot path.
 * Calls whose workspace would exceed 48 MiB (cdb_workspace_bytes of the model
 * at n_rows: e.g. more than 256 rows of the Ouro-shaped model) return
 * CDB_ERR_CAPACITY before anything is enqueued.  Nothing carries over between
 * calls in the scratch.  Every call on one GPU shares its scratch: calls that
 * overlap on a GPU (different streams without ordering, several threads) race
 * and must not be issued. */
cdb_status cdb_loop_step_noalloc(const cdb_model* model, const cdb_kv* kv, const cdb_state* state,
                                 const cdb_rows* rows, const cdb_step_out* out, int32_t* d_error, hipStream_t stream);

/* Coda stage (Section 4.1; Eq. 1 p(x_{t+1}) = softmax(C(h))): coda layers with
 * KV plane r_max + 1 on h = state.h[slot], final RMSNorm, LM head.  logits:
 * device fp32 [n_rows][vocab], required (CDB_ERR_INVALID_ARG if NULL);
 * next_ids: device int32 [n_rows] = argmax (lowest index on ties). */
cdb_status cdb_boundary_coda(const cdb_model* model, const cdb_kv* kv, const cdb_state* state,
                             const cdb_rows* rows, float* logits, int32_t* next_ids, void* ws, size_t ws_bytes,
                             hipStream_t stream);

/* Chunked prefill of one sequence (the prompt KV every decode reads; Section
 * 6.1 runs prompts before decoding): rows i = 0..n_rows-1 are positions
 * pos0 + i with input ids tokens[i] (device int32).  Runs the prelude layers
 * (plane 0), r_max core loops over the whole chunk (loop r writes plane r;
 * prompt tokens take every loop), the coda layers (plane r_max + 1), the final
 * RMSNorm and the LM head: logits device fp32 [n_rows][vocab], next_ids device
 * int32 [n_rows] (argmax, lowest index on ties).  logits may be NULL: then
 * only the last row's greedy id is produced, in next_ids[0] (the LM head runs
 * for the 32-row tile holding that row only).  Positions < pos0 of the
 * sequence must already be in the cache (earlier chunks); every plane's pages
 * of positions < pos0 + n_rows must be mapped.  Earlier positions are read from
 * what each plane's page holds: with aliased planes (the shared layouts) that
 * is an earlier chunk's last loop, so chunking matches one whole-prompt block
 * under the full layout only.  Attention is query-tiled on
 * MFMA; above 256 rows the projections use compute-bound tiles.
 * 1 <= n_rows <= 512, else CDB_ERR_CAPACITY (an empty chunk has no last row to
 * take an id from); the workspace must be sized for n_rows.  One call spans at
 * most 10240 positions: pos0 + n_rows > 10240 returns CDB_ERR_CAPACITY before
 * anything is enqueued (the page ids of the key range are held on chip). */
cdb_status cdb_prefill(const cdb_model* model, const cdb_kv* kv, int32_t seq, int32_t pos0, int32_t n_rows,
                       const int32_t* tokens, float* logits, int32_t* next_ids, void* ws, size_t ws_bytes,
                       hipStream_t stream);

/* Paged decode attention of one layer, alone (the operation every layer of the
 * stage calls runs after writing its K/V; Section 4.2): for row i and head h,
 *   out[i][h*hd + :] = softmax_s(q[i][h*hd + :] . K_s / sqrt(hd)) V_s
 * over positions s = 0..pos[i] of sequence seq[i] in the row's plane of stage
 * `stage` (0 prelude, 1 core -> plane c[i] + 1, 2 coda), layer `layer` of that
 * stage.  q: device fp32 [n_rows][d] (after RoPE); out: device bf16 in the
 * fragment order of the output projection's input: element (m, k) at
 * ((m/32 * d/16 + k/16) * 64 + m%32 + 32*((k%16)/8)) * 8 + k%8, rows rounded up
 * to 32/64/128/256.  order: optional device int32 [n_rows], the rows ranked by
 * descending pos (ties by index); NULL makes the call compute it into the
 * workspace at byte offset 256, from where later calls on the same rows may
 * pass it.  ws: at least 256 + 4 * 256 bytes.  Reads the cache only. */
cdb_status cdb_paged_attention(const cdb_model_desc* desc, const cdb_kv* kv, const cdb_rows* rows, int32_t stage,
                               int32_t layer, const float* q, const int32_t* order, void* out, void* ws,
                               size_t ws_bytes, hipStream_t stream);

/* Reads (and clears) the workspace's sticky device error code.  Synchronises
 * `stream`; not for the hot path. */
cdb_status cdb_read_device_error(void* ws, hipStream_t stream, int32_t* code);

const char* cdb_status_str(cdb_status s);

#ifdef __cplusplus
}
#endif
#endif
