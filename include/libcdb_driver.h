/*
 * libcdb driver -- host-side continuous-depth-batching scheduler (paper
 * Section 4.1) over the libcdb stage calls.  Not part of the optimised path:
 * it decides which rows each stage call gets, maps KV pages, and enqueues the
 * calls; it never reads device results back (exit decisions are replayed from
 * each sequence's depth table, App. B.2).
 *
 * Two queues: the boundary queue (tokens that left the core -> coda, then the
 * prelude of their next input; newly admitted sequences -> prelude) and the
 * loop queue (tokens in the core).  Boundary work runs first once
 * min_coda_batch exits are waiting, or when no loop work is left.
 *   refill       running loop rows stay in the batch; freed rows are filled
 *                from the loop queue at the next step (Section 4.1, Fig. 1)
 *   no-refill    a batch is formed once per round and shrinks until all its
 *                tokens exited; coda and prelude then run for the round
 *   fixed_depth  every token runs r_max loops (continuous batching baseline)
 *   gated        exits decided on the device by a threshold (Section 4.3;
 *                App. C.2).  With lookahead the device's decision after one
 *                loop step governs the step after next, so the host plans
 *                each step from results one step old and never stalls the
 *                device; without it every loop step waits for its own result.
 * Pages: every plane of a sequence is mapped at admission (lowest free id
 * first, (sequence, page, plane) order) and released when it finishes.
 */
#ifndef LIBCDB_DRIVER_H
#define LIBCDB_DRIVER_H

#include <stddef.h>
#include <stdint.h>

#include "libcdb.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct cdb_driver cdb_driver;

typedef struct {
    int32_t max_batch;       /* rows per loop step (<= 256) */
    int32_t max_active;      /* sequences in flight at once */
    int32_t refill;          /* 1 refill, 0 no-refill */
    int32_t fixed_depth;     /* 1: every token loops r_max times */
    int32_t min_coda_batch;  /* exits to accumulate before the coda runs (>= 1) */
    int32_t r_max;
    int32_t has_prelude, has_coda;  /* whether the model has prelude / coda layers (their pools are used) */
    int32_t max_seqs, max_pages;    /* page-table shape [max_seqs][r_max + 2][max_pages] */
    int32_t pre_pages, core_pages, coda_pages;  /* pool sizes */
    int32_t kv_layout;              /* CDB_KV_FULL, CDB_KV_SHARED or CDB_KV_FIRST_THEN_SHARED */
    int32_t gated;                  /* 1: exits decided on the device by a threshold (cdb_gate) */
    int32_t lookahead;              /* gated: the decision after loop r ends the token after loop r + 1 */
    float threshold;                /* gated: the criterion's threshold */
    int32_t prefill_chunk;          /* 0: prompts are prefilled by the caller (cdb_driver_add_sequence);
                                       1..512: prompts of requests added with cdb_driver_add_request run
                                       through cdb_prefill in chunks of at most this many tokens */
    int32_t sync_steps;             /* 1: the runner waits for every loop step before planning the next
                                       (the synchronous scheduler, for comparison); 0: never waits */
    int32_t boundary_stream;        /* 0: every call on one stream.  1, 2: prelude, coda and prefill calls
                                       run on a second stream with their own workspace, ordered with the
                                       loop steps by events (Section 4.3).  In refill mode the tokens whose
                                       prelude was planned since the last loop step are held back from
                                       the next step, which so does not wait for that boundary work:
                                       with 1 they still fill rows the loop queue leaves free (no row
                                       idles; the step then waits for their prelude), with 2 they always
                                       join the step after next (the boundary work of step k overlaps
                                       step k + 1 whole, at the cost of rows idling one step) */
    int32_t graph_loop;             /* 1: the loop step is captured once in a HIP graph at max_batch rows with
                                       the row count in device memory (cdb_rows.d_n_rows) and each loop tick
                                       replays it: one launch instead of the step's kernels (Section 4.3,
                                       static shapes and graphs).  Results are those of the direct calls. */
} cdb_driver_config;

/* Core KV layouts (Section 4.2, App. C.1, Table 1), all by page-table aliasing:
 *   FULL              one page per core plane (depth-indexed, last-exited copies)
 *   SHARED            every core plane maps the same page: one slot per layer,
 *                     overwritten at every loop
 *   FIRST_THEN_SHARED plane 1 private, planes 2..r_max share a second page */
enum { CDB_KV_FULL = 0, CDB_KV_SHARED = 1, CDB_KV_FIRST_THEN_SHARED = 2 };

enum { CDB_TICK_NONE = 0, CDB_TICK_PRELUDE_FIRST = 1, CDB_TICK_LOOP = 2, CDB_TICK_CODA = 3, CDB_TICK_PREFILL = 4 };

/* One planned stage call (host arrays of up to 256 rows).  For CDB_TICK_CODA
 * the first n_continue rows continue (the prelude of their next input follows
 * in the same tick, at pos + 1); the rest finish their sequence.  For
 * CDB_TICK_PREFILL the call is one prompt chunk of sequence seq[0]: n_rows
 * tokens from position pos[0]; n_continue = 1 when it ends the prompt (its last
 * row's greedy id is the first decode input). */
typedef struct {
    int32_t stage;
    int32_t n_rows, n_continue;
    int32_t slot[256], seq[256], pos[256], c[256], depth[256], decode_index[256];
    double wait_until;
} cdb_driver_tick;

typedef struct {
    int64_t loop_steps, loop_rows, idle_rows;  /* idle_rows: max_batch - rows, summed over loop steps */
    int64_t coda_calls, coda_rows, prelude_calls, prelude_rows;
    int64_t tokens;                            /* decode tokens finished (coda rows) */
    int64_t prefill_calls, prefill_tokens;     /* prompt chunks run by the driver */
    int64_t host_wait_us;                      /* cdb_driver_run: time the host spent waiting on the device
                                                  (staging-buffer reuse, page-table uploads, gated
                                                  decisions, sync_steps), microseconds */
    int64_t pt_uploads, pt_upload_bytes;       /* page-table uploads and the bytes they copied */
    int64_t graph_launches;                    /* loop steps run as graph replays (graph_loop) */
} cdb_driver_stats;

cdb_driver* cdb_driver_create(const cdb_driver_config* cfg);
void cdb_driver_destroy(cdb_driver* d);

/* Adds a request in arrival order: its prompt (already prefilled: its KV must
 * be present when the sequence is admitted) and the exit depth of each of its
 * n_decode decode inputs (NULL in gated mode).  Returns the sequence id (= its
 * row of the page table and its state slot) or -1: a bad argument, max_seqs
 * reached, an arrival before the previous one, a depth outside [1, r_max], or
 * a sequence that could never be admitted (prompt_len + n_decode positions
 * need more pages per plane than max_pages, or more pages than a pool holds
 * in all). */
int32_t cdb_driver_add_sequence(cdb_driver* d, int32_t prompt_len, int32_t n_decode, const int32_t* depths,
                                double arrival);

/* Adds a request whose prompt the driver prefills (prefill_chunk > 0):
 * prompt_ids (host, prompt_len ids, copied).  Scheduling priority (Section
 * 4.1): the coda, then prompt chunks (one per call, first admitted first),
 * then the prelude of first decode inputs, then loop steps.  The first decode
 * input is the prompt's greedy continuation, passed on the device.  Returns
 * the sequence id or -1 (the reasons of cdb_driver_add_sequence, or a prompt
 * longer than the 10240 positions one cdb_prefill call spans). */
int32_t cdb_driver_add_request(cdb_driver* d, int32_t prompt_len, const int32_t* prompt_ids, int32_t n_decode,
                               const int32_t* depths, double arrival);

/* Host page table [max_seqs][r_max + 2][max_pages] as the driver maintains it. */
const int32_t* cdb_driver_page_table(cdb_driver* d);

/* Scheduler stepping without a device (tests, simulations): next() plans a
 * call (1), reports completion of all work (0) or that nothing can run before
 * t->wait_until (-1); complete() applies a planned call's effect. */
int32_t cdb_driver_next(cdb_driver* d, cdb_driver_tick* t);
int32_t cdb_driver_complete(cdb_driver* d, const cdb_driver_tick* t);

/* Gated mode: the device's exit_mask and exit_next (uint8 per row, in the
 * tick's row order) of a completed loop tick.  Without lookahead it must be
 * given before that tick is completed; with lookahead before the next loop
 * tick is completed.  Returns -1 if the mask disagrees with the exits the
 * scheduler applied. */
int32_t cdb_driver_loop_result(cdb_driver* d, const cdb_driver_tick* t, const uint8_t* exit_mask,
                               const uint8_t* exit_next);
void cdb_driver_set_time(cdb_driver* d, double now_seconds);

int32_t cdb_driver_get_stats(const cdb_driver* d, cdb_driver_stats* out);

/* Pages currently mapped in each pool (aliased pages count once). */
int32_t cdb_driver_pages_in_use(const cdb_driver* d, int32_t* pre, int32_t* core, int32_t* coda);

/* Normalised latency per sequence (finish - arrival) / n_decode, in seconds;
 * -1 for unfinished ones.  Returns the number written. */
int32_t cdb_driver_latencies(const cdb_driver* d, double* normalized, int32_t n);

/* Device scratch cdb_driver_run needs for this driver and a model with
 * `vocab` logits. */
size_t cdb_driver_scratch_bytes(const cdb_driver* d, int32_t vocab);

/* Runs every added request to completion on the device: plans each call,
 * stages its rows through pinned host memory, enqueues the stage call on
 * `stream`.  first_tokens (host, per sequence) is each sequence's first decode
 * input (may be NULL when every request was added with
 * cdb_driver_add_request: their first inputs come from the prefill); later
 * inputs are the coda's greedy ids, passed on device.  With prefill_chunk >
 * 256 the workspace must be sized for prefill_chunk rows.  The page
 * table in kv->page_table (device) is overwritten from the driver's.
 * state needs a slot per sequence (n_slots >= max_seqs).  scratch: device,
 * cdb_driver_scratch_bytes(d, vocab).  tokens_out (device,
 * optional): int32 [max_seqs][tokens_stride] receives, at [seq][k], the greedy
 * id the coda produced after decode input k (tokens_stride >= every
 * sequence's n_decode, else CDB_ERR_INVALID_ARG).  Gated mode: the device's
 * exit decisions are copied back after every loop step and fed to the
 * scheduler (one step late with lookahead, the last step's after the run);
 * CDB_ERR_INVALID_ARG if they ever disagree with the exits applied.
 * boundary_stream: the loop steps run on `stream`, the prelude, coda and
 * prefill calls on a second stream the runner creates (default priority) and
 * destroys before returning; ws then holds two workspaces, ws_bytes / 2 each
 * (rounded down to 256 bytes; the second starts there), the first for loop
 * steps, the second for boundary stages (its device error word covers those).
 * Page-table changes after the first upload copy only the blocks of
 * sequences admitted or released.  Returns a cdb_status; *seconds = wall
 * time including the final synchronisation.  With the environment variable
 * CDB_DRIVER_PROGRESS set, a progress line goes to stderr every 10 s. */
int32_t cdb_driver_run(cdb_driver* d, const cdb_model* model, const cdb_kv* kv, const cdb_state* state, void* scratch,
                       size_t scratch_bytes, const int32_t* first_tokens, int32_t* tokens_out,
                       int32_t tokens_stride, void* ws, size_t ws_bytes, hipStream_t stream, double* seconds);

#ifdef __cplusplus
}
#endif
#endif
