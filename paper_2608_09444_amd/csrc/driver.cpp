// Host driver for continuous depth batching (paper Section 4.1): a two-queue
// scheduler (boundary stages, loop steps) that builds every stage call's
// batch, a page allocator, and a runner that enqueues the libcdb stage calls.
//
// Scheduling (host only, no device access):
//  * Sequences are admitted in arrival order while fewer than `max_active` are
//    in flight and their pages fit; pages of every plane are mapped at
//    admission, lowest free id first.
//  * Boundary queue: tokens that just exited the core (coda, then the prelude
//    of the next token) and newly admitted sequences (prelude of the first
//    decode input).  It runs first when it holds at least `min_coda_batch`
//    exits, or when no loop work is left (Section 4.1: coda has priority, the
//    prelude follows it directly; a minimum coda batch lets exits accumulate).
//  * Loop queue: tokens in the core.  Refill mode keeps the rows of the
//    running batch at the front and fills freed rows from the queue; no-refill
//    mode forms a batch once per round and lets it shrink until every token has
//    exited (Section 4.1, Fig. 1 right).  Fixed-depth mode runs every token for
//    r_max loops (continuous batching, the baseline the paper compares with).
//  * Exit decisions are replayed from each sequence's depth table
//    (App. B.2), so the host knows every exit without reading the device; in
//    gated mode they come from the device (cdb_driver_loop_result), one loop
//    step late with the lookahead gate (Section 4.3).
//
// Running (cdb_driver_run): each tick's rows go through pinned host buffers and
// one asynchronous copy to the device, then the stage call; the coda batch
// lists continuing sequences first, so its device-side next-token ids are the
// prelude's tokens for the next tick without any host round trip.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <chrono>
#include <deque>
#include <vector>

#include "../../include/libcdb.h"
#include "../../include/libcdb_driver.h"

namespace cdb {
// defined with the row kernels
hipError_t launch_scatter_ids(int M, const int32_t* ids, const int32_t* seq, const int32_t* index, int max_seqs,
                              int stride, int32_t* out, hipStream_t st);
hipError_t launch_gather_ids(int M, const int32_t* seq, const int32_t* src, int max_seqs, int32_t* dst,
                             hipStream_t st);
}  // namespace cdb

namespace {

enum SeqState { WAITING = 0, PRELUDE = 1, LOOP = 2, EXITED = 3, DONE = 4, PREFILL = 5 };

struct Seq {
    int32_t prompt_len = 0, n_decode = 0;
    std::vector<int32_t> prompt;  // ids of a prompt the driver prefills (empty: prefilled by the caller)
    int32_t prefilled = 0;        // prompt positions done
    std::vector<int32_t> depth;  // per decode input
    double arrival = 0.0;
    int state = WAITING;
    int32_t t = 0;  // decode input index of the token in flight (position prompt_len + t)
    int32_t c = 0;  // loops completed by that token
    int32_t pages = 0;
    double admit_time = -1.0, done_time = -1.0;
    bool exit_now = false;  // gated: the current loop is the token's last (known before the step completes)
};

struct Allocator {
    std::vector<int32_t> free_ids;  // kept sorted descending: back() is the lowest
    explicit Allocator(int32_t n = 0) {
        for (int32_t i = n - 1; i >= 0; --i) free_ids.push_back(i);
    }
    int32_t available() const { return (int32_t)free_ids.size(); }
    int32_t take() {
        const int32_t id = free_ids.back();
        free_ids.pop_back();
        return id;
    }
    void give(int32_t id) {
        free_ids.insert(std::upper_bound(free_ids.begin(), free_ids.end(), id, std::greater<int32_t>()), id);
    }
};

}  // namespace

struct cdb_driver {
    cdb_driver_config cfg;
    std::vector<Seq> seqs;
    std::vector<int32_t> page_table;  // [max_seqs][r_max + 2][max_pages]
    Allocator pre, core, coda;
    size_t next_arrival = 0;  // index into seqs in arrival order (sequences are added in arrival order)
    int32_t active = 0;
    std::deque<int32_t> exited;   // sequences whose token left the core, awaiting the coda
    std::deque<int32_t> prefillq; // admitted sequences whose prompt is still being prefilled
    std::deque<int32_t> fresh;    // admitted sequences awaiting the prelude of their first input
    std::deque<int32_t> loopq;    // sequences whose token waits for its next loop
    std::vector<int32_t> batch;   // rows of the running loop batch (refill keeps it)
    bool round_open = false;      // no-refill: a round is running
    cdb_driver_stats stats;
    double now = 0.0;  // seconds, advanced by the runner (or by tests)
    bool table_all_dirty = true;         // the whole page table must be uploaded (first run)
    std::vector<int32_t> dirty_seqs;     // sequences whose page-table block changed since the last upload
    std::vector<uint8_t> seq_dirty;      // per sequence: listed in dirty_seqs
    std::deque<int32_t> loop_hold;       // boundary stream: tokens prelude'd since the last loop tick
    std::vector<uint8_t> last_plan;  // gated: exits applied to the last completed loop tick, in row order
    bool result_pending = false;     // gated lookahead: the last completed loop tick's result is still due
};

static int32_t planes(const cdb_driver* d) { return d->cfg.r_max + 2; }

static void mark_dirty(cdb_driver* d, int32_t q) {
    if (!d->seq_dirty[q]) {
        d->seq_dirty[q] = 1;
        d->dirty_seqs.push_back(q);
    }
}

// Tokens whose prelude was just planned: with boundary stages on their own
// stream they join the loop step after next, so the next loop step does not
// wait for that prelude (refill mode); otherwise the loop queue directly.
static void to_loop_queue(cdb_driver* d, int32_t q) {
    if (d->cfg.boundary_stream && d->cfg.refill)
        d->loop_hold.push_back(q);
    else
        d->loopq.push_back(q);
}

static int32_t depth_of(const cdb_driver* d, const Seq& s) {
    if (d->cfg.fixed_depth) return d->cfg.r_max;
    if (d->cfg.gated) return 0;  // decided on the device
    return s.depth[s.t];
}

// Whether the token's current loop (index s.c) is its last.
static bool exits_now(const cdb_driver* d, const Seq& s) {
    if (s.c + 1 >= d->cfg.r_max) return true;
    if (d->cfg.gated) return s.exit_now;
    return s.c + 1 == depth_of(d, s);
}

// Distinct core pages per token page under the layout.
static int32_t core_slots(const cdb_driver* d) {
    if (d->cfg.kv_layout == CDB_KV_SHARED) return 1;
    if (d->cfg.kv_layout == CDB_KV_FIRST_THEN_SHARED) return d->cfg.r_max > 1 ? 2 : 1;
    return d->cfg.r_max;
}

static bool try_admit(cdb_driver* d, int32_t q) {
    Seq& s = d->seqs[q];
    const int32_t need = (s.prompt_len + s.n_decode + 15) / 16;
    if (need > d->cfg.max_pages) return false;
    const bool use_pre = d->cfg.has_prelude, use_coda = d->cfg.has_coda;
    if (d->core.available() < need * core_slots(d) || (use_pre && d->pre.available() < need) ||
        (use_coda && d->coda.available() < need))
        return false;
    // (sequence, page, plane) order, lowest free id first; aliased planes reuse
    // the page of the plane they share with
    for (int32_t pg = 0; pg < need; ++pg) {
        int32_t shared_id = -1;
        for (int32_t pl = 0; pl < planes(d); ++pl) {
            int32_t id = -1;
            if (pl == 0) {
                if (use_pre) id = d->pre.take();
            } else if (pl == d->cfg.r_max + 1) {
                if (use_coda) id = d->coda.take();
            } else if (d->cfg.kv_layout == CDB_KV_SHARED ||
                       (d->cfg.kv_layout == CDB_KV_FIRST_THEN_SHARED && pl >= 2)) {
                if (shared_id < 0) shared_id = d->core.take();
                id = shared_id;
            } else {
                id = d->core.take();
            }
            d->page_table[((size_t)q * planes(d) + pl) * d->cfg.max_pages + pg] = id;
        }
    }
    s.pages = need;
    s.t = 0;
    s.c = 0;
    s.admit_time = d->now;
    d->active++;
    if (!s.prompt.empty()) {
        s.state = PREFILL;
        s.prefilled = 0;
        d->prefillq.push_back(q);
    } else {
        s.state = PRELUDE;
        d->fresh.push_back(q);
    }
    mark_dirty(d, q);
    return true;
}

static void release(cdb_driver* d, int32_t q) {
    for (int32_t pg = 0; pg < d->seqs[q].pages; ++pg) {
        std::vector<int32_t> core_given;
        for (int32_t pl = 0; pl < planes(d); ++pl) {
            int32_t& id = d->page_table[((size_t)q * planes(d) + pl) * d->cfg.max_pages + pg];
            if (id < 0) continue;
            if (pl == 0) {
                d->pre.give(id);
            } else if (pl == d->cfg.r_max + 1) {
                d->coda.give(id);
            } else if (std::find(core_given.begin(), core_given.end(), id) == core_given.end()) {
                d->core.give(id);  // aliased planes give their page back once
                core_given.push_back(id);
            }
            id = -1;
        }
    }
    d->active--;
    mark_dirty(d, q);
}

static void admit(cdb_driver* d) {
    while (d->next_arrival < d->seqs.size() && d->active < d->cfg.max_active &&
           d->seqs[d->next_arrival].arrival <= d->now) {
        if (!try_admit(d, (int32_t)d->next_arrival)) break;
        d->next_arrival++;
    }
}

static void fill_rows(const cdb_driver* d, const std::vector<int32_t>& qs, cdb_driver_tick* t, bool loop, int32_t dpos) {
    t->n_rows = (int32_t)qs.size();
    for (size_t i = 0; i < qs.size(); ++i) {
        const Seq& s = d->seqs[qs[i]];
        t->seq[i] = qs[i];
        t->slot[i] = qs[i];
        t->pos[i] = s.prompt_len + s.t + dpos;
        t->c[i] = loop ? s.c : 0;
        t->depth[i] = loop ? depth_of(d, s) : 0;
        t->decode_index[i] = s.t + dpos;
    }
}

extern "C" {

cdb_driver* cdb_driver_create(const cdb_driver_config* cfg) {
    if (!cfg || cfg->max_batch < 1 || cfg->max_batch > 256 || cfg->r_max < 1 || cfg->max_seqs < 1 ||
        cfg->max_pages < 1 || cfg->max_active < 1 || cfg->min_coda_batch < 1 || cfg->kv_layout < 0 ||
        cfg->kv_layout > 2 || (cfg->gated && cfg->fixed_depth) || cfg->prefill_chunk < 0 || cfg->prefill_chunk > 512 ||
        cfg->boundary_stream < 0 || cfg->boundary_stream > 2 || cfg->graph_loop < 0 || cfg->graph_loop > 1)
        return nullptr;
    cdb_driver* d = new cdb_driver();
    d->cfg = *cfg;
    d->page_table.assign((size_t)cfg->max_seqs * (cfg->r_max + 2) * cfg->max_pages, -1);
    d->seq_dirty.assign(cfg->max_seqs, 0);
    d->pre = Allocator(cfg->has_prelude ? cfg->pre_pages : 0);
    d->core = Allocator(cfg->core_pages);
    d->coda = Allocator(cfg->has_coda ? cfg->coda_pages : 0);
    memset(&d->stats, 0, sizeof(d->stats));
    return d;
}

void cdb_driver_destroy(cdb_driver* d) { delete d; }

int32_t cdb_driver_add_sequence(cdb_driver* d, int32_t prompt_len, int32_t n_decode, const int32_t* depths,
                                double arrival) {
    if (!d || prompt_len < 1 || n_decode < 1 || (!depths && !d->cfg.gated)) return -1;
    if ((int32_t)d->seqs.size() >= d->cfg.max_seqs) return -1;
    if (!d->seqs.empty() && arrival < d->seqs.back().arrival) return -1;  // arrival order
    if (depths)
        for (int32_t i = 0; i < n_decode; ++i)
            if (depths[i] < 1 || depths[i] > d->cfg.r_max) return -1;
    // a sequence no pool state could ever admit would stall the queue behind it
    const int64_t need = ((int64_t)prompt_len + n_decode + 15) / 16;  // pages per plane
    if (need > d->cfg.max_pages || need * core_slots(d) > d->cfg.core_pages ||
        (d->cfg.has_prelude && need > d->cfg.pre_pages) || (d->cfg.has_coda && need > d->cfg.coda_pages))
        return -1;
    Seq s;
    s.prompt_len = prompt_len;
    s.n_decode = n_decode;
    if (depths) s.depth.assign(depths, depths + n_decode);
    s.arrival = arrival;
    d->seqs.push_back(std::move(s));
    return (int32_t)d->seqs.size() - 1;
}

int32_t cdb_driver_add_request(cdb_driver* d, int32_t prompt_len, const int32_t* prompt_ids, int32_t n_decode,
                               const int32_t* depths, double arrival) {
    // one cdb_prefill call spans at most 10240 positions
    if (!d || d->cfg.prefill_chunk < 1 || !prompt_ids || prompt_len < 1 || prompt_len > 10240) return -1;
    const int32_t q = cdb_driver_add_sequence(d, prompt_len, n_decode, depths, arrival);
    if (q >= 0) d->seqs[q].prompt.assign(prompt_ids, prompt_ids + prompt_len);
    return q;
}

const int32_t* cdb_driver_page_table(cdb_driver* d) { return d ? d->page_table.data() : nullptr; }

void cdb_driver_set_time(cdb_driver* d, double now) {
    if (d) d->now = now;
}

// Plans the next stage call.  Returns 1 with *t filled, 0 when all work is done,
// -1 when nothing can run until a later arrival (t->wait_until holds it).
int32_t cdb_driver_next(cdb_driver* d, cdb_driver_tick* t) {
    if (!d || !t) return -1;
    admit(d);
    t->n_continue = 0;
    auto coda_tick = [&]() {
        const int32_t n = std::min<int32_t>((int32_t)d->exited.size(), 256);
        std::vector<int32_t> rows(d->exited.begin(), d->exited.begin() + n);
        // continuing sequences first, so the coda's ids feed the next prelude in order
        std::stable_partition(rows.begin(), rows.end(),
                              [&](int32_t q) { return d->seqs[q].t + 1 < d->seqs[q].n_decode; });
        t->stage = CDB_TICK_CODA;
        fill_rows(d, rows, t, false, 0);
        for (int32_t q : rows) t->n_continue += d->seqs[q].t + 1 < d->seqs[q].n_decode;
        return 1;
    };
    auto prelude_tick = [&]() {
        const int32_t n = std::min<int32_t>((int32_t)d->fresh.size(), 256);
        std::vector<int32_t> rows(d->fresh.begin(), d->fresh.begin() + n);
        t->stage = CDB_TICK_PRELUDE_FIRST;
        fill_rows(d, rows, t, false, 0);
        return 1;
    };
    auto loop_tick = [&]() {
        t->stage = CDB_TICK_LOOP;
        fill_rows(d, d->batch, t, true, 0);
        return 1;
    };
    auto prefill_tick = [&]() {
        const int32_t q = d->prefillq.front();
        const Seq& s = d->seqs[q];
        const int32_t n = std::min(d->cfg.prefill_chunk, s.prompt_len - s.prefilled);
        t->stage = CDB_TICK_PREFILL;
        t->n_rows = n;
        t->n_continue = s.prefilled + n == s.prompt_len ? 1 : 0;
        t->seq[0] = q;
        t->slot[0] = q;
        t->pos[0] = s.prefilled;
        t->c[0] = 0;
        t->depth[0] = 0;
        t->decode_index[0] = 0;
        return 1;
    };
    if (d->cfg.refill) {
        // held tokens join now when nothing else is left to run in the core
        if (d->loopq.empty() && d->batch.empty())
            while (!d->loop_hold.empty()) {
                d->loopq.push_back(d->loop_hold.front());
                d->loop_hold.pop_front();
            }
        const bool loop_left = !d->loopq.empty() || !d->batch.empty();
        const int32_t n_exit = (int32_t)d->exited.size();
        if (n_exit > 0 && (n_exit >= d->cfg.min_coda_batch || !loop_left)) return coda_tick();
        if (!d->prefillq.empty()) return prefill_tick();
        if (!d->fresh.empty()) return prelude_tick();
        if (loop_left) {
            // keep the running rows, fill freed rows from the loop queue
            while ((int32_t)d->batch.size() < d->cfg.max_batch && !d->loopq.empty()) {
                d->batch.push_back(d->loopq.front());
                d->loopq.pop_front();
            }
            // boundary_stream 1: held tokens still take rows the queue left free
            // (this step then waits for their prelude); 2: they join the next step
            if (d->cfg.boundary_stream == 1)
                while ((int32_t)d->batch.size() < d->cfg.max_batch && !d->loop_hold.empty()) {
                    d->batch.push_back(d->loop_hold.front());
                    d->loop_hold.pop_front();
                }
            // tokens held back from this step join the next one
            while (!d->loop_hold.empty()) {
                d->loopq.push_back(d->loop_hold.front());
                d->loop_hold.pop_front();
            }
            return loop_tick();
        }
    } else {
        if (d->round_open) {
            if (!d->batch.empty()) return loop_tick();
            if (!d->exited.empty()) return coda_tick();
            d->round_open = false;
        }
        if (!d->exited.empty()) return coda_tick();
        if (!d->prefillq.empty()) return prefill_tick();
        if (!d->fresh.empty()) return prelude_tick();
        if (!d->loopq.empty()) {
            while ((int32_t)d->batch.size() < d->cfg.max_batch && !d->loopq.empty()) {
                d->batch.push_back(d->loopq.front());
                d->loopq.pop_front();
            }
            d->round_open = true;
            return loop_tick();
        }
    }
    if (d->next_arrival < d->seqs.size()) {
        t->stage = CDB_TICK_NONE;
        t->n_rows = 0;
        t->wait_until = d->seqs[d->next_arrival].arrival;
        return -1;
    }
    return 0;
}

// Applies a planned stage call's effect on the schedule.
int32_t cdb_driver_complete(cdb_driver* d, const cdb_driver_tick* t) {
    if (!d || !t) return -1;
    if (t->stage == CDB_TICK_CODA) {
        std::vector<int32_t> cont;
        for (int32_t i = 0; i < t->n_rows; ++i) {
            const int32_t q = t->seq[i];
            Seq& s = d->seqs[q];
            d->exited.erase(std::find(d->exited.begin(), d->exited.end(), q));
            d->stats.tokens++;
            if (s.t + 1 < s.n_decode) {
                s.t++;
                s.c = 0;
                s.exit_now = false;
                s.state = LOOP;
                cont.push_back(q);
            } else {
                s.state = DONE;
                s.done_time = d->now;
                release(d, q);
            }
        }
        d->stats.coda_calls++;
        d->stats.coda_rows += t->n_rows;
        // the prelude of the continuing sequences' next inputs runs right after
        d->stats.prelude_calls += cont.empty() ? 0 : 1;
        d->stats.prelude_rows += (int64_t)cont.size();
        for (int32_t q : cont) to_loop_queue(d, q);
        if (!d->cfg.refill && d->exited.empty() && d->batch.empty()) d->round_open = false;  // round over
    } else if (t->stage == CDB_TICK_PREFILL) {
        const int32_t q = t->seq[0];
        if (d->prefillq.empty() || d->prefillq.front() != q) return -1;
        Seq& s = d->seqs[q];
        if (t->pos[0] != s.prefilled || t->n_rows < 1 || s.prefilled + t->n_rows > s.prompt_len) return -1;
        s.prefilled += t->n_rows;
        d->stats.prefill_calls++;
        d->stats.prefill_tokens += t->n_rows;
        if (s.prefilled == s.prompt_len) {
            d->prefillq.pop_front();
            s.state = PRELUDE;
            d->fresh.push_back(q);
        }
    } else if (t->stage == CDB_TICK_PRELUDE_FIRST) {
        for (int32_t i = 0; i < t->n_rows; ++i) {
            const int32_t q = t->seq[i];
            d->fresh.erase(std::find(d->fresh.begin(), d->fresh.end(), q));
            d->seqs[q].state = LOOP;
            to_loop_queue(d, q);
        }
        d->stats.prelude_calls++;
        d->stats.prelude_rows += t->n_rows;
    } else if (t->stage == CDB_TICK_LOOP) {
        if (d->cfg.gated && d->cfg.lookahead && d->result_pending) return -1;  // previous loop's result not given
        std::vector<int32_t> keep;
        d->last_plan.assign(t->n_rows, 0);
        for (int32_t i = 0; i < t->n_rows; ++i) {
            const int32_t q = t->seq[i];
            Seq& s = d->seqs[q];
            if (exits_now(d, s)) {
                s.state = EXITED;
                d->exited.push_back(q);
                d->last_plan[i] = 1;
            } else {
                s.c++;
                s.exit_now = false;
                keep.push_back(q);
            }
        }
        d->result_pending = d->cfg.gated && d->cfg.lookahead;
        d->batch = keep;
        d->stats.loop_steps++;
        d->stats.loop_rows += t->n_rows;
        d->stats.idle_rows += d->cfg.max_batch - t->n_rows;
    }
    return 0;
}

int32_t cdb_driver_loop_result(cdb_driver* d, const cdb_driver_tick* t, const uint8_t* exit_mask,
                               const uint8_t* exit_next) {
    if (!d || !t || !exit_mask || t->stage != CDB_TICK_LOOP || !d->cfg.gated) return -1;
    if (!d->cfg.lookahead) {
        // before completion: the step's own decisions end the tokens
        for (int32_t i = 0; i < t->n_rows; ++i) d->seqs[t->seq[i]].exit_now = exit_mask[i] != 0;
        return 0;
    }
    // after completion: check the exits applied, carry the next decisions
    if (!d->result_pending || (int32_t)d->last_plan.size() != t->n_rows) return -1;
    d->result_pending = false;
    int32_t status = 0;
    for (int32_t i = 0; i < t->n_rows; ++i) {
        if ((exit_mask[i] != 0) != (d->last_plan[i] != 0)) status = -1;
        Seq& s = d->seqs[t->seq[i]];
        if (!d->last_plan[i] && exit_next) s.exit_now = exit_next[i] != 0;
    }
    return status;
}

int32_t cdb_driver_pages_in_use(const cdb_driver* d, int32_t* pre, int32_t* core, int32_t* coda) {
    if (!d) return -1;
    if (pre) *pre = (d->cfg.has_prelude ? d->cfg.pre_pages : 0) - d->pre.available();
    if (core) *core = d->cfg.core_pages - d->core.available();
    if (coda) *coda = (d->cfg.has_coda ? d->cfg.coda_pages : 0) - d->coda.available();
    return 0;
}

int32_t cdb_driver_get_stats(const cdb_driver* d, cdb_driver_stats* out) {
    if (!d || !out) return -1;
    *out = d->stats;
    return 0;
}

int32_t cdb_driver_latencies(const cdb_driver* d, double* normalized, int32_t n) {
    if (!d || !normalized) return -1;
    int32_t k = 0;
    for (const Seq& s : d->seqs) {
        if (k >= n) break;
        normalized[k++] = s.done_time >= 0 ? (s.done_time - s.arrival) / s.n_decode : -1.0;
    }
    return k;
}

// ------------------------------------------------------------------ runner

// Device scratch: three row sets (6 x 256 int32 each: the loop step's, the
// boundary stage's, the prelude's after a coda), next ids (256), loop-step
// outputs (scores, mask, cont, exited, counts, exit_next), the gate's pending
// flags (max_seqs), each sequence's first decode input (max_seqs int32),
// logits (256 x vocab fp32).
struct ScratchLayout {
    size_t rows, ids, step, pending, first, logits, total;
};
// one set of stage rows on the device: slot, seq, pos, c, depth and a sixth
// array (decode index or token) of 256 entries each, then the live row count
// a captured loop step reads (cdb_rows.d_n_rows)
constexpr int kRowSetInts = 6 * 256 + 64;
constexpr int kRowCount = 6 * 256;

static ScratchLayout scratch_layout(int32_t max_seqs, int32_t vocab) {
    ScratchLayout L;
    size_t off = 0;
    L.rows = off;
    off += 3 * (size_t)kRowSetInts * 4;
    L.ids = off;
    off += 256 * 4;
    L.step = off;
    off += 256 * 4 + 256 + 256 * 4 * 2 + 2 * 4 + 256;
    off = (off + 255) & ~(size_t)255;
    L.pending = off;
    off += ((size_t)max_seqs + 255) & ~(size_t)255;
    L.first = off;
    off += ((size_t)max_seqs * 4 + 255) & ~(size_t)255;
    L.logits = off;
    off += (size_t)256 * vocab * 4;
    L.total = off;
    return L;
}

size_t cdb_driver_scratch_bytes(const cdb_driver* d, int32_t vocab) {
    return d && vocab > 0 ? scratch_layout(d->cfg.max_seqs, vocab).total : 0;
}

namespace {

// Host-side waits on the device, timed for the driver's statistics.
struct Waits {
    std::chrono::steady_clock::duration total{};
    void on(hipEvent_t e) {
        const auto t0 = std::chrono::steady_clock::now();
        hipEventSynchronize(e);
        total += std::chrono::steady_clock::now() - t0;
    }
    hipError_t on(hipStream_t s) {
        const auto t0 = std::chrono::steady_clock::now();
        const hipError_t r = hipStreamSynchronize(s);
        total += std::chrono::steady_clock::now() - t0;
        return r;
    }
};

// A ring of events recorded on one stream, numbered by a running count, so
// another stream can wait for "the n-th record" (a later record of the same
// slot orders at least as late, which keeps such waits correct).
struct EventRing {
    static constexpr int N = 64;
    hipEvent_t ev[N];
    int64_t count = 0;  // records so far; record k (1-based) sits in slot (k - 1) % N
    EventRing() {
        for (int i = 0; i < N; ++i) hipEventCreateWithFlags(&ev[i], hipEventDisableTiming);
    }
    ~EventRing() {
        for (int i = 0; i < N; ++i) hipEventDestroy(ev[i]);
    }
    int64_t record(hipStream_t s) {
        hipEventRecord(ev[count % N], s);
        return ++count;
    }
    hipEvent_t at(int64_t k) const { return ev[(k - 1) % N]; }
};

}  // namespace

int32_t cdb_driver_run(cdb_driver* d, const cdb_model* model, const cdb_kv* kv, const cdb_state* state, void* scratch,
                       size_t scratch_bytes, const int32_t* first_tokens, int32_t* tokens_out,
                       int32_t tokens_stride, void* ws, size_t ws_bytes, hipStream_t stream, double* seconds) {
    if (!d || !model || !kv || !state || !scratch || !ws || !kv->page_table) return CDB_ERR_INVALID_ARG;
    for (const Seq& s : d->seqs)
        if (s.prompt.empty() && !first_tokens) return CDB_ERR_INVALID_ARG;  // its first input must be given
    if (tokens_out) {
        for (const Seq& s : d->seqs)
            if (s.n_decode > tokens_stride) return CDB_ERR_INVALID_ARG;
    }
    const ScratchLayout SL = scratch_layout(d->cfg.max_seqs, model->desc.vocab);
    if (scratch_bytes < SL.total) return CDB_ERR_CAPACITY;
    if (kv->max_seqs != d->cfg.max_seqs || kv->max_pages != d->cfg.max_pages) return CDB_ERR_INVALID_ARG;
    if (state->n_slots < d->cfg.max_seqs) return CDB_ERR_INVALID_ARG;
    const bool two = d->cfg.boundary_stream != 0;
    // the loop steps' stream and workspace (A), the boundary stages' (B)
    hipStream_t sA = stream, sB = stream;
    unsigned char* wsA = static_cast<unsigned char*>(ws);
    unsigned char* wsB = wsA;
    size_t wsA_bytes = ws_bytes, wsB_bytes = ws_bytes;
    if (two) {
        wsA_bytes = wsB_bytes = (ws_bytes / 2) & ~(size_t)255;
        wsB = wsA + wsA_bytes;
        if (hipStreamCreateWithFlags(&sB, hipStreamNonBlocking) != hipSuccess) return CDB_ERR_HIP;
    }
    unsigned char* base = static_cast<unsigned char*>(scratch);
    int32_t* drowsA = reinterpret_cast<int32_t*>(base + SL.rows);  // loop-step rows
    int32_t* drowsB = drowsA + kRowSetInts;                        // coda / prelude / prefill rows
    int32_t* drows2 = drowsB + kRowSetInts;                        // prelude rows after a coda
    int32_t* dids = reinterpret_cast<int32_t*>(base + SL.ids);
    int32_t* dfirst = reinterpret_cast<int32_t*>(base + SL.first);  // first decode input per sequence
    float* dlogits = reinterpret_cast<float*>(base + SL.logits);
    cdb_step_out out;
    out.exit_score = reinterpret_cast<float*>(base + SL.step);
    out.exit_mask = reinterpret_cast<uint8_t*>(base + SL.step + 256 * 4);
    out.cont = reinterpret_cast<int32_t*>(base + SL.step + 256 * 4 + 256);
    out.exited = out.cont + 256;
    out.counts = out.exited + 256;
    out.exit_next = reinterpret_cast<uint8_t*>(out.counts + 2);
    int32_t status = CDB_OK;
    cdb_gate gate;
    gate.threshold = d->cfg.threshold;
    gate.lookahead = d->cfg.lookahead;
    gate.pending = base + SL.pending;
    const bool gated = d->cfg.gated != 0;
    Waits waits;
    if (gated && hipMemsetAsync(gate.pending, 0, d->cfg.max_seqs, sA) != hipSuccess) status = CDB_ERR_HIP;

    // pinned host staging: a ring of row buffers and one of page-table blocks,
    // each slot reused only after the copy that last read it has completed; a
    // third ring receives the gated steps' decisions
    const int RING = 8, PT_RING = 64;
    const size_t slot_ints = kRowSetInts;
    const size_t block_ints = (size_t)planes(d) * d->cfg.max_pages;  // one sequence's page-table block
    const size_t pt_bytes = d->page_table.size() * 4;
    int32_t* pinned = nullptr;
    int32_t* pinned_pt = nullptr;  // the whole table (first upload) and the caller's first inputs
    int32_t* pinned_blk = nullptr;
    uint8_t* pinned_rb = nullptr;
    bool alloc_ok = hipHostMalloc(reinterpret_cast<void**>(&pinned), RING * slot_ints * 4) == hipSuccess;
    alloc_ok = alloc_ok && hipHostMalloc(reinterpret_cast<void**>(&pinned_pt),
                                         std::max(pt_bytes, d->seqs.size() * 4 + 4)) == hipSuccess;
    alloc_ok = alloc_ok && hipHostMalloc(reinterpret_cast<void**>(&pinned_blk), PT_RING * block_ints * 4) == hipSuccess;
    alloc_ok = alloc_ok && hipHostMalloc(reinterpret_cast<void**>(&pinned_rb), RING * 512) == hipSuccess;
    hipEvent_t ev[RING], rb_ev[RING], blk_ev[PT_RING], pt_ev;
    for (int i = 0; i < RING; ++i) {
        hipEventCreateWithFlags(&ev[i], hipEventDisableTiming);
        hipEventCreateWithFlags(&rb_ev[i], hipEventDisableTiming);
    }
    for (int i = 0; i < PT_RING; ++i) hipEventCreateWithFlags(&blk_ev[i], hipEventDisableTiming);
    hipEventCreateWithFlags(&pt_ev, hipEventDisableTiming);
    EventRing evA, evB;          // after loop steps (A); after boundary calls and uploads (B)
    int64_t waitedA = 0, waitedB = 0;  // latest record of the other stream each stream already waits for
    std::vector<int64_t> ready(d->cfg.max_seqs, 0);  // B record after each sequence's latest boundary call
    bool pt_used = false;
    if (!alloc_ok) status = CDB_ERR_HIP;
    // the caller's first inputs (prefilled prompts) to the device
    if (status == CDB_OK && first_tokens) {
        const size_t nb = d->seqs.size() * 4;  // one entry per added sequence
        memcpy(pinned_pt, first_tokens, nb);
        if (nb && hipMemcpyAsync(dfirst, pinned_pt, nb, hipMemcpyHostToDevice, sA) != hipSuccess)
            status = CDB_ERR_HIP;
        hipEventRecord(pt_ev, sA);
        pt_used = true;
    }
    int ring = 0, rb_ring = 0, blk_ring = 0;
    // live: the row count written after the arrays (read by a captured loop step)
    auto stage = [&](const int32_t* slot, const int32_t* seq, const int32_t* pos, const int32_t* c,
                     const int32_t* dep, const int32_t* tok, int32_t n, int32_t* dst, hipStream_t s,
                     int32_t live = -1) -> hipError_t {
        waits.on(ev[ring]);
        int32_t* h = pinned + ring * slot_ints;
        memcpy(h, slot, n * 4);
        memcpy(h + 256, seq, n * 4);
        memcpy(h + 512, pos, n * 4);
        if (c) memcpy(h + 768, c, n * 4);
        if (dep) memcpy(h + 1024, dep, n * 4);
        if (tok) memcpy(h + 1280, tok, n * 4);
        h[kRowCount] = live < 0 ? n : live;
        hipError_t e = hipMemcpyAsync(dst, h, slot_ints * 4, hipMemcpyHostToDevice, s);
        hipEventRecord(ev[ring], s);
        ring = (ring + 1) % RING;
        return e;
    };
    auto stage_ids = [&](const int32_t* ids, int32_t n, int32_t* dst, hipStream_t s) -> hipError_t {
        waits.on(ev[ring]);
        int32_t* h = pinned + ring * slot_ints;
        memcpy(h, ids, (size_t)n * 4);
        hipError_t e = hipMemcpyAsync(dst, h, (size_t)n * 4, hipMemcpyHostToDevice, s);
        hipEventRecord(ev[ring], s);
        ring = (ring + 1) % RING;
        return e;
    };
    // cross-stream ordering (no-ops with one stream)
    auto b_waits_for_a = [&]() {
        if (two && evA.count > waitedB) {
            hipStreamWaitEvent(sB, evA.at(evA.count), 0);
            waitedB = evA.count;
        }
    };
    auto a_waits_for_b = [&](int64_t k) {
        if (two && k > waitedA) {
            hipStreamWaitEvent(sA, evB.at(k), 0);
            waitedA = k;
        }
    };
    // page-table changes to the device: the whole table once, then only the
    // blocks of sequences admitted or released since, each through its own
    // pinned slot; they go on the boundary stream, which runs every new
    // sequence's first call (the loop steps reach a new sequence only after
    // waiting for that call)
    auto upload_table = [&]() -> hipError_t {
        hipError_t e = hipSuccess;
        int32_t* dpt = const_cast<int32_t*>(kv->page_table);
        if (d->table_all_dirty) {
            if (pt_used) waits.on(pt_ev);
            memcpy(pinned_pt, d->page_table.data(), pt_bytes);
            e = hipMemcpyAsync(dpt, pinned_pt, pt_bytes, hipMemcpyHostToDevice, sA);
            hipEventRecord(pt_ev, sA);
            pt_used = true;
            if (two) {
                hipStreamWaitEvent(sB, pt_ev, 0);
            }
            d->stats.pt_uploads++;
            d->stats.pt_upload_bytes += (int64_t)pt_bytes;
            d->table_all_dirty = false;
        } else {
            for (int32_t q : d->dirty_seqs) {
                if (e != hipSuccess) break;
                waits.on(blk_ev[blk_ring]);
                int32_t* hb = pinned_blk + blk_ring * block_ints;
                memcpy(hb, d->page_table.data() + (size_t)q * block_ints, block_ints * 4);
                e = hipMemcpyAsync(dpt + (size_t)q * block_ints, hb, block_ints * 4, hipMemcpyHostToDevice, sB);
                hipEventRecord(blk_ev[blk_ring], sB);
                blk_ring = (blk_ring + 1) % PT_RING;
                d->stats.pt_uploads++;
                d->stats.pt_upload_bytes += (int64_t)block_ints * 4;
            }
        }
        for (int32_t q : d->dirty_seqs) d->seq_dirty[q] = 0;
        d->dirty_seqs.clear();
        return e;
    };
    // gated: the previous loop tick and the ring slot of its decisions
    cdb_driver_tick prev;
    int prev_rb = -1;

    // graph_loop: the loop step captured once at max_batch rows, the live count
    // read from the row set's count entry; replayed on the loop-step stream
    const bool use_graph = d->cfg.graph_loop != 0;
    hipGraphExec_t gexec = nullptr;
    const cdb_rows rows_cap{d->cfg.max_batch, drowsA, drowsA + 256, drowsA + 512, drowsA + 768,
                            gated ? nullptr : drowsA + 1024, drowsA + kRowCount};
    auto loop_call = [&](const cdb_rows* r, hipStream_t st) -> cdb_status {
        return gated ? cdb_loop_step_gated(model, kv, state, r, &gate, &out, wsA, wsA_bytes, st)
                     : cdb_loop_step(model, kv, state, r, &out, wsA, wsA_bytes, st);
    };
    // capture on a private stream (the caller's may be the null stream); the
    // captured launches run only when the graph is launched
    auto capture = [&]() -> cdb_status {
        hipStream_t cs = nullptr;
        if (hipStreamCreateWithFlags(&cs, hipStreamNonBlocking) != hipSuccess) return CDB_ERR_HIP;
        cdb_status cst = CDB_ERR_HIP;
        if (hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal) == hipSuccess) {
            cst = loop_call(&rows_cap, cs);
            hipGraph_t g = nullptr;
            const hipError_t e = hipStreamEndCapture(cs, &g);  // ends the capture whatever the call returned
            if (cst == CDB_OK && (e != hipSuccess || !g)) cst = CDB_ERR_HIP;
            if (cst == CDB_OK && hipGraphInstantiate(&gexec, g, nullptr, nullptr, 0) != hipSuccess) {
                gexec = nullptr;
                cst = CDB_ERR_HIP;
            }
            if (g) hipGraphDestroy(g);  // the executable graph keeps what it needs
        }
        hipStreamDestroy(cs);
        (void)hipGetLastError();
        return cst;
    };

    cdb_driver_tick t;
    std::vector<int32_t> toks(256), npos(256);
    // CDB_DRIVER_PROGRESS set: a line on stderr every 10 s of a long run
    const bool progress = getenv("CDB_DRIVER_PROGRESS") != nullptr;
    double next_report = 10.0;
    const auto t0 = std::chrono::steady_clock::now();
    while (status == CDB_OK) {
        d->now = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
        if (progress && d->now >= next_report) {
            fprintf(stderr, "[driver] %.0f s: %lld tokens, %lld loop steps, %lld prompt tokens, %d active\n", d->now,
                    (long long)d->stats.tokens, (long long)d->stats.loop_steps, (long long)d->stats.prefill_tokens,
                    d->active);
            next_report += 10.0;
        }
        const int32_t r = cdb_driver_next(d, &t);
        if (r == 0) break;
        if (r < 0) continue;  // the next request has not arrived yet
        if (d->table_all_dirty || !d->dirty_seqs.empty()) {
            if (upload_table() != hipSuccess) {
                status = CDB_ERR_HIP;
                break;
            }
        }
        const int32_t n = t.n_rows;
        cdb_status s = CDB_OK;
        if (t.stage == CDB_TICK_PREFILL) {
            // the chunk's prompt ids through the staging ring; the chunk's last
            // greedy id lands in the sequence's first-input entry
            const int32_t q = t.seq[0];
            if (stage_ids(d->seqs[q].prompt.data() + t.pos[0], n, drowsB, sB) != hipSuccess) {
                status = CDB_ERR_HIP;
                break;
            }
            s = cdb_prefill(model, kv, q, t.pos[0], n, drowsB, nullptr, dfirst + q, wsB, wsB_bytes, sB);
            if (s != CDB_OK) {
                status = s;
                break;
            }
            ready[q] = two ? evB.record(sB) : 0;
            if (cdb_driver_complete(d, &t) != 0) {
                status = CDB_ERR_INVALID_ARG;
                break;
            }
            continue;
        }
        // sixth row array: the decode index (coda); the prelude of first inputs
        // gathers its tokens from the first-input entries on the device
        for (int32_t i = 0; i < n; ++i) toks[i] = t.stage == CDB_TICK_CODA ? t.decode_index[i] : 0;
        const bool on_b = t.stage != CDB_TICK_LOOP;
        int32_t* drows = on_b ? drowsB : drowsA;
        if (t.stage == CDB_TICK_CODA) b_waits_for_a();  // its rows exited in loop steps already enqueued
        if (t.stage == CDB_TICK_LOOP) {
            int64_t need = 0;
            for (int32_t i = 0; i < n; ++i) need = std::max(need, ready[t.seq[i]]);
            a_waits_for_b(need);
            if (use_graph && !gexec) {
                // one direct call at capacity with a live count of zero (no rows
                // are touched; every kernel of the capacity's launch shapes has then
                // run once, which sets their first-use attributes outside capture)
                if (stage(t.slot, t.seq, t.pos, t.c, t.depth, toks.data(), n, drowsA, sA, 0) != hipSuccess) {
                    status = CDB_ERR_HIP;
                    break;
                }
                s = loop_call(&rows_cap, sA);
                if (s == CDB_OK) s = capture();
                if (s != CDB_OK) {
                    status = s;
                    break;
                }
            }
        }
        if (stage(t.slot, t.seq, t.pos, t.c, t.depth, toks.data(), n, drows, on_b ? sB : sA) != hipSuccess) {
            status = CDB_ERR_HIP;
            break;
        }
        cdb_rows rows{n, drows, drows + 256, drows + 512, drows + 768, drows + 1024, nullptr};
        if (t.stage == CDB_TICK_PRELUDE_FIRST) {
            if (cdb::launch_gather_ids(n, drows + 256, dfirst, d->cfg.max_seqs, drows + 1280, sB) != hipSuccess) {
                status = CDB_ERR_HIP;
                break;
            }
            s = cdb_boundary_prelude(model, kv, state, &rows, drows + 1280, wsB, wsB_bytes, sB);
            if (s == CDB_OK && two) {
                const int64_t k = evB.record(sB);
                for (int32_t i = 0; i < n; ++i) ready[t.seq[i]] = k;
            }
        } else if (t.stage == CDB_TICK_LOOP) {
            if (gated) rows.depth = nullptr;
            if (use_graph) {
                s = hipGraphLaunch(gexec, sA) == hipSuccess ? CDB_OK : CDB_ERR_HIP;
                if (s == CDB_OK) d->stats.graph_launches++;
            } else {
                s = loop_call(&rows, sA);
            }
            if (gated) {
                if (s == CDB_OK) {
                    // this step's decisions to the host
                    const int rs = rb_ring;
                    rb_ring = (rb_ring + 1) % RING;
                    waits.on(rb_ev[rs]);
                    uint8_t* hb = pinned_rb + rs * 512;
                    if (hipMemcpyAsync(hb, out.exit_mask, n, hipMemcpyDeviceToHost, sA) != hipSuccess ||
                        hipMemcpyAsync(hb + 256, out.exit_next, n, hipMemcpyDeviceToHost, sA) != hipSuccess) {
                        status = CDB_ERR_HIP;
                        break;
                    }
                    hipEventRecord(rb_ev[rs], sA);
                    if (!d->cfg.lookahead) {
                        // the step's own exits are needed before it completes
                        waits.on(rb_ev[rs]);
                        cdb_driver_loop_result(d, &t, hb, hb + 256);
                    } else {
                        // lookahead: the previous step's decisions complete this one
                        if (prev_rb >= 0) {
                            waits.on(rb_ev[prev_rb]);
                            const uint8_t* pb = pinned_rb + prev_rb * 512;
                            if (cdb_driver_loop_result(d, &prev, pb, pb + 256) != 0) s = CDB_ERR_INVALID_ARG;
                        }
                        prev = t;
                        prev_rb = rs;
                    }
                }
            }
            if (s == CDB_OK && two) evA.record(sA);
        } else if (t.stage == CDB_TICK_CODA) {
            s = cdb_boundary_coda(model, kv, state, &rows, dlogits, dids, wsB, wsB_bytes, sB);
            if (s == CDB_OK && tokens_out &&
                cdb::launch_scatter_ids(n, dids, drows + 256, drows + 1280, d->cfg.max_seqs, tokens_stride, tokens_out,
                                        sB) != hipSuccess)
                s = CDB_ERR_HIP;
            if (s == CDB_OK && t.n_continue > 0) {
                // the continuing sequences are the coda batch's first rows: the
                // coda's ids are the prelude's tokens, one position further
                for (int32_t i = 0; i < t.n_continue; ++i) npos[i] = t.pos[i] + 1;
                if (stage(t.slot, t.seq, npos.data(), nullptr, nullptr, nullptr, t.n_continue, drows2, sB) !=
                    hipSuccess) {
                    status = CDB_ERR_HIP;
                    break;
                }
                cdb_rows prow{t.n_continue, drows2, drows2 + 256, drows2 + 512, nullptr, nullptr, nullptr};
                s = cdb_boundary_prelude(model, kv, state, &prow, dids, wsB, wsB_bytes, sB);
            }
            if (s == CDB_OK && two) {
                const int64_t k = evB.record(sB);
                for (int32_t i = 0; i < t.n_continue; ++i) ready[t.seq[i]] = k;
            }
        }
        if (s != CDB_OK) {
            status = s;
            break;
        }
        if (cdb_driver_complete(d, &t) != 0) {
            status = CDB_ERR_INVALID_ARG;
            break;
        }
        if (d->cfg.sync_steps && t.stage == CDB_TICK_LOOP && waits.on(sA) != hipSuccess) {
            status = CDB_ERR_HIP;
            break;
        }
    }
    // gated lookahead: the last loop step's decisions are still due; a device
    // decision the scheduler did not apply is an error, as for every earlier step
    if (status == CDB_OK && gated && d->cfg.lookahead && d->result_pending && prev_rb >= 0) {
        waits.on(rb_ev[prev_rb]);
        const uint8_t* pb = pinned_rb + prev_rb * 512;
        if (cdb_driver_loop_result(d, &prev, pb, pb + 256) != 0) status = CDB_ERR_INVALID_ARG;
    }
    if (waits.on(sA) != hipSuccess && status == CDB_OK) status = CDB_ERR_HIP;
    if (two) {
        if (waits.on(sB) != hipSuccess && status == CDB_OK) status = CDB_ERR_HIP;
        hipStreamDestroy(sB);
    }
    if (gexec) hipGraphExecDestroy(gexec);
    const double secs = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
    d->now = secs;
    d->stats.host_wait_us += (int64_t)std::chrono::duration_cast<std::chrono::microseconds>(waits.total).count();
    if (seconds) *seconds = secs;
    for (int i = 0; i < RING; ++i) {
        hipEventDestroy(ev[i]);
        hipEventDestroy(rb_ev[i]);
    }
    for (int i = 0; i < PT_RING; ++i) hipEventDestroy(blk_ev[i]);
    hipEventDestroy(pt_ev);
    if (pinned) hipHostFree(pinned);
    if (pinned_pt) hipHostFree(pinned_pt);
    if (pinned_blk) hipHostFree(pinned_blk);
    if (pinned_rb) hipHostFree(pinned_rb);
    return status;
}

}  // extern "C"
