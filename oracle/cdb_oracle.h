/*
 * cdb_oracle.h -- interface of the CPU oracle (test infrastructure only; the
 * product path never includes or links this).  All floating point is fp64;
 * weights are bf16 bit patterns in plain row-major [out][in] matrices.
 */
#ifndef CDB_ORACLE_H
#define CDB_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORC_OK = 0, ORC_ERR_ARG = 1, ORC_ERR_UNMAPPED = 2 };

typedef struct {
    int32_t d, n_heads, head_dim, d_ff, vocab;
    int32_t n_prelude, n_core, n_coda, r_max;
    int32_t injection;    /* 0: core input is h; 1: core input is W_a [h; e] */
    int32_t exit_kind;    /* 0: sigmoid(w_exit . RMSNorm(h)); 1: ||h_new - h_old||_2 */
    int32_t bf16_storage; /* 1: round the values the model stores in bf16 */
    double rms_eps, rope_base;
    int32_t kv_layout;    /* core KV layout: ORC_KV_FULL, ORC_KV_SHARED, ORC_KV_FIRST_THEN_SHARED */
} orc_desc;

/* Core KV layouts (Section 4.2; App. C.1, Table 1). */
enum { ORC_KV_FULL = 0, ORC_KV_SHARED = 1, ORC_KV_FIRST_THEN_SHARED = 2 };

typedef struct {
    const uint16_t* embed;        /* [vocab][d] */
    const uint16_t* lm_head;      /* [vocab][d] */
    const uint16_t* w_exit;       /* [d] */
    const uint16_t* adapter;      /* [d][2d], injection only */
    const uint16_t* const* layer; /* layer[7*L + j], j = q,k,v,o,gate,up,down; layers are
                                     prelude, then core, then coda */
} orc_weights;

typedef struct {
    double* pre_pool;  /* pages of [n_prelude][2][H][16][hd] */
    double* core_pool; /* pages of [n_core][2][H][16][hd] */
    double* coda_pool; /* pages of [n_coda][2][H][16][hd] */
    int32_t pre_pages, core_pages, coda_pages;
    const int32_t* page_table; /* [max_seqs][r_max + 2][max_pages] */
    int32_t max_seqs, max_pages, r_max;
} orc_paged;

int orc_ref_sequence(const orc_desc* m, const orc_weights* w, int32_t T, int32_t* tokens, int32_t n_given,
                     int32_t n_prefill, const int32_t* depth, double* logits_out, double* h_out, double* scores_out,
                     double* core_kv_out);
/* As orc_ref_sequence, with each decode token's depth decided by the
 * threshold rule on its own exit scores (lookahead: the decision after loop r
 * ends the token after loop r + 1); prefill tokens run r_max loops.
 * depth_out [T] receives every token's depth. */
int orc_ref_sequence_gated(const orc_desc* m, const orc_weights* w, int32_t T, int32_t* tokens, int32_t n_given,
                           int32_t n_prefill, double threshold, int32_t lookahead, int32_t* depth_out,
                           double* logits_out, double* h_out, double* scores_out);
int orc_gate_decide(const orc_desc* m, int32_t n, const int32_t* c, const double* score, double threshold,
                    int32_t lookahead, uint8_t* pending, uint8_t* exit_mask, uint8_t* exit_next);
int orc_brute_force(const orc_desc* m, const orc_weights* w, int32_t T, const int32_t* tokens, int32_t n_prefill,
                    const int32_t* depth, double* logits_out, double* h_out, double* scores_out);
int orc_prelude(const orc_desc* m, const orc_weights* w, const orc_paged* p, double* state_h, double* state_e,
                int32_t n_slots, int32_t n, const int32_t* slot, const int32_t* seq, const int32_t* pos,
                const int32_t* tokens);
int orc_loop_step(const orc_desc* m, const orc_weights* w, const orc_paged* p, double* state_h,
                  const double* state_e, int32_t n_slots, int32_t n, const int32_t* slot, const int32_t* seq,
                  const int32_t* pos, const int32_t* c, const int32_t* depth, double* score, uint8_t* exit_mask,
                  int32_t* cont, int32_t* exited, int32_t* counts);
int orc_coda(const orc_desc* m, const orc_weights* w, const orc_paged* p, const double* state_h,
             int32_t n_slots, int32_t n, const int32_t* slot, const int32_t* seq, const int32_t* pos,
             double* logits, int32_t* next_ids);
/* Threads of the OpenMP loops over rows (timing only); returns the count in use. */
int orc_set_threads(int n);

int orc_exit_compact(int32_t n, const int32_t* c, const int32_t* depth, int32_t r_max, uint8_t* exit_mask,
                     int32_t* cont, int32_t* exited, int32_t* counts);

void orc_rmsnorm(const double* x, int32_t n, double eps, double* y);
void orc_rope(double* v, int32_t n_heads, int32_t hd, int32_t pos, double base);
void orc_attend(const double* q, const double* k, const double* v, int32_t n, int32_t hd, double* out);
double orc_silu(double x);
double orc_to_bf16(double x);

#ifdef __cplusplus
}
#endif
#endif
