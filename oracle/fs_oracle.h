/*
 * CPU oracle for the FairServe policy hot path.  TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, obviously correct host code that states what the policy
 * computes, written from the paper (Alg. 1, Eq. 1, Eq. 2 and the OIT/WSC
 * prose of Sec. 4).  It shares no code with the HIP library: only the tests,
 * the smoke check and the CPU-baseline leg of the benchmark may load it.
 *
 * All pointers are host pointers.  Functions return an fso_code; on failure
 * the outputs are unspecified.  When several problems are present the largest
 * code is returned (validation looks at every record).
 */
#ifndef FS_ORACLE_H
#define FS_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum fso_code { FSO_OK = 0, FSO_E_ARG = 1, FSO_E_ORDER = 2, FSO_E_RANGE = 3, FSO_E_OVERFLOW = 4 };

typedef struct fso_trace {
  int32_t n_replicas, n_users, n_apps;
  const int64_t *rep_off;            /* [R+1] record offsets */
  const int64_t *ts_us;              /* arrival time, non-decreasing per replica */
  const int32_t *user, *app;         /* [0,U), [0,A) */
  const int32_t *call, *head, *prev; /* all NULL => every record is a first call */
  const int32_t *len_in, *len_sys, *len_out; /* len_sys may be NULL (=0) */
} fso_trace;

/* Eq. 1 and the fixed-point coefficients: w_aj = a*E[in] + b*E[sys] + g*E[out]
 * with (a,b,g) = (1,2,1); coef[a][j][x] = round_half_even(2^16 * K * x_weight / w_aj). */
int fso_coef_from_expectations(int32_t n_apps, int32_t n_stages, const double *e_in,
                               const double *e_sys, const double *e_out, int64_t K,
                               int64_t *coef /* [A][J][3] */);

/* Offline derivation from a historical trace (Eq. 1 with the expectations taken as
 * the history's sample means; the OIT app limit scaled by the app's mean number of
 * LLM calls per interaction).  Over all replicas, with stage j = min(call, J - 1):
 *   stats[a][j] = {records, first calls, sum L_I, sum L_S, sum L_O}
 *   coef[a][j][x] = round_half_even(2^16 K x_weight / w_aj), w_aj = D / n, computed
 *                   exactly as round_half_even(2^16 K x_weight n / D) with
 *                   n = records, D = sum(1 L_I + 2 L_S + 1 L_O) of the group;
 *                   a group with n = 0 or D = 0 takes its app's pooled (n, D) over all
 *                   stages, then the whole history's, and w_aj = K when all are empty;
 *   t_app[a]     = ceil(base_limit * records_a / first_calls_a), base_limit when the
 *                   app has no first call.
 * K in [1, 2^20], base_limit >= 0, fewer than 2^36 records.  coef and t_app may be
 * NULL.  FSO_E_RANGE for an id or length out of range, a coefficient >= 2^36 or a
 * limit above INT32_MAX. */
int fso_weights_from_history(const fso_trace *t, int32_t n_stages, int64_t K, int32_t base_limit,
                             int64_t *stats /* [A][J][5] */, int64_t *coef /* [A][J][3] */,
                             int32_t *t_app /* [A] */);

/* Eq. 2, one LLM call: cost = floor(E_u * (c_in*L_I + c_sys*L_S + c_out*L_O) / 2^8). */
int fso_cost(const fso_trace *t, int32_t n_stages, int64_t coef_rep_stride, const int64_t *coef,
             int64_t prio_rep_stride, const int32_t *prio, int64_t *cost);

/* OIT window counts and limit test (Alg. 1 monitoring stream).  reason[i]:
 * raw mode: 0 within limits, 1 user limit exceeded, 2 app limit exceeded;
 * gated mode: 0 not blocked, 1/2 head blocked by that limit, 3 inherited.
 * bitmap bit i = (reason[i] != 0).  cnt_* may be NULL. */
int fso_throttle(const fso_trace *t, int64_t window_us, int32_t t_user, const int32_t *t_app,
                 const uint8_t *overloaded /* NULL => always */, int32_t raw, uint8_t *reason,
                 uint32_t *bitmap, int32_t *cnt_user, int32_t *cnt_app);
/* The same with the application limit counted per application over all users
 * (app_scope = 1: the app-level rate limit the paper discusses) instead of per
 * (user, application) (app_scope = 0, fso_throttle). */
int fso_throttle_scoped(const fso_trace *t, int64_t window_us, int32_t t_user,
                        const int32_t *t_app, int32_t app_scope, const uint8_t *overloaded,
                        int32_t raw, uint8_t *reason, uint32_t *bitmap, int32_t *cnt_user,
                        int32_t *cnt_app);

/* flags: FSO_FCFS serves queued requests first come, first served (no service counter
 * or interaction priority in the choice; counters are still charged); FSO_BLIND checks
 * every call against the limits (not only first calls) and drops the rest of an
 * interaction once one of its calls is dropped.  FSO_FCFS | FSO_BLIND with
 * overload_tokens = -1 is the request-rate-limit (RPM) policy the paper compares with. */
/* FSO_LITERAL runs the execution stream as Alg. 1 writes it: an admitted call is
 * prefilled in its admission step (its first output token), decodes one more output
 * token per step and finishes in step admit + max(L_O, 1) - 1, when its user is charged
 * the call's cost (Eq. 2); cap_tokens is then the KV-cache capacity: a call holds
 * L_I + L_S + L_O tokens from admission to the end of its finish step, and the
 * admissions of a step stop at the first chosen call that does not fit (a call runs
 * alone when nothing else does).  Counters do not move between admissions. */
typedef struct fso_engine { int64_t step_us, cap_tokens, overload_tokens; uint32_t flags; } fso_engine;
enum { FSO_FCFS = 1, FSO_BLIND = 2, FSO_LITERAL = 4 };

typedef struct fso_outputs {
  int8_t *status;             /* [N] 0 admitted, 1/2/3 blocked, -1 not processed (bounded run) */
  int32_t *admit_step;        /* [N] or NULL, -1 if not admitted */
  int32_t *admit_seq;         /* [N] or NULL */
  int64_t *counter_after;     /* [N] or NULL */
  int64_t *counter_on_arrival;/* [N] or NULL, -1 if not processed */
  int64_t *counter;           /* [R][U] or NULL */
  int64_t *steps, *decisions, *max_gap; /* [R] or NULL */
} fso_outputs;

/* Per-replica step simulation (Alg. 1 execution + monitoring streams under the
 * token-budget step model).  exceed_reason: raw throttle reasons (NULL = none).
 * max_steps < 0: run until drained.  check != 0 verifies the paper's invariants
 * on every decision and returns FSO_E_ARG (with a message on stderr) if one fails. */
int fso_simulate(const fso_trace *t, const int64_t *cost, const uint8_t *exceed_reason,
                 const fso_engine *e, int64_t max_steps, int32_t n_threads, int32_t check,
                 fso_outputs *out);

typedef struct fso_metrics {
  double *jain, *max_gap_tokens, *svc_req_pct, *svc_int_pct, *served_users_pct, *delayed_users_pct;
  int64_t *throttled, *aborted_midway, *wasted_tokens;
} fso_metrics;

int fso_fairness_metrics(const fso_trace *t, const int64_t *cost, const int8_t *status,
                         const int32_t *admit_step, const int64_t *max_gap, int64_t step_us,
                         int32_t delay_steps, fso_metrics *m);

/* Workload analysis of Sec. 3 (the users' request and token rates of Fig. 2 overall and
 * per application, the token lengths per application of Figs. 3 and 5, the LLM calls per
 * interaction of Fig. 4, and the graph-size table, Table 2), per replica.  minute_us is
 * the length of a minute; the replica's horizon is M = floor(max ts / minute_us) + 1
 * minutes (0 without requests), a user's RPM = requests / M and TPM = tokens / M
 * (tokens = L_I + L_S + L_O), overall and within each application.
 * Bins:
 *   rate bin of x / M:   0 if x == 0, else 64 + floor(log2(x / M))  (exact, in [1, 127])
 *   length bin of L:     0 if L == 0, else 1 + floor(log2 L)
 *   size bin of s calls: min(s, 64) - 1
 *   graph bins (Table 2 rows): 1, 2-10, 11-20, 21-30, 31-40, 41-50, more than 50 calls
 * An interaction's size is the number of the replica's records whose first call
 * (head) is its first call.
 * Outputs (host arrays, every one written in full):
 *   minutes     [R]
 *   user_req, user_tok            [R][U]
 *   user_app_req, user_app_tok    [R][U][A]  (may be NULL)
 *   rate_hist   [R][A + 1][2][FSO_RATE_BINS]  users with a request (overall: row A; in app
 *               a: row a) by the rate bin of their RPM ([0]) and TPM ([1])
 *   len_hist    [R][A][3][FSO_LEN_BINS]  requests by the length bin of L_I, L_S, L_O
 *   len_sum     [R][A][3]                sums of L_I, L_S, L_O
 *   size_hist   [R][A][FSO_SIZE_BINS]    interactions (by their first call's app) by size bin
 *   graph       [R][FSO_GRAPH_BINS][5]   per graph bin: interactions, requests, sum L_I,
 *                                        sum L_O, sum L_S over those requests
 * FSO_E_ARG for minute_us <= 0; FSO_E_RANGE for an id, a length, a link or an arrival
 * time (negative) out of range. */
enum { FSO_RATE_BINS = 128, FSO_LEN_BINS = 32, FSO_SIZE_BINS = 64, FSO_GRAPH_BINS = 7 };
typedef struct fso_wstats {
  int64_t *minutes, *user_req, *user_tok, *user_app_req, *user_app_tok;
  int64_t *rate_hist, *len_hist, *len_sum, *size_hist, *graph;
} fso_wstats;
int fso_workload_stats(const fso_trace *t, int64_t minute_us, fso_wstats *out);

#ifdef __cplusplus
}
#endif
#endif
