/*
 * fairserve.h -- C-ABI of libfairserve.so, the MI355X (gfx950) implementation of
 * the FairServe policy hot path (Ensuring Fair LLM Serving Amid Diverse
 * Applications, arXiv 2411.15997): per-request weighted cost, OIT throttling from
 * sliding-window request counts, and the WSC scheduler step, run over many
 * independent trace replicas at once.
 *
 * Conventions for every entry point:
 *   - Pointers are DEVICE (HBM) pointers unless their name ends in _h (host).
 *   - Every call validates its arguments on the host and returns FS_E_ARG (or
 *     FS_E_WORKSPACE) synchronously; it then enqueues kernels on `stream` and
 *     returns without synchronising.  Data-dependent errors (unsorted times, ids or
 *     token counts out of range, fixed-point overflow) are written by the kernels to
 *     the caller's device status word `err` (int32, zeroed by the call itself);
 *     fs_sync_status() waits for the stream and returns it.  When several errors
 *     occur the largest code is reported.  Outputs are unspecified after an error.
 *   - The caller owns every buffer, including workspace and state.  The library
 *     allocates no device memory and keeps no pointer after the call returns.
 *   - Results are bit-deterministic.
 *
 * Trace layout (structure of arrays, replicas concatenated, record g of replica r
 * lives at rep_off[r] + i with replica-local index i):
 *   ts_us   int64  arrival time (microseconds, >= 0), non-decreasing within a replica;
 *                  equal times keep stream order
 *   user    int32  in [0, n_users);  app int32 in [0, n_apps)
 *   call    int32  stage j of the LLM interaction (0 = its first call)
 *   head    int32  replica-local index of the interaction's first call (itself when call == 0)
 *   prev    int32  replica-local index of call j-1 (-1 when call == 0); same user and head
 *   len_in, len_sys, len_out  int32 input / system / output tokens, each in [0, 2^24)
 *   call, head and prev are either all NULL (every record is a single-call
 *   interaction) or all set.  len_sys may be NULL (= 0).
 *   A trace without requests (rep_off_h[n_replicas] == 0) may leave every per-request
 *   array NULL, here and in the calls below (cost, reasons, bitmap, per-request
 *   outputs); the calls then write only their per-replica and per-user outputs.
 */
#ifndef FAIRSERVE_H
#define FAIRSERVE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum fs_status {
  FS_OK = 0,
  FS_E_ARG = 1,       /* bad argument or shape (synchronous) */
  FS_E_ORDER = 2,     /* ts_us decreases inside a replica */
  FS_E_RANGE = 3,     /* id, token count, coefficient, priority, cost or chain link out of range */
  FS_E_OVERFLOW = 4,  /* a cost, a service counter or a replica's charged total reaches 2^62 */
  FS_E_WORKSPACE = 5, /* workspace or state buffer too small (synchronous) */
  FS_E_STATE = 6,     /* state buffer not initialised for this trace, or wrong version */
  FS_E_HIP = 7        /* a HIP runtime call failed */
} fs_status;

typedef struct fs_trace {
  int32_t n_replicas, n_users, n_apps;
  const int64_t *rep_off_h; /* host   [R+1], rep_off_h[0] = 0, non-decreasing */
  const int64_t *rep_off;   /* device [R+1], same values */
  const int64_t *ts_us;
  const int32_t *user, *app;
  const int32_t *call, *head, *prev;
  const int32_t *len_in, *len_sys, *len_out;
} fs_trace;

/* Service weights (Sec. 4, WSC).  The paper's per-call service is
 *   E_i * (alpha L_I + beta L_S + gamma L_O) / w_aj            (one term of Eq. 2)
 * with alpha, beta, gamma = 1, 2, 1 and w_aj from Eq. 1.  Here the token-class
 * weight divided by w_aj is a Q16 fixed-point coefficient per (app, stage, class),
 * and E_i is a Q8 priority:
 *   cost = floor(E_u * (c_in*L_I + c_sys*L_S + c_out*L_O) / 2^8),   exact, < 2^62.
 * coef:  device [R or 1][n_apps][n_stages][3] int64 {in, sys, out}, each in [0, 2^36);
 *        coef_rep_stride = n_apps*n_stages*3 for a per-replica table, 0 for a shared one.
 * prio:  device [R or 1][n_users] int32 in [0, 2^16), or NULL for E = 1.0 (256).
 * Stage j = min(call, n_stages - 1). */
typedef struct fs_weights {
  int32_t n_stages;
  int64_t coef_rep_stride;
  const int64_t *coef;
  int64_t prio_rep_stride;
  const int32_t *prio;
} fs_weights;

/* OIT limits (Alg. 1 monitoring stream; Sec. 4, OIT).  For request i the counts are
 *   c_user(i) = #{ j <= i : user_j = user_i, ts_j > ts_i - window_us }
 *   c_app(i)  = #{ j <= i : user_j = user_i, app_j = app_i, ts_j > ts_i - window_us }
 * (every arrival is counted, whatever its fate).  The user limit is checked first:
 * exceeded if c_user > t_user, else if c_app > t_app_h[app].  t_user = INT32_MAX
 * disables the user limit.  window_us > 0; limits >= 0; t_app_h is a host array
 * [n_apps], n_apps <= 1024.  app_scope = 1 counts c_app over every user of the app
 * (drop the user_j = user_i term: the app-level rate limit of Sec. 3); 0 is the
 * per-(user, app) count above. */
typedef struct fs_limits {
  int64_t window_us;
  int32_t t_user;
  const int32_t *t_app_h;
  int32_t app_scope;
} fs_limits;

/* Engine model for the execution stream (the paper leaves the LLM engine's
 * admission test unspecified).  Time advances in steps of step_us; each step has
 * cap_tokens of capacity, and a step admits requests while its remaining budget is
 * positive; overshoot is carried as debt into the next step.  The system counts as
 * overloaded while the queued tokens exceed overload_tokens (-1: always).
 * flags: FS_ENGINE_GLOBAL_ONLY runs the scheduler with all of its state in global
 * memory (the path taken when the on-chip capacities overflow); for testing.
 * The policies the paper compares against (Sec. 2 and Sec. 5: request-rate limits and
 * the virtual token counter) run on the same kernels:
 *   FS_ENGINE_FCFS   admit the earliest queued request (first come, first served):
 *                    neither the service counters nor the interaction priority choose;
 *                    counters are still lifted and charged, so the metrics compare;
 *   FS_ENGINE_BLIND  interaction-blind limits: every call, not only an interaction's
 *                    first, is checked against the raw limit reasons (when overloaded),
 *                    and once a call is dropped every later call of its interaction is
 *                    dropped too (status 3), as a client abandons the interaction.
 * FS_ENGINE_FCFS | FS_ENGINE_BLIND with overload_tokens = -1 is the per-user
 * request-rate-limit policy (RPM); the virtual token counter is the default policy with
 * equal coefficients for every app and no limits (t_user = t_app = INT32_MAX); the
 * paper's WSC-only ablation is the default policy with no limits.
 *   FS_ENGINE_LITERAL  the execution stream as Alg. 1 writes it: an admitted call is
 *                    prefilled in its admission step (its first output token), decodes
 *                    one more output token per step and finishes in step
 *                    admit + max(L_O, 1) - 1, when its user is charged its cost (charge at
 *                    finish; counters do not move between a step's admissions).  cap_tokens
 *                    is then the KV-cache capacity in tokens: a call holds L_I + L_S + L_O
 *                    tokens from admission to the end of its finish step, and a step's
 *                    admissions stop at the first chosen call that does not fit (a call
 *                    runs alone when nothing else runs).  Finishes of a step are charged in
 *                    admission order after its admissions; counter_after is the counter
 *                    after the finish charge (-1 while the call runs).  Runs with all
 *                    state in global memory; combines with FCFS and BLIND. */
typedef struct fs_engine {
  int64_t step_us, cap_tokens, overload_tokens;
  uint32_t flags;
} fs_engine;
#define FS_ENGINE_GLOBAL_ONLY 1u
#define FS_ENGINE_FCFS 2u
#define FS_ENGINE_BLIND 4u
#define FS_ENGINE_LITERAL 8u

/* Per-record and per-replica scheduler outputs (device pointers).
 *   status       [N] int8: 0 admitted, 1 throttled by the user limit, 2 by the app limit,
 *                3 dropped because its interaction's first call was throttled (or, with
 *                FS_ENGINE_BLIND, an earlier call of its interaction was dropped),
 *                -1 not yet decided (bounded runs only)
 *   admit_step   [N] int32: step of admission, -1 otherwise
 *   admit_seq    [N] int32 or NULL: global admission order within the replica
 *   counter_after[N] int64 or NULL: the user's counter just after charging this request
 *   counter_on_arrival [N] int64 or NULL: the user's counter after the arrival lift
 *   counter      [R][n_users] int64: service counters when the call returns
 *   steps, decisions, max_gap [R] int64: steps simulated, admissions, and the largest
 *                counter gap max_X u - min_X u sampled after each step's admissions
 *   err          device int32 status word (see the conventions above) */
typedef struct fs_outputs {
  int8_t *status;
  int32_t *admit_step;
  int32_t *admit_seq;
  int64_t *counter_after;
  int64_t *counter_on_arrival;
  int64_t *counter;
  int64_t *steps, *decisions, *max_gap;
  int32_t *err;
} fs_outputs;

/* Per-replica fairness and served-experience metrics (device arrays [R] each).
 *   jain              Jain's index of the charged service over users with >= 1 request
 *   max_gap_tokens    max_gap / 2^16
 *   svc_req_pct       admitted requests / requests (service provided, Sec. 5)
 *   svc_int_pct       interactions with every call admitted / interactions
 *   served_users_pct  users with >= 1 fully served interaction / users with requests
 *   delayed_users_pct users with an admitted request whose admit_step exceeds its
 *                     arrival step by more than delay_steps / users with requests
 *   throttled         requests with status 1..3
 *   aborted_midway    interactions with both admitted and dropped calls
 *   wasted_tokens     tokens of admitted calls of such interactions */
typedef struct fs_metrics {
  double *jain, *max_gap_tokens, *svc_req_pct, *svc_int_pct, *served_users_pct,
      *delayed_users_pct;
  int64_t *throttled, *aborted_midway, *wasted_tokens;
} fs_metrics;

/* Eq. 2, one term per LLM call (and the charge of Alg. 1's execution stream):
 * writes cost[N] (int64) as defined for fs_weights.  Errors: FS_E_RANGE for a
 * token count, coefficient or priority out of range, FS_E_OVERFLOW for cost >= 2^62. */
fs_status fs_cost(const fs_trace *t, const fs_weights *w, int64_t *cost, int32_t *err,
                  hipStream_t stream);

/* Bytes of device workspace fs_throttle needs for this trace (0 for a trace it
 * rejects, see the key-space limit below). */
size_t fs_throttle_workspace(const fs_trace *t);

/* OIT (Alg. 1 monitoring stream, limit checks; Sec. 4, OIT).  For each record the
 * raw reason is 0 (within limits), 1 (user limit exceeded) or 2 (app limit exceeded).
 * flags & FS_THROTTLE_RAW: bitmap bit i = raw reason != 0, reason[i] = raw reason.
 * Otherwise (gated): a first call (head == its own index) is throttled iff
 * overloaded[i] (NULL = always) and its raw reason is nonzero; a later call is never
 * checked and is dropped iff its interaction's first call was throttled (code 3);
 * bitmap bit i = throttled.  The call reads ts_us, user, app and (gated) head, with
 * 0 <= head <= own index (else FS_E_RANGE); call and prev are not read.
 * bitmap: [ceil(N/32)] uint32, bit i%32 of word i/32 (global record index).
 * reason [N] uint8, cnt_user [N], cnt_app [N] int32 (the window counts) may be NULL.
 * ws: device workspace of at least fs_throttle_workspace(t) bytes, 256-byte aligned.
 * Key-space limit: with b(x) the bits of x - 1 (at least 1), the trace must have
 * b(n_replicas * n_users) + b(n_apps) <= 32 and that sum + b(N) + 1 <= 64 (N records);
 * otherwise FS_E_ARG (also from fs_run_trace, before anything is enqueued). */
#define FS_THROTTLE_RAW 1u
fs_status fs_throttle(const fs_trace *t, const fs_limits *lim, const uint8_t *overloaded,
                      uint32_t flags, uint32_t *bitmap, uint8_t *reason, int32_t *cnt_user,
                      int32_t *cnt_app, void *ws, size_t ws_bytes, int32_t *err,
                      hipStream_t stream);

/* Scheduler state (Alg. 1 state: counters u_i, waiting queue Q, throttling state),
 * resumable between calls.  fs_state_bytes gives its size; fs_state_init resets it
 * for trace t (all counters 0, nothing processed). */
size_t fs_state_bytes(const fs_trace *t);
fs_status fs_state_init(void *state, size_t state_bytes, const fs_trace *t, hipStream_t stream);

/* WSC scheduler steps (Alg. 1, both streams, under the fs_engine step model) for
 * every replica, starting from `state` and advancing it by n_steps steps (n_steps < 0:
 * until every request has arrived and the queue is empty).  Per step s: requests with
 * floor(ts/step_us) <= s arrive in stream order (counter lift when the user has nothing
 * queued, then OIT gating with exceed_reason, then enqueue); then, while the budget is
 * positive, the user with the least counter among users with a ready later call of an
 * incomplete interaction (else among all queued users) is served, ties to the lowest
 * user id, its earliest eligible request is admitted and its cost charged at once.
 * cost: [N] from fs_cost; exceed_reason: [N] raw reasons from fs_throttle (NULL = none).
 * Repeated calls with the same `out` must see the same trace, cost and reasons.
 * A run in k calls gives the same outputs as one call. */
fs_status fs_schedule_step(void *state, const fs_trace *t, const int64_t *cost,
                           const uint8_t *exceed_reason, const fs_engine *eng, fs_outputs *out,
                           int64_t n_steps, hipStream_t stream);

/* The whole hot path of Alg. 1 over a trace: the per-call service of Eq. 2 (fs_cost),
 * the OIT window tests of the monitoring stream (fs_throttle, raw), then the
 * monitoring and execution streams step by step (fs_state_init, fs_schedule_step until
 * drained), using caller workspace of at least fs_run_trace_workspace(t) bytes
 * (256-byte aligned; 0 is returned for a trace outside fs_throttle's key-space limit).
 * The cost and raw reasons stay in the workspace: the cost at offset 0 (int64 [N]),
 * the reasons (uint8 [N]) at the next 256-byte boundary. */
size_t fs_run_trace_workspace(const fs_trace *t);
fs_status fs_run_trace(const fs_trace *t, const fs_weights *w, const fs_limits *lim,
                       const fs_engine *eng, fs_outputs *out, void *ws, size_t ws_bytes,
                       hipStream_t stream);

/* Per-replica metrics from a finished run (Sec. 5 definitions plus Jain's index).
 * ws: device workspace of at least fs_metrics_workspace(t) bytes (256-byte aligned).
 * out->err receives data-dependent errors: FS_E_RANGE for an id or interaction link out
 * of range or an admitted request whose cost is outside [0, 2^62) (not counted), and
 * FS_E_OVERFLOW when a replica's total charged service (the sum of its admitted costs)
 * reaches 2^62; below that every sum of Jain's index is exact. */
size_t fs_metrics_workspace(const fs_trace *t);
fs_status fs_fairness_metrics(const fs_trace *t, const int64_t *cost, const fs_outputs *out,
                              const fs_engine *eng, int32_t delay_steps, fs_metrics *m, void *ws,
                              size_t ws_bytes, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): fs_fairness_metrics with the
 * library's own workspace, a fixed device array of fs_metrics_noalloc_limit() bytes
 * (32 MiB) per GPU, held until the process ends.  Same arguments and results as
 * fs_fairness_metrics without ws/ws_bytes; FS_E_WORKSPACE (synchronous) when
 * fs_metrics_workspace(t) exceeds the limit.  The call allocates nothing.  Every call on
 * one GPU uses that GPU's array (each call clears it first): calls that overlap on one
 * GPU (other streams, other host threads) race and must be serialised by the caller. */
size_t fs_metrics_noalloc_limit(void);
fs_status fs_fairness_metrics_noalloc(const fs_trace *t, const int64_t *cost,
                                      const fs_outputs *out, const fs_engine *eng,
                                      int32_t delay_steps, fs_metrics *m, hipStream_t stream);

/* Eq. 1 host helper: w_aj = 1*e_in + 2*e_sys + 1*e_out (expected tokens of app a at
 * stage j) and coef_h[a][j][x] = round-half-even(double(2^16 * K * class_weight_x) / w_aj)
 * computed in IEEE double.  Host arrays [A][J]; coef_h [A][J][3].  Synchronous. */
fs_status fs_coef_from_expectations(int32_t n_apps, int32_t n_stages, const double *e_in_h,
                                    const double *e_sys_h, const double *e_out_h, int64_t K,
                                    int64_t *coef_h);

/* Offline derivation of the weights and app limits from a historical trace (Eq. 1 with
 * each expectation taken as the history's sample mean; Sec. 4, OIT: the app limit scaled
 * by the app's mean number of LLM calls per interaction).  Over every record of `hist`
 * (all replicas pooled), with stage j = min(call, n_stages - 1):
 *   stats[a][j][5] int64 = {records, first calls (call == 0), sum L_I, sum L_S, sum L_O}
 *   coef [a][j][3] int64 = round-half-even(2^16 K x / w_aj) for x = 1, 2, 1 (input,
 *          system, output), w_aj = D / n the group's mean of L_I + 2 L_S + L_O,
 *          evaluated exactly as round-half-even(2^16 K x n / D).  A group with no
 *          records or no tokens takes its app's stages pooled, then the whole history,
 *          and w_aj = K when there are no tokens at all.  The table plugs into
 *          fs_weights (coef_rep_stride 0, n_stages as here).
 *   t_app[a] int32 = ceil(base_limit * records_a / first calls_a) (base_limit when app a
 *          has no first call), usable as fs_limits.t_app_h after a copy to the host.
 * Device arrays; coef and t_app may be NULL, stats is required (it is cleared by the
 * call).  ws: device workspace of at least fs_history_workspace(hist, n_stages) bytes,
 * 256-byte aligned (may be NULL when that size is 0), else FS_E_WORKSPACE.  K in [1, 2^20], base_limit >= 0, n_stages in [1, 4096],
 * fewer than 2^36 records, else FS_E_ARG.  Device errors (err): FS_E_RANGE for an app,
 * call or token count out of range (the record is skipped), a coefficient >= 2^36 or a
 * limit above INT32_MAX.  The trace's ts_us and user are not read. */
size_t fs_history_workspace(const fs_trace *hist, int32_t n_stages);
fs_status fs_weights_from_history(const fs_trace *hist, int32_t n_stages, int64_t K,
                                  int32_t base_limit, int64_t *stats, int64_t *coef,
                                  int32_t *t_app, void *ws, size_t ws_bytes, int32_t *err,
                                  hipStream_t stream);

/* Workload analysis of Sec. 3, per replica: the users' requests and tokens per minute
 * overall and within each application (Fig. 2), the token lengths per application
 * (Figs. 3 and 5), the LLM calls per interaction per application (Fig. 4) and the
 * graph-size table (Table 2).  minute_us > 0 is a minute's length; a replica's horizon
 * is M = floor(max ts / minute_us) + 1 minutes (0 without requests), a user's RPM is
 * requests / M and TPM tokens / M (tokens = L_I + L_S + L_O).  Bins:
 *   rate bin of x / M     0 if x == 0, else 64 + floor(log2(x / M)), exact (1..127)
 *   length bin of L       0 if L == 0, else 1 + floor(log2 L)
 *   size bin of s calls   min(s, 64) - 1 (an interaction's size is the number of the
 *                         replica's requests whose first call is its first call)
 *   graph bins            1, 2-10, 11-20, 21-30, 31-40, 41-50, more than 50 calls
 * Device outputs (int64, each written in full):
 *   minutes [R]; user_req, user_tok [R][U]; user_app_req, user_app_tok [R][U][A] (may be
 *   NULL); rate_hist [R][A + 1][2][FS_RATE_BINS]: users with a request by the rate bin of
 *   their RPM ([0]) and TPM ([1]), within app a (row a) or overall (row A);
 *   len_hist [R][A][3][FS_LEN_BINS]: requests by the length bin of L_I, L_S, L_O;
 *   len_sum [R][A][3]; size_hist [R][A][FS_SIZE_BINS]: interactions (by the app of their
 *   first call) by size bin; graph [R][FS_GRAPH_BINS][5]: per graph bin its
 *   interactions, requests, and the sums of L_I, L_O, L_S over those requests.
 * ws: at least fs_workload_workspace(t) bytes, 256-byte aligned.  Device errors (err):
 * FS_E_RANGE for an id, length, interaction link or negative arrival time (the request
 * is not counted). */
#define FS_RATE_BINS 128
#define FS_LEN_BINS 32
#define FS_SIZE_BINS 64
#define FS_GRAPH_BINS 7
typedef struct fs_wstats {
  int64_t *minutes, *user_req, *user_tok, *user_app_req, *user_app_tok;
  int64_t *rate_hist, *len_hist, *len_sum, *size_hist, *graph;
} fs_wstats;
size_t fs_workload_workspace(const fs_trace *t);
fs_status fs_workload_stats(const fs_trace *t, int64_t minute_us, const fs_wstats *out, void *ws,
                            size_t ws_bytes, int32_t *err, hipStream_t stream);

/* Waits for `stream` and returns the device status word `err`. */
fs_status fs_sync_status(hipStream_t stream, const int32_t *err);

const char *fs_status_string(fs_status s);

#ifdef __cplusplus
}
#endif
#endif
