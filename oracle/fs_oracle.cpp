// CPU oracle for the FairServe policy hot path.  TEST INFRASTRUCTURE ONLY:
// only tests/, the smoke check and the benchmark's CPU-baseline leg load it.
//
// Written for a reader holding the paper.  Every function follows one passage:
//   fso_coef_from_expectations  Eq. 1 and the token-class weights (Sec. 4, WSC)
//   fso_weights_from_history    Eq. 1 from a historical trace's sample means, and the app
//                               limit scaled by the mean calls per interaction (Sec. 4)
//   fso_cost                    Eq. 2, one term of the sum (one LLM call), Alg. 1 charge
//   fso_throttle                Alg. 1 monitoring stream: counting, OIT limit checks, the
//                               interaction exemption (Sec. 4, OIT)
//   fso_simulate                Alg. 1 both streams under a token-budget step engine
//   fso_fairness_metrics        Sec. 5 served-experience definitions plus Jain's index
// The data structures are the paper's own: a dictionary from user and from
// (user, app) to the list of arrival times (OIT), a per-user FIFO queue and the
// service counters (WSC), with an ordered set standing in for "argmin".
// Nothing here is blocked, fused or reordered for speed.
#include "fs_oracle.h"

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdio>
#include <deque>
#include <set>
#include <thread>
#include <unordered_map>
#include <utility>
#include <vector>

namespace {

constexpr int64_t kLenLimit = int64_t(1) << 24;   // token counts are in [0, 2^24)
constexpr int64_t kCoefLimit = int64_t(1) << 36;  // Q16 coefficients are in [0, 2^36)
constexpr int64_t kPrioLimit = int64_t(1) << 16;  // Q8 user priority in [0, 2^16)
constexpr int64_t kValueLimit = int64_t(1) << 62; // costs and counters stay below 2^62
constexpr int64_t kCapLimit = int64_t(1) << 40;   // engine token capacity per step

struct Replica {
  int64_t base, n;
};

Replica replica(const fso_trace *t, int32_t r) {
  return Replica{t->rep_off[r], t->rep_off[r + 1] - t->rep_off[r]};
}

int worse(int a, int b) { return a > b ? a : b; }

// Structural checks.  Each entry point checks the fields it reads.
// kIds: app ids and stages; kApps: app ids only; kUsers: user ids; kChain: the whole
// interaction chain (head and previous call); kHeads: only each request's link to its
// interaction's first call (itself for a first call), 0 <= head <= own index.
enum Need : unsigned {
  kIds = 1, kOrder = 2, kChain = 4, kLengths = 8, kUsers = 16, kHeads = 32, kApps = 64
};

int validate_trace(const fso_trace *t, unsigned need) {
  if (!t || t->n_replicas < 1 || t->n_users < 1 || t->n_apps < 1 || !t->rep_off || !t->ts_us ||
      !t->user || !t->app)
    return FSO_E_ARG;
  bool any = t->call || t->head || t->prev;
  bool all = t->call && t->head && t->prev;
  if (any && !all) return FSO_E_ARG;
  if ((need & kLengths) && (!t->len_in || !t->len_out)) return FSO_E_ARG;
  if (t->rep_off[0] != 0) return FSO_E_ARG;
  for (int32_t r = 0; r < t->n_replicas; ++r)
    if (t->rep_off[r + 1] < t->rep_off[r] || t->rep_off[r + 1] - t->rep_off[r] > INT32_MAX)
      return FSO_E_ARG;
  int code = FSO_OK;
  for (int32_t r = 0; r < t->n_replicas; ++r) {
    Replica rp = replica(t, r);
    for (int64_t i = 0; i < rp.n; ++i) {
      int64_t g = rp.base + i;
      if (need & kOrder) {
        if (t->ts_us[g] < 0) code = worse(code, FSO_E_RANGE);
        if (i > 0 && t->ts_us[g] < t->ts_us[g - 1]) code = worse(code, FSO_E_ORDER);
      }
      if ((need & kUsers) && (t->user[g] < 0 || t->user[g] >= t->n_users))
        code = worse(code, FSO_E_RANGE);
      if ((need & kApps) && (t->app[g] < 0 || t->app[g] >= t->n_apps))
        code = worse(code, FSO_E_RANGE);
      if (need & kIds) {
        if (t->app[g] < 0 || t->app[g] >= t->n_apps) code = worse(code, FSO_E_RANGE);
        if (all && t->call[g] < 0) code = worse(code, FSO_E_RANGE);
      }
      if ((need & kHeads) && all && (t->head[g] < 0 || t->head[g] > i))
        code = worse(code, FSO_E_RANGE);
      if ((need & kChain) && all) {
        int32_t c = t->call[g], h = t->head[g], p = t->prev[g];
        bool ok;
        if (c == 0) {
          ok = (h == i) && (p == -1);
        } else {
          ok = c > 0 && p >= 0 && p < i;
          if (ok) {
            int64_t gp = rp.base + p;
            ok = t->call[gp] == c - 1 && t->user[gp] == t->user[g] && t->head[gp] == h;
          }
        }
        if (!ok) code = worse(code, FSO_E_RANGE);
      }
      if (need & kLengths) {
        int64_t li = t->len_in[g], lo = t->len_out[g], ls = t->len_sys ? t->len_sys[g] : 0;
        if (li < 0 || li >= kLenLimit || lo < 0 || lo >= kLenLimit || ls < 0 || ls >= kLenLimit)
          code = worse(code, FSO_E_RANGE);
      }
    }
  }
  return code;
}

bool is_first_call(const fso_trace *t, int64_t g) { return !t->call || t->call[g] == 0; }

int64_t tokens(const fso_trace *t, int64_t g) {
  if (!t->len_in) return 0;
  return int64_t(t->len_in[g]) + (t->len_sys ? t->len_sys[g] : 0) + t->len_out[g];
}

// Runs fn(r) for every replica on n_threads threads (replicas are independent).
template <class Fn>
void for_each_replica(int32_t R, int32_t n_threads, Fn fn) {
  if (n_threads <= 1 || R <= 1) {
    for (int32_t r = 0; r < R; ++r) fn(r);
    return;
  }
  std::atomic<int32_t> next{0};
  std::vector<std::thread> pool;
  int32_t nt = std::min(n_threads, R);
  for (int32_t w = 0; w < nt; ++w)
    pool.emplace_back([&] {
      for (int32_t r = next.fetch_add(1); r < R; r = next.fetch_add(1)) fn(r);
    });
  for (auto &th : pool) th.join();
}

// ---------------------------------------------------------------------------
// Alg. 1, both streams, for one replica.
// ---------------------------------------------------------------------------
struct Simulation {
  const fso_trace *t;
  Replica rp;
  int32_t rep;
  const int64_t *cost;
  const uint8_t *reason;
  fso_engine e;
  int64_t max_steps;
  bool check;
  fso_outputs *out;

  int fail(const char *what, int64_t i) {
    std::fprintf(stderr, "fs_oracle: invariant violated in replica %d at record %lld: %s\n", rep,
                 (long long)i, what);
    return FSO_E_ARG;
  }

  int run() {
    const int32_t U = t->n_users;
    const int64_t n = rp.n, base = rp.base;
    auto G = [&](int64_t i) { return base + i; };

    // WSC service counters u_i, initialised to 0 (Alg. 1 state).
    std::vector<int64_t> u(U, 0);
    // Waiting queue Q: a dictionary from user to that user's queued requests,
    // kept in arrival (stream) order.
    std::vector<std::set<int64_t>> queued(U);
    // Queued later calls of an interaction whose previous call has been served:
    // the "incomplete interactions" the execution stream serves first.
    std::vector<std::set<int64_t>> ready(U);
    // X = users with a queued request, T0 = users with a ready later call,
    // both ordered by (counter, user id) so that begin() is the argmin.
    std::set<std::pair<int64_t, int32_t>> X, T0;
    // Every queued request, by arrival (the first-come, first-served order).
    std::set<int64_t> arrival_order;
    const bool fcfs = (e.flags & FSO_FCFS) != 0, blind = (e.flags & FSO_BLIND) != 0;
    // Literal engine (Alg. 1 execution stream as written): the batch B of running calls
    // in admission order with the step of their last output token; each holds its
    // L_I + L_S + L_O tokens of KV cache from admission to finish, and is charged at
    // finish.
    const bool literal = (e.flags & FSO_LITERAL) != 0;
    struct Running {
      int64_t rec, fin;
    };
    std::vector<Running> batch;
    int64_t kv_used = 0;
    std::vector<uint8_t> served(n, 0), aborted(n, 0), dropped(n, 0);
    std::vector<int64_t> next_call(n, -1);
    if (t->call)
      for (int64_t i = 0; i < n; ++i)
        if (t->call[G(i)] > 0) next_call[t->prev[G(i)]] = i;

    for (int64_t i = 0; i < n; ++i) {
      out->status[G(i)] = -1;
      if (out->admit_step) out->admit_step[G(i)] = -1;
      if (out->admit_seq) out->admit_seq[G(i)] = -1;
      if (out->counter_after) out->counter_after[G(i)] = -1;
      if (out->counter_on_arrival) out->counter_on_arrival[G(i)] = -1;
    }

    auto set_counter = [&](int32_t k, int64_t v) {
      bool inX = !queued[k].empty(), inT0 = !ready[k].empty();
      if (inX) X.erase({u[k], k});
      if (inT0) T0.erase({u[k], k});
      u[k] = v;
      if (inX) X.insert({v, k});
      if (inT0) T0.insert({v, k});
    };
    auto make_ready = [&](int64_t i) {
      int32_t k = t->user[G(i)];
      if (ready[k].empty()) T0.insert({u[k], k});
      ready[k].insert(i);
    };

    const int64_t tau = e.step_us, C = e.cap_tokens, theta = e.overload_tokens;
    int32_t last_exit = -1;  // the most recent user to exit Q
    int64_t debt = 0, backlog = 0, seq = 0, gap = 0, nxt = 0, s = 0;

    while (true) {
      if (max_steps >= 0 && s >= max_steps) break;
      if (nxt == n && X.empty() && batch.empty()) break;
      if (X.empty() && literal) {
        // Nothing queued: nothing happens before the next arrival or the next finish.
        int64_t target = nxt < n ? t->ts_us[G(nxt)] / tau : INT64_MAX;
        for (const Running &b : batch) target = std::min(target, b.fin);
        if (max_steps >= 0 && target > max_steps) target = max_steps;
        if (target > s) {
          s = target;
          if (max_steps >= 0 && s >= max_steps) break;
        }
      } else if (X.empty() && nxt < n) {
        // Nothing queued: the steps before the next arrival only pay back debt.
        int64_t target = t->ts_us[G(nxt)] / tau;
        if (max_steps >= 0 && target > max_steps) target = max_steps;
        if (target > s) {
          int64_t k = target - s;
          debt = (k >= (-debt + C - 1) / C) ? 0 : debt + k * C;
          s = target;
          if (max_steps >= 0 && s >= max_steps) break;
        }
      }
      if (s >= INT32_MAX) return FSO_E_OVERFLOW;

      // Monitoring stream: every request that has arrived by the end of step s.
      while (nxt < n && t->ts_us[G(nxt)] / tau <= s) {
        int64_t i = nxt++;
        int32_t k = t->user[G(i)];
        if (queued[k].empty()) {  // user not in Q: counter lift (Alg. 1, lift on arrival)
          if (X.empty()) {
            if (last_exit >= 0) set_counter(k, std::max(u[k], u[last_exit]));
          } else {
            set_counter(k, std::max(u[k], X.begin()->first));
          }
        }
        if (out->counter_on_arrival) out->counter_on_arrival[G(i)] = u[k];
        bool blocked;
        int8_t code;
        if (!is_first_call(t, G(i)) && !blind) {
          // mid-interaction: never limit-checked, dropped only if its interaction was throttled
          blocked = aborted[t->head[G(i)]] != 0;
          code = 3;
        } else if (!is_first_call(t, G(i)) && dropped[t->prev[G(i)]]) {
          // interaction-blind limits: an earlier call was dropped, the interaction is abandoned
          blocked = true;
          code = 3;
        } else {
          // OIT: limits apply only while the system is overloaded
          uint8_t why = reason ? reason[G(i)] : 0;
          blocked = backlog > theta && why != 0;
          code = int8_t(why);
          if (check && blocked && !(backlog > theta)) return fail("throttled while not overloaded", i);
        }
        if (blocked) {
          out->status[G(i)] = code;
          dropped[i] = 1;
          if (is_first_call(t, G(i))) aborted[i] = 1;
        } else {
          if (queued[k].empty()) X.insert({u[k], k});
          queued[k].insert(i);
          arrival_order.insert(i);
          backlog += tokens(t, G(i));
          if (!is_first_call(t, G(i)) && served[t->prev[G(i)]]) make_ready(i);
        }
      }

      // Execution stream: admit least-served users while the step has budget (literal
      // engine: while the chosen request's tokens fit in the free KV cache, or nothing
      // runs at all).
      int64_t budget = C + debt;
      while ((literal || budget > 0) && !X.empty()) {
        bool tier0 = !T0.empty();
        int32_t k;
        int64_t r;
        if (fcfs) {
          // the earliest queued request (a later call waiting for its previous call
          // cannot be it: that call arrived earlier and is still queued)
          r = *arrival_order.begin();
          k = t->user[G(r)];
          tier0 = ready[k].count(r) != 0;
          if (check && !tier0 && !is_first_call(t, G(r))) return fail("FCFS picked a waiting call", r);
        } else if (tier0) {
          k = T0.begin()->second;
          r = *ready[k].begin();
        } else {
          k = X.begin()->second;
          r = *queued[k].begin();
          if (check && !is_first_call(t, G(r))) return fail("queue front is a later call", r);
          if (check && u[k] != X.begin()->first) return fail("argmin key stale", r);
        }
        if (literal && !batch.empty() && kv_used + tokens(t, G(r)) > C) break;
        if (tier0) {
          ready[k].erase(r);
          if (ready[k].empty()) T0.erase({u[k], k});
        }
        queued[k].erase(r);
        arrival_order.erase(r);
        bool emptied = queued[k].empty();
        if (emptied) X.erase({u[k], k});
        if (check && served[r]) return fail("served twice", r);
        served[r] = 1;
        out->status[G(r)] = 0;
        int64_t tok = tokens(t, G(r));
        budget -= tok;
        backlog -= tok;
        if (literal) {
          // prefill now (its first output token), one more token per step, charge at finish
          int64_t lo = t->len_out[G(r)];
          batch.push_back({r, s + std::max<int64_t>(lo, 1) - 1});
          kv_used += tok;
        } else {
          int64_t before = u[k];
          int64_t after = before + cost[G(r)];
          if (after >= kValueLimit) return FSO_E_OVERFLOW;
          set_counter(k, after);
          if (check && after < before) return fail("counter decreased", r);
          if (check && !fcfs && !tier0 && !X.empty() && after - X.begin()->first > cost[G(r)])
            return fail("served user ends more than one cost above the minimum", r);
          if (out->counter_after) out->counter_after[G(r)] = after;
        }
        if (out->admit_step) out->admit_step[G(r)] = int32_t(s);
        if (out->admit_seq) out->admit_seq[G(r)] = int32_t(seq);
        ++seq;
        if (emptied) last_exit = k;
        int64_t nc = next_call[r];
        if (nc >= 0 && nc < nxt && !dropped[nc]) {  // (interaction-blind limits may drop it)
          if (check && !queued[t->user[G(nc)]].count(nc)) return fail("next call not queued", nc);
          make_ready(nc);
        }
      }
      if (literal) {
        // Decode: calls whose last output token falls in step s finish, in admission
        // order; the user is charged the call's service (Eq. 2) and its KV is freed.
        if (check && kv_used > C && batch.size() > 1) return fail("KV cache over capacity", -1);
        std::vector<Running> still;
        for (const Running &b : batch) {
          if (b.fin != s) {
            still.push_back(b);
            continue;
          }
          int32_t k = t->user[G(b.rec)];
          int64_t after = u[k] + cost[G(b.rec)];
          if (after >= kValueLimit) return FSO_E_OVERFLOW;
          set_counter(k, after);
          if (out->counter_after) out->counter_after[G(b.rec)] = after;
          kv_used -= tokens(t, G(b.rec));
        }
        batch.swap(still);
      } else {
        debt = std::min<int64_t>(budget, 0);
      }
      if (!X.empty()) gap = std::max(gap, X.rbegin()->first - X.begin()->first);
      ++s;
    }

    if (check && max_steps < 0) {
      for (int64_t i = 0; i < n; ++i) {
        int8_t st = out->status[G(i)];
        if (st < 0 || st > 3) return fail("record never decided", i);
        if ((st == 0) != (served[i] != 0)) return fail("status and service disagree", i);
      }
    }
    if (out->counter)
      for (int32_t k = 0; k < U; ++k) out->counter[int64_t(rep) * U + k] = u[k];
    if (out->steps) out->steps[rep] = s;
    if (out->decisions) out->decisions[rep] = seq;
    if (out->max_gap) out->max_gap[rep] = gap;
    return FSO_OK;
  }
};

}  // namespace

extern "C" {

int fso_coef_from_expectations(int32_t n_apps, int32_t n_stages, const double *e_in,
                               const double *e_sys, const double *e_out, int64_t K,
                               int64_t *coef) {
  if (n_apps < 1 || n_stages < 1 || K < 1 || K > (int64_t(1) << 20) || !e_in || !e_sys || !e_out ||
      !coef)
    return FSO_E_ARG;
  // Token-class weights alpha, beta, gamma = 1, 2, 1 for input, system, output tokens.
  const int64_t cls[3] = {1, 2, 1};
  for (int32_t a = 0; a < n_apps; ++a)
    for (int32_t j = 0; j < n_stages; ++j) {
      int64_t at = int64_t(a) * n_stages + j;
      double w = cls[0] * e_in[at] + cls[1] * e_sys[at] + cls[2] * e_out[at];  // Eq. 1
      if (!(w > 0.0)) return FSO_E_ARG;
      for (int x = 0; x < 3; ++x) {
        double q = double(int64_t(65536) * K * cls[x]) / w;
        double c = std::nearbyint(q);  // default rounding mode: half to even
        if (!(c >= 0.0) || c >= double(kCoefLimit)) return FSO_E_RANGE;
        coef[at * 3 + x] = int64_t(c);
      }
    }
  return FSO_OK;
}

namespace {

// round_half_even(num / den) for den > 0, exact.
unsigned __int128 div_round_half_even(unsigned __int128 num, unsigned __int128 den) {
  unsigned __int128 q = num / den, r = num % den;
  if (2 * r > den || (2 * r == den && (q & 1))) ++q;
  return q;
}

}  // namespace

int fso_weights_from_history(const fso_trace *t, int32_t n_stages, int64_t K, int32_t base_limit,
                             int64_t *stats, int64_t *coef, int32_t *t_app) {
  if (n_stages < 1 || n_stages > 4096 || K < 1 || K > (int64_t(1) << 20) || base_limit < 0 ||
      !stats)
    return FSO_E_ARG;
  // Only the fields read here are checked: app, call and the token counts.
  int code = validate_trace(t, kLengths);
  if (code == FSO_E_ARG) return code;
  if (t->rep_off[t->n_replicas] >= (int64_t(1) << 36)) return FSO_E_ARG;
  const int32_t A = t->n_apps, J = n_stages;
  enum { kN, kFirst, kIn, kSys, kOut };
  std::vector<int64_t> st(size_t(A) * J * 5, 0);
  // The history's records per (app, stage): how many, how many first calls, token sums.
  for (int32_t r = 0; r < t->n_replicas; ++r) {
    Replica rp = replica(t, r);
    for (int64_t i = 0; i < rp.n; ++i) {
      int64_t g = rp.base + i;
      int32_t a = t->app[g];
      int64_t li = t->len_in[g], lo = t->len_out[g], ls = t->len_sys ? t->len_sys[g] : 0;
      bool bad = a < 0 || a >= A || (t->call && t->call[g] < 0) || li < 0 || li >= kLenLimit ||
                 lo < 0 || lo >= kLenLimit || ls < 0 || ls >= kLenLimit;
      if (bad) {
        code = worse(code, FSO_E_RANGE);
        continue;
      }
      int32_t j = t->call ? std::min(t->call[g], J - 1) : 0;
      int64_t *s = &st[(size_t(a) * J + j) * 5];
      s[kN] += 1;
      s[kFirst] += is_first_call(t, g) ? 1 : 0;
      s[kIn] += li;
      s[kSys] += ls;
      s[kOut] += lo;
    }
  }
  std::copy(st.begin(), st.end(), stats);
  // Eq. 1's weighted token sum D of a group of n records: w = D / n.
  const int64_t cls[3] = {1, 2, 1};
  auto D_of = [&](const int64_t *s) { return cls[0] * s[kIn] + cls[1] * s[kSys] + cls[2] * s[kOut]; };
  int64_t all_n = 0, all_D = 0;
  std::vector<int64_t> app_n(A, 0), app_D(A, 0), app_first(A, 0);
  for (int32_t a = 0; a < A; ++a)
    for (int32_t j = 0; j < J; ++j) {
      const int64_t *s = &st[(size_t(a) * J + j) * 5];
      app_n[a] += s[kN];
      app_D[a] += D_of(s);
      app_first[a] += s[kFirst];
    }
  for (int32_t a = 0; a < A; ++a) {
    all_n += app_n[a];
    all_D += app_D[a];
  }
  for (int32_t a = 0; a < A; ++a) {
    for (int32_t j = 0; coef && j < J; ++j) {
      const int64_t *s = &st[(size_t(a) * J + j) * 5];
      int64_t n = s[kN], D = D_of(s);
      if (n == 0 || D == 0) {  // too little history: pool the app's stages, then all apps
        n = app_n[a];
        D = app_D[a];
      }
      if (n == 0 || D == 0) {
        n = all_n;
        D = all_D;
      }
      if (n == 0 || D == 0) {  // no tokens anywhere: w_aj = K
        n = 1;
        D = K;
      }
      for (int x = 0; x < 3; ++x) {
        unsigned __int128 num = (unsigned __int128)(int64_t(65536) * K * cls[x]) * uint64_t(n);
        unsigned __int128 c = div_round_half_even(num, uint64_t(D));
        if (c >= (unsigned __int128)kCoefLimit) {
          code = worse(code, FSO_E_RANGE);
          c = 0;
        }
        coef[(size_t(a) * J + j) * 3 + x] = int64_t(c);
      }
    }
    if (t_app) {
      // mean LLM calls per interaction of app a = records / first calls, rounded up
      int64_t lim = base_limit;
      if (app_first[a] > 0) {
        unsigned __int128 num = (unsigned __int128)uint64_t(base_limit) * uint64_t(app_n[a]);
        unsigned __int128 v = (num + uint64_t(app_first[a]) - 1) / uint64_t(app_first[a]);
        if (v > (unsigned __int128)INT32_MAX) {
          code = worse(code, FSO_E_RANGE);
          v = 0;
        }
        lim = int64_t(v);
      }
      t_app[a] = int32_t(lim);
    }
  }
  return code;
}

int fso_cost(const fso_trace *t, int32_t n_stages, int64_t coef_rep_stride, const int64_t *coef,
             int64_t prio_rep_stride, const int32_t *prio, int64_t *cost) {
  if (n_stages < 1 || !coef || !cost || coef_rep_stride < 0 || prio_rep_stride < 0) return FSO_E_ARG;
  // Eq. 2 reads the user only through its priority E_i: user ids are checked only
  // when priorities are given.
  int code = validate_trace(t, kIds | kLengths | (prio ? unsigned(kUsers) : 0u));
  if (code == FSO_E_ARG) return code;
  for (int32_t r = 0; r < t->n_replicas; ++r) {
    Replica rp = replica(t, r);
    for (int64_t i = 0; i < rp.n; ++i) {
      int64_t g = rp.base + i;
      int32_t a = t->app[g], k = prio ? t->user[g] : 0;
      if (a < 0 || a >= t->n_apps || k < 0 || k >= t->n_users) continue;  // reported above
      int32_t j = t->call ? std::min(std::max(t->call[g], 0), n_stages - 1) : 0;
      const int64_t *c = coef + r * coef_rep_stride + (int64_t(a) * n_stages + j) * 3;
      int64_t E = prio ? prio[r * prio_rep_stride + k] : 256;  // E_i in Q8
      bool ok = E >= 0 && E < kPrioLimit;
      for (int x = 0; x < 3; ++x) ok = ok && c[x] >= 0 && c[x] < kCoefLimit;
      if (!ok) {
        code = worse(code, FSO_E_RANGE);
        continue;
      }
      unsigned __int128 L_I = uint32_t(std::max(t->len_in[g], 0));
      unsigned __int128 L_S = t->len_sys ? uint32_t(std::max(t->len_sys[g], 0)) : 0;
      unsigned __int128 L_O = uint32_t(std::max(t->len_out[g], 0));
      // Eq. 2 for one call: E_i * (alpha L_I + beta L_S + gamma L_O) / w_aj, with the
      // token-class weights and 1/w_aj folded into the Q16 coefficients.
      unsigned __int128 weighted = L_I * uint64_t(c[0]) + L_S * uint64_t(c[1]) + L_O * uint64_t(c[2]);
      unsigned __int128 v = (weighted * uint64_t(E)) >> 8;
      if (v >= (unsigned __int128)kValueLimit) {
        code = worse(code, FSO_E_OVERFLOW);
        cost[g] = 0;
      } else {
        cost[g] = int64_t(v);
      }
    }
  }
  return code;
}

int fso_throttle(const fso_trace *t, int64_t window_us, int32_t t_user, const int32_t *t_app,
                 const uint8_t *overloaded, int32_t raw, uint8_t *reason, uint32_t *bitmap,
                 int32_t *cnt_user, int32_t *cnt_app) {
  return fso_throttle_scoped(t, window_us, t_user, t_app, 0, overloaded, raw, reason, bitmap,
                             cnt_user, cnt_app);
}

int fso_throttle_scoped(const fso_trace *t, int64_t window_us, int32_t t_user,
                        const int32_t *t_app, int32_t app_scope, const uint8_t *overloaded,
                        int32_t raw, uint8_t *reason, uint32_t *bitmap, int32_t *cnt_user,
                        int32_t *cnt_app) {
  if (window_us <= 0 || t_user < 0 || !t_app || !reason || app_scope < 0 || app_scope > 1)
    return FSO_E_ARG;
  // The limit tests read arrival times, users and apps; the gated mode also each
  // request's link to its interaction's first call, which is itself for a first call.
  int code = validate_trace(t, kApps | kUsers | kOrder | (raw ? 0u : unsigned(kHeads)));
  if (code == FSO_E_ARG) return code;
  for (int32_t a = 0; a < t->n_apps; ++a)
    if (t_app[a] < 0) return FSO_E_ARG;
  if (code != FSO_OK) return code;
  const int64_t A = t->n_apps;
  for (int32_t r = 0; r < t->n_replicas; ++r) {
    Replica rp = replica(t, r);
    // OIT's dictionaries: user -> arrival times, (user, app) -> arrival times (or
    // app -> arrival times for the app-level limit).
    std::unordered_map<int64_t, std::deque<int64_t>> by_user, by_user_app;
    std::vector<uint8_t> raw_why(rp.n, 0);  // each request's own limit test
    for (int64_t i = 0; i < rp.n; ++i) {
      int64_t g = rp.base + i, ts = t->ts_us[g];
      std::deque<int64_t> &du = by_user[t->user[g]];
      std::deque<int64_t> &da =
          by_user_app[app_scope ? int64_t(t->app[g]) : int64_t(t->user[g]) * A + t->app[g]];
      du.push_back(ts);  // counted on arrival, whatever the request's fate
      da.push_back(ts);
      while (du.front() <= ts - window_us) du.pop_front();
      while (da.front() <= ts - window_us) da.pop_front();
      int64_t cu = int64_t(du.size()), ca = int64_t(da.size());
      if (cnt_user) cnt_user[g] = int32_t(cu);
      if (cnt_app) cnt_app[g] = int32_t(ca);
      // user limit first, then the application limit
      uint8_t why = cu > t_user ? 1 : (ca > t_app[t->app[g]] ? 2 : 0);
      raw_why[i] = why;
      if (raw) {
        reason[g] = why;
      } else if (!t->head || t->head[g] == i) {  // a first call
        bool over = overloaded ? overloaded[g] != 0 : true;
        reason[g] = over ? why : 0;
      } else {
        // a later call inherits its interaction's fate: stalled, never throttled itself;
        // dropped iff its first call (at head) was over a limit while overloaded
        const int64_t h = t->head[g];
        const bool hover = overloaded ? overloaded[rp.base + h] != 0 : true;
        reason[g] = (hover && raw_why[h] != 0) ? 3 : 0;
      }
    }
  }
  if (bitmap) {
    int64_t N = t->rep_off[t->n_replicas];
    for (int64_t w = 0; w < (N + 31) / 32; ++w) bitmap[w] = 0;
    for (int64_t g = 0; g < N; ++g)
      if (reason[g]) bitmap[g / 32] |= uint32_t(1) << (g % 32);
  }
  return FSO_OK;
}

int fso_simulate(const fso_trace *t, const int64_t *cost, const uint8_t *exceed_reason,
                 const fso_engine *e, int64_t max_steps, int32_t n_threads, int32_t check,
                 fso_outputs *out) {
  if (!e || !out || !out->status || !cost) return FSO_E_ARG;
  if (e->step_us <= 0 || e->cap_tokens <= 0 || e->cap_tokens > kCapLimit) return FSO_E_ARG;
  if (e->flags & ~uint32_t(FSO_FCFS | FSO_BLIND | FSO_LITERAL)) return FSO_E_ARG;
  int code = validate_trace(t, kIds | kUsers | kOrder | kChain | kLengths);
  if (code != FSO_OK) return code;
  int64_t N = t->rep_off[t->n_replicas];
  for (int64_t g = 0; g < N; ++g) {
    if (cost[g] < 0 || cost[g] >= kValueLimit) code = worse(code, FSO_E_RANGE);
    if (exceed_reason && exceed_reason[g] > 2) code = worse(code, FSO_E_RANGE);
  }
  if (code != FSO_OK) return code;
  std::vector<int> codes(t->n_replicas, FSO_OK);
  for_each_replica(t->n_replicas, n_threads, [&](int32_t r) {
    Simulation sim{t, replica(t, r), r, cost, exceed_reason, *e, max_steps, check != 0, out};
    codes[r] = sim.run();
  });
  for (int c : codes) code = worse(code, c);
  return code;
}

int fso_fairness_metrics(const fso_trace *t, const int64_t *cost, const int8_t *status,
                         const int32_t *admit_step, const int64_t *max_gap, int64_t step_us,
                         int32_t delay_steps, fso_metrics *m) {
  if (!cost || !status || !admit_step || !m || step_us <= 0 || delay_steps < 0) return FSO_E_ARG;
  int code = validate_trace(t, kIds | kUsers | kChain);
  if (code != FSO_OK) return code;
  const int32_t U = t->n_users;
  for (int32_t r = 0; r < t->n_replicas; ++r) {
    Replica rp = replica(t, r);
    std::vector<uint8_t> has(U, 0), full_user(U, 0), delayed(U, 0);
    std::vector<int64_t> charged(U, 0);
    std::vector<uint8_t> any_served(rp.n, 0), any_blocked(rp.n, 0);  // indexed by interaction head
    int64_t admitted = 0, throttled = 0, interactions = 0;
    unsigned __int128 total = 0;  // the replica's charged service, exact
    for (int64_t i = 0; i < rp.n; ++i) {
      int64_t g = rp.base + i;
      int32_t k = t->user[g];
      int64_t h = is_first_call(t, g) ? i : t->head[g];
      has[k] = 1;
      if (is_first_call(t, g)) ++interactions;
      if (status[g] == 0) {
        ++admitted;
        // charged service is a cost in [0, 2^62); another value is an error (not added)
        if (cost[g] < 0 || cost[g] >= kValueLimit) {
          code = worse(code, FSO_E_RANGE);
        } else {
          total += uint64_t(cost[g]);
          // below 2^62 in total (else an overflow error below), so no sum wraps
          if (total < (unsigned __int128)kValueLimit) charged[k] += cost[g];
        }
        any_served[h] = 1;
        if (admit_step[g] - t->ts_us[g] / step_us > delay_steps) delayed[k] = 1;
      } else {
        any_blocked[h] = 1;
        if (status[g] > 0) ++throttled;
      }
    }
    int64_t full = 0, aborted = 0, wasted = 0;
    for (int64_t i = 0; i < rp.n; ++i) {
      int64_t g = rp.base + i;
      if (!is_first_call(t, g)) continue;
      if (!any_blocked[i]) {
        ++full;
        full_user[t->user[g]] = 1;
      }
      if (any_served[i] && any_blocked[i]) ++aborted;
    }
    for (int64_t i = 0; i < rp.n; ++i) {
      int64_t g = rp.base + i;
      int64_t h = is_first_call(t, g) ? i : t->head[g];
      if (status[g] == 0 && any_served[h] && any_blocked[h]) wasted += tokens(t, g);
    }
    if (total >= (unsigned __int128)kValueLimit) code = worse(code, FSO_E_OVERFLOW);
    // Jain's index over users with at least one request: (sum x)^2 / (n * sum x^2),
    // exact: sum x < 2^62 and sum x^2 <= (sum x)^2 < 2^124.
    unsigned __int128 s1 = 0, s2 = 0;
    int64_t n_users = 0, n_full = 0, n_delayed = 0;
    for (int32_t k = 0; k < U; ++k) {
      if (!has[k]) continue;
      ++n_users;
      s1 += uint64_t(charged[k]);
      s2 += (unsigned __int128)uint64_t(charged[k]) * uint64_t(charged[k]);
      n_full += full_user[k];
      n_delayed += delayed[k];
    }
    double jain = s2 == 0 ? 1.0 : (double(s1) * double(s1)) / (double(n_users) * double(s2));
    auto pct = [](int64_t a, int64_t b) { return b == 0 ? 0.0 : 100.0 * double(a) / double(b); };
    if (m->jain) m->jain[r] = jain;
    if (m->max_gap_tokens) m->max_gap_tokens[r] = max_gap ? double(max_gap[r]) / 65536.0 : 0.0;
    if (m->svc_req_pct) m->svc_req_pct[r] = pct(admitted, rp.n);
    if (m->svc_int_pct) m->svc_int_pct[r] = pct(full, interactions);
    if (m->served_users_pct) m->served_users_pct[r] = pct(n_full, n_users);
    if (m->delayed_users_pct) m->delayed_users_pct[r] = pct(n_delayed, n_users);
    if (m->throttled) m->throttled[r] = throttled;
    if (m->aborted_midway) m->aborted_midway[r] = aborted;
    if (m->wasted_tokens) m->wasted_tokens[r] = wasted;
  }
  return code;
}

// ---------------------------------------------------------------------------
// Workload analysis (Sec. 3: Fig. 2 rates per user overall and per application,
// Figs. 3 and 5 token lengths per application, Fig. 4 calls per interaction, Table 2
// graph sizes and their tokens).

// floor(log2(x / M)) for x >= 1, M >= 1, by plain comparison: the largest k with
// M * 2^k <= x (k may be negative: then M <= x * 2^-k).
static int64_t floor_log2_ratio(int64_t x, int64_t M) {
  const unsigned __int128 X = uint64_t(x), Mm = uint64_t(M);
  int64_t k = 0;
  if (X >= Mm) {
    while ((Mm << (k + 1)) <= X) ++k;
  } else {
    k = -1;
    while ((X << (-k)) < Mm) --k;
  }
  return k;
}

static int rate_bin(int64_t x, int64_t M) {
  if (x == 0) return 0;
  return int(64 + floor_log2_ratio(x, M));
}

static int len_bin(int64_t L) {
  if (L == 0) return 0;
  int b = 0;
  while ((int64_t(1) << (b + 1)) <= L) ++b;  // floor(log2 L)
  return 1 + b;
}

static int graph_bin(int64_t s) {
  if (s <= 1) return 0;
  if (s <= 10) return 1;
  if (s <= 20) return 2;
  if (s <= 30) return 3;
  if (s <= 40) return 4;
  if (s <= 50) return 5;
  return 6;
}

int fso_workload_stats(const fso_trace *t, int64_t minute_us, fso_wstats *o) {
  if (minute_us <= 0 || !o || !o->minutes || !o->user_req || !o->user_tok || !o->rate_hist ||
      !o->len_hist || !o->len_sum || !o->size_hist || !o->graph)
    return FSO_E_ARG;
  int code = validate_trace(t, kIds | kUsers | kLengths);
  if (code == FSO_E_ARG) return code;
  const int32_t R = t->n_replicas, U = t->n_users, A = t->n_apps;
  for (int32_t r = 0; r < R; ++r) {
    Replica rp = replica(t, r);
    int64_t max_ts = -1;
    for (int64_t i = 0; i < rp.n; ++i) max_ts = std::max(max_ts, t->ts_us[rp.base + i]);
    const int64_t M = rp.n > 0 ? max_ts / minute_us + 1 : 0;
    o->minutes[r] = M;
    std::vector<int64_t> req(U, 0), tok(U, 0), areq(int64_t(U) * A, 0), atok(int64_t(U) * A, 0);
    std::vector<int64_t> lh(int64_t(A) * 3 * FSO_LEN_BINS, 0), ls(int64_t(A) * 3, 0);
    std::vector<int64_t> size(rp.n, 0);  // records per first call (interaction)
    for (int64_t i = 0; i < rp.n; ++i) {
      const int64_t g = rp.base + i;
      const int32_t u = t->user[g], a = t->app[g];
      const int64_t L[3] = {t->len_in[g], t->len_sys ? t->len_sys[g] : 0, t->len_out[g]};
      bool ok = u >= 0 && u < U && a >= 0 && a < A && t->ts_us[g] >= 0;
      for (int x = 0; x < 3; ++x) ok = ok && L[x] >= 0 && L[x] < kLenLimit;
      int64_t h = i;
      if (!is_first_call(t, g)) {
        h = t->head[g];
        if (h < 0 || h >= i) ok = false;
      }
      if (!ok) {
        code = worse(code, FSO_E_RANGE);
        continue;
      }
      const int64_t tk = L[0] + L[1] + L[2];
      req[u] += 1;
      tok[u] += tk;
      areq[int64_t(u) * A + a] += 1;
      atok[int64_t(u) * A + a] += tk;
      for (int x = 0; x < 3; ++x) {
        lh[(int64_t(a) * 3 + x) * FSO_LEN_BINS + len_bin(L[x])] += 1;
        ls[int64_t(a) * 3 + x] += L[x];
      }
      size[h] += 1;
    }
    int64_t *rh = o->rate_hist + int64_t(r) * (A + 1) * 2 * FSO_RATE_BINS;
    for (int64_t k = 0; k < int64_t(A + 1) * 2 * FSO_RATE_BINS; ++k) rh[k] = 0;
    for (int32_t u = 0; u < U; ++u) {
      o->user_req[int64_t(r) * U + u] = req[u];
      o->user_tok[int64_t(r) * U + u] = tok[u];
      if (req[u] > 0) {  // a user with a request, overall (row A)
        rh[(int64_t(A) * 2 + 0) * FSO_RATE_BINS + rate_bin(req[u], M)] += 1;
        rh[(int64_t(A) * 2 + 1) * FSO_RATE_BINS + rate_bin(tok[u], M)] += 1;
      }
      for (int32_t a = 0; a < A; ++a) {
        const int64_t n_ua = areq[int64_t(u) * A + a], t_ua = atok[int64_t(u) * A + a];
        if (o->user_app_req) o->user_app_req[(int64_t(r) * U + u) * A + a] = n_ua;
        if (o->user_app_tok) o->user_app_tok[(int64_t(r) * U + u) * A + a] = t_ua;
        if (n_ua > 0) {  // a user of application a
          rh[(int64_t(a) * 2 + 0) * FSO_RATE_BINS + rate_bin(n_ua, M)] += 1;
          rh[(int64_t(a) * 2 + 1) * FSO_RATE_BINS + rate_bin(t_ua, M)] += 1;
        }
      }
    }
    for (int64_t k = 0; k < int64_t(A) * 3 * FSO_LEN_BINS; ++k)
      o->len_hist[int64_t(r) * A * 3 * FSO_LEN_BINS + k] = lh[k];
    for (int64_t k = 0; k < int64_t(A) * 3; ++k) o->len_sum[int64_t(r) * A * 3 + k] = ls[k];
    int64_t *sh = o->size_hist + int64_t(r) * A * FSO_SIZE_BINS;
    for (int64_t k = 0; k < int64_t(A) * FSO_SIZE_BINS; ++k) sh[k] = 0;
    int64_t *gr = o->graph + int64_t(r) * FSO_GRAPH_BINS * 5;
    for (int k = 0; k < FSO_GRAPH_BINS * 5; ++k) gr[k] = 0;
    for (int64_t i = 0; i < rp.n; ++i) {  // interactions, at their first call
      const int64_t g = rp.base + i;
      if (!is_first_call(t, g) || size[i] == 0) continue;
      const int32_t a = t->app[g];
      if (a < 0 || a >= A) continue;
      sh[int64_t(a) * FSO_SIZE_BINS + std::min<int64_t>(size[i], FSO_SIZE_BINS) - 1] += 1;
      gr[graph_bin(size[i]) * 5 + 0] += 1;
    }
    for (int64_t i = 0; i < rp.n; ++i) {  // requests, by the size of their interaction
      const int64_t g = rp.base + i;
      const bool first = is_first_call(t, g);
      const int64_t h = first ? i : t->head[g];
      if (h < 0 || (first ? h != i : h >= i) || t->user[g] < 0 || t->user[g] >= U ||
          t->app[g] < 0 || t->app[g] >= A)
        continue;
      int64_t *row = gr + graph_bin(size[h]) * 5;
      row[1] += 1;
      row[2] += t->len_in[g];
      row[3] += t->len_out[g];
      row[4] += t->len_sys ? t->len_sys[g] : 0;
    }
  }
  return code;
}

}  // extern "C"
