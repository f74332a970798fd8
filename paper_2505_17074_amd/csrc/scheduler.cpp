// LAPS-SD request scheduler (arXiv 2505.17074, Algorithm 1, Sec. 4) and the
// FCFS, predicted-length SJF, exact SJF and LAS baselines: host C++ behind
// the C ABI of specsched.h.
//
// Every arrived, unfinished request sits in one ordered set keyed by what its
// policy ranks on, so a decision is a set minimum:
//   FCFS       (arrival, id)
//   LP_SJF     (predicted length, arrival, id)
//   SJF_EXACT  (size hint, arrival, id)
//   LAS        (attained service, arrival, id)
//   LAPS_SD    per queue j: perceptible (Eq. (6) estimate, arrival, id) and
//              non-perceptible (arrival, id)
// A request is taken out of its set while its round is reported and put back
// under its new key.  Floating point (rates, the stability window, Eq. (6))
// follows the operation order of the header exactly, with contraction off.
#pragma clang fp contract(off)

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <limits>
#include <new>
#include <set>
#include <vector>

#include "specsched.h"

namespace {

struct Key {
  int64_t i0;       // integer rank (length, hint, attained service) or 0
  double d0;        // Eq. (6) estimate for perceptible LAPS-SD requests, else 0
  int64_t arrival;
  int32_t id;
  bool operator<(const Key& o) const {
    if (i0 != o.i0) return i0 < o.i0;
    if (d0 != o.d0) return d0 < o.d0;
    if (arrival != o.arrival) return arrival < o.arrival;
    return id < o.id;
  }
};

struct ReqState {
  int64_t arrival = 0;
  int64_t hint = 0;
  int64_t attained = 0;
  int64_t acc_sum = 0;
  int64_t drafted = 0;
  int32_t prompt = 0;
  int32_t pred_len = 1;
  int32_t draft = 0;
  int32_t queue = 0;
  int32_t rounds = 0;
  int32_t n_rates = 0;          // rates recorded (window holds the last gamma)
  bool arrived = false;
  bool finished = false;
  bool perceptible = false;
  double A = 0.0;
  double T = 0.0;
  Key key{};
  int set_index = -1;           // which ready set holds it, -1 = none
};

bool params_ok(const spec_sched_params_t* p) {
  return p && p->K >= 1 && p->M >= 2 && p->S1_up_us >= 1 && p->gamma >= 1 && std::isfinite(p->delta) &&
         p->delta >= 0.0 && p->t_ssm_us >= 0 && p->t_llm_us >= 0 && p->swap_us_per_token >= 0;
}

}  // namespace

struct spec_sched {
  int policy = 0;
  spec_sched_params_t P{};
  int32_t capacity = 0;
  std::vector<ReqState> req;
  std::vector<double> rates;                 // capacity x gamma ring buffers
  std::set<std::pair<int64_t, int32_t>> pending;   // (arrival, id) not yet arrived
  std::vector<std::set<Key>> sets;           // ready sets (see the file comment)
  int32_t running = -1;                      // request of the last reported round
  int64_t n_ready = 0;

  // queue of attained service E: the first j with E < S1_up * M^j, else K-1
  int32_t queue_of(int64_t E) const {
    int64_t up = P.S1_up_us;
    for (int32_t j = 0; j < P.K - 1; ++j) {
      if (E < up) return j;
      if (up > std::numeric_limits<int64_t>::max() / P.M) return j + 1 < P.K - 1 ? j + 1 : P.K - 1;
      up *= P.M;
    }
    return P.K - 1;
  }

  // Eq. (6), in the operation order of the header
  static double eq6(int32_t n, int32_t Lp, double A, int64_t t_ssm, int64_t t_llm) {
    const int64_t num = (int64_t)n * Lp * t_ssm + (int64_t)Lp * t_llm;
    return (double)num / ((double)n * A + 1.0);
  }

  void place(int32_t id) {
    ReqState& r = req[id];
    Key k{0, 0.0, r.arrival, id};
    int idx = 0;
    switch (policy) {
      case SPEC_SCHED_FCFS: break;
      case SPEC_SCHED_LP_SJF: k.i0 = r.pred_len; break;
      case SPEC_SCHED_SJF_EXACT: k.i0 = r.hint; break;
      case SPEC_SCHED_LAS: k.i0 = r.attained; break;
      default:                                // LAPS-SD: sets 2j (perceptible), 2j+1
        if (r.perceptible) {
          k.d0 = r.T;
          idx = 2 * r.queue;
        } else {
          idx = 2 * r.queue + 1;
        }
    }
    r.key = k;
    r.set_index = idx;
    sets[idx].insert(k);
  }

  void unplace(int32_t id) {
    ReqState& r = req[id];
    if (r.set_index >= 0) sets[r.set_index].erase(r.key);
    r.set_index = -1;
  }

  void admit(int64_t now) {
    while (!pending.empty() && pending.begin()->first <= now) {
      const int32_t id = pending.begin()->second;
      pending.erase(pending.begin());
      req[id].arrived = true;
      place(id);
      ++n_ready;
    }
  }

  int32_t pick() const {
    if (n_ready == 0) return -1;
    const bool nonpreemptive =
        policy == SPEC_SCHED_FCFS || policy == SPEC_SCHED_LP_SJF || policy == SPEC_SCHED_SJF_EXACT;
    if (nonpreemptive && running >= 0 && !req[running].finished) return running;
    if (policy != SPEC_SCHED_LAPS_SD) return sets[0].begin()->id;
    int32_t top = 0;
    while (sets[2 * top].empty() && sets[2 * top + 1].empty()) ++top;   // n_ready > 0: some set is non-empty
    if (running >= 0 && !req[running].finished && req[running].perceptible && req[running].queue == top)
      return running;
    if (!sets[2 * top].empty()) return sets[2 * top].begin()->id;
    return sets[2 * top + 1].begin()->id;
  }

  void report(int32_t id, int32_t accepted, int64_t round_us, bool finished) {
    ReqState& r = req[id];
    const int32_t a = std::min(std::max(accepted, 0), r.draft);
    unplace(id);
    r.attained += round_us;
    r.rounds += 1;
    running = id;
    if (finished) {
      r.finished = true;
      --n_ready;
      return;
    }
    if (policy == SPEC_SCHED_LAPS_SD) {
      if (!r.perceptible && r.draft > 0) {
        r.acc_sum += a;
        r.drafted += r.draft;
        const int32_t g = P.gamma;
        double* ring = rates.data() + (size_t)id * g;
        ring[r.n_rates % g] = (double)r.acc_sum / (double)r.drafted;
        r.n_rates += 1;
        if (r.n_rates >= g) {
          // the window oldest to newest
          const int32_t first = r.n_rates - g;
          double lo = ring[first % g], hi = lo, s = 0.0;
          for (int32_t t = 0; t < g; ++t) {
            const double x = ring[(first + t) % g];
            lo = std::min(lo, x);
            hi = std::max(hi, x);
          }
          if (hi - lo < P.delta) {
            for (int32_t t = 0; t < g; ++t) s += ring[(first + t) % g];
            r.perceptible = true;
            r.A = s / (double)g;
            r.T = eq6(r.draft, r.pred_len, r.A, P.t_ssm_us, P.t_llm_us);
          }
        }
      }
      // a perceptible request goes to the queue of max(E, T): its estimate
      // places it, attained service takes over if it overruns
      r.queue = queue_of(r.perceptible ? std::max(r.attained, (int64_t)r.T) : r.attained);
    }
    place(id);
  }
};

namespace {

// Rounds a request needs with its true trace (the SJF_EXACT hint uses them).
int64_t rounds_needed(const spec_sched_request_t& q) {
  int64_t tok = 0, k = 0;
  while (tok < q.out_len) {
    tok += std::min(std::max(q.accepted[k], 0), q.draft) + 1;
    ++k;
  }
  return k;
}

}  // namespace

extern "C" {

spec_status_t spec_sched_create(int32_t policy, const spec_sched_params_t* params, int32_t capacity,
                                spec_sched_t** out) {
  if (!out || policy < SPEC_SCHED_FCFS || policy > SPEC_SCHED_LAPS_SD || !params_ok(params) || capacity < 1)
    return SPEC_ERR_INVALID_ARG;
  spec_sched_t* s = nullptr;
  try {
    s = new spec_sched();
    s->policy = policy;
    s->P = *params;
    s->capacity = capacity;
    s->req.reserve((size_t)capacity);
    if (policy == SPEC_SCHED_LAPS_SD) s->rates.assign((size_t)capacity * (size_t)params->gamma, 0.0);
    s->sets.resize(policy == SPEC_SCHED_LAPS_SD ? 2 * (size_t)params->K : 1);
  } catch (const std::bad_alloc&) {
    delete s;
    return SPEC_ERR_WORKSPACE;
  }
  *out = s;
  return SPEC_OK;
}

void spec_sched_destroy(spec_sched_t* s) { delete s; }

spec_status_t spec_sched_submit(spec_sched_t* s, int64_t arrival_us, int32_t prompt_tokens, int32_t pred_len,
                                int32_t draft, int64_t size_hint_us, int32_t* id_out) {
  if (!s || !id_out || (int64_t)s->req.size() >= s->capacity || arrival_us < 0 || prompt_tokens < 0 ||
      pred_len < 1 || draft < 0 || size_hint_us < 0)
    return SPEC_ERR_INVALID_ARG;
  const int32_t id = (int32_t)s->req.size();
  try {
    ReqState r;
    r.arrival = arrival_us;
    r.hint = size_hint_us;
    r.prompt = prompt_tokens;
    r.pred_len = pred_len;
    r.draft = draft;
    s->req.push_back(r);
    s->pending.insert({arrival_us, id});
  } catch (const std::bad_alloc&) {
    if ((int32_t)s->req.size() > id) s->req.pop_back();
    return SPEC_ERR_WORKSPACE;
  }
  *id_out = id;
  return SPEC_OK;
}

spec_status_t spec_sched_next(spec_sched_t* s, int64_t now_us, int32_t* id_out) {
  if (!s || !id_out) return SPEC_ERR_INVALID_ARG;
  try {
    s->admit(now_us);
  } catch (const std::bad_alloc&) {
    return SPEC_ERR_WORKSPACE;
  }
  *id_out = s->pick();
  return SPEC_OK;
}

spec_status_t spec_sched_report(spec_sched_t* s, int32_t id, int32_t accepted, int64_t round_us,
                                int32_t finished) {
  if (!s || id < 0 || id >= (int32_t)s->req.size() || round_us < 0) return SPEC_ERR_INVALID_ARG;
  const ReqState& r = s->req[id];
  if (!r.arrived || r.finished) return SPEC_ERR_INVALID_ARG;
  try {
    s->report(id, accepted, round_us, finished != 0);
  } catch (const std::bad_alloc&) {
    return SPEC_ERR_WORKSPACE;
  }
  return SPEC_OK;
}

spec_status_t spec_sched_query(const spec_sched_t* s, int32_t id, spec_sched_state_t* out) {
  if (!s || !out || id < 0 || id >= (int32_t)s->req.size()) return SPEC_ERR_INVALID_ARG;
  const ReqState& r = s->req[id];
  out->attained_us = r.attained;
  out->queue = r.queue;
  out->perceptible = r.perceptible ? 1 : 0;
  out->finished = r.finished ? 1 : 0;
  out->rounds = r.rounds;
  out->A = r.A;
  out->T_est_us = r.T;
  return SPEC_OK;
}

spec_status_t spec_sched_simulate(const spec_sched_request_t* reqs, int32_t n, int32_t policy,
                                  const spec_sched_params_t* params, spec_sched_result_t* out) {
  if (!reqs || n < 1 || !out || !out->completion_us || !params_ok(params)) return SPEC_ERR_INVALID_ARG;
  if (out->max_rounds < 0 || (out->max_rounds > 0 && (!out->round_req || !out->round_start_us)))
    return SPEC_ERR_INVALID_ARG;
  for (int32_t i = 0; i < n; ++i) {
    const spec_sched_request_t& q = reqs[i];
    if (q.arrival_us < 0 || q.round_us < 1 || q.prompt_tokens < 0 || q.out_len < 1 || q.pred_len < 1 ||
        q.draft < 0 || !q.accepted || q.n_accepted < q.out_len)
      return SPEC_ERR_INVALID_ARG;
  }
  spec_sched_t* s = nullptr;
  spec_status_t st = spec_sched_create(policy, params, n, &s);
  if (st != SPEC_OK) return st;
  std::vector<int64_t> emitted, rounds;
  std::vector<char> swapped, done;
  try {
    emitted.assign(n, 0);
    rounds.assign(n, 0);
    swapped.assign(n, 0);
    done.assign(n, 0);
  } catch (const std::bad_alloc&) {
    spec_sched_destroy(s);
    return SPEC_ERR_WORKSPACE;
  }
  for (int32_t i = 0; i < n; ++i) {
    const spec_sched_request_t& q = reqs[i];
    const int64_t hint = policy == SPEC_SCHED_SJF_EXACT ? rounds_needed(q) * q.round_us : 0;
    int32_t id = -1;
    st = spec_sched_submit(s, q.arrival_us, q.prompt_tokens, q.pred_len, q.draft, hint, &id);
    if (st != SPEC_OK) {
      spec_sched_destroy(s);
      return st;
    }
  }
  const int64_t swap = params->swap_us_per_token;
  int64_t now = 0, n_rounds = 0, switches = 0, switch_us = 0;
  int32_t left = n, running = -1;
  bool log_full = false;
  while (left > 0) {
    int32_t i = -1;
    st = spec_sched_next(s, now, &i);
    if (st != SPEC_OK) break;
    if (i < 0) {                       // idle until the next arrival
      int64_t t = std::numeric_limits<int64_t>::max();
      for (int32_t j = 0; j < n; ++j)
        if (!done[j]) t = std::min(t, reqs[j].arrival_us);
      now = t;
      continue;
    }
    const spec_sched_request_t& q = reqs[i];
    if (running >= 0 && running != i && !done[running]) {
      const int64_t c = swap * (reqs[running].prompt_tokens + emitted[running]);
      swapped[running] = 1;
      now += c;
      switch_us += c;
      ++switches;
    }
    if (swapped[i]) {
      const int64_t c = swap * (q.prompt_tokens + emitted[i]);
      swapped[i] = 0;
      now += c;
      switch_us += c;
    }
    const int32_t a = std::min(std::max(q.accepted[rounds[i]], 0), q.draft);
    if (n_rounds < out->max_rounds) {
      out->round_req[n_rounds] = i;
      out->round_start_us[n_rounds] = now;
    } else if (out->max_rounds > 0) {
      log_full = true;
    }
    ++n_rounds;
    now += q.round_us;
    rounds[i] += 1;
    emitted[i] += a + 1;
    const bool fin = emitted[i] >= q.out_len;
    if (fin) {
      done[i] = 1;
      --left;
      out->completion_us[i] = now;
    }
    st = spec_sched_report(s, i, a, q.round_us, fin ? 1 : 0);
    if (st != SPEC_OK) break;
    running = i;
  }
  out->n_rounds = n_rounds;
  out->switches = switches;
  out->switch_us = switch_us;
  for (int32_t i = 0; i < n; ++i) {
    const ReqState& r = s->req[i];
    if (out->perceptible) out->perceptible[i] = r.perceptible ? 1 : 0;
    if (out->A) out->A[i] = r.A;
    if (out->T_est_us) out->T_est_us[i] = r.T;
  }
  spec_sched_destroy(s);
  if (st != SPEC_OK) return st;
  return log_full ? SPEC_ERR_INVALID_ARG : SPEC_OK;
}

}  // extern "C"
