/*
 * specsched.h -- C ABI of the LAPS-SD request scheduler (arXiv 2505.17074,
 * Algorithm 1, Sec. 4) and its baselines, host-side C++ in the same library
 * as the verify step (specverify.h).
 *
 * The serving model is the paper's (Sec. 3): one request is served at a
 * time, in speculative decoding rounds.  A round of request i drafts n_i
 * tokens and verifies them in one LLM pass (one verify step, specverify.h);
 * it lasts round_us and yields a + 1 tokens, where a is the round's accepted
 * count (the verify step's accepted_len) and the +1 is the LLM's additional
 * token (Sec. 4.3).  After every round the scheduler chooses the request for
 * the next one.
 *
 * Policies
 *   SPEC_SCHED_FCFS       non-preemptive, earliest arrival first (Sec. 1).
 *   SPEC_SCHED_LP_SJF     non-preemptive, smallest predicted output length
 *                         first (the length-prediction SJF baseline, Sec. 5.1).
 *   SPEC_SCHED_SJF_EXACT  non-preemptive, smallest `size_hint_us` first: with
 *                         the true execution times as hints, the optimum of
 *                         Fig. 1(c) for simultaneous arrivals.
 *   SPEC_SCHED_LAS        least attained service first, re-decided after
 *                         every round (Sec. 3, the LAS baseline of Sec. 5.1).
 *   SPEC_SCHED_LAPS_SD    Algorithm 1:
 *     - K priority queues; queue j (0-based) covers service times in
 *       [S_down(j), S_up(j)), with S_up(j) = S1_up_us * M^j for j < K-1,
 *       the last queue unbounded, and S_down(j) = S_up(j-1), S_down(0) = 0.
 *       New requests enter queue 0.  After every round a non-perceptible
 *       request moves to the queue holding its attained service E (the sum
 *       of its round times: speculation plus verification, Sec. 4.2); a
 *       perceptible one to the queue holding max(E, T), T its Eq. (6)
 *       estimate truncated to an integer ("moved to the corresponding
 *       queue", Sec. 4.1).
 *     - The highest-priority non-empty queue is served (Sec. 4.2).  Inside
 *       it, perceptible requests go first, smallest Eq. (6) estimate first;
 *       then non-perceptible requests, earliest arrival first (Sec. 4.3).
 *     - A running perceptible request keeps the server while its queue is
 *       the highest non-empty one (no preemption inside a queue).
 *     - After every round of a request that drafts (n > 0) and is not yet
 *       perceptible, its acceptance rate so far (accepted / drafted) is
 *       recorded.  Once the last gamma rates differ by less than delta
 *       (max - min), it becomes perceptible, with A = the mean of those gamma
 *       rates and the Eq. (6) estimate
 *         T = (n*Lp*t_ssm_us + Lp*t_llm_us) / (n*A + 1).
 *   All ties go to the earlier arrival, then the smaller request id.
 *
 * Conventions: host memory only and no HIP call; argument errors return
 * SPEC_ERR_INVALID_ARG and change nothing; a failed allocation returns
 * SPEC_ERR_WORKSPACE.  Each decision costs O(log n + K) (ordered sets of the
 * arrived requests, one per key).  Results are deterministic, and floating point is used only for
 * the rates, the stability test and Eq. (6), in the operation order written
 * above (left-to-right sum of the window, then / gamma; the numerator of
 * Eq. (6) in 64-bit integers, converted once).  A scheduler object is not
 * thread-safe: one caller at a time.
 */
#ifndef SPECSCHED_H
#define SPECSCHED_H

#include "specverify.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum spec_sched_policy {
  SPEC_SCHED_FCFS = 0,
  SPEC_SCHED_LP_SJF = 1,
  SPEC_SCHED_SJF_EXACT = 2,
  SPEC_SCHED_LAS = 3,
  SPEC_SCHED_LAPS_SD = 4
} spec_sched_policy_t;

/* Parameters of Algorithm 1 and Eq. (6) (the LAPS-SD policy reads all but
 * swap_us_per_token, which only spec_sched_simulate reads).
 *   K >= 1 queues; M >= 2 (integer threshold ratio); S1_up_us >= 1;
 *   gamma >= 1 rounds in the stability window; delta >= 0 (finite);
 *   t_ssm_us, t_llm_us >= 0: drafting time per token and verification time
 *   per round in Eq. (6); swap_us_per_token >= 0: KV swap cost per cached
 *   token, each direction (spec_sched_simulate). */
typedef struct spec_sched_params {
  int32_t K;
  int32_t M;
  int64_t S1_up_us;
  int32_t gamma;
  int32_t pad0;
  double delta;
  int64_t t_ssm_us;
  int64_t t_llm_us;
  int64_t swap_us_per_token;
} spec_sched_params_t;

typedef struct spec_sched spec_sched_t;   /* opaque */

/* A request's state as the scheduler sees it. */
typedef struct spec_sched_state {
  int64_t attained_us;     /* E: sum of its reported round times */
  int32_t queue;           /* LAPS-SD queue index (0 for other policies) */
  int32_t perceptible;     /* 1 once stable (LAPS-SD) */
  int32_t finished;        /* 1 once reported finished */
  int32_t rounds;          /* rounds reported */
  double A;                /* predicted acceptance rate (when perceptible) */
  double T_est_us;         /* Eq. (6) estimate (when perceptible) */
} spec_sched_state_t;

/* Create a scheduler for up to `capacity` >= 1 requests.  *out receives the
 * object; free it with spec_sched_destroy. */
SPEC_API spec_status_t spec_sched_create(int32_t policy, const spec_sched_params_t* params, int32_t capacity,
                                         spec_sched_t** out);
SPEC_API void spec_sched_destroy(spec_sched_t* s);

/* Register a request: it becomes eligible once `now_us` passed to
 * spec_sched_next reaches arrival_us.  Ids are given in submission order
 * from 0.  pred_len >= 1 is the predicted output length (Sec. 4.3's
 * predictor, LP_SJF and Eq. (6)); draft >= 0 is n; prompt_tokens >= 0;
 * size_hint_us >= 0 is read by SJF_EXACT only.  SPEC_ERR_INVALID_ARG when
 * full or an argument is out of range. */
SPEC_API spec_status_t spec_sched_submit(spec_sched_t* s, int64_t arrival_us, int32_t prompt_tokens,
                                         int32_t pred_len, int32_t draft, int64_t size_hint_us, int32_t* id_out);

/* The request to serve for the next round at time now_us (non-decreasing
 * across calls), or -1 in *id_out when no submitted, unfinished request has
 * arrived by then. */
SPEC_API spec_status_t spec_sched_next(spec_sched_t* s, int64_t now_us, int32_t* id_out);

/* Report the round just served for request `id` (the one spec_sched_next
 * returned last): its accepted count (clamped to [0, draft]), its duration
 * round_us >= 0, and whether the request has now finished. */
SPEC_API spec_status_t spec_sched_report(spec_sched_t* s, int32_t id, int32_t accepted, int64_t round_us,
                                         int32_t finished);

SPEC_API spec_status_t spec_sched_query(const spec_sched_t* s, int32_t id, spec_sched_state_t* out);

/* One request of a simulated workload (host memory). */
typedef struct spec_sched_request {
  int64_t arrival_us;
  int64_t round_us;          /* duration of each of its rounds, >= 1 */
  int32_t prompt_tokens;     /* >= 0 */
  int32_t out_len;           /* true output length, >= 1 */
  int32_t pred_len;          /* predicted output length, >= 1 */
  int32_t draft;             /* n >= 0 */
  const int32_t* accepted;   /* accepted count of each round, >= out_len entries */
  int32_t n_accepted;
  int32_t pad0;
} spec_sched_request_t;

/* Outputs of spec_sched_simulate (host memory, caller-owned).  completion_us
 * [n] is required; the per-round log (round_req, round_start_us, capacity
 * max_rounds) and the per-request perceptible / A / T_est_us [n] arrays may
 * be NULL.  n_rounds, switches and switch_us are written always. */
typedef struct spec_sched_result {
  int64_t* completion_us;
  int32_t* round_req;
  int64_t* round_start_us;
  int64_t max_rounds;
  int64_t n_rounds;
  int64_t switches;          /* preemptions of an unfinished request */
  int64_t switch_us;         /* time spent swapping KV caches */
  int32_t* perceptible;
  double* A;
  double* T_est_us;
} spec_sched_result_t;

/* Serve n >= 1 requests to completion under `policy` with the scheduler
 * above, round by round on the server model of Sec. 3: a round of request i
 * starts when the server is free (or at the next arrival when it idles),
 * lasts round_us and yields accepted[round] + 1 tokens (accepted clamped to
 * [0, draft]); the request completes at the end of the round whose output
 * reaches out_len.  Moving the server away from an unfinished request swaps
 * its KV cache out, and resuming a preempted request swaps it in, each
 * costing swap_us_per_token x (prompt_tokens + tokens emitted so far).
 * SJF_EXACT receives each request's true execution time as its hint.
 * SPEC_ERR_INVALID_ARG on a bad request or a round log too small for the
 * rounds served (then completion_us is still written). */
SPEC_API spec_status_t spec_sched_simulate(const spec_sched_request_t* reqs, int32_t n, int32_t policy,
                                           const spec_sched_params_t* params, spec_sched_result_t* out);

#ifdef __cplusplus
}
#endif

#endif /* SPECSCHED_H */
