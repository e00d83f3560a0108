/*
 * tetri_sched.h -- C ABI of the round-based step scheduler (host code, no GPU).
 *
 * TetriServe (arXiv 2510.01565) serves diffusion requests step by step: at the
 * start of every round of fixed length tau it decides, for each pending
 * request, whether it runs this round and on how many GPUs (its
 * sequence-parallel degree k, a power of two), so that as many requests as
 * possible still meet their deadlines (section 4.2).  This library makes the
 * two per-round decisions:
 *
 *  - ts_allocate: deadline-aware GPU allocation of one request (section
 *    4.2.1): the split of its remaining steps over degrees k that meets its
 *    deadline with the least GPU time sum n_k * k * T(k), T(k) coming from the
 *    offline cost model (per-step time of the request's resolution on k GPUs);
 *  - ts_round_schedule: request packing (section 4.2.2, Algorithm 1): at most
 *    one option per request (run one of its allocations for this round, or
 *    not at all) with total width at most N GPUs, maximising the number of
 *    requests that are not definitely late at the next round start -- a group
 *    knapsack solved by dynamic programming over capacity, O(R N) time;
 *    requests that cannot survive then get at most one leftover GPU each, best
 *    effort (section 4.2.2, last paragraph before Algorithm 1);
 *  - ts_select_batch: selective continuous batching of identical requests.
 *
 * Conventions
 *  - Times are integers in microseconds, so every comparison is exact.
 *  - A cost-model row step_us[j] is the step time on k = 2^j GPUs; 0 marks a
 *    degree that was not profiled (never chosen).  At most TS_MAX_DEGREES
 *    degrees (k <= 2^(TS_MAX_DEGREES-1)).
 *  - All pointers are host memory owned by the caller; nothing is retained
 *    after a call returns.  The calls are thread-safe (no global state).
 *  - Arguments are validated first; on error nothing is written and the call
 *    returns TS_ERR_INVALID_ARG.
 */
#ifndef TETRI_SCHED_H
#define TETRI_SCHED_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TS_MAX_DEGREES 8  /* k = 1, 2, 4, ..., 128 */
#define TS_MAX_ALLOCS 8   /* allocations per request (one per degree at most) */
#define TS_MAX_STEPS 256  /* remaining steps of one request */
#define TS_MAX_GPUS 4096  /* cluster size N */

typedef enum {
  TS_OK = 0,
  TS_ERR_INVALID_ARG = 1, /* null pointer, negative or out-of-range size */
  TS_INFEASIBLE = 2       /* ts_allocate: no split meets the budget (a fallback is still written) */
} ts_status;

/* One allocation (s^m, A^m): `steps` steps run on `gpus` GPUs. */
typedef struct {
  int32_t steps;
  int32_t gpus;
} ts_alloc;

/*
 * Deadline-aware GPU allocation of one request (section 4.2.1).
 *   step_us[n_degrees]  cost-model row of the request's resolution (see above)
 *   max_gpus            cluster size N (1 .. TS_MAX_GPUS); degrees k > N are not used
 *   steps               remaining steps S, 0 <= S <= TS_MAX_STEPS
 *   budget_us           time left until the deadline (D - now); may be <= 0
 * Chooses n_k >= 0 with sum n_k = S and sum n_k T(k) <= budget_us minimising
 * the GPU time sum n_k k T(k); ties go to less total time, then to more steps
 * on smaller degrees (lexicographically from k = 1).  Writes the nonzero
 * (n_k, k) in increasing k to out[0 .. *n_out) (room for TS_MAX_ALLOCS), the
 * GPU time and the total time.  Returns TS_OK, or TS_INFEASIBLE when no split
 * meets the budget, in which case every step is placed on the fastest degree
 * (ties: the smaller k) and written the same way.  Exact (a Pareto dynamic
 * program over degrees and steps), not a heuristic.
 */
ts_status ts_allocate(const int64_t* step_us, int32_t n_degrees, int32_t max_gpus, int32_t steps, int64_t budget_us,
                      ts_alloc* out, int32_t* n_out, int64_t* gpu_time_us, int64_t* time_us);

/* A pending request at a round start. */
typedef struct {
  int64_t deadline_us;                /* absolute deadline D_i */
  int64_t step_us[TS_MAX_DEGREES];    /* cost-model row T_i(2^j), 0 = not profiled */
  int32_t n_allocs;                   /* allocations from ts_allocate, 0 .. TS_MAX_ALLOCS */
  ts_alloc allocs[TS_MAX_ALLOCS];     /* (s_i^m, A_i^m) */
} ts_request;

/* The decision for one request. */
typedef struct {
  int32_t option;      /* -1 = none, else the index m of the allocation that runs this round */
  int32_t gpus;        /* GPUs it occupies this round (w_i(o); 1 for a best-effort grant) */
  int32_t steps;       /* steps it completes this round: q_i^m = min(s_i^m, floor(tau / T_i(A_i^m))) */
  int32_t survives;    /* sv_i(o): next round start + (remaining steps) * T_i^min <= D_i */
  int32_t best_effort; /* 1: a request none of whose options survives, granted one leftover GPU */
} ts_decision;

/*
 * One round of request packing (Algorithm 1).
 *   reqs[n_req]   pending requests (n_req >= 0)
 *   n_gpus        N, 1 <= N <= TS_MAX_GPUS
 *   round_us      round length tau > 0; now_us the round start t_r
 *   out[n_req]    decisions, in request order
 *   survivors     number of requests with survives = 1 in the chosen plan
 *   gpus_used     GPUs occupied this round (best-effort grants included)
 * Options of request i: none, and every allocation m with q_i^m > 0 and
 * A_i^m <= N.  The DP keeps, for every capacity c, the best survivor count
 * (first option in the order none, m = 0, 1, ... on ties), and the plan is
 * read back from the smallest capacity reaching the maximum.  Requests none
 * of whose options survives are then granted one leftover GPU each (on one
 * GPU, min(remaining steps, floor(tau / T_i(1))) steps) in order of deadline,
 * ties by request index, while GPUs remain and T_i(1) fits the round.
 */
ts_status ts_round_schedule(const ts_request* reqs, int32_t n_req, int32_t n_gpus, int64_t round_us, int64_t now_us,
                            ts_decision* out, int32_t* survivors, int32_t* gpus_used);

/*
 * Selective continuous batching (sections 3 and 5: steps of identical
 * small-resolution requests are merged only when no deadline suffers).
 *   reqs[n_req]        pending requests of one resolution (same step shape)
 *   batch_us[max_b+1]  batch_us[b] = time of one step of b such requests
 *                      batched on one GPU (0 = not measured; batch_us[0]
 *                      unused); batch_us[1] is the unbatched step time
 *   round_us, now_us   round length tau > 0 and round start t_r
 *   members[n_req]     out: indices of the chosen requests, earliest deadline
 *                      first (ties: lower index); the first *b are the batch
 *   b                  out: batch size, 1 .. min(n_req, max_b) (0 if n_req = 0)
 * A request left alone on one GPU completes q_1 = floor(tau / batch_us[1])
 * steps this round, in a batch of b it completes q_b = floor(tau /
 * batch_us[b]).  It survives when t_r + tau + (remaining - min(remaining, q)) *
 * T_i^min <= D_i, T_i^min over its profiled degrees.  The batch is the
 * largest measured b whose b earliest-deadline requests each survive in the
 * batch whenever they would survive alone (and q_b > 0).
 * Remaining steps of a request: the sum of its allocations' steps.
 */
ts_status ts_select_batch(const ts_request* reqs, int32_t n_req, const int64_t* batch_us, int32_t max_b,
                          int64_t round_us, int64_t now_us, int32_t* members, int32_t* b);

#ifdef __cplusplus
}
#endif

#endif /* TETRI_SCHED_H */
