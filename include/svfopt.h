/*
 * svfopt.h -- exact offline optimum of tiny burst instances (host code).
 *
 * Part of libsvfsim.so.  Used to measure competitive ratios: the total
 * latency of the integer program of Section 3.1 (objective eq:obj under
 * eq:c1 - eq:c3) for instances whose requests all arrive at step 0, next to
 * the bound 1 + 2/(1 - alpha) of Theorem thm:svf-burst (Table tab:alpha-cr).
 *
 * The optimum may start any set of waiting requests at any step as long as
 * the memory of every future step stays <= M (a request started at k holds
 * s + (tau - k) at tau in [k+1, k+o]); it may also wait while something
 * runs.  It is computed by dynamic programming over the state (requests not
 * started, running requests and their progress), with identical requests
 * merged; the cost of a step is the number of unfinished requests.
 *
 * Return codes are those of svfsim.h, plus SVF_ELIMIT.
 */
#ifndef SVFOPT_H
#define SVFOPT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* The search visited more states than allowed. */
#define SVF_ELIMIT (-6)

/*
 * Optimal total latency sum_i (k_i + o_i) of one burst instance.
 *   n             number of requests, 0 <= n <= 16
 *   prompt        s_i >= 1                                   host int32 [n]
 *   output        o_i >= 1, o_i <= 16                        host int32 [n]
 *   M             budget, s_i + o_i <= M for every i (SVF_EINFEASIBLE if not)
 *   state_limit   largest number of distinct states to store (<= 0: 2^26)
 *   total_latency result                                     host int64 [1]
 *   states        number of states stored (may be NULL)      host int64 [1]
 * Errors: SVF_EINVAL (bad sizes or NULL pointers), SVF_EINFEASIBLE,
 * SVF_ELIMIT (state_limit reached; *total_latency is then undefined),
 * SVF_ENOMEM.  Thread-safe.
 */
int svf_opt_burst(int32_t n, const int32_t *prompt, const int32_t *output, int64_t M,
                  int64_t state_limit, int64_t *total_latency, int64_t *states);

/*
 * The same for num_instances instances in CSR form (req_offsets [num + 1]),
 * each with its own budget M[i], solved on ``threads`` host threads
 * (<= 0: all hardware threads).  total_latency[i] and states[i] receive the
 * results; status[i] the return code of instance i.  Returns SVF_OK when
 * every instance succeeded, else the first failing instance's code.
 */
int svf_opt_burst_batch(int32_t num_instances, const int64_t *req_offsets,
                        const int32_t *prompt, const int32_t *output, const int64_t *M,
                        int64_t state_limit, int32_t threads, int64_t *total_latency,
                        int64_t *states, int32_t *status);

#ifdef __cplusplus
}
#endif

#endif /* SVFOPT_H */
