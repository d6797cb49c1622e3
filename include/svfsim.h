/*
 * svfsim.h -- C ABI of the MI355X batched scheduling simulator.
 *
 * What is simulated (Section 3.1 of "Geometry-Aware Online Scheduling for LLM
 * Serving", integer program eq:obj / eq:c1 / eq:c2 / eq:c3): an instance is a
 * set of n requests, request i arriving at step a_i with prompt size s_i and
 * output length o_i, served under a KV budget of M tokens.  Time is discrete;
 * a request started at step k holds s_i + (tau - k) tokens at every step
 * tau in [k+1, k+o_i] and finishes at k + o_i (latency k + o_i - a_i).
 * The scheduler decides every start: each step it admits waiting requests in
 * priority order (Alg. 1 / Alg. 2, Process 2) while the forward-looking
 * memory check passes (no future step may exceed M; Appendix E.2, proof of the
 * waiting-time lemma), and stops at the first one that does not fit.
 *
 * Priorities (Section 2.2): FCFS by arrival; SJF by believed length o^;
 * SVF by volume s*o^ + (o^^2 + o^)/2 (Eq. 1); 1-bit SVF by the same volume
 * with o^ = O_b for a long/short bit b (Eq. 2).  Ties go to the earlier
 * arrival, then the lower index.
 *
 * Many independent instances, and several policies over the same instances,
 * are advanced together on one GPU; every integer output matches the CPU
 * oracle exactly.
 *
 * Conventions
 *   - All arrays are structure-of-arrays, little-endian, CSR over instances.
 *   - Every function returns SVF_OK (0) or a negative SVF_E* code; the text of
 *     the last error of the calling thread is returned by svf_last_error().
 *   - A handle is not thread-safe; distinct handles are independent.
 *   - Work is enqueued on the HIP stream given at creation; functions marked
 *     "asynchronous" return before the GPU has finished.
 */
#ifndef SVFSIM_H
#define SVFSIM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SVFSIM_ABI_VERSION 1

/* Scheduling policies. */
enum {
    SVF_POLICY_FCFS = 0,    /* key a_i                                      */
    SVF_POLICY_SJF = 1,     /* key o^_i                                     */
    SVF_POLICY_SVF = 2,     /* key s_i o^_i + (o^_i^2 + o^_i)/2  (Eq. 1)     */
    SVF_POLICY_SVF1BIT = 3  /* the same with o^_i = b_i ? O1 : O0  (Eq. 2)   */
};

/* Admission rule, added to a policy number (e.g. SVF_POLICY_SVF |
 * SVF_ADMIT_CURRENT).  The default is the forward-looking check (no future
 * step over M, Appendix E.2).  SVF_ADMIT_CURRENT reads Alg. 1's Process 2
 * literally: the head is admitted while the memory of the next step, with the
 * head's first token, fits; growth beyond M later is resolved by evicting the
 * running request with the largest believed remaining volume. */
enum {
    SVF_ADMIT_LOOKAHEAD = 0,
    SVF_ADMIT_CURRENT = 0x100
};

/* Return codes. */
enum {
    SVF_OK = 0,
    SVF_EINVAL = -1,        /* bad argument or malformed input arrays        */
    SVF_ENOMEM = -2,        /* device or host allocation failed              */
    SVF_EHIP = -3,          /* a HIP runtime call failed                     */
    SVF_EINFEASIBLE = -4,   /* some s_i + max(o_i, o^_i) > M: never fits     */
    SVF_ESTATE = -5         /* call not allowed in the handle's state        */
};

/* Per-instance status reported by svf_stats. */
enum {
    SVF_STATUS_DONE = 0,      /* every request finished                       */
    SVF_STATUS_EXHAUSTED = 1, /* max_steps passed first                       */
    SVF_STATUS_RUNNING = 2    /* svf_step stopped before the end               */
};

typedef struct svf_batch svf_batch; /* opaque handle */

/*
 * Description of a batch.  Requests of instance i occupy indices
 * [req_offsets[i], req_offsets[i+1]) of every per-request array and are given
 * in arrival order (a nondecreasing inside an instance).
 *
 *   num_instances    >= 0
 *   req_offsets      host array [num_instances + 1], req_offsets[0] == 0,
 *                    nondecreasing; each instance holds < 2^31 requests
 *   arrival          a_i >= 0                                  int32 [N]
 *   prompt           s_i >= 1                                  int32 [N]
 *   output           o_i >= 1, the true length (drives completion)   int32 [N]
 *   plan_len         o^_i >= 1, the length the scheduler believes for SJF,
 *                    SVF and FCFS (keys and the memory check); NULL means the
 *                    true length is known (o^ = o)             int32 [N] or NULL
 *   long_bit         b_i in {0,1}; required iff SVF_POLICY_SVF1BIT is listed
 *                                                               int8 [N] or NULL
 *   M                KV budget in tokens, 1 <= M < 2^30
 *   num_policies     1..8 policies run side by side on the same instances
 *   policies         host array [num_policies] of SVF_POLICY_*, each optionally
 *                    plus SVF_ADMIT_CURRENT
 *   O0, O1           1-bit proxy lengths (>= 1 when SVF1BIT is listed)
 *   max_steps        stop an instance after step max_steps (0 <= max_steps
 *                    < 2^30); such instances report SVF_STATUS_EXHAUSTED
 *   inputs_on_device 0: the per-request arrays are host memory and are copied
 *                    at creation (the caller keeps ownership); 1: they are
 *                    device memory on the current device and are only read
 *                    during svf_create (copied into the handle's own buffers)
 *
 * The packed priority key (key << 32 | index) must fit: every key < 2^32.
 * Memory totals are kept in 32 bits: M + max_steps + 2 * (longest planned
 * length rounded up to a power of two) < 2^31, where under SVF_ADMIT_CURRENT
 * an instance's sum of s_i + o^_i takes M's place when larger.
 */
typedef struct svf_batch_desc {
    int32_t num_instances;
    const int64_t *req_offsets;
    const int32_t *arrival;
    const int32_t *prompt;
    const int32_t *output;
    const int32_t *plan_len;
    const int8_t *long_bit;
    int64_t M;
    int32_t num_policies;
    const int32_t *policies;
    int32_t O0, O1;
    int64_t max_steps;
    int32_t inputs_on_device;
} svf_batch_desc;

/* Per-instance results of one policy slot. */
typedef struct svf_instance_stats {
    int32_t makespan;       /* largest finish step (0 if none finished)       */
    int32_t status;         /* SVF_STATUS_*                                   */
    int64_t sum_latency;    /* sum over finished requests of finish - a       */
    int64_t request_steps;  /* sum over steps of the number of running
                               requests (sum o_i without preemption)          */
    int64_t peak_mem;       /* largest total memory held at any step          */
    int64_t preemptions;    /* evictions (only when o^ differs from o)        */
    int64_t t_end;          /* next step to simulate (simulated time reached) */
} svf_instance_stats;

/* Timing of the kernels enqueued by the last svf_reset / svf_step / svf_run
 * calls since profiling was enabled, measured with HIP events on the handle's
 * stream (milliseconds, summed over launches). */
typedef struct svf_timing {
    double init_ms;     /* state reset, priority keys and their sort         */
    double sim_ms;      /* the simulation kernel                             */
    double final_ms;    /* output finalisation and per-instance statistics   */
    int64_t sim_launches;
} svf_timing;

/*
 * Build a batch of instances.  An instance is the problem of Section 3.1:
 * requests (a_i, s_i, o_i) and a budget M, with the start steps as the
 * decisions of the integer program (the x_{i,t} of eq:c1) and the policy's
 * order of Section 2.2 (Eq. 1, Eq. 2, SJF, FCFS).
 *
 * Validate ``desc`` on the host and build a handle: allocates the device
 * buffers and copies the inputs (host-to-device, or device-to-device when
 * inputs_on_device).  ``hip_stream`` is a hipStream_t (NULL: the null stream)
 * on which every later call enqueues its work.  No simulation work runs yet.
 * Errors: SVF_EINVAL (malformed arrays, NULL pointers, unknown policy,
 * arrivals out of order, key overflow), SVF_EINFEASIBLE (a request that can
 * never fit), SVF_ENOMEM, SVF_EHIP.  Validation happens before any HIP call.
 */
int svf_create(const svf_batch_desc *desc, void *hip_stream, svf_batch **out);

/*
 * Process 1 of Alg. 1 / Alg. 2 (every request's priority from its prompt and
 * believed length: the volume of Eq. 1, its 1-bit form Eq. 2, or the SJF and
 * FCFS keys), for all requests up front.
 *
 * Asynchronous.  Restart every instance and policy slot at step 0: computes
 * the priority keys (Eq. 1 / Eq. 2), sorts each instance's requests by
 * (key, arrival, index) and clears the per-instance state.
 */
int svf_reset(svf_batch *h);

/*
 * The discrete decode steps of Section 3.1 (one token per running request
 * per step, constraint eq:c2 on the memory of every step), each one pass of
 * the scheduling loop of Alg. 1 / Alg. 2, Process 2: arrivals, completions,
 * eviction on overflow, strict head-of-line admission under the
 * forward-looking check, advance.
 *
 * Asynchronous.  Advance every unfinished instance by ``nsteps`` simulated
 * steps (nsteps >= 0), or until it finishes or passes max_steps.  Calls
 * svf_reset first if the handle was never reset.  State stays on the GPU
 * between calls, so k calls of svf_step(1) equal one svf_run.
 */
int svf_step(svf_batch *h, int64_t nsteps);

/*
 * The same loop (Alg. 1 / Alg. 2, Process 2, over the steps of Section 3.1)
 * until every request has finished: the schedule whose total latency is the
 * objective eq:obj.
 *
 * Asynchronous.  Run every instance from its current step to completion (or
 * max_steps).  Calls svf_reset first if the handle was never reset.
 */
int svf_run(svf_batch *h);

/*
 * The decisions and their outcome per request (Section 3.1): the start step
 * k_i chosen by the scheduler and the finish k_i + o_i whose difference to
 * a_i is the request's latency in the objective eq:obj.
 *
 * Copy the per-request results of policy slot ``policy_slot`` (an index into
 * desc.policies) into caller buffers of N int32 each, for the state reached so
 * far (synchronises the stream when outputs_on_device == 0):
 *   start      step of the request's current run (-1 while waiting)
 *   finish     completion step (-1 until it has completed)
 *   preempt    number of evictions suffered
 *   admit_seq  position of its last admission in its instance (-1 if none)
 * Any pointer may be NULL to skip that array.  outputs_on_device == 1: the
 * buffers are device memory and the copy is enqueued on the stream.
 * Errors: SVF_EINVAL (slot out of range), SVF_ESTATE (never reset).
 */
int svf_read(svf_batch *h, int32_t policy_slot, int32_t *start, int32_t *finish,
             int32_t *preempt, int32_t *admit_seq, int32_t outputs_on_device);

/*
 * Per-instance aggregates of the schedule: the total latency of eq:obj
 * (sum of finish - a_i, exact in 64 bits), the largest memory of any step
 * (at most M by eq:c2), request-steps (running requests summed over steps,
 * one token each per step), the makespan (duration behind the throughput of
 * Section 4.1) and the eviction count.
 *
 * Copy per-instance statistics of policy slot ``policy_slot`` into ``out``
 * (host array [num_instances]); synchronises the stream.  Errors: SVF_EINVAL
 * (slot out of range, NULL ``out``), SVF_ESTATE (never reset), SVF_EHIP.
 */
int svf_stats(svf_batch *h, int32_t policy_slot, svf_instance_stats *out);

/* Enable (1) or disable (0) kernel timing with HIP events, and clear it. */
int svf_set_profiling(svf_batch *h, int32_t enable);

/* Read the accumulated kernel timing (synchronises the stream). */
int svf_timings(svf_batch *h, svf_timing *out);

/* Sizes of the batch: requests N, instances, policy slots. */
int svf_shape(const svf_batch *h, int64_t *num_requests, int32_t *num_instances,
              int32_t *num_policies);

/* Release the handle and its device buffers (synchronises the stream).
 * Passing NULL is allowed and does nothing. */
int svf_destroy(svf_batch *h);

/*
 * Limits of svf_run_noalloc: its device scratch per GPU (bytes), and the
 * largest number of instances of one call.
 */
#define SVF_NOALLOC_SCRATCH_BYTES (128u << 20)
#define SVF_NOALLOC_MAX_INSTANCES 65536

/*
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The same
 * computation as svf_create + svf_run + svf_read / svf_stats of every policy
 * slot, with every intermediate buffer (inputs staged on the device, priority
 * records, rank bitmaps, memory profiles, running lists, per-segment state)
 * carved from one static device array of SVF_NOALLOC_SCRATCH_BYTES per GPU,
 * which the library holds until the process ends.  Calls no hipMalloc or
 * hipFree and allocates no host memory.
 *
 *   desc       as for svf_create; the per-request arrays must be host memory
 *              (inputs_on_device == 0), each instance must hold at most 8192
 *              requests and num_instances <= SVF_NOALLOC_MAX_INSTANCES
 *   hip_stream hipStream_t (NULL: the null stream) the work is enqueued on
 *   start, finish, preempt, admit_seq
 *              caller-owned device arrays of num_policies * N int32 each,
 *              policy-slot major (slot p at [p * N, (p + 1) * N)), with the
 *              meaning of svf_read's outputs after a run to completion
 *   stats      caller-owned device array of num_policies * num_instances
 *              svf_instance_stats, policy-slot major
 *
 * The inputs are copied into the scratch and the stream is synchronised
 * before the call returns (the caller may then reuse its host arrays); the
 * simulation and the outputs are asynchronous on ``hip_stream``.
 *
 * Every call on one GPU uses that GPU's single scratch array: calls that
 * overlap on one GPU (on different streams, or from several threads) race
 * and give undefined results; calls on one stream are ordered and safe.
 * Each call clears and rebuilds everything it reads from the scratch.
 *
 * Errors: those of svf_create, and SVF_EINVAL when the batch needs more
 * scratch than SVF_NOALLOC_SCRATCH_BYTES (the message gives both sizes),
 * has an instance of more than 8192 requests or more than
 * SVF_NOALLOC_MAX_INSTANCES instances, passes device inputs, or a NULL
 * output for a non-empty batch.
 */
int svf_run_noalloc(const svf_batch_desc *desc, void *hip_stream, int32_t *start,
                    int32_t *finish, int32_t *preempt, int32_t *admit_seq,
                    svf_instance_stats *stats);

/* Message of the calling thread's last non-zero return ("" if none). */
const char *svf_last_error(void);

/* SVFSIM_ABI_VERSION of the built library. */
int svf_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SVFSIM_H */
