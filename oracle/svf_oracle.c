/*
 * svf_oracle.c -- plain CPU reference for the batched, discrete-time simulation
 * of memory-constrained online LLM-serving scheduling (SVF, 1-bit SVF, SJF,
 * FCFS) from "Geometry-Aware Online Scheduling for LLM Serving".
 *
 * TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load this file's library.  It shares no
 * code with the GPU path and it is deliberately slow and literal: every step of
 * every instance is simulated, the waiting queue is an unsorted array scanned
 * for its minimum, and every memory total is summed afresh over the active set.
 *
 * Model (Section 3.1, integer program eq:obj / eq:c1 / eq:c2):
 *   - time is discrete; one decode step produces one token per active request;
 *   - a request i started at step k occupies s_i + (tau - k) memory units at
 *     every step tau in [k+1, k+o_i] (constraint eq:c2) and nothing at step k;
 *     its latency is k + o_i - a_i (objective eq:obj);
 *   - the total over all active requests must stay <= M at every step.
 *
 * Per step t, in this order (readings of the paper recorded in the design
 * notes; the paper leaves the intra-step order open):
 *   1. arrivals:    requests with a_i = t join the waiting set W;
 *   2. completions: active i with t - k_i = o_i leave, finish_i = t;
 *   3. overflow:    only possible when the scheduler plans with lengths other
 *                   than the true ones.  While the true memory of the next step
 *                   exceeds M, evict the active request with the largest
 *                   believed remaining volume (ties: latest arrival).  The
 *                   victim loses its progress (KV eviction and recompute,
 *                   Section 1) and is eligible again from step t+1;
 *   4. admission:   repeatedly take the highest-priority eligible waiting
 *                   request h (Alg. 1/Alg. 2, Process 2) and start it at t if
 *                   the forward-looking memory check passes (Appendix E.2, proof
 *                   of the waiting-time lemma: no future step may exceed M);
 *                   otherwise stop (strict head of line, no backfilling);
 *   5. advance:     request_steps += |A|, peak = max(peak, memory at t+1).
 *
 * Admission rule.  The default is the forward-looking check above.  The
 * alternative "current capacity" rule reads Alg. 1's Process 2 literally (pop
 * the head while the KV cache has room): h is admitted iff the memory of the
 * next step, sum_{i in A} (s_i + t+1 - k_i) + (s_h + 1), stays <= M; later
 * growth beyond M is then resolved by step 3's eviction.  A policy code selects
 * it by adding RULE_CURRENT (0x100) to the policy number.
 *
 * Priority keys (lower first; ties by arrival then index):
 *   FCFS      a_i
 *   SJF       o^_i
 *   SVF       s_i*o^_i + (o^_i^2 + o^_i)/2          (Section 2.2, Eq. 1)
 *   1-bit SVF the same with o^_i = O_{b_i}          (Section 2.2, Eq. 2)
 * where o^ is the length the scheduler believes (o itself when known).
 *
 * Forward-looking check.  With F_i = k_i + max(o^_i, t - k_i + 1) (an active
 * request that has outlived its planned length is planned to finish next
 * step), h started at t fits iff for every future step tau
 *     sum_{i in A u {h}, k_i < tau <= F_i} (s_i + tau - k_i) <= M.
 * Between consecutive planned finishes every term grows by one per step, so the
 * total can only peak at a planned finish; and beyond F_h the active set alone
 * is already feasible (it passed the same test when its last member was
 * admitted, and step 3 guarantees step t+1).  The check below therefore sums
 * at tau in {F_i <= F_h} u {F_h}; the pure-Python literal oracle evaluates
 * every tau and the tests require both to agree.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <pthread.h>

#define POL_FCFS 0
#define POL_SJF 1
#define POL_SVF 2
#define POL_SVF1BIT 3
#define RULE_CURRENT 0x100

#define NSTATS 8
/* stats layout per instance: makespan, status, sum_latency, request_steps,
 * peak_mem, preemptions, t_end, n_finished */

typedef struct {
    int32_t n;
    const int32_t *a, *s, *o, *plan; /* plan may be NULL */
    const int8_t *bit;               /* may be NULL */
    int64_t M;
    int32_t policy, rule, O0, O1;
    int64_t max_steps, t_stop;
    int32_t *start, *finish, *preempt, *admit_seq;
    int64_t *stats;
} inst_job;

/* Section 2.2, Eq. 1: the memory-time volume of a request. */
int64_t oracle_volume(int64_t s, int64_t o) { return s * o + (o * o + o) / 2; }

static int64_t believed_len(const inst_job *J, int32_t i) {
    if (J->policy == POL_SVF1BIT) return J->bit[i] ? J->O1 : J->O0;
    if (J->plan) return J->plan[i];
    return J->o[i];
}

int64_t oracle_key(int32_t policy, int64_t a, int64_t s, int64_t ohat) {
    switch (policy) {
    case POL_FCFS: return a;
    case POL_SJF: return ohat;
    default: return oracle_volume(s, ohat); /* SVF and 1-bit SVF */
    }
}

/* (key, arrival, index) lexicographic order */
static int precedes(const int64_t *key, const int32_t *a, int32_t i, int32_t j) {
    if (key[i] != key[j]) return key[i] < key[j];
    if (a[i] != a[j]) return a[i] < a[j];
    return i < j;
}

static void simulate(inst_job *J) {
    const int32_t n = J->n;
    const int32_t *a = J->a, *s = J->s, *o = J->o;
    const int64_t M = J->M;
    int64_t *key = (int64_t *)malloc(sizeof(int64_t) * (n ? n : 1));
    int64_t *ohat = (int64_t *)malloc(sizeof(int64_t) * (n ? n : 1));
    int32_t *W = (int32_t *)malloc(sizeof(int32_t) * (n ? n : 1));
    int32_t *A = (int32_t *)malloc(sizeof(int32_t) * (n ? n : 1));
    int32_t *evicted = (int32_t *)malloc(sizeof(int32_t) * (n ? n : 1));
    int64_t *k = (int64_t *)malloc(sizeof(int64_t) * (n ? n : 1));
    int32_t nW = 0, nA = 0, cursor = 0, nfin = 0;
    int64_t t = 0, seq = 0, peak = 0, req_steps = 0, status = 0;

    for (int32_t i = 0; i < n; ++i) {
        ohat[i] = believed_len(J, i);
        key[i] = oracle_key(J->policy, a[i], s[i], ohat[i]);
        k[i] = -1;
        J->start[i] = -1;
        J->finish[i] = -1;
        J->preempt[i] = 0;
        J->admit_seq[i] = -1;
    }

    for (;;) {
        if (nfin == n) { status = 0; break; }
        if (t > J->max_steps) { status = 1; break; }
        if (t >= J->t_stop) { status = 2; break; }

        /* 1. arrivals */
        while (cursor < n && a[cursor] == t) W[nW++] = cursor++;

        /* 2. completions: true length reached */
        for (int32_t x = 0; x < nA;) {
            int32_t i = A[x];
            if (t - k[i] == o[i]) {
                J->finish[i] = (int32_t)t;
                ++nfin;
                A[x] = A[--nA];
            } else {
                ++x;
            }
        }

        /* 3. overflow of the next step's true memory */
        int32_t nev = 0;
        for (;;) {
            int64_t mem_next = 0;
            for (int32_t x = 0; x < nA; ++x) {
                int32_t i = A[x];
                mem_next += s[i] + (t + 1) - k[i];
            }
            if (mem_next <= M) break;
            int32_t best = -1;
            int64_t bestR = -1;
            for (int32_t x = 0; x < nA; ++x) {
                int32_t i = A[x];
                int64_t e = t - k[i];
                int64_t L = ohat[i] > e + 1 ? ohat[i] : e + 1;
                int64_t R = 0;
                for (int64_t y = e + 1; y <= L; ++y) R += s[i] + y;
                /* largest remaining volume; ties go to the latest arrival */
                if (best < 0 || R > bestR ||
                    (R == bestR && (a[i] > a[best] || (a[i] == a[best] && i > best)))) {
                    best = i;
                    bestR = R;
                }
            }
            for (int32_t x = 0; x < nA; ++x)
                if (A[x] == best) { A[x] = A[--nA]; break; }
            J->preempt[best] += 1;
            k[best] = -1;
            J->start[best] = -1;     /* waiting again: no current run */
            J->admit_seq[best] = -1;
            evicted[nev++] = best;
        }

        /* 4. admission, strict head of line */
        for (;;) {
            int32_t hx = -1;
            for (int32_t x = 0; x < nW; ++x)
                if (hx < 0 || precedes(key, a, W[x], W[hx])) hx = x;
            if (hx < 0) break;
            int32_t h = W[hx];
            int64_t Fh = t + ohat[h];
            int feasible = 1;
            if (J->rule == RULE_CURRENT) {
                /* memory of the next step only */
                int64_t mem_next = s[h] + 1;
                for (int32_t x = 0; x < nA; ++x) {
                    int32_t j = A[x];
                    mem_next += s[j] + (t + 1) - k[j];
                }
                if (mem_next > M) break;
                k[h] = t;
                J->start[h] = (int32_t)t;
                J->admit_seq[h] = (int32_t)seq++;
                A[nA++] = h;
                W[hx] = W[--nW];
                continue;
            }
            /* checkpoints: every planned finish of an active request up to F_h,
             * and F_h itself */
            for (int32_t c = -1; c < nA && feasible; ++c) {
                int64_t tau;
                if (c < 0) {
                    tau = Fh;
                } else {
                    int32_t i = A[c];
                    int64_t e = t - k[i];
                    int64_t L = ohat[i] > e + 1 ? ohat[i] : e + 1;
                    tau = k[i] + L;
                    if (tau > Fh) continue;
                }
                int64_t mem = s[h] + (tau - t);
                for (int32_t x = 0; x < nA; ++x) {
                    int32_t j = A[x];
                    int64_t e = t - k[j];
                    int64_t L = ohat[j] > e + 1 ? ohat[j] : e + 1;
                    int64_t Fj = k[j] + L;
                    if (tau <= Fj) mem += s[j] + (tau - k[j]);
                }
                if (mem > M) feasible = 0;
            }
            if (!feasible) break;
            k[h] = t;
            J->start[h] = (int32_t)t;
            J->admit_seq[h] = (int32_t)seq++;
            A[nA++] = h;
            W[hx] = W[--nW];
        }

        /* evicted requests may compete again from the next step */
        for (int32_t x = 0; x < nev; ++x) W[nW++] = evicted[x];

        /* 5. advance */
        req_steps += nA;
        int64_t mem = 0;
        for (int32_t x = 0; x < nA; ++x) {
            int32_t i = A[x];
            mem += s[i] + (t + 1) - k[i];
        }
        if (mem > peak) peak = mem;
        ++t;
    }

    int64_t makespan = 0, sum_lat = 0, pre = 0, nf = 0;
    for (int32_t i = 0; i < n; ++i) {
        if (J->finish[i] >= 0) {
            if (J->finish[i] > makespan) makespan = J->finish[i];
            sum_lat += (int64_t)J->finish[i] - a[i];
            ++nf;
        }
        pre += J->preempt[i];
    }
    int64_t *st = J->stats;
    st[0] = makespan;
    st[1] = status;
    st[2] = sum_lat;
    st[3] = req_steps;
    st[4] = peak;
    st[5] = pre;
    st[6] = t;
    st[7] = nf;

    free(key); free(ohat); free(W); free(A); free(evicted); free(k);
}

typedef struct {
    inst_job *jobs;
    int32_t count, stride, first;
} worker_arg;

static void *worker(void *p) {
    worker_arg *w = (worker_arg *)p;
    for (int32_t j = w->first; j < w->count; j += w->stride) simulate(&w->jobs[j]);
    return NULL;
}

/*
 * Simulate every instance of a batch under one policy (policy number, plus
 * RULE_CURRENT for the current-capacity admission rule).
 *   offsets[num_instances+1]: CSR offsets into the per-request arrays
 *   plan, bit: may be NULL (plan NULL => believed length = true length)
 *   t_stop: stop before processing step t_stop (status 2), or a huge value
 *   threads: worker threads (instances are independent)
 *   outputs: start, finish, preempt, admit_seq [N]; stats [num_instances*8]
 * Returns 0.
 */
int oracle_run(int32_t num_instances, const int64_t *offsets, const int32_t *a,
               const int32_t *s, const int32_t *o, const int32_t *plan,
               const int8_t *bit, int64_t M, int32_t policy, int32_t O0, int32_t O1,
               int64_t max_steps, int64_t t_stop, int32_t threads, int32_t *start,
               int32_t *finish, int32_t *preempt, int32_t *admit_seq, int64_t *stats) {
    inst_job *jobs = (inst_job *)calloc(num_instances ? num_instances : 1, sizeof(inst_job));
    for (int32_t i = 0; i < num_instances; ++i) {
        int64_t lo = offsets[i], hi = offsets[i + 1];
        inst_job *J = &jobs[i];
        J->n = (int32_t)(hi - lo);
        J->a = a + lo; J->s = s + lo; J->o = o + lo;
        J->plan = plan ? plan + lo : NULL;
        J->bit = bit ? bit + lo : NULL;
        J->M = M; J->policy = policy & 0xFF; J->rule = policy & RULE_CURRENT;
        J->O0 = O0; J->O1 = O1;
        J->max_steps = max_steps; J->t_stop = t_stop;
        J->start = start + lo; J->finish = finish + lo;
        J->preempt = preempt + lo; J->admit_seq = admit_seq + lo;
        J->stats = stats + (int64_t)NSTATS * i;
    }
    if (threads < 1) threads = 1;
    if (threads > num_instances) threads = num_instances > 0 ? num_instances : 1;
    if (threads == 1) {
        for (int32_t i = 0; i < num_instances; ++i) simulate(&jobs[i]);
    } else {
        pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * threads);
        worker_arg *wa = (worker_arg *)malloc(sizeof(worker_arg) * threads);
        for (int32_t w = 0; w < threads; ++w) {
            wa[w].jobs = jobs; wa[w].count = num_instances; wa[w].stride = threads; wa[w].first = w;
            pthread_create(&th[w], NULL, worker, &wa[w]);
        }
        for (int32_t w = 0; w < threads; ++w) pthread_join(th[w], NULL);
        free(th); free(wa);
    }
    free(jobs);
    return 0;
}
