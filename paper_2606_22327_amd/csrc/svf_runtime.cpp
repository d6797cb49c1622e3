// svf_runtime.cpp -- host side of the C ABI declared in include/svfsim.h:
// validation, buffer ownership, launch configuration, timing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <vector>

#include "svf_kernels.h"
#include "svfsim.h"

using svfk::SegState;
using svfk::StatsOut;

static_assert(sizeof(StatsOut) == sizeof(svf_instance_stats), "stats layout");
static_assert(sizeof(SegState) == 80, "state layout");

namespace {

// message of the calling thread's last failure (a fixed buffer: no call
// allocates host memory for it)
thread_local char g_err[512];

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

int ok() { return SVF_OK; }

constexpr int64_t kLimit30 = int64_t(1) << 30;

int64_t next_pow2(int64_t x) {
    int64_t p = 1;
    while (p < x) p <<= 1;
    return p;
}

struct Timed {
    int kind;  // 0 init, 1 sim, 2 final
    hipEvent_t a, b;
};

}  // namespace

struct svf_batch {
    hipStream_t stream = nullptr;
    // Second stream (default priority) on which the per-step segments run
    // concurrently with the event-driven ones, forked from and joined back
    // into ``stream`` with events; null: both launches on ``stream``.
    hipStream_t aux = nullptr;
    hipEvent_t fork_ev = nullptr, join_ev = nullptr;
    int device = 0;
    int32_t I = 0, P = 0;
    int64_t N = 0;
    int32_t M = 0, O0 = 0, O1 = 0, max_steps = 0;
    std::vector<int32_t> policies;
    std::vector<int64_t> offsets;
    int32_t H = 1, CH = 64, nchunks = 0, bw_max = 0, max_n = 0;
    bool fused_sort = false;  // every instance fits one workgroup of k_sort_rec
    bool list_known = false;  // event path: profile as the finish-ordered list
    bool ring_used = true;    // some segment keeps its profile in the ring
    int32_t list_stride = 0;  // list entries per segment in HBM (the bound)
    int32_t list_cap = 0;     // list entries per segment in LDS (first launch)
    size_t lds_list = 0;      // LDS of the event kernel with the list
    size_t lds_list_full = 0; //   and with room for the bound (continuation)
    bool list_stepped = false; // per-step path: profile as the finish-ordered list
    int32_t step_cap = 0;      // its entries in LDS (first launch)
    size_t lds_step = 0;       // LDS of the per-step kernel with the list
    size_t lds_step_full = 0;  //   and with room for the bound (continuation)
    int32_t res_known = 0;     // workgroups resident at once: first event launch
    int32_t res_stepped = 0;   //   and first per-step launch (0: no issue priorities)
    int32_t kbits[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    int64_t bw_total = 0;
    bool d_lds = true;
    size_t lds_bytes = 0;
    bool any_stepped = false;
    int64_t n_known = 0, n_stepped = 0;
    bool was_reset = false, dirty = false;
    bool prof = false;
    std::vector<Timed> timed;
    double acc_ms[3] = {0, 0, 0};
    int64_t sim_launches = 0;

    // device buffers
    int64_t* d_off = nullptr;
    int32_t *d_a = nullptr, *d_s = nullptr, *d_o = nullptr, *d_plan = nullptr;
    int8_t* d_bit = nullptr;
    int32_t* d_pol = nullptr;
    int32_t *d_chunk_seg = nullptr, *d_chunk_lo = nullptr;
    uint64_t *d_keys0 = nullptr, *d_keys1 = nullptr;
    int4* d_rec = nullptr;
    int32_t* d_rank = nullptr;
    uint8_t* d_stepped = nullptr;
    int64_t* d_bw_off = nullptr;
    uint64_t* d_bitmap = nullptr;
    int32_t* d_ring = nullptr;
    int32_t *d_start = nullptr, *d_fin = nullptr, *d_pre = nullptr, *d_seq = nullptr;
    int4* d_act = nullptr;
    int2* d_actkr = nullptr;
    int32_t* d_evl = nullptr;
    SegState* d_st = nullptr;
    int32_t* d_fin_out = nullptr;
    StatsOut* d_stats = nullptr;
    int32_t* d_lst_f = nullptr;
    uint32_t* d_lst_q = nullptr;
    unsigned long long* d_prog = nullptr;  // [2] progress counters of the simulation launches
    const uint64_t* sorted_keys = nullptr;  // which key buffer holds the final order
};

namespace {

template <typename T>
int dalloc(T** p, int64_t count) {
    *p = nullptr;
    if (count <= 0) return SVF_OK;
    hipError_t e = hipMalloc((void**)p, sizeof(T) * (size_t)count);
    if (e != hipSuccess) {
        *p = nullptr;
        return fail(SVF_ENOMEM, "hipMalloc of %lld bytes failed: %s",
                    (long long)(sizeof(T) * count), hipGetErrorString(e));
    }
    return SVF_OK;
}

void free_all(svf_batch* h) {
    void* ptrs[] = {h->d_off, h->d_a, h->d_s, h->d_o, h->d_plan, h->d_bit, h->d_pol,
                    h->d_chunk_seg, h->d_chunk_lo, h->d_keys0, h->d_keys1, h->d_rec,
                    h->d_rank, h->d_stepped, h->d_bw_off, h->d_bitmap, h->d_ring,
                    h->d_start, h->d_fin, h->d_pre, h->d_seq, h->d_act, h->d_actkr, h->d_evl,
                    h->d_st, h->d_fin_out, h->d_stats, h->d_lst_f, h->d_lst_q, h->d_prog};
    for (void* p : ptrs)
        if (p) (void)hipFree(p);
    for (auto& t : h->timed) {
        (void)hipEventDestroy(t.a);
        (void)hipEventDestroy(t.b);
    }
    h->timed.clear();
    if (h->fork_ev) (void)hipEventDestroy(h->fork_ev);
    if (h->join_ev) (void)hipEventDestroy(h->join_ev);
    if (h->aux) (void)hipStreamDestroy(h->aux);
    h->fork_ev = h->join_ev = nullptr;
    h->aux = nullptr;
}

#define HIPCHK(expr)                                                                  \
    do {                                                                              \
        hipError_t e_ = (expr);                                                       \
        if (e_ != hipSuccess)                                                         \
            return fail(SVF_EHIP, "%s failed: %s", #expr, hipGetErrorString(e_));     \
    } while (0)

#define RETCHK(expr)              \
    do {                          \
        int r_ = (expr);          \
        if (r_ != SVF_OK) return r_; \
    } while (0)

struct HostView {
    const int32_t *a, *s, *o, *plan;
    const int8_t* bit;
};

// Largest number of requests of one instance that can run at the same time.
// A running request holds at least s + 1 tokens at the next step, and the
// planned (and true) total of that step stays <= M once a step's admissions
// are done, so at most the k smallest values of s + 1 fit.  Values at or
// above kCap count as kCap (a lower bound on each), which keeps k an upper
// bound.
int64_t running_bound(const int32_t* s, const int64_t* off, int32_t I, int64_t M) {
    constexpr int kCap = 4096;
    int64_t h[kCap + 1];
    int64_t best = 0;
    for (int32_t i = 0; i < I; ++i) {
        std::fill(h, h + kCap + 1, 0);
        for (int64_t j = off[i]; j < off[i + 1]; ++j)
            h[std::min<int64_t>((int64_t)s[j] + 1, kCap)] += 1;
        int64_t sum = 0, k = 0;
        for (int v = 1; v <= kCap; ++v) {
            if (!h[v]) continue;
            const int64_t take = std::min<int64_t>(h[v], (M - sum) / v);
            k += take;
            sum += take * v;
            if (take < h[v]) break;
        }
        best = std::max(best, k);
    }
    return best;
}

// Everything that can be checked without a GPU.  Writes each segment's path
// (1: per-step) to stepped[P*I] and each policy's largest key to max_key[P].
int validate(const svf_batch_desc* d, const HostView& v, const int64_t* off, int64_t N,
             uint8_t* stepped, int64_t* max_plan, int64_t* max_profile, uint64_t* max_key) {
    const int32_t I = d->num_instances, P = d->num_policies;
    bool has1bit = false;
    for (int p = 0; p < P; ++p) has1bit |= (d->policies[p] & 0xFF) == SVF_POLICY_SVF1BIT;
    if (N > 0 && (!v.a || !v.s || !v.o))
        return fail(SVF_EINVAL, "arrival, prompt and output must not be NULL");
    if (has1bit && N > 0 && !v.bit) return fail(SVF_EINVAL, "SVF1BIT needs long_bit");
    if (has1bit && (d->O0 < 1 || d->O1 < 1)) return fail(SVF_EINVAL, "SVF1BIT needs O0, O1 >= 1");
    *max_plan = 1;
    // Largest planned memory total at one future step.  The forward-looking
    // check keeps it <= M; with next-step admission only, the requests of an
    // instance bound it together: sum of s + o^.
    *max_profile = d->M;
    std::fill(stepped, stepped + (size_t)P * I, 0);
    std::fill(max_key, max_key + P, 0);
    int64_t cur_total[8];
    for (int32_t i = 0; i < I; ++i) {
        const int64_t lo = off[i], hi = off[i + 1];
        std::fill(cur_total, cur_total + P, 0);
        for (int64_t j = lo; j < hi; ++j) {
            const int32_t a = v.a[j], s = v.s[j], o = v.o[j];
            if (a < 0 || a >= kLimit30)
                return fail(SVF_EINVAL, "instance %d request %lld: arrival %d out of [0, 2^30)", i,
                            (long long)(j - lo), a);
            if (j > lo && a < v.a[j - 1])
                return fail(SVF_EINVAL, "instance %d: arrivals not in order at request %lld", i,
                            (long long)(j - lo));
            if (s < 1) return fail(SVF_EINVAL, "instance %d request %lld: prompt %d < 1", i, (long long)(j - lo), s);
            if (o < 1) return fail(SVF_EINVAL, "instance %d request %lld: output %d < 1", i, (long long)(j - lo), o);
            if (v.plan && v.plan[j] < 1)
                return fail(SVF_EINVAL, "instance %d request %lld: plan_len %d < 1", i, (long long)(j - lo), v.plan[j]);
            if (v.bit && v.bit[j] != 0 && v.bit[j] != 1)
                return fail(SVF_EINVAL, "instance %d request %lld: long_bit %d not 0/1", i, (long long)(j - lo), v.bit[j]);
            for (int p = 0; p < P; ++p) {
                const int pol = d->policies[p] & 0xFF;
                const bool current_rule = (d->policies[p] & SVF_ADMIT_CURRENT) != 0;
                int64_t oh;
                if (pol == SVF_POLICY_SVF1BIT) oh = v.bit[j] ? d->O1 : d->O0;
                else oh = v.plan ? v.plan[j] : o;
                if ((int64_t)s + std::max<int64_t>(o, oh) > d->M)
                    return fail(SVF_EINFEASIBLE,
                                "instance %d request %lld: s + max(o, planned) = %lld exceeds M = %lld",
                                i, (long long)(j - lo), (long long)s + std::max<int64_t>(o, oh),
                                (long long)d->M);
                uint64_t key;
                if (pol == SVF_POLICY_FCFS) key = (uint64_t)a;
                else if (pol == SVF_POLICY_SJF) key = (uint64_t)oh;
                else key = (uint64_t)s * (uint64_t)oh + (((uint64_t)oh * oh + oh) >> 1);
                if (key >= (uint64_t(1) << 32))
                    return fail(SVF_EINVAL, "instance %d request %lld: priority key %llu >= 2^32", i,
                                (long long)(j - lo), (unsigned long long)key);
                max_key[p] = std::max(max_key[p], key);
                // eviction is only possible when plans differ from the truth
                // or when admission looks at the next step only
                if (oh != o || current_rule) stepped[(size_t)p * I + i] = 1;
                *max_plan = std::max(*max_plan, oh);
                if (current_rule) cur_total[p] += s + oh;
            }
        }
        for (int p = 0; p < P; ++p) *max_profile = std::max(*max_profile, cur_total[p]);
    }
    return SVF_OK;
}

int check_desc_shape(const svf_batch_desc* d, int64_t* N) {
    if (!d) return fail(SVF_EINVAL, "desc is NULL");
    if (d->num_instances < 0) return fail(SVF_EINVAL, "num_instances < 0");
    if (!d->req_offsets) return fail(SVF_EINVAL, "req_offsets is NULL");
    if (d->num_policies < 1 || d->num_policies > 8)
        return fail(SVF_EINVAL, "num_policies must be in 1..8 (got %d)", d->num_policies);
    if (!d->policies) return fail(SVF_EINVAL, "policies is NULL");
    for (int p = 0; p < d->num_policies; ++p) {
        const int base = d->policies[p] & 0xFF, rule = d->policies[p] & ~0xFF;
        if (base < SVF_POLICY_FCFS || base > SVF_POLICY_SVF1BIT ||
            (rule != SVF_ADMIT_LOOKAHEAD && rule != SVF_ADMIT_CURRENT))
            return fail(SVF_EINVAL, "unknown policy %d", d->policies[p]);
    }
    if (d->M < 1 || d->M >= kLimit30) return fail(SVF_EINVAL, "M must be in [1, 2^30)");
    if (d->max_steps < 0 || d->max_steps >= kLimit30)
        return fail(SVF_EINVAL, "max_steps must be in [0, 2^30)");
    const int64_t* off = d->req_offsets;
    if (off[0] != 0) return fail(SVF_EINVAL, "req_offsets[0] must be 0");
    for (int32_t i = 0; i < d->num_instances; ++i) {
        const int64_t n = off[i + 1] - off[i];
        if (n < 0) return fail(SVF_EINVAL, "req_offsets decreases at instance %d", i);
        if (n >= (int64_t(1) << 31) - 1)
            return fail(SVF_EINVAL, "instance %d holds too many requests", i);
    }
    *N = off[d->num_instances];
    if (*N * (int64_t)d->num_policies >= (int64_t(1) << 31))
        return fail(SVF_EINVAL, "requests x policies must stay below 2^31");
    return SVF_OK;
}

// The launch plan of a validated batch: sizes, sort shape, profile kind
// (ring or finish-ordered list) and its LDS capacity per path, issue
// priorities.  Fills the host fields of ``h`` (not its buffers) and the
// bitmap word offsets bw_off[I+1].
int plan_batch(svf_batch* h, const svf_batch_desc* d, const HostView& v, const int64_t* off,
               const uint8_t* stepped, int64_t max_plan, int64_t max_profile,
               const uint64_t* max_key, int64_t* bw_off) {
    const int32_t I = d->num_instances, P = d->num_policies;
    const int64_t N = off[I];
    h->I = I; h->P = P; h->N = N;
    h->M = (int32_t)d->M;
    h->O0 = d->O0; h->O1 = d->O1;
    h->max_steps = (int32_t)d->max_steps;
    h->H = (int32_t)next_pow2(std::max<int64_t>(max_plan, 1));
    for (int32_t i = 0; i < I; ++i) h->max_n = std::max<int32_t>(h->max_n, (int32_t)(off[i + 1] - off[i]));
    h->CH = (int32_t)std::min<int64_t>(8192, std::max<int64_t>(64, next_pow2(h->max_n)));
    h->fused_sort = h->max_n <= svfk::SORT_REC_MAX;
    for (int32_t p = 0; p < P; ++p)
        h->kbits[p] = max_key[p] ? 64 - __builtin_clzll(max_key[p]) : 0;
    for (int64_t g = 0; g < (int64_t)P * I; ++g) {
        h->any_stepped |= stepped[g] != 0;
        (stepped[g] ? h->n_stepped : h->n_known) += 1;
    }
    // the profile ring stores memory + step index in int32
    if (max_profile + h->max_steps + 2 * (int64_t)h->H >= (int64_t(1) << 31) - 1)
        return fail(SVF_EINVAL, "M (or, under SVF_ADMIT_CURRENT, an instance's sum of s + planned "
                                "length) + max_steps + 2 * (longest planned length, rounded up to "
                                "a power of two) must stay below 2^31");

    // bitmap word offsets of the instances
    bw_off[0] = 0;
    for (int32_t i = 0; i < I; ++i) {
        const int64_t n = off[i + 1] - off[i];
        const int64_t W0 = (n + 63) / 64, W1 = (W0 + 63) / 64;
        bw_off[i + 1] = bw_off[i] + W0 + W1;
        h->bw_max = std::max<int32_t>(h->bw_max, (int32_t)(W0 + W1));
    }
    h->bw_total = bw_off[I];

    // ring placement: LDS when the ring and bitmap fit comfortably
    const char* env = getenv("SVFSIM_RING");
    const size_t ring_bytes = ((size_t)h->H + 64) * 4;  // H slots + spare slot
    const size_t bm_bytes = (size_t)h->bw_max * 8;
    h->d_lds = ring_bytes + bm_bytes <= 65536;
    if (env && !strcmp(env, "global")) h->d_lds = false;
    if (env && !strcmp(env, "lds") && ring_bytes + bm_bytes <= 160 * 1024) h->d_lds = true;
    h->lds_bytes = std::max<size_t>(8, bm_bytes + (h->d_lds ? ring_bytes : 0));
    // The event path keeps its profile as the finish-ordered list (8 bytes
    // per running request) when the ring does not fit in LDS, or when few
    // requests run at once: the list's checks and insertions touch the
    // running requests that finish before the candidate, the ring's the
    // candidate's whole planned length.  Measured: the list is faster at
    // about 140-280 concurrent requests (4096 x 1000 and 16384 x 5000
    // workloads), 4x slower at about 930 (64 x 200,000); the estimate is
    // M / (mean s + mean o / 2) and the crossover is taken at 512.  The list
    // in LDS gets the largest capacity that still lets as many waves reside
    // as the list kernel's registers allow; segments that outgrow it stop,
    // and a second launch with room for the bound on concurrent requests
    // continues them.
    const int64_t bound = (h->n_known > 0 || h->any_stepped)
                              ? std::max<int64_t>(1, running_bound(v.s, off, I, d->M)) : 1;
    const size_t full_bytes = bm_bytes + (size_t)svfk::list_slots((int)std::min<int64_t>(bound, 1 << 24)) * 8;
    if (h->n_known > 0) {
        const char* pe = getenv("SVFSIM_PROFILE");
        bool use = false;
        int64_t cap = bound;
        if (full_bytes <= 160 * 1024) {
            auto occ = [&](bool list, bool dl, size_t bytes) {
                int w = 0;
                return svfk::sim_known_occupancy(list, dl, bytes, &w) == hipSuccess ? w : -1;
            };
            const int w_top = occ(true, false, bm_bytes + (size_t)svfk::list_slots(64) * 8);
            int64_t lo = std::min<int64_t>(bound, 64), hi = bound;  // occ(lo) >= w_top
            while (lo < hi) {
                const int64_t mid = lo + (hi - lo + 1) / 2;
                if (occ(true, false, bm_bytes + (size_t)svfk::list_slots((int)mid) * 8) >= w_top) lo = mid;
                else hi = mid - 1;
            }
            cap = lo;
            const char* pc = getenv("SVFSIM_LIST_LDS_CAP");  // testing: a smaller LDS list
            if (pc && atoll(pc) > 0) cap = std::min<int64_t>(cap, atoll(pc));
            double sum_s = 0.0, sum_o = 0.0;
            for (int64_t x = 0; x < N; ++x) {
                sum_s += v.s[x];
                sum_o += v.o[x];
            }
            const double running = N > 0 ? (double)d->M / ((sum_s + 0.5 * sum_o) / (double)N) : 0.0;
            if (w_top > 0) use = !h->d_lds || running <= 512.0;
        }
        if (pe && !strcmp(pe, "ring")) use = false;
        if (pe && !strcmp(pe, "list")) use = full_bytes <= 160 * 1024;
        if (use) {
            h->list_known = true;
            h->list_cap = (int32_t)cap;
            h->lds_list = bm_bytes + (size_t)svfk::list_slots((int)cap) * 8;
            h->lds_list_full = full_bytes;
        }
    }
    // The per-step path keeps its planned profile as the finish-ordered list
    // when the list with room for the bound fits in 64 KB of LDS.  As on the
    // event path, the first launch gives it the largest capacity that keeps
    // the kernel at the occupancy its registers allow, and a continuation
    // launch has room for the bound.
    if (h->any_stepped) {
        const char* ps = getenv("SVFSIM_STEP_PROFILE");
        bool use = full_bytes <= 64 * 1024;
        if (ps && !strcmp(ps, "ring")) use = false;
        if (ps && !strcmp(ps, "list")) use = full_bytes <= 160 * 1024;
        if (use) {
            auto occ = [&](size_t bytes) {
                int w = 0;
                return svfk::sim_step_occupancy(bytes, &w) == hipSuccess ? w : -1;
            };
            const int w_top = occ(bm_bytes + (size_t)svfk::list_slots(64) * 8);
            int64_t lo = std::min<int64_t>(bound, 64), hi = bound;
            while (w_top > 0 && lo < hi) {
                const int64_t mid = lo + (hi - lo + 1) / 2;
                if (occ(bm_bytes + (size_t)svfk::list_slots((int)mid) * 8) >= w_top) lo = mid;
                else hi = mid - 1;
            }
            int64_t cap = w_top > 0 ? lo : bound;
            const char* pc = getenv("SVFSIM_STEP_LDS_CAP");  // testing: a smaller LDS list
            if (pc && atoll(pc) > 0) cap = std::min<int64_t>(cap, atoll(pc));
            h->list_stepped = true;
            h->step_cap = (int32_t)cap;
            h->lds_step = bm_bytes + (size_t)svfk::list_slots((int)cap) * 8;
            h->lds_step_full = full_bytes;
        }
    }
    if (h->list_known || h->list_stepped) h->list_stride = (int32_t)bound;
    h->ring_used = (h->n_known > 0 && !h->list_known) || (h->any_stepped && !h->list_stepped);
    // Resident workgroups of the first simulation launch of each path; the
    // waves set their issue priorities only when it is known (timing only).
    // With at most one segment per CU there is nothing to arbitrate.
    {
        int ncu = 0;
        const char* pp = getenv("SVFSIM_ISSUE_PRIO");  // "0": all waves at one priority
        const bool on = !(pp && !strcmp(pp, "0"));
        if (on && hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, h->device) == hipSuccess &&
            ncu > 0 && (int64_t)P * I > ncu) {
            int w = 0;
            if (h->n_known > 0 &&
                svfk::sim_occupancy(false, h->list_known, h->d_lds,
                                    h->list_known ? h->lds_list : h->lds_bytes, &w) == hipSuccess)
                h->res_known = w * ncu;
            w = 0;
            if (h->any_stepped &&
                svfk::sim_occupancy(true, h->list_stepped, h->d_lds,
                                    h->list_stepped ? h->lds_step : h->lds_bytes, &w) == hipSuccess)
                h->res_stepped = w * ncu;
        }
        (void)hipGetLastError();
    }
    if (h->lds_bytes > 160 * 1024)
        return fail(SVF_EINVAL, "an instance's rank bitmap needs %zu bytes of LDS (> 160 KB)", h->lds_bytes);

    return SVF_OK;
}

void record(svf_batch* h, int kind, hipEvent_t* a) {
    if (!h->prof) return;
    (void)hipEventCreate(a);
    (void)hipEventRecord(*a, h->stream);
    (void)kind;
}

void record_end(svf_batch* h, int kind, hipEvent_t a) {
    if (!h->prof) return;
    hipEvent_t b;
    (void)hipEventCreate(&b);
    (void)hipEventRecord(b, h->stream);
    h->timed.push_back({kind, a, b});
}

int do_reset(svf_batch* h) {
    const int32_t G = h->P * h->I;
    const int64_t PN = (int64_t)h->P * h->N;
    hipEvent_t e0 = nullptr;
    record(h, 0, &e0);
    HIPCHK(svfk::launch_init_state(h->d_st, G, h->stream));
    HIPCHK(svfk::launch_fill_u64(h->d_bitmap, (int64_t)h->P * h->bw_total, 0ull, h->stream));
    if (h->ring_used)
        HIPCHK(svfk::launch_init_ring(h->d_ring, (int64_t)G * (h->H + 64), h->H, h->stream));
    if (!h->fused_sort) {
        HIPCHK(svfk::launch_fill_i32(h->d_start, PN, -1, h->stream));
        HIPCHK(svfk::launch_fill_i32(h->d_fin, PN, -1, h->stream));
        HIPCHK(svfk::launch_fill_i32(h->d_pre, PN, 0, h->stream));
        HIPCHK(svfk::launch_fill_i32(h->d_seq, PN, -1, h->stream));
    }
    if (PN > 0) {
        svfk::SortArgs A{};
        A.offsets = h->d_off;
        A.a = h->d_a; A.s = h->d_s; A.o = h->d_o; A.plan = h->d_plan; A.bit = h->d_bit;
        A.policies = h->d_pol;
        A.chunk_seg = h->d_chunk_seg;
        A.chunk_lo = h->d_chunk_lo;
        A.rec = h->d_rec;
        A.rank = h->d_rank;
        A.I = h->I; A.P = h->P; A.N = h->N; A.O0 = h->O0; A.O1 = h->O1; A.CH = h->CH;
        for (int p = 0; p < 8; ++p) A.kbits[p] = h->kbits[p];
        A.start = h->d_start; A.fin = h->d_fin; A.preempt = h->d_pre; A.admit_seq = h->d_seq;
        A.stepped = h->d_stepped;
        if (h->fused_sort) {
            // keys, sort, records, ranks and cleared outputs in one kernel
            HIPCHK(svfk::launch_sort_rec(A, G, h->max_n, h->stream));
            record_end(h, 0, e0);
            h->was_reset = true;
            h->dirty = true;
            return SVF_OK;
        }
        A.keys_in = nullptr;
        A.keys_out = h->d_keys0;
        HIPCHK(svfk::launch_chunk_sort(A, h->nchunks, h->stream));
        uint64_t* cur = h->d_keys0;
        uint64_t* other = h->d_keys1;
        for (int64_t w = h->CH; w < h->max_n; w *= 2) {
            A.keys_in = cur;
            A.keys_out = other;
            HIPCHK(svfk::launch_merge_pass(A, h->nchunks, (int)w, h->stream));
            std::swap(cur, other);
        }
        A.keys_in = cur;
        A.keys_out = nullptr;
        HIPCHK(svfk::launch_build_rec(A, h->nchunks, h->stream));
    }
    record_end(h, 0, e0);
    h->was_reset = true;
    h->dirty = true;
    return SVF_OK;
}

int do_sim(svf_batch* h, int64_t delta) {
    const int32_t G = h->P * h->I;
    if (G <= 0) return SVF_OK;
    svfk::SimArgs S{};
    S.offsets = h->d_off;
    S.a = h->d_a;
    S.rec = h->d_rec;
    S.rank = h->d_rank;
    S.stepped = h->d_stepped;
    S.policies = h->d_pol;
    S.bw_off = h->d_bw_off;
    S.bitmap = h->d_bitmap;
    S.ring = h->d_ring;
    S.start = h->d_start;
    S.fin = h->d_fin;
    S.preempt = h->d_pre;
    S.admit_seq = h->d_seq;
    S.act = h->d_act;
    S.actkr = h->d_actkr;
    S.evl = h->d_evl;
    S.st = h->d_st;
    S.I = h->I; S.P = h->P; S.N = h->N;
    S.bw_total = h->bw_total;
    S.bw_max = h->bw_max;
    S.H = h->H;
    S.M = h->M;
    S.max_steps = h->max_steps;
    S.step_delta = delta;
    S.lst_f = h->d_lst_f;
    S.lst_q = h->d_lst_q;
    S.list_stride = h->list_stride;
    S.list_cap = h->list_cap;
    S.list_resume = 0;
    S.resident = h->res_known;
    S.prog = h->d_prog;
    HIPCHK(svfk::launch_fill_u64(reinterpret_cast<uint64_t*>(h->d_prog), 2, 0ull, h->stream));
    hipEvent_t e0 = nullptr;
    record(h, 1, &e0);
    // The two paths simulate disjoint segments (each kernel leaves the other
    // path's segments alone) and keep separate progress counters, so with
    // segments on both the event-driven launch runs on the second stream,
    // concurrently with the per-step one.  The per-step launch (long serial
    // segments at low occupancy) goes first, on the caller's stream, so that
    // its waves are resident from the start; the event-driven waves fill the
    // remaining slots.
    const bool fork = h->aux && h->n_known > 0 && h->n_stepped > 0;
    const hipStream_t st_stepped = h->stream;
    hipStream_t st_known = h->stream;
    if (fork) {
        HIPCHK(hipEventRecord(h->fork_ev, h->stream));
        HIPCHK(hipStreamWaitEvent(h->aux, h->fork_ev, 0));
        st_known = h->aux;
    }
    // launch errors are kept until the second stream has been joined back
    hipError_t le = hipSuccess;
    if (h->n_stepped > 0) {
        svfk::SimArgs T = S;
        T.list_cap = h->step_cap;
        T.list_resume = 0;
        T.resident = h->res_stepped;
        T.prog = h->d_prog + 1;
        le = svfk::launch_sim(T, G, h->d_lds, true, h->list_stepped,
                              h->list_stepped ? h->lds_step : h->lds_bytes, st_stepped);
        if (le == hipSuccess && h->list_stepped && h->step_cap < h->list_stride) {
            // segments whose list outgrew the LDS capacity, up to the same step
            T.list_cap = h->list_stride;
            T.list_resume = 1;
            T.resident = 0;
            le = svfk::launch_sim(T, G, false, true, true, h->lds_step_full, st_stepped);
        }
    }
    if (le == hipSuccess && h->n_known > 0) {
        le = svfk::launch_sim(S, G, h->d_lds, false, h->list_known,
                              h->list_known ? h->lds_list : h->lds_bytes, st_known);
        if (le == hipSuccess && h->list_known && h->list_cap < h->list_stride) {
            // segments whose list outgrew the LDS capacity, up to the same step
            S.list_cap = h->list_stride;
            S.list_resume = 1;
            S.resident = 0;
            le = svfk::launch_sim(S, G, false, false, true, h->lds_list_full, st_known);
        }
    }
    if (fork) {
        HIPCHK(hipEventRecord(h->join_ev, h->aux));
        HIPCHK(hipStreamWaitEvent(h->stream, h->join_ev, 0));
    }
    if (le != hipSuccess)
        return fail(SVF_EHIP, "simulation launch failed: %s", hipGetErrorString(le));
    record_end(h, 1, e0);
    h->sim_launches += 1;
    h->dirty = true;
    return SVF_OK;
}

int do_finalize(svf_batch* h) {
    if (!h->dirty) return SVF_OK;
    const int32_t G = h->P * h->I;
    svfk::FinArgs F{};
    F.offsets = h->d_off;
    F.a = h->d_a;
    F.o = h->d_o;
    F.stepped = h->d_stepped;
    F.start = h->d_start;
    F.fin = h->d_fin;
    F.preempt = h->d_pre;
    F.st = h->d_st;
    F.fin_out = h->d_fin_out;
    F.stats = h->d_stats;
    F.I = h->I; F.P = h->P; F.N = h->N;
    hipEvent_t e0 = nullptr;
    record(h, 2, &e0);
    HIPCHK(svfk::launch_finalize(F, G, h->stream));
    record_end(h, 2, e0);
    h->dirty = false;
    return SVF_OK;
}

// Sequential placement of buffers in a fixed device region (256-byte
// aligned); ``used`` may exceed the region, and is checked before any use.
struct Carve {
    char* base;
    size_t used;
    template <typename T>
    T* take(int64_t count) {
        if (count <= 0) return nullptr;
        used = (used + 255) & ~size_t(255);
        T* p = reinterpret_cast<T*>(base + used);
        used += sizeof(T) * (size_t)count;
        return p;
    }
};

// Host tables of svf_run_noalloc (per-segment path flags, bitmap word
// offsets), static so that the call allocates nothing; guarded by g_na_mu.
std::mutex g_na_mu;
uint8_t g_na_stepped[(size_t)SVF_NOALLOC_MAX_INSTANCES * 8];
int64_t g_na_bw_off[SVF_NOALLOC_MAX_INSTANCES + 1];

}  // namespace

extern "C" {

const char* svf_last_error(void) { return g_err; }

int svf_abi_version(void) { return SVFSIM_ABI_VERSION; }

int svf_create(const svf_batch_desc* d, void* hip_stream, svf_batch** out) {
    g_err[0] = 0;
    if (!out) return fail(SVF_EINVAL, "out is NULL");
    *out = nullptr;
    int64_t N = 0;
    RETCHK(check_desc_shape(d, &N));
    const int32_t I = d->num_instances, P = d->num_policies;
    const std::vector<int64_t> off(d->req_offsets, d->req_offsets + I + 1);

    // host view of the per-request arrays (device inputs are fetched first)
    std::vector<int32_t> ha, hs, ho, hp;
    std::vector<int8_t> hb;
    HostView v{d->arrival, d->prompt, d->output, d->plan_len, d->long_bit};
    if (d->inputs_on_device && N > 0) {
        if (!d->arrival || !d->prompt || !d->output)
            return fail(SVF_EINVAL, "arrival, prompt and output must not be NULL");
        ha.resize(N); hs.resize(N); ho.resize(N);
        HIPCHK(hipMemcpy(ha.data(), d->arrival, 4 * N, hipMemcpyDeviceToHost));
        HIPCHK(hipMemcpy(hs.data(), d->prompt, 4 * N, hipMemcpyDeviceToHost));
        HIPCHK(hipMemcpy(ho.data(), d->output, 4 * N, hipMemcpyDeviceToHost));
        v.a = ha.data(); v.s = hs.data(); v.o = ho.data();
        if (d->plan_len) {
            hp.resize(N);
            HIPCHK(hipMemcpy(hp.data(), d->plan_len, 4 * N, hipMemcpyDeviceToHost));
            v.plan = hp.data();
        }
        if (d->long_bit) {
            hb.resize(N);
            HIPCHK(hipMemcpy(hb.data(), d->long_bit, N, hipMemcpyDeviceToHost));
            v.bit = hb.data();
        }
    }
    std::vector<uint8_t> stepped((size_t)P * I);
    int64_t max_plan = 1, max_profile = 0;
    uint64_t max_key[8];
    RETCHK(validate(d, v, off.data(), N, stepped.data(), &max_plan, &max_profile, max_key));

    svf_batch* h = new (std::nothrow) svf_batch();
    if (!h) return fail(SVF_ENOMEM, "host allocation failed");
    h->stream = (hipStream_t)hip_stream;
    (void)hipGetDevice(&h->device);
    h->policies.assign(d->policies, d->policies + P);
    h->offsets = off;
    std::vector<int64_t> bw_off(I + 1, 0);
    {
        const int rc = plan_batch(h, d, v, off.data(), stepped.data(), max_plan, max_profile,
                                  max_key, bw_off.data());
        if (rc != SVF_OK) {
            delete h;
            return rc;
        }
    }
    // chunk table (segment, first position) of the sort for large instances
    std::vector<int32_t> cseg, clo;
    for (int32_t p = 0; p < P; ++p)
        for (int32_t i = 0; i < I; ++i) {
            const int64_t n = off[i + 1] - off[i];
            for (int64_t lo = 0; lo < n; lo += h->CH) {
                cseg.push_back(p * I + i);
                clo.push_back((int32_t)lo);
            }
        }
    h->nchunks = (int32_t)cseg.size();

    const int64_t G = (int64_t)P * I;
    const int64_t PN = (int64_t)P * N;
    int rc = SVF_OK;
#define ALLOC(ptr, cnt) \
    if (rc == SVF_OK) rc = dalloc(&h->ptr, (cnt));
    ALLOC(d_off, I + 1);
    ALLOC(d_a, N);
    ALLOC(d_s, N);
    ALLOC(d_o, N);
    if (d->plan_len) ALLOC(d_plan, N);
    if (d->long_bit) ALLOC(d_bit, N);
    ALLOC(d_pol, P);
    ALLOC(d_chunk_seg, h->nchunks);
    ALLOC(d_chunk_lo, h->nchunks);
    if (!h->fused_sort) {
        ALLOC(d_keys0, PN);
        ALLOC(d_keys1, PN);
    }
    ALLOC(d_rec, PN);
    ALLOC(d_rank, PN);
    ALLOC(d_stepped, G);
    ALLOC(d_bw_off, I + 1);
    ALLOC(d_bitmap, (int64_t)P * h->bw_total);
    if (h->ring_used) ALLOC(d_ring, G * (h->H + 64));
    if (h->list_known || h->list_stepped) {
        ALLOC(d_lst_f, G * (int64_t)h->list_stride);
        ALLOC(d_lst_q, G * (int64_t)h->list_stride);
    }
    ALLOC(d_start, PN);
    ALLOC(d_fin, PN);
    ALLOC(d_pre, PN);
    ALLOC(d_seq, PN);
    if (h->any_stepped) {
        ALLOC(d_act, PN);
        ALLOC(d_actkr, PN);
        ALLOC(d_evl, PN);
    }
    ALLOC(d_st, G);
    ALLOC(d_prog, 2);
    ALLOC(d_fin_out, PN);
    ALLOC(d_stats, G);
#undef ALLOC
    if (rc != SVF_OK) {
        free_all(h);
        delete h;
        return rc;
    }
    const hipMemcpyKind kind = d->inputs_on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;
    hipError_t e = hipSuccess;
#define CPY(dst, src, bytes, k) \
    if (e == hipSuccess && (bytes) > 0) e = hipMemcpyAsync((dst), (src), (bytes), (k), h->stream);
    CPY(h->d_off, off.data(), 8 * (I + 1), hipMemcpyHostToDevice);
    CPY(h->d_a, d->arrival, 4 * N, kind);
    CPY(h->d_s, d->prompt, 4 * N, kind);
    CPY(h->d_o, d->output, 4 * N, kind);
    if (d->plan_len) CPY(h->d_plan, d->plan_len, 4 * N, kind);
    if (d->long_bit) CPY(h->d_bit, d->long_bit, N, kind);
    CPY(h->d_pol, h->policies.data(), 4 * P, hipMemcpyHostToDevice);
    CPY(h->d_chunk_seg, cseg.data(), 4 * (int64_t)cseg.size(), hipMemcpyHostToDevice);
    CPY(h->d_chunk_lo, clo.data(), 4 * (int64_t)clo.size(), hipMemcpyHostToDevice);
    CPY(h->d_stepped, stepped.data(), G, hipMemcpyHostToDevice);
    CPY(h->d_bw_off, bw_off.data(), 8 * (I + 1), hipMemcpyHostToDevice);
#undef CPY
    // Finishes and preemption counts are written only by the per-step path;
    // event-path segments keep these initial values (the reset's sort clears
    // them for per-step segments only).
    if (e == hipSuccess) e = svfk::launch_fill_i32(h->d_fin, PN, -1, h->stream);
    if (e == hipSuccess) e = svfk::launch_fill_i32(h->d_pre, PN, 0, h->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->stream);
    if (e == hipSuccess) {
        hipError_t a = svfk::prepare_sim(h->d_lds, h->lds_bytes, h->list_known || h->list_stepped,
                                         std::max(h->lds_list_full, h->lds_step_full));
        if (a != hipSuccess) e = a;
    }
    if (e == hipSuccess && h->fused_sort) {
        hipError_t a = svfk::prepare_sort_rec(h->max_n);
        if (a != hipSuccess) e = a;
    }
    // both paths in one batch: a second stream for the per-step launches
    // (SVFSIM_CONCURRENT=0 keeps them on one stream)
    const char* pc = getenv("SVFSIM_CONCURRENT");
    if (e == hipSuccess && h->n_known > 0 && h->n_stepped > 0 && !(pc && !strcmp(pc, "0"))) {
        e = hipStreamCreateWithFlags(&h->aux, hipStreamNonBlocking);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&h->fork_ev, hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&h->join_ev, hipEventDisableTiming);
    }
    if (e != hipSuccess) {
        free_all(h);
        delete h;
        return fail(SVF_EHIP, "copying the inputs failed: %s", hipGetErrorString(e));
    }
    *out = h;
    return ok();
}

int svf_reset(svf_batch* h) {
    if (!h) return fail(SVF_EINVAL, "handle is NULL");
    return do_reset(h);
}

int svf_step(svf_batch* h, int64_t nsteps) {
    if (!h) return fail(SVF_EINVAL, "handle is NULL");
    if (nsteps < 0) return fail(SVF_EINVAL, "nsteps < 0");
    if (!h->was_reset) RETCHK(do_reset(h));
    // nsteps == 0 still launches: instances that are already complete at their
    // current step (e.g. empty ones) get their final status
    return do_sim(h, std::min<int64_t>(nsteps, int64_t(1) << 40));
}

int svf_run(svf_batch* h) {
    if (!h) return fail(SVF_EINVAL, "handle is NULL");
    if (!h->was_reset) RETCHK(do_reset(h));
    return do_sim(h, int64_t(1) << 40);
}

int svf_read(svf_batch* h, int32_t slot, int32_t* start, int32_t* finish, int32_t* preempt,
             int32_t* admit_seq, int32_t outputs_on_device) {
    if (!h) return fail(SVF_EINVAL, "handle is NULL");
    if (slot < 0 || slot >= h->P) return fail(SVF_EINVAL, "policy slot %d out of range", slot);
    if (!h->was_reset) return fail(SVF_ESTATE, "nothing simulated yet (call svf_reset/svf_run)");
    RETCHK(do_finalize(h));
    const int64_t base = (int64_t)slot * h->N;
    const size_t bytes = 4 * (size_t)h->N;
    const hipMemcpyKind k = outputs_on_device ? hipMemcpyDeviceToDevice : hipMemcpyDeviceToHost;
    if (bytes) {
        if (start) HIPCHK(hipMemcpyAsync(start, h->d_start + base, bytes, k, h->stream));
        if (finish) HIPCHK(hipMemcpyAsync(finish, h->d_fin_out + base, bytes, k, h->stream));
        if (preempt) HIPCHK(hipMemcpyAsync(preempt, h->d_pre + base, bytes, k, h->stream));
        if (admit_seq) HIPCHK(hipMemcpyAsync(admit_seq, h->d_seq + base, bytes, k, h->stream));
    }
    if (!outputs_on_device) HIPCHK(hipStreamSynchronize(h->stream));
    return ok();
}

int svf_stats(svf_batch* h, int32_t slot, svf_instance_stats* out) {
    if (!h) return fail(SVF_EINVAL, "handle is NULL");
    if (slot < 0 || slot >= h->P) return fail(SVF_EINVAL, "policy slot %d out of range", slot);
    if (!out && h->I > 0) return fail(SVF_EINVAL, "out is NULL");
    if (!h->was_reset) return fail(SVF_ESTATE, "nothing simulated yet (call svf_reset/svf_run)");
    RETCHK(do_finalize(h));
    if (h->I > 0)
        HIPCHK(hipMemcpyAsync(out, h->d_stats + (int64_t)slot * h->I,
                              sizeof(svf_instance_stats) * h->I, hipMemcpyDeviceToHost, h->stream));
    HIPCHK(hipStreamSynchronize(h->stream));
    return ok();
}

int svf_set_profiling(svf_batch* h, int32_t enable) {
    if (!h) return fail(SVF_EINVAL, "handle is NULL");
    HIPCHK(hipStreamSynchronize(h->stream));
    for (auto& t : h->timed) {
        (void)hipEventDestroy(t.a);
        (void)hipEventDestroy(t.b);
    }
    h->timed.clear();
    h->acc_ms[0] = h->acc_ms[1] = h->acc_ms[2] = 0;
    h->sim_launches = 0;
    h->prof = enable != 0;
    return ok();
}

int svf_timings(svf_batch* h, svf_timing* out) {
    if (!h || !out) return fail(SVF_EINVAL, "NULL argument");
    HIPCHK(hipStreamSynchronize(h->stream));
    for (auto& t : h->timed) {
        float ms = 0;
        HIPCHK(hipEventElapsedTime(&ms, t.a, t.b));
        h->acc_ms[t.kind] += ms;
        (void)hipEventDestroy(t.a);
        (void)hipEventDestroy(t.b);
    }
    h->timed.clear();
    out->init_ms = h->acc_ms[0];
    out->sim_ms = h->acc_ms[1];
    out->final_ms = h->acc_ms[2];
    out->sim_launches = h->sim_launches;
    return ok();
}

int svf_shape(const svf_batch* h, int64_t* num_requests, int32_t* num_instances,
              int32_t* num_policies) {
    if (!h) return fail(SVF_EINVAL, "handle is NULL");
    if (num_requests) *num_requests = h->N;
    if (num_instances) *num_instances = h->I;
    if (num_policies) *num_policies = h->P;
    return ok();
}

int svf_destroy(svf_batch* h) {
    if (!h) return ok();
    (void)hipStreamSynchronize(h->stream);
    free_all(h);
    delete h;
    return ok();
}

int svf_run_noalloc(const svf_batch_desc* d, void* hip_stream, int32_t* start, int32_t* finish,
                    int32_t* preempt, int32_t* admit_seq, svf_instance_stats* stats) {
    g_err[0] = 0;
    int64_t N = 0;
    RETCHK(check_desc_shape(d, &N));
    const int32_t I = d->num_instances, P = d->num_policies;
    if (d->inputs_on_device)
        return fail(SVF_EINVAL, "svf_run_noalloc: the inputs must be host memory (inputs_on_device = 0)");
    if (I > SVF_NOALLOC_MAX_INSTANCES)
        return fail(SVF_EINVAL, "svf_run_noalloc: %d instances, at most %d", I,
                    SVF_NOALLOC_MAX_INSTANCES);
    const int64_t G = (int64_t)P * I, PN = (int64_t)P * N;
    if (PN > 0 && (!start || !finish || !preempt || !admit_seq))
        return fail(SVF_EINVAL, "svf_run_noalloc: an output array is NULL");
    if (G > 0 && !stats) return fail(SVF_EINVAL, "svf_run_noalloc: stats is NULL");
    const int64_t* off = d->req_offsets;
    for (int32_t i = 0; i < I; ++i)
        if (off[i + 1] - off[i] > svfk::SORT_REC_MAX)
            return fail(SVF_EINVAL, "svf_run_noalloc: instance %d holds %lld requests, at most %d",
                        i, (long long)(off[i + 1] - off[i]), (int)svfk::SORT_REC_MAX);

    std::lock_guard<std::mutex> lock(g_na_mu);
    const HostView v{d->arrival, d->prompt, d->output, d->plan_len, d->long_bit};
    int64_t max_plan = 1, max_profile = 0;
    uint64_t max_key[8];
    RETCHK(validate(d, v, off, N, g_na_stepped, &max_plan, &max_profile, max_key));
    svf_batch h;  // the launch plan; its buffers are the scratch and the caller's outputs
    h.stream = (hipStream_t)hip_stream;
    HIPCHK(hipGetDevice(&h.device));
    RETCHK(plan_batch(&h, d, v, off, g_na_stepped, max_plan, max_profile, max_key, g_na_bw_off));

    void* base = nullptr;
    size_t cap = 0;
    HIPCHK(svfk::noalloc_scratch(&base, &cap));
    Carve c{static_cast<char*>(base), 0};
    h.d_off = c.take<int64_t>(I + 1);
    h.d_a = c.take<int32_t>(N);
    h.d_s = c.take<int32_t>(N);
    h.d_o = c.take<int32_t>(N);
    if (d->plan_len) h.d_plan = c.take<int32_t>(N);
    if (d->long_bit) h.d_bit = c.take<int8_t>(N);
    h.d_pol = c.take<int32_t>(P);
    h.d_rec = c.take<int4>(PN);
    h.d_rank = c.take<int32_t>(PN);
    h.d_stepped = c.take<uint8_t>(G);
    h.d_bw_off = c.take<int64_t>(I + 1);
    h.d_bitmap = c.take<uint64_t>((int64_t)P * h.bw_total);
    if (h.ring_used) h.d_ring = c.take<int32_t>(G * (h.H + 64));
    if (h.list_known || h.list_stepped) {
        h.d_lst_f = c.take<int32_t>(G * (int64_t)h.list_stride);
        h.d_lst_q = c.take<uint32_t>(G * (int64_t)h.list_stride);
    }
    h.d_fin = c.take<int32_t>(PN);
    if (h.any_stepped) {
        h.d_act = c.take<int4>(PN);
        h.d_actkr = c.take<int2>(PN);
        h.d_evl = c.take<int32_t>(PN);
    }
    h.d_st = c.take<SegState>(G);
    h.d_prog = c.take<unsigned long long>(2);
    if (c.used > cap)
        return fail(SVF_EINVAL, "svf_run_noalloc: the batch needs %zu bytes of device scratch, "
                                "more than the %zu this entry point has", c.used, cap);
    h.d_start = start;
    h.d_pre = preempt;
    h.d_seq = admit_seq;
    h.d_fin_out = finish;
    h.d_stats = reinterpret_cast<StatsOut*>(stats);

    // inputs and host tables into the scratch; everything else the call reads
    // is rebuilt by its own kernels (the scratch keeps the previous call's data)
    const hipMemcpyKind k = hipMemcpyHostToDevice;
    hipError_t e = hipSuccess;
#define CPY(dst, src, bytes) \
    if (e == hipSuccess && (bytes) > 0) e = hipMemcpyAsync((dst), (src), (bytes), k, h.stream);
    CPY(h.d_off, off, 8 * (I + 1));
    CPY(h.d_a, d->arrival, 4 * N);
    CPY(h.d_s, d->prompt, 4 * N);
    CPY(h.d_o, d->output, 4 * N);
    if (d->plan_len) CPY(h.d_plan, d->plan_len, 4 * N);
    if (d->long_bit) CPY(h.d_bit, d->long_bit, N);
    CPY(h.d_pol, d->policies, 4 * P);
    CPY(h.d_stepped, g_na_stepped, G);
    CPY(h.d_bw_off, g_na_bw_off, 8 * (I + 1));
#undef CPY
    // finishes and preemption counts start cleared, as at svf_create
    if (e == hipSuccess) e = svfk::launch_fill_i32(h.d_fin, PN, -1, h.stream);
    if (e == hipSuccess) e = svfk::launch_fill_i32(h.d_pre, PN, 0, h.stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h.stream);
    if (e != hipSuccess)
        return fail(SVF_EHIP, "svf_run_noalloc: copying the inputs failed: %s", hipGetErrorString(e));
    HIPCHK(svfk::prepare_sim(h.d_lds, h.lds_bytes, h.list_known || h.list_stepped,
                             std::max(h.lds_list_full, h.lds_step_full)));
    if (h.max_n > 0) HIPCHK(svfk::prepare_sort_rec(h.max_n));
    RETCHK(do_reset(&h));
    RETCHK(do_sim(&h, int64_t(1) << 40));
    RETCHK(do_finalize(&h));
    return ok();
}

}  // extern "C"
