// svf_opt.cpp -- exact optimum of tiny burst instances (host code).
//
// Dynamic programming over the scheduler's state for the integer program of
// Section 3.1 with every arrival at step 0.  The state is the multiset of
// requests not started and the multiset of running requests with their
// progress; identical (s, o) requests are merged into one type, so a state is
// a vector of counts.  The value of a state is the least number of
// (request, step) pairs still to be spent unfinished, which for a burst does
// not depend on the current step:
//
//   V(U, R) = |U| + |R| + min over admissible S of V(U - S, advance(R + S)),
//
// where S is any sub-multiset of U whose start keeps every future step's
// memory <= M given R (S may be empty unless nothing runs), and advance moves
// every running request one step on and drops those that complete.  The
// recursion is searched depth first with a budget (branch and bound): a
// state's lower bound is the remaining length of its unfinished requests.

#include <stdint.h>

#include <algorithm>
#include <cstring>
#include <map>
#include <new>
#include <string>
#include <thread>
#include <unordered_map>
#include <vector>

#include "svfopt.h"
#include "svfsim.h"

namespace {

constexpr int kMaxN = 16;
constexpr int kMaxO = 16;  // keeps the recursion (one frame per type per step) shallow

struct Entry {
    int64_t v;    // exact value, or a lower bound when !exact
    bool exact;
};

struct Solver {
    int T = 0;                    // number of request types
    std::vector<int> s, o, cnt;   // per type
    std::vector<int> slot;        // first progress slot of each type
    int nslots = 0;               // sum of o over types
    int64_t M = 0;
    int64_t limit = 0;
    bool overflow = false;
    std::unordered_map<std::string, Entry> memo;

    // Cost still to come is at least the remaining length of every
    // unfinished request: o - e for a running one, o for one not started.
    int64_t floor_of(const uint8_t* u, const uint8_t* r) const {
        int64_t lb = 0;
        for (int t = 0; t < T; ++t) {
            lb += (int64_t)u[t] * o[t];
            for (int e = 0; e < o[t]; ++e) lb += (int64_t)r[slot[t] + e] * (o[t] - e);
        }
        return lb;
    }

    // Branch and bound over the recursion above: returns the exact value of
    // state st if it is <= budget, otherwise some lower bound > budget.
    // Exact values and lower bounds are both remembered.
    int64_t value(const std::string& st, int64_t budget) {
        auto it = memo.find(st);
        int64_t known_lb = 0;
        if (it != memo.end()) {
            if (it->second.exact) return it->second.v;
            known_lb = it->second.v;
        }
        if (overflow) return 0;
        const uint8_t* u = reinterpret_cast<const uint8_t*>(st.data());
        const uint8_t* r = u + T;
        int here = 0, running = 0;
        for (int t = 0; t < T; ++t) here += u[t];
        for (int k = 0; k < nslots; ++k) running += r[k];
        here += running;
        if (here == 0) return 0;
        const int64_t lb = std::max(known_lb, floor_of(u, r));
        if (lb > budget) return lb;
        // memory of the running requests at future steps d = 1..max o
        int64_t mem[kMaxO + 1] = {0};
        for (int t = 0; t < T; ++t)
            for (int e = 0; e < o[t]; ++e) {
                const int c = r[slot[t] + e];
                if (!c) continue;
                for (int d = 1; e + d <= o[t]; ++d) mem[d] += (int64_t)c * (s[t] + e + d);
            }
        std::vector<std::string> kids;
        int x[kMaxN];
        children(0, mem, x, u, r, running == 0, kids);
        int64_t best = INT64_MAX, fail_lb = INT64_MAX;
        for (const std::string& k : kids) {
            const int64_t cap = std::min(budget, best == INT64_MAX ? INT64_MAX : best - 1);
            if (cap < here) break;  // no child can beat best within the budget
            const int64_t v = value(k, cap - here);
            if (overflow) return 0;
            if (v <= cap - here) best = std::min(best, here + v);
            else fail_lb = std::min(fail_lb, here + v);
        }
        if ((int64_t)memo.size() >= limit) {
            overflow = true;
            return 0;
        }
        if (best <= budget) {
            memo[st] = {best, true};
            return best;
        }
        // every child failed: the smallest of their bounds (> budget) holds
        const int64_t out = std::max(lb, std::min(fail_lb, best));
        memo[st] = {std::max(out, budget + 1), false};
        return std::max(out, budget + 1);
    }

    // Every admissible start set, most starts first (good schedules early
    // tighten the budget): x[t] requests of type t, types in order; mem is
    // the future memory with the choices so far.
    void children(int t, const int64_t* mem, int* x, const uint8_t* u, const uint8_t* r,
                  bool must_start, std::vector<std::string>& kids) {
        if (t == T) {
            int started = 0;
            for (int k = 0; k < T; ++k) started += x[k];
            if (must_start && started == 0) return;
            std::string nx(T + nslots, '\0');
            uint8_t* nu = reinterpret_cast<uint8_t*>(&nx[0]);
            uint8_t* nr = nu + T;
            for (int k = 0; k < T; ++k) {
                nu[k] = (uint8_t)(u[k] - x[k]);
                // progress e -> e + 1; the new starts enter at progress 1
                for (int e = 0; e + 1 < o[k]; ++e) nr[slot[k] + e + 1] = r[slot[k] + e];
                if (o[k] > 1) nr[slot[k] + 1] = (uint8_t)(nr[slot[k] + 1] + x[k]);
            }
            kids.push_back(std::move(nx));
            return;
        }
        // largest count of this type that still fits
        int64_t cur[kMaxO + 1];
        std::memcpy(cur, mem, sizeof(cur));
        int cmax = 0;
        for (int c = 1; c <= u[t]; ++c) {
            bool ok = true;
            for (int d = 1; d <= o[t]; ++d) ok &= cur[d] + (int64_t)c * (s[t] + d) <= M;
            if (!ok) break;
            cmax = c;
        }
        for (int c = cmax; c >= 0; --c) {
            for (int d = 0; d <= kMaxO; ++d)
                cur[d] = mem[d] + (d >= 1 && d <= o[t] ? (int64_t)c * (s[t] + d) : 0);
            x[t] = c;
            children(t + 1, cur, x, u, r, must_start, kids);
        }
        x[t] = 0;
    }
};

int solve_one(int32_t n, const int32_t* prompt, const int32_t* output, int64_t M,
              int64_t state_limit, int64_t* total, int64_t* states) {
    if (n < 0 || n > kMaxN) return SVF_EINVAL;
    if (n > 0 && (!prompt || !output)) return SVF_EINVAL;
    if (!total) return SVF_EINVAL;
    std::map<std::pair<int, int>, int> types;
    for (int i = 0; i < n; ++i) {
        if (prompt[i] < 1 || output[i] < 1 || output[i] > kMaxO) return SVF_EINVAL;
        if ((int64_t)prompt[i] + output[i] > M) return SVF_EINFEASIBLE;
        types[{prompt[i], output[i]}] += 1;
    }
    Solver S;
    S.M = M;
    S.limit = state_limit > 0 ? state_limit : (int64_t(1) << 26);
    for (auto& kv : types) {
        S.s.push_back(kv.first.first);
        S.o.push_back(kv.first.second);
        S.cnt.push_back(kv.second);
        S.slot.push_back(S.nslots);
        S.nslots += kv.first.second;
    }
    S.T = (int)S.s.size();
    std::string st(S.T + S.nslots, '\0');
    for (int t = 0; t < S.T; ++t) st[t] = (char)(uint8_t)S.cnt[t];
    int64_t v = 0;
    try {
        v = S.value(st, INT64_MAX - 1);
    } catch (const std::bad_alloc&) {
        return SVF_ENOMEM;
    }
    if (states) *states = (int64_t)S.memo.size();
    if (S.overflow) return SVF_ELIMIT;
    *total = v;
    return SVF_OK;
}

}  // namespace

extern "C" int svf_opt_burst(int32_t n, const int32_t* prompt, const int32_t* output, int64_t M,
                             int64_t state_limit, int64_t* total_latency, int64_t* states) {
    return solve_one(n, prompt, output, M, state_limit, total_latency, states);
}

extern "C" int svf_opt_burst_batch(int32_t num_instances, const int64_t* req_offsets,
                                   const int32_t* prompt, const int32_t* output,
                                   const int64_t* M, int64_t state_limit, int32_t threads,
                                   int64_t* total_latency, int64_t* states, int32_t* status) {
    if (num_instances < 0 || (num_instances > 0 && (!req_offsets || !M || !total_latency ||
                                                    !status)))
        return SVF_EINVAL;
    for (int32_t i = 0; i < num_instances; ++i)
        if (req_offsets[i + 1] < req_offsets[i] || req_offsets[i + 1] - req_offsets[i] > kMaxN)
            return SVF_EINVAL;
    int nt = threads > 0 ? threads : (int)std::max(1u, std::thread::hardware_concurrency());
    nt = std::max(1, std::min(nt, std::max(1, num_instances)));
    auto work = [&](int w) {
        for (int32_t i = w; i < num_instances; i += nt) {
            const int64_t lo = req_offsets[i];
            int64_t st = 0;
            status[i] = solve_one((int32_t)(req_offsets[i + 1] - lo), prompt + lo, output + lo,
                                  M[i], state_limit, &total_latency[i], &st);
            if (states) states[i] = st;
        }
    };
    std::vector<std::thread> pool;
    for (int w = 1; w < nt; ++w) pool.emplace_back(work, w);
    work(0);
    for (auto& th : pool) th.join();
    for (int32_t i = 0; i < num_instances; ++i)
        if (status[i] != SVF_OK) return status[i];
    return SVF_OK;
}
