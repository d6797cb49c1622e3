// svf_kernels.hip -- gfx950 kernels of the batched scheduling simulator.
//
// One "segment" is one instance under one policy; segments are independent.
// Kernels, in launch order:
//   k_fill_*          clear state, bitmaps, rings and outputs (no memset nodes)
//   k_sort_rec<NT,E>  instances of at most 8192 requests: priority keys (Eq. 1 /
//                     Eq. 2), stable radix sort in LDS, rank-ordered records,
//                     index->rank map and cleared outputs, one workgroup per
//                     segment; larger instances take the next three kernels
//   k_chunk_sort<CH>  priority keys packed as key<<32|index and bitonic-sorted
//                     in LDS, one workgroup per chunk of CH
//   k_merge_pass      doubles the sorted run length of segments longer than CH
//                     (each element finds its output slot by binary search in
//                     the partner run)
//   k_build_rec       rank-ordered request records and the index->rank map
//   k_sim<D_LDS, STEPPED>, k_sim_list, k_sim_list_resume, k_sim_steplist,
//   k_sim_steplist_stop, k_sim_steplist_resume
//                     the simulation: one wave64 per segment (profile as a ring,
//                     per-step or event-driven; or as a finish-ordered list);
//                     the waves order their issue priorities by remaining work
//   k_finalize        per-request outputs as of the reached step (finish derived
//                     as start + o where lengths are known) + per-segment
//                     statistics, one 256-thread workgroup per segment
//
// Waiting set.  A segment's requests are sorted once by priority; the waiting
// set is then a bitmap over priority ranks (bit r set iff the request of rank
// r has arrived and is not running), with a summary word per 64 bitmap words.
// The highest-priority waiting request is the lowest set bit: one ballot over
// at most 64 summary words, then two count-trailing-zeros.  Both levels live
// in LDS for the whole launch.
//
// Future memory profile.  D[tau mod H] holds the memory that the running
// requests are planned to hold at future step tau (each request started at k
// with planned length L adds s + (tau - k) for tau in [k+1, k+L]; Section 3.1,
// eq:c2).  H is a power of two >= the longest planned length, so the window
// [t+1, t+H] never wraps onto itself.  The forward-looking check of a
// candidate h at step t (no future step above M; Appendix E.2) is then one
// pass over its own window: max_{j<o^_h} D[t+1+j] + (s_h + j + 1) <= M.
// Admitting h adds its growth to the same window; a step that becomes past is
// folded into the peak statistic and cleared.  The other form of the profile
// is the list of running requests ordered by planned finish, with prefix sums
// of s - k: between admissions the memory only drops at finishes, so the
// check visits just the finishes inside the candidate's window and its last
// step (ListProf, StepList).  The host picks the form per batch: the list
// where few requests run at once, the ring where many do.
//
// Known lengths (the scheduler plans with the true length) make D change only
// at admissions, so a blocked head stays blocked until a computable step t_f
// (every violating tau stops violating once t >= min(tau, D[tau]+tau+s_h-M))
// or until a request of higher priority arrives.  Such segments jump from
// event to event; the skipped steps are exactly the ones where the per-step
// scheduler admits nothing.  Segments whose planned lengths differ from the
// truth (1-bit SVF, noisy predictions) are advanced step by step: they track
// true completions, requests running past their planned length (planned to
// finish at the next step, kept as two running sums), and evictions when the
// true memory of the next step would exceed M; they too jump over the steps
// at which none of these can happen (memory then grows by one token per
// running request per step).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "svf_kernels.h"

namespace svfk {

// ------------------------------------------------------------ wave helpers

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

__device__ __forceinline__ int wave_max_i32(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o));
    return v;
}

__device__ __forceinline__ int wave_min_i32(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o));
    return v;
}

__device__ __forceinline__ long long wave_sum_i64(long long v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

__device__ __forceinline__ long long wave_max_i64(long long v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        long long w = __shfl_xor(v, o);
        v = w > v ? w : v;
    }
    return v;
}

__device__ __forceinline__ int bcast_i32(int v, int src) { return __shfl(v, src); }

__device__ __forceinline__ void wave_sync() { __syncthreads(); }

// The planned length the scheduler uses for request i under a policy.
__device__ __forceinline__ int planned_len(int policy, const int32_t* o, const int32_t* plan,
                                           const int8_t* bit, int O0, int O1, int64_t i) {
    if (policy == POLICY_SVF1BIT) return bit[i] ? O1 : O0;
    return plan ? plan[i] : o[i];
}

// Priority key (lower runs first): Section 2.2, Eq. 1 (volume) and Eq. 2 (the
// same volume with the 1-bit proxy length), SJF by length, FCFS by arrival.
__device__ __forceinline__ uint64_t priority_key(int policy, int32_t a, int32_t s, int32_t oh) {
    if (policy == POLICY_FCFS) return (uint64_t)(uint32_t)a;
    if (policy == POLICY_SJF) return (uint64_t)(uint32_t)oh;
    const uint64_t L = (uint64_t)(uint32_t)oh;
    return (uint64_t)(uint32_t)s * L + ((L * L + L) >> 1);
}

// ------------------------------------------------------------ fills

__global__ void k_fill_i32(int32_t* __restrict__ p, int64_t n, int32_t v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void k_fill_u64(uint64_t* __restrict__ p, int64_t n, uint64_t v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// A fresh ring represents the window [1, H] with D = 0: G[slot] = tau.  Each
// segment's ring has stride H + 64 (slot H is the spare slot).
__global__ void k_init_ring(int32_t* __restrict__ ring, int64_t n, int32_t H) {
    const int64_t RS = (int64_t)H + 64;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int32_t s = (int32_t)(i % RS);
        ring[i] = s == 0 ? H : (s < H ? s : 0);
    }
}

__global__ void k_init_state(SegState* __restrict__ st, int32_t G) {
    int g = blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= G) return;
    SegState z;
    z.t = 0; z.cursor = 0; z.seq = 0; z.status = STATUS_RUNNING;
    z.nA = 0; z.nfin = 0; z.max_fin = 0; z.head_rank = -1;
    z.t_f = 0; z.N_O = 0; z.C_O = 0; z.peak = 0; z.req_steps = 0; z.ln = 0; z.lq = 0;
    z.resume_lim = 0; z.resume_nev = -1;
    st[g] = z;
}

// ------------------------------------------------------------ keys and sort

template <int CH, int NT>
__global__ __launch_bounds__(NT) void k_chunk_sort(SortArgs A) {
    __shared__ uint64_t sk[CH];
    const int c = blockIdx.x;
    const int g = A.chunk_seg[c];
    const int lo = A.chunk_lo[c];
    const int pol = g / A.I, inst = g - pol * A.I;
    const int64_t off = A.offsets[inst];
    const int n = (int)(A.offsets[inst + 1] - off);
    const int len = min(CH, n - lo);
    const int policy = A.policies[pol] & 0xFF;
    for (int j = threadIdx.x; j < CH; j += NT) {
        uint64_t v = ~0ull;
        if (j < len) {
            const int64_t i = off + lo + j;
            const int oh = planned_len(policy, A.o, A.plan, A.bit, A.O0, A.O1, i);
            v = (priority_key(policy, A.a[i], A.s[i], oh) << 32) | (uint32_t)(lo + j);
        }
        sk[j] = v;
    }
    __syncthreads();
    for (int k = 2; k <= CH; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int t = threadIdx.x; t < CH / 2; t += NT) {
                const int i = 2 * t - (t & (j - 1));
                const int l = i + j;
                const bool asc = (i & k) == 0;
                const uint64_t x = sk[i], y = sk[l];
                if ((x > y) == asc) { sk[i] = y; sk[l] = x; }
            }
            __syncthreads();
        }
    }
    uint64_t* out = A.keys_out + (int64_t)pol * A.N + off + lo;
    for (int j = threadIdx.x; j < len; j += NT) out[j] = sk[j];
}

// One merge level: runs of length w become runs of length 2w.  Keys are
// unique (the index is packed in), so "number of partner elements below x"
// is the exact displacement.
__global__ __launch_bounds__(256) void k_merge_pass(SortArgs A, int w) {
    const int c = blockIdx.x;
    const int g = A.chunk_seg[c];
    const int lo = A.chunk_lo[c];
    const int pol = g / A.I, inst = g - pol * A.I;
    const int64_t off = A.offsets[inst];
    const int n = (int)(A.offsets[inst + 1] - off);
    const int len = min(A.CH, n - lo);
    const uint64_t* in = A.keys_in + (int64_t)pol * A.N + off;
    uint64_t* out = A.keys_out + (int64_t)pol * A.N + off;
    for (int j = threadIdx.x; j < len; j += blockDim.x) {
        const int p = lo + j;
        const uint64_t x = in[p];
        const int q = p / w;
        const int pair_base = (q >> 1) * 2 * w;
        const int local = p - q * w;
        int plo, phi;  // partner run [plo, phi)
        if ((q & 1) == 0) { plo = (q + 1) * w; phi = min(n, plo + w); }
        else { plo = (q - 1) * w; phi = plo + w; }
        int below = 0;
        if (plo < phi) {
            int L = plo, R = phi;  // first element >= x
            while (L < R) {
                const int m = (L + R) >> 1;
                if (in[m] < x) L = m + 1; else R = m;
            }
            below = L - plo;
        }
        out[pair_base + local + below] = x;
    }
}

__global__ __launch_bounds__(256) void k_build_rec(SortArgs A) {
    const int c = blockIdx.x;
    const int g = A.chunk_seg[c];
    const int lo = A.chunk_lo[c];
    const int pol = g / A.I, inst = g - pol * A.I;
    const int64_t off = A.offsets[inst];
    const int n = (int)(A.offsets[inst + 1] - off);
    const int len = min(A.CH, n - lo);
    const int policy = A.policies[pol] & 0xFF;
    const uint64_t* keys = A.keys_in + (int64_t)pol * A.N + off;
    int4* rec = A.rec + (int64_t)pol * A.N + off;
    int32_t* rank = A.rank + (int64_t)pol * A.N + off;
    for (int j = threadIdx.x; j < len; j += blockDim.x) {
        const int r = lo + j;
        const int idx = (int)(uint32_t)keys[r];
        if ((unsigned)idx >= (unsigned)n) continue;  // only a broken sort gets here
        const int64_t i = off + idx;
        int4 q;
        q.x = idx;
        q.y = A.s[i];
        q.z = planned_len(policy, A.o, A.plan, A.bit, A.O0, A.O1, i);
        q.w = A.o[i];
        rec[r] = q;
        rank[idx] = r;
    }
}

// One workgroup per segment whose instance holds n <= NT*E requests: the
// priority keys (Eq. 1 / Eq. 2, SJF, FCFS), a stable least-significant-digit
// radix sort on them (4-bit digits, as many passes as the policy's largest key
// needs; requests start in index order, which is arrival order, so equal keys
// stay in (arrival, index) order), then the rank-ordered records, the
// index -> rank map and the cleared outputs.  Thread t holds the elements
// t*E .. t*E+E-1 of the current order.  One pass: each element takes a
// running count of its digit among the thread's earlier elements (a 16-bit
// LDS counter per digit and thread, two to a 32-bit word for the atomic add),
// an exclusive scan over the counters in digit-major order turns them into
// start positions, and the elements are scattered through LDS and read back
// in thread order.  The element array is padded by one entry per 32 so that
// the thread-strided reads spread over the banks.  Global memory is read and
// written in batches of 8 elements per thread, so that a thread has 8
// requests in flight.
__device__ __forceinline__ int pad32(int f) { return f + (f >> 5); }

template <int NT, int E>
__global__ __launch_bounds__(NT) void k_sort_rec(SortArgs A) {
    constexpr int CH = NT * E;
    constexpr int B8 = 8;
    extern __shared__ uint64_t smem[];
    uint64_t* buf = smem;                                                 // [pad32(CH)]
    uint16_t* cnt = reinterpret_cast<uint16_t*>(smem + CH + CH / 32);     // [16 NT]
    uint32_t* cnt32 = reinterpret_cast<uint32_t*>(cnt);
    uint32_t* wsum = reinterpret_cast<uint32_t*>(cnt + 16 * NT);          // [NT / 64]
    const int g = blockIdx.x;
    const int pol = g / A.I, inst = g - pol * A.I;
    const int64_t off = A.offsets[inst];
    const int n = (int)(A.offsets[inst + 1] - off);
    const int policy = A.policies[pol] & 0xFF;
    const bool stepped = A.stepped[g] != 0;
    const int tid = threadIdx.x;
    const int lane = tid & 63, w = tid >> 6;
    const int64_t base = (int64_t)pol * A.N + off;

    // keys, read coalesced (element j = (e0 + u) NT + t) and handed over through LDS
    for (int e0 = 0; e0 * NT < n; e0 += B8) {
        int ra[B8], rs[B8], ro[B8];
#pragma unroll
        for (int u = 0; u < B8; ++u) {
            const int j = (e0 + u) * NT + tid;
            if (j < n) {
                const int64_t i = off + j;
                ra[u] = A.a[i];
                rs[u] = A.s[i];
                ro[u] = planned_len(policy, A.o, A.plan, A.bit, A.O0, A.O1, i);
            }
        }
#pragma unroll
        for (int u = 0; u < B8; ++u) {
            const int j = (e0 + u) * NT + tid;
            if (j < n) buf[pad32(j)] = (priority_key(policy, ra[u], rs[u], ro[u]) << 32) | (uint32_t)j;
        }
    }
    __syncthreads();
    uint64_t v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int j = tid * E + e;
        v[e] = j < n ? buf[pad32(j)] : ~0ull;
    }
    const int kb = A.kbits[pol];
    for (int sh = 0; sh < kb; sh += 4) {
#pragma unroll
        for (int d = 0; d < 16; ++d) cnt[d * NT + tid] = 0;
        int dg[E];
        uint32_t rk[E];
#pragma unroll
        for (int e = 0; e < E; ++e) {
            dg[e] = (int)((v[e] >> (32 + sh)) & 15u);
            rk[e] = 0u;
            if (tid * E + e < n) {
                const int f = dg[e] * NT + tid;
                const int hs = 16 * (f & 1);
                rk[e] = (atomicAdd(&cnt32[f >> 1], 1u << hs) >> hs) & 0xFFFFu;
            }
        }
        __syncthreads();
        // exclusive scan of the counters in digit-major order: thread t takes
        // the entries 16t .. 16t+15, then the threads' totals are scanned
        uint32_t c[16];
        uint32_t tot = 0u;
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            const uint32_t x = cnt[16 * tid + k];
            c[k] = tot;
            tot += x;
        }
        uint32_t inc = tot;  // inclusive scan of the thread totals inside the wave
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const uint32_t y = (uint32_t)__shfl_up((int)inc, o);
            if (lane >= o) inc += y;
        }
        if (lane == 63) wsum[w] = inc;
        __syncthreads();
        uint32_t woff = 0u;
        for (int k = 0; k < w; ++k) woff += wsum[k];
        const uint32_t add = woff + inc - tot;
#pragma unroll
        for (int k = 0; k < 16; ++k) cnt[16 * tid + k] = (uint16_t)(c[k] + add);
        __syncthreads();
#pragma unroll
        for (int e = 0; e < E; ++e)
            if (tid * E + e < n) buf[pad32((int)(cnt[dg[e] * NT + tid] + rk[e]))] = v[e];
        __syncthreads();
#pragma unroll
        for (int e = 0; e < E; ++e)
            if (tid * E + e < n) v[e] = buf[pad32(tid * E + e)];
        __syncthreads();
    }
    // (with no pass, buf already holds the index order)
    // records in rank order (consecutive ranks across a wave), the index ->
    // rank map, and the outputs cleared
    int4* rec = A.rec + base;
    int32_t* rank = A.rank + base;
    for (int e0 = 0; e0 * NT < n; e0 += B8) {
        int idx[B8];
        int4 q[B8];
#pragma unroll
        for (int u = 0; u < B8; ++u) {
            const int r = (e0 + u) * NT + tid;
            idx[u] = r < n ? (int)(uint32_t)buf[pad32(r)] : -1;
            if ((unsigned)idx[u] >= (unsigned)n) idx[u] = -1;  // only a broken sort
        }
#pragma unroll
        for (int u = 0; u < B8; ++u) {
            if (idx[u] >= 0) {
                const int64_t i = off + idx[u];
                q[u].x = idx[u];
                q[u].y = A.s[i];
                q[u].z = planned_len(policy, A.o, A.plan, A.bit, A.O0, A.O1, i);
                q[u].w = A.o[i];
            }
        }
#pragma unroll
        for (int u = 0; u < B8; ++u) {
            const int r = (e0 + u) * NT + tid;
            if (idx[u] >= 0) {
                rec[r] = q[u];
                rank[idx[u]] = r;
            }
            if (r < n) {
                A.start[base + r] = -1;
                A.admit_seq[base + r] = -1;
                if (stepped) {  // the event path never writes these (cleared at creation)
                    A.fin[base + r] = -1;
                    A.preempt[base + r] = 0;
                }
            }
        }
    }
}

// ------------------------------------------------------------ simulation

struct Seg {
    int n;
    const int4* __restrict__ rec;
    const int32_t* __restrict__ rank;
    const int32_t* __restrict__ a;
    int32_t* __restrict__ start;
    int32_t* __restrict__ fin;
    int32_t* __restrict__ preempt;
    int32_t* __restrict__ admit_seq;
    int4* __restrict__ act;      // running list (per-step path): record {index, s, o^, o}
    int2* __restrict__ actkr;    //   and {start step, rank}
    int32_t* __restrict__ evl;
};

// Order LDS accesses of different lanes of this wave.  LDS executes one
// wave's instructions in issue order, so only the compiler has to be stopped
// from moving accesses across this point.
__device__ __forceinline__ void lds_order() {
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
}

// Values the whole wave agrees on, kept in scalar registers.
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Wave-wide max/min with DPP: within quads, half rows and rows, then the
// row broadcasts of lanes 15 and 31; lane 63 ends with the result.  Each step
// is one DPP-modified max/min (two wait states before it: a DPP source written
// by the previous VALU instruction).  Must be called with every lane active.
__device__ __forceinline__ int wmax(int v) {
    asm volatile(
        "s_nop 1\n\t"
        "v_max_i32_dpp %0, %0, %0 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_max_i32_dpp %0, %0, %0 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_max_i32_dpp %0, %0, %0 row_half_mirror row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_max_i32_dpp %0, %0, %0 row_mirror row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_max_i32_dpp %0, %0, %0 row_bcast:15 row_mask:0xa bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_max_i32_dpp %0, %0, %0 row_bcast:31 row_mask:0xc bank_mask:0xf\n\t"
        "s_nop 1"
        : "+v"(v));
    return __builtin_amdgcn_readlane(v, 63);
}

__device__ __forceinline__ int wmin(int v) {
    asm volatile(
        "s_nop 1\n\t"
        "v_min_i32_dpp %0, %0, %0 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_min_i32_dpp %0, %0, %0 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_min_i32_dpp %0, %0, %0 row_half_mirror row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_min_i32_dpp %0, %0, %0 row_mirror row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_min_i32_dpp %0, %0, %0 row_bcast:15 row_mask:0xa bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_min_i32_dpp %0, %0, %0 row_bcast:31 row_mask:0xc bank_mask:0xf\n\t"
        "s_nop 1"
        : "+v"(v));
    return __builtin_amdgcn_readlane(v, 63);
}

// Issue priority of a wave by its remaining work.  A launch runs one
// single-wave workgroup per segment, more of them than the GPU holds at once;
// the hardware starts them in order of blockIdx as slots free up.  At equal
// priority the arbiter favours older waves, so the last waves to start are
// the last to finish and the launch drains as a long tail of ever fewer
// waves, which issue far less per cycle than a full CU.  Instead the waves
// keep one counter per launch: the number of running waves and the sum of
// their remaining requests (admissions still to make, or requests still to
// finish), updated every 32 requests and when a wave starts and ends.  A
// wave with more remaining than the mean gets a higher level (four levels,
// 1/64 of its segment apart): remaining work evens out, and the waves that
// are running when the last ones start end at about the same time.  The
// counter value used is the one returned by the wave's previous update, so
// no wave waits for it.  Issue order changes only timing: every output is
// the same at any priority.
struct IssuePrio {
    static constexpr int SH = 40;  // counter: running waves << SH | sum of remaining
    unsigned long long* ctr;
    unsigned long long pend;       // the counter as returned by the last update (lane 0)
    int n, th, next, last;

    __device__ __forceinline__ void add(unsigned long long v) {
        if (lane_id() == 0) pend = atomicAdd(ctr, v);
    }
    __device__ __forceinline__ void init(const SimArgs& P, int n_, int done) {
        next = INT32_MAX;
        ctr = nullptr;
        if (P.resident <= 0 || n_ <= 0 || P.prog == nullptr || done >= n_) return;
        ctr = P.prog;
        n = n_;
        th = max(n / 64, 1);
        last = done;
        pend = 0ull;
        add((1ull << SH) + (unsigned long long)(n - done));
        next = done + 32;
        __builtin_amdgcn_s_setprio(2);
    }
    __device__ __forceinline__ void set(int done) {
        const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)pend);
        const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(pend >> 32));
        const uint64_t c = ((uint64_t)hi << 32) | lo;
        const int64_t cnt = (int64_t)(c >> SH), sum = (int64_t)(c & ((1ull << SH) - 1ull));
        // (my remaining - mean remaining) * cnt, against the level step * cnt
        const int64_t d = (int64_t)(n - done) * cnt - sum, s = (int64_t)th * cnt;
        if (d > s) __builtin_amdgcn_s_setprio(3);
        else if (d > 0) __builtin_amdgcn_s_setprio(2);
        else if (d > -s) __builtin_amdgcn_s_setprio(1);
        else __builtin_amdgcn_s_setprio(0);
        add(0ull - (unsigned long long)(done - last));
        last = done;
        next = done + 32;
    }
    __device__ __forceinline__ void update(int done) {
        if (done >= next) set(done);
    }
    // the wave leaves the count (every exit of the simulation loop)
    __device__ __forceinline__ void leave() {
        if (ctr != nullptr) add(0ull - ((1ull << SH) + (unsigned long long)(n - last)));
    }
};

// One record at a uniform index, loaded through the scalar cache: the records
// are written by the sort before the simulation and only read while it runs.
__device__ __forceinline__ int4 record(const int4* rec, int r) {
    typedef __attribute__((address_space(4))) const int cint;
    const cint* p = (const cint*)(rec + r);
    return make_int4(p[0], p[1], p[2], p[3]);
}

__device__ __forceinline__ int4 readlane4(const int4& v, int src) {
    int4 r;
    r.x = __builtin_amdgcn_readlane(v.x, src);
    r.y = __builtin_amdgcn_readlane(v.y, src);
    r.z = __builtin_amdgcn_readlane(v.z, src);
    r.w = __builtin_amdgcn_readlane(v.w, src);
    return r;
}

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int src) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, src);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), src);
    return ((uint64_t)hi << 32) | lo;
}

// The future memory profile.  Slot tau mod H holds G[tau] = D[tau] + tau,
// where D[tau] is the memory the running requests are planned to hold at
// future step tau (a request started at k with planned length L contributes
// s + (tau - k) for tau in [k+1, k+L]; Section 3.1, eq:c2).  Storing D + tau
// turns the forward-looking check of a candidate (size s_h) started at t into
// a plain maximum: every tau in its window needs D[tau] + s_h + (tau - t) <= M,
// i.e. max G <= (M - s_h) + t.  A slot always represents the one tau of the
// current window [t+1, t+H] congruent to it; when that step becomes past the
// slot is rewritten as G = tau' for the next tau' it will represent (D = 0).
// In LDS, one wave's accesses are ordered by issue; in global memory a
// workgroup barrier (which also waits for outstanding stores) orders them.
template <bool LDS>
struct Ring {
    int32_t* p;  // H slots, then one spare slot (index H) that absorbs masked-off stores
    int H;
    int mask;
    __device__ __forceinline__ int ld(int tau) const { return p[tau & mask]; }
    __device__ __forceinline__ void st(int tau, int v) const { p[tau & mask] = v; }
    // store only if ok; otherwise the value goes to the spare slot (no branch)
    __device__ __forceinline__ void st_if(bool ok, int tau, int v) const {
        p[ok ? (tau & mask) : H] = v;
    }
    __device__ __forceinline__ static void order() {
        if (LDS) lds_order(); else __syncthreads();
    }
    // Visit the window [t+1, t+len] (len <= H) as at most two runs of
    // consecutive slots: op(first slot, run length, tau of the first slot).
    template <class Op>
    __device__ __forceinline__ void runs(int t, int len, Op op) const {
        const int s0 = uni((t + 1) & mask);
        const int L1 = uni(min(len, H - s0));
        op(s0, L1, t + 1);
        if (len > L1) op(0, uni(len - L1), uni(t + 1 + L1));
    }
};

// Lowest set bit of the two-level rank bitmap, or -1.
__device__ __forceinline__ int bitmap_first(const uint64_t* B, const uint64_t* S, int W1) {
    const int lane = lane_id();
    for (int base = 0; base < W1; base += 64) {
        const uint64_t v = (base + lane < W1) ? S[base + lane] : 0ull;
        const uint64_t m = ballot(v != 0ull);
        if (m) {
            const int f = __builtin_ctzll(m);
            const uint64_t sv = readlane64(v, f);
            const int w = (base + f) * 64 + __builtin_ctzll(sv);
            const uint64_t bw = B[w];
            const uint32_t lo = (uint32_t)uni((int)(uint32_t)bw);
            const uint32_t hi = (uint32_t)uni((int)(uint32_t)(bw >> 32));
            return w * 64 + __builtin_ctzll(((uint64_t)hi << 32) | lo);
        }
    }
    return -1;
}

__device__ __forceinline__ void bitmap_set_atomic(uint64_t* B, uint64_t* S, int r) {
    const int w = r >> 6;
    atomicOr((unsigned long long*)&B[w], 1ull << (r & 63));
    atomicOr((unsigned long long*)&S[w >> 6], 1ull << (w & 63));
}

// called by one lane
__device__ __forceinline__ void bitmap_clear(uint64_t* B, uint64_t* S, int r) {
    const int w = r >> 6;
    const uint64_t nb = B[w] & ~(1ull << (r & 63));
    B[w] = nb;
    if (nb == 0ull) S[w >> 6] &= ~(1ull << (w & 63));
}

// Largest G over the window [t+1, t+len], per lane (INT32_MIN if empty).
// Runs are walked in uniform blocks of 256 slots (four per lane, two paired
// LDS reads), then a predicated tail.
template <bool LDS>
__device__ __forceinline__ int window_max(const Ring<LDS>& R, int t, int len) {
    const int lane = lane_id();
    int m = INT32_MIN;
    R.runs(t, len, [&](int s, int L, int) {
        const int32_t* q = R.p + s + lane;
        const int nb = L >> 8;
        for (int b = 0; b < nb; ++b, q += 256)
            m = max(m, max(max(q[0], q[64]), max(q[128], q[192])));
        const int rem = L & 255;
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (lane + 64 * u < rem) m = max(m, q[64 * u]);
    });
    return m;
}

// Scan of the window [t+1, t+len] in batches of 64*NB slots (NB loads per
// lane in flight): MODE 0 takes the largest G, MODE 1 the largest
// min(tau, G - X), MODE 2 both.
template <int NB, int MODE, bool LDS>
__device__ __forceinline__ void window_scan(const Ring<LDS>& R, int t, int len, int X, int& m,
                                            int& rel) {
    const int lane = lane_id();
    R.runs(t, len, [&](int s, int L, int tau0) {
        const int32_t* q = R.p + s + lane;
        int tau = tau0 + lane;
        int b = 0;
        for (; b + 64 * NB <= L; b += 64 * NB, q += 64 * NB, tau += 64 * NB) {
            int x[NB];
#pragma unroll
            for (int u = 0; u < NB; ++u) x[u] = q[64 * u];
#pragma unroll
            for (int u = 0; u < NB; ++u) {
                if (MODE != 1) m = max(m, x[u]);
                if (MODE != 0) rel = max(rel, min(tau + 64 * u, x[u] - X));
            }
        }
        for (; b + 256 <= L; b += 256, q += 256, tau += 256) {
            int x[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) x[u] = q[64 * u];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                if (MODE != 1) m = max(m, x[u]);
                if (MODE != 0) rel = max(rel, min(tau + 64 * u, x[u] - X));
            }
        }
        const int rem = uni(L - b);
        if (rem > 0) {
            const int base = s + b + lane;
            int x[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) x[u] = R.p[min(base + 64 * u, R.H - 1)];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const bool in = lane + 64 * u < rem;
                if (MODE != 1) m = max(m, in ? x[u] : INT32_MIN);
                if (MODE != 0) rel = max(rel, in ? min(tau + 64 * u, x[u] - X) : INT32_MIN);
            }
        }
    });
}

// Add c0 + SLOPE * tau (SLOPE = +1 or -1) to every slot of the window
// [t+1, t+len] (len <= H), in batches of 64*NB slots, then 256, then a tail
// with clamped loads and masked-off stores to the spare slot.
template <int NB, int SLOPE, bool LDS>
__device__ __forceinline__ void window_add(const Ring<LDS>& R, int t, int len, int c0) {
    const int lane = lane_id();
    R.runs(t, len, [&](int s, int L, int tau0) {
        int32_t* q = R.p + s + lane;
        int c = c0 + SLOPE * (tau0 + lane);
        int b = 0;
        for (; b + 64 * NB <= L; b += 64 * NB, q += 64 * NB, c += SLOPE * 64 * NB) {
            int x[NB];
#pragma unroll
            for (int u = 0; u < NB; ++u) x[u] = q[64 * u];
#pragma unroll
            for (int u = 0; u < NB; ++u) q[64 * u] = x[u] + c + SLOPE * 64 * u;
        }
        for (; b + 256 <= L; b += 256, q += 256, c += SLOPE * 256) {
            int x[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) x[u] = q[64 * u];
#pragma unroll
            for (int u = 0; u < 4; ++u) q[64 * u] = x[u] + c + SLOPE * 64 * u;
        }
        const int rem = uni(L - b);
        if (rem > 0) {
            const int base = s + b + lane;
            int x[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) x[u] = R.p[min(base + 64 * u, R.H - 1)];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const bool ok = lane + 64 * u < rem;
                R.p[ok ? base + 64 * u : R.H] = x[u] + c + SLOPE * 64 * u;
            }
        }
    });
    Ring<LDS>::order();
}

// fit_and_admit for windows of at most 64*U steps: one LDS round trip with U
// loads per lane in flight, values kept in registers for the update.
template <int U, bool LDS>
__device__ __forceinline__ bool fit_small(const Ring<LDS>& R, int t, int s_h, int oh, int len,
                                          int live, int X, int lim, int extra1, int* t_free) {
    const int lane = lane_id();
    int g[U];
    int m = INT32_MIN;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int j = lane + 64 * u;
        const int tau = t + 1 + j;
        const int x = R.ld(tau);
        g[u] = j < live ? x : tau;  // beyond maxF the slot holds tau (D = 0)
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int j = lane + 64 * u;
        const int v = g[u] + (j == 0 ? extra1 : 0);
        m = max(m, j < len ? v : INT32_MIN);
    }
    if (ballot(m > lim) != 0ull) {
        // the release step, from the values still in registers
        int rel = INT32_MIN;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int j = lane + 64 * u;
            const int v = g[u] + (j == 0 ? extra1 : 0);
            rel = max(rel, j < len ? min(t + 1 + j, v - X) : INT32_MIN);
        }
        *t_free = wmax(rel);
        return false;
    }
    const int c = s_h - t;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int j = lane + 64 * u;
        const int tau = t + 1 + j;
        R.st_if(j < oh, tau, g[u] + c + tau);
    }
    Ring<LDS>::order();
    return true;
}

// Forward-looking check of a candidate (size s_h, planned length oh) started
// at step t, and its admission when it fits; chk = 1 checks the next step
// only (current-capacity admission).  extra1 is memory held at t+1
// only (requests past their planned length).  maxF is a step after which no
// running request is planned to hold memory (D = 0 there, so the candidate
// alone, s_h + oh <= M, always fits); the check stops there.  If the
// candidate fits, its growth s_h + (tau - t) is added over its whole window
// and true is returned.  Otherwise *t_free receives the first step at which
// every violation has disappeared while the profile stays unchanged: a
// violation at tau persists while tau is ahead and the start is earlier than
// G[tau] - (M - s_h); max_tau min(tau, G[tau] - X) over the window is that
// step (steps that do not violate contribute at most t).
// Windows of at most 512 steps take one LDS round trip (fit_small).
template <bool LDS>
__device__ __forceinline__ bool fit_and_admit(const Ring<LDS>& R, int t, int s_h, int oh, int M,
                                              int extra1, int maxF, int* t_free, int chk = 1 << 30) {
    const int X = M - s_h;
    const int lim = X + t;
    // steps of the candidate's window that hold planned memory, and the part checked
    const int live = uni(max(0, min(oh, maxF - t)));
    int len = min(live, chk);
    if (extra1 != 0) len = max(len, 1);  // step t+1 always carries extra1
    len = uni(len);
    const int ld = max(len, live);
    if (oh <= 64) return fit_small<1>(R, t, s_h, oh, len, ld, X, lim, extra1, t_free);
    if (oh <= 128) return fit_small<2>(R, t, s_h, oh, len, ld, X, lim, extra1, t_free);
    if (oh <= 256) return fit_small<4>(R, t, s_h, oh, len, ld, X, lim, extra1, t_free);
    if (oh <= 512) return fit_small<8>(R, t, s_h, oh, len, ld, X, lim, extra1, t_free);
    // longer windows: the check takes only the maximum; the release step is
    // computed in a second pass when the candidate does not fit
    int m = INT32_MIN, rel = INT32_MIN;
    window_scan<16, 0>(R, t, len, X, m, rel);
    if (extra1 != 0) m = max(m, R.ld(t + 1) + extra1);
    if (ballot(m > lim) != 0ull) {
        window_scan<16, 1>(R, t, len, X, m, rel);
        if (extra1 != 0) rel = max(rel, min(t + 1, R.ld(t + 1) + extra1 - X));
        *t_free = wmax(rel);
        return false;
    }
    window_add<16, 1>(R, t, oh, s_h - t);
    return true;
}

// Remove the planned profile of a request started at k with planned length L
// for the future steps tau in [t+1, k+L].
template <bool LDS>
__device__ __forceinline__ void remove_future(const Ring<LDS>& R, int t, int s, int k, int L) {
    window_add<16, -1>(R, t, k + L - t, k - s);
}

// Fold the past steps (lo, hi] (hi <= t): their memory is final; add it to
// the per-lane peak and relabel each slot for the step H later.  Steps are
// visited in increasing order, so a slot met twice (hi - lo > H) is relabelled
// twice in order.
template <int U, bool LDS>
__device__ __forceinline__ void fold_block(const Ring<LDS>& R, int b, int hi, int& peak_lane) {
    const int lane = lane_id();
    int x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) x[u] = R.ld(b + lane + 64 * u);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int tau = b + lane + 64 * u;
        const bool ok = tau <= hi;
        peak_lane = max(peak_lane, ok ? x[u] - tau : 0);
        R.st_if(ok, tau, tau + R.H);
    }
    // a slot can come round again H steps later in the same fold
    Ring<LDS>::order();
}

template <bool LDS>
__device__ __forceinline__ void fold_range(const Ring<LDS>& R, int lo, int hi, int& peak_lane) {
    int b = lo + 1;
    for (; hi - b >= 1023; b += 1024) fold_block<16>(R, b, hi, peak_lane);
    for (; hi - b >= 255; b += 256) fold_block<4>(R, b, hi, peak_lane);
    for (; b <= hi; b += 64) fold_block<1>(R, b, hi, peak_lane);
}

// ---- known lengths: event-driven

// The event path keeps the future memory profile of the running requests in
// one of two forms (chosen per batch by the host from the LDS each needs):
// the ring of G = D + tau values (RingProf) or a list of the running requests
// ordered by planned finish (ListProf).  Both offer begin (at each visited
// step, before admissions), fit (the forward-looking check of a candidate
// started at t, and its admission when it fits; *t_free as in fit_and_admit
// otherwise, or -1: the segment has to leave the launch at the current step)
// and end (the peak of the steps up to t).

template <bool LDS>
struct RingProf {
    const Ring<LDS>& D;
    int folded;     // slots of steps <= folded are labelled for the current window
    int peak_lane;  // per-lane largest memory total of the folded steps
    __device__ __forceinline__ RingProf(const Ring<LDS>& d, int t) : D(d), folded(t), peak_lane(0) {}
    __device__ __forceinline__ void begin(int) {}
    __device__ __forceinline__ bool fit(int t, int s_h, int oh, int M, int maxF, int* t_free) {
        // slots up to t + oh must be labelled for the current window
        if (t + oh - D.H > folded) {
            const int to = min(t, t + oh - D.H + 512);
            fold_range(D, folded, to, peak_lane);
            folded = to;
        }
        return fit_and_admit(D, t, s_h, oh, M, 0, maxF, t_free);
    }
    __device__ __forceinline__ int end(int t) {
        // every past step folded: the ring is canonical again
        fold_range(D, folded, t, peak_lane);
        return wmax(peak_lane);
    }
};

// The running requests sorted by planned finish F, latest first (entry 0 has
// the largest F), with Q_j = sum over the entries 0..j of (s - k), k the step a
// request was started at, in wrapping 32-bit arithmetic (every quantity formed
// from it fits in int32).  The memory at step tau is D(tau) = sum over running
// requests with F >= tau of (s - k + tau).  Between two finish steps it grows with tau, so the check of
// a candidate (size s_h, planned length oh) started at t needs only the steps
// tau = F_j <= te = t + oh and tau = te:
//   D(F_j) + F_j = Q_j + F_j (j + 2)      (the entries 0..j have F >= F_j),
//   D(te) + te   = Q_{c-1} + te (c + 1)   (c entries have F >= te),
// each at most M - s_h + t (Appendix E.2, eq:c2).  These are the last entries
// of the list, read from the end in groups of 64 until an entry with F > te
// shows up; a short candidate touches one group.  Admission inserts the
// candidate at c: the entries behind it move up by one and gain s_h - t in
// Q.  Requests finished by t are the last entries and are dropped at each
// visited step; D at their finish step goes into the peak.  The host bounds
// the requests that can run at once; the list in LDS may hold fewer (more
// waves then fit on a compute unit).  A candidate that fits into a full list
// gets *t_free = -1 (a real failure always gives a step after t): the segment
// stops at that step with the candidate as the head, and a later launch with
// room for the bound continues it.
//
// Every lane of a group takes part in every step, so that no lane is masked
// off (the scalar unit, which would juggle the masks, is the busiest unit of
// this kernel): lanes past the last entry of a group read a copy of that
// entry, which leaves maxima unchanged and is taken out of counts, and the
// shift of an insertion writes each lane's entry to a position of its own (a
// lane whose entry stays rewrites it in place; the lane of entry c-1 writes
// the candidate; lanes past the group's end write to a slot of their own
// behind the capacity, so the arrays have 65 slots more than the list may
// hold).
struct ListProf {
    int32_t* F;     // [list_slots(cap)] planned finish, descending
    uint32_t* Q;    // [list_slots(cap)] prefix sums of s - k
    int cap;        // capacity
    int ln;         // entries
    uint32_t tot;   // Q of the last entry (0 if none)
    int peak_lane;
    __device__ __forceinline__ void begin(int t) {
        const int lane = lane_id();
        while (ln > 0) {
            const int top = ln, base = max(top - 64, 0);
            const int jr = min(base + lane, top - 1);
            const int f = F[jr];
            const uint32_t q = Q[jr];
            const bool done = f <= t;
            const uint64_t dm = ballot(done);
            if (dm == 0ull) break;
            // the memory at the finish step of a finished request
            peak_lane = max(peak_lane, done ? (int)(q + (uint32_t)f * (uint32_t)(jr + 1)) : 0);
            // the finished ones end the group; copies of the last entry are
            // among them
            ln = top - ((int)__popcll(dm) - (64 - (top - base)));
            if (ln > base) {
                tot = (uint32_t)__builtin_amdgcn_readlane((int)q, ln - 1 - base);
                break;
            }
            if (ln == 0) {
                tot = 0u;
                if (lane == 0) F[0] = INT32_MAX;  // an empty list reads as "finishes last"
                lds_order();
            }
        }
    }
    __device__ __forceinline__ bool fit(int t, int s_h, int oh, int M, int maxF, int* t_free) {
        (void)maxF;
        const int lane = lane_id();
        const int te = t + oh;
        const int X = M - s_h;
        const int lim = X + t;
        // groups of 64 entries from the end, down to the one holding an entry
        // with F > te (its first entry has the largest F) or the first entry
        int m = INT32_MIN;
        int top = ln, base, f, jr;
        uint32_t q;
        for (;;) {
            base = max(top - 64, 0);
            jr = min(base + lane, max(top - 1, 0));
            f = F[jr];
            q = Q[jr];
            m = max(m, f <= te ? (int)(q + (uint32_t)f * (uint32_t)(jr + 2)) : INT32_MIN);
            if (base == 0) break;
            if (__builtin_amdgcn_readfirstlane(f) > te) break;
            top = base;
        }
        // c = entries with F >= te (a prefix of the group, copies excluded)
        const int ge = min((int)__popcll(ballot(f >= te)), top - base);
        const int c = base + ge;
        const uint32_t qc1 = ge > 0 ? (uint32_t)__builtin_amdgcn_readlane((int)q, ge - 1) : 0u;
        const int ve = (int)(qc1 + (uint32_t)te * (uint32_t)(c + 1));
        if (ballot(max(m, ve) > lim) != 0ull) {
            // the release step: max over the violating steps of min(tau, D + tau - X),
            // over the same groups again (base: the lowest one scanned)
            int rel = min(te, ve - X);
            if (top == ln) {  // one group, still in the registers
                const int v = (int)(q + (uint32_t)f * (uint32_t)(jr + 2));
                rel = max(rel, f <= te ? min(f, v - X) : INT32_MIN);
            } else {
                for (int tp = ln;;) {
                    const int b = max(tp - 64, 0);
                    const int jj = min(b + lane, tp - 1);
                    const int ff = F[jj];
                    const int v = (int)(Q[jj] + (uint32_t)ff * (uint32_t)(jj + 2));
                    rel = max(rel, ff <= te ? min(ff, v - X) : INT32_MIN);
                    if (b <= base) break;
                    tp = b;
                }
            }
            *t_free = wmax(rel);
            return false;
        }
        if (ln >= cap) {
            *t_free = -1;
            return false;
        }
        // the entries c .. ln-1 move up by one and gain s_h - t, group by
        // group from the end (no entry is overwritten unread); entry c-1
        // writes the candidate behind itself
        const uint32_t ch = (uint32_t)(s_h - t);
        const uint32_t qn = qc1 + ch;
        auto shift = [&](int b, int tp, int ff, uint32_t qq) {
            const int j = b + lane;
            const bool mv = j >= c - 1;
            const bool nw = j == c - 1;
            // lanes past the group's end: a slot of their own behind the capacity
            const int pos = j < tp ? (mv ? j + 1 : j) : cap + 1 + lane;
            F[pos] = nw ? te : ff;
            Q[pos] = nw ? qn : (mv ? qq + ch : qq);
        };
        if (top == ln) {
            // the check read only the last group, which holds entry c-1 (or
            // is the first group): shift it from the registers
            shift(base, top, f, q);
        } else {
            // groups down to the one holding entry max(c-1, 0)
            const int groups = max((ln - max(c - 1, 0) + 63) >> 6, 1);
            for (int g = 0, tp = ln; g < groups; ++g, tp -= 64) {
                const int b = max(tp - 64, 0);
                const int jj = min(b + lane, max(tp - 1, 0));
                shift(b, tp, F[jj], Q[jj]);
            }
        }
        if (c == 0) {  // no entry before the candidate (every lane stores the same values)
            F[0] = te;
            Q[0] = qn;
        }
        lds_order();
        ++ln;
        tot += ch;
        return true;
    }
    __device__ __forceinline__ int end(int t) {
        begin(t);
        // the memory at step t of the requests still running
        if (ln > 0) peak_lane = max(peak_lane, (int)(tot + (uint32_t)t * (uint32_t)ln));
        return wmax(peak_lane);
    }
};


template <class PROF>
__device__ void run_known(const SimArgs& P, const Seg& sg, uint64_t* B, uint64_t* S, int W1,
                          PROF& prof, SegState& st, int t_lim) {
    const int lane = lane_id();
    const int M = P.M;
    const int n = sg.n;
    // admissions so far: seq0 + nstg (known lengths: every admitted request
    // is finished at start + o, so no other count is needed)
    int t = uni(st.t), cursor = uni(st.cursor), seq0 = uni(st.seq);
    int max_fin = uni(st.max_fin), head = uni(st.head_rank), t_f = uni(st.t_f);
    int status = STATUS_RUNNING;

    // Arrival window: lane l holds request wb + l (arrival, rank, record).
    int wb = 0, a_reg = INT32_MAX, rk_reg = 0;
    int4 aq = make_int4(0, 0, 0, 0);
    auto load_arrivals = [&](int base) {
        wb = uni(base);
        const int i = base + lane;
        a_reg = INT32_MAX;
        rk_reg = 0;
        if (i < n) {
            a_reg = sg.a[i];
            rk_reg = sg.rank[i];
            if ((unsigned)rk_reg >= (unsigned)n) rk_reg = 0;  // only a broken sort
            aq = sg.rec[rk_reg];
        }
    };
    load_arrivals(cursor);

    // the record of one rank: a scalar load (read-only while the simulation runs)
    auto rec_of = [&](int r) -> int4 { return record(sg.rec, r); };
    int4 hq = make_int4(0, 0, 0, 0);  // record of the blocked head
    if (head >= 0) hq = rec_of(head);
    // Admissions are staged in registers, lane j holding the j-th of up to 64
    // (request index and start step), and written out 64 at a time with their
    // admission numbers, so that no store is in flight behind each admission;
    // the finish (start + o) is derived when the outputs are finalised.
    int stg_idx = 0, stg_t = 0, nstg = 0;
    IssuePrio prio;
    prio.init(P, n, seq0);
    auto flush = [&]() {
        if (lane < nstg) {
            sg.start[stg_idx] = stg_t;
            sg.admit_seq[stg_idx] = seq0 + lane;
        }
        seq0 += nstg;
        nstg = 0;
        prio.update(seq0);
    };

    // Bitmap word of the current candidate, mirrored in scalar registers for
    // the admission loop of one step (nothing else writes the bitmap there).
    int cw = -1;
    uint64_t cbits = 0ull;
    auto load_word = [&](int w) {
        const uint64_t v = B[w];
        const uint32_t lo = (uint32_t)uni((int)(uint32_t)v);
        const uint32_t hi = (uint32_t)uni((int)(uint32_t)(v >> 32));
        cbits = ((uint64_t)hi << 32) | lo;
        cw = w;
    };

    for (;;) {
        // every request finished by step t-1 (an empty instance is done at t = 0)
        if (seq0 + nstg == n) {
            if (n == 0 || max_fin <= t - 1) { status = STATUS_DONE; break; }
        }
        if (t > P.max_steps) { status = STATUS_EXHAUSTED; break; }
        if (t >= t_lim) break;

        // 1. arrivals up to t: a prefix of the window (arrivals are sorted;
        //    those of earlier steps were ranked below the blocked head, so
        //    nothing could happen at their steps).  n_below counts those
        //    ranked above the blocked head (the lowest waiting rank before
        //    this step; none if nothing was waiting).
        const int old_head = head < 0 ? INT32_MAX : head;
        int new_min = INT32_MAX, n_below = 0;
        int4 nq = make_int4(0, 0, 0, 0);
        for (;;) {
            const bool arr = (wb + lane >= cursor) && (a_reg <= t);
            const uint64_t m = ballot(arr);
            if (m == 0ull) break;
            if (arr) bitmap_set_atomic(B, S, rk_reg);
            n_below += __popcll(ballot(arr && rk_reg < old_head));
            int mn, src;
            if ((m & (m - 1ull)) == 0ull) {  // a single arrival
                src = __builtin_ctzll(m);
                mn = __builtin_amdgcn_readlane(rk_reg, src);
            } else {
                mn = wmin(arr ? rk_reg : INT32_MAX);
                src = __builtin_ctzll(ballot(arr && rk_reg == mn));
            }
            if (mn < new_min) {
                new_min = mn;
                nq = readlane4(aq, src);
            }
            cursor += __popcll(m);
            if (cursor < wb + 64) break;
            load_arrivals(cursor);
        }
        lds_order();

        // 4. admissions (known lengths: completions change nothing ahead)
        if (new_min < old_head || (head >= 0 && t >= t_f)) {
            int r = head;
            int4 q = hq;
            if (new_min < old_head) { r = new_min; q = nq; }
            load_word(r >> 6);  // arrivals may have changed any word
            prof.begin(t);
            for (;;) {
                int tf = 0;
                if (!prof.fit(t, q.y, q.z, M, max_fin, &tf)) { head = r; hq = q; t_f = tf; break; }
                if (lane == nstg) {
                    stg_idx = q.x;
                    stg_t = t;
                }
                if (++nstg == 64) flush();
                cbits &= ~(1ull << (r & 63));
                // every lane stores the same word (no lane mask to set up)
                B[cw] = cbits;
                if (cbits == 0ull) S[cw >> 6] &= ~(1ull << (cw & 63));
                lds_order();
                max_fin = max(max_fin, t + q.w);
                // Once every arrival ranked above the old head is running, the
                // old head is next, or nothing is left waiting.
                // Before t_f it still does not fit: the profile has only grown
                // since t_f was computed, which can only delay the release.
                // (Candidates come in rank order, so the first n_below of them
                // are exactly those arrivals.)
                // (n_below <= 0 stays below zero)
                if (--n_below == 0) {
                    if (old_head == INT32_MAX) { head = -1; break; }
                    if (t < t_f) break;
                    // the old head is now the lowest waiting rank: found below
                }
                if (cbits != 0ull) {
                    r = cw * 64 + __builtin_ctzll(cbits);
                } else {
                    r = bitmap_first(B, S, W1);
                    if (r < 0) { head = -1; break; }
                    load_word(r >> 6);
                }
                q = rec_of(r);
            }
        }

        // a full list: the candidate is the head, checked again at t when the
        // segment resumes
        if (t_f < 0) break;

        // 5. advance to the next step where anything can happen: with a
        //    blocked head, its release or the next arrival ranked above it
        //    (past the window: the window's end)
        int nt;
        if (head >= 0) {
            const uint64_t up = ballot((wb + lane >= cursor) && rk_reg < head);
            const int next_up = up != 0ull ? __builtin_amdgcn_readlane(a_reg, __builtin_ctzll(up))
                                           : (wb + 64 < n ? uni(sg.a[wb + 64]) : INT32_MAX);
            nt = min(t_f, next_up);
        } else if (cursor < n) {
            nt = cursor < wb + 64 ? __builtin_amdgcn_readlane(a_reg, cursor - wb) : uni(sg.a[cursor]);
        } else {
            nt = max_fin + 1;
        }
        nt = max(nt, t + 1);
        nt = min(nt, t_lim);
        nt = min(nt, P.max_steps + 1);
        if (nt <= t) nt = t + 1;
        t = uni(nt);
    }
    flush();
    prio.leave();
    // the peak over the steps up to t
    const int pk = prof.end(t);
    st.t = t; st.cursor = cursor; st.seq = seq0; st.nfin = seq0; st.max_fin = max_fin;
    st.head_rank = head; st.t_f = t_f; st.status = status;
    st.peak = max(st.peak, (int64_t)pk);
}

// ---- planned lengths differ from the truth: one step at a time

// The per-step path keeps the planned memory of the requests that are still
// within their planned length (each started at k with planned length L holds
// s + tau - k at the steps tau in [k+1, k+L]) in one of two forms: the ring
// (RingStep) or the finish-ordered list (StepList).  Both offer begin (at
// step t, before anything reads the profile: requests whose planned length
// ends by t leave it), next (their memory at step t+1), fit (the check of a
// candidate over the steps t+1 .. t+min(oh, chk), with extra1 added at t+1,
// and its admission for its whole planned length; *t_free as in
// fit_and_admit), remove (a request's planned memory after t) and end_step.
template <bool LDS>
struct RingStep {
    const Ring<LDS>& D;
    __device__ __forceinline__ explicit RingStep(const Ring<LDS>& d) : D(d) {}
    __device__ __forceinline__ void begin(int) {}
    __device__ __forceinline__ int64_t next(int t) const { return (int64_t)D.ld(t + 1) - (t + 1); }
    __device__ __forceinline__ bool fit(int t, int s_h, int oh, int M, int extra1, int maxF,
                                        int* t_free, int chk) {
        return fit_and_admit(D, t, s_h, oh, M, extra1, maxF, t_free, chk);
    }
    __device__ __forceinline__ void remove(int t, int s, int k, int L) { remove_future(D, t, s, k, L); }
    // the next step is tn > t: the slots of steps t+1 .. tn become those of
    // steps t+1+H .. tn+H (nothing is planned that far; the last H of them
    // when more than H steps pass)
    __device__ __forceinline__ void end_step(int t, int tn) {
        Ring<LDS>::order();
        const int J = tn - t;
        if (J == 1) {
            if (lane_id() == 0) D.st(t + 1, t + 1 + D.H);
        } else {
            for (int x = max(J - D.H, 0) + lane_id(); x < J; x += 64) D.st(t + 1 + x, t + 1 + x + D.H);
        }
        Ring<LDS>::order();
    }
};

// The list of the event path, with what the per-step path needs besides:
// entries leave at their planned finish (the request then either completes
// or runs on past its plan, which the caller accounts for), an entry can be
// removed from the middle (early completion, eviction), the check may stop
// short of the candidate's planned finish (next-step admission) and carries
// the memory of the requests past their plan at t+1.  As on the event path,
// the LDS may hold fewer entries than the host's bound: a candidate that fits
// into a full list gets *t_free = -1 (a real failure always gives a step
// after t), which stops the segment inside the admission phase of its step;
// a launch with room for the bound resumes it there.
struct StepList {
    int32_t* F;     // [list_slots(cap)] planned finish, descending
    uint32_t* Q;    // [list_slots(cap)] prefix sums of s - k
    int cap;
    int ln;
    uint32_t tot;
    struct Scan {
        int m, base, top, f, jr, c;
        uint32_t q, qc1;
    };
    // Groups of 64 from the end down to the one holding an entry with F > tx
    // (or the first): m = the lanes' largest D(F_j) + F_j over F_j <= tx, c =
    // #{F >= tx}, qc1 = Q_{c-1} (0 if c = 0).
    __device__ __forceinline__ Scan scan_to(int tx) const {
        const int lane = lane_id();
        Scan r;
        r.m = INT32_MIN;
        r.top = ln;
        for (;;) {
            r.base = max(r.top - 64, 0);
            r.jr = min(r.base + lane, max(r.top - 1, 0));
            r.f = F[r.jr];
            r.q = Q[r.jr];
            r.m = max(r.m, r.f <= tx ? (int)(r.q + (uint32_t)r.f * (uint32_t)(r.jr + 2)) : INT32_MIN);
            if (r.base == 0) break;
            if (__builtin_amdgcn_readfirstlane(r.f) > tx) break;
            r.top = r.base;
        }
        const int ge = min((int)__popcll(ballot(r.f >= tx)), r.top - r.base);
        r.c = r.base + ge;
        r.qc1 = ge > 0 ? (uint32_t)__builtin_amdgcn_readlane((int)r.q, ge - 1) : 0u;
        return r;
    }
    __device__ __forceinline__ void begin(int t) {
        const int lane = lane_id();
        if (ln == 0 || __builtin_amdgcn_readfirstlane(F[ln - 1]) > t) return;
        while (ln > 0) {
            const int top = ln, base = max(top - 64, 0);
            const int jr = min(base + lane, top - 1);
            const uint64_t dm = ballot(F[jr] <= t);
            if (dm == 0ull) break;
            const uint32_t q = Q[jr];
            ln = top - ((int)__popcll(dm) - (64 - (top - base)));
            if (ln > base) {
                tot = (uint32_t)__builtin_amdgcn_readlane((int)q, ln - 1 - base);
                break;
            }
            if (ln == 0) {
                tot = 0u;
                if (lane == 0) F[0] = INT32_MAX;  // an empty list reads as "finishes last"
                lds_order();
            }
        }
    }
    // all entries have F >= t+1 (begin(t) ran)
    __device__ __forceinline__ int64_t next(int t) const {
        return (int64_t)(int)(tot + (uint32_t)ln * (uint32_t)(t + 1));
    }
    __device__ __forceinline__ bool fit(int t, int s_h, int oh, int M, int extra1, int maxF,
                                        int* t_free, int chk) {
        (void)maxF;
        const int lane = lane_id();
        const int te = t + oh;
        const int tc = t + min(oh, chk);  // the last step checked
        const int X = M - s_h;
        const int lim = X + t;
        // step t+1 with the memory of the requests past their plan
        const int v1 = (int)(tot + (uint32_t)(ln + 1) * (uint32_t)(t + 1)) + extra1;
        Scan a = scan_to(tc);
        const int vc = (int)(a.qc1 + (uint32_t)tc * (uint32_t)(a.c + 1));
        if (ballot(max(a.m, max(vc, v1)) > lim) != 0ull) {
            // the release step: max over the violating steps of min(tau, D + tau - X)
            int rel = max(min(tc, vc - X), min(t + 1, v1 - X));
            if (a.top == ln) {
                const int v = (int)(a.q + (uint32_t)a.f * (uint32_t)(a.jr + 2));
                rel = max(rel, a.f <= tc ? min(a.f, v - X) : INT32_MIN);
            } else {
                for (int tp = ln;;) {
                    const int b = max(tp - 64, 0);
                    const int jj = min(b + lane, tp - 1);
                    const int ff = F[jj];
                    const int v = (int)(Q[jj] + (uint32_t)ff * (uint32_t)(jj + 2));
                    rel = max(rel, ff <= tc ? min(ff, v - X) : INT32_MIN);
                    if (b <= a.base) break;
                    tp = b;
                }
            }
            *t_free = wmax(rel);
            return false;
        }
        if (ln >= cap) {
            *t_free = -1;
            return false;
        }
        // the candidate goes in at its planned finish te
        if (tc != te) a = scan_to(te);
        const int c = a.c;
        const uint32_t ch = (uint32_t)(s_h - t);
        const uint32_t qn = a.qc1 + ch;
        auto shift = [&](int b, int tp, int ff, uint32_t qq) {
            const int j = b + lane;
            const bool mv = j >= c - 1;
            const bool nw = j == c - 1;
            const int pos = j < tp ? (mv ? j + 1 : j) : cap + 1 + lane;
            F[pos] = nw ? te : ff;
            Q[pos] = nw ? qn : (mv ? qq + ch : qq);
        };
        if (a.top == ln) {
            shift(a.base, a.top, a.f, a.q);
        } else {
            const int groups = max((ln - max(c - 1, 0) + 63) >> 6, 1);
            for (int g = 0, tp = ln; g < groups; ++g, tp -= 64) {
                const int b = max(tp - 64, 0);
                const int jj = min(b + lane, max(tp - 1, 0));
                shift(b, tp, F[jj], Q[jj]);
            }
        }
        if (c == 0) {
            if (lane == 0) {
                F[0] = te;
                Q[0] = qn;
            }
        }
        lds_order();
        ++ln;
        tot += ch;
        return true;
    }
    // Remove the entry of a request started at k with planned length L
    // (planned finish k + L > t); entries with equal F and s - k are
    // interchangeable.
    __device__ __forceinline__ void remove(int t, int s, int k, int L) {
        (void)t;
        const int lane = lane_id();
        const int fd = k + L;
        const uint32_t cd = (uint32_t)(s - k);
        // find it: groups from the end (its F is at least that of the last entry)
        int p = -1;
        for (int top = ln; top > 0;) {
            const int base = max(top - 64, 0);
            const int j = base + lane;
            const int jr = min(j, top - 1);
            const int f = F[jr];
            const uint32_t qp = jr > 0 ? Q[jr - 1] : 0u;
            const uint64_t hit = ballot(j < top && f == fd && Q[jr] - qp == cd);
            if (hit != 0ull) {
                p = base + (int)__builtin_ctzll(hit);
                break;
            }
            if (base == 0 || __builtin_amdgcn_readfirstlane(f) > fd) break;
            top = base;
        }
        if (p < 0) return;  // not in the list (cannot happen)
        // entries p+1 .. ln-1 move down by one and lose s - k
        for (int b = p; b < ln; b += 64) {
            const int j = b + lane;
            const int jr = min(j, ln - 1);
            const int f = F[jr];
            const uint32_t q = Q[jr];
            const int pos = (j > p && j < ln) ? j - 1 : cap + 1 + lane;
            F[pos] = f;
            Q[pos] = q - cd;
        }
        lds_order();
        --ln;
        tot -= cd;
        if (ln == 0) {
            if (lane == 0) F[0] = INT32_MAX;
            lds_order();
        }
    }
    __device__ __forceinline__ void end_step(int, int) {}
};


// The running list (global memory, small enough to stay in L2): entry x
// holds the record {index, s, planned length, true length} of a running
// request and {start step, rank}.
struct RunList {
    int4* q;
    int2* kr;
    // Entries written by one lane are read by others next.  The list is read
    // and written by the lanes of one wave only, which see
    // each other's memory operations in program order without waiting; the
    // fence keeps the compiler from reordering them.
    __device__ __forceinline__ static void order() { lds_order(); }
};

// STOP: the profile may fill up (a list with less room than the host's
// bound); the segment then leaves the launch inside the step.
template <bool STOP, class PROF>
__device__ void run_stepped(const SimArgs& P, const Seg& sg, uint64_t* B, uint64_t* S, int W1,
                            PROF& D, const RunList& A, SegState& st, int t_lim) {
    const int lane = lane_id();
    const int M = P.M;
    const int n = sg.n;
    int t = uni(st.t), cursor = uni(st.cursor), seq = uni(st.seq), nfin = uni(st.nfin);
    int nA = uni(st.nA), N_O = uni(st.N_O);
    int64_t C_O = st.C_O, peak = st.peak, req_steps = st.req_steps;
    int status = STATUS_RUNNING;
    // no request admitted so far is planned to hold memory after step maxF
    int maxF = uni(st.max_fin);
    // current-capacity admission checks the next step only
    const int pol = blockIdx.x / P.I;
    const int chk = (P.policies[pol] & ADMIT_CURRENT) ? 1 : (1 << 30);
    // memory planned for step t+1 by requests within their planned length
    auto planned_next = [&]() -> int64_t { return D.next(t); };

    // arrival window: lane l holds the arrival and rank of request wb + l
    int wb = 0, a_reg = INT32_MAX, rk_reg = 0;
    auto load_arrivals = [&](int b) {
        wb = uni(b);
        const int i = b + lane;
        a_reg = INT32_MAX;
        rk_reg = 0;
        if (i < n) {
            a_reg = sg.a[i];
            rk_reg = sg.rank[i];
            if ((unsigned)rk_reg >= (unsigned)n) rk_reg = 0;  // only a broken sort
        }
    };
    load_arrivals(cursor);
    // the record of one rank: a scalar load (read-only while the simulation runs)
    auto rec_of = [&](int r) -> int4 { return record(sg.rec, r); };
    // Steps that provably change nothing are not scanned or checked:
    //  - next_ev: no running request completes or reaches its planned length
    //    before this step (the list is scanned only from then on);
    //  - blk, blk_tf: the highest-priority waiting request (rank blk) failed
    //    the check and cannot fit before step blk_tf while the planned
    //    profile has not shrunk and no request of higher priority is waiting
    //    (relaxed is set by completions, evictions and such arrivals).
    //    A violation at a future step tau persists until tau or until
    //    G[tau] - (M - s) is reached; one at the next step persists until
    //    something is released, since the true memory of the next step only
    //    grows while no request completes or leaves.
    int next_ev = t;  // scan at the first step of a launch
    int blk = -1, blk_tf = 0;
    bool relaxed = true;
    IssuePrio prio;
    prio.init(P, n, nfin);

    for (;;) {
        if (nfin == n) { status = STATUS_DONE; break; }
        if (t > P.max_steps) { status = STATUS_EXHAUSTED; break; }
        if (t >= t_lim) break;
        // 1. arrivals up to t: a prefix of the window (arrivals are sorted;
        //    those of earlier steps were ranked below the blocked head, which
        //    stayed blocked, so nothing could happen at their steps)
        for (;;) {
            const bool arr = (wb + lane >= cursor) && (a_reg <= t);
            const uint64_t m = ballot(arr);
            if (m == 0ull) break;
            if (arr) bitmap_set_atomic(B, S, rk_reg);
            if (ballot(arr && (blk < 0 || rk_reg < blk)) != 0ull) relaxed = true;
            cursor += __popcll(m);
            if (cursor < wb + 64) break;
            load_arrivals(cursor);
        }
        lds_order();
        // 2. completions and requests reaching their planned length: groups
        //    of up to 256 entries are read at once.  The list's order does
        //    not matter (evictions choose by volume, then index), so the
        //    entries that leave are replaced by the entries that stay from
        //    the end of the list: one move per hole instead of shifting
        //    everything behind the first one.
        if (nA > 0 && t >= next_ev) {
            int64_t dC = 0;
            int dN = 0, dfin = 0;
            int nxt = INT32_MAX;  // next event of the entries that stay
            int rem = 0;          // lane i: position of the i-th entry that leaves (first 64)
            for (int base = 0; base < nA; base += 256) {
                int4 qq[4];
                int2 kr[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int x = min(base + 64 * u + lane, nA - 1);
                    qq[u] = A.q[x];
                    kr[u] = A.kr[x];
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int x = base + 64 * u + lane;
                    const bool live = x < nA;
                    const int idx = qq[u].x, s = qq[u].y, oh = qq[u].z, o = qq[u].w, k = kr[u].x;
                    bool done = false;
                    if (live) {
                        const int e = t - k;
                        if (e == o) {
                            done = true;
                            sg.fin[idx] = t;
                            if (o > oh) { dC -= (int64_t)(s - k); dN -= 1; }
                        } else if (e == oh) {
                            dC += (int64_t)(s - k);
                            dN += 1;
                        }
                        if (!done) nxt = min(nxt, (e < oh && oh < o) ? k + oh : k + o);
                    }
                    uint64_t dm = ballot(done);
                    if (dm == 0ull) continue;
                    // early finishers give back their planned future
                    uint64_t early = ballot(done && oh > o);
                    while (early) {
                        const int src = __builtin_ctzll(early);
                        early &= early - 1;
                        D.remove(t, __builtin_amdgcn_readlane(s, src), __builtin_amdgcn_readlane(k, src),
                                 __builtin_amdgcn_readlane(oh, src));
                    }
                    while (dm) {
                        const int b = __builtin_ctzll(dm);
                        dm &= dm - 1;
                        if (lane == dfin) rem = base + 64 * u + b;
                        ++dfin;
                    }
                }
            }
            const int newA = nA - dfin;
            if (dfin > 64) {
                // many at once: compact in place, keeping the order (an
                // entry's place only moves down, after its group was read)
                int pos0 = 0;
                for (int base = 0; base < nA; base += 256) {
                    int4 qq[4];
                    int2 kr[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int x = min(base + 64 * u + lane, nA - 1);
                        qq[u] = A.q[x];
                        kr[u] = A.kr[x];
                    }
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int x = base + 64 * u + lane;
                        const bool stay = x < nA && t - kr[u].x != qq[u].w;
                        const uint64_t keep = ballot(stay);
                        const int pos = pos0 + __popcll(keep & ((1ull << lane) - 1ull));
                        if (stay && pos != x) {
                            A.q[pos] = qq[u];
                            A.kr[pos] = kr[u];
                        }
                        pos0 += __popcll(keep);
                    }
                }
            } else if (dfin > 0) {
                // holes: the positions that left below newA (the first h, in
                // order); the entries that stay at or above newA fill them
                const int h = (int)__popcll(ballot(lane < dfin && rem < newA));
                uint64_t gone = 0ull;  // positions newA + j that left
                for (int i = h; i < dfin; ++i)
                    gone |= 1ull << (__builtin_amdgcn_readlane(rem, i) - newA);
                uint64_t stay = ~gone & (dfin == 64 ? ~0ull : ((1ull << dfin) - 1ull));
                int src = 0;
                for (int i = 0; i < h; ++i) {
                    if (lane == i) src = newA + __builtin_ctzll(stay);
                    stay &= stay - 1ull;
                }
                if (lane < h) {
                    const int4 mq = A.q[src];
                    const int2 mk = A.kr[src];
                    A.q[rem] = mq;
                    A.kr[rem] = mk;
                }
            }
            nA = uni(newA);
            C_O += wave_sum_i64(dC);
            N_O += (int)wave_sum_i64(dN);
            if (dfin > 0) relaxed = true;
            nfin += dfin;
            prio.update(nfin);
            next_ev = wmin(nxt);
            RunList::order();  // the compacted list is read again below
        }
        // requests whose planned length ends by t leave the planned profile
        D.begin(t);
        // 3. overflow of the true memory at t+1: evict the largest believed
        //    remaining volume (latest arrival on ties)
        int nev = 0;
        {
            int64_t mem_next = planned_next() + C_O + (int64_t)N_O * (t + 1);
            while (mem_next > M && nA > 0) {
                // the scan keeps each lane's best entry and the list's last
                // entry in registers: no load after it
                long long bestR = -1;
                int bestIdx = -1, bestPos = -1;
                int4 bq = make_int4(0, 0, 0, 0), lq = make_int4(0, 0, 0, 0);
                int2 bkr = make_int2(0, 0), lkr = make_int2(0, 0);
                for (int base = 0; base < nA; base += 256) {
                    int4 qq[4];
                    int2 kr[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int x = min(base + 64 * u + lane, nA - 1);
                        qq[u] = A.q[x];
                        kr[u] = A.kr[x];
                    }
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int x = base + 64 * u + lane;
                        if (x >= nA) continue;
                        // sum over x = e+1 .. L of (s + x) = (L - e)(2s + L + e + 1) / 2:
                        // one 32 x 32 -> 64-bit product (L - e < 2^30, and
                        // 2s + L + e + 1 < 2^32 with s, L, e < 2^30)
                        const int e = t - kr[u].x;
                        const int L = max(qq[u].z, e + 1);
                        const long long R = (long long)(((unsigned long long)(uint32_t)(L - e) *
                                                         (uint32_t)(2 * (uint32_t)qq[u].y + (uint32_t)L +
                                                                    (uint32_t)e + 1u)) >> 1);
                        if (R > bestR || (R == bestR && qq[u].x > bestIdx)) {
                            bestR = R;
                            bestIdx = qq[u].x;
                            bestPos = x;
                            bq = qq[u];
                            bkr = kr[u];
                        }
                        if (x == nA - 1) {
                            lq = qq[u];
                            lkr = kr[u];
                        }
                    }
                }
                const long long gR = wave_max_i64(bestR);
                const int gIdx = wmax(bestR == gR ? bestIdx : -1);
                const uint64_t who = ballot(bestR == gR && bestIdx == gIdx);
                const int src = __builtin_ctzll(who);
                const int vpos = __builtin_amdgcn_readlane(bestPos, src);
                const int4 q = readlane4(bq, src);
                const int2 vkr = make_int2(__builtin_amdgcn_readlane(bkr.x, src),
                                           __builtin_amdgcn_readlane(bkr.y, src));
                const int lsrc = (nA - 1) & 63;
                const int4 last_q = readlane4(lq, lsrc);
                const int2 last_kr = make_int2(__builtin_amdgcn_readlane(lkr.x, lsrc),
                                               __builtin_amdgcn_readlane(lkr.y, lsrc));
                const int k = vkr.x;
                const int e = t - k;
                if (e < q.z) D.remove(t, q.y, k, q.z);
                else { C_O -= (int64_t)(q.y - k); N_O -= 1; }
                if (lane == 0) {
                    A.q[vpos] = last_q;
                    A.kr[vpos] = last_kr;
                    sg.preempt[q.x] += 1;
                    sg.start[q.x] = -1;
                    sg.admit_seq[q.x] = -1;
                    sg.evl[nev] = vkr.y;
                }
                RunList::order();
                --nA;
                ++nev;
                relaxed = true;
                mem_next = planned_next() + C_O + (int64_t)N_O * (t + 1);
            }
        }
        // 4. admissions
        for (;;) {
            if (!relaxed && blk >= 0 && t < blk_tf) break;  // still blocked
            const int r = bitmap_first(B, S, W1);
            if (r < 0) { blk = -1; break; }
            const int4 q = rec_of(r);
            int tf = 0;
            // memory of requests past their plan at t+1; <= M after step 3
            const int extra1 = (int)(C_O + (int64_t)N_O * (t + 1));
            // If the next step alone is over (true memory at t+1 plus the
            // candidate's first token), the candidate fails the check and
            // stays blocked until something is released: without completions
            // or evictions the running set only grows, by one token per
            // request per step.
            if (planned_next() + extra1 + q.y + 1 > M) {
                blk = r;
                blk_tf = INT32_MAX;
                relaxed = false;
                break;
            }
            if (!D.fit(t, q.y, q.z, M, extra1, maxF, &tf, chk)) {
                blk = r;
                blk_tf = tf;
                relaxed = false;
                break;
            }
            maxF = max(maxF, t + q.z);
            next_ev = min(next_ev, q.z < q.w ? t + q.z : t + q.w);
            if (lane == 0) {
                bitmap_clear(B, S, r);
                sg.start[q.x] = t;
                sg.admit_seq[q.x] = seq;
                A.q[nA] = q;
                A.kr[nA] = make_int2(t, r);
            }
            RunList::order();
            ++seq;
            ++nA;
        }
        if (STOP && blk_tf < 0) {  // a full list: leave the launch inside this step
            st.resume_nev = nev;
            break;
        }
        // evicted requests compete again from the next step
        if (nev > 0) {
            lds_order();  // their ranks were stored by lane 0 of this wave
            for (int x = lane; x < nev; x += 64) {
                const int r = sg.evl[x];
                if ((unsigned)r < (unsigned)n) bitmap_set_atomic(B, S, r);
            }
            lds_order();
            relaxed = true;  // one of them may rank above the blocked head
        }
        // 5. advance to the next step at which anything can happen.  Until
        //    then no request arrives, completes, reaches its planned length or
        //    is evicted, no request ranked above the blocked head arrives (with
        //    nothing waiting: no request arrives), and the blocked head stays
        //    blocked, so every running request grows by one token per step:
        //    the true memory at step tau+1 is mem + nA (tau - t), below M
        //    until tau_ov.  Evicted requests compete again at t+1, and a
        //    segment whose requests have all finished ends at t+1.
        const int64_t mem = planned_next() + C_O + (int64_t)N_O * (t + 1);
        int tn = t + 1;
        if (nev == 0 && nfin < n) {
            int tj = min(next_ev, min(t_lim, P.max_steps + 1));
            if (cursor < n) {
                int na;
                if (blk >= 0) {  // the next arrival ranked above the head (past the window: its end)
                    const uint64_t up = ballot((wb + lane >= cursor) && rk_reg < blk);
                    na = up != 0ull ? __builtin_amdgcn_readlane(a_reg, __builtin_ctzll(up))
                                    : (wb + 64 < n ? uni(sg.a[wb + 64]) : INT32_MAX);
                } else {
                    na = cursor < wb + 64 ? __builtin_amdgcn_readlane(a_reg, cursor - wb)
                                          : uni(sg.a[cursor]);
                }
                tj = min(tj, na);
            }
            if (blk >= 0) tj = min(tj, blk_tf);
            if (nA > 0 && tj > t + 1) {
                const int64_t room = (int64_t)M - mem;  // >= 0 after the admissions
                tj = room < 0 ? t + 1 : min(tj, t + 1 + (int)((uint32_t)room / (uint32_t)nA));
            }
            tn = max(tj, t + 1);
        }
        req_steps += (int64_t)nA * (tn - t);
        peak = max(peak, mem + (int64_t)nA * (tn - 1 - t));
        D.end_step(t, tn);
        t = uni(tn);
    }
    prio.leave();
    st.t = t; st.cursor = cursor; st.seq = seq; st.nfin = nfin; st.nA = nA; st.N_O = N_O;
    st.C_O = C_O; st.peak = peak; st.req_steps = req_steps; st.status = status;
    st.max_fin = maxF;
}

// The rest of step st.t for a segment that stopped inside its admissions
// (its steps 1-3 ran in the launch before, evicting nev requests whose ranks
// are in evl): the admissions with room for the host's bound, the evicted
// requests back into the waiting set, and the advance to the next step.
template <class PROF>
__device__ void stepped_resume_tail(const SimArgs& P, const Seg& sg, uint64_t* B, uint64_t* S,
                                    int W1, PROF& D, const RunList& A, SegState& st, int nev) {
    const int lane = lane_id();
    const int M = P.M;
    const int t = uni(st.t);
    int seq = uni(st.seq), nA = uni(st.nA), maxF = uni(st.max_fin);
    const int64_t C_O = st.C_O;
    const int N_O = st.N_O;
    const int pol = blockIdx.x / P.I;
    const int chk = (P.policies[pol] & ADMIT_CURRENT) ? 1 : (1 << 30);
    const int extra1 = (int)(C_O + (int64_t)N_O * (t + 1));
    for (;;) {
        const int r = bitmap_first(B, S, W1);
        if (r < 0) break;
        const int4 q = record(sg.rec, r);
        if (D.next(t) + extra1 + q.y + 1 > M) break;
        int tf = 0;
        if (!D.fit(t, q.y, q.z, M, extra1, maxF, &tf, chk)) break;
        maxF = max(maxF, t + q.z);
        if (lane == 0) {
            bitmap_clear(B, S, r);
            sg.start[q.x] = t;
            sg.admit_seq[q.x] = seq;
            A.q[nA] = q;
            A.kr[nA] = make_int2(t, r);
        }
        RunList::order();
        ++seq;
        ++nA;
    }
    if (nev > 0) {
        for (int x = lane; x < nev; x += 64) {
            const int r = sg.evl[x];
            if ((unsigned)r < (unsigned)sg.n) bitmap_set_atomic(B, S, r);
        }
        lds_order();
    }
    st.req_steps += nA;
    st.peak = max(st.peak, D.next(t) + C_O + (int64_t)N_O * (t + 1));
    D.end_step(t, t + 1);
    st.t = t + 1;
    st.seq = seq;
    st.nA = nA;
    st.max_fin = maxF;
}

// One wave64 per segment; launched once for segments that plan with the
// true lengths (event-driven) and once for the others (per step), so each
// kernel carries only its own path.  LIST: the event path keeps its profile
// as the finish-ordered list (LDS after the bitmap, kept in global memory
// between launches) instead of the ring.
template <bool D_LDS, bool STEPPED, bool LIST, bool RESUME = false, bool STOP = false>
__device__ __forceinline__ void sim_segment(const SimArgs& P) {
    extern __shared__ uint64_t smem[];
    const int g = blockIdx.x;
    if ((P.stepped[g] != 0) != STEPPED) return;
    const int lane = lane_id();
    const int pol = g / P.I, inst = g - pol * P.I;
    const int64_t off = P.offsets[inst];
    const int n = (int)(P.offsets[inst + 1] - off);
    SegState st = P.st[g];
    if (st.status != STATUS_RUNNING) return;
    if (LIST && P.list_resume && st.resume_lim == 0) return;

    Seg sg;
    sg.n = n;
    const int64_t base = (int64_t)pol * P.N + off;
    sg.rec = P.rec + base;
    sg.rank = P.rank + base;
    sg.a = P.a + off;
    sg.start = P.start + base;
    sg.fin = P.fin + base;
    sg.preempt = P.preempt + base;
    sg.admit_seq = P.admit_seq + base;
    sg.act = P.act ? P.act + base : nullptr;
    sg.actkr = P.actkr ? P.actkr + base : nullptr;
    sg.evl = P.evl ? P.evl + base : nullptr;

    // rank bitmap (two levels) staged in LDS for the launch
    const int W0 = (n + 63) >> 6;
    const int W1 = (W0 + 63) >> 6;
    const int64_t bw_base = (int64_t)pol * P.bw_total + P.bw_off[inst];
    uint64_t* Bg = P.bitmap + bw_base;
    uint64_t* B = smem;
    uint64_t* S = smem + W0;
    for (int x = lane; x < W0 + W1; x += 64) B[x] = Bg[x];

    // steps t < t_lim are simulated in this launch
    const int64_t want = (int64_t)st.t + P.step_delta;
    int t_lim = (int)min(want, (int64_t)P.max_steps + 2);

    if (LIST && STEPPED) {
        const int cap = P.list_cap;
        int32_t* Fg = P.lst_f + (int64_t)g * P.list_stride;
        uint32_t* Qg = P.lst_q + (int64_t)g * P.list_stride;
        StepList L;
        L.cap = cap;
        L.F = reinterpret_cast<int32_t*>(smem + P.bw_max);
        L.Q = reinterpret_cast<uint32_t*>(L.F + list_slots(cap));
        L.ln = uni(st.ln);
        L.tot = (uint32_t)uni((int)st.lq);
        // resumed inside a step (>= 0), or from the start of one (-1)
        const int mid = RESUME ? uni(st.resume_nev) : -1;
        if (RESUME) t_lim = st.resume_lim;
        st.resume_lim = 0;
        st.resume_nev = -1;
        if (L.ln > cap) {
            // more planned requests than this launch has room for
            st.resume_lim = t_lim;
        } else {
            for (int x = lane; x < L.ln; x += 64) {
                L.F[x] = Fg[x];
                L.Q[x] = Qg[x];
            }
            if (L.ln == 0 && lane == 0) L.F[0] = INT32_MAX;  // the empty list's sentinel
            __syncthreads();
            RunList A;
            A.q = sg.act;
            A.kr = sg.actkr;
            if (RESUME && mid >= 0) {
                lds_order();  // the evicted ranks were stored by lane 0 of this wave
                stepped_resume_tail(P, sg, B, S, W1, L, A, st, mid);
            }
            run_stepped<STOP>(P, sg, B, S, W1, L, A, st, t_lim);
            __syncthreads();
            for (int x = lane; x < L.ln; x += 64) {
                Fg[x] = L.F[x];
                Qg[x] = L.Q[x];
            }
            st.ln = L.ln;
            st.lq = L.tot;
            if (st.resume_nev >= 0) st.resume_lim = t_lim;  // stopped inside step st.t
        }
    } else if (LIST) {
        const int cap = P.list_cap;
        int32_t* Fg = P.lst_f + (int64_t)g * P.list_stride;
        uint32_t* Qg = P.lst_q + (int64_t)g * P.list_stride;
        ListProf L;
        L.cap = cap;
        L.F = reinterpret_cast<int32_t*>(smem + P.bw_max);
        L.Q = reinterpret_cast<uint32_t*>(L.F + list_slots(cap));
        L.ln = uni(st.ln);
        L.tot = (uint32_t)uni((int)st.lq);
        L.peak_lane = 0;
        if (P.list_resume) t_lim = st.resume_lim;
        st.resume_lim = 0;
        if (L.ln > cap) {
            // more running than this launch has room for: left to the continuation
            st.resume_lim = t_lim;
        } else {
            for (int x = lane; x < L.ln; x += 64) {
                L.F[x] = Fg[x];
                L.Q[x] = Qg[x];
            }
            if (L.ln == 0 && lane == 0) L.F[0] = INT32_MAX;  // the empty list's sentinel
            // a stop on a full list left t_f = -1: the head is checked again at t
            if (st.t_f < 0) st.t_f = st.t;
            __syncthreads();
            run_known(P, sg, B, S, W1, L, st, t_lim);
            __syncthreads();
            for (int x = lane; x < L.ln; x += 64) {
                Fg[x] = L.F[x];
                Qg[x] = L.Q[x];
            }
            st.ln = L.ln;
            st.lq = L.tot;
            if (st.t_f < 0) st.resume_lim = t_lim;  // stopped on a full list
        }
    } else {
        const int RS = P.H + 64;  // ring stride: H slots and the spare slot, padded
        int32_t* Dg = P.ring + (int64_t)g * RS;
        int32_t* Dl = reinterpret_cast<int32_t*>(smem + P.bw_max);
        if (D_LDS) {
            for (int x = lane; x < P.H; x += 64) Dl[x] = Dg[x];
        }
        __syncthreads();
        Ring<D_LDS> D;
        D.p = D_LDS ? Dl : Dg;
        D.H = P.H;
        D.mask = P.H - 1;
        if (STEPPED) {
            RunList A;
            A.q = sg.act;
            A.kr = sg.actkr;
            RingStep<D_LDS> R(D);
            run_stepped<false>(P, sg, B, S, W1, R, A, st, t_lim);
        } else {
            RingProf<D_LDS> R(D, uni(st.t));
            run_known(P, sg, B, S, W1, R, st, t_lim);
        }
        __syncthreads();
        if (D_LDS) {
            for (int x = lane; x < P.H; x += 64) Dg[x] = Dl[x];
        }
    }
    for (int x = lane; x < W0 + W1; x += 64) Bg[x] = B[x];
    if (lane == 0) P.st[g] = st;
}

template <bool D_LDS, bool STEPPED>
__global__ __launch_bounds__(64) void k_sim(SimArgs P) {
    sim_segment<D_LDS, STEPPED, false>(P);
}

// The list kernel needs few vector registers; its scalar state is squeezed
// (spilled to vector lanes) so that eight waves fit on each SIMD, which the
// short LDS footprint of the list allows.
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(8, 8)))
void k_sim_list(SimArgs P) {
    sim_segment<false, false, true>(P);
}

// The per-step path with the finish-ordered list: with room for the bound,
// with less (segments may stop inside a step), and the continuation.
__global__ __launch_bounds__(64) void k_sim_steplist(SimArgs P) {
    sim_segment<false, true, true>(P);
}
__global__ __launch_bounds__(64) void k_sim_steplist_stop(SimArgs P) {
    sim_segment<false, true, true, false, true>(P);
}
__global__ __launch_bounds__(64) void k_sim_steplist_resume(SimArgs P) {
    sim_segment<false, true, true, true>(P);
}

// The same for the continuation of segments whose list outgrew the first
// launch's LDS (a kernel of its own, so that timings keep the two apart).
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(8, 8)))
void k_sim_list_resume(SimArgs P) {
    sim_segment<false, false, true>(P);
}

// ------------------------------------------------------------ finalize

// One workgroup of FIN_NT threads per segment, FIN_U requests per thread in
// flight: the outputs are a streaming pass over start, o and a (plus the
// per-step path's finish and preemption counts, which the event path never
// writes: its finish is start + o and it never evicts).
constexpr int FIN_NT = 256, FIN_U = 4;

__global__ __launch_bounds__(FIN_NT) void k_finalize(FinArgs F) {
    __shared__ long long red[3][FIN_NT / 64];
    __shared__ int redm[FIN_NT / 64];
    const int g = blockIdx.x;
    const int tid = threadIdx.x, lane = lane_id(), w = tid >> 6;
    const int pol = g / F.I, inst = g - pol * F.I;
    const int64_t off = F.offsets[inst];
    const int n = (int)(F.offsets[inst + 1] - off);
    const int64_t base = (int64_t)pol * F.N + off;
    const SegState st = F.st[g];
    const bool stepped = F.stepped[g] != 0;
    const int t_end = st.t;
    long long lat = 0, rs = 0, pre = 0;
    int mk = 0;
    for (int j0 = 0; j0 < n; j0 += FIN_NT * FIN_U) {
        int k[FIN_U], o[FIN_U], a[FIN_U], f[FIN_U], p[FIN_U];
#pragma unroll
        for (int u = 0; u < FIN_U; ++u) {
            const int j = j0 + u * FIN_NT + tid;
            k[u] = -1; o[u] = 0; a[u] = 0; f[u] = -1; p[u] = 0;
            if (j < n) {
                k[u] = F.start[base + j];
                o[u] = F.o[off + j];
                a[u] = F.a[off + j];
                if (stepped) {
                    f[u] = F.fin[base + j];
                    p[u] = F.preempt[base + j];
                }
            }
        }
#pragma unroll
        for (int u = 0; u < FIN_U; ++u) {
            const int j = j0 + u * FIN_NT + tid;
            if (j >= n) continue;
            // known lengths: the finish is start + o (not stored by the simulation)
            int fj = stepped ? f[u] : (k[u] >= 0 ? k[u] + o[u] : -1);
            if (fj > t_end - 1) fj = -1;
            F.fin_out[base + j] = fj;
            if (fj >= 0) {
                lat += (long long)fj - a[u];
                mk = max(mk, fj);
            }
            if (!stepped && k[u] >= 0) rs += (long long)min(k[u] + o[u], t_end) - k[u];
            pre += p[u];
        }
    }
    lat = wave_sum_i64(lat);
    rs = wave_sum_i64(rs);
    pre = wave_sum_i64(pre);
    mk = wave_max_i32(mk);
    if (lane == 0) {
        red[0][w] = lat;
        red[1][w] = rs;
        red[2][w] = pre;
        redm[w] = mk;
    }
    __syncthreads();
    if (tid == 0) {
        for (int x = 1; x < FIN_NT / 64; ++x) {
            lat += red[0][x];
            rs += red[1][x];
            pre += red[2][x];
            mk = max(mk, redm[x]);
        }
        StatsOut so;
        so.makespan = mk;
        so.status = st.status;
        so.sum_latency = lat;
        so.request_steps = stepped ? st.req_steps : rs;
        so.peak_mem = st.peak;
        so.preemptions = pre;
        so.t_end = t_end;
        F.stats[g] = so;
    }
}

// ------------------------------------------------------------ launchers

static inline int grid_for(int64_t n, int bs) {
    int64_t g = (n + bs - 1) / bs;
    if (g > 65536) g = 65536;
    return (int)(g < 1 ? 1 : g);
}

hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill_i32, dim3(grid_for(n, 256)), dim3(256), 0, s, p, n, v);
    return hipGetLastError();
}

hipError_t launch_fill_u64(uint64_t* p, int64_t n, uint64_t v, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill_u64, dim3(grid_for(n, 256)), dim3(256), 0, s, p, n, v);
    return hipGetLastError();
}

hipError_t launch_init_ring(int32_t* ring, int64_t n, int32_t H, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_init_ring, dim3(grid_for(n, 256)), dim3(256), 0, s, ring, n, H);
    return hipGetLastError();
}

hipError_t launch_init_state(SegState* st, int32_t G, hipStream_t s) {
    if (G <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_init_state, dim3((G + 255) / 256), dim3(256), 0, s, st, G);
    return hipGetLastError();
}

hipError_t launch_chunk_sort(const SortArgs& A, int nchunks, hipStream_t s) {
    if (nchunks <= 0) return hipSuccess;
    switch (A.CH) {
    case 64: hipLaunchKernelGGL((k_chunk_sort<64, 64>), dim3(nchunks), dim3(64), 0, s, A); break;
    case 128: hipLaunchKernelGGL((k_chunk_sort<128, 64>), dim3(nchunks), dim3(64), 0, s, A); break;
    case 256: hipLaunchKernelGGL((k_chunk_sort<256, 128>), dim3(nchunks), dim3(128), 0, s, A); break;
    case 512: hipLaunchKernelGGL((k_chunk_sort<512, 256>), dim3(nchunks), dim3(256), 0, s, A); break;
    case 1024: hipLaunchKernelGGL((k_chunk_sort<1024, 256>), dim3(nchunks), dim3(256), 0, s, A); break;
    case 2048: hipLaunchKernelGGL((k_chunk_sort<2048, 512>), dim3(nchunks), dim3(512), 0, s, A); break;
    case 4096: hipLaunchKernelGGL((k_chunk_sort<4096, 512>), dim3(nchunks), dim3(512), 0, s, A); break;
    case 8192: hipLaunchKernelGGL((k_chunk_sort<8192, 1024>), dim3(nchunks), dim3(1024), 0, s, A); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_merge_pass(const SortArgs& A, int nchunks, int w, hipStream_t s) {
    if (nchunks <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_merge_pass, dim3(nchunks), dim3(256), 0, s, A, w);
    return hipGetLastError();
}

hipError_t launch_build_rec(const SortArgs& A, int nchunks, hipStream_t s) {
    if (nchunks <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_build_rec, dim3(nchunks), dim3(256), 0, s, A);
    return hipGetLastError();
}

template <int NT, int E>
static size_t sort_rec_lds() {
    return (size_t)(NT * E + NT * E / 32) * 8 + (size_t)16 * NT * 2 + (size_t)(NT / 64) * 4;
}

template <int NT, int E>
static hipError_t sort_rec_attr() {
    const size_t b = sort_rec_lds<NT, E>();
    if (b <= 65536) return hipSuccess;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(&k_sort_rec<NT, E>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)b);
}

template <int NT, int E>
static hipError_t sort_rec_go(const SortArgs& A, int G, hipStream_t s) {
    const size_t lds = sort_rec_lds<NT, E>();
    hipLaunchKernelGGL((k_sort_rec<NT, E>), dim3(G), dim3(NT), lds, s, A);
    return hipGetLastError();
}

// workgroup shapes (threads, elements per thread) by the largest instance
hipError_t prepare_sort_rec(int max_n) {
    if (max_n <= 64 * 4) return sort_rec_attr<64, 4>();
    if (max_n <= 128 * 8) return sort_rec_attr<128, 8>();
    if (max_n <= 128 * 16) return sort_rec_attr<128, 16>();
    if (max_n <= 256 * 16) return sort_rec_attr<256, 16>();
    if (max_n <= 256 * 20) return sort_rec_attr<256, 20>();
    if (max_n <= 256 * 24) return sort_rec_attr<256, 24>();
    if (max_n <= 256 * 32) return sort_rec_attr<256, 32>();
    return hipErrorInvalidValue;
}

hipError_t launch_sort_rec(const SortArgs& A, int G, int max_n, hipStream_t s) {
    if (G <= 0) return hipSuccess;
    if (max_n <= 64 * 4) return sort_rec_go<64, 4>(A, G, s);
    if (max_n <= 128 * 8) return sort_rec_go<128, 8>(A, G, s);
    if (max_n <= 128 * 16) return sort_rec_go<128, 16>(A, G, s);
    if (max_n <= 256 * 16) return sort_rec_go<256, 16>(A, G, s);
    if (max_n <= 256 * 20) return sort_rec_go<256, 20>(A, G, s);
    if (max_n <= 256 * 24) return sort_rec_go<256, 24>(A, G, s);
    if (max_n <= 256 * 32) return sort_rec_go<256, 32>(A, G, s);
    return hipErrorInvalidValue;
}

hipError_t launch_sim(const SimArgs& P, int G, bool d_lds, bool stepped, bool list,
                      size_t lds_bytes, hipStream_t s) {
    if (G <= 0) return hipSuccess;
    if (stepped && list) {
        if (P.list_resume) hipLaunchKernelGGL(k_sim_steplist_resume, dim3(G), dim3(64), lds_bytes, s, P);
        else if (P.list_cap < P.list_stride) hipLaunchKernelGGL(k_sim_steplist_stop, dim3(G), dim3(64), lds_bytes, s, P);
        else hipLaunchKernelGGL(k_sim_steplist, dim3(G), dim3(64), lds_bytes, s, P);
    } else if (!stepped && list) {
        if (P.list_resume) hipLaunchKernelGGL(k_sim_list_resume, dim3(G), dim3(64), lds_bytes, s, P);
        else hipLaunchKernelGGL(k_sim_list, dim3(G), dim3(64), lds_bytes, s, P);
    } else if (d_lds) {
        if (stepped) hipLaunchKernelGGL((k_sim<true, true>), dim3(G), dim3(64), lds_bytes, s, P);
        else hipLaunchKernelGGL((k_sim<true, false>), dim3(G), dim3(64), lds_bytes, s, P);
    } else {
        if (stepped) hipLaunchKernelGGL((k_sim<false, true>), dim3(G), dim3(64), lds_bytes, s, P);
        else hipLaunchKernelGGL((k_sim<false, false>), dim3(G), dim3(64), lds_bytes, s, P);
    }
    return hipGetLastError();
}

static hipError_t sim_attr(const void* f, size_t lds_bytes) {
    if (lds_bytes <= 65536) return hipSuccess;
    return hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
}

hipError_t prepare_sim(bool d_lds, size_t lds_ring, bool list, size_t lds_list) {
    hipError_t e;
    if (d_lds) {
        e = sim_attr((const void*)k_sim<true, true>, lds_ring);
        if (e == hipSuccess) e = sim_attr((const void*)k_sim<true, false>, lds_ring);
    } else {
        e = sim_attr((const void*)k_sim<false, true>, lds_ring);
        if (e == hipSuccess) e = sim_attr((const void*)k_sim<false, false>, lds_ring);
    }
    if (e == hipSuccess && list) e = sim_attr((const void*)k_sim_list, lds_list);
    if (e == hipSuccess && list) e = sim_attr((const void*)k_sim_steplist, lds_list);
    if (e == hipSuccess && list) e = sim_attr((const void*)k_sim_steplist_resume, lds_list);
    if (e == hipSuccess && list) e = sim_attr((const void*)k_sim_steplist_stop, lds_list);
    if (e == hipSuccess && list) e = sim_attr((const void*)k_sim_list_resume, lds_list);
    return e;
}

hipError_t sim_known_occupancy(bool list, bool d_lds, size_t lds_bytes, int* blocks) {
    const void* f = list ? (const void*)k_sim_list
                         : (d_lds ? (const void*)k_sim<true, false>
                                  : (const void*)k_sim<false, false>);
    hipError_t e = sim_attr(f, lds_bytes);
    if (e != hipSuccess) return e;
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, f, 64, lds_bytes);
}

hipError_t sim_occupancy(bool stepped, bool list, bool d_lds, size_t lds_bytes, int* blocks) {
    const void* f;
    if (list) f = stepped ? (const void*)k_sim_steplist : (const void*)k_sim_list;
    else if (stepped) f = d_lds ? (const void*)k_sim<true, true> : (const void*)k_sim<false, true>;
    else f = d_lds ? (const void*)k_sim<true, false> : (const void*)k_sim<false, false>;
    hipError_t e = sim_attr(f, lds_bytes);
    if (e != hipSuccess) return e;
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, f, 64, lds_bytes);
}

hipError_t sim_step_occupancy(size_t lds_bytes, int* blocks) {
    const void* f = (const void*)k_sim_steplist_stop;
    hipError_t e = sim_attr(f, lds_bytes);
    if (e != hipSuccess) return e;
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, f, 64, lds_bytes);
}

hipError_t launch_finalize(const FinArgs& F, int G, hipStream_t s) {
    if (G <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_finalize, dim3(G), dim3(FIN_NT), 0, s, F);
    return hipGetLastError();
}

}  // namespace svfk
