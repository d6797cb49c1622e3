// svf_kernels.h -- internal interface between the host runtime and the gfx950
// kernels of the batched scheduling simulator (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace svfk {

enum { POLICY_FCFS = 0, POLICY_SJF = 1, POLICY_SVF = 2, POLICY_SVF1BIT = 3 };
enum { ADMIT_CURRENT = 0x100 };  // added to a policy code: next-step admission
enum { STATUS_DONE = 0, STATUS_EXHAUSTED = 1, STATUS_RUNNING = 2 };

// Per-segment (instance x policy) simulation state, kept in HBM between launches.
struct SegState {
    int32_t t;          // next step to simulate
    int32_t cursor;     // next request (instance-local index) still to arrive
    int32_t seq;        // admissions so far
    int32_t status;     // STATUS_*
    int32_t nA;         // running requests (per-step path)
    int32_t nfin;       // finished (per-step path) / admitted (event path)
    int32_t max_fin;    // event path: latest scheduled finish
    int32_t head_rank;  // event path: blocked head (-1: none known)
    int32_t t_f;        // event path: the head cannot fit before this step
    int32_t N_O;        // per-step path: requests past their planned length
    int64_t C_O;        // per-step path: sum of (s - k) over those requests
    int64_t peak;       // largest memory total over the steps folded so far
    int64_t req_steps;  // per-step path: sum over steps of running requests
    int32_t ln;         // event path with the list profile: running requests
    uint32_t lq;        //   and the prefix sum of (s - k) of the last entry
    int32_t resume_lim; // list full before step resume_lim: continue up to there (0: no)
    int32_t resume_nev; // per-step path: -1, or stopped in the admission phase of step t
                        //   with this many evictions of that step (ranks in evl)
};

// Same layout as svf_instance_stats of the public header.
struct StatsOut {
    int32_t makespan;
    int32_t status;
    int64_t sum_latency;
    int64_t request_steps;
    int64_t peak_mem;
    int64_t preemptions;
    int64_t t_end;
};

struct SortArgs {
    const int64_t* offsets;   // [I+1]
    const int32_t* a;         // [N]
    const int32_t* s;
    const int32_t* o;
    const int32_t* plan;      // [N] or null
    const int8_t* bit;        // [N] or null
    const int32_t* policies;  // [P] (device)
    const uint8_t* stepped;   // [G] 1: per-step path (its finishes and preemptions are cleared too)
    const int32_t* chunk_seg; // [nchunks] segment of each chunk
    const int32_t* chunk_lo;  // [nchunks] first rank position of each chunk
    const uint64_t* keys_in;  // [P*N]
    uint64_t* keys_out;       // [P*N]
    int4* rec;                // [P*N] rank-ordered {index, s, planned length, o}
    int32_t* rank;            // [P*N] index -> rank
    int32_t I, P;
    int64_t N;
    int32_t O0, O1;
    int32_t CH;
    int32_t kbits[8];         // [P] bits of the largest priority key of each policy
    int32_t* start;           // [P*N] outputs cleared by the fused sort (k_sort_rec)
    int32_t* fin;
    int32_t* preempt;
    int32_t* admit_seq;
};

struct SimArgs {
    const int64_t* offsets;
    const int32_t* a;
    const int4* rec;
    const int32_t* rank;
    const uint8_t* stepped;   // [G] 1: per-step path (plans differ or next-step admission)
    const int32_t* policies;  // [P] policy codes
    const int64_t* bw_off;    // [I+1] bitmap word offset of each instance
    uint64_t* bitmap;         // [P*bw_total]
    int32_t* ring;            // [G*(H+64)] future profile plus step index (G = D + tau)
    int32_t* start;           // [P*N]
    int32_t* fin;
    int32_t* preempt;
    int32_t* admit_seq;
    int4* act;                // [P*N] or null: running list, record of each entry
    int2* actkr;              // [P*N] or null: running list, {start step, rank}
    int32_t* evl;             // [P*N] or null
    SegState* st;             // [G]
    int32_t I, P;
    int64_t N;
    int64_t bw_total;
    int32_t bw_max;           // largest bitmap size of one instance (words)
    int32_t H;                // ring length (power of two)
    int32_t M;
    int32_t max_steps;
    int64_t step_delta;       // steps to simulate in this launch
    int32_t* lst_f;           // [G*list_stride] event path, list profile: planned finishes
    uint32_t* lst_q;          // [G*list_stride]   and prefix sums of s - k
    int32_t list_stride;      // entries per segment in HBM (bound on concurrent requests)
    int32_t list_cap;         // entries per segment in LDS in this launch (<= list_stride)
    int32_t list_resume;      // 1: only continue the segments that stopped with a full list
    int32_t resident;         // workgroups of this launch resident at once (0: no issue priorities)
    unsigned long long* prog; // [1] progress counter of this launch, cleared before it
};

struct FinArgs {
    const int64_t* offsets;
    const int32_t* a;
    const int32_t* o;
    const uint8_t* stepped;
    const int32_t* start;
    const int32_t* fin;
    const int32_t* preempt;
    const SegState* st;
    int32_t* fin_out;
    StatsOut* stats;
    int32_t I, P;
    int64_t N;
};

hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s);
hipError_t launch_fill_u64(uint64_t* p, int64_t n, uint64_t v, hipStream_t s);
hipError_t launch_init_ring(int32_t* ring, int64_t n, int32_t H, hipStream_t s);
hipError_t launch_init_state(SegState* st, int32_t G, hipStream_t s);
hipError_t launch_chunk_sort(const SortArgs& A, int nchunks, hipStream_t s);
hipError_t launch_merge_pass(const SortArgs& A, int nchunks, int w, hipStream_t s);
hipError_t launch_build_rec(const SortArgs& A, int nchunks, hipStream_t s);
// Instances of at most SORT_REC_MAX requests: keys, stable radix sort, records,
// ranks and cleared outputs in one kernel, one workgroup per segment.
enum { SORT_REC_MAX = 8192 };
hipError_t prepare_sort_rec(int max_n);
hipError_t launch_sort_rec(const SortArgs& A, int G, int max_n, hipStream_t s);
hipError_t prepare_sim(bool d_lds, size_t lds_ring, bool list, size_t lds_list);
// entries of LDS the finish-ordered list of capacity cap takes (F and Q each)
__host__ __device__ inline int list_slots(int cap) { return cap + 65; }
// list: the event path keeps its profile as the finish-ordered list
hipError_t launch_sim(const SimArgs& P, int G, bool d_lds, bool stepped, bool list,
                      size_t lds_bytes, hipStream_t s);
// resident waves per compute unit of the event kernel (ring or list profile)
hipError_t sim_known_occupancy(bool list, bool d_lds, size_t lds_bytes, int* blocks);
// resident waves per compute unit of the per-step kernel with the list
hipError_t sim_step_occupancy(size_t lds_bytes, int* blocks);
// resident waves per compute unit of the first simulation kernel of a path
hipError_t sim_occupancy(bool stepped, bool list, bool d_lds, size_t lds_bytes, int* blocks);
hipError_t launch_finalize(const FinArgs& F, int G, hipStream_t s);
// Device address and size of the calling thread's current device's scratch
// array of the no-allocation entry point (svf_noalloc.hip).
hipError_t noalloc_scratch(void** addr, size_t* bytes);

}  // namespace svfk
