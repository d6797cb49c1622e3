// Test driver for the C ABI of include/svfsim.h, built with the runtime's
// host code under the address and undefined-behaviour sanitizers (device
// code is not instrumented).  tests/test_sanitizers.py runs it.
//
//   abi_asan errors            malformed calls; validation happens before any
//                              HIP call, so this mode needs no GPU
//   abi_asan create IN         svf_create on a valid batch (on a machine
//                              without a GPU it stops at the first HIP call)
//   abi_asan run IN OUT        svf_create + svf_run, the same batch in svf_step
//                              chunks and through svf_run_noalloc (all three must
//                              agree), outputs of the first written to OUT
//
// IN (native byte order): int64 I, N, M, P, O0, O1, max_steps, has_plan,
// has_bit; int64 policies[P]; int64 offsets[I + 1]; int32 a[N], s[N], o[N];
// int32 plan[N] if has_plan; int8 bit[N] if has_bit.
// OUT, per policy slot: int32 start[N], finish[N], preempt[N], admit_seq[N];
// svf_instance_stats[I].
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "svfsim.h"

namespace {

struct Batch {
    std::vector<int64_t> off;
    std::vector<int32_t> a, s, o, plan, pol;
    std::vector<int8_t> bit;
    int64_t I = 0, N = 0, M = 0, O0 = 0, O1 = 0, max_steps = 0;
    svf_batch_desc desc() const {
        svf_batch_desc d{};
        d.num_instances = (int32_t)I;
        d.req_offsets = off.data();
        d.arrival = a.data();
        d.prompt = s.data();
        d.output = o.data();
        d.plan_len = plan.empty() ? nullptr : plan.data();
        d.long_bit = bit.empty() ? nullptr : bit.data();
        d.M = M;
        d.num_policies = (int32_t)pol.size();
        d.policies = pol.data();
        d.O0 = (int32_t)O0;
        d.O1 = (int32_t)O1;
        d.max_steps = max_steps;
        d.inputs_on_device = 0;
        return d;
    }
};

template <typename T>
void get(FILE* f, std::vector<T>& v, int64_t n) {
    v.resize((size_t)n);
    if (n > 0 && fread(v.data(), sizeof(T), (size_t)n, f) != (size_t)n) {
        fprintf(stderr, "short input\n");
        exit(2);
    }
}

Batch load(const char* path) {
    FILE* f = fopen(path, "rb");
    if (!f) exit(2);
    std::vector<int64_t> h;
    get(f, h, 9);
    Batch b;
    b.I = h[0]; b.N = h[1]; b.M = h[2]; b.O0 = h[4]; b.O1 = h[5]; b.max_steps = h[6];
    std::vector<int64_t> p;
    get(f, p, h[3]);
    for (int64_t x : p) b.pol.push_back((int32_t)x);
    get(f, b.off, b.I + 1);
    get(f, b.a, b.N);
    get(f, b.s, b.N);
    get(f, b.o, b.N);
    if (h[7]) get(f, b.plan, b.N);
    if (h[8]) get(f, b.bit, b.N);
    fclose(f);
    return b;
}

int failures = 0;

void expect(bool ok, const char* what) {
    if (!ok) {
        fprintf(stderr, "FAILED: %s (last error: %s)\n", what, svf_last_error());
        ++failures;
    }
}

// A malformed variant of a small valid batch must be refused by svf_create
// and by svf_run_noalloc with the given code, before any HIP call.
void refuse(const svf_batch_desc& d, int code, const char* what) {
    svf_batch* h = nullptr;
    expect(svf_create(&d, nullptr, &h) == code && h == nullptr, what);
    int32_t dummy[64];
    svf_instance_stats st[8];
    expect(svf_run_noalloc(&d, nullptr, dummy, dummy, dummy, dummy, st) == code, what);
}

int errors_mode() {
    const int64_t off[3] = {0, 3, 5};
    const int32_t a[5] = {0, 1, 1, 0, 4}, s[5] = {2, 3, 4, 1, 1}, o[5] = {5, 6, 7, 2, 2};
    const int32_t pol[2] = {SVF_POLICY_SVF, SVF_POLICY_FCFS};
    svf_batch_desc ok{};
    ok.num_instances = 2; ok.req_offsets = off; ok.arrival = a; ok.prompt = s; ok.output = o;
    ok.M = 20; ok.num_policies = 2; ok.policies = pol;
    svf_batch_desc d = ok;
    d.req_offsets = nullptr;
    refuse(d, SVF_EINVAL, "NULL offsets");
    d = ok; d.arrival = nullptr;
    refuse(d, SVF_EINVAL, "NULL arrival");
    d = ok; d.num_instances = -1;
    refuse(d, SVF_EINVAL, "negative instance count");
    const int64_t off_bad[3] = {0, 4, 3};
    d = ok; d.req_offsets = off_bad;
    refuse(d, SVF_EINVAL, "decreasing offsets");
    const int32_t a_bad[5] = {2, 1, 1, 0, 4};
    d = ok; d.arrival = a_bad;
    refuse(d, SVF_EINVAL, "arrivals out of order");
    const int32_t s_bad[5] = {2, 0, 4, 1, 1};
    d = ok; d.prompt = s_bad;
    refuse(d, SVF_EINVAL, "prompt < 1");
    const int32_t o_bad[5] = {5, 6, 7, 2, 0};
    d = ok; d.output = o_bad;
    refuse(d, SVF_EINVAL, "output < 1");
    d = ok; d.M = 8;
    refuse(d, SVF_EINFEASIBLE, "request larger than M");
    d = ok; d.M = int64_t(1) << 30;
    refuse(d, SVF_EINVAL, "M too large");
    d = ok; d.num_policies = 0;
    refuse(d, SVF_EINVAL, "no policy");
    d = ok; d.num_policies = 9;
    refuse(d, SVF_EINVAL, "too many policies");
    const int32_t pol_bad[2] = {SVF_POLICY_SVF, 77};
    d = ok; d.policies = pol_bad;
    refuse(d, SVF_EINVAL, "unknown policy");
    const int32_t pol_bit[1] = {SVF_POLICY_SVF1BIT};
    d = ok; d.policies = pol_bit; d.num_policies = 1;
    refuse(d, SVF_EINVAL, "1-bit policy without bits");
    const int8_t bits[5] = {0, 1, 1, 0, 0};
    d.long_bit = bits; d.O0 = 0; d.O1 = 3;
    refuse(d, SVF_EINVAL, "1-bit policy with O0 = 0");
    d.O0 = 1; d.O1 = 40;
    refuse(d, SVF_EINFEASIBLE, "1-bit proxy larger than M");
    const int32_t plan_bad[5] = {1, 1, 0, 1, 1};
    d = ok; d.plan_len = plan_bad;
    refuse(d, SVF_EINVAL, "plan < 1");
    d = ok; d.max_steps = -1;
    refuse(d, SVF_EINVAL, "negative step budget");
    const int32_t s_key[5] = {65535, 3, 4, 1, 1}, o_key[5] = {65535, 6, 7, 2, 2};
    d = ok; d.prompt = s_key; d.output = o_key; d.M = int64_t(1) << 29;
    refuse(d, SVF_EINVAL, "key overflow");
    expect(svf_create(nullptr, nullptr, nullptr) == SVF_EINVAL, "NULL out");
    svf_batch* h = nullptr;
    expect(svf_create(nullptr, nullptr, &h) == SVF_EINVAL, "NULL desc");
    expect(svf_reset(nullptr) == SVF_EINVAL, "reset NULL");
    expect(svf_step(nullptr, 1) == SVF_EINVAL, "step NULL");
    expect(svf_run(nullptr) == SVF_EINVAL, "run NULL");
    expect(svf_read(nullptr, 0, nullptr, nullptr, nullptr, nullptr, 0) == SVF_EINVAL, "read NULL");
    expect(svf_stats(nullptr, 0, nullptr) == SVF_EINVAL, "stats NULL");
    expect(svf_destroy(nullptr) == SVF_OK, "destroy NULL");
    expect(svf_run_noalloc(nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr) ==
               SVF_EINVAL, "noalloc NULL desc");
    d = ok;
    expect(svf_run_noalloc(&d, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr) == SVF_EINVAL,
           "noalloc NULL outputs");
    d.inputs_on_device = 1;
    int32_t dummy[16];
    svf_instance_stats st[4];
    expect(svf_run_noalloc(&d, nullptr, dummy, dummy, dummy, dummy, st) == SVF_EINVAL,
           "noalloc device inputs");
    printf("errors: %s\n", failures ? "FAILED" : "ok");
    return failures ? 1 : 0;
}

int create_mode(const char* in) {
    const Batch b = load(in);
    const svf_batch_desc d = b.desc();
    svf_batch* h = nullptr;
    const int rc = svf_create(&d, nullptr, &h);
    // on a machine without a GPU the first HIP call fails after validation
    printf("create: rc %d (%s)\n", rc, rc ? svf_last_error() : "ok");
    if (rc == SVF_OK) svf_destroy(h);
    return (rc == SVF_OK || rc == SVF_EHIP || rc == SVF_ENOMEM) ? 0 : 1;
}

struct Outputs {
    std::vector<int32_t> v;  // per slot: start, finish, preempt, admit_seq
    std::vector<svf_instance_stats> st;
};

bool collect(svf_batch* h, const Batch& b, Outputs& out) {
    const size_t P = b.pol.size(), N = (size_t)b.N, I = (size_t)b.I;
    out.v.assign(P * 4 * N, 0);
    out.st.assign(P * I, svf_instance_stats{});
    for (size_t p = 0; p < P; ++p) {
        int32_t* base = out.v.data() + p * 4 * N;
        if (svf_read(h, (int32_t)p, base, base + N, base + 2 * N, base + 3 * N, 0) != SVF_OK)
            return false;
        if (svf_stats(h, (int32_t)p, out.st.data() + p * I) != SVF_OK) return false;
    }
    return true;
}

bool same(const Outputs& x, const Outputs& y) {
    return x.v == y.v && x.st.size() == y.st.size() &&
           (x.st.empty() || !memcmp(x.st.data(), y.st.data(), x.st.size() * sizeof(svf_instance_stats)));
}

int run_mode(const char* in, const char* outp) {
    const Batch b = load(in);
    const svf_batch_desc d = b.desc();
    const size_t P = b.pol.size(), N = (size_t)b.N, I = (size_t)b.I;
    Outputs whole, chunks, na;
    svf_batch* h = nullptr;
    expect(svf_create(&d, nullptr, &h) == SVF_OK, "create");
    if (!h) return 1;
    expect(svf_run(h) == SVF_OK, "run");
    expect(collect(h, b, whole), "read whole run");
    // again after a reset, in steps of irregular size
    expect(svf_reset(h) == SVF_OK, "reset");
    for (int64_t k : {int64_t(7), int64_t(1), int64_t(100), int64_t(1) << 40})
        expect(svf_step(h, k) == SVF_OK, "step");
    expect(collect(h, b, chunks), "read chunked run");
    expect(same(whole, chunks), "chunked run equals the whole run");
    expect(svf_destroy(h) == SVF_OK, "destroy");
    // the no-allocation entry point, outputs in device memory of the caller
    int32_t* dv = nullptr;
    svf_instance_stats* ds = nullptr;
    const size_t nv = std::max<size_t>(P * N, 1), ns = std::max<size_t>(P * I, 1);
    expect(hipMalloc(&dv, 4 * 4 * nv) == hipSuccess, "hipMalloc outputs");
    expect(hipMalloc(&ds, sizeof(svf_instance_stats) * ns) == hipSuccess, "hipMalloc stats");
    if (dv && ds) {
        expect(svf_run_noalloc(&d, nullptr, dv, dv + nv, dv + 2 * nv, dv + 3 * nv, ds) == SVF_OK,
               "run_noalloc");
        std::vector<int32_t> hv(4 * nv);
        na.st.assign(P * I, svf_instance_stats{});
        expect(hipMemcpy(hv.data(), dv, 4 * 4 * nv, hipMemcpyDeviceToHost) == hipSuccess, "copy");
        if (P * I)
            expect(hipMemcpy(na.st.data(), ds, sizeof(svf_instance_stats) * P * I,
                             hipMemcpyDeviceToHost) == hipSuccess, "copy stats");
        na.v.assign(P * 4 * N, 0);
        for (size_t p = 0; p < P; ++p)
            for (size_t f = 0; f < 4; ++f)
                memcpy(na.v.data() + (p * 4 + f) * N, hv.data() + f * nv + p * N, 4 * N);
        expect(same(whole, na), "run_noalloc equals the handle");
    }
    (void)hipFree(dv);
    (void)hipFree(ds);
    FILE* f = fopen(outp, "wb");
    if (!f) return 2;
    for (size_t p = 0; p < P; ++p) {
        fwrite(whole.v.data() + p * 4 * N, 4, 4 * N, f);
        fwrite(whole.st.data() + p * I, sizeof(svf_instance_stats), I, f);
    }
    fclose(f);
    printf("run: %s\n", failures ? "FAILED" : "ok");
    return failures ? 1 : 0;
}

}  // namespace

int main(int argc, char** argv) {
    if (argc >= 2 && !strcmp(argv[1], "errors")) return errors_mode();
    if (argc >= 3 && !strcmp(argv[1], "create")) return create_mode(argv[2]);
    if (argc >= 4 && !strcmp(argv[1], "run")) return run_mode(argv[2], argv[3]);
    fprintf(stderr, "usage: %s errors | create IN | run IN OUT\n", argv[0]);
    return 2;
}
