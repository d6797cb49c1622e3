/*
 * Test driver: runs the CPU oracle (oracle/svf_oracle.c) on one batch read
 * from a file and writes its outputs to another, so that the oracle can be
 * built with the address and undefined-behaviour sanitizers into a program
 * of its own (tests/test_sanitizers.py).
 *
 * Input (native byte order): int64 I, N, M, policy, O0, O1, max_steps,
 * t_stop, threads, has_plan, has_bit; int64 offsets[I + 1]; int32 a[N],
 * s[N], o[N]; int32 plan[N] if has_plan; int8 bit[N] if has_bit.
 * Output: int32 start[N], finish[N], preempt[N], admit_seq[N]; int64
 * stats[I * 8].
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_run(int32_t num_instances, const int64_t *offsets, const int32_t *a,
               const int32_t *s, const int32_t *o, const int32_t *plan,
               const int8_t *bit, int64_t M, int32_t policy, int32_t O0, int32_t O1,
               int64_t max_steps, int64_t t_stop, int32_t threads, int32_t *start,
               int32_t *finish, int32_t *preempt, int32_t *admit_seq, int64_t *stats);

static void *read_array(FILE *f, size_t elem, int64_t count) {
    void *p = malloc(elem * (size_t)(count > 0 ? count : 1));
    if (!p || fread(p, elem, (size_t)count, f) != (size_t)count) {
        fprintf(stderr, "short input\n");
        exit(2);
    }
    return p;
}

int main(int argc, char **argv) {
    if (argc != 3) {
        fprintf(stderr, "usage: %s input output\n", argv[0]);
        return 2;
    }
    FILE *in = fopen(argv[1], "rb");
    if (!in) return 2;
    int64_t h[11];
    if (fread(h, sizeof(int64_t), 11, in) != 11) return 2;
    const int64_t I = h[0], N = h[1];
    int64_t *off = read_array(in, 8, I + 1);
    int32_t *a = read_array(in, 4, N), *s = read_array(in, 4, N), *o = read_array(in, 4, N);
    int32_t *plan = h[9] ? read_array(in, 4, N) : NULL;
    int8_t *bit = h[10] ? read_array(in, 1, N) : NULL;
    fclose(in);
    const size_t n1 = (size_t)(N > 0 ? N : 1), i1 = (size_t)(I > 0 ? I : 1);
    int32_t *start = malloc(4 * n1), *finish = malloc(4 * n1), *pre = malloc(4 * n1),
            *seq = malloc(4 * n1);
    int64_t *stats = calloc(8 * i1, 8);
    if (!start || !finish || !pre || !seq || !stats) return 2;
    oracle_run((int32_t)I, off, a, s, o, plan, bit, h[2], (int32_t)h[3], (int32_t)h[4],
               (int32_t)h[5], h[6], h[7], (int32_t)h[8], start, finish, pre, seq, stats);
    FILE *out = fopen(argv[2], "wb");
    if (!out) return 2;
    fwrite(start, 4, (size_t)N, out);
    fwrite(finish, 4, (size_t)N, out);
    fwrite(pre, 4, (size_t)N, out);
    fwrite(seq, 4, (size_t)N, out);
    fwrite(stats, 8, (size_t)(8 * I), out);
    fclose(out);
    free(off); free(a); free(s); free(o); free(plan); free(bit);
    free(start); free(finish); free(pre); free(seq); free(stats);
    return 0;
}
