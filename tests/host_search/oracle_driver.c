/* oracle_driver.c -- test harness: runs the oracle's threaded entry points
 * (argmin over every mapping, evaluation of every index, both contention
 * readings) on one instance read from stdin, for builds of the oracle under
 * AddressSanitizer + UndefinedBehaviorSanitizer and ThreadSanitizer.
 * Input: n n_edges n_levels budget, n lines "gpu cpu load xfer mem", n_edges
 * lines "src dst", n_levels Q16 factors.  Prints "<index> <makespan>" for the
 * fixed-at-start argmin, the processor-sharing argmin, and the sum of the
 * feasible makespans of every index. */
#include <inttypes.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_problem_size(void);
int oracle_problem_init(void *P, int32_t n, const int64_t *tools, int32_t n_edges,
                        const int32_t *edges, int32_t n_levels, const int64_t *contention,
                        int64_t budget);
void oracle_set_sharing(void *P, int32_t sharing);
uint64_t oracle_num_mappings(const void *P);
void oracle_argmin(const void *P, uint64_t lo, uint64_t hi, int32_t nthreads,
                   uint64_t *best_index, int64_t *best_makespan);
void oracle_eval_many(const void *P, const uint64_t *idx, int64_t count, int32_t nthreads,
                      int64_t *out);

int main(void) {
    int n, ne, nl;
    long long budget;
    if (scanf("%d %d %d %lld", &n, &ne, &nl, &budget) != 4 || n < 1 || n > 40 || ne < 0 ||
        nl < 1 || nl > 64)
        return 2;
    int64_t *tools = malloc(sizeof(int64_t) * 5 * (size_t)n);
    int32_t *edges = malloc(sizeof(int32_t) * 2 * (size_t)(ne > 0 ? ne : 1));
    int64_t *f = malloc(sizeof(int64_t) * (size_t)nl);
    for (int i = 0; i < 5 * n; i++) {
        long long x;
        if (scanf("%lld", &x) != 1) return 2;
        tools[i] = x;
    }
    for (int i = 0; i < 2 * ne; i++)
        if (scanf("%d", &edges[i]) != 1) return 2;
    for (int i = 0; i < nl; i++) {
        long long x;
        if (scanf("%lld", &x) != 1) return 2;
        f[i] = x;
    }
    void *P = malloc((size_t)oracle_problem_size());
    if (oracle_problem_init(P, n, tools, ne, edges, nl, f, budget) != 0) return 3;
    const uint64_t total = oracle_num_mappings(P);
    uint64_t bi;
    int64_t bm;
    oracle_argmin(P, 0, total, 4, &bi, &bm);
    printf("%" PRIu64 " %" PRId64 "\n", bi, bm);
    oracle_set_sharing(P, 1);
    oracle_argmin(P, 0, total, 4, &bi, &bm);
    printf("%" PRIu64 " %" PRId64 "\n", bi, bm);
    oracle_set_sharing(P, 0);
    uint64_t *idx = malloc(sizeof(uint64_t) * total);
    int64_t *out = malloc(sizeof(int64_t) * total);
    for (uint64_t x = 0; x < total; x++) idx[x] = x;
    oracle_eval_many(P, idx, (int64_t)total, 4, out);
    int64_t sum = 0;
    for (uint64_t x = 0; x < total; x++)
        if (out[x] != INT64_MAX) sum += out[x];
    printf("%" PRId64 "\n", sum);
    free(idx);
    free(out);
    free(P);
    free(tools);
    free(edges);
    free(f);
    return 0;
}
