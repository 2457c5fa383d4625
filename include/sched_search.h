/*
 * sched_search.h -- brute-force device-mapping search on one AMD Instinct MI355X.
 *
 * A workflow is a DAG of tools; every tool runs in one of three modes
 * (Section 2.1): 0 = cpu, 1 = gpu_now (immediate GPU, holds its footprint
 * while it runs, an over-budget start is an out-of-memory failure), 2 =
 * gpu_queue (serialized GPU queue, holds no VRAM while waiting, pays load-in).
 * A mapping assigns a mode to every tool; its index is sum_v mode_v * 3^v
 * (tool 0 is the least significant digit).  A problem may restrict each tool
 * to a subset of the modes (sched_problem_create_masked): then the index is
 * mixed radix, sum_v digit_v * W_v, where digit_v is the rank of the tool's
 * mode among its r_v allowed modes (ascending) and W_v = r_0 ... r_(v-1); with
 * every mode allowed this is the base-3 index above.  The library scores mappings with
 * an integer event-driven schedule (GPU-utilisation contention as a Q16
 * slowdown fixed at each GPU start by the number of co-running GPU tools,
 * VRAM admission, FIFO queue on (ready time, tool), PCIe transfer charged to
 * the consumer of an edge whose ends sit on different devices) and returns
 * the feasible mapping of lowest makespan, ties to the lowest index: the
 * exhaustive-search reference of Sections 2.3 and 4.1, with the measured
 * latency replaced by the model.
 *
 * Units: time in integer microseconds, memory in integer MiB, contention
 * factors in Q16 (65536 = 1.0x).  All calls are thread-safe on distinct
 * workspaces; a problem handle is immutable after creation.
 *
 * Ownership: every host pointer argument is owned by the caller and only
 * read (or, for outputs, written) during the call.  The library never
 * allocates device memory: device work runs in the caller's workspace on the
 * caller's HIP stream, and every entry point that launches work waits for
 * that stream before returning.  On error no output is written.
 */
#ifndef SCHED_SEARCH_H
#define SCHED_SEARCH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Error codes (negative; 0 is success). */
#define SCHED_OK 0
#define SCHED_E_NULL (-1)      /* a required pointer is null */
#define SCHED_E_SIZE (-2)      /* n_tools not in [1,40], n_levels not in [1,64],
                                  a negative count, n_replicas < 1 */
#define SCHED_E_VALUE (-3)     /* gpu_us or cpu_us < 1; load, xfer, mem or
                                  budget < 0; a factor < 65536 or > 2^24; an
                                  option mask outside [1, 7]; a mode that the
                                  problem does not allow; a contention mode
                                  other than 0 or 1 */
#define SCHED_E_EDGE (-4)      /* edge endpoint out of range, or a self-loop */
#define SCHED_E_CYCLE (-5)     /* the edges contain a cycle */
#define SCHED_E_RANGE (-6)     /* lo >= hi or hi > the number of mappings; an
                                  index beyond it; replica map out of range */
#define SCHED_E_OVERFLOW (-7)  /* the worst-case makespan bound reaches 2^30 us,
                                  or (N+1)*(budget+1) reaches 2^32: the device
                                  path keeps times and VRAM sums in 32 bits */
#define SCHED_E_WORKSPACE (-8) /* workspace null, misaligned (256 B) or too small */
#define SCHED_E_DEVICE (-9)    /* a HIP runtime call failed */
#define SCHED_E_NOMEM (-10)    /* host allocation failed */

/* Tool card: the per-tool profile of Section 3.1 (CPU, GPU and load-in times,
 * VRAM footprint) plus the input-transfer cost paid when a predecessor runs
 * on the other device. */
typedef struct {
    int64_t gpu_us;  /* isolated GPU latency, >= 1 */
    int64_t cpu_us;  /* isolated CPU latency, >= 1 */
    int64_t load_us; /* load-in paid by gpu_queue, >= 0 */
    int64_t xfer_us; /* input transfer across devices, >= 0 */
    int64_t mem_mib; /* VRAM footprint while running on the GPU, >= 0 */
} sched_tool;

/* Re-measured latencies of one replica (running averages, Section 3.2);
 * footprints, edges, budget and contention stay those of its problem. */
typedef struct {
    int64_t gpu_us, cpu_us, load_us, xfer_us;
} sched_lat;

/* Data dependency: dst starts only after src completes (Section 2.1). */
typedef struct {
    int32_t src, dst;
} sched_edge;

/* Search result.  With no feasible mapping in the range: best_index =
 * UINT64_MAX and makespan_us = INT64_MAX (on a full range this cannot
 * happen: index 0, all tools on the CPU, is always feasible). */
typedef struct {
    uint64_t best_index;
    int64_t makespan_us;
} sched_result;

typedef struct sched_problem sched_problem;

/* Validate and freeze a problem (Section 2.1: DAG G=(V,E), modes, tau,
 * budget M).  tools: n_tools cards; edges: n_edges pairs (duplicates are
 * ignored); contention_q16: F[k-1] for k = 1..n_levels co-running GPU tools,
 * each in [65536, 2^24], levels beyond n_levels use the last one;
 * vram_budget_mib: the budget M.  On success *out receives a handle to free
 * with sched_problem_destroy.  Host-only: touches no device. */
int sched_problem_create(const sched_tool *tools, int32_t n_tools,
                         const sched_edge *edges, int32_t n_edges,
                         const uint32_t *contention_q16, int32_t n_levels,
                         int64_t vram_budget_mib, sched_problem **out);

/* The same with a per-tool decision space: allowed[v] (n_tools entries) has
 * bit m set when tool v may run in mode m (bit 0 cpu, bit 1 gpu_now, bit 2
 * gpu_queue), each in [1, 7].  Covers the binary GPU/CPU space of S1-S10
 * (Section 4.1 and Table 3: cpu or gpu_now, 2^N mappings) and tools with no
 * GPU implementation (the neutral tools of Table 1: cpu only).  A tool with a
 * single allowed mode takes no digit of the index. */
int sched_problem_create_masked(const sched_tool *tools, int32_t n_tools,
                                const sched_edge *edges, int32_t n_edges,
                                const uint32_t *contention_q16, int32_t n_levels,
                                int64_t vram_budget_mib, const uint8_t *allowed,
                                sched_problem **out);

/* All creation parameters in one place (the two calls above are shorthands).
 * allowed: as for sched_problem_create_masked, or null for every mode.
 * contention_mode: how concurrent GPU tools slow each other (Section 2.3,
 * Factor A; the paper measures it and states no rule):
 *   0  fixed at start: a GPU tool starting while k GPU tools run (itself
 *      included) lasts round(b * F[min(k, K)] / 2^16), for its whole run;
 *   1  processor sharing: every running GPU tool advances at 1 / F[min(k, K)]
 *      of its isolated speed, k recounted at every start and end (work in
 *      units of 2^-16 us, rates round(2^32 / F) halves up). */
typedef struct {
    const sched_tool *tools;
    int32_t n_tools;
    const sched_edge *edges;
    int32_t n_edges;
    const uint32_t *contention_q16;
    int32_t n_levels;
    int64_t vram_budget_mib;
    const uint8_t *allowed;
    int32_t contention_mode;
} sched_problem_desc;

int sched_problem_create_desc(const sched_problem_desc *desc, sched_problem **out);

void sched_problem_destroy(sched_problem *p);

/* Modes of mapping `index` (n_tools entries written to modes), and the index
 * of per-tool modes (SCHED_E_VALUE if a mode is not allowed).  Host-only. */
int sched_mapping_modes(const sched_problem *p, uint64_t index, int32_t *modes);
int sched_mapping_index(const sched_problem *p, const int32_t *modes, uint64_t *index);

/* Number of tools and of mappings (3^N, or the product of the radices) of a
 * problem. */
int sched_num_tools(const sched_problem *p, int32_t *out);
int sched_num_mappings(const sched_problem *p, uint64_t *out);

/* Bytes of device workspace sufficient for any call below on these
 * problems with up to n_replicas replicas (n_replicas = 0 for calls without
 * replicas).  Host-only. */
int sched_workspace_bytes(const sched_problem *const *problems, int32_t n_problems,
                          int32_t n_replicas, size_t *out);

/* Exhaustive search over mapping indices [lo, hi) of problem p (the oracle
 * of Sections 2.3 and 4.1).  d_workspace: device memory of ws_bytes, 256-byte
 * aligned; hip_stream: a hipStream_t (null = default stream).  Writes *h_out
 * (host) after the stream has finished. */
int sched_bruteforce_argmin(const sched_problem *p, uint64_t lo, uint64_t hi,
                            void *d_workspace, size_t ws_bytes, void *hip_stream,
                            sched_result *h_out);

/* For callers that cannot allocate device memory or pass a workspace (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): sched_bruteforce_argmin without a workspace argument.  The
 * table, block partials and result live in a fixed per-GPU array of the
 * library (2 MiB, held by each GPU the library runs on until the process
 * ends); the call allocates nothing (no hipMalloc, hipFree or heap memory).
 * Every call on a GPU shares that GPU's array: calls that overlap on one GPU
 * (several host threads or streams at once) race and must be serialized by
 * the caller.  Nothing in the array needs to start at zero: each call writes
 * what it reads.  Errors as for sched_bruteforce_argmin; SCHED_E_WORKSPACE if
 * the problem's table and partials do not fit the array (never for problems
 * sched_problem_create accepts). */
int sched_bruteforce_argmin_noalloc(const sched_problem *p, uint64_t lo, uint64_t hi,
                                    void *hip_stream, sched_result *h_out);

/* Diagnostic for parity tests, not part of the method: the full-range search
 * of sched_bruteforce_argmin over [0, number of mappings), with the same plan
 * and kernels (shared schedule prefixes included), that also writes the
 * makespan of every mapping it scores to d_makespan[index] (device, uint32,
 * 0xFFFFFFFF when infeasible).  Every mapping is scored exactly once, so each
 * entry is written once.  capacity: entries of d_makespan, at least the
 * number of mappings (else SCHED_E_WORKSPACE); d_workspace as for
 * sched_bruteforce_argmin.  *h_out receives the search result. */
int sched_bruteforce_record(const sched_problem *p, void *d_workspace, size_t ws_bytes,
                            void *hip_stream, uint32_t *d_makespan, uint64_t capacity,
                            sched_result *h_out);

/* Batched re-scoring of perturbed profiles (the running-average feedback of
 * Section 3.2): replica r is problem replica_problem[r] with the latencies
 * replica_lat[off_r .. off_r + N_r), where off_r is the sum of N over the
 * earlier replicas.  Each replica gets its own exhaustive search over all
 * mappings of its problem; h_out[r] receives its result. */
int sched_eval_batch(const sched_problem *const *problems, int32_t n_problems,
                     const int32_t *replica_problem, const sched_lat *replica_lat,
                     int32_t n_replicas, void *d_workspace, size_t ws_bytes,
                     void *hip_stream, sched_result *h_out);

/* Score explicit mappings (the what-if probes of Section 3.2): h_idx is a
 * host array of n indices, each below the number of mappings (else
 * SCHED_E_RANGE, checked before any device work); h_makespan (host, n
 * entries) receives each mapping's makespan in us, or INT64_MAX when it is
 * infeasible.  The library copies the indices through d_workspace in chunks
 * (at least one index beyond the problem table must fit; the bytes of
 * sched_workspace_bytes take 65,536 per chunk) and waits for the stream. */
int sched_eval_mappings(const sched_problem *p, const uint64_t *h_idx, int64_t n,
                        void *d_workspace, size_t ws_bytes, void *hip_stream,
                        int64_t *h_makespan);

/* The same on device arrays (no host copies): d_idx and d_makespan hold n
 * entries each; an index beyond the number of mappings yields INT64_MAX.  The
 * workspace holds the problem table only. */
int sched_eval_mappings_device(const sched_problem *p, const uint64_t *d_idx, int64_t n,
                               int64_t *d_makespan, void *d_workspace, size_t ws_bytes,
                               void *hip_stream);

/* One what-if probe around a base mapping. */
typedef struct {
    uint64_t index;      /* mapping probed */
    int64_t makespan_us; /* INT64_MAX when infeasible */
    int32_t kind;        /* 0: the base mapping, 1: single-tool move, 2: swap */
    int32_t tool;        /* tool moved (-1 for the base) */
    int32_t mode;        /* its new mode (0 cpu, 1 gpu_now, 2 gpu_queue) */
    int32_t swap_tool;   /* swap: tool moved from gpu_now to gpu_queue; else -1 */
} sched_probe;

/* Bounded what-if exploration around base_index, the runtime monitor's active
 * path (Section 3.2, Algorithm 1): the base mapping first; then for each tool
 * i in order and each other allowed mode a of tool i in the order cpu,
 * gpu_now, gpu_queue, the single-tool move i -> a; right after a move to
 * gpu_now that is infeasible (over the VRAM budget), one swap per tool j on
 * gpu_now in the base mapping that may use gpu_queue (ascending j):
 * i -> gpu_now with j -> gpu_queue.
 * lat: optional re-measured latencies (N entries, e.g. running averages) that
 * replace the problem's own for these probes; null keeps the profiles.
 * h_out: host array of capacity entries; capacity must be at least
 * 1 + 2N + N(N-1).  *n_out receives the number of probes written. */
int sched_eval_reprobes(const sched_problem *p, uint64_t base_index, const sched_lat *lat,
                        void *d_workspace, size_t ws_bytes, void *hip_stream,
                        sched_probe *h_out, int32_t capacity, int32_t *n_out);

/* Counters of one pruned search. */
typedef struct {
    uint64_t prefixes;          /* assignments of the prefix tools that were bounded */
    uint64_t prefixes_searched; /* prefixes whose subspace was searched exhaustively */
    uint64_t mappings_searched; /* mappings scored by those searches */
    int64_t initial_bound_us;   /* makespan of the descent's mapping (INT64_MAX if none) */
    int32_t prefix_tools;       /* tools in the prefix (0: one exhaustive search) */
    int32_t descent_rounds;     /* neighbourhood evaluations of the descent */
    int32_t launches;           /* exhaustive-search launches */
    int32_t shared_prefix_launches; /* of those, launches on the shared-prefix plan */
} sched_prune_stats;

/* Exact search with pruning: the same result as sched_bruteforce_argmin over
 * every mapping (the lowest makespan, ties to the lowest index), for spaces
 * too large to enumerate (the problem is NP-hard, Section 2.3).  An upper
 * bound comes from steepest descent over the what-if neighbourhood of
 * Algorithm 1 from index 0.  The tools whose modes move the bound most form a
 * prefix; every prefix assignment gets a lower bound (critical path of the
 * shortest durations, queued durations summed) and only assignments whose
 * bound does not exceed the best makespan found so far have their remaining
 * tools searched exhaustively, most promising first.  Spaces below 2^22
 * mappings get one exhaustive search.  d_workspace: at least
 * sched_pruned_workspace_bytes(p) bytes, 256-byte aligned.  stats: optional
 * counters (host). */
int sched_pruned_workspace_bytes(const sched_problem *p, size_t *out);
int sched_pruned_argmin(const sched_problem *p, void *d_workspace, size_t ws_bytes,
                        void *hip_stream, sched_result *h_out, sched_prune_stats *stats);

/* Sliding-window latency statistics: the runtime monitor's observation
 * feedback (Section 3.2, Algorithm 1, passive path).  For every tool and mode
 * the monitor keeps the `window` most recent measured latencies and reports
 * their running average; re-scoring with those averages in place of the
 * isolated profiles (sched_eval_batch, sched_eval_reprobes) exposes the
 * latency the previous mappings actually induced.  Host-only. */
typedef struct sched_monitor sched_monitor;

/* n_tools in [1, 40], window >= 1. */
int sched_monitor_create(int32_t n_tools, int32_t window, sched_monitor **out);
void sched_monitor_destroy(sched_monitor *m);

/* Record one executed round: tool v ran in mode modes[v] (0, 1 or 2) for
 * latency_us[v] (for gpu_queue, load-in included); a negative latency means
 * tool v was not observed.  The oldest value of a full window is dropped. */
int sched_monitor_observe(sched_monitor *m, const int32_t *modes, const int64_t *latency_us);

/* Running averages: for tool v and mode k, entry 3v + k of mean_us gets the
 * mean of its window rounded half up (0 if empty) and of count the number of
 * values in it.  Both arrays hold 3 * n_tools entries. */
int sched_monitor_averages(const sched_monitor *m, int64_t *mean_us, int32_t *count);

/* Latencies for re-scoring (n_tools entries): the profile (n_tools cards)
 * with every observed quantity replaced by its running average: cpu_us by
 * the cpu average, gpu_us by the gpu_now average, load_us by the gpu_queue
 * average minus that gpu_us (at least 0); xfer_us is kept.  An average is
 * used as a base latency: the schedule model still applies its contention
 * factor on top. */
int sched_monitor_latencies(const sched_monitor *m, const sched_tool *profile, sched_lat *out);

/* Diagnostic, not part of the method: the integer VALU throughput probe that
 * gives the search's roofline an empirical ceiling next to the published
 * peak.  Launches `blocks` blocks of 256 lanes on hip_stream; every lane runs
 * `iters` steps of 8 independent chains of an add, a max, a compare and a
 * select (32 int32 VALU operations per step) and writes one word of d_out
 * (device, at least blocks * 256 uint32).  *lane_ops (host) receives the
 * int32 lane operations of the launch.  Waits for the stream before
 * returning.  Errors: SCHED_E_NULL (d_out or lane_ops null), SCHED_E_SIZE
 * (blocks or iters 0, blocks > 2^24), SCHED_E_DEVICE. */
int sched_valu_probe(uint32_t blocks, uint32_t iters, uint32_t *d_out, void *hip_stream,
                     double *lane_ops);

/* Diagnostic, not part of the method: a check of the wave-wide OR through
 * LDS that the search uses to skip tools no lane of a wave needs to visit.
 * Launches `blocks` blocks of 256 lanes on hip_stream; lane g takes part when
 * d_active[g] is non-zero and then writes to d_out64[g] the bitwise OR of
 * d_in over the active lanes of its wave (64 consecutive lanes), and to
 * d_out32[g] the OR of bits 16..47 of d_in over the same lanes; lanes that do
 * not take part write all ones.  All arrays are device memory of blocks * 256
 * entries, owned by the caller.  Waits for the stream before returning.
 * Errors: SCHED_E_NULL (an array null), SCHED_E_SIZE (blocks 0 or > 2^16),
 * SCHED_E_DEVICE. */
int sched_wave_or_probe(const uint64_t *d_in, const uint8_t *d_active, uint32_t blocks,
                        uint64_t *d_out64, uint32_t *d_out32, void *hip_stream);

/* Static text for an error code. */
const char *sched_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* SCHED_SEARCH_H */
