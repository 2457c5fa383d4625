/*
 * oracle.c -- plain CPU reference for the brute-force device-mapping search.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the bench's
 * CPU-baseline leg load this file's library.  It shares no code, header or
 * table with the HIP path and must never be used as a fallback for it.
 *
 * What it computes.  A workflow is a DAG of tools (Section 2.1).  Each tool v
 * runs in one mode a_v of {cpu, gpu_now, gpu_queue}, digit 0, 1 or 2 of the
 * mapping index (tool 0 is the least significant base-3 digit).  A mapping is
 * scored by an integer, event-driven simulation of the schedule; the paper's
 * own oracle measures wall-clock time instead (Sections 2.3 and 4.1), and
 * gives no analytical model, so the simulation rules below are a reading of
 * Section 2.1 (modes, VRAM inequality, T_e2e = max over sinks of C_v) and
 * Section 2.3 (Factor A: concurrent GPU tools slow each other while CPU time
 * is unaffected; Factor B: an immediate GPU start over the budget is an
 * out-of-memory failure, queued tools wait and pay load-in).
 *
 *   base latency   b(v,cpu) = cpu_us, b(v,gpu_now) = gpu_us,
 *                  b(v,gpu_queue) = gpu_us + load_us           (tau, Sec. 2.1)
 *   ready time     r_v = max over edges u->v of C_u + xfer_us[v] when u and v
 *                  sit on different devices (0 for sources)
 *   at each event time t, in this order:
 *     1. release   running tasks with C_u <= t finish and free their VRAM
 *     2. starts    every waiting cpu / gpu_now task with all predecessors
 *                  finished and r_v <= t starts at t; if the VRAM held by
 *                  running GPU tasks plus the new gpu_now starts exceeds the
 *                  budget M, the mapping is infeasible (out of memory)
 *     3. queue     if no gpu_queue task is running, the waiting gpu_queue
 *                  task with the smallest (r_v, v) among the ready ones is
 *                  admitted iff its footprint fits the free VRAM
 *     4. durations k = number of GPU tasks running after steps 2-3; a GPU
 *                  task starting now gets C_v = t + round(b * F[min(k,K)] /
 *                  2^16) (Q16, halves up), fixed for its lifetime; a CPU task
 *                  gets C_v = t + cpu_us
 *     5. next      t = the smallest finish time or ready time after t; with
 *                  tasks left and no such time the mapping is infeasible
 *   makespan = max_v C_v (equal to the max over sinks, Sec. 2.1).
 *
 * Processor sharing (the other reading of Factor A, selected per problem):
 * a GPU task's duration is not fixed at its start; every running GPU task
 * advances at the same rate, 1 / F[min(k, K)] of the isolated speed, with k
 * recounted at every event.  In integers: a GPU task holds W = b * 2^16 units
 * of work; while k GPU tasks run, each completes w_k = round(2^32 / F[k])
 * units per microsecond (halves up); the next GPU finish is t + ceil(R_min /
 * w_k) for the least remaining work R_min; at the next event every running
 * GPU task's remaining work drops by (t' - t) * w_k and those at or below 0
 * finish at t'.  Steps 1-3 and the CPU are as above.
 *
 * Search: the lowest makespan over an index range [lo, hi), ties to the
 * lowest index; infeasible mappings are never chosen.  Everything is int64.
 */
#include <pthread.h>
#include <stdint.h>
#include <string.h>

#define OR_MAXN 40
#define OR_MAXLEV 64
#define OR_INFEASIBLE INT64_MAX

enum { OR_CPU = 0, OR_GPU_NOW = 1, OR_GPU_QUEUE = 2 };
enum { WAITING = 0, RUNNING = 1, DONE = 2 };

typedef struct {
    int32_t n;
    int32_t n_levels;
    int64_t budget;
    int64_t gpu[OR_MAXN], cpu[OR_MAXN], load[OR_MAXN], xfer[OR_MAXN], mem[OR_MAXN];
    int64_t contention[OR_MAXLEV]; /* F[k-1] for k = 1..K, Q16 */
    int32_t npred[OR_MAXN];
    int32_t pred[OR_MAXN][OR_MAXN];
    int32_t sharing; /* 0: fixed at start, 1: processor sharing */
} or_problem;

int oracle_problem_size(void) { return (int)sizeof(or_problem); }

/* Fill a problem from flat arrays.  tools: n rows of (gpu, cpu, load, xfer,
 * mem); edges: n_edges pairs (src, dst), duplicates ignored.  Returns 0, or
 * -1 when a size or endpoint is out of range. */
int oracle_problem_init(or_problem *P, int32_t n, const int64_t *tools,
                        int32_t n_edges, const int32_t *edges,
                        int32_t n_levels, const int64_t *contention,
                        int64_t budget) {
    if (n < 1 || n > OR_MAXN || n_levels < 1 || n_levels > OR_MAXLEV) return -1;
    memset(P, 0, sizeof(*P));
    P->n = n;
    P->n_levels = n_levels;
    P->budget = budget;
    for (int v = 0; v < n; v++) {
        P->gpu[v] = tools[5 * v + 0];
        P->cpu[v] = tools[5 * v + 1];
        P->load[v] = tools[5 * v + 2];
        P->xfer[v] = tools[5 * v + 3];
        P->mem[v] = tools[5 * v + 4];
    }
    for (int k = 0; k < n_levels; k++) P->contention[k] = contention[k];
    for (int e = 0; e < n_edges; e++) {
        int u = edges[2 * e], v = edges[2 * e + 1];
        if (u < 0 || u >= n || v < 0 || v >= n || u == v) return -1;
        int dup = 0;
        for (int j = 0; j < P->npred[v]; j++)
            if (P->pred[v][j] == u) dup = 1;
        if (!dup) P->pred[v][P->npred[v]++] = u;
    }
    return 0;
}

static int on_gpu(int mode) { return mode != OR_CPU; }

/* b(v, a): isolated latency of tool v in mode a (tau of Section 2.1). */
static int64_t base_latency(const or_problem *P, int v, int mode) {
    if (mode == OR_CPU) return P->cpu[v];
    if (mode == OR_GPU_NOW) return P->gpu[v];
    return P->gpu[v] + P->load[v];
}

/* Duration of a GPU task that starts while k GPU tasks run (itself included);
 * the contention table clamps at its last level. */
static int64_t gpu_duration(const or_problem *P, int v, int mode, int k) {
    int level = k < P->n_levels ? k : P->n_levels;
    unsigned __int128 prod =
        (unsigned __int128)(uint64_t)base_latency(P, v, mode) *
        (uint64_t)P->contention[level - 1];
    return (int64_t)((prod + 32768u) >> 16);
}

/* Simulate one mapping.  mode[v] in {0,1,2}.  On success returns the makespan
 * and, when the pointers are non-null, each tool's start and finish time.
 * Returns OR_INFEASIBLE when the mapping is infeasible. */
/* Steps of one fixed-at-start schedule, counted for the work model of a
 * sequential event-driven evaluation (tools whose ready time was computed,
 * their in-edges, tools started); the counting changes no result. */
typedef struct {
    int64_t edges;   /* in-edges of the tools whose ready time was computed */
    int64_t started; /* tools started before the schedule ended */
} or_counts;

static int64_t schedule_fs(const or_problem *P, const int32_t *mode, int64_t *start_out,
                           int64_t *finish_out, or_counts *cnt) {
    const int n = P->n;
    int state[OR_MAXN];
    int64_t S[OR_MAXN], C[OR_MAXN], r[OR_MAXN];
    int preds_done[OR_MAXN], starting[OR_MAXN], seen[OR_MAXN];
    int n_started = 0;
    int64_t t = 0;

    for (int v = 0; v < n; v++) {
        state[v] = WAITING;
        seen[v] = 0;
    }

    for (;;) {
        /* 1. release */
        for (int v = 0; v < n; v++)
            if (state[v] == RUNNING && C[v] <= t) state[v] = DONE;

        /* ready times of waiting tasks whose predecessors have all finished */
        for (int v = 0; v < n; v++) {
            preds_done[v] = 0;
            if (state[v] != WAITING) continue;
            int all = 1;
            int64_t rv = 0;
            for (int j = 0; j < P->npred[v]; j++) {
                int u = P->pred[v][j];
                if (state[u] != DONE) { all = 0; break; }
                int64_t arrive = C[u];
                if (on_gpu(mode[u]) != on_gpu(mode[v])) arrive += P->xfer[v];
                if (arrive > rv) rv = arrive;
            }
            preds_done[v] = all;
            r[v] = rv;
            if (all && !seen[v]) {
                seen[v] = 1;
                if (cnt) cnt->edges += P->npred[v];
            }
        }

        /* 2. immediate starts (cpu and gpu_now never wait) */
        int64_t in_use = 0;
        for (int v = 0; v < n; v++)
            if (state[v] == RUNNING && on_gpu(mode[v])) in_use += P->mem[v];
        for (int v = 0; v < n; v++) {
            starting[v] = 0;
            if (state[v] == WAITING && mode[v] != OR_GPU_QUEUE && preds_done[v] &&
                r[v] <= t) {
                starting[v] = 1;
                if (mode[v] == OR_GPU_NOW) in_use += P->mem[v];
            }
        }
        if (in_use > P->budget) return OR_INFEASIBLE;

        /* 3. serialized gpu_queue admission, FIFO on (r_v, v) */
        int queue_busy = 0;
        for (int v = 0; v < n; v++)
            if (state[v] == RUNNING && mode[v] == OR_GPU_QUEUE) queue_busy = 1;
        if (!queue_busy) {
            int head = -1;
            for (int v = 0; v < n; v++) {
                if (state[v] == WAITING && mode[v] == OR_GPU_QUEUE && preds_done[v] &&
                    r[v] <= t && (head < 0 || r[v] < r[head]))
                    head = v;
            }
            if (head >= 0 && P->mem[head] <= P->budget - in_use) {
                starting[head] = 1;
                in_use += P->mem[head];
            }
        }

        /* 4. durations, with k counting co-starting GPU tasks */
        int k = 0;
        for (int v = 0; v < n; v++)
            if (on_gpu(mode[v]) && (state[v] == RUNNING || starting[v])) k++;
        for (int v = 0; v < n; v++) {
            if (!starting[v]) continue;
            state[v] = RUNNING;
            S[v] = t;
            C[v] = t + (mode[v] == OR_CPU ? P->cpu[v] : gpu_duration(P, v, mode[v], k));
            n_started++;
            if (cnt) cnt->started++;
        }
        if (n_started == n) break;

        /* 5. next event: a finish or a ready time after t */
        int64_t next = OR_INFEASIBLE;
        for (int v = 0; v < n; v++) {
            if (state[v] == RUNNING && C[v] > t && C[v] < next) next = C[v];
            if (state[v] == WAITING && preds_done[v] && r[v] > t && r[v] < next) next = r[v];
        }
        if (next == OR_INFEASIBLE) return OR_INFEASIBLE; /* a queued task never fits */
        t = next;
    }

    int64_t makespan = 0;
    for (int v = 0; v < n; v++) {
        if (C[v] > makespan) makespan = C[v];
        if (start_out) start_out[v] = S[v];
        if (finish_out) finish_out[v] = C[v];
    }
    return makespan;
}

int64_t oracle_schedule(const or_problem *P, const int32_t *mode,
                        int64_t *start_out, int64_t *finish_out) {
    return schedule_fs(P, mode, start_out, finish_out, 0);
}

/* Work rate of a GPU task while k GPU tasks run: round(2^32 / F[k]) units of
 * 2^-16 us per us, halves up. */
static int64_t ps_rate(const or_problem *P, int k) {
    int level = k < P->n_levels ? k : P->n_levels;
    int64_t f = P->contention[level - 1];
    return (((int64_t)1 << 33) + f) / (2 * f);
}

/* The same simulation under processor sharing (see the header). */
int64_t oracle_schedule_ps(const or_problem *P, const int32_t *mode,
                           int64_t *start_out, int64_t *finish_out) {
    const int n = P->n;
    int state[OR_MAXN];
    int64_t S[OR_MAXN], C[OR_MAXN], r[OR_MAXN], R[OR_MAXN];
    int preds_done[OR_MAXN], starting[OR_MAXN];
    int n_done = 0;
    int64_t t = 0;

    for (int v = 0; v < n; v++) state[v] = WAITING;

    for (;;) {
        /* 1. release: CPU tasks at their finish, GPU tasks out of work */
        for (int v = 0; v < n; v++) {
            if (state[v] != RUNNING) continue;
            if (on_gpu(mode[v]) ? R[v] <= 0 : C[v] <= t) {
                state[v] = DONE;
                C[v] = t;
                n_done++;
            }
        }
        if (n_done == n) break;

        /* ready times of waiting tasks whose predecessors have all finished */
        for (int v = 0; v < n; v++) {
            preds_done[v] = 0;
            if (state[v] != WAITING) continue;
            int all = 1;
            int64_t rv = 0;
            for (int j = 0; j < P->npred[v]; j++) {
                int u = P->pred[v][j];
                if (state[u] != DONE) { all = 0; break; }
                int64_t arrive = C[u];
                if (on_gpu(mode[u]) != on_gpu(mode[v])) arrive += P->xfer[v];
                if (arrive > rv) rv = arrive;
            }
            preds_done[v] = all;
            r[v] = rv;
        }

        /* 2. immediate starts */
        int64_t in_use = 0;
        for (int v = 0; v < n; v++)
            if (state[v] == RUNNING && on_gpu(mode[v])) in_use += P->mem[v];
        for (int v = 0; v < n; v++) {
            starting[v] = 0;
            if (state[v] == WAITING && mode[v] != OR_GPU_QUEUE && preds_done[v] &&
                r[v] <= t) {
                starting[v] = 1;
                if (mode[v] == OR_GPU_NOW) in_use += P->mem[v];
            }
        }
        if (in_use > P->budget) return OR_INFEASIBLE;

        /* 3. serialized gpu_queue admission, FIFO on (r_v, v) */
        int queue_busy = 0;
        for (int v = 0; v < n; v++)
            if (state[v] == RUNNING && mode[v] == OR_GPU_QUEUE) queue_busy = 1;
        if (!queue_busy) {
            int head = -1;
            for (int v = 0; v < n; v++) {
                if (state[v] == WAITING && mode[v] == OR_GPU_QUEUE && preds_done[v] &&
                    r[v] <= t && (head < 0 || r[v] < r[head]))
                    head = v;
            }
            if (head >= 0 && P->mem[head] <= P->budget - in_use) {
                starting[head] = 1;
                in_use += P->mem[head];
            }
        }

        /* 4. starts: CPU finish times fixed, GPU tasks take their work */
        for (int v = 0; v < n; v++) {
            if (!starting[v]) continue;
            state[v] = RUNNING;
            S[v] = t;
            if (mode[v] == OR_CPU) C[v] = t + P->cpu[v];
            else R[v] = base_latency(P, v, mode[v]) << 16;
        }

        /* 5. next event, at the rate of the GPU tasks running from t on */
        int k = 0;
        int64_t rmin = 0;
        for (int v = 0; v < n; v++)
            if (state[v] == RUNNING && on_gpu(mode[v])) {
                if (k == 0 || R[v] < rmin) rmin = R[v];
                k++;
            }
        int64_t w = k ? ps_rate(P, k) : 0;
        int64_t next = OR_INFEASIBLE;
        if (k) next = t + (rmin + w - 1) / w;
        for (int v = 0; v < n; v++) {
            if (state[v] == RUNNING && !on_gpu(mode[v]) && C[v] > t && C[v] < next) next = C[v];
            if (state[v] == WAITING && preds_done[v] && r[v] > t && r[v] < next) next = r[v];
        }
        if (next == OR_INFEASIBLE) return OR_INFEASIBLE; /* a queued task never fits */
        for (int v = 0; v < n; v++)
            if (state[v] == RUNNING && on_gpu(mode[v])) R[v] -= (next - t) * w;
        t = next;
    }

    int64_t makespan = 0;
    for (int v = 0; v < n; v++) {
        if (C[v] > makespan) makespan = C[v];
        if (start_out) start_out[v] = S[v];
        if (finish_out) finish_out[v] = C[v];
    }
    return makespan;
}

void oracle_set_sharing(or_problem *P, int32_t sharing) { P->sharing = sharing ? 1 : 0; }

/* Simulate one mapping under the problem's contention reading. */
int64_t oracle_simulate(const or_problem *P, const int32_t *mode, int64_t *start_out,
                        int64_t *finish_out) {
    if (P->sharing) return oracle_schedule_ps(P, mode, start_out, finish_out);
    return oracle_schedule(P, mode, start_out, finish_out);
}

/* Mode of every tool for mapping index x: digit v of x in base 3. */
static void decode_index(int n, uint64_t x, int32_t *mode) {
    for (int v = 0; v < n; v++) {
        mode[v] = (int32_t)(x % 3u);
        x /= 3u;
    }
}

int64_t oracle_eval_index(const or_problem *P, uint64_t x) {
    int32_t mode[OR_MAXN];
    decode_index(P->n, x, mode);
    return oracle_simulate(P, mode, 0, 0);
}

/* Summed step counts of the fixed-at-start schedules of mappings idx[0..count):
 * out[0] in-edges of tools whose ready time was computed, out[1] tools
 * started, out[2] feasible mappings. */
void oracle_count_steps(const or_problem *P, const uint64_t *idx, int64_t count, int64_t *out) {
    out[0] = out[1] = out[2] = 0;
    for (int64_t i = 0; i < count; i++) {
        int32_t mode[OR_MAXN];
        decode_index(P->n, idx[i], mode);
        or_counts c = {0, 0};
        if (schedule_fs(P, mode, 0, 0, &c) != OR_INFEASIBLE) out[2]++;
        out[0] += c.edges;
        out[1] += c.started;
    }
}

uint64_t oracle_num_mappings(const or_problem *P) {
    uint64_t m = 1;
    for (int v = 0; v < P->n; v++) m *= 3u;
    return m;
}

/* ---- threaded search: contiguous slices, merged by (makespan, index) ---- */

typedef struct {
    const or_problem *P;
    uint64_t lo, hi;
    uint64_t best_index;
    int64_t best_makespan;
} search_slice;

static void *search_worker(void *arg) {
    search_slice *s = (search_slice *)arg;
    s->best_index = UINT64_MAX;
    s->best_makespan = OR_INFEASIBLE;
    for (uint64_t x = s->lo; x < s->hi; x++) {
        int64_t m = oracle_eval_index(s->P, x);
        if (m < s->best_makespan) { /* strict: ties keep the lower index */
            s->best_makespan = m;
            s->best_index = x;
        }
    }
    return 0;
}

#define OR_MAXTHREADS 256

/* Lowest makespan over [lo, hi), ties to the lowest index.  With no feasible
 * mapping in range: best_index = UINT64_MAX, best_makespan = INT64_MAX. */
void oracle_argmin(const or_problem *P, uint64_t lo, uint64_t hi, int32_t nthreads,
                   uint64_t *best_index, int64_t *best_makespan) {
    if (nthreads < 1) nthreads = 1;
    if (nthreads > OR_MAXTHREADS) nthreads = OR_MAXTHREADS;
    uint64_t total = hi > lo ? hi - lo : 0;
    if ((uint64_t)nthreads > total) nthreads = total ? (int32_t)total : 1;
    search_slice sl[OR_MAXTHREADS];
    pthread_t th[OR_MAXTHREADS];
    for (int i = 0; i < nthreads; i++) {
        sl[i].P = P;
        sl[i].lo = lo + total * (uint64_t)i / (uint64_t)nthreads;
        sl[i].hi = lo + total * (uint64_t)(i + 1) / (uint64_t)nthreads;
        pthread_create(&th[i], 0, search_worker, &sl[i]);
    }
    *best_index = UINT64_MAX;
    *best_makespan = OR_INFEASIBLE;
    for (int i = 0; i < nthreads; i++) {
        pthread_join(th[i], 0);
        if (sl[i].best_makespan < *best_makespan ||
            (sl[i].best_makespan == *best_makespan && sl[i].best_index < *best_index)) {
            *best_makespan = sl[i].best_makespan;
            *best_index = sl[i].best_index;
        }
    }
}

/* ---- threaded evaluation of a list of indices ---- */

typedef struct {
    const or_problem *P;
    const uint64_t *idx;
    int64_t *out;
    int64_t lo, hi;
} eval_slice;

static void *eval_worker(void *arg) {
    eval_slice *s = (eval_slice *)arg;
    for (int64_t i = s->lo; i < s->hi; i++) s->out[i] = oracle_eval_index(s->P, s->idx[i]);
    return 0;
}

void oracle_eval_many(const or_problem *P, const uint64_t *idx, int64_t count,
                      int32_t nthreads, int64_t *out) {
    if (nthreads < 1) nthreads = 1;
    if (nthreads > OR_MAXTHREADS) nthreads = OR_MAXTHREADS;
    if (count < nthreads) nthreads = count > 0 ? (int32_t)count : 1;
    eval_slice sl[OR_MAXTHREADS];
    pthread_t th[OR_MAXTHREADS];
    for (int i = 0; i < nthreads; i++) {
        sl[i].P = P;
        sl[i].idx = idx;
        sl[i].out = out;
        sl[i].lo = count * i / nthreads;
        sl[i].hi = count * (i + 1) / nthreads;
        pthread_create(&th[i], 0, eval_worker, &sl[i]);
    }
    for (int i = 0; i < nthreads; i++) pthread_join(th[i], 0);
}
