/*
 * cfp.h -- C ABI of the min-plus chain search library (libcfp.so, gfx950).
 *
 * The library computes the plan search of CFP (arXiv 2504.00598, Sec. 4.4,
 * "Plan Cost Estimation and Optimization"): a model is a chain of N blocks
 * (ParallelBlocks or segments); block i picks one of K strategies; a plan
 * x = (x_0 .. x_{N-1}) costs, by Eq. T,
 *
 *     T(x) = sum_i c[i][x_i] + sum_{i=1}^{N-1} R_{e(i)}[x_{i-1}][x_i]
 *
 * where c[i][s] is the profiled time of block i under strategy s (the
 * paper's p_n + c_n, computation plus communication) and R_e[t][s] is the
 * profiled resharding time from strategy t of a block to strategy s of the
 * next one (the paper's r_n).  Resharding tables are shared by all edges
 * with the same e(i) = redge[i], as profiles of matched segments are reused
 * (Sec. 4.1).  Optionally each block/strategy has a quantised peak memory
 * mem[i][s] and the plan must satisfy Eq. M, sum_i mem[i][x_i] <= budget
 * (Sec. 4.4: least cost under the memory limit, memory quantised).
 *
 * Every call answers B independent searches that share rtab/redge but have
 * their own cost (and mem, budget) tables.  Results are exact: the optimum
 * is the int64 minimum of Eq. T, and the plan is, among all optimal plans,
 * the one chosen by taking the lowest index at every tie (equivalently the
 * least optimal plan in reversed lexicographic order (x_{N-1}, ..., x_0)).
 *
 * Conventions for every call:
 *  - Arrays are C-contiguous, row-major.  "device" pointers are HIP device
 *    memory of the current device; "host" pointers are ordinary host memory.
 *  - The caller owns all memory.  The library allocates no device memory,
 *    frees nothing of the caller's and keeps no pointer after a call
 *    returns.  Its only allocations are host-side: per device, on the first
 *    call that uploads a workspace header, a ring of 32 pinned host slots of
 *    64 KiB and one event per slot (held until the process ends), so that
 *    the header copy is asynchronous; and the benchmarking timer's events.
 *  - Work is enqueued on `stream` (a hipStream_t passed as void*; NULL is
 *    the default stream) and ordered like any other stream work; inputs must
 *    stay valid until that work has run.
 *  - Argument errors (descriptor fields, NULL pointers, host redge out of
 *    range, workspace too small, unsupported K) are returned synchronously,
 *    as a negative CFP_ERR_* code, before any HIP call is made.
 *  - Outcomes found on the device are written per search to status[b]:
 *    CFP_ST_BADINPUT when a device array holds a value outside its
 *    documented range, CFP_ST_INFEASIBLE when no plan exists (a block with
 *    every strategy unavailable, or no plan within the memory budget).  When
 *    status[b] != CFP_ST_OK, opt[b] = INT64_MAX and the traced plan is all -1.
 *  - No global mutable state apart from the opt-in benchmarking timer and
 *    the static workspace of cfp_search_chain_noalloc (both declared
 *    below): calls on different streams with different workspaces may
 *    run concurrently.  Three paths wait on the device for other workgroups of
 *    the same launch and need them resident at the same time: the memory
 *    variant (cfp_dp_chain_mem, cfp_mem_frontier), the split chain kernel
 *    that cfp_dp_chain uses for K > 64 when the chunk-parallel kernels do not
 *    apply, and the chunk-parallel chain search for 256 < K <= 512 with at
 *    most 8 searches (four workgroups per chunk exchange every row).  Their
 *    waits are bounded; if another long kernel keeps their
 *    workgroups from being dispatched (a shared GPU, concurrent calls), a
 *    wait may expire and the search ends with CFP_ST_TIMEOUT, never with a
 *    wrong answer.
 */
#ifndef CFP_H
#define CFP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* A cost entry equal to CFP_COST_INF marks a strategy that is unavailable at
 * that block (used to pad blocks with fewer than K strategies). */
#define CFP_COST_INF 0x7FFFFFFF

/* Synchronous return codes. */
enum {
  CFP_OK = 0,
  CFP_ERR_ARG = -1,         /* NULL pointer or a descriptor field out of range */
  CFP_ERR_RANGE = -2,       /* host array (redge) holds an out-of-range value */
  CFP_ERR_WORKSPACE = -3,   /* ws is NULL or ws_bytes < cfp_workspace_bytes() */
  CFP_ERR_UNSUPPORTED = -4, /* K or n_mem beyond what the library supports */
  CFP_ERR_HIP = -5          /* a HIP runtime call or kernel launch failed */
};

/* Per-search status written on the device. */
enum {
  CFP_ST_OK = 0,
  CFP_ST_INFEASIBLE = 1, /* no plan (all strategies unavailable at a block, or budget too small) */
  CFP_ST_OVERFLOW = 2,   /* reserved: device arithmetic left its exact range (not reachable with valid inputs) */
  CFP_ST_TIMEOUT = 3,    /* a bounded device wait expired (memory variant, K > 64 split chain kernel,
                            or 256 < K <= 512 chunk-parallel teams, while other work held the GPU;
                            see above) */
  CFP_ST_BADINPUT = 4    /* a device array value is outside its documented range */
};

/* Forward variants (the argument `variant` of cfp_workspace_bytes / cfp_traceback). */
enum { CFP_V_CHAIN = 0, CFP_V_MEM = 1, CFP_V_SCAN = 2, CFP_V_SEG = 3 };

/* Largest supported number of strategies per block. */
#define CFP_MAX_K 512

typedef struct {
  int32_t n_blocks;     /* N >= 1 */
  int32_t k;            /* strategies per block, 1 <= K <= CFP_MAX_K */
  int32_t batch;        /* independent searches B >= 1 */
  int32_t n_tables;     /* distinct resharding tables E >= 1 */
  const int32_t *cost;  /* device [B][N][K]; each entry in [0, CFP_COST_INF] (CFP_COST_INF = unavailable) */
  const int32_t *rtab;  /* device [E][K][K]; rtab[e][t][s]: strategy t of block i-1 -> strategy s of block i;
                           each entry in [0, cfp_r_limit(variant, K)) */
  const int32_t *redge; /* HOST [N]; redge[i] in [0, E) names the table of edge (i-1 -> i); redge[0] is ignored */
} cfp_chain_desc;

/* Exclusive upper bound on resharding-table entries for which `variant` with
 * K strategies is exact.  The kernels carry (cost, argmin) packed in one
 * 32-bit word with ceil(log2 K) index bits (at least 4), so the bound depends
 * on K: 2^(30-b) for K <= 64, 2^(32-b) - 1 for K > 64 (chain and scan) and
 * 2^(32-b) - 1 for the boundary tables of the segment search, with
 * b = max(4, ceil(log2 K)); 2^(31-b) with b = max(5, ceil(log2 K)) for the
 * memory variant (K <= 256).  Returns 0 for an unsupported K or variant. */
int32_t cfp_r_limit(int32_t variant, int32_t k);

/* Bytes of device workspace a forward call of `variant` needs (n_mem is the
 * memory axis size M for CFP_V_MEM, ignored otherwise).  Returns 0 for an
 * invalid descriptor. */
size_t cfp_workspace_bytes(const cfp_chain_desc *d, int32_t variant, int32_t n_mem);

/* Unconstrained search by the forward chain recurrence
 *     D[0][s] = c[0][s],   D[i][s] = c[i][s] + min_t (D[i-1][t] + R_{e(i)}[t][s])
 * (Sec. 4.4; the dynamic program that starts at the first block).
 *   ws     device workspace of at least cfp_workspace_bytes(d, CFP_V_CHAIN, 0)
 *          bytes; on return (in stream order) it holds the argmin tables that
 *          cfp_traceback reads.
 *   opt    device [B] int64: min_x T(x), or INT64_MAX when status != OK.
 *   status device [B] int32: CFP_ST_*.  */
int cfp_dp_chain(const cfp_chain_desc *d, void *ws, size_t ws_bytes, int64_t *opt, int32_t *status,
                 void *stream);

/* Search under a memory budget (Sec. 4.4 with Eq. M as the constraint):
 *     D[i][s][m] = c[i][s] + min_t D[i-1][t][m - mem[i][s]] + R_{e(i)}[t][s]
 * with D[0][s][m] = c[0][s] if mem[0][s] <= m; the answer is
 * min_s D[N-1][s][budget[b]] (total memory <= budget, inclusive).
 *   mem    device [B][N][K] uint8, each entry in [0, n_mem) and at most 16
 *          (the memory of one block is a small number of buckets; a larger
 *          entry gives status CFP_ST_BADINPUT)
 *   n_mem  M, the number of memory buckets, 1 <= M <= 4096
 *   budget device [B] int32, each in [0, M)
 * Supported for 1 <= K <= 256 and any n_tables >= 1 (CFP_ERR_UNSUPPORTED for
 * K > 256).  Every cost and resharding entry in its documented range gives
 * the exact optimum (CFP_ST_OVERFLOW is not reachable).  The buckets of a
 * search are cut into chunks of 64 that run as a pipeline of workgroups;
 * searches are launched in rounds small enough that every chunk of a round
 * is resident at once.  A chunk that waits too long for the chunk below it
 * (which cannot happen when the GPU is not shared) ends its search with
 * CFP_ST_TIMEOUT.  ws must hold cfp_workspace_bytes(d, CFP_V_MEM, n_mem)
 * bytes. */
int cfp_dp_chain_mem(const cfp_chain_desc *d, const uint8_t *mem, int32_t n_mem, const int32_t *budget,
                     void *ws, size_t ws_bytes, int64_t *opt, int32_t *status, void *stream);

/* Budget frontier: the least cost at every memory budget, from one pass
 * (Sec. 4.4 with Eq. M as the constraint).  D[i][s][m] is the least cost of a
 * prefix ending in s with memory total at most m, so one pass at the largest
 * budget M-1 holds every budget's answer in its last row:
 *     frontier[b][m] = min_s D[N-1][s][m],   m = 0 .. M-1
 * (INT64_MAX where no plan fits within m).  The frontier does not increase
 * with m; its last entry equals cfp_dp_chain_mem at budget M-1, and
 * cfp_traceback(d, CFP_V_MEM, n_mem, ...) on the same workspace returns the
 * plans at budget M-1.
 *   mem, n_mem  as for cfp_dp_chain_mem (K <= 256, any n_tables)
 *   frontier    device [B][n_mem] int64
 *   status      device [B] int32: CFP_ST_OK, CFP_ST_INFEASIBLE when no plan
 *               fits even M-1 buckets (frontier all INT64_MAX), or an error
 *               status, in which case the frontier of that search is not
 *               meaningful.
 * ws must hold cfp_workspace_bytes(d, CFP_V_MEM, n_mem) bytes. */
int cfp_mem_frontier(const cfp_chain_desc *d, const uint8_t *mem, int32_t n_mem, void *ws, size_t ws_bytes,
                     int64_t *frontier, int32_t *status, void *stream);

/* The same optimum as cfp_dp_chain computed as a min-plus parallel scan:
 * block i becomes the transfer matrix T_i[t][s] = R_{e(i)}[t][s] + c[i][s]
 * (T_0[t][s] = c[0][s]), the matrices are composed by a tree of min-plus
 * matrix products (min-plus matrix product is associative), and a down-sweep
 * recovers every prefix vector D[i].  For long chains.  Products are kept in
 * 32-bit words relative to their minimum, so besides the R bound of
 * cfp_r_limit the available costs of every block must lie within 2^30 of
 * each other (max_s c[i][s] - min_s c[i][s] < 2^30 over available s);
 * otherwise the search ends with CFP_ST_BADINPUT.  ws must hold
 * cfp_workspace_bytes(d, CFP_V_SCAN, 0) bytes (about B * N * K * K * 4). */
int cfp_minplus_scan(const cfp_chain_desc *d, void *ws, size_t ws_bytes, int64_t *opt, int32_t *status,
                     void *stream);

/* Recover the plan x (Sec. 4.4: the plan tuple i = (i_1 .. i_N)) of every
 * search from a workspace filled by the forward call of `variant` with the
 * same descriptor (and n_mem for CFP_V_MEM): plan[b][N-1] is the lowest
 * optimal final strategy and plan[b][i-1] the lowest predecessor attaining
 * D[i][plan[b][i]].  The traceback reads the forward tables in ws and uses a
 * small scratch region of ws (chunk maps), so it writes to ws as well.
 *   plan   device [B][N] int32; all -1 for a search whose status is not OK. */
int cfp_traceback(const cfp_chain_desc *d, int32_t variant, int32_t n_mem, void *ws, size_t ws_bytes,
                  int32_t *plan, void *stream);

/* Segment-level search (Sec. 4.2-4.4).  The units are model segments; the
 * plan t of a segment combines the strategies of its blocks (K = prod of the
 * block strategy counts, e.g. 3^4 = 81 for four blocks of three strategies,
 * Sec. 5.5).  Resharding between consecutive segments is profiled only for
 * the boundary block pair (Sec. 4.2), so Eq. T's resharding term is
 *     R_{e(i)}[t][s] = rbound[e(i)][last[t]][first[s]]
 * with last[t] the strategy of the last block of plan t and first[s] that of
 * the first block of plan s.  The result is exactly cfp_dp_chain's on that
 * expanded table (same optimum, same lowest-index plan), found with O(K + L F)
 * work per segment instead of O(K^2). */
typedef struct {
  int32_t n_segments;    /* N >= 1 */
  int32_t k;             /* plans per segment, 1 <= K <= CFP_MAX_K */
  int32_t batch;         /* independent searches B >= 1 */
  int32_t n_tables;      /* distinct boundary tables E >= 1 */
  int32_t n_last;        /* L: strategies of a segment's last block, 1..8 */
  int32_t n_first;       /* F: strategies of a segment's first block, 1..8 */
  const int32_t *cost;   /* device [B][N][K]; each entry in [0, CFP_COST_INF] */
  const int32_t *rbound; /* device [E][L][F]; each entry in [0, cfp_r_limit(CFP_V_SEG, K)) */
  const uint8_t *last;   /* device [K]; each entry < L (else status CFP_ST_BADINPUT) */
  const uint8_t *first;  /* device [K]; each entry < F (else status CFP_ST_BADINPUT) */
  const int32_t *redge;  /* HOST [N]; redge[i] in [0, E): table of the boundary (i-1 -> i) */
} cfp_segment_desc;

/* Workspace bytes of a segment search (0 for an invalid descriptor). */
size_t cfp_segment_workspace_bytes(const cfp_segment_desc *d);

/* Forward segment search; opt/status as for cfp_dp_chain.  CFP_ERR_UNSUPPORTED
 * when K > CFP_MAX_K, L or F exceeds 8, or 8 N K exceeds 2^31 - 1 (device row
 * offsets are 32-bit).  Batches too small to occupy the device run each chain
 * as chunks made exact by rank convergence; the workspace then also holds the
 * speculative rows (B N K 4 bytes, counted by cfp_segment_workspace_bytes). */
int cfp_dp_segments(const cfp_segment_desc *d, void *ws, size_t ws_bytes, int64_t *opt, int32_t *status,
                    void *stream);

/* Plans [B][N] of a workspace filled by cfp_dp_segments with the same
 * descriptor (lowest optimal final plan, lowest predecessor at every step). */
int cfp_traceback_segments(const cfp_segment_desc *d, void *ws, size_t ws_bytes, int32_t *plan, void *stream);

/* Whole search in one call: cfp_dp_chain followed by cfp_traceback (Sec. 4.4:
 * the Eq. T recurrence, then the lowest-index optimal plan), with the same
 * results, statuses and plans.
 *   ws, ws_bytes  as for cfp_dp_chain.  Small searches (K <= 64, N <= 512,
 *                 B <= 256, n_tables <= 255 and
 *                 E*KP*(KP+4)*4 + N*(5*KP+1) <= 61440 with KP = K rounded
 *                 up to 16, 32 or 64) do not use it (it may then be NULL):
 *                 they run as one kernel launch that also checks the range
 *                 of R, with the edge map passed in the launch's arguments
 *                 (no host-to-device copy).  Larger searches run the two
 *                 calls and return CFP_ERR_WORKSPACE for a missing or short
 *                 workspace.
 *   opt, status   device [B], as cfp_dp_chain writes them.
 *   plan          device [B][N] int32, as cfp_traceback writes it.
 * opt, status and plan may also be pinned host memory mapped into the
 * device's address space (hipHostMalloc) on the one-launch path, which then
 * needs no copy back. */
int cfp_search_chain(const cfp_chain_desc *d, void *ws, size_t ws_bytes, int64_t *opt, int32_t *status,
                     int32_t *plan, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * search as cfp_dp_chain followed by cfp_traceback, with the workspace taken
 * from a static device array of CFP_NOALLOC_MAX_BYTES bytes that the library
 * holds on every GPU it runs on until the process ends.  The call allocates
 * nothing: the header and the edge map reach the device as kernel arguments
 * and the upload ring of the other calls is not used.
 *   d       as for cfp_dp_chain (redge on the host)
 *   opt     device [B] int64, status device [B] int32, plan device [B][N] int32:
 *           as cfp_dp_chain and cfp_traceback write them.
 * Returns CFP_ERR_WORKSPACE when the search needs more than
 * CFP_NOALLOC_MAX_BYTES of workspace (cfp_workspace_bytes(d, CFP_V_CHAIN, 0)),
 * CFP_ERR_HIP if the array's device address cannot be obtained, otherwise as
 * cfp_dp_chain.  Every call on one GPU uses that GPU's one array: calls that
 * overlap on a GPU (different streams or threads with work in flight at the
 * same time) race and must be serialised by the caller; calls in one stream
 * are ordered and safe. */
#define CFP_NOALLOC_MAX_BYTES (32u << 20)
int cfp_search_chain_noalloc(const cfp_chain_desc *d, int64_t *opt, int32_t *status, int32_t *plan, void *stream);

/* Benchmarking aid (not needed for searching).  cfp_timer_start creates
 * max_launches pairs of HIP events (1 <= max_launches <= 2^20) and arms
 * recording: from then on every launch of a forward call's main kernel (the
 * chain step kernel of cfp_dp_chain, the step kernel of cfp_dp_chain_mem,
 * each min-plus matrix-product launch of cfp_minplus_scan) carries one pair
 * as the start and stop events of its dispatch (on the call's stream), until
 * the pairs run out.
 * cfp_timer_stop waits for the recorded events, writes the summed device
 * time in milliseconds and the number of bracketed launches, disarms
 * recording and destroys the events.  The timer is process-wide state behind
 * a lock, meant for one benchmarking thread; besides the header-upload ring
 * it is the only global state of the library.  Returns CFP_OK, CFP_ERR_ARG (bad count, start while armed,
 * stop while not armed) or CFP_ERR_HIP. */
int cfp_timer_start(int32_t max_launches);
int cfp_timer_stop(double *total_ms, int32_t *launches);

/* Static string for a CFP_ERR_* or CFP_ST_* code (status codes are >= 0). */
const char *cfp_status_string(int code);

#ifdef __cplusplus
}
#endif

#endif /* CFP_H */
