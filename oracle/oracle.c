/*
 * CPU oracle for the chain dynamic program of CFP's plan search.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is compiled into liboracle.so, which
 * only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * load.  The product library never links, loads or calls it, and it shares no
 * code, header or table with the GPU path.
 *
 * What it computes (paper Sec. 4.4, "Plan Cost Estimation and Optimization"):
 * a plan x = (x_0 .. x_{N-1}) picks one strategy per block.  Its cost is
 * Eq. T with the per-block time p_n + c_n folded into one table c:
 *
 *     T(x) = sum_i c[i][x_i] + sum_{i=1}^{N-1} R_{e(i)}[x_{i-1}][x_i]
 *
 * and its memory is Eq. M, M(x) = sum_i mem[i][x_i].  The search returns the
 * plan of least T, optionally among those with M(x) <= budget (Sec. 4.4: the
 * plan of minimal cost under the memory limit, found by a dynamic program
 * that starts at the first segment, with quantised memory).
 *
 * Because T is a sum of unary terms and terms on adjacent pairs only, the
 * forward recurrence
 *
 *     D[0][s] = c[0][s]
 *     D[i][s] = c[i][s] + min_t (D[i-1][t] + R_{e(i)}[t][s])
 *
 * reaches exactly min_x T(x) = min_s D[N-1][s].  All arithmetic is int64.
 *
 * Readings where the paper is silent (each stated again where it is used):
 *  - c[i][s] == 0x7FFFFFFF means "strategy s is unavailable at block i";
 *    such states are unreachable (cost +infinity).
 *  - Ties: the lowest index wins at every choice (final state and every
 *    traceback step), which yields, among all optimal plans, the one that is
 *    smallest in reversed lexicographic order (x_{N-1}, ..., x_0).
 *  - Memory: the budget is inclusive; D[i][s][m] is the least cost of a
 *    prefix ending in state s whose memory total is at most m.
 *
 * Status codes: 0 ok, 1 infeasible (no plan, or no plan within the budget).
 */
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_COST_INF 0x7FFFFFFF
#define ORC_INF INT64_MAX

enum { ORC_OK = 0, ORC_INFEASIBLE = 1 };

static int64_t cost_value(int32_t c) { return c == ORC_COST_INF ? ORC_INF : (int64_t)c; }

static int64_t add_inf(int64_t a, int64_t b) {
  if (a == ORC_INF || b == ORC_INF) return ORC_INF;
  return a + b;
}

/* ---------------------------------------------------------------- chain -- */

/* One search: c is [N][K], D is caller scratch of N*K entries. */
static void chain_one(int N, int K, const int32_t *c, const int32_t *rtab, const int32_t *redge,
                      int64_t *D, int64_t *opt, int32_t *plan, int32_t *status) {
  for (int s = 0; s < K; ++s) D[s] = cost_value(c[s]);

  for (int i = 1; i < N; ++i) {
    const int32_t *R = rtab + (size_t)redge[i] * K * K; /* R[t][s]: t earlier, s later */
    const int64_t *prev = D + (size_t)(i - 1) * K;
    int64_t *cur = D + (size_t)i * K;
    for (int s = 0; s < K; ++s) {
      int64_t best = ORC_INF;
      for (int t = 0; t < K; ++t) {
        int64_t v = add_inf(prev[t], (int64_t)R[(size_t)t * K + s]);
        if (v < best) best = v;
      }
      cur[s] = add_inf(best, cost_value(c[(size_t)i * K + s]));
    }
  }

  const int64_t *last = D + (size_t)(N - 1) * K;
  int64_t best = ORC_INF;
  int arg = -1;
  for (int s = 0; s < K; ++s)
    if (last[s] < best) { best = last[s]; arg = s; }

  if (best == ORC_INF) {
    *opt = ORC_INF;
    *status = ORC_INFEASIBLE;
    for (int i = 0; i < N; ++i) plan[i] = -1;
    return;
  }
  *opt = best;
  *status = ORC_OK;

  /* Traceback: the earliest predecessor that attains the recorded value. */
  int s = arg;
  plan[N - 1] = s;
  for (int i = N - 1; i >= 1; --i) {
    const int32_t *R = rtab + (size_t)redge[i] * K * K;
    const int64_t *prev = D + (size_t)(i - 1) * K;
    int64_t target = D[(size_t)i * K + s] - (int64_t)c[(size_t)i * K + s];
    int pick = -1;
    for (int t = 0; t < K; ++t) {
      if (add_inf(prev[t], (int64_t)R[(size_t)t * K + s]) == target) { pick = t; break; }
    }
    plan[i - 1] = pick;
    s = pick;
  }
}

/* ------------------------------------------------------ memory variant -- */

/* One search under a memory budget.  D is [N][K][W] with W = budget + 1. */
static void chain_mem_one(int N, int K, const int32_t *c, const int32_t *rtab, const int32_t *redge,
                          const uint8_t *mem, int budget, int64_t *D, int64_t *opt, int32_t *plan,
                          int32_t *status) {
  const int W = budget + 1;
#define DIDX(i, s, m) (((size_t)(i) * K + (s)) * W + (m))
  for (int s = 0; s < K; ++s)
    for (int m = 0; m < W; ++m)
      D[DIDX(0, s, m)] = (mem[s] <= m) ? cost_value(c[s]) : ORC_INF;

  for (int i = 1; i < N; ++i) {
    const int32_t *R = rtab + (size_t)redge[i] * K * K;
    for (int s = 0; s < K; ++s) {
      int ms = mem[(size_t)i * K + s];
      int64_t cs = cost_value(c[(size_t)i * K + s]);
      for (int m = 0; m < W; ++m) {
        if (m < ms) { D[DIDX(i, s, m)] = ORC_INF; continue; }
        int64_t best = ORC_INF;
        for (int t = 0; t < K; ++t) {
          int64_t v = add_inf(D[DIDX(i - 1, t, m - ms)], (int64_t)R[(size_t)t * K + s]);
          if (v < best) best = v;
        }
        D[DIDX(i, s, m)] = add_inf(best, cs);
      }
    }
  }

  int64_t best = ORC_INF;
  int arg = -1;
  for (int s = 0; s < K; ++s)
    if (D[DIDX(N - 1, s, budget)] < best) { best = D[DIDX(N - 1, s, budget)]; arg = s; }
  if (best == ORC_INF) {
    *opt = ORC_INF;
    *status = ORC_INFEASIBLE;
    for (int i = 0; i < N; ++i) plan[i] = -1;
    return;
  }
  *opt = best;
  *status = ORC_OK;

  int s = arg, m = budget;
  plan[N - 1] = s;
  for (int i = N - 1; i >= 1; --i) {
    const int32_t *R = rtab + (size_t)redge[i] * K * K;
    int mp = m - mem[(size_t)i * K + s];
    int64_t target = D[DIDX(i, s, m)] - (int64_t)c[(size_t)i * K + s];
    int pick = -1;
    for (int t = 0; t < K; ++t) {
      if (add_inf(D[DIDX(i - 1, t, mp)], (int64_t)R[(size_t)t * K + s]) == target) { pick = t; break; }
    }
    plan[i - 1] = pick;
    s = pick;
    m = mp;
  }
#undef DIDX
}

/* Budget frontier of one search: F[m] = least cost of a plan whose memory
 * total is at most m, for every m in [0, M) (Sec. 4.4 with Eq. M as the
 * constraint, every budget at once).  With D[i][s][m] meaning "total memory
 * at most m", F[m] = min_s D[N-1][s][m].  D is [N][K][M]. */
static void mem_frontier_one(int N, int K, const int32_t *c, const int32_t *rtab, const int32_t *redge,
                             const uint8_t *mem, int M, int64_t *D, int64_t *F) {
  int64_t opt;
  int32_t status;
  int32_t *plan = (int32_t *)malloc(sizeof(int32_t) * (size_t)N);
  if (!plan) {
    for (int m = 0; m < M; ++m) F[m] = -1;
    return;
  }
  chain_mem_one(N, K, c, rtab, redge, mem, M - 1, D, &opt, plan, &status);
  free(plan);
  for (int m = 0; m < M; ++m) {
    int64_t best = ORC_INF;
    for (int s = 0; s < K; ++s) {
      const int64_t v = D[((size_t)(N - 1) * K + s) * M + m];
      if (v < best) best = v;
    }
    F[m] = best;
  }
}

/* ------------------------------------------------------------ threading -- */

typedef struct {
  int N, K, B, variant, M;
  const int32_t *cost, *rtab, *redge, *budget;
  const uint8_t *mem;
  int64_t *opt, *frontier;
  int32_t *plan, *status;
  int next; /* next search to take, guarded by lock */
  int failed;
  pthread_mutex_t lock;
} job_t;

static void *worker(void *arg) {
  job_t *j = (job_t *)arg;
  int64_t *D = NULL;
  size_t cap = 0;
  for (;;) {
    pthread_mutex_lock(&j->lock);
    int b = j->next++;
    pthread_mutex_unlock(&j->lock);
    if (b >= j->B) break;
    size_t need = (size_t)j->N * j->K;
    if (j->variant == 1) need *= (size_t)j->budget[b] + 1;
    if (j->variant == 2) need *= (size_t)j->M;
    if (need > cap) {
      free(D);
      D = (int64_t *)malloc(need * sizeof(int64_t));
      cap = need;
      if (!D) { j->failed = 1; break; }
    }
    const int32_t *c = j->cost + (size_t)b * j->N * j->K;
    int32_t *plan = j->plan + (size_t)b * j->N;
    if (j->variant == 0)
      chain_one(j->N, j->K, c, j->rtab, j->redge, D, &j->opt[b], plan, &j->status[b]);
    else if (j->variant == 2)
      mem_frontier_one(j->N, j->K, c, j->rtab, j->redge, j->mem + (size_t)b * j->N * j->K, j->M, D,
                       j->frontier + (size_t)b * j->M);
    else
      chain_mem_one(j->N, j->K, c, j->rtab, j->redge, j->mem + (size_t)b * j->N * j->K, j->budget[b], D,
                    &j->opt[b], plan, &j->status[b]);
  }
  free(D);
  return NULL;
}

static int run(job_t *j, int nthreads) {
  if (nthreads < 1) nthreads = 1;
  if (nthreads > j->B) nthreads = j->B;
  pthread_mutex_init(&j->lock, NULL);
  j->next = 0;
  j->failed = 0;
  pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)nthreads);
  if (!th) return -1;
  for (int k = 0; k < nthreads; ++k) pthread_create(&th[k], NULL, worker, j);
  for (int k = 0; k < nthreads; ++k) pthread_join(th[k], NULL);
  free(th);
  pthread_mutex_destroy(&j->lock);
  return j->failed ? -1 : 0;
}

/* ------------------------------------------------------------- exported -- */

/* Unconstrained search for B independent chains.  cost [B][N][K],
 * rtab [E][K][K], redge [N] (redge[0] unused), outputs opt [B], plan [B][N],
 * status [B].  Returns 0, or -1 on bad arguments / allocation failure. */
int oracle_chain(int N, int K, int B, int E, const int32_t *cost, const int32_t *rtab,
                 const int32_t *redge, int64_t *opt, int32_t *plan, int32_t *status, int nthreads) {
  if (N < 1 || K < 1 || B < 1 || E < 1) return -1;
  for (int i = 1; i < N; ++i)
    if (redge[i] < 0 || redge[i] >= E) return -1;
  job_t j;
  memset(&j, 0, sizeof j);
  j.N = N; j.K = K; j.B = B; j.variant = 0;
  j.cost = cost; j.rtab = rtab; j.redge = redge;
  j.opt = opt; j.plan = plan; j.status = status;
  return run(&j, nthreads);
}

/* Memory-budgeted search.  mem [B][N][K] (buckets), budget [B] (inclusive). */
int oracle_chain_mem(int N, int K, int B, int E, const int32_t *cost, const int32_t *rtab,
                     const int32_t *redge, const uint8_t *mem, const int32_t *budget, int64_t *opt,
                     int32_t *plan, int32_t *status, int nthreads) {
  if (N < 1 || K < 1 || B < 1 || E < 1) return -1;
  for (int i = 1; i < N; ++i)
    if (redge[i] < 0 || redge[i] >= E) return -1;
  for (int b = 0; b < B; ++b)
    if (budget[b] < 0) return -1;
  job_t j;
  memset(&j, 0, sizeof j);
  j.N = N; j.K = K; j.B = B; j.variant = 1;
  j.cost = cost; j.rtab = rtab; j.redge = redge; j.mem = mem; j.budget = budget;
  j.opt = opt; j.plan = plan; j.status = status;
  return run(&j, nthreads);
}

/* Budget frontier of B searches: frontier [B][M] int64, entry m = least cost
 * with memory total <= m (INT64_MAX where no plan fits). */
int oracle_mem_frontier(int N, int K, int B, int E, const int32_t *cost, const int32_t *rtab,
                        const int32_t *redge, const uint8_t *mem, int M, int64_t *frontier, int nthreads) {
  if (N < 1 || K < 1 || B < 1 || E < 1 || M < 1) return -1;
  for (int i = 1; i < N; ++i)
    if (redge[i] < 0 || redge[i] >= E) return -1;
  job_t j;
  memset(&j, 0, sizeof j);
  j.N = N; j.K = K; j.B = B; j.variant = 2; j.M = M;
  j.cost = cost; j.rtab = rtab; j.redge = redge; j.mem = mem;
  j.frontier = frontier;
  return run(&j, nthreads);
}

/* All forward values D[i][s] of one chain (int64, INT64_MAX = unreachable). */
int oracle_chain_values(int N, int K, int E, const int32_t *cost, const int32_t *rtab,
                        const int32_t *redge, int64_t *D) {
  if (N < 1 || K < 1 || E < 1) return -1;
  for (int i = 1; i < N; ++i)
    if (redge[i] < 0 || redge[i] >= E) return -1;
  int64_t opt;
  int32_t status;
  int32_t *plan = (int32_t *)malloc(sizeof(int32_t) * (size_t)N);
  if (!plan) return -1;
  chain_one(N, K, cost, rtab, redge, D, &opt, plan, &status);
  free(plan);
  return 0;
}

/* Eq. T of one plan of one chain (INT64_MAX if it uses an unavailable
 * strategy), and Eq. M of the same plan if mem is not NULL. */
int64_t oracle_plan_cost(int N, int K, const int32_t *cost, const int32_t *rtab, const int32_t *redge,
                         const int32_t *plan) {
  int64_t t = 0;
  for (int i = 0; i < N; ++i) t = add_inf(t, cost_value(cost[(size_t)i * K + plan[i]]));
  for (int i = 1; i < N; ++i) {
    const int32_t *R = rtab + (size_t)redge[i] * K * K;
    t = add_inf(t, (int64_t)R[(size_t)plan[i - 1] * K + plan[i]]);
  }
  return t;
}

int64_t oracle_plan_mem(int N, int K, const uint8_t *mem, const int32_t *plan) {
  int64_t m = 0;
  for (int i = 0; i < N; ++i) m += mem[(size_t)i * K + plan[i]];
  return m;
}
