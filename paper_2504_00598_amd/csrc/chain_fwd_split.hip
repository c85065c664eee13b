// Forward pass of the unconstrained chain search (Sec. 4.4, Eq. T recurrence)
// for few, long chains with 64 < K <= 512: each search is split over P
// workgroups (CUs) so that the resharding tables stay in registers.
//
// Workgroup p of a search owns the SPW = 4096 / KP states
// s = p*SPW .. p*SPW + SPW-1 (P = KP / SPW: 64 for K <= 512, 16 for K <= 256,
// 4 for K <= 128).  Thread (s_local, g) keeps, for every table e (at most 12),
// the 16 predecessors t = 16g .. 16g+15 of its state pre-shifted and tagged:
//     RP[e][j] = (R_e[t][s] << b) | t
// (12 x 16 = 192 registers), so a step is 16 saturating adds and 8 three-input
// minima per thread against the full previous row Q, read from LDS.
//
// Every step the workgroups of a search exchange their new values: each
// publishes its SPW values as 64-bit words (step << 32) | value with
// device-scope stores into one of two slots, and gathers the whole row by
// device-scope loads that wait (boundedly) for the step's tag.  A slot is
// rewritten two steps later, which cannot happen before every workgroup has
// gathered it: a workgroup publishes step i+1 only after it has gathered all
// of step i, which every workgroup publishes only after gathering step i-1.
// Every workgroup thus holds the same full row and normalises it exactly:
//     Q_i[t] = min(D[i][t] - min_t D[i][t], cap) << b,   cap = 2^(32-b) - 1,
// so the best candidate of every state is at most R_max (through the row's
// argmin), exact for R below cfp_r_limit; a state at the cap is beaten through
// that argmin by every continuation.  All workgroups of a launch must be
// resident at once (the launcher only uses this kernel when B * P fits the
// device); a wait that expires ends the search with CFP_ST_TIMEOUT.
#include "cfp_internal.h"
#include "common.h"

namespace cfp {

constexpr int kSplitThreads = 256;
constexpr int kSplitTables = 12;
constexpr int kSplitSpin = 1 << 20;  // polls of one word before the search gives up

template <int KP>
struct SplitShape {
  static constexpr int SPW = 4096 / KP;              // states per workgroup
  static constexpr int P = KP / SPW;                 // workgroups per search
  static constexpr int GROUPS = kSplitThreads / SPW;  // predecessor groups of 16
  static_assert(GROUPS * 16 == KP, "16 predecessors per thread");
};

__global__ void split_init_kernel(uint64_t *xb, size_t nxb, int32_t *sflags, int B) {
  for (size_t x = (size_t)blockIdx.x * blockDim.x + threadIdx.x; x < nxb + B; x += (size_t)gridDim.x * blockDim.x) {
    if (x < nxb) xb[x] = ~0ull;  // tag 0xFFFFFFFF: no step
    else sflags[x - nxb] = 0;
  }
}

template <int KP>
__global__ __launch_bounds__(kSplitThreads, 1) void chain_fwd_split_kernel(
    const int32_t *__restrict__ cost, const int32_t *__restrict__ rtab, const int32_t *__restrict__ redge, int N,
    int K, int E, uint8_t *__restrict__ table, uint64_t *xb, int32_t *sflags, SearchResult *__restrict__ res,
    const WsHeader *__restrict__ hdr, int64_t *__restrict__ opt, int32_t *__restrict__ status) {
  using S = SplitShape<KP>;
  constexpr int SPW = S::SPW, P = S::P, BITS = Pow2Bits<KP>::value;
  constexpr uint32_t CAP = (1u << (32 - BITS)) - 1u;
  constexpr int NW = kSplitThreads / 64;

  __shared__ __align__(16) uint32_t Qs[KP];
  __shared__ uint32_t part[NW][SPW];
  __shared__ uint32_t wmin[NW];
  __shared__ int flags;  // bit 0: negative cost, bit 1: a wait expired

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int b = blockIdx.x / P, p = blockIdx.x % P;
  const int sl = tid % SPW, g = tid / SPW;
  const int s = p * SPW + sl;  // the state this thread works for
  const int32_t *cb = cost + (size_t)b * N * K;
  uint64_t *xbs = xb + (size_t)b * 2 * KP;
  const bool ELEM2 = KP > 256;

  if (tid == 0) flags = 0;

  // Tables of this thread: 16 predecessors of state s for every table.
  uint32_t rp[kSplitTables][16];
#pragma unroll
  for (int e = 0; e < kSplitTables; ++e)
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int t = 16 * g + j;
      // unconditional, in-bounds loads (entry 0 for padding) stay in flight together
      const bool ok = e < E && t < K && s < K;
      const uint32_t r = (uint32_t)rtab[ok ? ((size_t)e * K + t) * K + s : 0];
      rp[e][j] = ok ? ((r << BITS) | (uint32_t)t) : kSat;
    }

  // Block-wide minimum of one value per thread (one barrier).
  auto block_min = [&](uint32_t v) __attribute__((always_inline)) {
    v = wave_min(v);
    if (lane == 0) wmin[wid] = v;
    __syncthreads();
    return umin(umin(wmin[0], wmin[1]), umin(wmin[2], wmin[3]));
  };

  // Row 0, read whole by every workgroup.
  constexpr int GPT = (KP + kSplitThreads - 1) / kSplitThreads;  // row entries per thread
  uint32_t yv[GPT];
  __syncthreads();
  uint32_t lm = kSat;
#pragma unroll
  for (int k = 0; k < GPT; ++k) {
    const int x = tid + kSplitThreads * k;
    const int32_t c = x < K ? cb[x] : CFP_COST_INF;
    if (c < 0) atomicOr(&flags, 1);
    yv[k] = c == CFP_COST_INF ? kSat : (uint32_t)c;
    lm = umin(lm, yv[k]);
  }
  uint32_t rmin = block_min(lm);
  int64_t o = rmin;
  bool infeasible = rmin == kSat;
#pragma unroll
  for (int k = 0; k < GPT; ++k)
    if (tid + kSplitThreads * k < KP) Qs[tid + kSplitThreads * k] = umin(yv[k] - rmin, CAP) << BITS;
  __syncthreads();

  const bool comb = tid < SPW;
  int32_t cnext = (comb && s < K && N > 1) ? cb[(size_t)K + s] : CFP_COST_INF;
  bool aborted = false;

  for (int i = 1; i < N && !aborted; ++i) {
    // 1. partial minimum over this thread's 16 predecessors
    const int e = __builtin_amdgcn_readfirstlane(redge[i]);
    const uint4 *qp = (const uint4 *)&Qs[16 * g];
    const uint4 q0 = qp[0], q1 = qp[1], q2 = qp[2], q3 = qp[3];
    const uint32_t q[16] = {q0.x, q0.y, q0.z, q0.w, q1.x, q1.y, q1.z, q1.w,
                            q2.x, q2.y, q2.z, q2.w, q3.x, q3.y, q3.z, q3.w};
    auto row = [&](const uint32_t(&r)[16]) __attribute__((always_inline)) {
      uint32_t a = sat_add(q[0], r[0]);
#pragma unroll
      for (int j = 1; j < 16; j += 2) a = umin(umin(a, sat_add(q[j], r[j])), j + 1 < 16 ? sat_add(q[j + 1], r[j + 1]) : kSat);
      return a;
    };
    uint32_t acc;
    switch (e) {
#define CFP_CASE(E_) \
  case E_: acc = row(rp[E_]); break;
      CFP_CASE(0) CFP_CASE(1) CFP_CASE(2) CFP_CASE(3) CFP_CASE(4) CFP_CASE(5)
      CFP_CASE(6) CFP_CASE(7) CFP_CASE(8) CFP_CASE(9) CFP_CASE(10)
      default: acc = row(rp[11]); break;
#undef CFP_CASE
    }
    // lanes of one state inside the wave: s_local + SPW * k
#pragma unroll
    for (int off = SPW; off < 64; off <<= 1) acc = umin(acc, (uint32_t)__shfl_xor((int)acc, off, 64));
    if (lane < SPW) part[wid][lane] = acc;
    __syncthreads();

    // 2. the workgroup's states: value, argmin, publication
    const int slot = i & 1;
    if (comb) {
      const uint32_t m = umin(umin(part[0][sl], part[1][sl]), umin(part[2][sl], part[3][sl]));
      uint32_t y = kSat;
      if (s < K) {
        const size_t cell = ((size_t)b * N + i) * K + s;
        if (ELEM2) ((uint16_t *)table)[cell] = (uint16_t)(m & (KP - 1));
        else table[cell] = (uint8_t)(m & (KP - 1));
        if (cnext < 0) atomicOr(&flags, 1);
        if (cnext != CFP_COST_INF && m != kSat) y = (m >> BITS) + (uint32_t)cnext;
        cnext = i + 1 < N ? cb[(size_t)(i + 1) * K + s] : CFP_COST_INF;
      }
      __hip_atomic_store(&xbs[(size_t)slot * KP + s], ((uint64_t)(uint32_t)i << 32) | y, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }

    // 3. gather the whole row of step i
    lm = kSat;
#pragma unroll
    for (int k = 0; k < GPT; ++k) {
      const int x = tid + kSplitThreads * k;
      yv[k] = kSat;
      if (x >= KP) continue;
      uint64_t w = 0;
      int spins = 0;
      while (true) {
        w = __hip_atomic_load(&xbs[(size_t)slot * KP + x], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if ((uint32_t)(w >> 32) == (uint32_t)i) break;
        ++spins;
        // another workgroup of the search gave up (checked every 256 polls), or this wait expired
        if (spins > kSplitSpin ||
            ((spins & 255) == 0 && __hip_atomic_load(&sflags[b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0)) {
          atomicOr(&flags, 2);
          __hip_atomic_store(&sflags[b], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          w = kSat;
          break;
        }
        __builtin_amdgcn_s_sleep(1);  // spaces the polls of the many waiting threads
      }
      yv[k] = (uint32_t)w;
      lm = umin(lm, yv[k]);
    }
    rmin = block_min(lm);
    o += rmin;
    infeasible |= rmin == kSat;
#pragma unroll
    for (int k = 0; k < GPT; ++k)
      if (tid + kSplitThreads * k < KP) Qs[tid + kSplitThreads * k] = umin(yv[k] - rmin, CAP) << BITS;
    aborted = (flags & 2) != 0;  // uniform: read after the barrier inside block_min
    __syncthreads();
  }

  // Lowest final state of least value; workgroup 0 of the search reports it.
  uint32_t pk = kSat;
#pragma unroll
  for (int k = 0; k < GPT; ++k) {
    const int x = tid + kSplitThreads * k;
    if (x < K) pk = umin(pk, Qs[x] | (uint32_t)x);
  }
  const uint32_t fin = block_min(pk);
  if (p == 0 && tid == 0) {
    int st = CFP_ST_OK;
    if (flags & 2) st = CFP_ST_TIMEOUT;
    else if ((flags & 1) || hdr->rflag) st = CFP_ST_BADINPUT;
    else if (infeasible) st = CFP_ST_INFEASIBLE;
    else if ((fin >> BITS) != 0) st = CFP_ST_OVERFLOW;
    status[b] = st;
    opt[b] = st == CFP_ST_OK ? o : INT64_MAX;
    res[b].final_state = st == CFP_ST_OK ? (int32_t)(fin & (KP - 1)) : -1;
    res[b].status = st;
    res[b].final_m = 0;
  }
}

// Streaming variant, for batches too large to keep the tables in registers
// (e.g. 64 searches with K = 256): P = KP / 64 workgroups per search, each
// owning 64 states, streaming its 64-column slice of the edge's table from
// L2 every step (packed (R << b) | t in the workspace).  The slices are loaded
// two steps ahead into two register buffers that alternate: loads complete in
// issue order, so a slice loaded one step ahead would hold up the exchange
// loads of the step in between.
constexpr int kSplitWThreads = 512;

template <int KP>
struct SplitWShape {
  static constexpr int SPW = 64;                   // states per workgroup
  static constexpr int P = KP / SPW;               // workgroups per search
  static constexpr int SQ = SPW / 4;               // threads per table row (4 states each)
  static constexpr int TG = kSplitWThreads / SQ;   // row groups
  static constexpr int TPG = KP / TG;              // rows per group
};

template <int KP>
__global__ __launch_bounds__(kSplitWThreads, 1) void chain_fwd_splitw_kernel(
    const int32_t *__restrict__ cost, const uint32_t *__restrict__ rpk, const int32_t *__restrict__ redge, int N,
    int K, uint8_t *__restrict__ table, uint64_t *xb, int32_t *sflags, SearchResult *__restrict__ res,
    const WsHeader *__restrict__ hdr, int64_t *__restrict__ opt, int32_t *__restrict__ status) {
  using S = SplitWShape<KP>;
  constexpr int SPW = S::SPW, P = S::P, SQ = S::SQ, TPG = S::TPG, BITS = Pow2Bits<KP>::value;
  constexpr uint32_t CAP = (1u << (32 - BITS)) - 1u;
  constexpr int NW = kSplitWThreads / 64;
  static_assert(TPG % 4 == 0, "rows per group");

  __shared__ __align__(16) uint32_t Qs[KP];
  __shared__ __align__(16) uint32_t part[NW][SPW];
  __shared__ uint32_t wmin[NW];
  __shared__ int flags;  // bit 0: negative cost, bit 1: a wait expired

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int b = blockIdx.x / P, p = blockIdx.x % P;
  const int sq = tid % SQ, g = tid / SQ;
  const int32_t *cb = cost + (size_t)b * N * K;
  uint64_t *xbs = xb + (size_t)b * 2 * KP;
  const bool comb = tid < SPW;
  const int s = p * SPW + tid;  // combiner state
  const bool ELEM2 = KP > 256;

  auto block_min = [&](uint32_t v) __attribute__((always_inline)) {
    v = wave_min(v);
    if (lane == 0) wmin[wid] = v;
    __syncthreads();
    uint32_t m = wmin[0];
#pragma unroll
    for (int w = 1; w < NW; ++w) m = umin(m, wmin[w]);
    return m;
  };
  const uint32_t lane_off = (uint32_t)(g * TPG * KP + p * SPW + 4 * sq);  // words within a table
  auto load_r = [&](int i, uint4(&R)[TPG]) __attribute__((always_inline)) {
    const int e = __builtin_amdgcn_readfirstlane(redge[i < N ? i : N - 1]);
    const uint32_t *tab = rpk + (size_t)e * KP * KP;
#pragma unroll
    for (int r = 0; r < TPG; ++r) R[r] = *(const uint4 *)(tab + lane_off + r * KP);
  };

  if (tid == 0) flags = 0;
  __syncthreads();
  // Row 0, read whole by every workgroup.
  uint32_t yv = kSat;
  if (tid < K) {
    const int32_t c = cb[tid];
    if (c < 0) atomicOr(&flags, 1);
    yv = c == CFP_COST_INF ? kSat : (uint32_t)c;
  }
  uint32_t rmin = block_min(yv);
  int64_t o = rmin;
  bool infeasible = rmin == kSat;
  if (tid < KP) Qs[tid] = umin(yv - rmin, CAP) << BITS;
  int32_t cnext = (comb && s < K && N > 1) ? cb[(size_t)K + s] : CFP_COST_INF;
  uint4 RA[TPG], RB[TPG];
  load_r(1, RA);
  load_r(2, RB);
  __syncthreads();
  bool aborted = false;

  auto step = [&](int i, uint4(&R)[TPG]) __attribute__((always_inline)) {
    // 1. partials of this thread's 4 states over its TPG rows
    uint32_t a0 = kSat, a1 = kSat, a2 = kSat, a3 = kSat;
#pragma unroll
    for (int r4 = 0; r4 < TPG; r4 += 4) {
      const uint4 qq = *(const uint4 *)&Qs[g * TPG + r4];
      const uint32_t q[4] = {qq.x, qq.y, qq.z, qq.w};
#pragma unroll
      for (int r = 0; r < 4; r += 2) {
        const uint4 x = R[r4 + r], y = R[r4 + r + 1];
        a0 = umin(umin(a0, sat_add(q[r], x.x)), sat_add(q[r + 1], y.x));
        a1 = umin(umin(a1, sat_add(q[r], x.y)), sat_add(q[r + 1], y.y));
        a2 = umin(umin(a2, sat_add(q[r], x.z)), sat_add(q[r + 1], y.z));
        a3 = umin(umin(a3, sat_add(q[r], x.w)), sat_add(q[r + 1], y.w));
      }
    }
    // the groups of one wave (lanes sq + SQ k)
#pragma unroll
    for (int off = SQ; off < 64; off <<= 1) {
      a0 = umin(a0, (uint32_t)__shfl_xor((int)a0, off, 64));
      a1 = umin(a1, (uint32_t)__shfl_xor((int)a1, off, 64));
      a2 = umin(a2, (uint32_t)__shfl_xor((int)a2, off, 64));
      a3 = umin(a3, (uint32_t)__shfl_xor((int)a3, off, 64));
    }
    if (lane < SQ) *(uint4 *)&part[wid][4 * lane] = make_uint4(a0, a1, a2, a3);
    __syncthreads();

    // 2. this workgroup's states: value, argmin, publication
    const int slot = i & 1;
    if (comb) {
      uint32_t m = part[0][tid];
#pragma unroll
      for (int w = 1; w < NW; ++w) m = umin(m, part[w][tid]);
      uint32_t y = kSat;
      if (s < K) {
        const size_t cell = ((size_t)b * N + i) * K + s;
        if (ELEM2) ((uint16_t *)table)[cell] = (uint16_t)(m & (KP - 1));
        else table[cell] = (uint8_t)(m & (KP - 1));
        if (cnext < 0) atomicOr(&flags, 1);
        if (cnext != CFP_COST_INF && m != kSat) y = (m >> BITS) + (uint32_t)cnext;
        cnext = i + 1 < N ? cb[(size_t)(i + 1) * K + s] : CFP_COST_INF;
      }
      __hip_atomic_store(&xbs[(size_t)slot * KP + s], ((uint64_t)(uint32_t)i << 32) | y, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }

    // 3. gather the row of step i
    uint32_t yg = kSat;
    if (tid < KP) {
      int spins = 0;
      while (true) {
        const uint64_t w = __hip_atomic_load(&xbs[(size_t)slot * KP + tid], __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT);
        if ((uint32_t)(w >> 32) == (uint32_t)i) {
          yg = (uint32_t)w;
          break;
        }
        ++spins;
        if (spins > kSplitSpin ||
            ((spins & 255) == 0 && __hip_atomic_load(&sflags[b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0)) {
          atomicOr(&flags, 2);
          __hip_atomic_store(&sflags[b], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          break;
        }
        __builtin_amdgcn_s_sleep(1);  // spaces the polls of the many waiting threads
      }
    }
    rmin = block_min(yg);
    o += rmin;
    infeasible |= rmin == kSat;
    if (tid < KP) Qs[tid] = umin(yg - rmin, CAP) << BITS;
    aborted = (flags & 2) != 0;  // uniform: read after the barrier inside block_min
    // 4. the slice of step i+2 into the buffer this step has consumed
    load_r(i + 2, R);
    __syncthreads();
  };

  int i = 1;
  for (; i + 1 < N && !aborted; i += 2) {
    step(i, RA);
    if (aborted) break;
    step(i + 1, RB);
  }
  if (i < N && !aborted) step(i, RA);

  // Lowest final state of least value; workgroup 0 of the search reports it.
  const uint32_t pk = tid < K ? (Qs[tid] | (uint32_t)tid) : kSat;
  const uint32_t fin = block_min(pk);
  if (p == 0 && tid == 0) {
    int st = CFP_ST_OK;
    if (flags & 2) st = CFP_ST_TIMEOUT;
    else if ((flags & 1) || hdr->rflag) st = CFP_ST_BADINPUT;
    else if (infeasible) st = CFP_ST_INFEASIBLE;
    else if ((fin >> BITS) != 0) st = CFP_ST_OVERFLOW;
    status[b] = st;
    opt[b] = st == CFP_ST_OK ? o : INT64_MAX;
    res[b].final_state = st == CFP_ST_OK ? (int32_t)(fin & (KP - 1)) : -1;
    res[b].status = st;
    res[b].final_m = 0;
  }
}

static int split_kp(int k) { return k <= 128 ? 128 : k <= 256 ? 256 : 512; }

// The workgroups of every search of one launch must be resident together:
// at most one per compute unit, with the tables held in registers.
static int device_cus() {
  static int cus = -1;
  if (cus < 0) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      n = 0;
    cus = n;
  }
  return cus;
}

// Which split form fits: 1 = tables in registers, 2 = streamed slices, 0 = none.
static int split_form(int k, int n_tables, int batch) {
  if (k <= 64 || k > 512) return 0;
  const int kp = split_kp(k), cus = device_cus();
  if (n_tables <= kSplitTables && (long long)batch * (kp / (4096 / kp)) <= cus) return 1;
  if ((long long)batch * (kp / 64) <= cus) return 2;
  return 0;
}

// The workgroups of every search of one launch must be resident together:
// at most one per compute unit.
bool chain_fwd_split_supported(int k, int n_tables, int batch) { return split_form(k, n_tables, batch) != 0; }

size_t split_region_bytes(int k, int batch) {
  const size_t kp = split_kp(k);
  return align_up((size_t)batch * 2 * kp * 8) + align_up((size_t)batch * 4);
}

template <int KP>
static void launch_split_kp(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *region, uint32_t *rpk,
                            uint8_t *table, SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status,
                            hipStream_t st) {
  uint64_t *xb = (uint64_t *)region;
  const size_t nxb = (size_t)d.batch * 2 * KP;
  int32_t *sflags = (int32_t *)(region + align_up(nxb * 8));
  hipLaunchKernelGGL(split_init_kernel, dim3(64), dim3(256), 0, st, xb, nxb, sflags, d.batch);
  if (split_form(d.k, d.n_tables, d.batch) == 1) {
    timer_begin(st);
    timed_launch(chain_fwd_split_kernel<KP>, dim3(d.batch * SplitShape<KP>::P), dim3(kSplitThreads), 0, st,
                       d.cost, d.rtab, redge_dev, d.n_blocks, d.k, d.n_tables, table, xb, sflags, res, hdr, opt,
                       status);
    timer_end(st);
  } else {
    launch_pack_rtab(d.rtab, d.n_tables, d.k, KP, Pow2Bits<KP>::value, rpk, st);
    timer_begin(st);
    timed_launch(chain_fwd_splitw_kernel<KP>, dim3(d.batch * SplitWShape<KP>::P), dim3(kSplitWThreads), 0,
                       st, d.cost, rpk, redge_dev, d.n_blocks, d.k, table, xb, sflags, res, hdr, opt, status);
    timer_end(st);
  }
}

hipError_t launch_chain_fwd_split(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *region, uint32_t *rpk,
                                  uint8_t *table, SearchResult *res, const WsHeader *hdr, int64_t *opt,
                                  int32_t *status, hipStream_t st) {
  switch (split_kp(d.k)) {
    case 128: launch_split_kp<128>(d, redge_dev, region, rpk, table, res, hdr, opt, status, st); break;
    case 256: launch_split_kp<256>(d, redge_dev, region, rpk, table, res, hdr, opt, status, st); break;
    default: launch_split_kp<512>(d, redge_dev, region, rpk, table, res, hdr, opt, status, st); break;
  }
  return hipGetLastError();
}

}  // namespace cfp
