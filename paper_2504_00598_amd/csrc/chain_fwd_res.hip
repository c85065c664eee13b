// Forward pass of the unconstrained chain search for K <= 32 with the
// resharding tables held in registers (Sec. 4.4, Eq. T recurrence).
//
// Work split of one search (one workgroup of 4 waves): wave w owns the SW =
// KP/4 states s in [w*SW, (w+1)*SW); the GROUPS = 64/SW adjacent lanes of a
// state split the predecessors t into groups of TL = KP/GROUPS, so lane
// (s', g) = lane s'*GROUPS + g.  Each lane keeps, for the whole search and
// for every table e, its TL entries pre-shifted and tagged with t:
//     RP[e][j] = (R_e[t][s] << b) | t,   t = g*TL + j.
// A step is TL saturating adds and mins per lane, a DPP reduction over the
// GROUPS lanes of the state, and one barrier.  The tables are the same for
// every search, so each workgroup reads them once (from L2).
//
// Normalisation is one step behind: the row written at step i is
//     Q_i[s] = min(D[i][s] - o_i, cap) << b,   o_i = rowmin_{i-1} + min_s c[i][s],
// which each wave can form before the minimum of row i is known.  With v the
// cheapest strategy of block i, D[i][v] - o_i <= R_max, so the best
// candidate of every state at step i+1 is at most 2 R_max; the packed minimum
// is exact while 2 R_max < cap = 2^(32-b) - 1, i.e. for R < 2^(31-b).  A
// state whose relative value saturates is beaten through v by every
// continuation, so it never lies on an optimal plan.  In int64,
// opt = sum_i min_s c[i][s] + sum_i (rowmin_i - o_i).  The row minimum is
// gathered with an LDS atomic min into one of three rotating words.
//
// The step loop is unrolled by U = 12 steps.  Costs arrive through LDS in
// blocks of U rows, loaded one block ahead and rewritten as
// cadj[i][s] = c[i][s] - min_s c[i][s] (2^31 for an unavailable strategy,
// which always saturates); argmin bytes are collected in LDS per block and
// written to the table with one coalesced store per thread.  When the edge
// map is periodic, redge[i] = i mod E with E dividing U (the repeated-layer
// case), the table of every unrolled step is a compile-time register set;
// otherwise a per-step switch selects it.
#include "res_common.h"

namespace cfp {

template <int KP>
struct ResGeo {
  static constexpr int SW = KP / 4;        // states per wave
  static constexpr int GROUPS = 64 / SW;   // lanes per state
  static constexpr int TL = KP / GROUPS;   // predecessors per lane
  static constexpr int BITS = Pow2Bits<KP>::value;
  static constexpr uint32_t CAP = (1u << (32 - BITS)) - 1u;
  static constexpr int QPAD = TL >= 4 ? 4 : 0;
  static constexpr int QSTRIDE = TL + QPAD;  // LDS words per predecessor group
};

template <int TL>
__device__ __forceinline__ uint32_t minplus_lane(const uint32_t (&q)[TL], const uint32_t (&r)[TL]) {
  uint32_t acc = sat_add(q[0], r[0]);
#pragma unroll
  for (int j = 1; j < TL; ++j) acc = umin(acc, sat_add(q[j], r[j]));
  return acc;
}

// EP = period of the edge map (divides kUnroll), or 0 for an arbitrary map.
template <int KP, int EP>
__global__ __launch_bounds__(kThreads, 1) void chain_fwd_res_kernel(
    const int32_t *__restrict__ cost, const int32_t *__restrict__ rtab, const int32_t *__restrict__ redge, int N,
    int K, int E, uint8_t *__restrict__ table, SearchResult *__restrict__ res, const WsHeader *__restrict__ hdr,
    int64_t *__restrict__ opt, int32_t *__restrict__ status) {
  using G = ResGeo<KP>;
  constexpr int SW = G::SW, GROUPS = G::GROUPS, TL = G::TL, BITS = G::BITS;
  constexpr int QSTRIDE = G::QSTRIDE;
  constexpr int U = kUnroll;
  constexpr uint32_t CAP = G::CAP;
  static_assert(EP == 0 || U % EP == 0, "period must divide the unroll");

  __shared__ __align__(16) uint32_t Qs[2][GROUPS * QSTRIDE];
  __shared__ __align__(16) uint32_t cadj[2][U][KP];
  __shared__ __align__(16) uint8_t argb[2][U][KP];
  __shared__ uint32_t dmin[3];  // row minima of Q, rotating
  __shared__ int flags;         // bit 0: negative cost seen; bit 1: a block with no available strategy

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int sl = lane / GROUPS, g = lane % GROUPS;
  const int s = wid * SW + sl;
  const int t0 = g * TL;
  const int b = blockIdx.x;
  const int qslot = (s / TL) * QSTRIDE + s % TL;  // where state s is written in Qs
  const bool owner = (g == 0);                     // one lane per state writes it
  CostStager<KP> cs(cost + (size_t)b * N * K, table + (size_t)b * N * K, N, K, tid);

  if (tid == 0) {
    flags = 0;
    dmin[0] = dmin[1] = dmin[2] = kSat;
  }

  // Resident tables.
  uint32_t rp[kResTables][TL];
#pragma unroll
  for (int e = 0; e < kResTables; ++e)
#pragma unroll
    for (int j = 0; j < TL; ++j) {
      const int t = t0 + j;
      // unconditional, in-bounds loads (entry 0 for padding) stay in flight together
      const bool ok = e < E && t < K && s < K;
      const uint32_t r = (uint32_t)rtab[ok ? ((size_t)e * K + t) * K + s : 0];
      rp[e][j] = ok ? ((r << BITS) | (uint32_t)t) : kSat;
    }

  // Table index of every step of a block, per wave: lane r holds redge[blk*U + r].
  auto load_edges = [&](int blk) __attribute__((always_inline)) {
    const int i = blk * U + lane;
    return (EP == 0 && lane < U && i < N) ? redge[i] : 0;
  };
  int32_t ecur = load_edges(0), enext = N > U ? load_edges(1) : 0;

  const int nblk = (N + U - 1) / U;
  cs.load(0);
  __syncthreads();  // flags / dmin initialised
  cs.store(0, cadj[0], &flags);
  if (nblk > 1) cs.load(1);
  __syncthreads();

  // Row 0: Q_0[s] = min(c[0][s] - cmin_0, cap) << b.
  uint64_t dsum = 0;
  {
    const uint32_t qn = umin(cadj[0][0][s], CAP) << BITS;
    if (owner) {
      Qs[0][qslot] = qn;
      atomicMin(&dmin[0], qn);
    }
  }
  __syncthreads();

  // One step i = blk*U + J (J static).  guard: skip steps outside [1, N).
  auto step = [&](auto Jc, int blk, bool guard) __attribute__((always_inline)) {
    constexpr int J = decltype(Jc)::value;
    const int i = blk * U + J;
    if (guard && (i < 1 || i >= N)) return;
    constexpr int cur = (J + 1) & 1, nxt = J & 1;  // U is even: parity of i-1 and i
    uint32_t q[TL];
    if (TL >= 4) {
#pragma unroll
      for (int j = 0; j < TL; j += 4) {
        const uint4 v = *(const uint4 *)&Qs[cur][g * QSTRIDE + j];
        q[j] = v.x; q[j + 1] = v.y; q[j + 2] = v.z; q[j + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int j = 0; j < TL; ++j) q[j] = Qs[cur][g * QSTRIDE + j];
    }
    const uint32_t dv = dmin[(J + 2) % 3];  // minimum of row i-1 (U is a multiple of 3)
    const uint32_t ca = cadj[blk & 1][J][s];
    asm volatile("" ::"v"(ca));  // issue the cost read with the row reads, not after the reduction
    uint32_t acc;
    if constexpr (EP != 0) {
      acc = minplus_lane<TL>(q, rp[J % (EP ? EP : 1)]);
    } else {
      const int e = __builtin_amdgcn_readlane(ecur, J);
      switch (e) {
#define CFP_CASE(E_) \
  case E_: acc = minplus_lane<TL>(q, rp[E_]); break;
        CFP_CASE(0) CFP_CASE(1) CFP_CASE(2) CFP_CASE(3) CFP_CASE(4) CFP_CASE(5)
        CFP_CASE(6) CFP_CASE(7) CFP_CASE(8) CFP_CASE(9) CFP_CASE(10)
        default: acc = minplus_lane<TL>(q, rp[11]); break;
#undef CFP_CASE
      }
    }
    acc = group_min<GROUPS>(acc);
    const uint32_t d = __builtin_amdgcn_readfirstlane(dv) >> BITS;
    dsum += d;
    const uint32_t qn = umin((acc >> BITS) - d + ca, CAP) << BITS;
    if (owner) {
      Qs[nxt][qslot] = qn;
      argb[blk & 1][J][s] = (uint8_t)acc;
      atomicMin(&dmin[J % 3], qn);
    }
    if (tid == 0) dmin[(J + 1) % 3] = kSat;  // read at step i-1, next written at step i+1
    if (J == 0) cs.flush(blk - 1, argb[(blk - 1) & 1]);
    if (J == U - 1 && blk + 1 < nblk) {
      cs.store(blk + 1, cadj[(blk + 1) & 1], &flags);
      if (EP == 0) ecur = enext;
      if (blk + 2 < nblk) {
        cs.load(blk + 2);
        if (EP == 0) enext = load_edges(blk + 2);
      }
    }
    __syncthreads();
  };
  auto group = [&](int blk, bool guard) __attribute__((always_inline)) {
    step(std::integral_constant<int, 0>{}, blk, guard);
    step(std::integral_constant<int, 1>{}, blk, guard);
    step(std::integral_constant<int, 2>{}, blk, guard);
    step(std::integral_constant<int, 3>{}, blk, guard);
    step(std::integral_constant<int, 4>{}, blk, guard);
    step(std::integral_constant<int, 5>{}, blk, guard);
    step(std::integral_constant<int, 6>{}, blk, guard);
    step(std::integral_constant<int, 7>{}, blk, guard);
    step(std::integral_constant<int, 8>{}, blk, guard);
    step(std::integral_constant<int, 9>{}, blk, guard);
    step(std::integral_constant<int, 10>{}, blk, guard);
    step(std::integral_constant<int, 11>{}, blk, guard);
  };

  // Block 0 starts with row 0 (done above); the last block may be partial.
  group(0, true);
  int blk = 1;
  for (; (blk + 1) * U <= N; ++blk) group(blk, false);
  if (blk < nblk) group(blk, true);

  // The block of the last row has not been flushed yet.
  cs.flush((N - 1) / U, argb[((N - 1) / U) & 1]);

  const int last = (N - 1) & 1;
  const uint32_t pk = (owner && s < K) ? (Qs[last][qslot] | (uint32_t)s) : kSat;
  finish_search(pk, cs.csum, dsum, BITS, CAP, flags, hdr, b, opt, status, res);
}

bool chain_fwd_res_supported(int k, int e) { return k <= 64 && e <= kResTables; }

// Period of the edge map if redge[i] == i mod E for all i >= 1 with E
// dividing the unroll, else 0.
static int edge_period(const int32_t *redge, int n, int e) {
  if (kUnroll % e != 0) return 0;
  for (int i = 1; i < n; ++i)
    if (redge[i] != i % e) return 0;
  return e;
}

template <int KP>
static void launch_res(const cfp_chain_desc &d, int period, const int32_t *redge_dev, uint8_t *table,
                       SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st) {
#define CFP_LAUNCH(EP)                                                                                      \
  timed_launch(chain_fwd_res_kernel<KP, EP>, dim3(d.batch), dim3(kThreads), 0, st, d.cost, d.rtab, \
                     redge_dev, d.n_blocks, d.k, d.n_tables, table, res, hdr, opt, status)
  switch (period) {
    case 1: CFP_LAUNCH(1); break;
    case 2: CFP_LAUNCH(2); break;
    case 3: CFP_LAUNCH(3); break;
    case 4: CFP_LAUNCH(4); break;
    case 6: CFP_LAUNCH(6); break;
    case 12: CFP_LAUNCH(12); break;
    default: CFP_LAUNCH(0); break;
  }
#undef CFP_LAUNCH
}

void launch_chain_fwd_k64(const cfp_chain_desc &d, int period, const int32_t *redge_dev, uint8_t *table,
                          SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st);

hipError_t launch_chain_fwd_res(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *table, SearchResult *res,
                                const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st) {
  const int period = edge_period(d.redge, d.n_blocks, d.n_tables);
  if (d.k <= 16) launch_res<16>(d, period, redge_dev, table, res, hdr, opt, status, st);
  else if (d.k <= 32) launch_res<32>(d, period, redge_dev, table, res, hdr, opt, status, st);
  else launch_chain_fwd_k64(d, period, redge_dev, table, res, hdr, opt, status, st);
  return hipGetLastError();
}

}  // namespace cfp
