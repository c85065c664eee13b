// Forward pass of the unconstrained chain search for 32 < K <= 64, resharding
// tables in registers (Sec. 4.4, Eq. T recurrence).
//
// One search per workgroup of 4 waves.  Wave w owns the predecessors
// t in [16w, 16w+16) of all 64 states: lane s keeps
//     RP[e][j] = (R_e[16w+j][s] << 6) | (16w+j)
// for every table e, and holds in a register one word of the current row,
// Q[16w + (s mod 16)], so every DPP row of 16 lanes carries the wave's 16
// predecessor values.  A step is
//   1. partial_w[s] = min_j (Q[16w+j] + RP[e][j]): 16 adds whose first operand
//      is broadcast from lane j of the row (DPP row_newbcast) and 8 mins;
//   2. one barrier to exchange the 4 partials of each state through LDS;
//   3. every lane combines the partials of the state it holds next and forms
//      the new word of that state itself, so the row never has to be
//      redistributed.
// Normalisation is one step behind (see the K <= 32 kernel):
//     Q_i[s] = min(D[i][s] - o_i, qcap) << 6,  o_i = rowmin_{i-1} + min_s c[i][s].
// The adds are not saturating (DPP has no clamp form), so the value field is
// capped at qcap = 2^25 - 1 and R < 2^24: Q + RP < 2^32 never wraps, the best
// candidate (at most 2 R_max) is exact, and any state at the cap exceeds
// 2 R_max and is beaten through the cheapest state of its block.
#include "res_common.h"

namespace cfp {

template <int EP>
__global__ __launch_bounds__(kThreads, 1) void chain_fwd_k64_kernel(
    const int32_t *__restrict__ cost, const int32_t *__restrict__ rtab, const int32_t *__restrict__ redge, int N,
    int K, int E, uint8_t *__restrict__ table, SearchResult *__restrict__ res, const WsHeader *__restrict__ hdr,
    int64_t *__restrict__ opt, int32_t *__restrict__ status) {
  constexpr int KP = 64, BITS = 6, U = kUnroll;
  constexpr uint32_t QCAP = (1u << (31 - BITS)) - 1u;
  constexpr uint32_t RP_NONE = 0x80000000u;  // "no such pair": above every exact candidate, never wraps
  static_assert(EP == 0 || U % EP == 0, "period must divide the unroll");

  __shared__ __align__(16) uint32_t part[2][KP][4];
  __shared__ __align__(16) uint32_t wmin[2][4];
  __shared__ __align__(16) uint32_t cadj[2][U][KP];
  __shared__ __align__(16) uint8_t argb[2][U][KP];
  __shared__ int flags;

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int myst = 16 * wid + (lane & 15);  // the state whose word this lane holds
  const int b = blockIdx.x;
  // Cost blocks alternate between two stagers (block b in csb[b & 1]) so that a
  // block is loaded two blocks (24 steps) before it is used: loaded one block
  // ahead, its wait showed in the step time.
  CostStager<KP> csb[2] = {CostStager<KP>(cost + (size_t)b * N * K, table + (size_t)b * N * K, N, K, tid),
                           CostStager<KP>(cost + (size_t)b * N * K, table + (size_t)b * N * K, N, K, tid)};

  if (tid == 0) flags = 0;

  uint32_t rp[kResTables][16];
#pragma unroll
  for (int e = 0; e < kResTables; ++e)
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int t = 16 * wid + j;
      // every load is unconditional and in bounds (entry 0 for padding), so the
      // 192 loads are in flight together instead of one after another
      const bool ok = e < E && t < K && lane < K;
      const uint32_t r = (uint32_t)rtab[ok ? ((size_t)e * K + t) * K + lane : 0];
      rp[e][j] = ok ? ((r << BITS) | (uint32_t)t) : RP_NONE;
    }

  auto load_edges = [&](int blk) __attribute__((always_inline)) {
    const int i = blk * U + lane;
    return (EP == 0 && lane < U && i < N) ? redge[i] : 0;
  };
  int32_t ecur = load_edges(0), enext = N > U ? load_edges(1) : 0;

  const int nblk = (N + U - 1) / U;
  csb[0].load(0);
  __syncthreads();  // flags initialised
  csb[0].store(0, cadj[0], &flags);
  if (nblk > 1) csb[1].load(1);
  if (nblk > 2) csb[0].load(2);
  __syncthreads();

  // Row 0.
  uint32_t qv = umin(cadj[0][0][myst], QCAP) << BITS;
  {
    const uint32_t wm = group_min<16>(qv);
    if (lane == 0) wmin[0][wid] = wm;
  }
  uint64_t dsum = 0;

  auto step = [&](auto Jc, auto Pc, int blk, bool guard) __attribute__((always_inline)) {
    constexpr int J = decltype(Jc)::value;
    constexpr int PB = decltype(Pc)::value;  // parity of blk
    const int i = blk * U + J;
    if (guard && (i < 1 || i >= N)) return;
    constexpr int cur = (J + 1) & 1, nxt = J & 1;  // parities of i-1 and i (U is even)

    // 1. partial over this wave's predecessors.
    uint32_t acc;
    auto row = [&](const uint32_t(&r)[16]) __attribute__((always_inline)) {
      uint32_t a = (uint32_t)__builtin_amdgcn_mov_dpp((int)qv, kRowBcast0 + 0, 0xF, 0xF, true) + r[0];
#define CFP_T(j) a = umin(a, (uint32_t)__builtin_amdgcn_mov_dpp((int)qv, kRowBcast0 + j, 0xF, 0xF, true) + r[j])
      CFP_T(1); CFP_T(2); CFP_T(3); CFP_T(4); CFP_T(5); CFP_T(6); CFP_T(7); CFP_T(8);
      CFP_T(9); CFP_T(10); CFP_T(11); CFP_T(12); CFP_T(13); CFP_T(14); CFP_T(15);
#undef CFP_T
      return a;
    };
    if constexpr (EP != 0) {
      acc = row(rp[J % (EP ? EP : 1)]);
    } else {
      const int e = __builtin_amdgcn_readlane(ecur, J);
      switch (e) {
#define CFP_CASE(E_) \
  case E_: acc = row(rp[E_]); break;
        CFP_CASE(0) CFP_CASE(1) CFP_CASE(2) CFP_CASE(3) CFP_CASE(4) CFP_CASE(5)
        CFP_CASE(6) CFP_CASE(7) CFP_CASE(8) CFP_CASE(9) CFP_CASE(10)
        default: acc = row(rp[11]); break;
#undef CFP_CASE
      }
    }
    part[nxt][lane][wid] = acc;
    __syncthreads();

    // 2. the state this lane holds: combine, normalise, keep.
    const uint4 p4 = *(const uint4 *)&part[nxt][myst][0];
    const uint4 w4 = *(const uint4 *)&wmin[cur][0];
    const uint32_t ca = cadj[blk & 1][J][myst];
    const uint32_t m = umin(umin(p4.x, p4.y), umin(p4.z, p4.w));
    const uint32_t d = __builtin_amdgcn_readfirstlane(umin(umin(w4.x, w4.y), umin(w4.z, w4.w))) >> BITS;
    dsum += d;
    qv = umin((m >> BITS) - d + ca, QCAP) << BITS;
    if (lane < 16) argb[blk & 1][J][myst] = (uint8_t)m;
    const uint32_t wm = group_min<16>(qv);
    if (lane == 0) wmin[nxt][wid] = wm;
    if (J == 0) csb[0].flush(blk - 1, argb[(blk - 1) & 1]);
    if (J == U - 1 && blk + 1 < nblk) {
      csb[1 - PB].store(blk + 1, cadj[(blk + 1) & 1], &flags);
      if (blk + 3 < nblk) csb[1 - PB].load(blk + 3);
      if (EP == 0) ecur = enext;
      if (EP == 0 && blk + 2 < nblk) enext = load_edges(blk + 2);
    }
  };
  auto group = [&](auto Pc, int blk, bool guard) __attribute__((always_inline)) {
    step(std::integral_constant<int, 0>{}, Pc, blk, guard);
    step(std::integral_constant<int, 1>{}, Pc, blk, guard);
    step(std::integral_constant<int, 2>{}, Pc, blk, guard);
    step(std::integral_constant<int, 3>{}, Pc, blk, guard);
    step(std::integral_constant<int, 4>{}, Pc, blk, guard);
    step(std::integral_constant<int, 5>{}, Pc, blk, guard);
    step(std::integral_constant<int, 6>{}, Pc, blk, guard);
    step(std::integral_constant<int, 7>{}, Pc, blk, guard);
    step(std::integral_constant<int, 8>{}, Pc, blk, guard);
    step(std::integral_constant<int, 9>{}, Pc, blk, guard);
    step(std::integral_constant<int, 10>{}, Pc, blk, guard);
    step(std::integral_constant<int, 11>{}, Pc, blk, guard);
  };
  const std::integral_constant<int, 0> even{};
  const std::integral_constant<int, 1> odd{};

  group(even, 0, true);
  int blk = 1;  // odd
  for (; (blk + 2) * U <= N; blk += 2) {
    group(odd, blk, false);
    group(even, blk + 1, false);
  }
  if (blk < nblk) group(odd, blk, true);
  if (blk + 1 < nblk) group(even, blk + 1, true);
  __syncthreads();
  csb[0].flush((N - 1) / U, argb[((N - 1) / U) & 1]);

  const uint32_t pk = (lane < 16 && myst < K) ? (qv | (uint32_t)myst) : kSat;
  finish_search(pk, csb[0].csum + csb[1].csum, dsum, BITS, QCAP, flags, hdr, b, opt, status, res);
}

template <int EP>
static void launch_k64_ep(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *table, SearchResult *res,
                          const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st) {
  timed_launch(chain_fwd_k64_kernel<EP>, dim3(d.batch), dim3(kThreads), 0, st, d.cost, d.rtab, redge_dev,
                     d.n_blocks, d.k, d.n_tables, table, res, hdr, opt, status);
}

void launch_chain_fwd_k64(const cfp_chain_desc &d, int period, const int32_t *redge_dev, uint8_t *table,
                          SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st) {
  switch (period) {
    case 1: launch_k64_ep<1>(d, redge_dev, table, res, hdr, opt, status, st); break;
    case 2: launch_k64_ep<2>(d, redge_dev, table, res, hdr, opt, status, st); break;
    case 3: launch_k64_ep<3>(d, redge_dev, table, res, hdr, opt, status, st); break;
    case 4: launch_k64_ep<4>(d, redge_dev, table, res, hdr, opt, status, st); break;
    case 6: launch_k64_ep<6>(d, redge_dev, table, res, hdr, opt, status, st); break;
    case 12: launch_k64_ep<12>(d, redge_dev, table, res, hdr, opt, status, st); break;
    default: launch_k64_ep<0>(d, redge_dev, table, res, hdr, opt, status, st); break;
  }
}

}  // namespace cfp
