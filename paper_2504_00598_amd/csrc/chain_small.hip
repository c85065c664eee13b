// One-launch search of small chains (Sec. 4.4: the Eq. T recurrence and the
// traceback of the lowest-index optimal plan), for callers that want one
// search's answer as soon as possible.  One workgroup of eight waves per search:
//   1. all eight waves stage the resharding tables into LDS, transposed and
//      packed as (R[t][s] << b) | t, checking every entry against the exact
//      range, the search's cost rows, checking for negative costs, and the
//      edge map (a batch of loads in flight per lane before any is used);
//   2. wave 0 runs the recurrence.  For K <= 16 all 64 lanes work on a step:
//      lane (g, s) (row g of 16 lanes) forms the candidates of state s from
//      the predecessors 4g .. 4g+3, whose values reach the row by a DPP row
//      broadcast of the previous row rotated by 4g lanes in row g; the four
//      rows' minima meet by two permlane swaps.  For larger K lane s works for
//      state s over all predecessors, whose values reach it by readlane.  One
//      unsigned minimum per candidate pair keeps the value and the lowest
//      predecessor; the argmin bytes go to LDS;
//   3. wave 0 walks the argmins back from the lowest optimal final state.
// The edge map travels in the kernel arguments, so a search needs no
// host-to-device copy and no workspace.
//
// Normalisation: x[s] = (m >> b) + c[i][s] with m the packed minimum; the row
// is split into d = min_s x[s] (summed exactly in 64 bits) and
// Q[s] = min(x[s] - d, cap) << b, cap = 2^(31-b) - 1, so Q < 2^31.  Packed
// table words are below 2^30 (R < 2^(30-b)); a padding predecessor t >= K
// has the word 2^31 | t.  So no candidate leaves 32 bits (plain adds), a
// padding predecessor never wins, and the best candidate of every state, at
// most R_max through the row's minimum, is below the cap: a capped state never
// wins.  Unavailable strategies and padding states take x = 2^32 - 1.
#include "cfp_internal.h"
#include "common.h"

namespace cfp {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct SmallArgs {
  const int32_t *cost;  // [B][N][K]
  const int32_t *rtab;  // [E][K][K]
  int64_t *opt;
  int32_t *status;
  int32_t *plan;        // [B][N]
  int N, K, E;
  int32_t rlimit;
  uint8_t redge[kSmallMaxN];  // table of edge (i-1 -> i); entry 0 unused
};

template <int KP>
struct SmallShape {
  static constexpr int BITS = KP <= 16 ? 4 : KP <= 32 ? 5 : 6;
  static constexpr int CS = KP + 4;  // LDS stride of a table column (words)
  static constexpr uint32_t CAP = (1u << (31 - BITS)) - 1u;
};

constexpr int kSmallThreads = 512;
constexpr int kSmallTab = 8, kSmallCost = 4;   // table and cost rows in flight per lane while staging
constexpr uint32_t kPadWord = 0x80000000u;     // | t: the word of a padding predecessor
constexpr int kRowBcast = 0x150;               // DPP row_newbcast:n = kRowBcast + n
constexpr int kRowRor = 0x120;                 // DPP row_ror:n = kRowRor + n

// min(keep, the partner lane's send): quad_perm partners lane ^ 1 and lane ^ 2;
// the half mirror pairs lane i with lane 7 - i of its eight, the mirror lane i
// with lane 15 - i of its row.
template <int CTRL>
__device__ __forceinline__ uint32_t min_dpp(uint32_t keep, uint32_t send) {
  return umin(keep, (uint32_t)__builtin_amdgcn_mov_dpp((int)send, CTRL, 0xF, 0xF, true));
}

// Minimum over each row of 16 lanes (every lane of the row gets it).
__device__ __forceinline__ uint32_t small_row_min(uint32_t x) {
  x = min_dpp<0xB1>(x, x);
  x = min_dpp<0x4E>(x, x);
  x = min_dpp<0x141>(x, x);
  return min_dpp<0x140>(x, x);
}

// Minimum over the 64 lanes (every lane gets it).
__device__ __forceinline__ uint32_t small_wave_min(uint32_t x) {
  x = small_row_min(x);
  const auto h = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  x = umin(h[0], h[1]);
  const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  return umin(r[0], r[1]);
}

template <int KP>
__global__ __launch_bounds__(kSmallThreads) void chain_small_kernel(SmallArgs a) {
  using S = SmallShape<KP>;
  constexpr int BITS = S::BITS, CS = S::CS;
  extern __shared__ __align__(16) uint32_t lds[];
  const int N = a.N, K = a.K, E = a.E;
  uint32_t *tab = lds;                        // [E][KP][CS]: column s of table e at (e KP + s) CS
  uint32_t *crow = tab + (size_t)E * KP * CS;  // [N][KP] costs (kSat for unavailable and padding)
  uint8_t *arg = (uint8_t *)(crow + (size_t)N * KP);  // [N][KP] argmins
  uint8_t *red = arg + (size_t)N * KP;                // [N] the edge map
  const int b = blockIdx.x, tid = threadIdx.x;

  // 1. Tables and costs into LDS, with the range checks.  Entries are read in
  // their natural order (rows of K words) from the two arrays' uniform bases:
  // a batch of kSmallTab table rows and kSmallCost cost rows per lane is in
  // flight before any is used, and no load sits behind a branch (rows past
  // the end and padding states are clamped to a valid word and not used).
  int bad = 0;
  const int32_t *cb = a.cost + (size_t)b * N * K;
  // thread tid covers state ss of rows r0, r0 + RPI, ... (RPI rows per load instruction)
  constexpr unsigned RPI = kSmallThreads / KP;
  const unsigned ss = (unsigned)tid % KP, r0 = (unsigned)tid / KP, ssc = min(ss, (unsigned)K - 1);
  const unsigned trows = (unsigned)(E * KP), crows = (unsigned)N, uK = (unsigned)K;
  for (unsigned tb = 0, cr = 0; tb < trows || cr < crows; tb += RPI * kSmallTab, cr += RPI * kSmallCost) {
    int32_t vt[kSmallTab], vc[kSmallCost];
#pragma unroll
    for (int u = 0; u < kSmallTab; ++u) {
      const unsigned r = min(tb + RPI * u + r0, trows - 1), e = r / KP, t = min(r % KP, uK - 1);
      vt[u] = a.rtab[__umul24(__umul24(e, uK) + t, uK) + ssc];
    }
#pragma unroll
    for (int u = 0; u < kSmallCost; ++u) {
      const unsigned i = min(cr + RPI * u + r0, crows - 1);
      vc[u] = cb[__umul24(i, uK) + ssc];
    }
#pragma unroll
    for (int u = 0; u < kSmallTab; ++u) {
      const unsigned r = tb + RPI * u + r0, e = r / KP, t = r % KP;
      if (r < trows) {
        uint32_t w = kPadWord | t;
        if (t < uK && ss < uK) {
          bad |= vt[u] < 0 || vt[u] >= a.rlimit;
          w = ((uint32_t)vt[u] << BITS) | t;
        }
        tab[(e * KP + ss) * CS + t] = w;
      }
    }
#pragma unroll
    for (int u = 0; u < kSmallCost; ++u) {
      const unsigned i = cr + RPI * u + r0;
      if (i < crows) {
        const bool real = ss < uK;
        bad |= real && vc[u] < 0;
        crow[i * KP + ss] = (!real || vc[u] == CFP_COST_INF) ? kSat : (uint32_t)vc[u];
      }
    }
  }
  for (int i = tid; i < N; i += kSmallThreads) red[i] = a.redge[i];
  __syncthreads();

  // 2. The recurrence, wave 0.  The table index of row i + 2 is read while row
  // i is computed and the table column of row i + 1 is read.
  const int lane = tid & 63;
  uint64_t dsum = 0;
  bool infeasible = false;
  uint32_t Q = 0;
  if (tid < 64) {
    if constexpr (KP == 16) {
      const int g = lane >> 4, l = lane & 15;  // row, state
      const bool sin = l < K;
      uint32_t x = crow[l];
      uint32_t dv = small_row_min(x);  // the row minimum, in every lane
      uint32_t d = __builtin_amdgcn_readfirstlane(dv);
      infeasible |= d == kSat;
      dsum += d;
      Q = umin(x - dv, S::CAP) << BITS;
      const uint32_t *colb = tab + l * CS + 4 * g;  // predecessors 4g .. 4g+3 of state l
      u32x4 rp = *(const u32x4 *)(colb + red[min(1, N - 1)] * KP * CS);
      uint32_t cnext = crow[min(1, N - 1) * KP + l];
      int enext = red[min(2, N - 1)];
      for (int i = 1; i < N; ++i) {
        const u32x4 rc = rp;
        const uint32_t cv = cnext;
        rp = *(const u32x4 *)(colb + enext * KP * CS);
        cnext = crow[min(i + 1, N - 1) * KP + l];
        enext = red[min(i + 2, N - 1)];
        // row g holds the previous row rotated by 4g lanes: lane j of the row is state 4g + j
        uint32_t qr = (uint32_t)__builtin_amdgcn_update_dpp((int)Q, (int)Q, kRowRor + 8, 0xC, 0xF, false);
        qr = (uint32_t)__builtin_amdgcn_update_dpp((int)qr, (int)qr, kRowRor + 12, 0xA, 0xF, false);
        const uint32_t c0 = (uint32_t)__builtin_amdgcn_mov_dpp((int)qr, kRowBcast + 0, 0xF, 0xF, true) + rc.x;
        const uint32_t c1 = (uint32_t)__builtin_amdgcn_mov_dpp((int)qr, kRowBcast + 1, 0xF, 0xF, true) + rc.y;
        const uint32_t c2 = (uint32_t)__builtin_amdgcn_mov_dpp((int)qr, kRowBcast + 2, 0xF, 0xF, true) + rc.z;
        const uint32_t c3 = (uint32_t)__builtin_amdgcn_mov_dpp((int)qr, kRowBcast + 3, 0xF, 0xF, true) + rc.w;
        uint32_t m = umin(umin(c0, c1), umin(c2, c3));
        const auto h = __builtin_amdgcn_permlane32_swap(m, m, false, false);
        m = umin(h[0], h[1]);
        const auto r = __builtin_amdgcn_permlane16_swap(m, m, false, false);
        m = umin(r[0], r[1]);  // state l over all predecessors, in every row
        // cv is 2^32 - 1 for an unavailable or padding state, so the
        // saturating add gives x = 2^32 - 1 there and is exact elsewhere
        x = sat_add(m >> BITS, cv);
        if (g == 0) arg[i * KP + l] = (uint8_t)(m & (KP - 1));
        dv = small_row_min(x);
        Q = umin(x - dv, S::CAP) << BITS;  // the next step needs only this
        d = __builtin_amdgcn_readfirstlane(dv);
        infeasible |= d == kSat;
        dsum += d;
      }
      Q = lane < 16 ? (sin ? (Q | (uint32_t)l) : kSat) : kSat;  // final packing, row 0
    } else {
      // Lanes s >= KP duplicate lane KP - 1's addresses and carry x = 2^32 - 1.
      const int s = lane, sl = min(s, KP - 1);
      const bool sin = s < K;
      uint32_t x = s < KP ? crow[sl] : kSat;
      uint32_t d = __builtin_amdgcn_readfirstlane(small_wave_min(x));
      infeasible |= d == kSat;
      dsum += d;
      Q = umin(x - d, S::CAP) << BITS;
      u32x4 col[KP / 4];  // the lane's column of the next edge's table
      auto load_col = [&](int e) __attribute__((always_inline)) {
        const uint32_t *c = tab + (e * KP + sl) * CS;
#pragma unroll
        for (int t = 0; t < KP / 4; ++t) col[t] = *(const u32x4 *)(c + 4 * t);
      };
      load_col(red[min(1, N - 1)]);
      const uint32_t cmask = s < KP ? 0u : kSat;  // lanes past KP carry 2^32 - 1
      uint32_t cnext = crow[min(1, N - 1) * KP + sl] | cmask;
      int enext = red[min(2, N - 1)];
      for (int i = 1; i < N; ++i) {
        u32x4 rp[KP / 4];
#pragma unroll
        for (int t = 0; t < KP / 4; ++t) rp[t] = col[t];
        const uint32_t cv = cnext;
        load_col(enext);
        cnext = crow[min(i + 1, N - 1) * KP + sl] | cmask;
        enext = red[min(i + 2, N - 1)];
        uint32_t m0 = kSat, m1 = kSat;
#pragma unroll
        for (int t = 0; t < KP / 4; ++t) {
          const uint32_t q0 = __builtin_amdgcn_readlane(Q, 4 * t), q1 = __builtin_amdgcn_readlane(Q, 4 * t + 1);
          const uint32_t q2 = __builtin_amdgcn_readlane(Q, 4 * t + 2), q3 = __builtin_amdgcn_readlane(Q, 4 * t + 3);
          m0 = umin(umin(m0, q0 + rp[t].x), q1 + rp[t].y);
          m1 = umin(umin(m1, q2 + rp[t].z), q3 + rp[t].w);
        }
        const uint32_t m = umin(m0, m1);
        x = sat_add(m >> BITS, cv);  // cv = 2^32 - 1: unavailable or padding
        if (s < KP) arg[i * KP + s] = (uint8_t)(m & (KP - 1));
        const uint32_t dv = small_wave_min(x);
        Q = umin(x - dv, S::CAP) << BITS;
        d = __builtin_amdgcn_readfirstlane(dv);
        infeasible |= d == kSat;
        dsum += d;
      }
      Q = sin ? (Q | (uint32_t)s) : kSat;  // final packing
    }
  }

  // 3. Final state and traceback (wave 0).
  const uint32_t pk = small_wave_min(Q);
  bad = __syncthreads_or(bad);  // also orders the argmin bytes before the walk
  const int st = bad ? CFP_ST_BADINPUT : infeasible ? CFP_ST_INFEASIBLE : CFP_ST_OK;
  // the plan is walked into LDS (over the cost rows, no longer needed) and
  // stored by all lanes of wave 0
  int32_t *pw = (int32_t *)crow;
  if (st == CFP_ST_OK && tid == 0) {
    int cur = (int)(pk & (KP - 1));
    pw[N - 1] = cur;
    for (int i = N - 1; i >= 1; --i) {
      cur = arg[i * KP + cur];
      pw[i - 1] = cur;
    }
  }
  __syncthreads();
  if (tid < 64) {
    int32_t *pl = a.plan + (size_t)b * N;
    for (int i = tid; i < N; i += 64) pl[i] = st == CFP_ST_OK ? pw[i] : -1;
    if (tid == 0) a.opt[b] = st == CFP_ST_OK ? (int64_t)dsum : INT64_MAX;
    // status last: a caller that polls it in host memory finds plan and opt
    // complete once it is written
    __threadfence_system();
    if (tid == 0) __hip_atomic_store(&a.status[b], st, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  }
}

int small_kp(int k) { return k <= 16 ? 16 : k <= 32 ? 32 : 64; }

// LDS of a search: tables, costs, argmins and the edge map (the bound
// documented in cfp.h).
size_t small_bytes(int kp, int n, int e) {
  return (size_t)e * kp * (kp + 4) * 4 + (size_t)n * (kp * 5 + 1);
}

}  // namespace

bool chain_small_supported(int n, int k, int n_tables, int batch) {
  if (k > 64 || n > kSmallMaxN || n_tables > 255 || batch > kSmallMaxBatch) return false;
  return small_bytes(small_kp(k), n, n_tables) <= kSmallMaxLds;
}

hipError_t launch_chain_small(const cfp_chain_desc &d, int64_t *opt, int32_t *status, int32_t *plan,
                              hipStream_t st) {
  SmallArgs a;
  a.cost = d.cost;
  a.rtab = d.rtab;
  a.opt = opt;
  a.status = status;
  a.plan = plan;
  a.N = d.n_blocks;
  a.K = d.k;
  a.E = d.n_tables;
  a.rlimit = cfp_r_limit(CFP_V_CHAIN, d.k);
  a.redge[0] = 0;
  for (int i = 1; i < d.n_blocks; ++i) a.redge[i] = (uint8_t)d.redge[i];
  const int kp = small_kp(d.k);
  const size_t lds = small_bytes(kp, d.n_blocks, d.n_tables);
  timer_begin(st);
  switch (kp) {
    case 16: timed_launch(chain_small_kernel<16>, dim3(d.batch), dim3(kSmallThreads), (uint32_t)lds, st, a); break;
    case 32: timed_launch(chain_small_kernel<32>, dim3(d.batch), dim3(kSmallThreads), (uint32_t)lds, st, a); break;
    default: timed_launch(chain_small_kernel<64>, dim3(d.batch), dim3(kSmallThreads), (uint32_t)lds, st, a); break;
  }
  timer_end(st);
  return hipGetLastError();
}

}  // namespace cfp
