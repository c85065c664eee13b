// Segment-level search with boundary resharding (Sec. 4.2-4.4).
//
// The chain is one of segments; segment i picks one of K plans.  A plan is a
// combination of the strategies of the segment's blocks, and the resharding
// cost between consecutive segments depends only on the strategy of the
// earlier segment's last block and of the later segment's first block: only
// those boundary block pairs are profiled (Sec. 4.2; 3 x 3 = 9 pairs for
// segments of four blocks with three strategies each, Sec. 5.5).  So Eq. T's
// resharding term is r_e[last(t)][first(s)] and the step of the recurrence
// factorises:
//     D[i][s] = c[i][s] + min_l (M_l + r_{e(i)}[l][first(s)]),
//     M_l     = min_{t : last(t) = l} D[i-1][t],
// O(K + L F) work per step instead of O(K^2).
//
// One wave per search, four searches per workgroup, no barrier: lane x holds
// the states x, x+64, ...  A row lives in registers as exact-normalised values
// Q[s] = min(D[i][s] - min_s D[i][s], cap).  With one wave per SIMD at the
// usual batch sizes a step costs what its instructions take to issue, so it is
// built from lane exchanges only (DPP, permlane swaps), with no LDS:
//   1. class minima: the packed words (Q << b) | t are reduced over the wave
//      per class by a reduce-scatter (each exchange halves the classes a lane
//      keeps, until a lane keeps one), then by plain exchanges; a minimum
//      carries the lowest predecessor t of least value.  Afterwards every lane
//      holds the minimum of the class its position names.
//   2. boundary minima: the lane that holds M_l for boundary pair (l, f)
//      forms M_l + r[l][f]; a minimum over the lanes of pair group f gives
//      G_f, which every state s then takes for f = first(s).
//   3. the new row: D = G + c, its minimum normalises the row.
// Through the row's argmin (Q = 0) the best candidate of every state is at
// most r_max, exact while r_max < cap = 2^(32-b) - 1; a state at the cap is
// beaten through that argmin by every continuation.  So while the previous row
// has a reachable state every G_f is finite, and an unavailable strategy alone
// makes D unreachable (a saturating add).  The cost rows and the boundary
// entries come from rings of kSegAhead rows in registers, loaded that many
// steps ahead (the edge indices twice as far), so the wait for a row's data
// never covers the loads and argmin stores of the steps since.
#include "cfp_internal.h"
#include "common.h"

namespace cfp {

namespace {

constexpr int kSegWaves = 4;  // searches per workgroup
constexpr int kSegMaxLF = 8;  // largest number of strategies of a boundary block
constexpr int kSegAhead = 8;  // rows in flight per lane

// DPP controls: quad_perm [1,0,3,2] and [2,3,0,1] (lane ^ 1, lane ^ 2),
// row_ror:4 and :8, row_half_mirror, row_mirror, row_newbcast:n.
constexpr int kXor1 = 0xB1, kXor2 = 0x4E, kRor4 = 0x124, kRor8 = 0x128, kHalfMirror = 0x141, kMirror = 0x140;
constexpr int kRowBcast = 0x150;

template <int CTRL>
__device__ __forceinline__ uint32_t from_dpp(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, CTRL, 0xF, 0xF, true);
}
template <int CTRL>
__device__ __forceinline__ uint32_t min_dpp(uint32_t keep, uint32_t send) {
  return umin(keep, from_dpp<CTRL>(send));
}

// Minimum over the lanes with equal lane % 16 (the four rows).
__device__ __forceinline__ uint32_t seg_cross_rows(uint32_t x) {
  const auto h = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  x = umin(h[0], h[1]);
  const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  return umin(r[0], r[1]);
}

// Raw buffer resource over [base, base + bytes): loads beyond it read 0 and
// stores beyond it are dropped (32-bit data format, no swizzle).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}

// Minimum over the 64 lanes of a wave; every lane gets it.
__device__ __forceinline__ uint32_t seg_wave_min(uint32_t x) {
  x = min_dpp<kXor1>(x, x);
  x = min_dpp<kXor2>(x, x);
  x = min_dpp<kHalfMirror>(x, x);
  x = min_dpp<kMirror>(x, x);
  return seg_cross_rows(x);
}

// Minimum over the 64 lanes of a wave, as a scalar: the four row minima are
// read independently and combined on the scalar unit.
__device__ __forceinline__ uint32_t seg_wave_min_s(uint32_t x) {
  x = min_dpp<kXor1>(x, x);
  x = min_dpp<kXor2>(x, x);
  x = min_dpp<kHalfMirror>(x, x);
  x = min_dpp<kMirror>(x, x);
  const uint32_t r0 = __builtin_amdgcn_readlane(x, 0), r1 = __builtin_amdgcn_readlane(x, 16);
  const uint32_t r2 = __builtin_amdgcn_readlane(x, 32), r3 = __builtin_amdgcn_readlane(x, 48);
  return umin(umin(r0, r1), umin(r2, r3));
}

}  // namespace

// SPL states per lane (K <= 64 SPL); LM >= n_last, n_first is 4 or 8.  The
// argmin entries are 16-bit exactly when K > 256, i.e. SPL = 8.
//
// Class of a lane after the reduce-scatter (bits b0, b1, b2 of the lane):
// LM = 4: 2 b0 + b1; LM = 8: 4 b0 + 2 b1 + b2.  Boundary pair (l, f) sits in
// the lanes of class l in group f: LM = 4, groups of 4 lanes, f = (lane / 4) %
// 4 (every row holds all pairs); LM = 8, groups of 8 lanes, f = lane / 8.
template <int SPL, int LM>
__global__ __launch_bounds__(kSegWaves * 64) void seg_fwd_kernel(
    const int32_t *__restrict__ cost, const int32_t *__restrict__ rbound, const uint8_t *__restrict__ last,
    const uint8_t *__restrict__ first, const int32_t *__restrict__ redge, int N, int K, int B, int L, int F,
    int bits, uint8_t *__restrict__ table, SearchResult *__restrict__ res, const WsHeader *__restrict__ hdr,
    int64_t *__restrict__ opt, int32_t *__restrict__ status) {
  static_assert(LM == 4 || LM == 8, "classes per boundary side");
  constexpr bool kWide = SPL == 8;
  constexpr int H = LM / 2;  // classes a lane keeps after the first exchange
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int b = blockIdx.x * kSegWaves + wid;
  if (b >= B) return;  // the waves are independent: nothing below waits for another wave
  const uint32_t CAP = (1u << (32 - bits)) - 1u, IMASK = (1u << bits) - 1u;
  const int32_t *cb = cost + (size_t)b * N * K;
  const int b0 = lane & 1, b1 = (lane >> 1) & 1, b2 = (lane >> 2) & 1;

  int ls[SPL], fs[SPL];
  bool real[SPL];
  uint32_t q[SPL];
  bool bad = false;
#pragma unroll
  for (int j = 0; j < SPL; ++j) {
    const int s = lane + 64 * j;
    real[j] = s < K;
    ls[j] = real[j] ? last[s] : 0;
    fs[j] = real[j] ? first[s] : 0;
    bad |= real[j] && (ls[j] >= L || fs[j] >= F);
    if (ls[j] >= L) ls[j] = 0;  // keep the selects in range; the search reports bad input
    if (fs[j] >= F) fs[j] = 0;
    if (!real[j]) ls[j] = -1;  // in no class
  }
  const uint32_t sl = lane < K ? (uint32_t)lane : 0u;  // a lane's first state, clamped for the loads

  // Memory goes through buffer resources: a scalar row offset plus a fixed
  // lane offset, so a step spends no vector instructions on addresses.  The
  // host keeps N K 4 below 2^31.
  const uint32_t K4 = (uint32_t)K * 4u, last_row = (uint32_t)(N - 1) * K4;
  const __amdgpu_buffer_rsrc_t crs = make_rsrc(cb, (uint32_t)N * K4);
  const __amdgpu_buffer_rsrc_t rrs = make_rsrc(rbound, 0x7FFFFFFFu);  // offsets come from checked edges
  const __amdgpu_buffer_rsrc_t ers = make_rsrc(redge, (uint32_t)N * 4u);

  // Ring of cost rows: row i >= 1 sits in slot (i - 1) % kSegAhead.
  int32_t ring[kSegAhead][SPL];
  uint32_t coff[SPL];  // byte offset of a lane's states within a row
#pragma unroll
  for (int j = 0; j < SPL; ++j) coff[j] = (real[j] ? (uint32_t)(lane + 64 * j) : sl) * 4u;
  auto load_row = [&](uint32_t roff, int32_t(&dst)[SPL]) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < SPL; ++j) dst[j] = __builtin_amdgcn_raw_buffer_load_b32(crs, (int)coff[j], (int)roff, 0);
  };
  int32_t c0[SPL];
  load_row(0, c0);

  // Boundary lanes and the ring of their entries r_{e(i)}[l][f]; the edge
  // index of a row is read kSegAhead steps before its entries, into a ring of
  // its own (every lane loads it; one lane's copy is read).
  const int lf_l = LM == 4 ? 2 * b0 + b1 : 4 * b0 + 2 * b1 + b2;
  const int lf_f = LM == 4 ? (lane >> 2) & 3 : lane >> 3;
  const bool lf = lf_l < L && lf_f < F;
  const uint32_t lf_off = lf ? (uint32_t)(lf_l * F + lf_f) * 4u : 0u;  // bytes
  const uint32_t LF4 = (uint32_t)(L * F) * 4u;
  auto load_r = [&](uint32_t e) __attribute__((always_inline)) {
    return (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(rrs, (int)lf_off, (int)(e * LF4), 0);
  };
  auto load_e = [&](uint32_t eoff) __attribute__((always_inline)) {
    return (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(ers, 0, (int)eoff, 0);
  };
  auto row_off = [&](int i) __attribute__((always_inline)) { return min((uint32_t)i * K4, last_row); };
  auto edge_off = [&](int i) __attribute__((always_inline)) { return (uint32_t)min(i, N - 1) * 4u; };
  uint32_t rring[kSegAhead], ering[kSegAhead];
#pragma unroll
  for (int u = 0; u < kSegAhead; ++u) {  // in the order the steps issue them
    rring[u] = load_r(__builtin_amdgcn_readfirstlane(load_e(edge_off(1 + u))));
    ering[u] = load_e(edge_off(1 + u + kSegAhead));
    load_row(row_off(1 + u), ring[u]);
  }

  // Row 0.
  uint32_t ym = kSat;
#pragma unroll
  for (int j = 0; j < SPL; ++j) {
    const int32_t c = c0[j];
    bad |= real[j] && c < 0;
    const uint32_t y = !real[j] || c == CFP_COST_INF ? kSat : (uint32_t)c;
    q[j] = y;
    ym = umin(ym, y);
  }
  uint32_t rmin = __builtin_amdgcn_readfirstlane(seg_wave_min(ym));
  int64_t o = rmin;
  uint32_t rmax = rmin;  // kSat once a row has no reachable state
#pragma unroll
  for (int j = 0; j < SPL; ++j) q[j] = umin(q[j] - rmin, CAP);

  uint32_t neg = 0;  // OR of the costs read: the sign bit flags a negative one

  // Wait here for every load above (once per search): the waits in the loop
  // then count only the loads the loop itself issued, several steps back
  // (the compiler orders the loads above by kind, not by slot).
#pragma unroll
  for (int u = 0; u < kSegAhead; ++u) {
    asm volatile("" ::"v"(rring[u]), "v"(ering[u]));
#pragma unroll
    for (int j = 0; j < SPL; ++j) asm volatile("" ::"v"(ring[u][j]));
  }

  // Argmin cells of this search: a lane without a state stores out of the
  // resource's range (dropped); in the steps past the last row every lane
  // stores into row 0, which is never read back.  So every step issues the
  // same loads and stores, with no branch between them.
  constexpr uint32_t kElem = kWide ? 2u : 1u;
  const __amdgpu_buffer_rsrc_t trs = make_rsrc(table + (size_t)b * N * K * kElem, (uint32_t)N * K * kElem);
  uint32_t toff[SPL];
#pragma unroll
  for (int j = 0; j < SPL; ++j) toff[j] = real[j] ? (uint32_t)(lane + 64 * j) * kElem : 0x80000000u;

  // The step of row i, with its data in ring slot U = (i - 1) % kSegAhead.
  // Steps with i >= N (the padding of the last group) change no state.
  auto step = [&](int i, auto Uc) __attribute__((always_inline)) {
    constexpr int U = decltype(Uc)::value;
    const bool valid = i < N;
    // 1. class minima of the previous row
    uint32_t pk[SPL];
#pragma unroll
    for (int j = 0; j < SPL; ++j) pk[j] = (q[j] << bits) | (uint32_t)(lane + 64 * j);
    auto part = [&](int cls) __attribute__((always_inline)) {
      uint32_t x[SPL];
#pragma unroll
      for (int j = 0; j < SPL; ++j) x[j] = ls[j] == cls ? pk[j] : kSat;
#pragma unroll
      for (int w = 1; w < SPL; w *= 2)  // a tree, not a chain
#pragma unroll
        for (int j = 0; j + w < SPL; j += 2 * w) x[j] = umin(x[j], x[j + w]);
      return x[0];
    };
    // first exchange (lane ^ 1): keep the classes H b0 + m, send H (1 - b0) + m
    uint32_t A[H];
#pragma unroll
    for (int m = 0; m < H; ++m) A[m] = min_dpp<kXor1>(part(H * b0 + m), part(H * (1 - b0) + m));
    uint32_t M;
    if constexpr (LM == 4) {
      // second (lane ^ 2): keep class 2 b0 + b1; then the rest of the row, the rows
      M = min_dpp<kXor2>(b1 ? A[1] : A[0], b1 ? A[0] : A[1]);
      M = min_dpp<kRor4>(M, M);
    } else {
      uint32_t Bv[2];
#pragma unroll
      for (int n = 0; n < 2; ++n) Bv[n] = min_dpp<kXor2>(b1 ? A[2 + n] : A[n], b1 ? A[n] : A[2 + n]);
      // third (lane +- 4 within the row, bit 2 flipped): keep class 4 b0 + 2 b1 + b2
      M = min_dpp<kRor4>(b2 ? Bv[1] : Bv[0], b2 ? Bv[0] : Bv[1]);
    }
    M = min_dpp<kRor8>(M, M);
    M = seg_cross_rows(M);
    // 2. boundary minima: the pair lanes offer M_l + r[l][f]; group minimum
    const uint32_t r = rring[U];
    uint32_t cand = sat_add(M, lf ? r << bits : kSat);
    cand = min_dpp<kXor1>(cand, cand);
    cand = min_dpp<kXor2>(cand, cand);
    uint32_t g[SPL];
    if constexpr (LM == 4) {
      uint32_t G[4];
      G[0] = from_dpp<kRowBcast + 0>(cand);
      G[1] = from_dpp<kRowBcast + 4>(cand);
      G[2] = from_dpp<kRowBcast + 8>(cand);
      G[3] = from_dpp<kRowBcast + 12>(cand);
#pragma unroll
      for (int j = 0; j < SPL; ++j) {
        const uint32_t lo = fs[j] & 1 ? G[1] : G[0], hi = fs[j] & 1 ? G[3] : G[2];
        g[j] = fs[j] & 2 ? hi : lo;
      }
    } else {
      cand = min_dpp<kHalfMirror>(cand, cand);
      uint32_t G[8];
#pragma unroll
      for (int f = 0; f < 8; ++f) G[f] = __builtin_amdgcn_readlane(cand, 8 * f);
#pragma unroll
      for (int j = 0; j < SPL; ++j) {
        uint32_t x = G[0];
#pragma unroll
        for (int f = 1; f < 8; ++f) x = fs[j] == f ? G[f] : x;
        g[j] = x;
      }
    }
    // 3. the new row; the low bits of an argmin entry are the predecessor
    // (the bits above it are not read back)
    const uint32_t trow = valid ? (uint32_t)i * (uint32_t)K * kElem : 0u;
    ym = kSat;
    uint32_t yn[SPL];
#pragma unroll
    for (int j = 0; j < SPL; ++j) {
      const int32_t cc = ring[U][j];
      if (kWide) __builtin_amdgcn_raw_buffer_store_b16((uint16_t)g[j], trs, (int)toff[j], (int)trow, 0);
      else __builtin_amdgcn_raw_buffer_store_b8((uint8_t)g[j], trs, (int)toff[j], (int)trow, 0);
      neg |= (uint32_t)cc;
      const bool dead = !real[j] | (cc == CFP_COST_INF);
      yn[j] = sat_add(g[j] >> bits, dead ? kSat : (uint32_t)cc);
      ym = umin(ym, yn[j]);
    }
    // The sign check is kept here: sunk to the end of the loop it would hold
    // every ring slot live across the refills below.
    asm volatile("" : "+v"(neg));
    // the loads of row i + kSegAhead, into the registers just read (kept
    // below their last reads, so each ring slot stays in its registers)
    __builtin_amdgcn_sched_barrier(0);
    rring[U] = load_r(__builtin_amdgcn_readfirstlane(ering[U]));
    ering[U] = load_e(edge_off(i + 2 * kSegAhead));
    load_row(row_off(i + kSegAhead), ring[U]);
    const uint32_t rm = seg_wave_min_s(ym);
    if (valid) {  // uniform; no memory operation below
      o += rm;
      rmax = max(rmax, rm);
#pragma unroll
      for (int j = 0; j < SPL; ++j) q[j] = umin(yn[j] - rm, CAP);
    }
  };
  // rows in groups of kSegAhead so that every ring slot is a constant
  for (int i0 = 1; i0 < N; i0 += kSegAhead) {
    step(i0 + 0, std::integral_constant<int, 0>{});
    step(i0 + 1, std::integral_constant<int, 1>{});
    step(i0 + 2, std::integral_constant<int, 2>{});
    step(i0 + 3, std::integral_constant<int, 3>{});
    step(i0 + 4, std::integral_constant<int, 4>{});
    step(i0 + 5, std::integral_constant<int, 5>{});
    step(i0 + 6, std::integral_constant<int, 6>{});
    step(i0 + 7, std::integral_constant<int, 7>{});
  }
  static_assert(kSegAhead == 8, "the group above has kSegAhead steps");

  // Lowest final state of least value (the least is 0 after normalisation).
  uint32_t pk = kSat;
#pragma unroll
  for (int j = 0; j < SPL; ++j)
    if (real[j]) pk = umin(pk, (q[j] << bits) | (uint32_t)(lane + 64 * j));
  const uint32_t fin = __builtin_amdgcn_readfirstlane(seg_wave_min(pk));
  const bool infeasible = rmax == kSat;
  bad = __any(bad || (int32_t)neg < 0);
  if (lane == 0) {
    int st = CFP_ST_OK;
    if (bad || hdr->rflag) st = CFP_ST_BADINPUT;
    else if (infeasible) st = CFP_ST_INFEASIBLE;
    else if ((fin >> bits) != 0) st = CFP_ST_OVERFLOW;
    status[b] = st;
    opt[b] = st == CFP_ST_OK ? o + (int64_t)(fin >> bits) : INT64_MAX;
    res[b].final_state = st == CFP_ST_OK ? (int32_t)(fin & IMASK) : -1;
    res[b].status = st;
    res[b].final_m = 0;
  }
}

bool seg_supported(int k, int n_last, int n_first) {
  return k >= 1 && k <= CFP_MAX_K && n_last >= 1 && n_last <= kSegMaxLF && n_first >= 1 && n_first <= kSegMaxLF;
}

template <int SPL, int LM>
static void launch_seg_spl(const cfp_segment_desc &d, const int32_t *redge_dev, uint8_t *table, SearchResult *res,
                           const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st) {
  const int grid = (d.batch + kSegWaves - 1) / kSegWaves;
  timed_launch(seg_fwd_kernel<SPL, LM>, dim3(grid), dim3(kSegWaves * 64), 0, st, d.cost, d.rbound, d.last,
               d.first, redge_dev, d.n_segments, d.k, d.batch, d.n_last, d.n_first, index_bits(d.k), table, res,
               hdr, opt, status);
}

template <int LM>
static void launch_seg_lm(const cfp_segment_desc &d, const int32_t *redge_dev, uint8_t *table, SearchResult *res,
                          const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st) {
  if (d.k <= 64) launch_seg_spl<1, LM>(d, redge_dev, table, res, hdr, opt, status, st);
  else if (d.k <= 128) launch_seg_spl<2, LM>(d, redge_dev, table, res, hdr, opt, status, st);
  else if (d.k <= 256) launch_seg_spl<4, LM>(d, redge_dev, table, res, hdr, opt, status, st);
  else launch_seg_spl<8, LM>(d, redge_dev, table, res, hdr, opt, status, st);
}

hipError_t launch_seg_fwd(const cfp_segment_desc &d, const int32_t *redge_dev, uint8_t *table, SearchResult *res,
                          const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st) {
  timer_begin(st);
  if (d.n_last <= 4 && d.n_first <= 4) launch_seg_lm<4>(d, redge_dev, table, res, hdr, opt, status, st);
  else launch_seg_lm<8>(d, redge_dev, table, res, hdr, opt, status, st);
  timer_end(st);
  return hipGetLastError();
}

}  // namespace cfp
