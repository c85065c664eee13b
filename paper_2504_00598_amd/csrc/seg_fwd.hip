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
// One wave runs one search, or one chunk of one: lane x holds the states x,
// x+64, ...  A row lives in registers as exact-normalised values
// Q[s] = min(D[i][s] - min_s D[i][s], cap).  With one wave per SIMD a step
// costs what its instructions take to issue, so it is built from lane
// exchanges only (DPP, permlane swaps), with no LDS:
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
//
// Parallelism over the chain.  A batch too small to give every SIMD a wave
// cuts each chain into P chunks that run at once, made exact by rank
// convergence (Maleki, Musuvathi and Mytkowicz, PPoPP 2014), as the chunked
// chain searches do; with only L F boundary pairs between segments the rows
// of a run become parallel to the true ones within a few steps.  One
// workgroup per search, wave p for chunk p, the passes separated by barriers:
//   1. speculative pass: chunk p starts at its first row from that row's
//      costs alone, writes its argmin rows and every normalised row with the
//      running sum of its row minima;
//   2. fix-up pass, chunks p >= 1: start again from the last speculative row
//      of chunk p-1 and recompute until the row equals chunk p's speculative
//      row of the same step (from there on every speculative row is the one
//      the true start gives), rewriting the argmins on the way;
//   3. final pass, wave 0: sums the chunks' row minima.  When a
//      chunk's fix-up met no speculative row, its end row is the true one but
//      the next chunk's fix-up started from a wrong row: that chunk is rerun
//      from the true row, at least as far as its fix-up went and then until
//      its row meets the speculative one (or to its end, and the next chunk
//      is rerun in turn).
// The result is the sequential recurrence's bit for bit for every input.
#include <algorithm>

#include "cfp_internal.h"
#include "common.h"

namespace cfp {

namespace {

constexpr int kSegWaves = 4;     // waves (searches or chunks) per workgroup
constexpr int kSegMaxLF = 8;     // largest number of strategies of a boundary block
constexpr int kSegAhead = 8;     // rows in flight per lane
constexpr int kSegMaxP = 8;      // chunks per search (waves of a workgroup)
constexpr int kSegMinRows = 16;  // least rows per chunk
constexpr int kSegSimds = 1024;  // SIMDs of the chip: waves at one per SIMD
constexpr int kSegArgN = 1536;   // longest edge map carried in the kernel arguments (16-bit entries)

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

// Raw buffer resource over [base, base + bytes): loads beyond it read 0 and
// stores beyond it are dropped (32-bit data format, no swizzle).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}

constexpr uint32_t kOob = 0x80000000u;  // a lane offset past every resource (its access is dropped)

enum { kSegFull = 0, kSegSpec = 1, kSegFix = 2, kSegRepair = 3 };

struct SegRec {
  int64_t dfix;   // fix-up: sum of the row minima of its rows (to the meeting row or the chunk end)
  int32_t conv;   // fix-up: meeting row, -1 if none
  int32_t flags;  // speculative pass: bit 0 bad input, bit 1 a row with no available strategy
};

struct SegArgs {
  const int32_t *cost;    // [B][N][K]
  const int32_t *rbound;  // [E][L][F]
  const uint8_t *last, *first;
  const int32_t *redge;   // device copy, entry 0 a valid table
  int N, K, B, E, L, F, bits;
  uint8_t *table;         // argmin entries [B][N][K], u8 or u16 (K > 256)
  // chunk-parallel form
  int P, CL;              // chunks per search, rows per chunk
  uint32_t *ckrow;        // speculative normalised rows [B][N][K]
  int64_t *dck;           // speculative running sum of row minima from the chunk's first row [B][N]
  SegRec *rec;            // [B][P]
  uint32_t *endrow;       // fix-up end rows of chunks that met no speculative row [B][P][K]
  // the edge map itself when N <= kSegArgN and E <= 65536 (no upload before the
  // launch): entry i in the 16-bit half i % 2 of word i / 2, so that a scalar
  // load reads it
  uint32_t earg[kSegArgN / 2];
};
static_assert(sizeof(SegArgs) + 64 <= 4096, "the arguments of a launch fit one 4 KiB block");

}  // namespace

// One run of the recurrence for search b over rows [r0, r1), in one wave.
//   kSegFull, kSegSpec: row r0 from its costs alone (its row minimum counts);
//     kSegSpec stores every normalised row and the running sum of minima.
//   kSegFix, kSegRepair: qs is the normalised row r0 - 1; rows r0 .. are
//     computed and compared with the speculative rows; the run stops at the
//     first row i >= lim that equals it (stop = i), else at r1 - 1 (stop = -1).
// Every computed row's argmins are stored (row r0 has none in kSegFull and
// kSegSpec).  o is the sum of the computed rows' minima, rmax the largest of
// them (kSat when a row has no available strategy); q ends as the last
// computed row; bad flags a negative cost or a boundary map out of range.
//
// SPL states per lane (K <= 64 SPL); LM >= n_last, n_first is 4 or 8.  The
// argmin entries are 16-bit exactly when K > 256, i.e. SPL = 8.  Class of a
// lane after the reduce-scatter (bits b0, b1, b2 of the lane): LM = 4:
// 2 b0 + b1; LM = 8: 4 b0 + 2 b1 + b2.  Boundary pair (l, f) sits in the lanes
// of class l in group f: LM = 4, groups of 4 lanes, f = (lane / 4) % 4 (every
// row holds all pairs); LM = 8, groups of 8 lanes, f = lane / 8.
template <int SPL, int LM, int MODE, bool EA>
__device__ __forceinline__ void seg_run(const SegArgs &a, int b, int r0, int r1, int lim, const uint32_t (&qs)[SPL],
                                        uint32_t (&q)[SPL], int64_t &o, uint32_t &rmax, int &stop, bool &bad) {
  static_assert(LM == 4 || LM == 8, "classes per boundary side");
  constexpr bool kWide = SPL == 8;
  constexpr bool kFromCost = MODE == kSegFull || MODE == kSegSpec;
  constexpr bool kCompare = MODE == kSegFix || MODE == kSegRepair;
  constexpr int H = LM / 2;  // classes a lane keeps after the first exchange
  const int lane = threadIdx.x & 63;
  const int N = a.N, K = a.K, L = a.L, F = a.F, bits = a.bits;
  const uint32_t CAP = (1u << (32 - bits)) - 1u;
  const int b0 = lane & 1, b1 = (lane >> 1) & 1, b2 = (lane >> 2) & 1;

  int ls[SPL], fs[SPL];
  bool real[SPL];
  bad = false;
#pragma unroll
  for (int j = 0; j < SPL; ++j) {
    const int s = lane + 64 * j;
    real[j] = s < K;
    ls[j] = real[j] ? a.last[s] : 0;
    fs[j] = real[j] ? a.first[s] : 0;
    bad |= real[j] && (ls[j] >= L || fs[j] >= F);
    if (ls[j] >= L) ls[j] = 0;  // keep the selects in range; the search reports bad input
    if (fs[j] >= F) fs[j] = 0;
    if (!real[j]) ls[j] = -1;  // in no class
  }
  const uint32_t sl = lane < K ? (uint32_t)lane : 0u;  // a lane's first state, clamped for the loads

  // Memory goes through buffer resources: a scalar row offset plus a fixed
  // lane offset, so a step spends no vector instructions on addresses.  The
  // host keeps N K 8 below 2^31.
  const size_t cells = (size_t)N * K;
  const uint32_t K4 = (uint32_t)K * 4u, last_row = (uint32_t)(N - 1) * K4;
  const __amdgpu_buffer_rsrc_t crs = make_rsrc(a.cost + (size_t)b * cells, (uint32_t)N * K4);
  const __amdgpu_buffer_rsrc_t rrs = make_rsrc(a.rbound, 0x7FFFFFFFu);  // offsets come from checked edges
  const __amdgpu_buffer_rsrc_t ers = make_rsrc(a.redge, (uint32_t)N * 4u);
  // speculative rows (stored by kSegSpec, compared by kSegFix and kSegRepair) and running sums
  const uint32_t *ckb = kFromCost && MODE != kSegSpec ? nullptr : a.ckrow + (size_t)b * cells;
  const __amdgpu_buffer_rsrc_t krs = make_rsrc(ckb, ckb ? (uint32_t)N * K4 : 0u);
  const int64_t *dkb = MODE == kSegSpec ? a.dck + (size_t)b * N : nullptr;
  const __amdgpu_buffer_rsrc_t drs = make_rsrc(dkb, dkb ? (uint32_t)N * 8u : 0u);

  // Rings: row i sits in slot (i - f0) % kSegAhead, f0 the first computed row.
  const int f0 = kFromCost ? r0 + 1 : r0;
  int32_t ring[kSegAhead][SPL];
  uint32_t kring[kCompare ? kSegAhead : 1][SPL];
  uint32_t coff[SPL];  // byte offset of a lane's states within a row
#pragma unroll
  for (int j = 0; j < SPL; ++j) coff[j] = (real[j] ? (uint32_t)(lane + 64 * j) : sl) * 4u;
  auto load_row = [&](uint32_t roff, int32_t(&dst)[SPL]) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < SPL; ++j) dst[j] = __builtin_amdgcn_raw_buffer_load_b32(crs, (int)coff[j], (int)roff, 0);
  };
  auto load_ck = [&](uint32_t roff, uint32_t(&dst)[SPL]) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < SPL; ++j)
      dst[j] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(krs, (int)coff[j], (int)roff, 0);
  };

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
  // table index of row i's boundary (EA: from the kernel arguments)
  auto edge_at = [&](int i) __attribute__((always_inline)) -> uint32_t {
    if constexpr (EA) {
      const int x = min(i, N - 1);
      return (a.earg[x >> 1] >> (16 * (x & 1))) & 0xFFFFu;
    }
    else return load_e(edge_off(i));
  };
  uint32_t rring[kSegAhead], ering[kSegAhead];
  int32_t c0[SPL];
  if constexpr (kFromCost) load_row(row_off(r0), c0);
#pragma unroll
  for (int u = 0; u < kSegAhead; ++u) {
    rring[u] = load_r(__builtin_amdgcn_readfirstlane(edge_at(f0 + u)));
    ering[u] = edge_at(f0 + u + kSegAhead);
    load_row(row_off(f0 + u), ring[u]);
    if constexpr (kCompare) load_ck(row_off(f0 + u), kring[u]);
  }

  // Speculative rows and running sums: a lane without a state, and every lane
  // in a step past the run's end, stores out of range (dropped).
  uint32_t ckoff[SPL];
#pragma unroll
  for (int j = 0; j < SPL; ++j) ckoff[j] = real[j] ? (uint32_t)(lane + 64 * j) * 4u : kOob;
  const uint32_t doff = lane == 0 ? 0u : kOob;
  auto store_spec = [&](int i, bool valid) __attribute__((always_inline)) {
    if constexpr (MODE == kSegSpec) {
      const uint32_t roff = valid ? (uint32_t)i * K4 : kOob;
#pragma unroll
      for (int j = 0; j < SPL; ++j) __builtin_amdgcn_raw_buffer_store_b32(q[j], krs, (int)(ckoff[j] + roff), 0, 0);
      const uint32_t droff = valid ? (uint32_t)i * 8u : kOob;
      typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
      const u32x2 ov = {(uint32_t)(uint64_t)o, (uint32_t)((uint64_t)o >> 32)};
      __builtin_amdgcn_raw_buffer_store_b64(ov, drs, (int)(doff + droff), 0, 0);
    }
  };

  // The start row.
  if constexpr (kFromCost) {
    uint32_t ym = kSat;
#pragma unroll
    for (int j = 0; j < SPL; ++j) {
      const int32_t c = c0[j];
      bad |= real[j] && c < 0;
      const uint32_t y = !real[j] || c == CFP_COST_INF ? kSat : (uint32_t)c;
      q[j] = y;
      ym = umin(ym, y);
    }
    const uint32_t rmin = __builtin_amdgcn_readfirstlane(seg_wave_min(ym));
    o = rmin;
    rmax = rmin;
#pragma unroll
    for (int j = 0; j < SPL; ++j) q[j] = umin(q[j] - rmin, CAP);
    store_spec(r0, true);
  } else {
#pragma unroll
    for (int j = 0; j < SPL; ++j) q[j] = qs[j];
    o = 0;
    rmax = 0;
  }
  stop = -1;
  bool done = false;

  uint32_t neg = 0;  // OR of the costs read: the sign bit flags a negative one

  // Wait here for every load above (once per run): the waits in the loop then
  // count only the loads the loop itself issued, several steps back (the
  // compiler orders the loads above by kind, not by slot).
#pragma unroll
  for (int u = 0; u < kSegAhead; ++u) {
    asm volatile("" ::"v"(rring[u]), "v"(ering[u]));
#pragma unroll
    for (int j = 0; j < SPL; ++j) asm volatile("" ::"v"(ring[u][j]));
    if constexpr (kCompare) {
#pragma unroll
      for (int j = 0; j < SPL; ++j) asm volatile("" ::"v"(kring[u][j]));
    }
  }

  // Argmin cells of this search: a lane without a state stores out of the
  // resource's range (dropped); in a step past the run's end every lane stores
  // into row 0, which is never read back.  So every step issues the same loads
  // and stores, with no branch between them.
  constexpr uint32_t kElem = kWide ? 2u : 1u;
  const __amdgpu_buffer_rsrc_t trs = make_rsrc(a.table + (size_t)b * cells * kElem, (uint32_t)N * K * kElem);
  uint32_t toff[SPL];
#pragma unroll
  for (int j = 0; j < SPL; ++j) toff[j] = real[j] ? (uint32_t)(lane + 64 * j) * kElem : kOob;

  // The step of row i, with its data in ring slot U = (i - f0) % kSegAhead.
  // A step past the run's end (the padding of the last group, or after the
  // run has met the speculative row) changes no state.
  auto step = [&](int i, auto Uc) __attribute__((always_inline)) {
    constexpr int U = decltype(Uc)::value;
    const bool valid = i < r1 && !done;
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
    uint32_t ym = kSat;
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
    ering[U] = edge_at(i + 2 * kSegAhead);
    load_row(row_off(i + kSegAhead), ring[U]);
    const uint32_t rm = seg_wave_min_s(ym);
    if (valid) {  // uniform; no memory operation below
      o += rm;
      rmax = max(rmax, rm);
#pragma unroll
      for (int j = 0; j < SPL; ++j) q[j] = umin(yn[j] - rm, CAP);
    }
    store_spec(i, valid);
    if constexpr (kCompare) {
      bool diff = false;
#pragma unroll
      for (int j = 0; j < SPL; ++j) diff |= real[j] && q[j] != kring[U][j];
      if (valid && i >= lim && __ballot(diff) == 0) {  // uniform
        stop = i;
        done = true;
      }
      // the speculative row i + kSegAhead, into the registers just compared
      __builtin_amdgcn_sched_barrier(0);
      load_ck(row_off(i + kSegAhead), kring[U]);
    }
  };
  // rows in groups of kSegAhead so that every ring slot is a constant
  for (int i0 = f0; i0 < r1 && !done; i0 += kSegAhead) {
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
  bad = bad || (int32_t)neg < 0;
}

// Status and outputs of search b from its last normalised row (lane 0 writes).
// Every boundary entry of every table must lie in [0, cap) (cfp_r_limit): the
// E L F entries are checked here, once per search.
template <int SPL>
__device__ __forceinline__ void seg_finish(const SegArgs &a, int b, const uint32_t (&q)[SPL], int64_t o, bool bad,
                                           bool infeasible, SearchResult *__restrict__ res,
                                           const WsHeader *__restrict__ hdr, int64_t *__restrict__ opt,
                                           int32_t *__restrict__ status) {
  const int lane = threadIdx.x & 63;
  const uint32_t IMASK = (1u << a.bits) - 1u, CAP = (1u << (32 - a.bits)) - 1u;
  const int nr = a.E * a.L * a.F;
  for (int x = lane; x < nr; x += 64) bad |= (uint32_t)a.rbound[x] >= CAP;
  // Lowest final state of least value (the least is 0 after normalisation).
  uint32_t pk = kSat;
#pragma unroll
  for (int j = 0; j < SPL; ++j)
    if (lane + 64 * j < a.K) pk = umin(pk, (q[j] << a.bits) | (uint32_t)(lane + 64 * j));
  const uint32_t fin = __builtin_amdgcn_readfirstlane(seg_wave_min(pk));
  bad = __any(bad);
  if (lane == 0) {
    int st = CFP_ST_OK;
    if (bad) st = CFP_ST_BADINPUT;
    else if (infeasible) st = CFP_ST_INFEASIBLE;
    else if ((fin >> a.bits) != 0) st = CFP_ST_OVERFLOW;
    status[b] = st;
    opt[b] = st == CFP_ST_OK ? o + (int64_t)(fin >> a.bits) : INT64_MAX;
    res[b].final_state = st == CFP_ST_OK ? (int32_t)(fin & IMASK) : -1;
    res[b].status = st;
    res[b].final_m = 0;
  }
}

// Whole searches, one wave each.
template <int SPL, int LM, bool EA>
__global__ __launch_bounds__(kSegWaves * 64) void seg_fwd_kernel(SegArgs a, SearchResult *__restrict__ res,
                                                                 const WsHeader *__restrict__ hdr,
                                                                 int64_t *__restrict__ opt,
                                                                 int32_t *__restrict__ status) {
  const int b = blockIdx.x * kSegWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (b >= a.B) return;  // the waves are independent: nothing below waits for another wave
  uint32_t q[SPL];
  int64_t o;
  uint32_t rmax;
  int stop;
  bool bad;
  seg_run<SPL, LM, kSegFull, EA>(a, b, 0, a.N, 0, q, q, o, rmax, stop, bad);
  seg_finish<SPL>(a, b, q, o, bad, rmax == kSat, res, hdr, opt, status);
}

// The final pass of search b (see the top of the file): the chunks' sums of
// row minima, the reruns a chunk whose predecessor met no speculative row
// needs, and the outputs.
template <int SPL, int LM, bool EA>
__device__ __forceinline__ void seg_final(const SegArgs &a, int b, SearchResult *__restrict__ res,
                                          const WsHeader *__restrict__ hdr, int64_t *__restrict__ opt,
                                          int32_t *__restrict__ status) {
  const int lane = threadIdx.x & 63;
  const int N = a.N, K = a.K, P = a.P, CL = a.CL;
  const SegRec *rc = a.rec + (size_t)b * P;
  const int64_t *dk = a.dck + (size_t)b * N;
  int fl = 0;
  for (int p = 0; p < P; ++p) fl |= rc[p].flags;
  int64_t total = dk[min(CL, N) - 1];  // chunk 0 started at the true first row
  bool end_true = true;                // the last speculative row of the previous chunk is the true one
  uint32_t t[SPL];                     // otherwise the true end row of the previous chunk
#pragma unroll
  for (int j = 0; j < SPL; ++j) t[j] = 0;
  for (int p = 1; p < P; ++p) {
    const int r0 = p * CL, r1 = min(r0 + CL, N);
    const int conv = rc[p].conv;
    if (end_true) {  // the fix-up of chunk p started from the true row
      total += rc[p].dfix;
      if (conv >= 0) {
        total += dk[r1 - 1] - dk[conv];
      } else {
        end_true = false;
        const uint32_t *er = a.endrow + ((size_t)b * P + p) * K;
#pragma unroll
        for (int j = 0; j < SPL; ++j) t[j] = er[min(lane + 64 * j, K - 1)];
      }
    } else {  // rerun chunk p from the true row, at least as far as its fix-up went
      uint32_t q[SPL];
      int64_t o;
      uint32_t rmax;
      int stop;
      bool bad;
      seg_run<SPL, LM, kSegRepair, EA>(a, b, r0, r1, conv >= 0 ? conv : r1 - 1, t, q, o, rmax, stop, bad);
      total += o;
      if (stop >= 0) {
        total += dk[r1 - 1] - dk[stop];
        end_true = true;
      } else {
#pragma unroll
        for (int j = 0; j < SPL; ++j) t[j] = q[j];
      }
    }
  }
  uint32_t q[SPL];
  if (end_true) {
    const uint32_t *lr = a.ckrow + ((size_t)b * N + N - 1) * K;
#pragma unroll
    for (int j = 0; j < SPL; ++j) q[j] = lr[min(lane + 64 * j, K - 1)];
  } else {
#pragma unroll
    for (int j = 0; j < SPL; ++j) q[j] = t[j];
  }
  seg_finish<SPL>(a, b, q, total, (fl & 1) != 0, (fl & 2) != 0, res, hdr, opt, status);
}

// The chunk-parallel search in one launch: one workgroup per search, wave p
// for chunk p.  The passes are separated by workgroup barriers (the waves of
// a workgroup share a compute unit, so a barrier also orders their global
// stores and loads): every wave runs its chunk speculatively, waves 1..P-1
// then fix up their chunks, and wave 0 runs the final pass.
template <int SPL, int LM, bool EA>
__global__ __launch_bounds__(64 * kSegMaxP) void seg_chunk_kernel(SegArgs a, SearchResult *__restrict__ res,
                                                                  const WsHeader *__restrict__ hdr,
                                                                  int64_t *__restrict__ opt,
                                                                  int32_t *__restrict__ status) {
  const int b = blockIdx.x, p = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int P = a.P, lane = threadIdx.x & 63;
  const int r0 = p * a.CL, r1 = min(r0 + a.CL, a.N);
  {  // 1. speculative run of chunk p
    uint32_t q[SPL];
    int64_t o;
    uint32_t rmax;
    int stop;
    bool bad;
    seg_run<SPL, LM, kSegSpec, EA>(a, b, r0, r1, 0, q, q, o, rmax, stop, bad);
    bad = __any(bad);
    if (lane == 0) a.rec[(size_t)b * P + p].flags = (bad ? 1 : 0) | (rmax == kSat ? 2 : 0);
  }
  __syncthreads();
  if (p >= 1) {  // 2. fix-up of chunk p from the last speculative row of chunk p-1
    const uint32_t *prev = a.ckrow + ((size_t)b * a.N + r0 - 1) * a.K;
    uint32_t qs[SPL];
#pragma unroll
    for (int x = 0; x < SPL; ++x) qs[x] = prev[min(lane + 64 * x, a.K - 1)];
    uint32_t q[SPL];
    int64_t o;
    uint32_t rmax;
    int stop;
    bool bad;
    seg_run<SPL, LM, kSegFix, EA>(a, b, r0, r1, r0, qs, q, o, rmax, stop, bad);
    const size_t ri = (size_t)b * P + p;
    if (stop < 0) {
      uint32_t *er = a.endrow + ri * a.K;
#pragma unroll
      for (int x = 0; x < SPL; ++x)
        if (lane + 64 * x < a.K) er[lane + 64 * x] = q[x];
    }
    if (lane == 0) {
      a.rec[ri].conv = stop;
      a.rec[ri].dfix = o;
    }
  }
  __syncthreads();
  if (p == 0) seg_final<SPL, LM, EA>(a, b, res, hdr, opt, status);  // 3. final pass
}

bool seg_supported(int k, int n_last, int n_first) {
  return k >= 1 && k <= CFP_MAX_K && n_last >= 1 && n_last <= kSegMaxLF && n_first >= 1 && n_first <= kSegMaxLF;
}

namespace {

// Chunks per search: enough waves for one per SIMD, chunks of at least
// kSegMinRows rows; P = 1 means the one-pass kernel.
struct SegPlan {
  int P, CL;
};

SegPlan seg_plan(int n, int batch) {
  int P = std::min(kSegMaxP, std::max(1, kSegSimds / std::max(1, batch)));
  P = std::min(P, n / kSegMinRows);
  if (P < 2) return SegPlan{1, n};
  const int CL = (n + P - 1) / P;
  return SegPlan{(n + CL - 1) / CL, CL};
}

template <int SPL, int LM, bool EA>
void launch_seg_ea(const SegArgs &a, SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status,
                   hipStream_t st) {
  const dim3 blk(kSegWaves * 64);
  auto grid = [](long waves) { return dim3((unsigned)((waves + kSegWaves - 1) / kSegWaves)); };
  if (a.P < 2) {
    timed_launch(seg_fwd_kernel<SPL, LM, EA>, grid(a.B), blk, 0, st, a, res, hdr, opt, status);
    return;
  }
  timed_launch(seg_chunk_kernel<SPL, LM, EA>, dim3(a.B), dim3(64 * a.P), 0, st, a, res, hdr, opt, status);
}

template <int SPL, int LM>
void launch_seg_spl(const SegArgs &a, bool ea, SearchResult *res, const WsHeader *hdr, int64_t *opt,
                    int32_t *status, hipStream_t st) {
  if (ea) launch_seg_ea<SPL, LM, true>(a, res, hdr, opt, status, st);
  else launch_seg_ea<SPL, LM, false>(a, res, hdr, opt, status, st);
}

template <int LM>
void launch_seg_lm(const SegArgs &a, bool ea, SearchResult *res, const WsHeader *hdr, int64_t *opt,
                   int32_t *status, hipStream_t st) {
  if (a.K <= 64) launch_seg_spl<1, LM>(a, ea, res, hdr, opt, status, st);
  else if (a.K <= 128) launch_seg_spl<2, LM>(a, ea, res, hdr, opt, status, st);
  else if (a.K <= 256) launch_seg_spl<4, LM>(a, ea, res, hdr, opt, status, st);
  else launch_seg_spl<8, LM>(a, ea, res, hdr, opt, status, st);
}

}  // namespace

size_t seg_region_bytes(int n, int k, int batch) {
  const SegPlan c = seg_plan(n, batch);
  if (c.P < 2) return 0;
  size_t off = align_up((size_t)batch * n * k * 4);           // speculative rows
  off += align_up((size_t)batch * n * 8);                     // running sums
  off += align_up((size_t)batch * c.P * sizeof(SegRec));      // chunk records
  off += align_up((size_t)batch * c.P * k * 4);               // fix-up end rows
  return off;
}

bool seg_edges_in_args(int n, int n_tables) { return n <= kSegArgN && n_tables <= 65536; }

hipError_t launch_seg_fwd(const cfp_segment_desc &d, const int32_t *redge_dev, uint8_t *table, uint8_t *region,
                          SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st) {
  SegArgs a{};
  const bool ea = seg_edges_in_args(d.n_segments, d.n_tables);
  if (ea)  // entry 0 is never read as a boundary; keep it a valid table
    for (int i = 1; i < d.n_segments; ++i) a.earg[i >> 1] |= (uint32_t)d.redge[i] << (16 * (i & 1));
  a.cost = d.cost;
  a.rbound = d.rbound;
  a.last = d.last;
  a.first = d.first;
  a.redge = redge_dev;
  a.N = d.n_segments;
  a.K = d.k;
  a.B = d.batch;
  a.E = d.n_tables;
  a.L = d.n_last;
  a.F = d.n_first;
  a.bits = index_bits(d.k);
  a.table = table;
  const SegPlan c = seg_plan(d.n_segments, d.batch);
  a.P = c.P;
  a.CL = c.CL;
  if (c.P >= 2) {
    size_t off = 0;
    a.ckrow = (uint32_t *)(region + off);
    off += align_up((size_t)d.batch * d.n_segments * d.k * 4);
    a.dck = (int64_t *)(region + off);
    off += align_up((size_t)d.batch * d.n_segments * 8);
    a.rec = (SegRec *)(region + off);
    off += align_up((size_t)d.batch * c.P * sizeof(SegRec));
    a.endrow = (uint32_t *)(region + off);
  }
  timer_begin(st);
  if (d.n_last <= 4 && d.n_first <= 4) launch_seg_lm<4>(a, ea, res, hdr, opt, status, st);
  else launch_seg_lm<8>(a, ea, res, hdr, opt, status, st);
  timer_end(st);
  return hipGetLastError();
}

}  // namespace cfp
