// Chunk-parallel forward pass of the chain search for 128 < K <= 512 (Sec. 4.4,
// Eq. T recurrence), for batches whose chains are long.
//
// Parallelism over the chain: as in the K <= 64 form, every chain is cut into
// P chunks that run at once, made exact by rank convergence (Maleki,
// Musuvathi and Mytkowicz, PPoPP 2014): a recurrence started from an
// arbitrary row becomes parallel to the true one after a few steps.
//   1. speculative pass: chunk p starts at its first row (or kCWarm rows
//      before it) from that row's costs alone, writes its argmin rows and, at
//      every quad end, its normalised row and running offset (a checkpoint);
//   2. fix-up pass, chunks p >= 1: start again from the last checkpoint row of
//      chunk p-1 and recompute until the row equals chunk p's checkpoint of the
//      same quad (from there on the speculative rows are the true ones);
//   3. final pass: sum the chunk offsets.  The fix-up of a chunk is valid when
//      the chunk before it ends on a true row; a chunk whose fix-up met no
//      checkpoint has its true end row, from which the next chunk is rerun
//      whole; the chunks after a rerun chunk whose rows met its checkpoints
//      are valid again.  The result is the sequential recurrence's bit for bit.
//
// One workgroup of 512 threads (8 waves) carries four chains (four searches of
// the same chunk: every chain of a launch is at the same row, so all use the
// same table) and all KP states, KP = 256 or 512.  Wave g works for the
// predecessors t = g KP/8 .. (g+1) KP/8 - 1 and lane q for the states
// q KP/64 .. (q+1) KP/64 - 1 of every chain, so every table load of a wave
// reads one row's KP words contiguously.  Per step a thread reads its share of
// the packed words (R_e[t][s] << b) | t of the edge's table (each word serves
// the four chains) in pieces of a few rows, four pieces in flight in their
// own registers (at KP = 256 that is the whole step, loaded a step ahead), and
// the predecessors' values from the previous rows in LDS (broadcast reads).
// A candidate is a saturating add, and one unsigned minimum keeps the value
// and the lowest predecessor.  The eight group minima of a state are combined
// through LDS, after which a thread holds one state of two chains (KP = 256)
// or of all four (KP = 512).
//
// The table stream is what bounds a step: KP^2 words per workgroup and step
// from the cache hierarchy (the step time does not change with the number of
// workgroups), hence four chains per workgroup.  At KP = 512 a batch of at
// most eight searches would leave most compute units idle; there teams of
// four workgroups split the states of each chunk (state-split teams, below).  Chunks are at least 16 rows
// long at KP = 256 and 64 at KP = 512, where runs take longer to become
// parallel (tens of rows on random costs).
//
// Normalisation: x[s] = (m >> b) + c[i][s]; the row is divided into the part
// d = min_s x[s] (summed exactly, per chain) and Q[s] = min(x[s] - d, cap) << b,
// cap = 2^(32-b) - 1.  The best candidate of every state is at most
// R_max << b | t through the row's minimum, so with R below cfp_r_limit a
// capped state never wins; unavailable strategies and padding states take
// x = 2^32 - 1 (capped).
#include <algorithm>
#include <type_traits>

#include "cfp_internal.h"
#include "common.h"

namespace cfp {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kCThreads = 512;          // threads per workgroup
constexpr int kCWaves = kCThreads / 64;
constexpr uint32_t kCX = 0xFFFFFFFFu;   // x of an unavailable or padding state
constexpr int kCMaxChunks = 64;
// Rows a speculative run starts before its chunk.  Starting early makes the
// run parallel to the true one sooner, so the fix-up pass stops earlier, but
// at K = 256 the rows saved there equal the rows added here (measured), so 0.
constexpr int kCWarm = 0;

constexpr int kCG = 4;                  // chains per workgroup (searches of the same chunk)
// Run modes: speculative; fix-up (stops once every chain met a checkpoint);
// repair (a whole chunk from a true row, noting where it meets).
constexpr int kCSpec = 0, kCFix = 1, kCRepair = 2;

template <int KP>
struct CwShape {
  static constexpr int BITS = KP <= 256 ? 8 : 9;   // index bits of a packed word
  static constexpr int PG = KP / kCWaves;           // predecessors per wave
  static constexpr int SPL = KP / 64;               // states per lane in the products
  static constexpr int V4 = SPL / 4;                // 4-word vectors per table row and lane
  static constexpr int ROWS = KP <= 256 ? 8 : 2;    // table rows per piece
  static constexpr int PIECES = PG / ROWS;          // pieces per step
  static constexpr int NB = 4;                      // pieces held in registers
  static constexpr int TPS = kCThreads / KP;        // threads per state after the reduction
  static constexpr int CH = kCG / TPS;              // chains per thread after the reduction
  static constexpr int QS = KP + KP / 8;            // LDS row stride: 4 words of padding after every 32
  static constexpr int MINROWS = KP <= 256 ? 16 : 64;  // least rows per chunk
  static constexpr uint32_t CAP = (1u << (32 - BITS)) - 1u;
  using Arg = typename std::conditional<(KP <= 256), uint8_t, uint16_t>::type;
  static_assert(PIECES % NB == 0 && ROWS % 2 == 0 && SPL % 4 == 0, "piece layout");
};

struct CwRec {
  int64_t dfix;   // fix-up pass: offset sum at the meeting checkpoint, or at the chunk end
  int32_t flags;  // bit 0 a negative cost, bit 1 a row with no available strategy (speculative
                  // pass); bit 2 a wait between the workgroups of a team expired
  int32_t conv;   // fix-up pass: quad of the meeting checkpoint, -1 if none
};

struct CwArgs {
  const int32_t *cost;
  const uint32_t *rpk;  // packed tables [E][KP][KP]
  const int32_t *redge;
  int N, K, B, P, CL, nq;  // CL rows per chunk (a multiple of 4); nq quads of rows
  uint8_t *table;          // argmin entries [B][N][K] (1 byte for KP = 256, 2 for 512)
  CwRec *rec;              // [B][P]
  int64_t *dck;            // speculative offset sum at every checkpoint [B][nq]
  uint32_t *ckrow;         // speculative row at every checkpoint [B][nq][KP]
  uint32_t *endrow;        // fix-up end row of chunks that met no checkpoint [B][P][KP]
  uint64_t *xb;            // state-split teams: exchanged rows [team][slot][chain][KP]
  int32_t *xflag;          // state-split teams: a member gave up waiting [team]
};

template <int KP>
struct CwSmem {
  uint32_t part[kCG][kCWaves][KP];         // partial minima [chain][predecessor group][state]
  uint32_t q[2][kCG][CwShape<KP>::QS];     // rows [buffer][chain][state, padded]
  uint32_t wm[kCWaves][kCG];               // wave minima of the new row, per chain
  int32_t wd[kCWaves][kCG];                // fix-up: the wave found a state off the checkpoint, per chain
};

__device__ __forceinline__ int qpad(int t) { return t + (t >> 5) * 4; }

// min(keep, the partner lane's send): quad_perm partners lane ^ 1 and lane ^ 2;
// the half mirror pairs lane i with lane 7 - i of its eight.
template <int CTRL>
__device__ __forceinline__ uint32_t min_dpp(uint32_t keep, uint32_t send) {
  return umin(keep, (uint32_t)__builtin_amdgcn_mov_dpp((int)send, CTRL, 0xF, 0xF, true));
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;

// Minimum over the 64 lanes of a wave (every lane gets it).
__device__ __forceinline__ uint32_t cw_wave_min(uint32_t x) {
  x = min_dpp<kDppXor1>(x, x);
  x = min_dpp<kDppXor2>(x, x);
  x = min_dpp<kDppHalfMirror>(x, x);
  x = min_dpp<kDppMirror>(x, x);
  const auto h = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  x = umin(h[0], h[1]);
  const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  return umin(r[0], r[1]);
}

// State of the workgroup's chains as seen by one thread.  After the
// reduction thread tid holds, for its state s = tid % KP, the chains
// h TPS + tid / KP, h = 0 .. CH - 1.
template <int KP>
struct CwChains {
  uint32_t x[CwShape<KP>::CH];  // the thread's values of the current row, normalised and shifted
  uint64_t dsum[kCG];   // offset sums since the start row (uniform)
  int conv[kCG];        // fix-up and repair: quad of the meeting checkpoint, -1 before
  uint64_t dconv[kCG];  // fix-up: dsum at that checkpoint
  uint32_t flags[kCG];  // speculative: bit 0 a negative cost, bit 1 a row with no available strategy
};

// Runs rows [r0, r1] of the workgroup's chains (searches bs[c], real where
// valid[c]).  Speculative: the start row is row rs <= r0 from its costs alone
// (rows before r0 warm the run up and write nothing); argmins from row r0 and
// checkpoints are written.  Fix-up: the start row (row r0 - 1) is start[c];
// stops at the first quad end where every real chain has met its checkpoint.
// Repair: like fix-up, run to r1.
template <int KP, int MODE>
__device__ __forceinline__ void cw_run(const CwArgs &a, const int *bs, const bool *valid, int rs, int r0, int r1,
                                       const uint32_t *const *start, CwSmem<KP> &sm, CwChains<KP> &ch) {
  using S = CwShape<KP>;
  using Arg = typename S::Arg;
  constexpr int CH = S::CH, TPS = S::TPS, BITS = S::BITS;
  constexpr bool CHECK = MODE != kCSpec;
  const int tid = threadIdx.x, lane = tid & 63, wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qd = lane, g = wid;  // state group, predecessor group (one wave each)
  const int N = a.N, K = a.K;
  // the thread's state and chains after the reduction
  const int sub = TPS == 1 ? 0 : tid / KP;
  const int ms = tid & (KP - 1);
  const bool sin = ms < K;
  // element h of the thread's chains from an array indexed by chain
  auto pick = [&](const auto &arr, int h) __attribute__((always_inline)) {
    return TPS == 1 ? arr[h] : (sub ? arr[TPS * h + 1] : arr[TPS * h]);
  };
  int hc[CH];  // chain of pair h
  bool hv[CH];
  // A chain's rows start at a wave-uniform address (scalar registers); the
  // thread's state adds one 32-bit byte offset, so no 64-bit address is held
  // per chain in vector registers.
  const int32_t *cbase[CH];
  Arg *tbase[CH];
  uint32_t *ckb[CH];
#pragma unroll
  for (int h = 0; h < CH; ++h) {
    hc[h] = TPS * h + sub;
    const int b = __builtin_amdgcn_readfirstlane(pick(bs, h));
    hv[h] = pick(valid, h);
    cbase[h] = a.cost + (size_t)b * N * K;
    tbase[h] = (Arg *)a.table + (size_t)b * N * K;
    ckb[h] = a.ckrow + (size_t)b * a.nq * KP;
  }
  const uint32_t coff = (uint32_t)min(ms, K - 1) * 4u, toffb = (uint32_t)ms * (uint32_t)sizeof(Arg),
                 koff = (uint32_t)ms * 4u;
  auto cost_at = [&](int h, size_t row, uint32_t off) __attribute__((always_inline)) {
    return *(const uint32_t *)((const char *)(cbase[h] + row * K) + off);
  };
  auto ck_at = [&](int h, size_t q) __attribute__((always_inline)) -> uint32_t & {
    uint32_t off = koff;
    asm volatile("" : "+v"(off));  // (no base + offset pair hoisted out of the loop, where it would spill)
    return *(uint32_t *)((char *)(ckb[h] + q * KP) + off);
  };
  // redge is read-only for the kernel's lifetime: read through the constant
  // address space, so a row's table index is one scalar load.
  const __attribute__((address_space(4))) int32_t *redge_c =
      (const __attribute__((address_space(4))) int32_t *)a.redge;
  auto edge = [&](int row) __attribute__((always_inline)) { return redge_c[row]; };
  const int i0 = MODE == kCSpec ? rs + 1 : r0;

  // Table pieces in flight, [buffer][row in piece][vector]; word offset of the
  // thread's first word within a table.
  const uint32_t toff = (uint32_t)(S::PG * g * KP + S::SPL * qd);
  u32x4 tb[S::NB][S::ROWS][S::V4];
  auto tload = [&](int buf, int piece, int row) __attribute__((always_inline)) {
    const uint32_t *tab = a.rpk + (size_t)edge(row) * KP * KP + toff + piece * S::ROWS * KP;
#pragma unroll
    for (int j = 0; j < S::ROWS; ++j)
#pragma unroll
      for (int v = 0; v < S::V4; ++v) tb[buf][j][v] = *(const u32x4 *)(tab + j * KP + 4 * v);
  };
  // Row minima of every chain from the threads' values: wave minima to LDS,
  // one barrier, then the minimum over the waves (uniform).
  auto row_min = [&](const uint32_t(&x)[CH], uint32_t(&d)[kCG]) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < kCG; ++c) {
      const uint32_t w = cw_wave_min((c % TPS) == sub ? x[c / TPS] : kCX);
      if (lane == 0) sm.wm[wid][c] = w;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < kCG; ++c) {
      uint32_t m = sm.wm[0][c];
#pragma unroll
      for (int w = 1; w < kCWaves; ++w) m = umin(m, sm.wm[w][c]);
      d[c] = __builtin_amdgcn_readfirstlane(m);
    }
  };

  // Start row.
#pragma unroll
  for (int c = 0; c < kCG; ++c) {
    ch.flags[c] = 0;
    ch.conv[c] = -1;
    ch.dconv[c] = 0;
    ch.dsum[c] = 0;
  }
  uint32_t cor[CH];
  if (MODE == kCSpec) {
    uint32_t x[CH], d[kCG];
#pragma unroll
    for (int h = 0; h < CH; ++h) {
      const uint32_t cv = cost_at(h, (size_t)rs, coff);
      cor[h] = cv;
      x[h] = (sin && cv != (uint32_t)CFP_COST_INF) ? cv : kCX;
    }
    row_min(x, d);
#pragma unroll
    for (int c = 0; c < kCG; ++c) {
      if (d[c] == kCX) ch.flags[c] |= 2;
      ch.dsum[c] = d[c];
    }
#pragma unroll
    for (int h = 0; h < CH; ++h) {
      ch.x[h] = umin(x[h] - pick(d, h), S::CAP) << BITS;
      sm.q[0][hc[h]][qpad(ms)] = ch.x[h];
    }
    if (i0 > r1) {  // a run of one row (rs = r0): the start row is its checkpoint
#pragma unroll
      for (int h = 0; h < CH; ++h)
        if (hv[h]) ck_at(h, (size_t)(r0 / 4)) = ch.x[h];
#pragma unroll
      for (int c = 0; c < kCG; ++c)
        if (tid == c && valid[c]) a.dck[(size_t)bs[c] * a.nq + r0 / 4] = (int64_t)ch.dsum[c];
    }
  } else {
#pragma unroll
    for (int h = 0; h < CH; ++h) {
      ch.x[h] = pick(start, h)[ms];
      sm.q[0][hc[h]][qpad(ms)] = ch.x[h];
      cor[h] = 0;
    }
  }
  auto negative_costs = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < kCG; ++c)
      if (__syncthreads_or(((c % TPS) == sub) && (cor[c / TPS] >> 31))) ch.flags[c] |= 1;
  };
  if (i0 > r1) {
    if (MODE == kCSpec) negative_costs();
    return;
  }
#pragma unroll
  for (int k = 0; k < S::NB; ++k) tload(k, k, i0);
  // Costs of the next two rows, [row parity][pair]: step i uses set i - i0 mod 2
  // and reloads it with row i + 2 (the loop runs two rows per turn, so every
  // index is a constant and no register is copied from a load in flight).
  uint32_t cq[2][CH], ckv[CH];
#pragma unroll
  for (int h = 0; h < CH; ++h) {
    cq[0][h] = cost_at(h, (size_t)i0, coff);
    cq[1][h] = cost_at(h, (size_t)min(i0 + 1, r1), coff);
    ckv[h] = 0;
    if (CHECK) ckv[h] = ck_at(h, (size_t)(i0 >> 2));
  }
  __syncthreads();

  // One row i with the previous rows in LDS buffer CUR; returns true when the
  // fix-up pass is done.
  auto step = [&](int i, auto Pc) __attribute__((always_inline)) -> bool {
    constexpr int cur = decltype(Pc)::value, nxt = cur ^ 1;
    uint32_t acc[kCG][S::SPL];
#pragma unroll
    for (int c = 0; c < kCG; ++c)
#pragma unroll
      for (int u = 0; u < S::SPL; ++u) acc[c][u] = kSat;
    const int inext = min(i + 1, r1);
    for (int kk = 0; kk < S::PIECES; kk += S::NB) {
#pragma unroll
      for (int bb = 0; bb < S::NB; ++bb) {
        const int k = kk + bb;
        uint32_t v[kCG][S::ROWS];  // the predecessors' values of this piece, per chain
#pragma unroll
        for (int c = 0; c < kCG; ++c) {
          const uint32_t *qc = &sm.q[cur][c][qpad(S::PG * g + S::ROWS * k)];
          if constexpr (S::ROWS % 4 == 0) {
#pragma unroll
            for (int r4 = 0; r4 < S::ROWS / 4; ++r4) {
              const u32x4 w = *(const u32x4 *)(qc + 4 * r4);
              v[c][4 * r4] = w.x;
              v[c][4 * r4 + 1] = w.y;
              v[c][4 * r4 + 2] = w.z;
              v[c][4 * r4 + 3] = w.w;
            }
          } else {
#pragma unroll
            for (int r2 = 0; r2 < S::ROWS / 2; ++r2) {
              const uint2 w = *(const uint2 *)(qc + 2 * r2);
              v[c][2 * r2] = w.x;
              v[c][2 * r2 + 1] = w.y;
            }
          }
        }
#pragma unroll
        for (int j = 0; j < S::ROWS; j += 2) {
#pragma unroll
          for (int vv = 0; vv < S::V4; ++vv) {
            const u32x4 w = tb[bb][j][vv], y = tb[bb][j + 1][vv];
#pragma unroll
            for (int c = 0; c < kCG; ++c) {
              uint32_t *ac = &acc[c][4 * vv];
              ac[0] = umin(umin(ac[0], sat_add(v[c][j], w.x)), sat_add(v[c][j + 1], y.x));
              ac[1] = umin(umin(ac[1], sat_add(v[c][j], w.y)), sat_add(v[c][j + 1], y.y));
              ac[2] = umin(umin(ac[2], sat_add(v[c][j], w.z)), sat_add(v[c][j + 1], y.z));
              ac[3] = umin(umin(ac[3], sat_add(v[c][j], w.w)), sat_add(v[c][j + 1], y.w));
            }
          }
        }
        // the registers just consumed take the piece NB further on (of this row or the next)
        const int nk = k + S::NB;
        if (nk < S::PIECES) tload(bb, nk, i);
        else tload(bb, nk - S::PIECES, inext);
      }
    }
    // Minima over the eight predecessor groups (one wave each) through LDS.
#pragma unroll
    for (int c = 0; c < kCG; ++c)
#pragma unroll
      for (int vv = 0; vv < S::V4; ++vv) {
        u32x4 pv;
        pv.x = acc[c][4 * vv];
        pv.y = acc[c][4 * vv + 1];
        pv.z = acc[c][4 * vv + 2];
        pv.w = acc[c][4 * vv + 3];
        *(u32x4 *)&sm.part[c][g][S::SPL * qd + 4 * vv] = pv;
      }
    __syncthreads();
    uint32_t m[CH];
#pragma unroll
    for (int h = 0; h < CH; ++h) {
      const int c = hc[h];
      uint32_t v = sm.part[c][0][ms];
#pragma unroll
      for (int w = 1; w < kCWaves; ++w) v = umin(v, sm.part[c][w][ms]);
      m[h] = v;
    }

    // New row: the thread's chains.
    uint32_t x[CH];
#pragma unroll
    for (int h = 0; h < CH; ++h) {
      const uint32_t cv = cq[cur][h];
      if (MODE == kCSpec) {
        cor[h] |= cv;
        asm volatile("" : "+v"(cor[h]));  // kept in its step (not sunk behind the argmin stores)
      }
      x[h] = (sin && cv != (uint32_t)CFP_COST_INF) ? (m[h] >> BITS) + cv : kCX;
      if (sin && hv[h] && i >= r0)
        *(Arg *)((char *)(tbase[h] + (size_t)i * K) + toffb) = (Arg)(m[h] & (KP - 1));
    }
    // The costs of row i + 2, into the registers just read.  The lane offset
    // passes through an empty asm that also takes x[h], so the load cannot be
    // issued before the last read of the old cost: the set keeps its registers
    // and no register copy at the end of the loop waits for a load.
#pragma unroll
    for (int h = 0; h < CH; ++h) {
      uint32_t off = coff;
      asm volatile("" : "+v"(off) : "v"(x[h]));
      cq[cur][h] = cost_at(h, (size_t)min(i + 2, r1), off);
    }
    uint32_t d[kCG];
    row_min(x, d);
#pragma unroll
    for (int c = 0; c < kCG; ++c) {
      if (MODE == kCSpec && d[c] == kCX) ch.flags[c] |= 2;
      ch.dsum[c] += d[c];
    }
#pragma unroll
    for (int h = 0; h < CH; ++h) {
      ch.x[h] = umin(x[h] - pick(d, h), S::CAP) << BITS;
      sm.q[nxt][hc[h]][qpad(ms)] = ch.x[h];
    }
    const bool qend = (i & 3) == 3 || i == r1;
    if (qend) {
      const int q = i >> 2;
      if (MODE == kCSpec && i >= r0) {
#pragma unroll
        for (int h = 0; h < CH; ++h)
          if (hv[h]) ck_at(h, (size_t)q) = ch.x[h];
#pragma unroll
        for (int c = 0; c < kCG; ++c)
          if (tid == c && valid[c]) a.dck[(size_t)bs[c] * a.nq + q] = (int64_t)ch.dsum[c];
      }
      if (CHECK) {
#pragma unroll
        for (int c = 0; c < kCG; ++c) {
          const uint64_t off = __ballot(((c % TPS) == sub) && ch.x[c / TPS] != ckv[c / TPS]);
          if (lane == 0) sm.wd[wid][c] = off != 0;
        }
        if (i < r1) {
#pragma unroll
          for (int h = 0; h < CH; ++h) ckv[h] = ck_at(h, (size_t)(q + 1));
        }
      }
    }
    __syncthreads();
    if (CHECK && qend) {
      const int q = i >> 2;
      bool all = true;
#pragma unroll
      for (int c = 0; c < kCG; ++c) {
        bool same = true;
#pragma unroll
        for (int w = 0; w < kCWaves; ++w) same = same && !sm.wd[w][c];
        if (ch.conv[c] < 0 && same) {
          ch.conv[c] = q;
          ch.dconv[c] = ch.dsum[c];
        }
        all = all && (ch.conv[c] >= 0 || !valid[c]);
      }
      if (MODE == kCFix && all) return true;
    }
    return false;
  };
  for (int i = i0; i <= r1; i += 2) {
    if (step(i, std::integral_constant<int, 0>{})) break;
    if (i + 1 > r1 || step(i + 1, std::integral_constant<int, 1>{})) break;
  }
  if (MODE == kCSpec) negative_costs();
}

// Speculative (MODE kCSpec, grid (ceil(B/kCG), P)) and fix-up (kCFix, grid
// (ceil(B/kCG), P-1)) passes.
template <int KP, int MODE>
__global__ __launch_bounds__(kCThreads, 1) void chain_cw_kernel(CwArgs a) {
  using S = CwShape<KP>;
  __shared__ __align__(16) CwSmem<KP> sm;
  int bs[kCG];
  bool valid[kCG];
#pragma unroll
  for (int c = 0; c < kCG; ++c) {
    const int b = kCG * blockIdx.x + c;
    valid[c] = b < a.B;
    bs[c] = min(b, a.B - 1);
  }
  const int p = MODE == kCFix ? blockIdx.y + 1 : blockIdx.y;
  const int r0 = p * a.CL, r1 = min(r0 + a.CL, a.N) - 1;
  // the speculative run of a chunk after the first starts kCWarm rows early
  const int rs = (MODE == kCSpec && p > 0) ? max(r0 - kCWarm, 0) : r0;
  const uint32_t *start[kCG];
#pragma unroll
  for (int c = 0; c < kCG; ++c) start[c] = a.ckrow + ((size_t)bs[c] * a.nq + (r0 > 0 ? r0 / 4 - 1 : 0)) * KP;
  CwChains<KP> ch;
  cw_run<KP, MODE>(a, bs, valid, rs, r0, r1, start, sm, ch);
  const int tid = threadIdx.x;
  const int sub = S::TPS == 1 ? 0 : tid / KP;
  const int ms = tid & (KP - 1);
  if (MODE == kCSpec) {
#pragma unroll
    for (int c = 0; c < kCG; ++c)
      if (tid == 0 && valid[c]) a.rec[(size_t)bs[c] * a.P + p].flags = (int32_t)ch.flags[c];
  } else {
#pragma unroll
    for (int h = 0; h < S::CH; ++h) {
      const int c0 = S::TPS * h;  // chain c0 + sub
      const bool v = sub ? valid[c0 + S::TPS - 1] : valid[c0];
      const int cv = sub ? ch.conv[c0 + S::TPS - 1] : ch.conv[c0];
      const int bh = sub ? bs[c0 + S::TPS - 1] : bs[c0];
      if (v && cv < 0) a.endrow[((size_t)bh * a.P + p) * KP + ms] = ch.x[h];
    }
#pragma unroll
    for (int c = 0; c < kCG; ++c) {
      if (tid != c || !valid[c]) continue;
      CwRec &r = a.rec[(size_t)bs[c] * a.P + p];
      r.conv = ch.conv[c];
      r.dfix = (int64_t)(ch.conv[c] >= 0 ? ch.dconv[c] : ch.dsum[c]);
    }
  }
}

// ---------------------------------------------------------------------------
// State-split teams (KP = 512 with few searches).  Four chains fill one
// workgroup, so a batch of a few searches leaves most compute units idle while
// each workgroup streams the whole 1 MiB table of every step.  Here a team of
// kXS workgroups carries the four chains of one chunk: part z computes the
// states z W .. z W + W - 1 (W = KP / kXS) of all four chains and so streams
// only those W columns of the table (a quarter).  After each row the parts
// exchange their new values x[s] (before normalisation) as 64-bit words
// (tag << 32) | x through device memory, every part gathers the whole row, and
// all parts normalise it the same way, exactly as one workgroup would.  A
// word's tag is its row (with the top bit set in the fix-up pass), and each
// team has two slots used in turn: a part publishes row i + 2 only after it
// has gathered row i + 1, which every part publishes only after gathering row
// i, so a slot is never rewritten before every part has read it.  Every
// decision that ends a run (the fix-up's meeting test) is taken by each part
// on the whole row, so the parts of a team always run the same rows.  All the
// workgroups of a launch must be resident at once (at most one per compute
// unit); a wait that expires marks the team, and the search ends with
// CFP_ST_TIMEOUT.

constexpr int kXS = 4;                      // workgroups per team
constexpr int kXW = 512 / kXS;              // states per part
constexpr int kXSpin = 1 << 20;             // poll rounds before a part gives up
constexpr uint32_t kXFixTag = 0x80000000u;  // tag bit of the fix-up pass
constexpr int kXMaxGroups = 2;              // teams are used for at most 2 x 4 searches
constexpr int kXQW = kXW + kXW / 8;         // padded LDS words of one part's states

struct CxSmem {
  uint32_t part[kCG][kCWaves][kXW];      // partial minima [chain][predecessor group][state of the part]
  uint32_t q[2][kCG][CwShape<512>::QS];  // whole rows [buffer][chain][state, padded]
  uint32_t wm[kCWaves];                  // wave minima of the new row (waves 2c and 2c+1 hold chain c)
  int32_t wd[kCWaves];                   // fix-up: the wave found a state off the checkpoint
  int32_t abort;                         // a wait expired, or another part of the team gave up
};

// A thread's view after the products: chain c = tid / W... of the four chains
// (two waves each), state sl = tid % W of every part.
struct CxChains {
  uint32_t q[kXS];      // the chain's normalised, shifted values at states sl + z W, z = 0 .. kXS - 1
  uint64_t dsum[kCG];   // offset sums since the start row (uniform)
  int conv[kCG];        // fix-up: quad of the meeting checkpoint, -1 before
  uint64_t dconv[kCG];  // fix-up: dsum at that checkpoint
  uint32_t flags[kCG];  // speculative: bit 1 a row with no available strategy
  uint32_t neg;         // speculative: OR of the thread's costs (bit 31: a negative cost)
  bool aborted;
};

// Runs rows [r0, r1] of the team's chains in part z.  Speculative: the start
// row r0 comes from its costs alone; argmins from row r0 + 1 and checkpoints
// are written.  Fix-up: the start row (row r0 - 1) is start[c]; stops at the
// first quad end where every real chain has met its checkpoint.
// Element idx (wave-uniform) of a four-element array, by selects rather than a
// dynamic index (which would move the array to scratch memory).
template <typename T>
__device__ __forceinline__ T sel4(const T (&v)[4], int idx) {
  return idx == 0 ? v[0] : idx == 1 ? v[1] : idx == 2 ? v[2] : v[3];
}

template <int MODE>
__device__ __forceinline__ void cx_run(const CwArgs &a, int z, int team, int grp, int r0, int r1, CxSmem &sm,
                                       CxChains &ch) {
  constexpr int KP = 512;
  using S = CwShape<KP>;
  constexpr int BITS = S::BITS;
  constexpr uint32_t CAP = S::CAP;
  constexpr int PG = S::PG;  // predecessors per wave
  constexpr uint32_t PASS = MODE == kCFix ? kXFixTag : 0u;
  const int tid = threadIdx.x, lane = tid & 63, wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = wid >> 1;          // the thread's chain after the products (uniform in the wave)
  const int sl = tid & (kXW - 1);  // the thread's state within each part
  const int N = a.N, K = a.K;
  const int b = min(kCG * grp + c, a.B - 1);  // chains past the batch repeat the last search and write nothing
  const bool hv = kCG * grp + c < a.B;
  const int s = z * kXW + sl;      // the thread's own state (computed by this part)
  const bool sin = s < K;
  const int qsl = qpad(sl);        // LDS index of state zz W + sl: zz kXQW + qsl
  const int32_t *cbase = a.cost + (size_t)b * N * K;
  uint16_t *tbase = (uint16_t *)a.table + (size_t)b * N * K;
  uint32_t *ckb = a.ckrow + (size_t)b * a.nq * KP;
  uint64_t *xbt = a.xb + (size_t)team * 2 * kCG * KP;
  const uint32_t coff = (uint32_t)min(s, K - 1) * 4u;
  auto cost_at = [&](size_t row, uint32_t off) __attribute__((always_inline)) {
    return *(const uint32_t *)((const char *)(cbase + row * K) + off);
  };
  const __attribute__((address_space(4))) int32_t *redge_c =
      (const __attribute__((address_space(4))) int32_t *)a.redge;

  // The step's table words of the wave's predecessors t = PG wid + j, states
  // z W + 2 lane and z W + 2 lane + 1: one 8-byte load per predecessor, the
  // whole step held in registers and loaded one step ahead.
  const uint32_t toff = (uint32_t)(PG * wid * KP + z * kXW + 2 * lane) * 4u;
  uint2 tb[PG];
  auto tload = [&](int j, int row, uint32_t dep) __attribute__((always_inline)) {
    const char *tab = (const char *)(a.rpk + (size_t)redge_c[row] * KP * KP);
    // The lane offset is formed by an asm add that also takes a value computed
    // from the register's last read: the load is issued after that read, and
    // no offset is hoisted out of the loop (64 of them would not fit).  One
    // 32-bit offset from the scalar base.
    uint32_t off;
    asm volatile("v_add_u32 %0, %1, %2" : "=v"(off) : "n"(j * KP * 4), "v"(toff), "v"(dep));
    tb[j] = *(const uint2 *)(tab + off);
  };

  // Publishes the part's value x of row i and gathers the other parts' values
  // of the same chain and state sl; returns the row's values in xv.
  auto exchange = [&](int i, uint32_t x, uint32_t (&xv)[kXS]) __attribute__((always_inline)) {
    const uint32_t tag = (uint32_t)i | PASS;
    char *slot = (char *)(xbt + (size_t)((i & 1) * kCG + c) * KP);  // uniform
    auto word = [&](int zz) __attribute__((always_inline)) {
      uint32_t off = (uint32_t)sl * 8u;
      asm volatile("" : "+v"(off));
      return (uint64_t *)(slot + off + (uint32_t)(zz * kXW * 8));
    };
    __hip_atomic_store(word(z), ((uint64_t)tag << 32) | x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    bool ok[kXS];
#pragma unroll
    for (int zz = 0; zz < kXS; ++zz) {
      ok[zz] = zz == z || ch.aborted;
      xv[zz] = zz == z ? x : kCX;
    }
    int spins = 0;
    // Every word is polled at once (the own word too), and twice, a few hundred
    // cycles apart: a word that lands just after the first poll left is seen
    // by the second rather than a whole round trip later.
    auto take = [&](const uint64_t (&w)[kXS]) __attribute__((always_inline)) {
      bool all = true;
#pragma unroll
      for (int zz = 0; zz < kXS; ++zz) {
        if (!ok[zz] && (uint32_t)(w[zz] >> 32) == tag) {
          xv[zz] = (uint32_t)w[zz];
          ok[zz] = true;
        }
        all = all && ok[zz];
      }
      return all;
    };
    while (true) {
      uint64_t w[kXS], w2[kXS];
#pragma unroll
      for (int zz = 0; zz < kXS; ++zz) w[zz] = __hip_atomic_load(word(zz), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __builtin_amdgcn_s_sleep(4);
#pragma unroll
      for (int zz = 0; zz < kXS; ++zz) w2[zz] = __hip_atomic_load(word(zz), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (take(w) || take(w2)) break;
      ++spins;
      // another part gave up (checked every 256 polls), or this wait expired
      if (spins > kXSpin ||
          ((spins & 255) == 0 && __hip_atomic_load(&a.xflag[team], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))) {
        sm.abort = 1;
        __hip_atomic_store(&a.xflag[team], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  };

  // Row minima of the four chains from the gathered values, the offsets, and
  // the normalised row into LDS buffer NXT.  Ends with every thread past a barrier.
  auto finish_row = [&](const uint32_t (&xv)[kXS], int nxt, uint32_t (&d)[kCG]) __attribute__((always_inline)) {
    uint32_t m = umin(umin(xv[0], xv[1]), umin(xv[2], xv[3]));
    m = cw_wave_min(m);
    if (lane == 0) sm.wm[wid] = m;
    __syncthreads();
#pragma unroll
    for (int cc = 0; cc < kCG; ++cc) d[cc] = __builtin_amdgcn_readfirstlane(umin(sm.wm[2 * cc], sm.wm[2 * cc + 1]));
    ch.aborted = sm.abort != 0;
    const uint32_t dc = sel4(d, c);
#pragma unroll
    for (int zz = 0; zz < kXS; ++zz) {
      ch.q[zz] = umin(xv[zz] - dc, CAP) << BITS;
      sm.q[nxt][c][zz * kXQW + qsl] = ch.q[zz];
    }
#pragma unroll
    for (int cc = 0; cc < kCG; ++cc) ch.dsum[cc] += d[cc];
  };

#pragma unroll
  for (int cc = 0; cc < kCG; ++cc) {
    ch.flags[cc] = 0;
    ch.conv[cc] = -1;
    ch.dconv[cc] = 0;
    ch.dsum[cc] = 0;
  }
  ch.neg = 0;
  ch.aborted = false;
  if (tid == 0) sm.abort = 0;
  __syncthreads();
  int i0;
  if (MODE == kCSpec) {
    // start row r0 from its costs alone
    const uint32_t cv = cost_at((size_t)r0, coff);
    ch.neg = cv;
    uint32_t xv[kXS], d[kCG];
    exchange(r0, (sin && cv != (uint32_t)CFP_COST_INF) ? cv : kCX, xv);
    finish_row(xv, 0, d);
#pragma unroll
    for (int cc = 0; cc < kCG; ++cc)
      if (d[cc] == kCX) ch.flags[cc] |= 2;
    if (r0 == r1) {  // a run of one row: the start row is its checkpoint
      if (hv) ckb[(size_t)(r0 / 4) * KP + s] = sel4(ch.q, z);
      if (z == 0 && sl == 0 && (wid & 1) == 0 && hv) a.dck[(size_t)b * a.nq + r0 / 4] = (int64_t)sel4(ch.dsum, c);
    }
    i0 = r0 + 1;
  } else {
    // the start row: chunk p - 1's last checkpoint (row r0 - 1, a quad end)
    const uint32_t *start = ckb + (size_t)(r0 / 4 - 1) * KP;
#pragma unroll
    for (int zz = 0; zz < kXS; ++zz) {
      ch.q[zz] = start[zz * kXW + sl];
      sm.q[0][c][zz * kXQW + qsl] = ch.q[zz];
    }
    i0 = r0;
  }
  __syncthreads();
  if (i0 > r1 || ch.aborted) return;

#pragma unroll
  for (int j = 0; j < PG; ++j) tload(j, i0, 0);
  // the own state's costs of the next two rows: step i uses set (i - i0) mod 2
  uint32_t cq[2], ckv[kXS];
  cq[0] = cost_at((size_t)i0, coff);
  cq[1] = cost_at((size_t)min(i0 + 1, r1), coff);
#pragma unroll
  for (int zz = 0; zz < kXS; ++zz) ckv[zz] = MODE == kCFix ? ckb[(size_t)(i0 >> 2) * KP + zz * kXW + sl] : 0u;

  // One row i with the previous row in LDS buffer CUR; returns true when the
  // run is over (fix-up: every chain met; any mode: the team gave up).
  auto step = [&](int i, auto Pc) __attribute__((always_inline)) -> bool {
    constexpr int cur = decltype(Pc)::value, nxt = cur ^ 1;
    const int inext = min(i + 1, r1);
    uint32_t acc[kCG][2];
#pragma unroll
    for (int cc = 0; cc < kCG; ++cc) acc[cc][0] = acc[cc][1] = kSat;
#pragma unroll
    for (int j4 = 0; j4 < PG / 4; ++j4) {
      u32x4 v[kCG];  // predecessors PG wid + 4 j4 .. + 3 of every chain (LDS broadcast reads)
#pragma unroll
      for (int cc = 0; cc < kCG; ++cc) v[cc] = *(const u32x4 *)&sm.q[cur][cc][qpad(PG * wid + 4 * j4)];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint2 w0 = tb[4 * j4 + 2 * h], w1 = tb[4 * j4 + 2 * h + 1];
#pragma unroll
        for (int cc = 0; cc < kCG; ++cc) {
          const uint32_t va = h ? v[cc].z : v[cc].x, vb = h ? v[cc].w : v[cc].y;
          acc[cc][0] = umin(umin(acc[cc][0], sat_add(va, w0.x)), sat_add(vb, w1.x));
          acc[cc][1] = umin(umin(acc[cc][1], sat_add(va, w0.y)), sat_add(vb, w1.y));
        }
      }
      // the four registers just read take the next row's words
#pragma unroll
      for (int u = 0; u < 4; ++u) tload(4 * j4 + u, inext, acc[u][u & 1]);
    }
    // minima over the eight predecessor groups through LDS
#pragma unroll
    for (int cc = 0; cc < kCG; ++cc) *(uint2 *)&sm.part[cc][wid][2 * lane] = make_uint2(acc[cc][0], acc[cc][1]);
    __syncthreads();
    uint32_t mv = sm.part[c][0][sl];
#pragma unroll
    for (int g = 1; g < kCWaves; ++g) mv = umin(mv, sm.part[c][g][sl]);
    const uint32_t cv = cq[cur];
    if (MODE == kCSpec) {
      ch.neg |= cv;
      asm volatile("" : "+v"(ch.neg));
    }
    const uint32_t x = (sin && cv != (uint32_t)CFP_COST_INF) ? (mv >> BITS) + cv : kCX;
    if (sin && hv) *(uint16_t *)((char *)(tbase + (size_t)i * K) + (uint32_t)s * 2u) = (uint16_t)(mv & (KP - 1));
    {
      uint32_t off = coff;
      asm volatile("" : "+v"(off) : "v"(x));
      cq[cur] = cost_at((size_t)min(i + 2, r1), off);
    }
    uint32_t xv[kXS], d[kCG];
    exchange(i, x, xv);
    finish_row(xv, nxt, d);
    if (MODE == kCSpec) {
#pragma unroll
      for (int cc = 0; cc < kCG; ++cc)
        if (d[cc] == kCX) ch.flags[cc] |= 2;
    }
    const bool qend = (i & 3) == 3 || i == r1;
    if (qend) {
      const int q = i >> 2;
      if (MODE == kCSpec) {
        if (hv) ckb[(size_t)q * KP + s] = sel4(ch.q, z);
        if (z == 0 && sl == 0 && (wid & 1) == 0 && hv) a.dck[(size_t)b * a.nq + q] = (int64_t)sel4(ch.dsum, c);
      } else {
        bool off = false;
#pragma unroll
        for (int zz = 0; zz < kXS; ++zz) off = off || ch.q[zz] != ckv[zz];
        const uint64_t bal = __ballot(off);
        if (lane == 0) sm.wd[wid] = bal != 0;
        if (i < r1) {
#pragma unroll
          for (int zz = 0; zz < kXS; ++zz) ckv[zz] = ckb[(size_t)(q + 1) * KP + zz * kXW + sl];
        }
      }
    }
    __syncthreads();
    if (MODE == kCFix && qend) {
      const int q = i >> 2;
      bool all = true;
#pragma unroll
      for (int cc = 0; cc < kCG; ++cc) {
        const bool same = !sm.wd[2 * cc] && !sm.wd[2 * cc + 1];
        if (ch.conv[cc] < 0 && same) {
          ch.conv[cc] = q;
          ch.dconv[cc] = ch.dsum[cc];
        }
        all = all && (ch.conv[cc] >= 0 || kCG * grp + cc >= a.B);
      }
      if (all) return true;
    }
    return ch.aborted;
  };
  for (int i = i0; i <= r1; i += 2) {
    if (step(i, std::integral_constant<int, 0>{})) break;
    if (i + 1 > r1 || step(i + 1, std::integral_constant<int, 1>{})) break;
  }
}

// Clears the exchange slots and abort flags of every team and the flags of
// every chunk record before a call's passes.
__global__ void chain_cx_init_kernel(uint64_t *xb, size_t nxb, int32_t *xflag, int teams, CwRec *rec, int nrec) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t x = (size_t)blockIdx.x * blockDim.x + threadIdx.x; x < nxb; x += stride) xb[x] = ~0ull;
  for (size_t x = (size_t)blockIdx.x * blockDim.x + threadIdx.x; x < (size_t)teams; x += stride) xflag[x] = 0;
  for (size_t x = (size_t)blockIdx.x * blockDim.x + threadIdx.x; x < (size_t)nrec; x += stride) rec[x].flags = 0;
}

// Speculative (MODE kCSpec, grid (kXS, ceil(B/kCG), P)) and fix-up (kCFix,
// grid (kXS, ceil(B/kCG), P-1)) passes of the state-split teams; part z is
// blockIdx.x, so consecutive workgroups form a team.
template <int MODE>
__global__ __launch_bounds__(kCThreads, 1) void chain_cx_kernel(CwArgs a) {
  __shared__ __align__(16) CxSmem sm;
  const int z = blockIdx.x, grp = blockIdx.y;
  const int p = MODE == kCFix ? blockIdx.z + 1 : blockIdx.z;
  const int team = grp * a.P + p;
  const int r0 = p * a.CL, r1 = min(r0 + a.CL, a.N) - 1;
  CxChains ch;
  cx_run<MODE>(a, z, team, grp, r0, r1, sm, ch);
  const int tid = threadIdx.x, wid = __builtin_amdgcn_readfirstlane(tid >> 6), c = wid >> 1, sl = tid & (kXW - 1);
  // flags of the run, one word per chain, ORed over the parts
  int32_t fl[kCG];
#pragma unroll
  for (int cc = 0; cc < kCG; ++cc) {
    fl[cc] = (MODE == kCSpec ? (int32_t)ch.flags[cc] : 0) | (ch.aborted ? 4 : 0);
    if (MODE == kCSpec && __syncthreads_or(c == cc && (ch.neg >> 31))) fl[cc] |= 1;
  }
#pragma unroll
  for (int cc = 0; cc < kCG; ++cc)
    if (tid == cc && kCG * grp + cc < a.B && fl[cc]) atomicOr(&a.rec[(size_t)(kCG * grp + cc) * a.P + p].flags, fl[cc]);
  if (MODE == kCFix) {
    const int s = z * kXW + sl, bc = kCG * grp + c;
    if (bc < a.B && sel4(ch.conv, c) < 0) a.endrow[((size_t)bc * a.P + p) * 512 + s] = sel4(ch.q, z);
#pragma unroll
    for (int cc = 0; cc < kCG; ++cc) {
      if (z != 0 || tid != cc || kCG * grp + cc >= a.B) continue;
      CwRec &r = a.rec[(size_t)(kCG * grp + cc) * a.P + p];
      r.conv = ch.conv[cc];
      r.dfix = (int64_t)(ch.conv[cc] >= 0 ? ch.dconv[cc] : ch.dsum[cc]);
    }
  }
}

// Final pass, one workgroup per search: the chunk offsets, the reruns after
// chunks whose fix-up met no checkpoint, and the lowest optimal final state.
template <int KP>
__global__ __launch_bounds__(kCThreads, 1) void chain_cw_final_kernel(CwArgs a, const WsHeader *__restrict__ hdr,
                                                                       SearchResult *__restrict__ res,
                                                                       int64_t *__restrict__ opt,
                                                                       int32_t *__restrict__ status) {
  using S = CwShape<KP>;
  __shared__ __align__(16) CwSmem<KP> sm;
  __shared__ uint32_t s_row[KP];  // a true end row of the last chunk accounted
  __shared__ int s_q, s_flags;
  __shared__ int64_t s_sum;
  __shared__ uint32_t s_fin[kCWaves];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int b = blockIdx.x, P = a.P;
  const int ms = tid & (KP - 1);
  const int64_t *dk = a.dck + (size_t)b * a.nq;
  const CwRec *rec = a.rec + (size_t)b * P;
  auto endq = [&](int p) __attribute__((always_inline)) { return (min((p + 1) * a.CL, a.N) - 1) >> 2; };
  if (wid == 0) {
    int fl = lane < P ? rec[lane].flags : 0;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) fl |= __shfl_xor(fl, off, 64);
    if (lane == 0) s_flags = fl;
  }
  // Chunk 0 runs from the true first row.  Invariant at the top of the loop:
  // chunks < p are accounted in `total`; if spec_true, the speculative end row
  // of chunk p-1 is a true row (so the fix-up of chunk p is valid), otherwise
  // s_row holds the true end row of chunk p-1.
  int64_t total = dk[endq(0)];
  bool spec_true = true;
  int p = 1;
  while (p < P) {
    if (spec_true) {
      // With wave 0: the first chunk q >= p whose fix-up met no checkpoint, and
      // the offsets of chunks p .. q (chunk q's fix-up ran from a true row to its end).
      if (wid == 0) {
        const int pl = p + lane;
        const bool in = pl < P;
        CwRec r{};
        if (in) r = rec[pl];
        const uint64_t nc = __ballot(in && r.conv < 0);
        const int q = nc ? p + __ffsll((long long)nc) - 1 : P;
        int64_t delta = 0;
        if (in && pl < q) delta = r.dfix + dk[endq(pl)] - dk[r.conv];
        else if (in && pl == q) delta = r.dfix;
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) delta += __shfl_xor(delta, off, 64);
        if (lane == 0) {
          s_q = q;
          s_sum = delta;
        }
      }
      __syncthreads();
      const int q = s_q;
      total += s_sum;
      if (q >= P) break;
      if (tid < KP) s_row[tid] = a.endrow[((size_t)b * P + q) * KP + tid];
      spec_true = false;
      p = q + 1;
      __syncthreads();
    } else {
      // Rerun chunk p whole from the true row in s_row; its rows are then
      // true, and so is its speculative end row if the rerun met a checkpoint.
      int bs[kCG];
      bool valid[kCG];
      const uint32_t *start[kCG];
#pragma unroll
      for (int c = 0; c < kCG; ++c) {
        bs[c] = b;
        valid[c] = c == 0;  // the other chains duplicate it and are discarded
        start[c] = s_row;
      }
      CwChains<KP> ch;
      const int r0 = p * a.CL, r1 = min(r0 + a.CL, a.N) - 1;
      cw_run<KP, kCRepair>(a, bs, valid, r0, r0, r1, start, sm, ch);
      total += (int64_t)ch.dsum[0];
      spec_true = ch.conv[0] >= 0;
      __syncthreads();  // every thread has read s_row
      if (!spec_true && tid < KP) s_row[tid] = ch.x[0];  // chain 0 of state tid is the thread's first
      __syncthreads();
      ++p;
    }
  }
  // The final row has minimum 0: the lowest state at the minimum.
  const uint32_t xv = spec_true ? a.ckrow[((size_t)b * a.nq + a.nq - 1) * KP + ms] : s_row[ms];
  const uint32_t pk = cw_wave_min((tid < KP && ms < a.K) ? (xv | (uint32_t)ms) : kSat);
  if (lane == 0) s_fin[wid] = pk;
  __syncthreads();
  if (tid == 0) {
    uint32_t fin = s_fin[0];
    for (int w = 1; w < kCWaves; ++w) fin = umin(fin, s_fin[w]);
    const int fl = s_flags;
    int st = CFP_ST_OK;
    if (fl & 4) st = CFP_ST_TIMEOUT;
    else if ((fl & 1) || hdr->rflag) st = CFP_ST_BADINPUT;
    else if (fl & 2) st = CFP_ST_INFEASIBLE;
    else if ((fin >> S::BITS) != 0) st = CFP_ST_OVERFLOW;
    status[b] = st;
    opt[b] = st == CFP_ST_OK ? total : INT64_MAX;
    res[b].final_state = st == CFP_ST_OK ? (int32_t)(fin & (KP - 1)) : -1;
    res[b].status = st;
    res[b].final_m = 0;
  }
}

struct CwPlan {
  int KP, P, CL, nq;
  int S;  // workgroups per chunk and group of four searches: 1, or kXS for state-split teams
};

// Compute units of the current device (256 if the query fails, as on a host
// without one, so that workspace sizes do not depend on it there).
int cw_device_cus() {
  static int cus = -1;
  if (cus < 0) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cus = n;
  }
  return cus;
}

CwPlan cw_plan(int n, int k, int batch) {
  CwPlan c{0, 0, 0, 0, 1};
  if (k <= 128 || k > 512) return c;
  const int kp = k <= 256 ? 256 : 512;
  const int minrows = kp == 256 ? CwShape<256>::MINROWS : CwShape<512>::MINROWS;
  if (n < 2 * minrows) return c;
  const int groups = (batch + kCG - 1) / kCG;
  // K > 256 with at most two groups of four searches: state-split teams, every
  // workgroup resident on its own compute unit.
  const int cus = cw_device_cus();
  const bool team = kp == 512 && groups <= kXMaxGroups && cus / (kXS * groups) >= 2;
  int P = team ? cus / (kXS * groups) : std::max(2, (256 + groups - 1) / groups);  // about one workgroup per CU
  P = std::min(P, std::min(kCMaxChunks, n / minrows));
  int CL = ((n + P - 1) / P + 3) & ~3;
  P = (n + CL - 1) / CL;
  if (P < 2) return c;
  c.KP = kp;
  c.P = P;
  c.CL = CL;
  c.nq = (n + 3) / 4;
  c.S = team ? kXS : 1;
  return c;
}

template <int KP>
void launch_cw_kp(const CwArgs &a, int groups, const WsHeader *hdr, SearchResult *res, int64_t *opt,
                  int32_t *status, hipStream_t st) {
  timer_begin(st);
  timed_launch(chain_cw_kernel<KP, kCSpec>, dim3(groups, a.P), dim3(kCThreads), 0, st, a);
  timer_end(st);
  hipLaunchKernelGGL((chain_cw_kernel<KP, kCFix>), dim3(groups, a.P - 1), dim3(kCThreads), 0, st, a);
  hipLaunchKernelGGL(chain_cw_final_kernel<KP>, dim3(a.B), dim3(kCThreads), 0, st, a, hdr, res, opt, status);
}

void launch_cx(const CwArgs &a, int groups, const WsHeader *hdr, SearchResult *res, int64_t *opt, int32_t *status,
               hipStream_t st) {
  const int teams = groups * a.P;
  hipLaunchKernelGGL(chain_cx_init_kernel, dim3(64), dim3(256), 0, st, a.xb, (size_t)teams * 2 * kCG * 512, a.xflag,
                     teams, a.rec, a.B * a.P);
  timer_begin(st);
  timed_launch(chain_cx_kernel<kCSpec>, dim3(kXS, groups, a.P), dim3(kCThreads), 0, st, a);
  timer_end(st);
  hipLaunchKernelGGL(chain_cx_kernel<kCFix>, dim3(kXS, groups, a.P - 1), dim3(kCThreads), 0, st, a);
  hipLaunchKernelGGL(chain_cw_final_kernel<512>, dim3(a.B), dim3(kCThreads), 0, st, a, hdr, res, opt, status);
}

}  // namespace

bool chain_cw_supported(int n, int k, int batch) { return cw_plan(n, k, batch).P >= 2; }

size_t cw_region_bytes(int n, int k, int n_tables, int batch) {
  const CwPlan c = cw_plan(n, k, batch);
  if (c.P < 2) return 0;
  const size_t kp = c.KP;
  size_t off = align_up((size_t)n_tables * kp * kp * 4);
  off += align_up((size_t)batch * c.P * sizeof(CwRec));
  off += align_up((size_t)batch * c.nq * 8);
  off += align_up((size_t)batch * c.nq * kp * 4);
  off += align_up((size_t)batch * c.P * kp * 4);
  if (c.S > 1) {
    const size_t teams = (size_t)((batch + kCG - 1) / kCG) * c.P;
    off += align_up(teams * 2 * kCG * kp * 8);
    off += align_up(teams * 4);
  }
  return off;
}

hipError_t launch_chain_cw(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *region, uint8_t *table,
                           SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st) {
  const CwPlan c = cw_plan(d.n_blocks, d.k, d.batch);
  const size_t kp = c.KP;
  CwArgs a;
  a.cost = d.cost;
  a.redge = redge_dev;
  a.N = d.n_blocks;
  a.K = d.k;
  a.B = d.batch;
  a.P = c.P;
  a.CL = c.CL;
  a.nq = c.nq;
  a.table = table;
  size_t off = 0;
  uint32_t *rpk = (uint32_t *)(region + off);
  a.rpk = rpk;
  off += align_up((size_t)d.n_tables * kp * kp * 4);
  a.rec = (CwRec *)(region + off);
  off += align_up((size_t)d.batch * c.P * sizeof(CwRec));
  a.dck = (int64_t *)(region + off);
  off += align_up((size_t)d.batch * c.nq * 8);
  a.ckrow = (uint32_t *)(region + off);
  off += align_up((size_t)d.batch * c.nq * kp * 4);
  a.endrow = (uint32_t *)(region + off);
  off += align_up((size_t)d.batch * c.P * kp * 4);
  const int groups = (d.batch + kCG - 1) / kCG;
  a.xb = nullptr;
  a.xflag = nullptr;
  if (c.S > 1) {
    a.xb = (uint64_t *)(region + off);
    off += align_up((size_t)groups * c.P * 2 * kCG * kp * 8);
    a.xflag = (int32_t *)(region + off);
  }
  launch_pack_rtab(d.rtab, d.n_tables, d.k, (int)kp, kp == 256 ? CwShape<256>::BITS : CwShape<512>::BITS, rpk, st,
                   cfp_r_limit(CFP_V_CHAIN, d.k), const_cast<WsHeader *>(hdr));
  if (c.S > 1) launch_cx(a, groups, hdr, res, opt, status, st);
  else if (kp == 256) launch_cw_kp<256>(a, groups, hdr, res, opt, status, st);
  else launch_cw_kp<512>(a, groups, hdr, res, opt, status, st);
  return hipGetLastError();
}

}  // namespace cfp
