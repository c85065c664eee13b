// Chunk-parallel forward pass of the chain search for 128 < K <= 256 (Sec. 4.4,
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
//   3. final pass: sum the chunk offsets; a chunk whose fix-up met no
//      checkpoint has its true end row, and the rest of the chain is rerun from
//      it.  The result is the sequential recurrence's bit for bit.
//
// One workgroup of 512 threads carries four chains (four searches of the same
// chunk: every chain of a launch is at the same row, so all use the same
// table) and all KP = 256 states.  Thread tid = 64 g + q (wave g) works for the
// states 4q .. 4q+3 of every chain over the predecessors t = 32 g .. 32 g + 31,
// so every table load of a wave reads 1 KiB of one row contiguously.  Per
// step it reads its 32 x 4 packed words (R_e[t][s] << 8) | t of the edge's
// table from the cache-resident array (each word serves the four chains), in
// four pieces of eight rows, each loaded one step ahead into its own registers,
// and the predecessors' values from the previous rows in LDS (broadcast
// reads).  A candidate is a saturating add, and one unsigned minimum keeps the
// value and the lowest predecessor.  The eight group minima of a state are
// combined through LDS, after which thread tid holds state tid % 256 of chains
// tid / 256 and 2 + tid / 256.
//
// The table stream is what bounds a step: 256 KiB per workgroup and step,
// which one CU takes in from L2 at about 14 bytes per clock (measured: the
// step time does not change with the number of workgroups), hence four chains
// per workgroup rather than two.
//
// Normalisation: x[s] = (m >> 8) + c[i][s]; the row is divided into the part
// d = min_s x[s] (summed exactly, per chain) and Q[s] = min(x[s] - d, cap) << 8,
// cap = 2^24 - 1.  The best candidate of every state is at most R_max << 8 | t
// through the row's minimum, so with R below cfp_r_limit a capped state never
// wins; unavailable strategies and padding states take x = 2^32 - 1 (capped).
#include <algorithm>

#include "cfp_internal.h"
#include "common.h"

namespace cfp {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kCKP = 256;               // states (padded)
constexpr int kCBits = 8;               // index bits of a packed word
constexpr int kCThreads = 512;          // threads per workgroup
constexpr int kCWaves = kCThreads / 64;
constexpr int kCRows = 8;               // predecessor rows per streamed piece
constexpr int kCPieces = 4;             // pieces per step (32 predecessors per thread)
constexpr int kCQS = kCKP + kCKP / 8;   // LDS row stride: 4 words of padding after every 32
constexpr uint32_t kCCap = (1u << (32 - kCBits)) - 1u;
constexpr uint32_t kCX = 0xFFFFFFFFu;   // x of an unavailable or padding state
constexpr int kCMaxChunks = 64;
constexpr int kCMinRows = 16;           // least rows per chunk
// Rows a speculative run starts before its chunk.  Starting early makes the
// run parallel to the true one sooner, so the fix-up pass stops earlier, but
// at K = 256 the rows saved there equal the rows added here (measured), so 0.
constexpr int kCWarm = 0;

constexpr int kCG = 4;                  // chains per workgroup (searches of the same chunk)
constexpr int kCH = kCG / 2;            // chains per thread after the reduce-scatter
constexpr int kCSpec = 0, kCFix = 1, kCRepair = 2;

struct CwRec {
  int64_t dfix;   // fix-up pass: offset sum at the meeting checkpoint, or at the chunk end
  int32_t flags;  // speculative pass: bit 0 a negative cost, bit 1 a row with no available strategy
  int32_t conv;   // fix-up pass: quad of the meeting checkpoint, -1 if none
};

struct CwArgs {
  const int32_t *cost;
  const uint32_t *rpk;  // packed tables [E][KP][KP]
  const int32_t *redge;
  int N, K, B, P, CL, nq;  // CL rows per chunk (a multiple of 4); nq quads of rows
  uint8_t *table;          // argmin entries [B][N][K]
  CwRec *rec;              // [B][P]
  int64_t *dck;            // speculative offset sum at every checkpoint [B][nq]
  uint32_t *ckrow;         // speculative row at every checkpoint [B][nq][KP]
  uint32_t *endrow;        // fix-up end row of chunks that met no checkpoint [B][P][KP]
};

struct CwSmem {
  uint32_t part[kCG][kCWaves][kCKP];  // partial minima [chain][predecessor group][state]
  uint32_t q[2][kCG][kCQS];   // rows [buffer][chain][state, padded]
  uint32_t wm[kCWaves][kCG];  // wave minima of the new row, per chain
  int32_t wd[kCWaves][kCG];   // fix-up: the wave found a state off the checkpoint, per chain
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
// reduction a thread holds, for its state s = tid % 256, the chains 2h + f2,
// h = 0 .. kCG/2 - 1 (f2 = tid / 256).
template <int MODE>
struct CwChains {
  uint32_t x[kCH];      // the thread's values of the current row, normalised and shifted
  uint64_t dsum[kCG];   // offset sums since the start row (uniform)
  int conv[kCG];        // fix-up: quad of the meeting checkpoint, -1 before
  uint64_t dconv[kCG];  // fix-up: dsum at that checkpoint
  uint32_t flags[kCG];  // speculative: bit 0 a negative cost, bit 1 a row with no available strategy
};

// Runs rows [r0, r1] of the workgroup's chains (searches bs[c], real where
// valid[c]).  Speculative: the start row is row rs <= r0 from its costs alone
// (rows before r0 warm the run up and write nothing); argmins from row r0 and
// checkpoints are written.  Fix-up: the start row (row r0 - 1)
// is start[c]; stops at the first quad end where every real chain has met its
// checkpoint.  Repair: like fix-up without checkpoints.
template <int MODE>
__device__ __forceinline__ void cw_run(const CwArgs &a, const int *bs, const bool *valid, int rs, int r0, int r1,
                                       const uint32_t *const *start, CwSmem &sm, CwChains<MODE> &ch) {
  const int tid = threadIdx.x, lane = tid & 63, wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qd = lane, g = wid;  // state quad, predecessor group (one wave each)
  const int N = a.N, K = a.K;
  // the thread's state and chains after the reduction
  const bool f2 = tid >= kCKP;
  const int ms = tid & (kCKP - 1);
  const bool sin = ms < K;
  int hc[kCH];  // chain of pair h
  bool hv[kCH];
  const int32_t *cbase[kCH];
  uint8_t *tbase[kCH];
  uint32_t *ckb[kCH];
#pragma unroll
  for (int h = 0; h < kCH; ++h) {
    hc[h] = 2 * h + (f2 ? 1 : 0);
    const int b = f2 ? bs[2 * h + 1] : bs[2 * h];
    hv[h] = f2 ? valid[2 * h + 1] : valid[2 * h];
    cbase[h] = a.cost + (size_t)b * N * K + min(ms, K - 1);
    tbase[h] = a.table + (size_t)b * N * K + ms;
    ckb[h] = a.ckrow + (size_t)b * a.nq * kCKP + ms;
  }
  // redge is read-only for the kernel's lifetime: read through the constant
  // address space, so a row's table index is one scalar load.
  const __attribute__((address_space(4))) int32_t *redge_c =
      (const __attribute__((address_space(4))) int32_t *)a.redge;
  auto edge = [&](int row) __attribute__((always_inline)) { return redge_c[row]; };
  const int i0 = MODE == kCSpec ? rs + 1 : r0;

  // Table pieces of the next row, [piece][row in piece]; word offset of the
  // thread's first word within a table.
  const uint32_t toff = (uint32_t)(32 * g * kCKP + 4 * qd);
  u32x4 tb[kCPieces][kCRows];
  auto tload = [&](int piece, int row) __attribute__((always_inline)) {
    const uint32_t *tab = a.rpk + (size_t)edge(row) * kCKP * kCKP + toff + piece * kCRows * kCKP;
#pragma unroll
    for (int j = 0; j < kCRows; ++j) tb[piece][j] = *(const u32x4 *)(tab + j * kCKP);
  };
  // Row minima of every chain from the threads' values: wave minima to LDS,
  // one barrier, then the minimum over the waves (uniform).
  auto row_min = [&](const uint32_t(&x)[kCH], uint32_t(&d)[kCG]) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < kCG; ++c) {
      const uint32_t w = cw_wave_min(((c & 1) == (f2 ? 1 : 0)) ? x[c >> 1] : kCX);
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
  uint32_t cor[kCH];
  if (MODE == kCSpec) {
    uint32_t x[kCH], d[kCG];
#pragma unroll
    for (int h = 0; h < kCH; ++h) {
      const uint32_t cv = (uint32_t)cbase[h][(size_t)rs * K];
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
    for (int h = 0; h < kCH; ++h) {
      ch.x[h] = umin(x[h] - (f2 ? d[2 * h + 1] : d[2 * h]), kCCap) << kCBits;
      sm.q[0][hc[h]][qpad(ms)] = ch.x[h];
    }
    if (i0 > r1) {  // a run of one row (rs = r0): the start row is its checkpoint
#pragma unroll
      for (int h = 0; h < kCH; ++h)
        if (hv[h]) ckb[h][(size_t)(r0 / 4) * kCKP] = ch.x[h];
#pragma unroll
      for (int c = 0; c < kCG; ++c)
        if (tid == c && valid[c]) a.dck[(size_t)bs[c] * a.nq + r0 / 4] = (int64_t)ch.dsum[c];
    }
  } else {
#pragma unroll
    for (int h = 0; h < kCH; ++h) {
      ch.x[h] = (f2 ? start[2 * h + 1] : start[2 * h])[ms];
      sm.q[0][hc[h]][qpad(ms)] = ch.x[h];
      cor[h] = 0;
    }
  }
  auto negative_costs = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < kCG; ++c)
      if (__syncthreads_or(((c & 1) == (f2 ? 1 : 0)) && (cor[c >> 1] >> 31))) ch.flags[c] |= 1;
  };
  if (i0 > r1) {
    if (MODE == kCSpec) negative_costs();
    return;
  }
#pragma unroll
  for (int k = 0; k < kCPieces; ++k) tload(k, i0);
  // Costs of the next two rows, [row parity][pair]: step i uses set i - i0 mod 2
  // and reloads it with row i + 2 (the loop runs two rows per turn, so every
  // index is a constant and no register is copied from a load in flight).
  uint32_t cq[2][kCH], ckv[kCH];
#pragma unroll
  for (int h = 0; h < kCH; ++h) {
    cq[0][h] = (uint32_t)cbase[h][(size_t)i0 * K];
    cq[1][h] = (uint32_t)cbase[h][(size_t)min(i0 + 1, r1) * K];
    ckv[h] = 0;
    if (MODE == kCFix) ckv[h] = ckb[h][(size_t)(i0 >> 2) * kCKP];
  }
  __syncthreads();

  // One row i with the previous rows in LDS buffer CUR; returns true when the
  // fix-up pass is done.
  auto step = [&](int i, auto Pc) __attribute__((always_inline)) -> bool {
    constexpr int cur = decltype(Pc)::value, nxt = cur ^ 1;
    uint32_t acc[kCG][4];
#pragma unroll
    for (int c = 0; c < kCG; ++c)
#pragma unroll
      for (int u = 0; u < 4; ++u) acc[c][u] = kSat;
    const int inext = min(i + 1, r1);
#pragma unroll
    for (int k = 0; k < kCPieces; ++k) {
      uint32_t v[kCG][kCRows];  // the predecessors' values of this piece, per chain
#pragma unroll
      for (int c = 0; c < kCG; ++c) {
        const uint32_t *qc = &sm.q[cur][c][qpad(32 * g) + 8 * k];
        const u32x4 lo = *(const u32x4 *)qc, hi = *(const u32x4 *)(qc + 4);
        v[c][0] = lo.x; v[c][1] = lo.y; v[c][2] = lo.z; v[c][3] = lo.w;
        v[c][4] = hi.x; v[c][5] = hi.y; v[c][6] = hi.z; v[c][7] = hi.w;
      }
#pragma unroll
      for (int j = 0; j < kCRows; j += 2) {
        const u32x4 w = tb[k][j], y = tb[k][j + 1];
#pragma unroll
        for (int c = 0; c < kCG; ++c) {
          acc[c][0] = umin(umin(acc[c][0], sat_add(v[c][j], w.x)), sat_add(v[c][j + 1], y.x));
          acc[c][1] = umin(umin(acc[c][1], sat_add(v[c][j], w.y)), sat_add(v[c][j + 1], y.y));
          acc[c][2] = umin(umin(acc[c][2], sat_add(v[c][j], w.z)), sat_add(v[c][j + 1], y.z));
          acc[c][3] = umin(umin(acc[c][3], sat_add(v[c][j], w.w)), sat_add(v[c][j + 1], y.w));
        }
      }
      tload(k, inext);  // this piece of the next row into the registers just consumed
    }
    // Minima over the eight predecessor groups (one wave each) through LDS.
#pragma unroll
    for (int c = 0; c < kCG; ++c) {
      u32x4 pv;
      pv.x = acc[c][0];
      pv.y = acc[c][1];
      pv.z = acc[c][2];
      pv.w = acc[c][3];
      *(u32x4 *)&sm.part[c][g][4 * qd] = pv;
    }
    __syncthreads();
    uint32_t m[kCH];
#pragma unroll
    for (int h = 0; h < kCH; ++h) {
      const int c = 2 * h + (f2 ? 1 : 0);
      uint32_t v = sm.part[c][0][ms];
#pragma unroll
      for (int w = 1; w < kCWaves; ++w) v = umin(v, sm.part[c][w][ms]);
      m[h] = v;
    }

    // New row: the thread's pairs.
    uint32_t x[kCH];
#pragma unroll
    for (int h = 0; h < kCH; ++h) {
      const uint32_t cv = cq[cur][h];
      cq[cur][h] = (uint32_t)cbase[h][(size_t)min(i + 2, r1) * K];
      if (MODE == kCSpec) cor[h] |= cv;
      x[h] = (sin && cv != (uint32_t)CFP_COST_INF) ? (m[h] >> kCBits) + cv : kCX;
      if (sin && hv[h] && i >= r0) tbase[h][(size_t)i * K] = (uint8_t)(m[h] & (kCKP - 1));
    }
    uint32_t d[kCG];
    row_min(x, d);
#pragma unroll
    for (int c = 0; c < kCG; ++c) {
      if (MODE == kCSpec && d[c] == kCX) ch.flags[c] |= 2;
      ch.dsum[c] += d[c];
    }
#pragma unroll
    for (int h = 0; h < kCH; ++h) {
      ch.x[h] = umin(x[h] - (f2 ? d[2 * h + 1] : d[2 * h]), kCCap) << kCBits;
      sm.q[nxt][hc[h]][qpad(ms)] = ch.x[h];
    }
    const bool qend = (i & 3) == 3 || i == r1;
    if (qend) {
      const int q = i >> 2;
      if (MODE == kCSpec && i >= r0) {
#pragma unroll
        for (int h = 0; h < kCH; ++h)
          if (hv[h]) ckb[h][(size_t)q * kCKP] = ch.x[h];
#pragma unroll
        for (int c = 0; c < kCG; ++c)
          if (tid == c && valid[c]) a.dck[(size_t)bs[c] * a.nq + q] = (int64_t)ch.dsum[c];
      }
      if (MODE == kCFix) {
#pragma unroll
        for (int c = 0; c < kCG; ++c) {
          const uint64_t off = __ballot(((c & 1) == (f2 ? 1 : 0)) && ch.x[c >> 1] != ckv[c >> 1]);
          if (lane == 0) sm.wd[wid][c] = off != 0;
        }
        if (i < r1) {
#pragma unroll
          for (int h = 0; h < kCH; ++h) ckv[h] = ckb[h][(size_t)(q + 1) * kCKP];
        }
      }
    }
    __syncthreads();
    if (MODE == kCFix && qend) {
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
      if (all) return true;
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
template <int MODE>
__global__ __launch_bounds__(kCThreads, 1) void chain_cw_kernel(CwArgs a) {
  __shared__ __align__(16) CwSmem sm;
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
  for (int c = 0; c < kCG; ++c) start[c] = a.ckrow + ((size_t)bs[c] * a.nq + (r0 > 0 ? r0 / 4 - 1 : 0)) * kCKP;
  CwChains<MODE> ch;
  cw_run<MODE>(a, bs, valid, rs, r0, r1, start, sm, ch);
  const int tid = threadIdx.x;
  const bool f2 = tid >= kCKP;
  const int ms = tid & (kCKP - 1);
  if (MODE == kCSpec) {
#pragma unroll
    for (int c = 0; c < kCG; ++c)
      if (tid == 0 && valid[c]) a.rec[(size_t)bs[c] * a.P + p].flags = (int32_t)ch.flags[c];
  } else {
#pragma unroll
    for (int h = 0; h < kCH; ++h) {
      const int c = 2 * h + (f2 ? 1 : 0);
      const bool v = f2 ? valid[2 * h + 1] : valid[2 * h];
      const int b = f2 ? bs[2 * h + 1] : bs[2 * h];
      const int cv = f2 ? ch.conv[2 * h + 1] : ch.conv[2 * h];
      (void)c;
      if (v && cv < 0) a.endrow[((size_t)b * a.P + p) * kCKP + ms] = ch.x[h];
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

// Final pass, one workgroup per search: chunk offsets, the rerun of the chain
// after a chunk whose fix-up met no checkpoint, and the lowest optimal final
// state.
__global__ __launch_bounds__(kCThreads, 1) void chain_cw_final_kernel(CwArgs a, const WsHeader *__restrict__ hdr,
                                                                       SearchResult *__restrict__ res,
                                                                       int64_t *__restrict__ opt,
                                                                       int32_t *__restrict__ status) {
  __shared__ __align__(16) CwSmem sm;
  __shared__ int s_q, s_flags;
  __shared__ int64_t s_dtot;
  __shared__ uint32_t s_fin[kCWaves];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int b = blockIdx.x, P = a.P;
  if (wid == 0) {
    const bool in = lane < P;
    CwRec r{};
    if (in) r = a.rec[(size_t)b * P + lane];
    const int endq = (min((lane + 1) * a.CL, a.N) - 1) >> 2;  // quad of the chunk's last row
    const uint64_t nc = __ballot(in && lane >= 1 && r.conv < 0);
    const int q = nc ? __ffsll((long long)nc) - 1 : P;  // first chunk whose fix-up met no checkpoint
    int64_t delta = 0;
    if (in && lane < q) {
      const int64_t *dk = a.dck + (size_t)b * a.nq;
      delta = lane == 0 ? dk[endq] : r.dfix + dk[endq] - dk[r.conv];
    } else if (lane == q) {
      delta = r.dfix;  // its fix-up started from the true row and ran to the end
    }
    int fl = in ? r.flags : 0;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      delta += __shfl_xor(delta, off, 64);
      fl |= __shfl_xor(fl, off, 64);
    }
    if (lane == 0) {
      s_q = q;
      s_dtot = delta;
      s_flags = fl;
    }
  }
  __syncthreads();
  const int q = s_q;
  uint64_t drep = 0;
  // the final row: chain 0 of state s is held by thread s, as pair 0
  const bool f2 = tid >= kCKP;
  const int ms = tid & (kCKP - 1);
  uint32_t xv;
  if (q < P - 1) {
    // Rerun the chain after chunk q from its true end row (the other chains
    // duplicate it and are discarded).
    const uint32_t *st = a.endrow + ((size_t)b * P + q) * kCKP;
    int bs[kCG];
    bool valid[kCG];
    const uint32_t *start[kCG];
#pragma unroll
    for (int c = 0; c < kCG; ++c) {
      bs[c] = b;
      valid[c] = c == 0;
      start[c] = st;
    }
    CwChains<kCRepair> ch;
    cw_run<kCRepair>(a, bs, valid, (q + 1) * a.CL, (q + 1) * a.CL, a.N - 1, start, sm, ch);
    xv = ch.x[0];
    drep = ch.dsum[0];
  } else if (q == P - 1) {
    xv = a.endrow[((size_t)b * P + q) * kCKP + ms];
  } else {
    xv = a.ckrow[((size_t)b * a.nq + a.nq - 1) * kCKP + ms];
  }
  // The final row has minimum 0: the lowest state at the minimum.
  const uint32_t pk = cw_wave_min((!f2 && ms < a.K) ? (xv | (uint32_t)ms) : kSat);
  if (lane == 0) s_fin[wid] = pk;
  __syncthreads();
  if (tid == 0) {
    uint32_t fin = s_fin[0];
    for (int w = 1; w < kCWaves; ++w) fin = umin(fin, s_fin[w]);
    const int fl = s_flags;
    int st = CFP_ST_OK;
    if ((fl & 1) || hdr->rflag) st = CFP_ST_BADINPUT;
    else if (fl & 2) st = CFP_ST_INFEASIBLE;
    else if ((fin >> kCBits) != 0) st = CFP_ST_OVERFLOW;
    status[b] = st;
    opt[b] = st == CFP_ST_OK ? s_dtot + (int64_t)drep : INT64_MAX;
    res[b].final_state = st == CFP_ST_OK ? (int32_t)(fin & (kCKP - 1)) : -1;
    res[b].status = st;
    res[b].final_m = 0;
  }
}

struct CwPlan {
  int P, CL, nq;
};

CwPlan cw_plan(int n, int k, int batch) {
  CwPlan c{0, 0, 0};
  if (k <= 128 || k > kCKP || n < 2 * kCMinRows) return c;
  const int groups = (batch + kCG - 1) / kCG;
  int P = std::max(2, (256 + groups - 1) / groups);  // about one workgroup per compute unit
  P = std::min(P, std::min(kCMaxChunks, n / kCMinRows));
  int CL = ((n + P - 1) / P + 3) & ~3;
  P = (n + CL - 1) / CL;
  if (P < 2) return c;
  c.P = P;
  c.CL = CL;
  c.nq = (n + 3) / 4;
  return c;
}

}  // namespace

bool chain_cw_supported(int n, int k, int batch) { return cw_plan(n, k, batch).P >= 2; }

size_t cw_region_bytes(int n, int k, int n_tables, int batch) {
  const CwPlan c = cw_plan(n, k, batch);
  if (c.P < 2) return 0;
  size_t off = align_up((size_t)n_tables * kCKP * kCKP * 4);
  off += align_up((size_t)batch * c.P * sizeof(CwRec));
  off += align_up((size_t)batch * c.nq * 8);
  off += align_up((size_t)batch * c.nq * kCKP * 4);
  off += align_up((size_t)batch * c.P * kCKP * 4);
  return off;
}

hipError_t launch_chain_cw(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *region, uint8_t *table,
                           SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st) {
  const CwPlan c = cw_plan(d.n_blocks, d.k, d.batch);
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
  off += align_up((size_t)d.n_tables * kCKP * kCKP * 4);
  a.rec = (CwRec *)(region + off);
  off += align_up((size_t)d.batch * c.P * sizeof(CwRec));
  a.dck = (int64_t *)(region + off);
  off += align_up((size_t)d.batch * c.nq * 8);
  a.ckrow = (uint32_t *)(region + off);
  off += align_up((size_t)d.batch * c.nq * kCKP * 4);
  a.endrow = (uint32_t *)(region + off);
  launch_pack_rtab(d.rtab, d.n_tables, d.k, kCKP, kCBits, rpk, st, cfp_r_limit(CFP_V_CHAIN, d.k),
                   const_cast<WsHeader *>(hdr));
  const int groups = (d.batch + kCG - 1) / kCG;
  timer_begin(st);
  timed_launch(chain_cw_kernel<kCSpec>, dim3(groups, c.P), dim3(kCThreads), 0, st, a);
  timer_end(st);
  hipLaunchKernelGGL(chain_cw_kernel<kCFix>, dim3(groups, c.P - 1), dim3(kCThreads), 0, st, a);
  hipLaunchKernelGGL(chain_cw_final_kernel, dim3(d.batch), dim3(kCThreads), 0, st, a, hdr, res, opt, status);
  return hipGetLastError();
}

}  // namespace cfp
