// Chunk-parallel forward pass of the chain search for 128 < K <= 256 (Sec. 4.4,
// Eq. T recurrence), for batches whose chains are long.
//
// Parallelism over the chain: as in the K <= 64 form, every chain is cut into
// P chunks that run at once, made exact by rank convergence (Maleki,
// Musuvathi and Mytkowicz, PPoPP 2014): a recurrence started from an
// arbitrary row becomes parallel to the true one after a few steps.
//   1. speculative pass: chunk p starts at its first row from that row's costs
//      alone, writes its argmin rows and, at every quad end, its normalised row
//      and running offset (a checkpoint);
//   2. fix-up pass, chunks p >= 1: start again from the last checkpoint row of
//      chunk p-1 and recompute until the row equals chunk p's checkpoint of the
//      same quad (from there on the speculative rows are the true ones);
//   3. final pass: sum the chunk offsets; a chunk whose fix-up met no
//      checkpoint has its true end row, and the rest of the chain is rerun from
//      it.  The result is the sequential recurrence's bit for bit.
//
// One workgroup of 512 threads carries two chains (two searches of the same
// chunk: every chain of a launch is at the same row, so both use the same
// table) and all KP = 256 states.  Thread tid = 8 q + g works for the states
// 4q .. 4q+3 of both chains over the predecessors t = 32 g .. 32 g + 31.  Per
// step it reads its 32 x 4 packed words (R_e[t][s] << 8) | t of the edge's
// table from the cache-resident array (each word serves both chains), in four
// pieces of eight rows, each loaded one step ahead into its own registers, and
// the predecessors' values from the previous row in LDS (broadcast reads).  A
// candidate is a saturating add, and one unsigned minimum keeps the value and
// the lowest predecessor.  The eight group minima of a state are combined by a
// reduce-scatter over the eight lanes of the state quad (two quad_perm steps and
// a half-mirror step, lanes of the upper half holding the complementary
// indices), after which lane g holds chain g / 4, state 4q + ((g ^ 3 (g / 4)) % 4).
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
  uint32_t q[2][2][kCQS];  // rows [buffer][chain][state, padded]
  uint32_t wm[kCWaves][2];  // wave minima of the new row, per chain
  int32_t wd[kCWaves][2];   // fix-up: the wave found a state off the checkpoint, per chain
};

__device__ __forceinline__ int qpad(int t) { return t + (t >> 5) * 4; }

// min(keep, lane ^ 1's send) and min(keep, lane ^ 2's send) by quad_perm; the
// half mirror pairs lane i with lane 7 - i of its eight.
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

// Runs rows [r0 (+1 in the speculative pass), r1] of the two chains b0, b1 of
// the workgroup (real: valid0, valid1).  Speculative: the start row is row r0
// from its costs; checkpoints are written.  Fix-up: the start row (row r0 - 1)
// is start[c]; stops at the first quad end where both chains meet their
// checkpoints.  Repair: like fix-up without checkpoints.
template <int MODE>
struct CwChains {
  uint32_t x;          // the lane's (chain, state) value of the current row, normalised and shifted
  uint64_t dsum[2];    // offset sums since the start row
  int conv[2];         // fix-up: quad of the meeting checkpoint, -1 before
  uint64_t dconv[2];   // fix-up: dsum at that checkpoint
  uint32_t flags[2];   // speculative, per chain: bit 0 a negative cost, bit 1 a row with no available strategy
};

template <int MODE>
__device__ __forceinline__ void cw_run(const CwArgs &a, int b0, int b1, bool valid0, bool valid1, int r0, int r1,
                                       const uint32_t *start0, const uint32_t *start1, CwSmem &sm,
                                       CwChains<MODE> &ch) {
  const int tid = threadIdx.x, lane = tid & 63, wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qd = tid >> 3, g = tid & 7;  // state quad, predecessor group
  const int N = a.N, K = a.K;
  // the lane's (chain, state) after the reduce-scatter
  const int mc = g >> 2;
  const int ms = 4 * qd + ((g ^ (mc ? 3 : 0)) & 3);
  const int mb = mc ? b1 : b0;
  const bool mvalid = mc ? valid1 : valid0;
  const bool sin = ms < K;
  const int32_t *cbase = a.cost + (size_t)mb * N * K + min(ms, K - 1);
  uint8_t *tbase = a.table + (size_t)mb * N * K + ms;
  auto edge = [&](int row) __attribute__((always_inline)) {
    return __builtin_amdgcn_readfirstlane(a.redge[row]);
  };
  const int i0 = MODE == kCSpec ? r0 + 1 : r0;

  // Table pieces of the next row, [piece][row in piece]; word offset of the
  // thread's first word within a table.
  const uint32_t toff = (uint32_t)(32 * g * kCKP + 4 * qd);
  u32x4 tb[kCPieces][kCRows];
  auto tload = [&](int piece, int row) __attribute__((always_inline)) {
    const uint32_t *tab = a.rpk + (size_t)edge(row) * kCKP * kCKP + toff + piece * kCRows * kCKP;
#pragma unroll
    for (int j = 0; j < kCRows; ++j) tb[piece][j] = *(const u32x4 *)(tab + j * kCKP);
  };

  // Start row.
  ch.flags[0] = ch.flags[1] = 0;
  ch.conv[0] = ch.conv[1] = -1;
  ch.dconv[0] = ch.dconv[1] = 0;
  uint32_t cor = 0;
  int cur = 0;
  if (MODE == kCSpec) {
    const uint32_t cv = (uint32_t)cbase[(size_t)r0 * K];
    cor = cv;
    const uint32_t x = (sin && cv != (uint32_t)CFP_COST_INF) ? cv : kCX;
    const uint32_t w0 = cw_wave_min(mc == 0 ? x : kCX), w1 = cw_wave_min(mc == 1 ? x : kCX);
    if (lane == 0) {
      sm.wm[wid][0] = w0;
      sm.wm[wid][1] = w1;
    }
    __syncthreads();
    uint32_t d0 = sm.wm[0][0], d1 = sm.wm[0][1];
#pragma unroll
    for (int w = 1; w < kCWaves; ++w) {
      d0 = umin(d0, sm.wm[w][0]);
      d1 = umin(d1, sm.wm[w][1]);
    }
    const uint32_t d = mc ? d1 : d0;
    if (d0 == kCX) ch.flags[0] |= 2;
    if (d1 == kCX) ch.flags[1] |= 2;
    ch.x = umin(x - d, kCCap) << kCBits;
    ch.dsum[0] = d0;
    ch.dsum[1] = d1;
    sm.q[0][mc][qpad(ms)] = ch.x;
    if (i0 > r1 && mvalid) {  // a run of one row: the start row is its checkpoint
      (a.ckrow + ((size_t)mb * a.nq + r0 / 4) * kCKP)[ms] = ch.x;
      if (tid == 0 && valid0) a.dck[(size_t)b0 * a.nq + r0 / 4] = (int64_t)ch.dsum[0];
      if (tid == 4 && valid1) a.dck[(size_t)b1 * a.nq + r0 / 4] = (int64_t)ch.dsum[1];
    }
  } else {
    ch.x = (mc ? start1 : start0)[ms];
    ch.dsum[0] = ch.dsum[1] = 0;
    sm.q[0][mc][qpad(ms)] = ch.x;
  }
  auto negative_costs = [&]() __attribute__((always_inline)) {
    if (__syncthreads_or(mc == 0 && (cor >> 31))) ch.flags[0] |= 1;
    if (__syncthreads_or(mc == 1 && (cor >> 31))) ch.flags[1] |= 1;
  };
  if (i0 > r1) {  // nothing to compute (a run of one row)
    if (MODE == kCSpec) negative_costs();
    return;
  }
#pragma unroll
  for (int k = 0; k < kCPieces; ++k) tload(k, i0);
  uint32_t c1 = (uint32_t)cbase[(size_t)i0 * K];                 // cost of the next row
  uint32_t c2 = (uint32_t)cbase[(size_t)min(i0 + 1, r1) * K];    // and of the one after
  uint32_t ckv = 0;
  if (MODE == kCFix) ckv = (mc ? a.ckrow + (size_t)b1 * a.nq * kCKP : a.ckrow + (size_t)b0 * a.nq * kCKP)[(size_t)(i0 >> 2) * kCKP + ms];
  __syncthreads();

  for (int i = i0; i <= r1; ++i) {
    const int nxt = cur ^ 1;
    const uint32_t *q0 = &sm.q[cur][0][qpad(32 * g)];
    const uint32_t *q1 = &sm.q[cur][1][qpad(32 * g)];
    uint32_t acc[2][4];
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int u = 0; u < 4; ++u) acc[c][u] = kSat;
    const int inext = min(i + 1, r1);
#pragma unroll
    for (int k = 0; k < kCPieces; ++k) {
      const u32x4 qa0 = *(const u32x4 *)(q0 + 8 * k), qb0 = *(const u32x4 *)(q0 + 8 * k + 4);
      const u32x4 qa1 = *(const u32x4 *)(q1 + 8 * k), qb1 = *(const u32x4 *)(q1 + 8 * k + 4);
      const uint32_t v0[8] = {qa0.x, qa0.y, qa0.z, qa0.w, qb0.x, qb0.y, qb0.z, qb0.w};
      const uint32_t v1[8] = {qa1.x, qa1.y, qa1.z, qa1.w, qb1.x, qb1.y, qb1.z, qb1.w};
#pragma unroll
      for (int j = 0; j < kCRows; j += 2) {
        const u32x4 w = tb[k][j], y = tb[k][j + 1];
        acc[0][0] = umin(umin(acc[0][0], sat_add(v0[j], w.x)), sat_add(v0[j + 1], y.x));
        acc[0][1] = umin(umin(acc[0][1], sat_add(v0[j], w.y)), sat_add(v0[j + 1], y.y));
        acc[0][2] = umin(umin(acc[0][2], sat_add(v0[j], w.z)), sat_add(v0[j + 1], y.z));
        acc[0][3] = umin(umin(acc[0][3], sat_add(v0[j], w.w)), sat_add(v0[j + 1], y.w));
        acc[1][0] = umin(umin(acc[1][0], sat_add(v1[j], w.x)), sat_add(v1[j + 1], y.x));
        acc[1][1] = umin(umin(acc[1][1], sat_add(v1[j], w.y)), sat_add(v1[j + 1], y.y));
        acc[1][2] = umin(umin(acc[1][2], sat_add(v1[j], w.z)), sat_add(v1[j + 1], y.z));
        acc[1][3] = umin(umin(acc[1][3], sat_add(v1[j], w.w)), sat_add(v1[j + 1], y.w));
      }
      tload(k, inext);  // this piece of the next row into the registers just consumed
    }
    // Reduce-scatter over the eight groups of the state quad.  Value index
    // k = 4 c + u; lane bits (b2 b1 b0) = g.  Step 1 keeps k0 = b0 ^ b2, step 2
    // k1 = b1 ^ b2 (quad_perm partners), step 3 k2 = b2 (half mirror: lane
    // 7 - g, whose kept k0, k1 equal this lane's).
    const bool f0 = ((g ^ (g >> 2)) & 1) != 0, f1 = (((g >> 1) ^ (g >> 2)) & 1) != 0, f2 = (g >> 2) != 0;
    uint32_t r1v[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {  // pairs (k, k + 1) with k = 2p: k0 = 0 / 1
      const uint32_t lo = acc[p >> 1][(p & 1) * 2], hi = acc[p >> 1][(p & 1) * 2 + 1];
      r1v[p] = min_dpp<kDppXor1>(f0 ? hi : lo, f0 ? lo : hi);
    }
    uint32_t r2v[2];
#pragma unroll
    for (int p = 0; p < 2; ++p) r2v[p] = min_dpp<kDppXor2>(f1 ? r1v[2 * p + 1] : r1v[2 * p], f1 ? r1v[2 * p] : r1v[2 * p + 1]);
    const uint32_t m = min_dpp<kDppHalfMirror>(f2 ? r2v[1] : r2v[0], f2 ? r2v[0] : r2v[1]);

    // New row: the lane's (chain, state).
    const uint32_t cv = c1;
    c1 = c2;
    c2 = (uint32_t)cbase[(size_t)min(i + 2, r1) * K];
    if (MODE == kCSpec) cor |= cv;
    const bool avail = sin && cv != (uint32_t)CFP_COST_INF;
    const uint32_t x = avail ? (m >> kCBits) + cv : kCX;
    if (sin && mvalid) tbase[(size_t)i * K] = (uint8_t)(m & (kCKP - 1));
    const uint32_t w0 = cw_wave_min(mc == 0 ? x : kCX), w1 = cw_wave_min(mc == 1 ? x : kCX);
    if (lane == 0) {
      sm.wm[wid][0] = w0;
      sm.wm[wid][1] = w1;
    }
    __syncthreads();
    uint32_t d0 = sm.wm[0][0], d1 = sm.wm[0][1];
#pragma unroll
    for (int w = 1; w < kCWaves; ++w) {
      d0 = umin(d0, sm.wm[w][0]);
      d1 = umin(d1, sm.wm[w][1]);
    }
    d0 = __builtin_amdgcn_readfirstlane(d0);
    d1 = __builtin_amdgcn_readfirstlane(d1);
    if (MODE == kCSpec && d0 == kCX) ch.flags[0] |= 2;
    if (MODE == kCSpec && d1 == kCX) ch.flags[1] |= 2;
    const uint32_t d = mc ? d1 : d0;
    ch.x = umin(x - d, kCCap) << kCBits;
    ch.dsum[0] += d0;
    ch.dsum[1] += d1;
    sm.q[nxt][mc][qpad(ms)] = ch.x;
    const bool qend = (i & 3) == 3 || i == r1;
    if (qend) {
      const int q = i >> 2;
      if (MODE == kCSpec) {
        if (mvalid) {
          (a.ckrow + ((size_t)mb * a.nq + q) * kCKP)[ms] = ch.x;
          if (tid == 0 && valid0) a.dck[(size_t)b0 * a.nq + q] = (int64_t)ch.dsum[0];
          if (tid == 4 && valid1) a.dck[(size_t)b1 * a.nq + q] = (int64_t)ch.dsum[1];
        }
      }
      if (MODE == kCFix) {
        const uint64_t off0 = __ballot(mc == 0 && ch.x != ckv), off1 = __ballot(mc == 1 && ch.x != ckv);
        if (lane == 0) {
          sm.wd[wid][0] = off0 != 0;
          sm.wd[wid][1] = off1 != 0;
        }
        if (i < r1) ckv = (mc ? a.ckrow + (size_t)b1 * a.nq * kCKP : a.ckrow + (size_t)b0 * a.nq * kCKP)[(size_t)(q + 1) * kCKP + ms];
      }
    }
    __syncthreads();
    cur = nxt;
    if (MODE == kCFix && qend) {
      bool same0 = true, same1 = true;
#pragma unroll
      for (int w = 0; w < kCWaves; ++w) {
        same0 = same0 && !sm.wd[w][0];
        same1 = same1 && !sm.wd[w][1];
      }
      const int q = i >> 2;
      if (ch.conv[0] < 0 && same0) {
        ch.conv[0] = q;
        ch.dconv[0] = ch.dsum[0];
      }
      if (ch.conv[1] < 0 && same1) {
        ch.conv[1] = q;
        ch.dconv[1] = ch.dsum[1];
      }
      if ((ch.conv[0] >= 0 || !valid0) && (ch.conv[1] >= 0 || !valid1)) break;
    }
  }
  if (MODE == kCSpec) negative_costs();
}

// Speculative (MODE kCSpec, grid (ceil(B/2), P)) and fix-up (kCFix, grid
// (ceil(B/2), P-1)) passes.
template <int MODE>
__global__ __launch_bounds__(kCThreads, 1) void chain_cw_kernel(CwArgs a) {
  __shared__ __align__(16) CwSmem sm;
  const int b0 = 2 * blockIdx.x, b1 = min(b0 + 1, a.B - 1);
  const bool valid1 = b0 + 1 < a.B;
  const int p = MODE == kCFix ? blockIdx.y + 1 : blockIdx.y;
  const int r0 = p * a.CL, r1 = min(r0 + a.CL, a.N) - 1;
  const uint32_t *s0 = nullptr, *s1 = nullptr;
  if (MODE == kCFix) {
    s0 = a.ckrow + ((size_t)b0 * a.nq + r0 / 4 - 1) * kCKP;
    s1 = a.ckrow + ((size_t)b1 * a.nq + r0 / 4 - 1) * kCKP;
  }
  CwChains<MODE> ch;
  cw_run<MODE>(a, b0, b1, true, valid1, r0, r1, s0, s1, sm, ch);
  const int tid = threadIdx.x;
  const int mc = (tid & 7) >> 2, ms = 4 * (tid >> 3) + (((tid & 7) ^ (mc ? 3 : 0)) & 3);
  if (MODE == kCSpec) {
    if (tid == 0) a.rec[(size_t)b0 * a.P + p].flags = (int32_t)ch.flags[0];
    if (tid == 0 && valid1) a.rec[(size_t)b1 * a.P + p].flags = (int32_t)ch.flags[1];
  } else {
    const int mb = mc ? b1 : b0;
    if ((mc == 0 || valid1) && ch.conv[mc] < 0) a.endrow[((size_t)mb * a.P + p) * kCKP + ms] = ch.x;
    for (int c = 0; c < 2; ++c) {
      if (tid != 4 * c || (c == 1 && !valid1)) continue;
      CwRec &r = a.rec[(size_t)(c ? b1 : b0) * a.P + p];
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
  // the final row: state s of chain 0 is held by lane (tid & 7) < 4 of its quad
  const int mc = (tid & 7) >> 2, ms = 4 * (tid >> 3) + (((tid & 7) ^ (mc ? 3 : 0)) & 3);
  uint32_t xv;
  if (q < P - 1) {
    // Rerun the chain after chunk q from its true end row (the second chain
    // duplicates the first and is discarded).
    const uint32_t *st = a.endrow + ((size_t)b * P + q) * kCKP;
    CwChains<kCRepair> ch;
    cw_run<kCRepair>(a, b, b, true, false, (q + 1) * a.CL, a.N - 1, st, st, sm, ch);
    xv = ch.x;
    drep = ch.dsum[0];
  } else if (q == P - 1) {
    xv = a.endrow[((size_t)b * P + q) * kCKP + ms];
  } else {
    xv = a.ckrow[((size_t)b * a.nq + a.nq - 1) * kCKP + ms];
  }
  // The final row has minimum 0: the lowest state at the minimum (chain 0 lanes).
  const uint32_t pk = cw_wave_min((mc == 0 && ms < a.K) ? (xv | (uint32_t)ms) : kSat);
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
  const int pairs = (batch + 1) / 2;
  int P = std::max(2, (256 + pairs - 1) / pairs);  // about one workgroup per compute unit
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
  launch_pack_rtab(d.rtab, d.n_tables, d.k, kCKP, kCBits, rpk, st);
  const int pairs = (d.batch + 1) / 2;
  timer_begin(st);
  hipLaunchKernelGGL(chain_cw_kernel<kCSpec>, dim3(pairs, c.P), dim3(kCThreads), 0, st, a);
  timer_end(st);
  hipLaunchKernelGGL(chain_cw_kernel<kCFix>, dim3(pairs, c.P - 1), dim3(kCThreads), 0, st, a);
  hipLaunchKernelGGL(chain_cw_final_kernel, dim3(d.batch), dim3(kCThreads), 0, st, a, hdr, res, opt, status);
  return hipGetLastError();
}

}  // namespace cfp
