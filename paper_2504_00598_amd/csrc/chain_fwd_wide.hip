// Forward pass of the unconstrained chain search for 64 < K <= 512 (Sec. 4.4,
// Eq. T recurrence), one workgroup of 8 waves per search.
//
// The resharding tables are too large to stay on chip (K=256: 256 KiB per
// table), so every step streams the table of its edge from L2.  Thread
// (sq, g) owns the four states s = 4sq .. 4sq+3 (one 16-byte load per table
// row) and the TPG rows t = g*TPG + j of group g.  The tables are packed once
// per call into the workspace with the row's index within its group,
//     RP[e][t][s] = (R_e[t][s] << lb) | (t mod TPG),   lb = log2(TPG)
// (padding rows and columns: all ones), so a candidate is one saturating add,
// Q[t] + RP[t][s], and one unsigned minimum over the group yields the least
// value and the lowest j attaining it.  The combiner of state s then takes the
// groups in order and keeps the first of least value, which is the lowest t.
//
// The thread's rows are read in chunks of 8, kept in a ring of registers: the
// chunk that a step has just consumed is reloaded at once with the same chunk
// of the next step, so the table stream continues through the two barriers
// that end a step (partials -> combine -> next row).
//
// Normalisation is one step behind, as in the register-resident kernels:
//     Q_i[s] = min(D[i][s] - o_i, cap),   o_i = o_{i-1} + d_{i-1} + cmin_i,
// with d_{i-1} = min_s Q_{i-1}[s] (reduced while row i-1 was written) and
// cmin_i = min_s c[i][s] (from a pre-pass over the cost rows), so no extra
// barrier waits for either.  Through the
// cheapest strategy of block i-1, Q_{i-1} <= R_max there, so the best
// candidate of every state is at most 2 R_max, exact while 2 R_max < cap =
// 2^(32-lb) - 1 (R < 2^24 is far inside for every K here); a state at the cap
// is beaten through that strategy by every continuation and can never lie on
// an optimal plan.  In int64, opt = sum_i cmin_i + sum_i d_i.
#include "cfp_internal.h"
#include "common.h"

namespace cfp {

constexpr int kWideThreads = 512;

// Minimum over the 64 lanes of a wave, returned to every lane: DPP within
// rows of 16, then the four row results through scalar registers.
__device__ __forceinline__ uint32_t wave_min_fast(uint32_t x) {
  x = umin(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0xB1, 0xF, 0xF, true));   // quad_perm [1,0,3,2]
  x = umin(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x4E, 0xF, 0xF, true));   // quad_perm [2,3,0,1]
  x = umin(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x141, 0xF, 0xF, true));  // row_half_mirror
  x = umin(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x140, 0xF, 0xF, true));  // row_mirror
  const uint32_t r0 = __builtin_amdgcn_readlane(x, 0), r1 = __builtin_amdgcn_readlane(x, 16);
  const uint32_t r2 = __builtin_amdgcn_readlane(x, 32), r3 = __builtin_amdgcn_readlane(x, 48);
  return umin(umin(r0, r1), umin(r2, r3));
}

template <int KP>
struct WideShape {
  static constexpr int SQ = KP / 4;                // threads per table row (4 states each)
  static constexpr int TG = kWideThreads / SQ;     // row groups
  static constexpr int TPG = KP / TG;              // rows per group
  static constexpr int LB = Pow2Bits<TPG>::value;  // index bits within a group
};

// With hdr set, the range check of R (entries in [0, limit)) is made on the
// way and flagged in the header.
__global__ void pack_rtab_kernel(const int32_t *__restrict__ rtab, int E, int K, int KP, int lb,
                                 uint32_t *__restrict__ rpk, int32_t limit, WsHeader *__restrict__ hdr) {
  const size_t total = (size_t)E * KP * KP;
  for (size_t x = (size_t)blockIdx.x * blockDim.x + threadIdx.x; x < total; x += (size_t)gridDim.x * blockDim.x) {
    const int s = (int)(x % KP);
    const int t = (int)((x / KP) % KP);
    const int e = (int)(x / ((size_t)KP * KP));
    uint32_t v = kSat;
    if (t < K && s < K) {
      const int32_t r = rtab[((size_t)e * K + t) * K + s];
      if (hdr && (r < 0 || r >= limit)) hdr->rflag = 1;
      v = ((uint32_t)r << lb) | (uint32_t)(t & ((1 << lb) - 1));
    }
    rpk[x] = v;
  }
}

// Minimum of every cost row, min_s c[b][i][s], one wave per row; a row that
// holds a negative cost gets INT32_MIN instead (valid costs are >= 0).
__global__ __launch_bounds__(256) void row_cmin_kernel(const int32_t *__restrict__ cost, int rows, int K,
                                                       int32_t *__restrict__ rowcmin) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const int32_t *c = cost + (size_t)row * K;
  int32_t m = CFP_COST_INF;
  bool neg = false;
  for (int s = lane; s < K; s += 64) {
    const int32_t v = c[s];
    neg |= v < 0;
    m = v < m ? v : m;
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const int32_t w = __shfl_xor(m, off, 64);
    m = w < m ? w : m;
  }
  neg = __any(neg);
  if (lane == 0) rowcmin[row] = neg ? INT32_MIN : m;
}

template <int KP>
__global__ __launch_bounds__(kWideThreads, 1) void chain_fwd_wide_kernel(
    const int32_t *__restrict__ cost, const int32_t *__restrict__ rowcmin, const uint32_t *__restrict__ rpk,
    const int32_t *__restrict__ redge, int N, int K, uint8_t *__restrict__ table, SearchResult *__restrict__ res,
    const WsHeader *__restrict__ hdr, int64_t *__restrict__ opt, int32_t *__restrict__ status) {
  using S = WideShape<KP>;
  constexpr int SQ = S::SQ, TG = S::TG, TPG = S::TPG, LB = S::LB;
  constexpr uint32_t CAP = (1u << (32 - LB)) - 1u;  // value field of a packed word
  constexpr int CH = 8;                              // rows per chunk
  constexpr int NCH = TPG / CH;                      // chunks per step
  constexpr int PF = NCH < 4 ? NCH : 4;              // chunks in the register ring
  constexpr int CW = KP / 64;                        // waves holding combiners
  constexpr int KB = Pow2Bits<KP>::value;            // bits of a final (Q | s) word
  static_assert(TPG % CH == 0 && NCH % PF == 0, "chunking");

  __shared__ __align__(16) uint32_t Qs[2][KP];
  __shared__ __align__(16) uint32_t part[TG][KP];
  __shared__ uint32_t wq[2][CW];  // per wave: min of the row just written

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int sq = tid % SQ, g = tid / SQ;
  const int b = blockIdx.x;
  const int32_t *cb = cost + (size_t)b * N * K;
  const int32_t *cmb = rowcmin + (size_t)b * N;
  const bool comb = tid < KP;
  const int s = tid;  // combiner state
  const bool real = comb && s < K;

  // c[i][s] of this combiner, loaded from an in-bounds address by every thread
  // (padding states read column 0; `avail` turns them into CFP_COST_INF).
  auto load_cost = [&](int i) __attribute__((always_inline)) { return cb[(size_t)i * K + (real ? s : 0)]; };
  auto avail = [&](int32_t c) __attribute__((always_inline)) { return real ? c : CFP_COST_INF; };

  // Row 0.
  int32_t cmin = cmb[0];
  bool bad = cmin < 0, infeasible = cmin == CFP_COST_INF;
  int64_t o = cmin;
  if (comb) {
    const int32_t c0 = avail(load_cost(0));
    const uint32_t q = c0 == CFP_COST_INF ? CAP : umin((uint32_t)c0 - (uint32_t)cmin, CAP);
    Qs[0][s] = q << LB;
    const uint32_t m = wave_min_fast(q);
    if (lane == 0) wq[0][wid] = m;
  }
  __syncthreads();

  // Register ring of table chunks: slot c % PF holds chunk c of the step in flight.
  uint4 ring[PF][CH];
  const uint32_t lane_off = (uint32_t)(g * TPG * KP + 4 * sq);  // words, within one table
  auto load_chunk = [&](int i, int c, uint4(&dst)[CH]) __attribute__((always_inline)) {
    const int e = __builtin_amdgcn_readfirstlane(redge[i]);
    const uint32_t *tab = rpk + (size_t)e * KP * KP + c * CH * KP;  // uniform
#pragma unroll
    for (int r = 0; r < CH; ++r) dst[r] = *(const uint4 *)(tab + lane_off + r * KP);
  };
  if (N > 1) {
#pragma unroll
    for (int c = 0; c < PF; ++c) load_chunk(1, c, ring[c]);
  }
  int32_t cm_next = cmb[N > 1 ? 1 : 0];  // cmin of the next row, one step ahead

  for (int i = 1; i < N; ++i) {
    const int cur = (i - 1) & 1, nxt = i & 1;
    // the costs of row i, issued before this step's table refills so that
    // using them after the barrier waits only for loads already consumed
    const int32_t craw = load_cost(i);
    __builtin_amdgcn_sched_barrier(0);
    uint32_t a0 = kSat, a1 = kSat, a2 = kSat, a3 = kSat;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      uint4(&R)[CH] = ring[c % PF];
      const uint4 *qp = (const uint4 *)&Qs[cur][g * TPG + c * CH];
      const uint4 qa = qp[0], qb = qp[1];
      const uint32_t q[CH] = {qa.x, qa.y, qa.z, qa.w, qb.x, qb.y, qb.z, qb.w};
#pragma unroll
      for (int r = 0; r < CH; r += 2) {
        a0 = umin(umin(a0, sat_add(q[r], R[r].x)), sat_add(q[r + 1], R[r + 1].x));
        a1 = umin(umin(a1, sat_add(q[r], R[r].y)), sat_add(q[r + 1], R[r + 1].y));
        a2 = umin(umin(a2, sat_add(q[r], R[r].z)), sat_add(q[r + 1], R[r + 1].z));
        a3 = umin(umin(a3, sat_add(q[r], R[r].w)), sat_add(q[r + 1], R[r + 1].w));
      }
      // refill this slot with the chunk PF positions further on in the stream
      // (not hoisted above the uses of the slot, which would double its
      // registers; the last step reloads its own table: in bounds, unused, and
      // no branch that would make the stream wait)
      __builtin_amdgcn_sched_barrier(0);
      const int c2 = c + PF;
      if (c2 < NCH) load_chunk(i, c2, R);
      else load_chunk(i + 1 < N ? i + 1 : i, c2 - NCH, R);
    }
    *(uint4 *)&part[g][4 * sq] = make_uint4(a0, a1, a2, a3);
    __syncthreads();

    // d_{i-1} was reduced while row i-1 was written; cmin_i comes from the pre-pass.
    uint32_t d = wq[cur][0];
#pragma unroll
    for (int w = 1; w < CW; ++w) d = umin(d, wq[cur][w]);
    const int32_t cm = cm_next;
    cm_next = cmb[i + 1 < N ? i + 1 : i];
    o += (int64_t)d + cm;
    infeasible |= cm == CFP_COST_INF;
    // used here by every thread, so the cost load cannot be sunk into the
    // combiner branch (where it would wait behind the table stream)
    const int32_t ccur = avail(craw);
    bad |= (cm | ccur) < 0;
    if (comb) {
      // first group of least value = lowest predecessor
      uint32_t best = part[0][s];
      int bg = 0;
#pragma unroll
      for (int gg = 1; gg < TG; ++gg) {
        const uint32_t p = part[gg][s];
        if ((p >> LB) < (best >> LB)) {
          best = p;
          bg = gg;
        }
      }
      if (real) {
        const size_t cell = ((size_t)b * N + i) * K + s;
        const uint32_t t = (uint32_t)bg * TPG + (best & (TPG - 1));
        if (KP > 256) ((uint16_t *)table)[cell] = (uint16_t)t;
        else table[cell] = (uint8_t)t;
      }
      const uint32_t v = (best >> LB) - d;  // >= 0: every candidate is >= the least Q
      const uint32_t q = ccur == CFP_COST_INF ? CAP : umin(v + ((uint32_t)ccur - (uint32_t)cm), CAP);
      Qs[nxt][s] = q << LB;
      const uint32_t m = wave_min_fast(q);
      if (lane == 0) wq[nxt][wid] = m;
    }
    __syncthreads();
  }

  // Lowest final state of least value
  // (a value at or above FCAP is not the least: the least is at most R_max).
  const int last = (N - 1) & 1;
  constexpr uint32_t FCAP = (1u << (32 - KB)) - 1u;
  __shared__ uint32_t fin4[CW];
  if (comb) {
    const uint32_t pk = real ? ((umin(Qs[last][s] >> LB, FCAP) << KB) | (uint32_t)s) : kSat;
    const uint32_t m = wave_min(pk);
    if (lane == 0) fin4[wid] = m;
  }
  __syncthreads();
  if (tid == 0) {
    uint32_t fin = fin4[0];
#pragma unroll
    for (int w = 1; w < CW; ++w) fin = umin(fin, fin4[w]);
    const int64_t total = o + (int64_t)(fin >> KB);
    int st = CFP_ST_OK;
    if (bad || hdr->rflag) st = CFP_ST_BADINPUT;
    else if (infeasible) st = CFP_ST_INFEASIBLE;
    else if ((fin >> KB) >= FCAP) st = CFP_ST_OVERFLOW;
    status[b] = st;
    opt[b] = st == CFP_ST_OK ? total : INT64_MAX;
    res[b].final_state = st == CFP_ST_OK ? (int32_t)(fin & (KP - 1)) : -1;
    res[b].status = st;
    res[b].final_m = 0;
  }
}

bool chain_fwd_wide_supported(int k) { return k > 64 && k <= 512; }

void launch_pack_rtab(const int32_t *rtab, int E, int K, int KP, int lb, uint32_t *rpk, hipStream_t st, int32_t limit,
                      WsHeader *hdr) {
  const size_t total = (size_t)E * KP * KP;
  const int grid = (int)((total + 255) / 256 < 4096 ? (total + 255) / 256 : 4096);
  hipLaunchKernelGGL(pack_rtab_kernel, dim3(grid), dim3(256), 0, st, rtab, E, K, KP, lb, rpk, limit, hdr);
}

// Workspace region of the kernel: packed tables [E][KP][KP] u32, then the
// cost-row minima [B][N] i32.
static size_t wide_rpk_bytes(int k, int n_tables) {
  const size_t kp = k <= 128 ? 128 : k <= 256 ? 256 : 512;
  return align_up((size_t)n_tables * kp * kp * 4);
}

size_t wide_region_bytes(int n, int k, int batch, int n_tables) {
  if (!chain_fwd_wide_supported(k)) return 0;
  return wide_rpk_bytes(k, n_tables) + align_up((size_t)batch * n * 4);
}

template <int KP>
static void launch_wide_kp(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *region, uint8_t *table,
                           SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st) {
  uint32_t *rpk = (uint32_t *)region;
  int32_t *rowcmin = (int32_t *)(region + wide_rpk_bytes(d.k, d.n_tables));
  const size_t total = (size_t)d.n_tables * KP * KP;
  const int grid = (int)((total + 255) / 256 < 4096 ? (total + 255) / 256 : 4096);
  hipLaunchKernelGGL(pack_rtab_kernel, dim3(grid), dim3(256), 0, st, d.rtab, d.n_tables, d.k, KP,
                     WideShape<KP>::LB, rpk, 0, (WsHeader *)nullptr);
  const int rows = d.batch * d.n_blocks;
  hipLaunchKernelGGL(row_cmin_kernel, dim3((rows + 3) / 4), dim3(256), 0, st, d.cost, rows, d.k, rowcmin);
  timer_begin(st);
  timed_launch(chain_fwd_wide_kernel<KP>, dim3(d.batch), dim3(kWideThreads), 0, st, d.cost, (const int32_t *)rowcmin,
               (const uint32_t *)rpk, redge_dev, d.n_blocks, d.k, table, res, hdr, opt, status);
  timer_end(st);
}

hipError_t launch_chain_fwd_wide(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *region, uint8_t *table,
                                 SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status,
                                 hipStream_t st) {
  if (d.k <= 128) launch_wide_kp<128>(d, redge_dev, region, table, res, hdr, opt, status, st);
  else if (d.k <= 256) launch_wide_kp<256>(d, redge_dev, region, table, res, hdr, opt, status, st);
  else launch_wide_kp<512>(d, redge_dev, region, table, res, hdr, opt, status, st);
  return hipGetLastError();
}

}  // namespace cfp
