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
// Q[s] = min(D[i][s] - min_s D[i][s], cap); the class minima and the L x F
// boundary candidates go through LDS atomic minima on packed words
// (Q << b) | t, so every minimum carries the lowest predecessor t of least
// value.  Through the row's argmin (Q = 0) the best candidate of every state is
// at most r_max, exact while r_max < cap = 2^(32-b) - 1; a state at the cap is
// beaten through that argmin by every continuation.
#include "cfp_internal.h"
#include "common.h"

namespace cfp {

constexpr int kSegWaves = 4;  // searches per workgroup
constexpr int kSegMaxLF = 8;  // largest number of strategies of a boundary block

// Minimum over the 64 lanes of a wave (DPP within rows, then the four row
// results through scalar registers); every lane gets it.
__device__ __forceinline__ uint32_t seg_wave_min(uint32_t x) {
  x = umin(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0xB1, 0xF, 0xF, true));   // quad_perm [1,0,3,2]
  x = umin(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x4E, 0xF, 0xF, true));   // quad_perm [2,3,0,1]
  x = umin(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x141, 0xF, 0xF, true));  // row_half_mirror
  x = umin(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x140, 0xF, 0xF, true));  // row_mirror
  const uint32_t r0 = __builtin_amdgcn_readlane(x, 0), r1 = __builtin_amdgcn_readlane(x, 16);
  const uint32_t r2 = __builtin_amdgcn_readlane(x, 32), r3 = __builtin_amdgcn_readlane(x, 48);
  return umin(umin(r0, r1), umin(r2, r3));
}

template <int SPL>
__global__ __launch_bounds__(kSegWaves * 64) void seg_fwd_kernel(
    const int32_t *__restrict__ cost, const int32_t *__restrict__ rbound, const uint8_t *__restrict__ last,
    const uint8_t *__restrict__ first, const int32_t *__restrict__ redge, int N, int K, int B, int L, int F,
    int bits, uint8_t *__restrict__ table, SearchResult *__restrict__ res, const WsHeader *__restrict__ hdr,
    int64_t *__restrict__ opt, int32_t *__restrict__ status) {
  __shared__ uint32_t Ml[kSegWaves][kSegMaxLF], Gl[kSegWaves][kSegMaxLF];
  const int wid = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int b = blockIdx.x * kSegWaves + wid;
  if (b >= B) return;  // the waves are independent: nothing below waits for another wave
  const uint32_t CAP = (1u << (32 - bits)) - 1u, IMASK = (1u << bits) - 1u;
  const int32_t *cb = cost + (size_t)b * N * K;
  const bool wide = K > 256;  // argmin entries are 16-bit

  int ls[SPL], fs[SPL];
  bool real[SPL];
  uint32_t q[SPL], y[SPL];
  int32_t cc[SPL], cn[SPL];
  bool bad = false;
#pragma unroll
  for (int j = 0; j < SPL; ++j) {
    const int s = lane + 64 * j;
    real[j] = s < K;
    ls[j] = real[j] ? last[s] : 0;
    fs[j] = real[j] ? first[s] : 0;
    bad |= real[j] && (ls[j] >= L || fs[j] >= F);
    if (ls[j] >= L) ls[j] = 0;  // keep LDS indices in range; the search reports bad input
    if (fs[j] >= F) fs[j] = 0;
  }

  // Row 0.
  uint32_t ym = kSat;
#pragma unroll
  for (int j = 0; j < SPL; ++j) {
    const int32_t c = real[j] ? cb[lane + 64 * j] : CFP_COST_INF;
    bad |= c < 0;
    y[j] = c == CFP_COST_INF ? kSat : (uint32_t)c;
    ym = umin(ym, y[j]);
  }
  uint32_t rmin = seg_wave_min(ym);
  int64_t o = rmin;
  bool infeasible = rmin == kSat;
#pragma unroll
  for (int j = 0; j < SPL; ++j) {
    q[j] = umin(y[j] - rmin, CAP);
    cn[j] = cb[(size_t)(N > 1 ? 1 : 0) * K + (real[j] ? lane + 64 * j : 0)];  // next row, in bounds
  }

  // lane l*F + f keeps its boundary entry of the next step (one step ahead)
  const int lf_l = lane / F, lf_f = lane - (lane / F) * F;
  const bool lf = lane < L * F;
  auto load_r = [&](int i) __attribute__((always_inline)) {
    const int e = redge[i < N ? i : N - 1];
    return lf ? (uint32_t)rbound[((size_t)e * L + lf_l) * F + lf_f] : 0u;
  };
  uint32_t rnext = load_r(1);

  for (int i = 1; i < N; ++i) {
    const uint32_t r = rnext;
    rnext = load_r(i + 1);
    // class minima of the previous row: M_l with its lowest argmin
    if (lane < L) Ml[wid][lane] = kSat;
#pragma unroll
    for (int j = 0; j < SPL; ++j)
      if (real[j]) atomicMin(&Ml[wid][ls[j]], (q[j] << bits) | (uint32_t)(lane + 64 * j));
    // boundary candidates: lane l*F + f offers M_l + r[l][f] to state class f
    if (lane < F) Gl[wid][lane] = kSat;
    if (lf) atomicMin(&Gl[wid][lf_f], sat_add(Ml[wid][lf_l], r << bits));
    // the new row
    ym = kSat;
#pragma unroll
    for (int j = 0; j < SPL; ++j) {
      cc[j] = cn[j];
      cn[j] = cb[(size_t)(i + 1 < N ? i + 1 : i) * K + (real[j] ? lane + 64 * j : 0)];
    }
#pragma unroll
    for (int j = 0; j < SPL; ++j) {
      y[j] = kSat;
      if (real[j]) {
        const uint32_t g = Gl[wid][fs[j]];
        const size_t cell = ((size_t)b * N + i) * K + lane + 64 * j;
        if (wide) ((uint16_t *)table)[cell] = (uint16_t)(g & IMASK);
        else table[cell] = (uint8_t)(g & IMASK);
        bad |= cc[j] < 0;
        if (cc[j] != CFP_COST_INF && g != kSat) y[j] = (g >> bits) + (uint32_t)cc[j];
      }
      ym = umin(ym, y[j]);
    }
    rmin = seg_wave_min(ym);
    o += rmin;
    infeasible |= rmin == kSat;
#pragma unroll
    for (int j = 0; j < SPL; ++j) q[j] = umin(y[j] - rmin, CAP);
  }

  // Lowest final state of least value (the least is 0 after normalisation).
  uint32_t pk = kSat;
#pragma unroll
  for (int j = 0; j < SPL; ++j)
    if (real[j]) pk = umin(pk, (q[j] << bits) | (uint32_t)(lane + 64 * j));
  const uint32_t fin = seg_wave_min(pk);
  bad = __any(bad);
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

template <int SPL>
static void launch_seg_spl(const cfp_segment_desc &d, const int32_t *redge_dev, uint8_t *table, SearchResult *res,
                           const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st) {
  const int grid = (d.batch + kSegWaves - 1) / kSegWaves;
  timed_launch(seg_fwd_kernel<SPL>, dim3(grid), dim3(kSegWaves * 64), 0, st, d.cost, d.rbound, d.last,
                     d.first, redge_dev, d.n_segments, d.k, d.batch, d.n_last, d.n_first, index_bits(d.k), table,
                     res, hdr, opt, status);
}

hipError_t launch_seg_fwd(const cfp_segment_desc &d, const int32_t *redge_dev, uint8_t *table, SearchResult *res,
                          const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st) {
  timer_begin(st);
  if (d.k <= 64) launch_seg_spl<1>(d, redge_dev, table, res, hdr, opt, status, st);
  else if (d.k <= 128) launch_seg_spl<2>(d, redge_dev, table, res, hdr, opt, status, st);
  else if (d.k <= 256) launch_seg_spl<4>(d, redge_dev, table, res, hdr, opt, status, st);
  else launch_seg_spl<8>(d, redge_dev, table, res, hdr, opt, status, st);
  timer_end(st);
  return hipGetLastError();
}

}  // namespace cfp
