// Forward pass of the unconstrained chain search (Sec. 4.4, Eq. T):
//     D[0][s] = c[0][s],   D[i][s] = c[i][s] + min_t (D[i-1][t] + R_{e(i)}[t][s]).
//
// One workgroup (256 threads) per search.  The current row lives in LDS as
// packed words Q[t] = min(D[i][t] - rowmin_i, cap) << b, where b = index bits
// and cap = 2^(32-b) - 1.  A candidate is the saturating sum
// Q[t] + ((R[t][s] << b) | t), so one unsigned minimum over t yields both
// the least value and the lowest index attaining it.  Exactness: after the
// row minimum is subtracted, the best candidate of every state is at most
// R_max (take t = the row's argmin), so it is exact when R_max < cap; a
// state whose relative value saturates exceeds every continuation through
// the row's argmin and can never lie on an optimal plan.  The running
// offset sum_i rowmin increments is kept exactly in int64.
#include "cfp_internal.h"
#include "common.h"

namespace cfp {

__global__ void validate_rtab_kernel(const int32_t *__restrict__ rtab, size_t count, int32_t limit, WsHeader *hdr) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += (size_t)gridDim.x * blockDim.x) {
    int32_t r = rtab[i];
    if (r < 0 || r >= limit) hdr->rflag = 1;
  }
}

hipError_t launch_validate_rtab(const int32_t *rtab, int e, int k, int32_t limit, WsHeader *hdr, hipStream_t st) {
  return launch_validate_range(rtab, (size_t)e * k * k, limit, hdr, st);
}

hipError_t launch_validate_range(const int32_t *rtab, size_t count, int32_t limit, WsHeader *hdr, hipStream_t st) {
  int grid = (int)((count + kThreads - 1) / kThreads);
  if (grid > 1024) grid = 1024;
  hipLaunchKernelGGL(validate_rtab_kernel, dim3(grid), dim3(kThreads), 0, st, rtab, count, limit, hdr);
  return hipGetLastError();
}

// Block-wide minimum for 256 threads; `red` is 4 words of LDS.  Contains one
// barrier; callers must not rewrite `red` before every thread has read it.
__device__ __forceinline__ uint32_t block_min(uint32_t v, uint32_t *red) {
  v = wave_min(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return umin(umin(red[0], red[1]), umin(red[2], red[3]));
}

template <int KP>
__global__ __launch_bounds__(kThreads) void chain_fwd_kernel(
    const int32_t *__restrict__ cost, const int32_t *__restrict__ rtab, const int32_t *__restrict__ redge, int N,
    int K, uint8_t *__restrict__ table, SearchResult *__restrict__ res, const WsHeader *__restrict__ hdr,
    int64_t *__restrict__ opt, int32_t *__restrict__ status) {
  constexpr int BITS = Pow2Bits<KP>::value;
  constexpr uint32_t CAP = (1u << (32 - BITS)) - 1u;
  constexpr int TG = KP >= kThreads ? 1 : kThreads / KP;  // t-groups per state
  constexpr int TPG = KP / TG;                            // t per group
  constexpr int SPT = KP > kThreads ? KP / kThreads : 1;  // states per thread
  constexpr int ELEM = KP > 256 ? 2 : 1;

  __shared__ uint32_t Qs[2][KP];
  __shared__ uint32_t part[TG][KP];
  __shared__ uint32_t red[2][4];
  __shared__ int bad;

  const int tid = threadIdx.x;
  const int b = blockIdx.x;
  const int g = KP <= kThreads ? tid / KP : 0;
  const bool owner = (g == 0);  // this thread finalises its states
  const int32_t *cb = cost + (size_t)b * N * K;

  auto sidx = [&](int j) { return KP <= kThreads ? tid % KP : tid + kThreads * j; };

  if (tid == 0) bad = 0;
  __syncthreads();

  bool infeasible = false;
  int64_t o;

  // Block 0: D[0][s] = c[0][s].
  {
    uint32_t y[SPT], mn = kSat;
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
      int s = sidx(j);
      y[j] = kSat;
      if (owner && s < K) {
        int32_t c = cb[s];
        if (c < 0) bad = 1;
        y[j] = c == CFP_COST_INF ? kSat : (uint32_t)c;
      }
      mn = umin(mn, y[j]);
    }
    uint32_t delta = block_min(mn, red[0]);
    if (delta == kSat) infeasible = true;
    o = (int64_t)delta;
#pragma unroll
    for (int j = 0; j < SPT; ++j)
      if (owner) Qs[0][sidx(j)] = umin(y[j] - delta, CAP) << BITS;
    __syncthreads();
  }

  for (int i = 1; i < N; ++i) {
    const int cur = (i - 1) & 1, nxt = i & 1;
    const int32_t *R = rtab + (size_t)redge[i] * K * K;
    uint32_t m[SPT];
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
      const int s = sidx(j);
      uint32_t acc = kSat;
      for (int tt = 0; tt < TPG; ++tt) {
        const int t = g * TPG + tt;
        uint32_t rp = (t < K && s < K) ? (((uint32_t)R[(size_t)t * K + s] << BITS) | (uint32_t)t) : kSat;
        acc = umin(acc, sat_add(Qs[cur][t], rp));
      }
      m[j] = acc;
      if (TG > 1) part[g][s] = acc;
    }
    if (TG > 1) {
      __syncthreads();
      if (owner) {
#pragma unroll
        for (int j = 0; j < SPT; ++j) {
          uint32_t acc = kSat;
          for (int gg = 0; gg < TG; ++gg) acc = umin(acc, part[gg][sidx(j)]);
          m[j] = acc;
        }
      }
    }
    uint32_t y[SPT], mn = kSat;
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
      const int s = sidx(j);
      y[j] = kSat;
      if (owner && s < K) {
        const size_t cell = ((size_t)b * N + i) * K + s;
        const uint32_t arg = m[j] & (KP - 1);
        if (ELEM == 1)
          table[cell] = (uint8_t)arg;
        else
          ((uint16_t *)table)[cell] = (uint16_t)arg;
        int32_t c = cb[(size_t)i * K + s];
        if (c < 0) bad = 1;
        y[j] = c == CFP_COST_INF ? kSat : (m[j] >> BITS) + (uint32_t)c;
      }
      mn = umin(mn, y[j]);
    }
    uint32_t delta = block_min(mn, red[i & 1]);
    if (delta == kSat) infeasible = true;
    o += (int64_t)delta;
#pragma unroll
    for (int j = 0; j < SPT; ++j)
      if (owner) Qs[nxt][sidx(j)] = umin(y[j] - delta, CAP) << BITS;
    __syncthreads();
  }

  // Lowest final state with the least value (value field 0 after normalisation).
  const int last = (N - 1) & 1;
  uint32_t pk = kSat;
#pragma unroll
  for (int j = 0; j < SPT; ++j) {
    const int s = sidx(j);
    if (owner && s < K) pk = umin(pk, Qs[last][s] | (uint32_t)s);
  }
  uint32_t fin = block_min(pk, red[N & 1]);
  if (tid == 0) {
    int st = CFP_ST_OK;
    if (bad || hdr->rflag) st = CFP_ST_BADINPUT;
    else if (infeasible) st = CFP_ST_INFEASIBLE;
    else if ((fin >> BITS) != 0) st = CFP_ST_OVERFLOW;
    status[b] = st;
    opt[b] = st == CFP_ST_OK ? o : INT64_MAX;
    res[b].final_state = st == CFP_ST_OK ? (int32_t)(fin & (KP - 1)) : -1;
    res[b].status = st;
    res[b].final_m = 0;
  }
}

template <int KP>
static void launch_kp(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *table, SearchResult *res,
                      const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st) {
  timed_launch(chain_fwd_kernel<KP>, dim3(d.batch), dim3(kThreads), 0, st, d.cost, d.rtab, redge_dev,
                     d.n_blocks, d.k, table, res, hdr, opt, status);
}

hipError_t launch_chain_fwd(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *table, int elem,
                            uint8_t *wide, SearchResult *res, const WsHeader *hdr, int64_t *opt,
                            int32_t *status, hipStream_t st) {
  (void)elem;
  if (chain_fwd_res_supported(d.k, d.n_tables)) {
    timer_begin(st);
    const hipError_t e = launch_chain_fwd_res(d, redge_dev, table, res, hdr, opt, status, st);
    timer_end(st);
    return e;
  }
  if (chain_fwd_wide_supported(d.k)) return launch_chain_fwd_wide(d, redge_dev, wide, table, res, hdr, opt, status, st);
  const int k = d.k;
  timer_begin(st);
  if (k <= 16) launch_kp<16>(d, redge_dev, table, res, hdr, opt, status, st);
  else if (k <= 32) launch_kp<32>(d, redge_dev, table, res, hdr, opt, status, st);
  else launch_kp<64>(d, redge_dev, table, res, hdr, opt, status, st);
  timer_end(st);
  return hipGetLastError();
}

}  // namespace cfp
