// Helpers shared by the register-resident chain kernels (K <= 64).
#pragma once

#include <type_traits>

#include "cfp_internal.h"
#include "common.h"

namespace cfp {

constexpr int kResTables = 12;  // resharding tables kept in registers
constexpr int kUnroll = 12;     // steps per unrolled group = cost rows per staging block

// DPP helpers (gfx9 encodings).
constexpr int kQuadSwap1 = 0xB1;   // quad_perm [1,0,3,2]
constexpr int kQuadSwap2 = 0x4E;   // quad_perm [2,3,0,1]
constexpr int kHalfMirror = 0x141;
constexpr int kMirror = 0x140;
constexpr int kRowBcast0 = 0x150;  // row_newbcast:n = kRowBcast0 + n: lane n of each row to the whole row

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_min(uint32_t x) {
  return umin(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, CTRL, 0xF, 0xF, true));
}
template <int CTRL>
__device__ __forceinline__ int32_t dpp_min_i32(int32_t x) {
  const int32_t y = __builtin_amdgcn_mov_dpp(x, CTRL, 0xF, 0xF, true);
  return y < x ? y : x;
}

// Minimum over aligned groups of N lanes (N = 1, 2, 4, 8 or 16); every lane
// of the group gets it.
template <int N>
__device__ __forceinline__ uint32_t group_min(uint32_t x) {
  if (N >= 2) x = dpp_min<kQuadSwap1>(x);
  if (N >= 4) x = dpp_min<kQuadSwap2>(x);
  if (N >= 8) x = dpp_min<kHalfMirror>(x);
  if (N >= 16) x = dpp_min<kMirror>(x);
  return x;
}
template <int N>
__device__ __forceinline__ int32_t group_min_i32(int32_t x) {
  if (N >= 2) x = dpp_min_i32<kQuadSwap1>(x);
  if (N >= 4) x = dpp_min_i32<kQuadSwap2>(x);
  if (N >= 8) x = dpp_min_i32<kHalfMirror>(x);
  if (N >= 16) x = dpp_min_i32<kMirror>(x);
  return x;
}

// Cost rows of one search staged through LDS in blocks of kUnroll rows.
// Threads tid < kUnroll*KP/4 each own 4 consecutive entries of one row
// (KP/4 threads per row, an aligned DPP group).  A block is loaded into
// registers one block ahead and stored as
//     cadj[r][s] = c[r][s] - min_s c[r][s]   (2^31 for CFP_COST_INF)
// together with the argmin bytes of the steps, which are written back to the
// table one block behind.
template <int KP>
struct CostStager {
  static constexpr int U = kUnroll;
  static constexpr int LPR = KP / 4;
  static constexpr int STAGERS = U * LPR;
  const int32_t *cb;  // cost rows of this search
  uint8_t *tb;        // argmin table rows of this search
  int N, K, tid;
  bool stager, full_rows;
  int st_r, st_c;
  int32_t creg[4];
  int64_t csum = 0;   // sum over the rows reduced by this thread of min_s c[r][s]

  __device__ CostStager(const int32_t *cb_, uint8_t *tb_, int N_, int K_, int tid_)
      : cb(cb_), tb(tb_), N(N_), K(K_), tid(tid_) {
    stager = tid < STAGERS;
    full_rows = (K == KP);
    st_r = tid / LPR;
    st_c = (tid % LPR) * 4;
  }

  __device__ __forceinline__ void load(int blk) {
    const int row = blk * U + st_r;
#pragma unroll
    for (int q = 0; q < 4; ++q) creg[q] = CFP_COST_INF;
    if (stager && row < N) {
      const int32_t *src = cb + (size_t)row * K + st_c;
      if (full_rows) {
        const int4 v = *(const int4 *)src;
        creg[0] = v.x; creg[1] = v.y; creg[2] = v.z; creg[3] = v.w;
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (st_c + q < K) creg[q] = src[q];
      }
    }
  }

  // flags: bit 0 = a negative cost, bit 1 = a row with no available strategy.
  __device__ __forceinline__ void store(int blk, uint32_t (*cadj)[KP], int *flags) {
    const int row = blk * U + st_r;
    int32_t cm = creg[0];
    bool neg = false;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      neg |= creg[q] < 0;
      cm = creg[q] < cm ? creg[q] : cm;
    }
    cm = group_min_i32<LPR>(cm);
    if (stager) {
      uint4 w;
      w.x = creg[0] == CFP_COST_INF ? 0x80000000u : (uint32_t)(creg[0] - cm);
      w.y = creg[1] == CFP_COST_INF ? 0x80000000u : (uint32_t)(creg[1] - cm);
      w.z = creg[2] == CFP_COST_INF ? 0x80000000u : (uint32_t)(creg[2] - cm);
      w.w = creg[3] == CFP_COST_INF ? 0x80000000u : (uint32_t)(creg[3] - cm);
      *(uint4 *)&cadj[st_r][st_c] = w;
      if (row < N) {
        if (neg) atomicOr(flags, 1);
        if ((tid % LPR) == 0) {
          if (cm == CFP_COST_INF) atomicOr(flags, 2);
          csum += cm;
        }
      }
    }
  }

  // Write the argmin bytes of block blk (rows blk*U ..) to the table.
  __device__ __forceinline__ void flush(int blk, const uint8_t (*argb)[KP]) {
    const int row = blk * U + st_r;
    if (!stager || row >= N) return;
    const uint32_t w = *(const uint32_t *)&argb[st_r][st_c];
    uint8_t *dst = tb + (size_t)row * K + st_c;
    if (full_rows) {
      *(uint32_t *)dst = w;
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (st_c + q < K) dst[q] = (uint8_t)(w >> (8 * q));
    }
  }
};

// Final answer of a search: lowest state of least value in the last row,
// opt = sum of row minima of the costs + sum of normalisation offsets + the
// value of that state.  pk: (Q | s) of this lane's state or kSat.
__device__ __forceinline__ void finish_search(uint32_t pk, int64_t csum, uint64_t dsum, int bits, uint32_t cap,
                                              int flags, const WsHeader *hdr, int b, int64_t *opt, int32_t *status,
                                              SearchResult *res) {
  __shared__ uint32_t fin4[4];
  __shared__ int64_t csum4[4];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  pk = wave_min(pk);
  int64_t cs = csum;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) cs += __shfl_xor(cs, off, 64);
  if (lane == 0) {
    fin4[wid] = pk;
    csum4[wid] = cs;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t fin = umin(umin(fin4[0], fin4[1]), umin(fin4[2], fin4[3]));
    const int64_t total = csum4[0] + csum4[1] + csum4[2] + csum4[3] + (int64_t)dsum + (int64_t)(fin >> bits);
    int st = CFP_ST_OK;
    if ((flags & 1) || hdr->rflag) st = CFP_ST_BADINPUT;
    else if (flags & 2) st = CFP_ST_INFEASIBLE;
    else if ((fin >> bits) >= cap) st = CFP_ST_OVERFLOW;
    status[b] = st;
    opt[b] = st == CFP_ST_OK ? total : INT64_MAX;
    res[b].final_state = st == CFP_ST_OK ? (int32_t)(fin & ((1u << bits) - 1u)) : -1;
    res[b].status = st;
    res[b].final_m = 0;
  }
}

}  // namespace cfp
