// Plan recovery from the argmin tables (the plan tuple of Sec. 4.4).
//
// table[b][i][s] (i >= 1) is the lowest predecessor t of state s at block i.
// Following it from the final state is a chain of N-1 dependent lookups, so
// the chain is cut into chunks of kChunk steps processed in three launches:
//   1. maps:   for every chunk and every possible end state, follow the chunk
//              in LDS to its start state (all chunks and states in parallel);
//   2. bounds: per search, compose the chunk maps from the final state to get
//              the state at every chunk boundary (nchunks dependent lookups);
//   3. fill:   per chunk, follow it again from its known end state and write
//              the plan entries.
// When one search's table fits in LDS the three steps run in a single launch
// with one workgroup per search (tb_lds_kernel below).
// The memory variant has states (s, m) and is followed step by step.
#include "cfp_internal.h"
#include "common.h"

#include <algorithm>
#include <cmath>
#include <type_traits>

namespace cfp {

// Index bits of the packed words (the stored argmin may carry value bits above them).
__device__ __forceinline__ int index_bits_dev(int k) {
  int b = 4;
  while ((1 << b) < k) ++b;
  return b;
}

struct ChunkSpan {
  int lo, hi;  // the chunk covers steps hi, hi-1, ..., lo+1 (block indices)
};

__device__ __forceinline__ ChunkSpan chunk_span(int c, int n) {
  ChunkSpan sp;
  sp.hi = n - 1 - c * kChunk;
  sp.lo = sp.hi - kChunk > 0 ? sp.hi - kChunk : 0;
  return sp;
}

// Copy the rows of steps lo+1 .. hi of one search into LDS (contiguous), in
// 16-byte pieces when the rows are so aligned.
template <typename T>
__device__ void load_chunk(const T *__restrict__ tab, int b, int n, int k, ChunkSpan sp, T *lds) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const size_t base = ((size_t)b * n + sp.lo + 1) * k;
  const int count = (sp.hi - sp.lo) * k;
  constexpr int PER = 16 / sizeof(T);
  if ((base % PER) == 0 && (count % PER) == 0) {
    const u32x4 *src = (const u32x4 *)(tab + base);
    u32x4 *dst = (u32x4 *)lds;
    for (int x = threadIdx.x; x < count / PER; x += blockDim.x) dst[x] = src[x];
  } else {
    for (int x = threadIdx.x; x < count; x += blockDim.x) lds[x] = tab[base + x];
  }
  __syncthreads();
}

template <typename T>
__global__ __launch_bounds__(kThreads) void tb_maps_kernel(int n, int k, const T *__restrict__ tab,
                                                           const SearchResult *__restrict__ res,
                                                           uint16_t *__restrict__ maps, int nchunks) {
  extern __shared__ __align__(16) uint8_t smem[];
  T *rows = (T *)smem;
  const int c = blockIdx.x, b = blockIdx.y;
  if (res[b].status != CFP_ST_OK) return;
  const ChunkSpan sp = chunk_span(c, n);
  load_chunk(tab, b, n, k, sp, rows);
  const int mask = (1 << index_bits_dev(k)) - 1;
  for (int s = threadIdx.x; s < k; s += blockDim.x) {
    int t = s;
    for (int i = sp.hi; i > sp.lo; --i) {
      int p = rows[(i - sp.lo - 1) * k + t] & mask;
      t = p < k ? p : k - 1;  // unreachable end states may carry any index; stay in bounds
    }
    maps[((size_t)b * nchunks + c) * k + s] = (uint16_t)t;
  }
}

// One search per workgroup: its chunk maps are staged in LDS (when they fit)
// so the composition is a chain of LDS reads rather than of memory loads.
constexpr int kBoundsThreads = 256;
constexpr size_t kBoundsLds = 48 * 1024;

__global__ __launch_bounds__(kBoundsThreads) void tb_bounds_kernel(int n, int k, int batch,
                                                                   const SearchResult *__restrict__ res,
                                                                   const uint16_t *__restrict__ maps,
                                                                   int32_t *__restrict__ bounds, int nchunks,
                                                                   int32_t *__restrict__ plan, int staged) {
  extern __shared__ __align__(16) uint16_t smaps[];
  const int b = blockIdx.x;
  if (res[b].status != CFP_ST_OK) {
    if (threadIdx.x == 0) plan[(size_t)b * n + n - 1] = -1;
    return;
  }
  const uint16_t *mb = maps + (size_t)b * nchunks * k;
  if (staged) {
    for (int x = threadIdx.x; x < nchunks * k; x += blockDim.x) smaps[x] = mb[x];
    __syncthreads();
  }
  if (threadIdx.x != 0) return;
  int s = res[b].final_state;
  plan[(size_t)b * n + n - 1] = s;
  for (int c = 0; c < nchunks; ++c) {
    bounds[(size_t)b * nchunks + c] = s;
    s = staged ? smaps[c * k + s] : mb[(size_t)c * k + s];
  }
}

template <typename T>
__global__ __launch_bounds__(kThreads) void tb_fill_kernel(int n, int k, const T *__restrict__ tab,
                                                           const SearchResult *__restrict__ res,
                                                           const int32_t *__restrict__ bounds, int nchunks,
                                                           int32_t *__restrict__ plan) {
  extern __shared__ __align__(16) uint8_t smem[];
  T *rows = (T *)smem;
  const int c = blockIdx.x, b = blockIdx.y;
  const ChunkSpan sp = chunk_span(c, n);
  int32_t *pb = plan + (size_t)b * n;
  if (res[b].status != CFP_ST_OK) {
    for (int i = sp.lo + threadIdx.x; i < sp.hi; i += blockDim.x) pb[i] = -1;
    return;
  }
  load_chunk(tab, b, n, k, sp, rows);
  __shared__ int32_t out[kChunk];
  if (threadIdx.x == 0) {
    const int mask = (1 << index_bits_dev(k)) - 1;
    int t = bounds[(size_t)b * nchunks + c];
    for (int i = sp.hi; i > sp.lo; --i) {
      int p = rows[(i - sp.lo - 1) * k + t] & mask;
      t = p < k ? p : k - 1;
      out[i - 1 - sp.lo] = t;
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < sp.hi - sp.lo; i += blockDim.x) pb[sp.lo + i] = out[i];
}

// Single-launch traceback: one workgroup of kTbWaves waves per search, the
// search's argmin rows staged in LDS.  The n - 1 steps are cut into nch
// chunks of span steps (span a multiple of kTbG, nch about sqrt(n), so that
// the chunk length and the number of chunks, both lengths of dependent lookup
// chains, are balanced); pad identity rows in front of row 1 make every chunk
// exactly span steps long, so the lookup loop has no per-step bounds.
//   1. Every (chunk, end state) pair is followed back to the chunk's start;
//      a wave task is one chunk and 64 end states, a wave carries up to
//      kTbMaxTasks of them stepped together, and the state at every kTbG-th
//      block is kept (the "marks").
//   2. One thread composes the chunk maps from the final state.
//   3. Every piece of kTbG steps is followed by its own thread from its known
//      end state and writes its plan entries.
constexpr int kTbWaves = 16;
constexpr int kTbThreads = 64 * kTbWaves;
constexpr int kTbLdsBytes = 152 * 1024;
constexpr int kTbMaxTasks = 8;  // chunk tasks per wave
constexpr int kTbG = 8;         // steps per piece

struct TbLdsPlan {
  int ok;
  int span, nch;   // steps per chunk (a multiple of kTbG), chunks
  int pad;         // identity rows in front: padded block = block + pad
  int tasks;       // chunk tasks per wave
  int marks_off;   // byte offset of the marks [nch][K][span / kTbG - 1]
  int maps_off;    // byte offset of the chunk maps [nch][K]
};

static TbLdsPlan tb_lds_plan(int n, int k, int elem) {
  TbLdsPlan p{};
  if (n < 1) return p;
  const int steps = n - 1;
  const int sb = (k + 63) / 64;  // blocks of 64 end states per chunk
  int nch = (int)std::lround(std::sqrt((double)std::max(steps, 1)));
  nch = std::max(1, std::min(nch, kTbWaves * kTbMaxTasks / sb));
  p.span = std::max(kTbG, (steps + nch - 1) / nch + kTbG - 1) / kTbG * kTbG;
  p.nch = steps > 0 ? (steps + p.span - 1) / p.span : 0;
  p.pad = p.nch * p.span - steps;
  p.tasks = (p.nch * sb + kTbWaves - 1) / kTbWaves;
  const long long rows = ((long long)p.nch * p.span * k * elem + 15) / 16 * 16;
  const long long marks = ((long long)p.nch * k * (p.span / kTbG - 1) * elem + 15) / 16 * 16;
  const long long maps = ((long long)p.nch * k * elem + 15) / 16 * 16;
  p.marks_off = (int)std::min<long long>(rows, 1 << 30);
  p.maps_off = (int)std::min<long long>(rows + marks, 1 << 30);
  p.ok = rows + marks + maps <= kTbLdsBytes && p.tasks <= kTbMaxTasks;
  return p;
}

template <typename T, int NT>
__global__ __launch_bounds__(kTbThreads) void tb_lds_kernel(int n, int k, const T *__restrict__ tab,
                                                            const SearchResult *__restrict__ res,
                                                            int32_t *__restrict__ plan, TbLdsPlan pl) {
  __shared__ __align__(16) uint8_t sm[kTbLdsBytes];
  __shared__ int32_t s_end[kTbThreads];  // state at the last block of each chunk
  const int b = blockIdx.x, tid = threadIdx.x;
  int32_t *pb = plan + (size_t)b * n;
  if (res[b].status != CFP_ST_OK) {
    for (int i = tid; i < n; i += kTbThreads) pb[i] = -1;
    return;
  }
  const int pad = pl.pad, span = pl.span, nm = span / kTbG - 1;
  T *rows = (T *)sm;  // padded row i' (1 <= i' <= nch span) at (i' - 1) k; real row i = i' - pad
  T *marks = (T *)(sm + pl.marks_off);
  T *maps = (T *)(sm + pl.maps_off);
  for (int x = tid; x < pad * k; x += kTbThreads) rows[x] = (T)(x % k);  // identity rows
  {
    // All loads of a batch are issued before any is stored (addresses past
    // the end are clamped, so every load is unconditional and completes in order).
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    constexpr int kBatch = 8;
    const size_t base = ((size_t)b * n + 1) * k;
    const int count = (n - 1) * k;
    T *dst0 = rows + (size_t)pad * k;
    constexpr int PER = 16 / sizeof(T);
    if ((base % PER) == 0 && (count % PER) == 0 && (((size_t)pad * k) % PER) == 0) {
      const u32x4 *src = (const u32x4 *)(tab + base);
      u32x4 *dst = (u32x4 *)dst0;
      const int m = count / PER;
      for (int x0 = tid; x0 < m; x0 += kBatch * kTbThreads) {
        u32x4 v[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) v[u] = src[min(x0 + u * kTbThreads, m - 1)];
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
          if (x0 + u * kTbThreads < m) dst[x0 + u * kTbThreads] = v[u];
      }
    } else {
      for (int x0 = tid; x0 < count; x0 += kBatch * kTbThreads) {
        T v[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) v[u] = tab[base + min(x0 + u * kTbThreads, count - 1)];
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
          if (x0 + u * kTbThreads < count) dst0[x0 + u * kTbThreads] = v[u];
      }
    }
  }
  __syncthreads();
  const int mask = (1 << index_bits_dev(k)) - 1;
  // 1. Chunk maps and marks.  Wave task w + kTbWaves j (j < NT) is chunk c and
  // end states 64 m + lane; its row offset is wave-uniform.  Tasks past the
  // last chunk and lanes past K follow chunk 0 from state 0 and store nothing.
  if (pl.nch > 0) {
    const int wid = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int sb = (k + 63) >> 6;
    int t[NT], off[NT], tau[NT];
    bool on[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const int wt = wid + kTbWaves * j;
      const int c = wt / sb, s = 64 * (wt - c * sb) + lane;
      const bool live = c < pl.nch;
      on[j] = live && s < k;
      t[j] = on[j] ? s : 0;
      off[j] = ((live ? c + 1 : 1) * span - 1) * k;  // padded row (c + 1) span
      tau[j] = c * k + s;
    }
    for (int x0 = 0; x0 < span; x0 += kTbG) {
#pragma unroll
      for (int u = 0; u < kTbG; ++u) {
        int p[NT];
#pragma unroll
        for (int j = 0; j < NT; ++j) p[j] = rows[off[j] + t[j]];
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          const int q = p[j] & mask;
          t[j] = q < k ? q : k - 1;  // unreachable end states may carry any index; stay in bounds
          off[j] -= k;
        }
      }
      if (x0 + kTbG < span) {
        const int m = x0 / kTbG;
#pragma unroll
        for (int j = 0; j < NT; ++j)
          if (on[j]) marks[tau[j] * nm + m] = (T)t[j];
      }
    }
#pragma unroll
    for (int j = 0; j < NT; ++j)
      if (on[j]) maps[tau[j]] = (T)t[j];
  }
  __syncthreads();
  // 2. Compose the chunk maps from the final state.
  if (tid == 0) {
    int s = res[b].final_state;
    pb[n - 1] = s;
    for (int c = pl.nch - 1; c >= 0; --c) {
      s_end[c] = s;
      s = maps[c * k + s];
    }
  }
  __syncthreads();
  // 3. Pieces of kTbG steps, one thread each; padded blocks below pad are not
  // real and are not written.
  const int ng = span / kTbG;
  for (int x = tid; x < pl.nch * ng; x += kTbThreads) {
    const int c = x / ng, j = x - c * ng;
    const int phi = (c + 1) * span - kTbG * j;  // padded block the piece starts from
    const int e = s_end[c];
    int t = j == 0 ? e : (int)marks[(c * k + e) * nm + j - 1];
#pragma unroll
    for (int u = 0; u < kTbG; ++u) {
      const int i = phi - u;  // padded row of this step
      const int q = rows[(i - 1) * k + t] & mask;
      t = q < k ? q : k - 1;
      if (i - 1 - pad >= 0) pb[i - 1 - pad] = t;
    }
  }
}

hipError_t launch_traceback_chain(int n, int k, int batch, int elem, const uint8_t *table,
                                  const SearchResult *res, uint16_t *maps, int32_t *bounds, int nchunks,
                                  int32_t *plan, hipStream_t st) {
  const TbLdsPlan pl = tb_lds_plan(n, k, elem);
  if (pl.ok) {
    auto go = [&](auto tp, auto ntc) {
      using T = decltype(tp);
      constexpr int NT = decltype(ntc)::value;
      hipLaunchKernelGGL((tb_lds_kernel<T, NT>), dim3(batch), dim3(kTbThreads), 0, st, n, k, (const T *)table, res,
                         plan, pl);
    };
    auto by_tasks = [&](auto tp) {
      switch (pl.tasks) {
        case 0:
        case 1: go(tp, std::integral_constant<int, 1>{}); break;
        case 2: go(tp, std::integral_constant<int, 2>{}); break;
        case 3: go(tp, std::integral_constant<int, 3>{}); break;
        case 4: go(tp, std::integral_constant<int, 4>{}); break;
        case 5: go(tp, std::integral_constant<int, 5>{}); break;
        case 6: go(tp, std::integral_constant<int, 6>{}); break;
        case 7: go(tp, std::integral_constant<int, 7>{}); break;
        default: go(tp, std::integral_constant<int, 8>{}); break;
      }
    };
    if (elem == 1) by_tasks(uint8_t{});
    else by_tasks(uint16_t{});
    return hipGetLastError();
  }
  const size_t lds = (size_t)kChunk * k * elem;
  if (nchunks > 0) {
    if (elem == 1)
      hipLaunchKernelGGL(tb_maps_kernel<uint8_t>, dim3(nchunks, batch), dim3(kThreads), lds, st, n, k, table, res,
                         maps, nchunks);
    else
      hipLaunchKernelGGL(tb_maps_kernel<uint16_t>, dim3(nchunks, batch), dim3(kThreads), lds, st, n, k,
                         (const uint16_t *)table, res, maps, nchunks);
  }
  const size_t mbytes = (size_t)nchunks * k * 2;
  const int staged = mbytes <= kBoundsLds ? 1 : 0;
  hipLaunchKernelGGL(tb_bounds_kernel, dim3(batch), dim3(kBoundsThreads), staged ? mbytes : 0, st, n, k, batch, res,
                     maps, bounds, nchunks, plan, staged);
  if (nchunks > 0) {
    if (elem == 1)
      hipLaunchKernelGGL(tb_fill_kernel<uint8_t>, dim3(nchunks, batch), dim3(kThreads), lds, st, n, k, table, res,
                         bounds, nchunks, plan);
    else
      hipLaunchKernelGGL(tb_fill_kernel<uint16_t>, dim3(nchunks, batch), dim3(kThreads), lds, st, n, k,
                         (const uint16_t *)table, res, bounds, nchunks, plan);
  }
  return hipGetLastError();
}

}  // namespace cfp
