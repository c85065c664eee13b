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
// The memory variant has states (s, m) and is followed step by step.
#include "cfp_internal.h"
#include "common.h"

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

hipError_t launch_traceback_chain(int n, int k, int batch, int elem, const uint8_t *table,
                                  const SearchResult *res, uint16_t *maps, int32_t *bounds, int nchunks,
                                  int32_t *plan, hipStream_t st) {
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
