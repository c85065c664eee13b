// Internal layout and launcher declarations of libcfp (not installed).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "cfp.h"

namespace cfp {

constexpr uint32_t kMagic = 0xCF900598u;
constexpr int kThreads = 256;   // threads of every search workgroup (4 waves of 64)
constexpr int kChunk = 64;      // traceback chunk length (steps)

// Number of index bits of the packed (value, index) word for K strategies.
inline int index_bits(int k) {
  int b = 4;
  while ((1 << b) < k) ++b;
  return b;
}

// Workspace header, written by the host at the start of every forward call.
struct WsHeader {
  uint32_t magic;
  int32_t variant, n, k, batch, n_mem, elem;  // elem: bytes per argmin entry
  int32_t rflag;                               // set to 1 by the device if rtab breaks its range
  // Paths that do not upload the header flag a range error with the number of
  // the call instead (no reset needed: call numbers start at a random point per
  // process and have the top bit set, so stale workspace bytes do not match).
  uint64_t rseq;
  int32_t pad[54];
};
static_assert(sizeof(WsHeader) == 256, "header is 256 bytes");

// Per-search record written by the forward kernels and read by the traceback.
struct SearchResult {
  int32_t final_state;  // lowest optimal final strategy, -1 if status != OK
  int32_t status;
  int32_t final_m;      // memory variant: budget of the search
  int32_t pad;
};

inline size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

struct WsLayout {
  size_t redge = 0;    // int32 [N]
  size_t result = 0;   // SearchResult [B]
  size_t table = 0;    // argmin entries [B][N][K] (chain, scan) or [B][N][K][M] (mem)
  size_t mem = 0;      // memory variant: copy of mem [B][N][K]
  size_t memreg = 0;   // memory variant: state order, packed tables, chunk flags and halo ring
  size_t memreg_bytes = 0;
  size_t fbudget = 0;  // memory variant: budgets [B] i32 and optima [B] i64 of a frontier call
  size_t fopt = 0;
  size_t maps = 0;     // traceback chunk maps uint16 [B][nchunks][K]
  size_t bounds = 0;   // traceback chunk boundary states int32 [B][nchunks]
  size_t wide = 0;     // chain variant, K > 64: packed tables and cost-row minima
  size_t split = 0;    // chain variant, K > 64: exchange slots and flags of the split kernel
  size_t wave = 0;     // chain variant, 32 < K <= 64 on long chains: packed tables, chunk records, checkpoints
  size_t cw = 0;       // chain variant, 128 < K <= 256 on long chains: packed tables, chunk records, checkpoints
  size_t seg = 0;      // segment variant, small batches: speculative rows, running sums, chunk records
  size_t scan = 0;     // scan variant: start of its private region
  size_t scan_bytes = 0;
  size_t total = 0;
  int elem = 1;
  int nchunks = 0;
};

WsLayout layout(int variant, int n, int k, int batch, int n_mem, int n_tables);

// Launchers (return hipSuccess or the launch error).
hipError_t launch_validate_rtab(const int32_t *rtab, int e, int k, int32_t limit, WsHeader *hdr,
                                hipStream_t st);
hipError_t launch_validate_range(const int32_t *a, size_t count, int32_t limit, WsHeader *hdr, hipStream_t st);
bool seg_supported(int k, int n_last, int n_first);
// Segment search: region of the chunk-parallel form (0 when one pass suffices);
// whether the edge map travels in the kernel arguments (then nothing of the
// header is read and no upload is needed).
size_t seg_region_bytes(int n, int k, int batch);
bool seg_edges_in_args(int n, int n_tables);
hipError_t launch_seg_fwd(const cfp_segment_desc &d, const int32_t *redge_dev, uint8_t *table, uint8_t *region,
                          SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st);
hipError_t launch_chain_fwd(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *table, int elem,
                            uint8_t *wide, SearchResult *res, const WsHeader *hdr, int64_t *opt,
                            int32_t *status, hipStream_t st);
bool chain_wave_supported(int n, int k, int n_tables, int batch);
size_t wave_region_bytes(int n, int k, int n_tables, int batch);
// True when the chunk-parallel K <= 64 path reads nothing of the uploaded
// header (periodic edge map, range errors flagged by call number).
bool chain_wave_headerless(const cfp_chain_desc &d);
hipError_t launch_chain_wave(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *region, uint8_t *table,
                             SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status,
                             hipStream_t st);
bool chain_cw_supported(int n, int k, int batch);
// One-launch search of small chains (forward, range checks and traceback).
constexpr int kSmallMaxN = 512;
constexpr int kSmallMaxBatch = 256;
constexpr size_t kSmallMaxLds = 60 * 1024;  // dynamic LDS, with room for the kernel's static words
bool chain_small_supported(int n, int k, int n_tables, int batch);
hipError_t launch_chain_small(const cfp_chain_desc &d, int64_t *opt, int32_t *status, int32_t *plan,
                              hipStream_t st);
size_t cw_region_bytes(int n, int k, int n_tables, int batch);
hipError_t launch_chain_cw(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *region, uint8_t *table,
                           SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st);
bool chain_fwd_split_supported(int k, int n_tables, int batch);
size_t split_region_bytes(int k, int batch);
hipError_t launch_chain_fwd_split(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *region, uint32_t *rpk,
                                  uint8_t *table, SearchResult *res, const WsHeader *hdr, int64_t *opt,
                                  int32_t *status, hipStream_t st);
// Packs R as (R << lb) | t; with hdr set it also flags an R entry outside [0, limit).
void launch_pack_rtab(const int32_t *rtab, int E, int K, int KP, int lb, uint32_t *rpk, hipStream_t st,
                      int32_t limit = 0, WsHeader *hdr = nullptr);
bool chain_fwd_wide_supported(int k);
size_t wide_region_bytes(int n, int k, int batch, int n_tables);
hipError_t launch_chain_fwd_wide(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *region, uint8_t *table,
                                 SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status,
                                 hipStream_t st);
bool chain_fwd_res_supported(int k, int n_tables);
hipError_t launch_chain_fwd_res(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *table, SearchResult *res,
                                const WsHeader *hdr, int64_t *opt, int32_t *status, hipStream_t st);
hipError_t launch_chain_fwd_generic(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *table,
                                    SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status,
                                    hipStream_t st);
bool chain_mem_supported(int k, int n_tables);
int32_t mem_r_limit(int k);
size_t mem_region_bytes(int n, int k, int batch, int n_mem, int n_tables);
hipError_t launch_chain_mem_fwd(const cfp_chain_desc &d, const uint8_t *mem, int n_mem, const int32_t *budget,
                                const int32_t *redge_dev, uint8_t *table, uint8_t *mem_copy, uint8_t *region,
                                SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status,
                                int64_t *frontier, hipStream_t st);
hipError_t launch_fill_i32(int32_t *p, int n, int32_t v, hipStream_t st);
hipError_t launch_traceback_chain(int n, int k, int batch, int elem, const uint8_t *table,
                                  const SearchResult *res, uint16_t *maps, int32_t *bounds, int nchunks,
                                  int32_t *plan, hipStream_t st);
hipError_t launch_traceback_mem(int n, int k, int batch, int n_mem, const uint8_t *table, const uint8_t *mem,
                                const SearchResult *res, int32_t *plan, hipStream_t st);
hipError_t launch_scan(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *region, size_t region_bytes,
                       uint8_t *table, int elem, SearchResult *res, const WsHeader *hdr, int64_t *opt,
                       int32_t *status, hipStream_t st);
size_t scan_region_bytes(int n, int k, int batch);

// Benchmarking timer: when armed, brackets each launch of a forward call's
// main kernel with a pair of HIP events on that launch's stream.
// Benchmarking timer: between timer_begin and timer_end the next timed_launch
// is timed by events attached to its dispatch (hipExtLaunchKernel), so the
// measured span is the kernel's own, without the gaps that separate event
// records add to a stream.
void timer_begin(hipStream_t st);
void timer_end(hipStream_t st);
bool timer_take(hipEvent_t *e0, hipEvent_t *e1);

template <typename... Args, typename... Params>
inline void timed_launch(void (*kernel)(Params...), dim3 grid, dim3 block, uint32_t shmem, hipStream_t st,
                         Args... args) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  timer_take(&e0, &e1);
  hipExtLaunchKernelGGL(kernel, grid, block, shmem, st, e0, e1, 0u, args...);
}

}  // namespace cfp
