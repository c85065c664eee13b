// Exported C ABI of libcfp: argument validation, workspace layout and launch
// sequencing.  Every check that can be made on the host is made before the
// first HIP call, so argument errors never touch the device.
#include <string.h>

#include <atomic>
#include <mutex>
#include <vector>

#include "cfp_internal.h"

namespace cfp {

WsLayout layout(int variant, int n, int k, int batch, int n_mem, int n_tables) {
  WsLayout L;
  L.elem = k > 256 ? 2 : 1;
  size_t off = sizeof(WsHeader);
  L.redge = off;
  off = align_up(off + (size_t)n * 4);
  L.result = off;
  off = align_up(off + (size_t)batch * sizeof(SearchResult));
  L.nchunks = n > 1 ? (n - 1 + kChunk - 1) / kChunk : 0;
  L.table = off;
  size_t cells = (size_t)batch * n * k;
  if (variant == CFP_V_MEM) {
    off = align_up(off + cells * (size_t)n_mem * L.elem);
    L.mem = off;
    off = align_up(off + cells);
    L.memreg = off;
    L.memreg_bytes = mem_region_bytes(n, k, batch, n_mem, n_tables);
    off = align_up(off + L.memreg_bytes);
    L.fbudget = off;
    off = align_up(off + (size_t)batch * 4);
    L.fopt = off;
    off = align_up(off + (size_t)batch * 8);
  } else {
    off = align_up(off + cells * L.elem);
  }
  L.maps = off;
  off = align_up(off + (size_t)batch * L.nchunks * k * 2);
  L.bounds = off;
  off = align_up(off + (size_t)batch * L.nchunks * 4);
  if (variant == CFP_V_CHAIN && chain_fwd_wide_supported(k)) {
    L.wide = off;
    off = align_up(off + wide_region_bytes(n, k, batch, n_tables));
    L.split = off;
    off = align_up(off + split_region_bytes(k, batch));
  }
  if (variant == CFP_V_CHAIN && chain_wave_supported(n, k, n_tables, batch)) {
    L.wave = off;
    off = align_up(off + wave_region_bytes(n, k, n_tables, batch));
  }
  if (variant == CFP_V_CHAIN && chain_cw_supported(n, k, batch)) {
    L.cw = off;
    off = align_up(off + cw_region_bytes(n, k, n_tables, batch));
  }
  if (variant == CFP_V_SEG) {
    L.seg = off;
    off = align_up(off + seg_region_bytes(n, k, batch));
  }
  if (variant == CFP_V_SCAN) {
    L.scan = off;
    L.scan_bytes = scan_region_bytes(n, k, batch);
    off = align_up(off + L.scan_bytes);
  }
  L.total = off;
  return L;
}

// Benchmarking timer (cfp_timer_start / cfp_timer_stop).  Slot 2j and 2j+1
// hold the start and stop events of the j-th timed launch.
namespace {
std::mutex g_timer_mu;
std::atomic<bool> g_timer_on{false};
std::vector<hipEvent_t> g_timer_ev;
size_t g_timer_used = 0;
bool g_timer_open = false;  // armed for the next timed_launch
}  // namespace

void timer_begin(hipStream_t) {
  if (!g_timer_on.load(std::memory_order_acquire)) return;
  std::lock_guard<std::mutex> lk(g_timer_mu);
  g_timer_open = true;
}

void timer_end(hipStream_t) {
  if (!g_timer_on.load(std::memory_order_acquire)) return;
  std::lock_guard<std::mutex> lk(g_timer_mu);
  g_timer_open = false;
}

bool timer_take(hipEvent_t *e0, hipEvent_t *e1) {
  if (!g_timer_on.load(std::memory_order_acquire)) return false;
  std::lock_guard<std::mutex> lk(g_timer_mu);
  if (!g_timer_open || 2 * g_timer_used + 1 >= g_timer_ev.size()) return false;
  *e0 = g_timer_ev[2 * g_timer_used];
  *e1 = g_timer_ev[2 * g_timer_used + 1];
  ++g_timer_used;
  g_timer_open = false;
  return true;
}

}  // namespace cfp

using namespace cfp;

namespace {

bool desc_ok(const cfp_chain_desc *d) {
  if (!d) return false;
  if (d->n_blocks < 1 || d->k < 1 || d->k > CFP_MAX_K || d->batch < 1 || d->n_tables < 1) return false;
  if (!d->cost || !d->rtab || !d->redge) return false;
  return true;
}

int check_desc(const cfp_chain_desc *d) {
  if (!d) return CFP_ERR_ARG;
  if (d->k > CFP_MAX_K) return CFP_ERR_UNSUPPORTED;
  if (!desc_ok(d)) return CFP_ERR_ARG;
  for (int i = 1; i < d->n_blocks; ++i)
    if (d->redge[i] < 0 || d->redge[i] >= d->n_tables) return CFP_ERR_RANGE;
  return CFP_OK;
}

// Host-to-device copies of the per-call header go through a ring of pinned
// host slots per device, so that the copy is asynchronous: a copy from pageable
// memory holds the calling thread until the stream has drained, which leaves
// the GPU idle while the next call's launches are issued.  A slot is reused
// only once the event recorded behind its previous copy has completed.
constexpr int kUpSlots = 32;
constexpr size_t kUpSlotBytes = 64 * 1024;
constexpr int kUpDevices = 64;

struct UploadRing {
  uint8_t *host = nullptr;
  hipEvent_t ev[kUpSlots] = {};
  bool pending[kUpSlots] = {};
  int next = 0;
  bool init = false, ok = false;
};
std::mutex g_up_mu;
UploadRing g_up[kUpDevices];

// Copy `bytes` bytes produced by fill(host_ptr) to dst on stream st.
template <typename F>
int upload(void *dst, size_t bytes, hipStream_t st, F fill) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return CFP_ERR_HIP;
  if (bytes <= kUpSlotBytes && dev >= 0 && dev < kUpDevices) {
    std::lock_guard<std::mutex> lk(g_up_mu);
    UploadRing &r = g_up[dev];
    if (!r.init) {
      r.init = true;
      r.ok = hipHostMalloc((void **)&r.host, kUpSlots * kUpSlotBytes, hipHostMallocDefault) == hipSuccess;
      for (int i = 0; r.ok && i < kUpSlots; ++i)
        r.ok = hipEventCreateWithFlags(&r.ev[i], hipEventDisableTiming) == hipSuccess;
    }
    if (r.ok) {
      const int slot = r.next;
      r.next = (r.next + 1) % kUpSlots;
      if (r.pending[slot] && hipEventSynchronize(r.ev[slot]) != hipSuccess) return CFP_ERR_HIP;
      r.pending[slot] = false;
      uint8_t *h = r.host + (size_t)slot * kUpSlotBytes;
      fill(h);
      if (hipMemcpyAsync(dst, h, bytes, hipMemcpyHostToDevice, st) != hipSuccess) return CFP_ERR_HIP;
      if (hipEventRecord(r.ev[slot], st) != hipSuccess) return CFP_ERR_HIP;
      r.pending[slot] = true;
      return CFP_OK;
    }
  }
  // Too large for a slot (or no pinned memory): a copy from pageable memory.
  std::vector<uint8_t> buf(bytes);
  fill(buf.data());
  if (hipMemcpyAsync(dst, buf.data(), bytes, hipMemcpyHostToDevice, st) != hipSuccess) return CFP_ERR_HIP;
  return CFP_OK;
}

// Header + device copy of redge, enqueued as one host-to-device copy.
int upload_header(const cfp_chain_desc *d, int variant, int n_mem, const WsLayout &L, void *ws, hipStream_t st) {
  const size_t bytes = L.redge + (size_t)d->n_blocks * 4;
  return upload(ws, bytes, st, [&](uint8_t *buf) {
    memset(buf, 0, L.redge);
    WsHeader h;
    memset(&h, 0, sizeof h);
    h.magic = kMagic;
    h.variant = variant;
    h.n = d->n_blocks;
    h.k = d->k;
    h.batch = d->batch;
    h.n_mem = n_mem;
    h.elem = L.elem;
    h.rflag = 0;
    memcpy(buf, &h, sizeof h);
    memcpy(buf + L.redge, d->redge, (size_t)d->n_blocks * 4);
    memset(buf + L.redge, 0, 4);  // redge[0] is ignored; keep it a valid table index
  });
}

// Workspace of cfp_search_chain_noalloc: a static device array, one per GPU,
// held until the process ends.  Host code never uses its name as an address:
// the device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) uint8_t scratch[CFP_NOALLOC_MAX_BYTES];

constexpr int kNoAllocDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kNoAllocDevices] = {};

// Device address of `scratch` on the current device (nullptr on failure).
void *scratch_address() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kNoAllocDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

// Words carried by one launch of put_words_kernel as its argument, so that
// host data reaches the device without a staging buffer.
constexpr int kPutWords = 960;
struct PutChunk {
  int32_t n, off;
  int32_t v[kPutWords];
};
static_assert(sizeof(PutChunk) + 16 < 4096, "one kernel argument block");

__global__ void put_words_kernel(int32_t *__restrict__ dst, PutChunk c) {
  for (int x = threadIdx.x; x < c.n; x += blockDim.x) dst[c.off + x] = c.v[x];
}

// Header and edge map of a chain call (the words [0, L.redge/4 + N) of the
// workspace) written by kernels whose arguments carry them.
int put_header(const cfp_chain_desc *d, const WsLayout &L, uint8_t *w, hipStream_t st) {
  WsHeader h;
  memset(&h, 0, sizeof h);
  h.magic = kMagic;
  h.variant = CFP_V_CHAIN;
  h.n = d->n_blocks;
  h.k = d->k;
  h.batch = d->batch;
  h.n_mem = 0;
  h.elem = L.elem;
  const int hw = (int)(L.redge / 4), total = hw + d->n_blocks;
  PutChunk c;
  for (int off = 0; off < total; off += kPutWords) {
    c.n = total - off < kPutWords ? total - off : kPutWords;
    c.off = off;
    for (int x = 0; x < c.n; ++x) {
      const int word = off + x;
      if (word < (int)(sizeof h / 4)) c.v[x] = ((const int32_t *)&h)[word];
      else if (word < hw) c.v[x] = 0;
      else c.v[x] = word == hw ? 0 : d->redge[word - hw];  // redge[0] is ignored; keep it a valid table index
    }
    hipLaunchKernelGGL(put_words_kernel, dim3(1), dim3(256), 0, st, (int32_t *)w, c);
    if (hipGetLastError() != hipSuccess) return CFP_ERR_HIP;
  }
  return CFP_OK;
}

// The launches of a chain forward call once the header and the edge map are
// in the workspace (or not needed: the periodic chunk-parallel K <= 64 path).
int dp_chain_launch(const cfp_chain_desc *d, const WsLayout &L, uint8_t *w, int64_t *opt, int32_t *status,
                    hipStream_t st) {
  WsHeader *hdr = (WsHeader *)w;
  const bool wave = chain_wave_supported(d->n_blocks, d->k, d->n_tables, d->batch);
  const bool cw = !wave && chain_cw_supported(d->n_blocks, d->k, d->batch);
  if (!wave && !cw &&
      launch_validate_rtab(d->rtab, d->n_tables, d->k, cfp_r_limit(CFP_V_CHAIN, d->k), hdr, st) != hipSuccess)
    return CFP_ERR_HIP;
  hipError_t e;
  if (wave)
    e = launch_chain_wave(*d, (const int32_t *)(w + L.redge), w + L.wave, w + L.table,
                          (SearchResult *)(w + L.result), hdr, opt, status, st);
  else if (cw)
    e = launch_chain_cw(*d, (const int32_t *)(w + L.redge), w + L.cw, w + L.table, (SearchResult *)(w + L.result),
                        hdr, opt, status, st);
  else if (chain_fwd_split_supported(d->k, d->n_tables, d->batch))
    e = launch_chain_fwd_split(*d, (const int32_t *)(w + L.redge), w + L.split, (uint32_t *)(w + L.wide),
                               w + L.table, (SearchResult *)(w + L.result), hdr, opt, status, st);
  else
    e = launch_chain_fwd(*d, (const int32_t *)(w + L.redge), w + L.table, L.elem, w + L.wide,
                         (SearchResult *)(w + L.result), hdr, opt, status, st);
  return e == hipSuccess ? CFP_OK : CFP_ERR_HIP;
}

}  // namespace

#pragma GCC visibility push(default)
extern "C" {

int32_t cfp_r_limit(int32_t variant, int32_t k) {
  if (k < 1 || k > CFP_MAX_K) return 0;
  int b = index_bits(k);
  switch (variant) {
    case CFP_V_CHAIN:
    case CFP_V_SCAN:
      return k <= 64 ? (int32_t)(1u << (30 - b)) : (int32_t)((1u << (32 - b)) - 1u);
    case CFP_V_MEM:
      return mem_r_limit(k);
    case CFP_V_SEG:
      return (int32_t)((1u << (32 - b)) - 1u);
    default:
      return 0;
  }
}

size_t cfp_workspace_bytes(const cfp_chain_desc *d, int32_t variant, int32_t n_mem) {
  if (!desc_ok(d)) return 0;
  if (variant == CFP_V_MEM) {
    if (n_mem < 1 || n_mem > 4096 || !chain_mem_supported(d->k, d->n_tables)) return 0;
  } else if (variant != CFP_V_CHAIN && variant != CFP_V_SCAN) {
    return 0;
  }
  return layout(variant, d->n_blocks, d->k, d->batch, variant == CFP_V_MEM ? n_mem : 0, d->n_tables).total;
}

int cfp_dp_chain(const cfp_chain_desc *d, void *ws, size_t ws_bytes, int64_t *opt, int32_t *status,
                 void *stream) {
  int rc = check_desc(d);
  if (rc != CFP_OK) return rc;
  if (!opt || !status) return CFP_ERR_ARG;
  WsLayout L = layout(CFP_V_CHAIN, d->n_blocks, d->k, d->batch, 0, d->n_tables);
  if (!ws || ws_bytes < L.total) return CFP_ERR_WORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  // The chunk-parallel paths check the range of R while packing it; the K <= 64
  // one with a periodic edge map reads nothing of the header, which is then not
  // uploaded (a host-to-device copy costs several microseconds of GPU time).
  const bool wave = chain_wave_supported(d->n_blocks, d->k, d->n_tables, d->batch);
  if (!(wave && chain_wave_headerless(*d)) && (rc = upload_header(d, CFP_V_CHAIN, 0, L, ws, st)) != CFP_OK)
    return rc;
  return dp_chain_launch(d, L, (uint8_t *)ws, opt, status, st);
}

int cfp_dp_chain_mem(const cfp_chain_desc *d, const uint8_t *mem, int32_t n_mem, const int32_t *budget,
                     void *ws, size_t ws_bytes, int64_t *opt, int32_t *status, void *stream) {
  int rc = check_desc(d);
  if (rc != CFP_OK) return rc;
  if (!mem || !budget || !opt || !status) return CFP_ERR_ARG;
  if (n_mem < 1) return CFP_ERR_ARG;
  if (n_mem > 4096 || !chain_mem_supported(d->k, d->n_tables)) return CFP_ERR_UNSUPPORTED;
  WsLayout L = layout(CFP_V_MEM, d->n_blocks, d->k, d->batch, n_mem, d->n_tables);
  if (!ws || ws_bytes < L.total) return CFP_ERR_WORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  uint8_t *w = (uint8_t *)ws;
  if ((rc = upload_header(d, CFP_V_MEM, n_mem, L, ws, st)) != CFP_OK) return rc;
  WsHeader *hdr = (WsHeader *)w;
  // the memory forward checks the range of R while packing it
  if (launch_chain_mem_fwd(*d, mem, n_mem, budget, (const int32_t *)(w + L.redge), w + L.table, w + L.mem,
                           w + L.memreg, (SearchResult *)(w + L.result), hdr, opt, status, nullptr, st) != hipSuccess)
    return CFP_ERR_HIP;
  return CFP_OK;
}

int cfp_mem_frontier(const cfp_chain_desc *d, const uint8_t *mem, int32_t n_mem, void *ws, size_t ws_bytes,
                     int64_t *frontier, int32_t *status, void *stream) {
  int rc = check_desc(d);
  if (rc != CFP_OK) return rc;
  if (!mem || !frontier || !status) return CFP_ERR_ARG;
  if (n_mem < 1) return CFP_ERR_ARG;
  if (n_mem > 4096 || !chain_mem_supported(d->k, d->n_tables)) return CFP_ERR_UNSUPPORTED;
  WsLayout L = layout(CFP_V_MEM, d->n_blocks, d->k, d->batch, n_mem, d->n_tables);
  if (!ws || ws_bytes < L.total) return CFP_ERR_WORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  uint8_t *w = (uint8_t *)ws;
  if ((rc = upload_header(d, CFP_V_MEM, n_mem, L, ws, st)) != CFP_OK) return rc;
  WsHeader *hdr = (WsHeader *)w;
  int32_t *budget = (int32_t *)(w + L.fbudget);
  if (launch_fill_i32(budget, d->batch, n_mem - 1, st) != hipSuccess) return CFP_ERR_HIP;
  // the memory forward checks the range of R while packing it
  if (launch_chain_mem_fwd(*d, mem, n_mem, budget, (const int32_t *)(w + L.redge), w + L.table, w + L.mem,
                           w + L.memreg, (SearchResult *)(w + L.result), hdr, (int64_t *)(w + L.fopt), status,
                           frontier, st) != hipSuccess)
    return CFP_ERR_HIP;
  return CFP_OK;
}

int cfp_minplus_scan(const cfp_chain_desc *d, void *ws, size_t ws_bytes, int64_t *opt, int32_t *status,
                     void *stream) {
  int rc = check_desc(d);
  if (rc != CFP_OK) return rc;
  if (!opt || !status) return CFP_ERR_ARG;
  WsLayout L = layout(CFP_V_SCAN, d->n_blocks, d->k, d->batch, 0, d->n_tables);
  if (!ws || ws_bytes < L.total) return CFP_ERR_WORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  uint8_t *w = (uint8_t *)ws;
  if ((rc = upload_header(d, CFP_V_SCAN, 0, L, ws, st)) != CFP_OK) return rc;
  WsHeader *hdr = (WsHeader *)w;
  if (launch_validate_rtab(d->rtab, d->n_tables, d->k, cfp_r_limit(CFP_V_SCAN, d->k), hdr, st) != hipSuccess)
    return CFP_ERR_HIP;
  if (launch_scan(*d, (const int32_t *)(w + L.redge), w + L.scan, L.scan_bytes, w + L.table, L.elem,
                  (SearchResult *)(w + L.result), hdr, opt, status, st) != hipSuccess)
    return CFP_ERR_HIP;
  return CFP_OK;
}

int cfp_traceback(const cfp_chain_desc *d, int32_t variant, int32_t n_mem, void *ws, size_t ws_bytes,
                  int32_t *plan, void *stream) {
  if (!desc_ok(d)) return d && d->k > CFP_MAX_K ? CFP_ERR_UNSUPPORTED : CFP_ERR_ARG;
  if (!plan) return CFP_ERR_ARG;
  if (variant != CFP_V_CHAIN && variant != CFP_V_MEM && variant != CFP_V_SCAN) return CFP_ERR_ARG;
  if (variant == CFP_V_MEM && (n_mem < 1 || n_mem > 4096 || !chain_mem_supported(d->k, d->n_tables)))
    return CFP_ERR_ARG;
  WsLayout L = layout(variant, d->n_blocks, d->k, d->batch, variant == CFP_V_MEM ? n_mem : 0, d->n_tables);
  if (!ws || ws_bytes < L.total) return CFP_ERR_WORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  uint8_t *w = (uint8_t *)ws;
  hipError_t e;
  if (variant == CFP_V_MEM)
    e = launch_traceback_mem(d->n_blocks, d->k, d->batch, n_mem, w + L.table, w + L.mem,
                             (const SearchResult *)(w + L.result), plan, st);
  else
    e = launch_traceback_chain(d->n_blocks, d->k, d->batch, L.elem, w + L.table,
                               (const SearchResult *)(w + L.result), (uint16_t *)(w + L.maps),
                               (int32_t *)(w + L.bounds), L.nchunks, plan, st);
  return e == hipSuccess ? CFP_OK : CFP_ERR_HIP;
}

int cfp_search_chain(const cfp_chain_desc *d, void *ws, size_t ws_bytes, int64_t *opt, int32_t *status,
                     int32_t *plan, void *stream) {
  int rc = check_desc(d);
  if (rc != CFP_OK) return rc;
  if (!opt || !status || !plan) return CFP_ERR_ARG;
  hipStream_t st = (hipStream_t)stream;
  if (chain_small_supported(d->n_blocks, d->k, d->n_tables, d->batch))
    return launch_chain_small(*d, opt, status, plan, st) == hipSuccess ? CFP_OK : CFP_ERR_HIP;
  if ((rc = cfp_dp_chain(d, ws, ws_bytes, opt, status, stream)) != CFP_OK) return rc;
  return cfp_traceback(d, CFP_V_CHAIN, 0, ws, ws_bytes, plan, stream);
}

int cfp_search_chain_noalloc(const cfp_chain_desc *d, int64_t *opt, int32_t *status, int32_t *plan,
                             void *stream) {
  int rc = check_desc(d);
  if (rc != CFP_OK) return rc;
  if (!opt || !status || !plan) return CFP_ERR_ARG;
  const WsLayout L = layout(CFP_V_CHAIN, d->n_blocks, d->k, d->batch, 0, d->n_tables);
  if (L.total > (size_t)CFP_NOALLOC_MAX_BYTES) return CFP_ERR_WORKSPACE;  // beyond the static scratch
  uint8_t *w = (uint8_t *)scratch_address();
  if (!w) return CFP_ERR_HIP;
  hipStream_t st = (hipStream_t)stream;
  // Every region the kernels read is written earlier in the same call; the
  // header (range flags included) is rewritten whole.
  if ((rc = put_header(d, L, w, st)) != CFP_OK) return rc;
  if ((rc = dp_chain_launch(d, L, w, opt, status, st)) != CFP_OK) return rc;
  const hipError_t e = launch_traceback_chain(d->n_blocks, d->k, d->batch, L.elem, w + L.table,
                                              (const SearchResult *)(w + L.result), (uint16_t *)(w + L.maps),
                                              (int32_t *)(w + L.bounds), L.nchunks, plan, st);
  return e == hipSuccess ? CFP_OK : CFP_ERR_HIP;
}

int cfp_timer_start(int32_t max_launches) {
  if (max_launches < 1 || max_launches > (1 << 20)) return CFP_ERR_ARG;
  std::lock_guard<std::mutex> lk(g_timer_mu);
  if (g_timer_on.load()) return CFP_ERR_ARG;
  g_timer_ev.assign(2 * (size_t)max_launches, nullptr);
  for (auto &e : g_timer_ev)
    if (hipEventCreate(&e) != hipSuccess) {
      for (auto &f : g_timer_ev)
        if (f) (void)hipEventDestroy(f);
      g_timer_ev.clear();
      return CFP_ERR_HIP;
    }
  g_timer_used = 0;
  g_timer_open = false;
  g_timer_on.store(true, std::memory_order_release);
  return CFP_OK;
}

int cfp_timer_stop(double *total_ms, int32_t *launches) {
  std::lock_guard<std::mutex> lk(g_timer_mu);
  if (!g_timer_on.load()) return CFP_ERR_ARG;
  g_timer_on.store(false, std::memory_order_release);
  int rc = CFP_OK;
  double sum = 0.0;
  for (size_t j = 0; j < g_timer_used; ++j) {
    float ms = 0.f;
    if (hipEventSynchronize(g_timer_ev[2 * j + 1]) != hipSuccess ||
        hipEventElapsedTime(&ms, g_timer_ev[2 * j], g_timer_ev[2 * j + 1]) != hipSuccess)
      rc = CFP_ERR_HIP;
    sum += ms;
  }
  for (auto &e : g_timer_ev) (void)hipEventDestroy(e);
  g_timer_ev.clear();
  if (total_ms) *total_ms = sum;
  if (launches) *launches = (int32_t)g_timer_used;
  g_timer_used = 0;
  return rc;
}

}  // extern "C"

namespace {

bool seg_desc_ok(const cfp_segment_desc *d) {
  if (!d) return false;
  if (d->n_segments < 1 || d->k < 1 || d->batch < 1 || d->n_tables < 1) return false;
  if (!d->cost || !d->rbound || !d->last || !d->first || !d->redge) return false;
  return true;
}

int check_seg(const cfp_segment_desc *d) {
  if (!d) return CFP_ERR_ARG;
  if (d->k > CFP_MAX_K || d->n_last > 8 || d->n_first > 8) return CFP_ERR_UNSUPPORTED;
  if (!seg_desc_ok(d) || d->n_last < 1 || d->n_first < 1) return CFP_ERR_ARG;
  if ((size_t)d->n_segments * d->k * 8 > (size_t)INT32_MAX) return CFP_ERR_UNSUPPORTED;  // 32-bit row offsets
  for (int i = 1; i < d->n_segments; ++i)
    if (d->redge[i] < 0 || d->redge[i] >= d->n_tables) return CFP_ERR_RANGE;
  return CFP_OK;
}

// The fields the workspace header and the traceback read, as a chain descriptor.
cfp_chain_desc as_chain(const cfp_segment_desc *d) {
  cfp_chain_desc c;
  c.n_blocks = d->n_segments;
  c.k = d->k;
  c.batch = d->batch;
  c.n_tables = d->n_tables;
  c.cost = d->cost;
  c.rtab = d->rbound;
  c.redge = d->redge;
  return c;
}

}  // namespace

extern "C" {

size_t cfp_segment_workspace_bytes(const cfp_segment_desc *d) {
  if (check_seg(d) != CFP_OK) return 0;
  return layout(CFP_V_SEG, d->n_segments, d->k, d->batch, 0, d->n_tables).total;
}

int cfp_dp_segments(const cfp_segment_desc *d, void *ws, size_t ws_bytes, int64_t *opt, int32_t *status,
                    void *stream) {
  int rc = check_seg(d);
  if (rc != CFP_OK) return rc;
  if (!opt || !status) return CFP_ERR_ARG;
  WsLayout L = layout(CFP_V_SEG, d->n_segments, d->k, d->batch, 0, d->n_tables);
  if (!ws || ws_bytes < L.total) return CFP_ERR_WORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  uint8_t *w = (uint8_t *)ws;
  const cfp_chain_desc c = as_chain(d);
  // the search kernels check the range of rbound themselves and read the edge
  // map from the workspace only when it is too long for the kernel arguments
  if (!seg_edges_in_args(d->n_segments, d->n_tables) && (rc = upload_header(&c, CFP_V_SEG, 0, L, ws, st)) != CFP_OK)
    return rc;
  WsHeader *hdr = (WsHeader *)w;
  if (launch_seg_fwd(*d, (const int32_t *)(w + L.redge), w + L.table, w + L.seg, (SearchResult *)(w + L.result), hdr,
                     opt, status, st) != hipSuccess)
    return CFP_ERR_HIP;
  return CFP_OK;
}

int cfp_traceback_segments(const cfp_segment_desc *d, void *ws, size_t ws_bytes, int32_t *plan, void *stream) {
  int rc = check_seg(d);
  if (rc != CFP_OK) return rc;
  if (!plan) return CFP_ERR_ARG;
  WsLayout L = layout(CFP_V_SEG, d->n_segments, d->k, d->batch, 0, d->n_tables);
  if (!ws || ws_bytes < L.total) return CFP_ERR_WORKSPACE;
  uint8_t *w = (uint8_t *)ws;
  const hipError_t e = launch_traceback_chain(d->n_segments, d->k, d->batch, L.elem, w + L.table,
                                              (const SearchResult *)(w + L.result), (uint16_t *)(w + L.maps),
                                              (int32_t *)(w + L.bounds), L.nchunks, plan, (hipStream_t)stream);
  return e == hipSuccess ? CFP_OK : CFP_ERR_HIP;
}

const char *cfp_status_string(int code) {
  switch (code) {
    case CFP_OK: return "ok";
    case CFP_ST_INFEASIBLE: return "infeasible: no plan satisfies the constraints";
    case CFP_ST_OVERFLOW: return "overflow: device arithmetic left its exact range";
    case CFP_ST_TIMEOUT: return "timeout: a bounded device wait expired";
    case CFP_ST_BADINPUT: return "bad input: a device array value is outside its documented range";
    case CFP_ERR_ARG: return "invalid argument";
    case CFP_ERR_RANGE: return "host array value out of range";
    case CFP_ERR_WORKSPACE: return "workspace missing or too small";
    case CFP_ERR_UNSUPPORTED: return "unsupported size";
    case CFP_ERR_HIP: return "HIP runtime error";
    default: return "unknown code";
  }
}

}  // extern "C"
#pragma GCC visibility pop
