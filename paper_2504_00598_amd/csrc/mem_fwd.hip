// Search under a memory budget (Sec. 4.4: least Eq. T cost with Eq. M within
// the memory limit, memory quantised into buckets):
//     D[0][s][m] = c[0][s]                                   if mem[0][s] <= m
//     D[i][s][m] = c[i][s] + min_t D[i-1][t][m - mem[i][s]] + R_{e(i)}[t][s]
// with D = +inf where m < mem[i][s]; the answer is min_s D[N-1][s][budget].
// D[i][s][m] is the least cost of a prefix whose memory total is at most m,
// so it does not increase with m.
//
// Layout.  Each search is cut into chunks of 64 memory buckets; one workgroup
// (8 waves) computes one chunk for all K <= 32 states.  Step i of a chunk
// only reads buckets m - mem[i][s] >= m - kMemShift of step i-1, so a chunk
// needs the top kMemShift buckets of the chunk below it: each chunk
// publishes what the chunk above needs of them in a device ring (one slot per
// step) and then raises a counter; the chunk above waits for the counter
// (bounded spin).  The ring
// and the counters are only touched by device-scope atomic stores and loads,
// and the counter is raised after every ring store has completed, so no cache
// write-back or invalidation is needed.  Chunks of one search have workgroup ids j*B + b, so a producer
// always has a lower id than its consumer and, for B a multiple of 8, all
// chunks of a search share one XCD and its L2.
//
// Arithmetic.  Column m carries an exact int64 offset o[m] = min_s D[s][m];
// LDS holds Q[s][m] = min(D[s][m] - o[m], cap) << b with cap = 2^(32-b) - 1.
// A candidate is the saturating sum Q[t][m-d] + ((R[t][s] << b) | t)
// with the resharding column of state s read from an LDS copy of the packed
// tables (every lane reads the same words); its value is
// relative to o[m-d], and o[m-d] - o[m] >= 0 (fewer buckets never cost
// less) converts it.  The best candidate of any state is at most R_max
// (through the minimum of column m-d), so it is exact for R < cap; a state
// whose relative value reaches the cap is beaten, at the same memory, by the
// minimum state of its column and can never lie on an optimal plan.  The
// kernel forms the products min_t Q[t][m'] + R[t][s] at unshifted buckets m'
// and applies each state's shift to them (see mem_fwd_kernel).
#include "cfp_internal.h"
#include "common.h"

namespace cfp {

constexpr int kMemChunk = 64;  // buckets per workgroup
constexpr int kMemShift = 16;  // largest supported mem entry (halo width)
constexpr int64_t kOffInf = (int64_t)1 << 62;
constexpr int kSpinLimit = 1 << 22;
constexpr int kMemTables = 12;  // resharding tables supported (kept in LDS)
constexpr int kMemThreads = 512;  // 8 waves: two per SIMD, so one wave's waits overlap the other's work

enum { MEMF_BAD = 1, MEMF_TIMEOUT = 2, MEMF_OVERFLOW = 4 };

// Per-search, per-block order of the states by memory shift (stable), as
// records (state | shift << 8, cost), so that a wave reads the records of its
// states with one scalar load; copies mem for the traceback; validates mem and
// the budget.  One wave per (b, i) row.
template <int KP>
__global__ __launch_bounds__(256) void mem_prep_kernel(const int32_t *__restrict__ cost, const uint8_t *__restrict__ mem,
                                                       const int32_t *__restrict__ budget, int N, int K, int M, int B,
                                                       uint2 *__restrict__ srec, uint8_t *__restrict__ mem_copy,
                                                       int32_t *__restrict__ mflags) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= B * N) return;
  const int b = row / N;
  const size_t base = (size_t)row * K;
  int d = 0, c = CFP_COST_INF;
  bool bad = false;
  if (lane < K) {
    d = mem[base + lane];
    c = cost[base + lane];
    mem_copy[base + lane] = (uint8_t)d;
    bad = d >= M || d > kMemShift || c < 0;
  }
  if (lane == 0 && (row % N) == 0 && (budget[b] < 0 || budget[b] >= M)) bad = true;
  if (__any(bad) && lane == 0) atomicOr(&mflags[b], MEMF_BAD);
  if (d > kMemShift) d = kMemShift;
  // stable rank by shift; states K..KP-1 (unavailable padding) sort last
  const int key = lane < K ? d : kMemShift + 1;
  int rank = 0;
  for (int o = 0; o < KP; ++o) {
    const int ko = __shfl(key, o, 64);
    rank += (ko < key) || (ko == key && o < lane);
  }
  if (lane < KP) {
    // record: x = state | shift << 8, y = cost
    srec[(size_t)row * KP + rank] = make_uint2((uint32_t)lane | ((uint32_t)(lane < K ? d : 0) << 8),
                                               (uint32_t)(lane < K ? c : CFP_COST_INF));
  }
}

// Resharding tables transposed and packed: rpT[e][s][t] = (R[e][t][s] << b) | t.
// Every R entry is read here, so the range check of R (entries in [0, limit))
// is made on the way and flagged in the header.
template <int KP>
__global__ void mem_pack_rtab_kernel(const int32_t *__restrict__ rtab, int E, int K, uint32_t *__restrict__ rpT,
                                     int32_t limit, WsHeader *__restrict__ hdr) {
  constexpr int BITS = Pow2Bits<KP>::value;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= E * KP * KP) return;
  const int e = idx / (KP * KP), s = (idx / KP) % KP, t = idx % KP;
  uint32_t v = kSat;
  if (s < K && t < K) {
    const int32_t r = rtab[((size_t)e * K + t) * K + s];
    if (r < 0 || r >= limit) hdr->rflag = 1;
    v = ((uint32_t)r << BITS) | (uint32_t)t;
  }
  rpT[idx] = v;
}

struct MemWs {
  uint2 *srec;       // [B][N][KP] records sorted by shift
  uint32_t *rpT;
  int32_t *mflags;   // [B]
  int32_t *pub;      // [B][nchunk]: last step published by each chunk
  uint32_t *ring;    // [B][nchunk][N][KP][kMemShift]
  int64_t *ring_off; // [B][nchunk][N][kMemShift]
  int nchunk;
};

// One step in product-then-shift form.  A state s with memory shift d takes
// its candidates from column m - d:
//     D[i][s][m] = c + min_t (Q[t][m-d] + R[t][s]) = c + P[s][m-d],
//     P[s][m']  = min_t (Q[t][m'] + R[t][s]),
// so a workgroup forms the products P at its own buckets once (each lane reads
// the K rows of its bucket's column once) and then shifts only P: one read per
// state and bucket instead of K per state and distinct shift.  The buckets
// below the chunk come from the chunk below, which passes its products (not
// its rows) for its top kMemShift buckets through the ring.
//   Phase A (products): wave w forms P for the states of rank SW w .. SW w +
//     SW - 1, lanes over the chunk's buckets.
//   Phase B (shift and normalise): wave w takes BPW = C / NW buckets; lane
//     (c = lane % BPW, g = lane / BPW) bucket BPW w + c and the SB states of
//     rank SB g ..; the column minimum is reduced over the lanes of a bucket.
// Step i of a chunk needs slot i of the ring below (P_i and the offsets of
// step i-1 of the top buckets) before its phase B.  A chunk stores slot i as
// soon as its products are in LDS (after the first barrier of step i), every
// lane one word (no branch around the stores, so the waits for later loads
// are exact), waits for the stores during phase B and publishes the slot
// after the second barrier: the chunk above runs about one step behind.
// Wave 0 reads the ring below.
template <int KP>
__global__ __launch_bounds__(kMemThreads) void mem_fwd_kernel(const int32_t *__restrict__ redge,
                                                           const int32_t *__restrict__ budget,
                                                           const uint2 *__restrict__ srec, const uint32_t *__restrict__ rpT,
                                                           int N, int K, int M, int B, MemWs w, uint8_t *__restrict__ table,
                                                           SearchResult *__restrict__ res, const WsHeader *__restrict__ hdr,
                                                           int64_t *__restrict__ opt, int32_t *__restrict__ status,
                                                           int64_t *__restrict__ frontier) {
  constexpr int BITS = Pow2Bits<KP>::value;
  constexpr uint32_t CAP = (1u << (32 - BITS)) - 1u;
  constexpr int NT = kMemThreads;
  constexpr int NW = NT / 64;           // waves per workgroup
  constexpr int SW = KP / NW;           // states per wave (phase A)
  constexpr int H = kMemShift, C = kMemChunk;
  constexpr int COLS = H + C;
  constexpr int BPW = C / NW;           // phase B: buckets per wave
  constexpr int LPB = 64 / BPW;         // lanes per bucket
  constexpr int SB = KP / LPB;          // states per lane
  constexpr int QS = C + 1;  // padded row stride: phase B writes several states of one bucket at once
  static_assert(SW >= 1 && SB >= 1 && BPW * NW == C && SB * LPB == KP, "work split");

  __shared__ uint32_t Q[KP][QS];       // normalised rows of the chunk's buckets
  __shared__ uint32_t P[2][KP][COLS];  // products of the step, [step parity]; columns < H: the chunk below
  __shared__ int64_t off[2][COLS];     // offsets of the previous step, [step parity]
  __shared__ __align__(16) uint8_t argb[KP][C];  // argmin bytes of the step, written back after it
  __shared__ int abort_flag;
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  __shared__ __align__(16) uint32_t rT[kMemTables][KP][KP];  // packed tables, read by broadcast

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int b = blockIdx.x % B, j = blockIdx.x / B;
  const int m0 = j * C;
  const int Bb = budget[b];
  const int mf = w.mflags[b];  // written by the prep kernel earlier in the stream
  if (mf & MEMF_BAD) {
    if (frontier && tid < C && m0 + tid < M) frontier[(size_t)b * M + m0 + tid] = INT64_MAX;
    if (j == 0 && tid == 0) {
      status[b] = CFP_ST_BADINPUT;
      opt[b] = INT64_MAX;
      res[b].final_state = -1;
      res[b].status = CFP_ST_BADINPUT;
      res[b].final_m = -1;
    }
    return;
  }
  if (m0 > Bb) return;  // no bucket of this chunk is within the budget
  const size_t rowbase = (size_t)b * N;
  int flags = 0;
  // phase B: this lane's bucket and states
  const int pc = lane % BPW, pg = lane / BPW;
  const int ml = BPW * wid + pc;  // bucket within the chunk
  const bool bact = m0 + ml <= Bb;

  for (int x = tid; x < kMemTables * KP * KP / 4; x += NT)
    ((u32x4 *)&rT[0][0][0])[x] = ((const u32x4 *)rpT)[x];
  // Chunk 0: buckets below 0 are infeasible.
  for (int x = tid; x < 2 * KP * H; x += NT) P[x / (KP * H)][(x / H) % KP][x % H] = kSat;
  if (tid < H) off[0][tid] = off[1][tid] = kOffInf;
  if (tid == 0) abort_flag = 0;

  const size_t chunk_id = (size_t)b * w.nchunk + j;
  uint32_t *my_ring = w.ring + chunk_id * N * KP * H;
  int64_t *my_roff = w.ring_off + chunk_id * N * H;
  const uint32_t *lo_ring = w.ring + (chunk_id - 1) * N * KP * H;
  const int64_t *lo_roff = w.ring_off + (chunk_id - 1) * N * H;
  const bool consumer = j > 0;

  // Phase B of step i from the values y of the lane's states: column minimum,
  // normalised rows, offsets of step i (into off[nxt]).
  // y: values of the lane's states (kSat unreachable, a reachable state at
  // most kSat - 1); rb: their records.
  uint32_t y[SB];
  uint2 rb[SB];
  auto normalise = [&](int i, int64_t od) __attribute__((always_inline)) {
    const int nxt = (i & 1) ^ 1;
    uint32_t x = y[0];
#pragma unroll
    for (int k = 1; k < SB; ++k) x = umin(x, y[k]);
#pragma unroll
    for (int o = BPW; o < 64; o *= 2) x = umin(x, (uint32_t)__shfl_xor((int)x, o, 64));
    const uint32_t cm = x;
    const bool feas = cm != kSat;
    if (feas && cm >= 0x80000000u) {  // rare: flagged at once, complete before the step is published
      flags |= MEMF_OVERFLOW;
      atomicOr(&w.mflags[b], MEMF_OVERFLOW);
      __builtin_amdgcn_s_waitcnt(0);
    }
    const int64_t onew = feas ? od + (int64_t)cm : kOffInf;
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      const int s = rb[k].x & 0xFF;
      Q[s][ml] = ((feas && y[k] != kSat) ? umin(y[k] - cm, CAP) : CAP) << BITS;
    }
    if (pg == 0) off[nxt][H + ml] = onew;
  };

  // Step 0: absolute values.
  {
    const uint2 *rec = srec + rowbase * KP + SB * pg;
#pragma unroll
    for (int k = 0; k < SB; ++k) rb[k] = rec[k];
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      const int d = (rb[k].x >> 8) & 0xFF;
      const int32_t c = (int32_t)rb[k].y;
      const bool rk = bact && m0 + ml >= d && c != CFP_COST_INF;
      y[k] = rk ? (uint32_t)c : kSat;
    }
    normalise(0, 0);
  }
  __syncthreads();

  // Slot i of this chunk's ring (P_i and the offsets of step i-1 of the top
  // buckets), read from LDS after the first barrier of step i: KP * H words,
  // one per thread when KP = 32, and the H offsets (each stored by several
  // lanes).
  constexpr int HW = KP * H / 64;
  constexpr int RPT = (KP * H + NT - 1) / NT;  // ring words per thread (repeats when fewer than NT)
  static_assert((KP * H) % NT == 0 || NT % (KP * H) == 0, "ring words split evenly");
  auto ring_store = [&](int i) __attribute__((always_inline)) {
    const int pi = i & 1;
#pragma unroll
    for (int k = 0; k < RPT; ++k) {
      const int x = (tid + NT * k) % (KP * H), st = x / H, h = x % H;
      __hip_atomic_store(&my_ring[(size_t)i * KP * H + x], P[pi][st][C + h], __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
    __hip_atomic_store(&my_roff[(size_t)i * H + (lane & (H - 1))], off[pi][C + (lane & (H - 1))], __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  };
  // Argmin bytes of step i from LDS to the table, buckets m0 .. min(m0 + C,
  // Bb + 1, M) - 1, in 16-byte pieces by the threads of waves 1 .. NW-1.
  const bool vec16 = (M % 16) == 0;
  auto flush = [&](int i) __attribute__((always_inline)) {
    for (int x = tid - 64; x >= 0 && x < KP * C / 16; x += NT - 64) {
      const int s = x / (C / 16), c0 = (x % (C / 16)) * 16;
      if (s >= K) continue;
      uint8_t *dst = table + ((rowbase + i) * K + s) * (size_t)M + m0 + c0;
      const int lim = min(Bb + 1, M) - (m0 + c0);
      if (vec16 && lim >= 16) {
        *(u32x4 *)dst = *(const u32x4 *)&argb[s][c0];
      } else {
        for (int q = 0; q < 16 && q < lim; ++q) dst[q] = argb[s][c0 + q];
      }
    }
  };

  int pubv = -1;  // wave 0: the producer's published step, read one step ahead
  if (consumer && wid == 0)
    pubv = __hip_atomic_load(&w.pub[chunk_id - 1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  for (int i = 1; i < N; ++i) {
    const int cur = i & 1;
    // Phase A.  Memory operations in issue order: the phase B records of the
    // step (all waves), then the halo loads of wave 0 when slot i is already
    // published (else it waits for it after its products), then the ring
    // stores of the last wave; so no wait for a load covers a store.
    {
      const uint2 *rec = srec + (rowbase + i) * KP + SB * pg;
#pragma unroll
      for (int k = 0; k < SB; ++k) rb[k] = rec[k];
    }
    uint32_t hq[HW];
    int64_t ho = kOffInf;
    bool early = false;
    if (consumer && wid == 0) {
      early = pubv >= i;
      if (early) {
#pragma unroll
        for (int k = 0; k < HW; ++k)
          hq[k] = __hip_atomic_load(&lo_ring[(size_t)i * KP * H + lane + 64 * k], __ATOMIC_RELAXED,
                                    __HIP_MEMORY_SCOPE_AGENT);
        if (lane < H) ho = __hip_atomic_load(&lo_roff[(size_t)i * H + lane], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    const int e = redge[i];
    {
      uint32_t A[KP];
#pragma unroll
      for (int t = 0; t < KP; ++t) A[t] = Q[t][lane];
      const uint2 *rec = srec + (rowbase + i) * KP + SW * wid;
#pragma unroll
      for (int k = 0; k < SW; ++k) {
        const int s = rec[k].x & 0xFF;
        uint32_t colc[KP];
#pragma unroll
        for (int q = 0; q < KP / 4; ++q) {
          const u32x4 v = ((const u32x4 *)&rT[e][s][0])[q];
          colc[4 * q] = v.x;
          colc[4 * q + 1] = v.y;
          colc[4 * q + 2] = v.z;
          colc[4 * q + 3] = v.w;
        }
        uint32_t acc = sat_add(A[0], colc[0]);
#pragma unroll
        for (int t = 1; t < KP; ++t) acc = umin(acc, sat_add(A[t], colc[t]));
        P[cur][s][H + lane] = acc;
      }
    }
    if (consumer && wid == 0) {
      if (!early) {
        int spins = 0;
        while (__hip_atomic_load(&w.pub[chunk_id - 1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < i) {
          if (++spins > kSpinLimit) {
            if (lane == 0) abort_flag = 1;
            flags |= MEMF_TIMEOUT;
            atomicOr(&w.mflags[b], MEMF_TIMEOUT);
            break;
          }
          __builtin_amdgcn_s_sleep(1);
        }
#pragma unroll
        for (int k = 0; k < HW; ++k)
          hq[k] = __hip_atomic_load(&lo_ring[(size_t)i * KP * H + lane + 64 * k], __ATOMIC_RELAXED,
                                    __HIP_MEMORY_SCOPE_AGENT);
        if (lane < H) ho = __hip_atomic_load(&lo_roff[(size_t)i * H + lane], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
#pragma unroll
      for (int k = 0; k < HW; ++k) {
        const int x = lane + 64 * k;
        P[cur][x / H][x % H] = hq[k];
      }
      if (lane < H) off[cur][lane] = ho;
    }
    __syncthreads();
    ring_store(i);

    // Phase B.
    {
      const int64_t od = off[cur][H + ml];
#pragma unroll
      for (int k = 0; k < SB; ++k) {
        const int s = rb[k].x & 0xFF;
        const int d = (rb[k].x >> 8) & 0xFF;
        const int32_t c = (int32_t)rb[k].y;
        const uint32_t pv = P[cur][s][H + ml - d];
        const int64_t os = off[cur][H + ml - d];
        const bool srcok = os < kOffInf;
        const int64_t g = srcok ? os - od : 0;
        const uint32_t goff = g > 0x7FFFFFFF ? 0x80000000u : (uint32_t)g;
        argb[s][ml] = (uint8_t)pv;
        const uint32_t v = pv >> BITS;
        const bool rk = bact && srcok && v < CAP && c != CFP_COST_INF;
        y[k] = rk ? umin(sat_add(sat_add(v, (uint32_t)c), goff), kSat - 1) : kSat;
      }
      normalise(i, od);
    }
    if (consumer && wid == 0 && i + 1 < N)
      pubv = __hip_atomic_load(&w.pub[chunk_id - 1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __builtin_amdgcn_s_waitcnt(0);  // the ring stores of slot i are complete
    __syncthreads();
    if (tid == 64 * (NW - 1)) __hip_atomic_store(&w.pub[chunk_id], i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    flush(i);
  }
  const int fin = N & 1;  // off buffer holding the last step's offsets
  const int m = m0 + lane;
  const bool active = m <= Bb;

  // Budget frontier: the exact offset of column m is min_s D[N-1][s][m], the
  // least cost with memory total at most m.
  if (frontier && wid == 0 && m < M)
    frontier[(size_t)b * M + m] = (active && off[fin][H + lane] < kOffInf) ? off[fin][H + lane] : INT64_MAX;

  // The chunk holding the budget bucket reports the search.
  if (abort_flag) flags |= MEMF_TIMEOUT;
  if (Bb >= m0 && Bb < m0 + C) {
    const int col = Bb - m0;
    if (tid == 0) {
      uint32_t f = kSat;
      for (int s = 0; s < K; ++s) f = umin(f, Q[s][col] | (uint32_t)s);
      const int64_t o = off[fin][H + col];
      const int sf = __hip_atomic_load(&w.mflags[b], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) | flags;
      int st = CFP_ST_OK;
      if (abort_flag || (sf & MEMF_TIMEOUT)) st = CFP_ST_TIMEOUT;
      else if (sf & MEMF_OVERFLOW) st = CFP_ST_OVERFLOW;
      else if (hdr->rflag) st = CFP_ST_BADINPUT;
      else if (o >= kOffInf) st = CFP_ST_INFEASIBLE;
      else if ((f >> BITS) != 0) st = CFP_ST_OVERFLOW;
      status[b] = st;
      opt[b] = st == CFP_ST_OK ? o : INT64_MAX;
      res[b].final_state = st == CFP_ST_OK ? (int32_t)(f & ((1u << BITS) - 1u)) : -1;
      res[b].status = st;
      res[b].final_m = Bb;
    }
  }
}

// Plan recovery for the memory variant.  The state is (s, m): the table gives
// the predecessor strategy t = arg[i][s][m] and the budget shrinks by
// mem[i][s].  The chase runs in windows of kMemWin steps: the argmin rows of
// the window are loaded into LDS for the only buckets it can reach,
// [m - kMemShift*(kMemWin-1), m], then one thread follows them.
constexpr int kMemWin = 12;
constexpr int kMemWinWidth = (kMemShift * (kMemWin - 1) + 16 + 15) / 16 * 16;  // covers [lo & ~15, top]

__device__ __forceinline__ int mem_index_bits(int k) {
  int b = 4;
  while ((1 << b) < k) ++b;
  return b;
}

constexpr int kMemTbThreads = 1024;  // every 16-byte piece of a window in flight at once
constexpr int kMemTbLoads = 8;       // pieces per thread and pass

__global__ __launch_bounds__(kMemTbThreads) void mem_tb_kernel(int N, int K, int M, const uint8_t *__restrict__ table,
                                                          const uint8_t *__restrict__ mem_copy,
                                                          const SearchResult *__restrict__ res,
                                                          int32_t *__restrict__ plan) {
  // window rows are 16-byte aligned copies of [lo16, lo16 + width) of a table row
  extern __shared__ __align__(16) uint8_t win[];  // [kMemWin][K][width] then mem rows [kMemWin][K]
  __shared__ int cur_s, cur_m;
  const int b = blockIdx.x, tid = threadIdx.x;
  int32_t *pb = plan + (size_t)b * N;
  if (res[b].status != CFP_ST_OK) {
    for (int i = tid; i < N; i += blockDim.x) pb[i] = -1;
    return;
  }
  const int mask = (1 << mem_index_bits(K)) - 1;
  const int width = kMemWinWidth;
  uint8_t *mrow = win + (size_t)kMemWin * K * width;
  const bool vec = (M % 16) == 0;
  if (tid == 0) {
    cur_s = res[b].final_state;
    cur_m = res[b].final_m;
    pb[N - 1] = cur_s;
  }
  __syncthreads();
  for (int i = N - 1; i >= 1;) {
    const int steps = i < kMemWin ? i : kMemWin;
    const int mtop = cur_m;
    const int lo = mtop - kMemShift * (steps - 1) > 0 ? mtop - kMemShift * (steps - 1) : 0;
    const int lo16 = lo & ~15;
    const int n16 = (mtop - lo16) / 16 + 1;  // 16-byte pieces covering [lo16, mtop]
    if (vec) {
      // all pieces of a pass are loaded before any is stored, so the window
      // costs about one memory latency
      const int total = steps * K * n16;
      for (int x0 = 0; x0 < total; x0 += kMemTbLoads * kMemTbThreads) {
        typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));  // copies stay in registers
        u32x4 v[kMemTbLoads];
#pragma unroll
        for (int u = 0; u < kMemTbLoads; ++u) {
          const int x = x0 + u * kMemTbThreads + tid;
          const int k = x / (K * n16), t = (x / n16) % K, c = x % n16;
          if (x < total)
            v[u] = *(const u32x4 *)&table[(((size_t)b * N + (i - k)) * K + t) * M + lo16 + 16 * c];
        }
#pragma unroll
        for (int u = 0; u < kMemTbLoads; ++u) {
          const int x = x0 + u * kMemTbThreads + tid;
          const int k = x / (K * n16), t = (x / n16) % K, c = x % n16;
          if (x < total) *(u32x4 *)&win[((size_t)k * K + t) * width + 16 * c] = v[u];
        }
      }
    } else {
      const int wd = mtop - lo16 + 1;
      const int total = steps * K * wd;
      for (int x0 = 0; x0 < total; x0 += 16 * kMemTbThreads) {
        uint8_t v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          const int x = x0 + u * kMemTbThreads + tid;
          const int k = x / (K * wd), t = (x / wd) % K, c = x % wd;
          v[u] = x < total ? table[(((size_t)b * N + (i - k)) * K + t) * M + lo16 + c] : 0;
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          const int x = x0 + u * kMemTbThreads + tid;
          const int k = x / (K * wd), t = (x / wd) % K, c = x % wd;
          if (x < total) win[((size_t)k * K + t) * width + c] = v[u];
        }
      }
    }
    for (int x = tid; x < steps * K; x += blockDim.x)
      mrow[x] = mem_copy[((size_t)b * N + (i - x / K)) * K + x % K];
    __syncthreads();
    if (tid == 0) {
      int s = cur_s, m = mtop;
      for (int k = 0; k < steps; ++k) {
        int t = win[((size_t)k * K + s) * width + (m - lo16)] & mask;
        if (t >= K) t = K - 1;
        m -= mrow[k * K + s];
        if (m < lo) m = lo;  // cannot happen on a consistent table; stay inside the window
        pb[i - k - 1] = t;
        s = t;
      }
      cur_s = s;
      cur_m = m;
    }
    __syncthreads();
    i -= steps;
  }
}

hipError_t launch_traceback_mem(int n, int k, int batch, int n_mem, const uint8_t *table, const uint8_t *mem,
                                const SearchResult *res, int32_t *plan, hipStream_t st) {
  const size_t lds = (size_t)kMemWin * k * kMemWinWidth + (size_t)kMemWin * k;
  hipLaunchKernelGGL(mem_tb_kernel, dim3(batch), dim3(kMemTbThreads), lds, st, n, k, n_mem, table, mem, res, plan);
  return hipGetLastError();
}

size_t mem_region_bytes(int n, int k, int batch, int n_mem) {
  const int KP = k <= 16 ? 16 : 32;
  const int nchunk = (n_mem + kMemChunk - 1) / kMemChunk;
  size_t off = 0;
  off = align_up(off + (size_t)batch * n * KP * 8);  // srec
  off = align_up(off + (size_t)12 * KP * KP * 4);    // rpT (tables beyond 12 are rejected)
  off = align_up(off + (size_t)batch * 4);           // mflags
  off = align_up(off + (size_t)batch * nchunk * 4);  // pub
  off = align_up(off + (size_t)batch * nchunk * n * KP * kMemShift * 4);
  off = align_up(off + (size_t)batch * nchunk * n * kMemShift * 8);
  return off;
}

static MemWs carve(uint8_t *region, int n, int k, int batch, int n_mem) {
  const int KP = k <= 16 ? 16 : 32;
  MemWs w;
  w.nchunk = (n_mem + kMemChunk - 1) / kMemChunk;
  size_t off = 0;
  w.srec = (uint2 *)(region + off); off = align_up(off + (size_t)batch * n * KP * 8);
  w.rpT = (uint32_t *)(region + off); off = align_up(off + (size_t)12 * KP * KP * 4);
  w.mflags = (int32_t *)(region + off); off = align_up(off + (size_t)batch * 4);
  w.pub = (int32_t *)(region + off); off = align_up(off + (size_t)batch * w.nchunk * 4);
  w.ring = (uint32_t *)(region + off); off = align_up(off + (size_t)batch * w.nchunk * n * KP * kMemShift * 4);
  w.ring_off = (int64_t *)(region + off);
  return w;
}

__global__ void mem_init_kernel(int32_t *mflags, int nb, int32_t *pub, int np) {
  for (int x = blockIdx.x * blockDim.x + threadIdx.x; x < nb + np; x += gridDim.x * blockDim.x) {
    if (x < nb) mflags[x] = 0;
    else pub[x - nb] = -1;
  }
}

template <int KP>
static void launch_mem(const cfp_chain_desc &d, const uint8_t *mem, int n_mem, const int32_t *budget,
                       const int32_t *redge_dev, uint8_t *table, uint8_t *mem_copy, uint8_t *region,
                       SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status, int64_t *frontier,
                       hipStream_t st) {
  const int N = d.n_blocks, K = d.k, B = d.batch, E = d.n_tables;
  MemWs w = carve(region, N, K, B, n_mem);
  hipLaunchKernelGGL(mem_init_kernel, dim3(64), dim3(256), 0, st, w.mflags, B, w.pub, B * w.nchunk);
  hipLaunchKernelGGL(mem_pack_rtab_kernel<KP>, dim3((E * KP * KP + 255) / 256), dim3(256), 0, st, d.rtab, E, K, w.rpT,
                     cfp_r_limit(CFP_V_MEM, K), const_cast<WsHeader *>(hdr));
  hipLaunchKernelGGL(mem_prep_kernel<KP>, dim3((B * N + 3) / 4), dim3(256), 0, st, d.cost, mem, budget, N, K, n_mem, B,
                     w.srec, mem_copy, w.mflags);
  timer_begin(st);
  timed_launch(mem_fwd_kernel<KP>, dim3(B * w.nchunk), dim3(kMemThreads), 0, st, redge_dev, budget,
               (const uint2 *)w.srec, (const uint32_t *)w.rpT, N, K, n_mem, B, w, table, res, hdr, opt, status, frontier);
  timer_end(st);
}

bool chain_mem_supported(int k, int n_tables) { return k <= 32 && n_tables <= 12; }

hipError_t launch_chain_mem_fwd(const cfp_chain_desc &d, const uint8_t *mem, int n_mem, const int32_t *budget,
                                const int32_t *redge_dev, uint8_t *table, uint8_t *mem_copy, uint8_t *region,
                                SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status,
                                int64_t *frontier, hipStream_t st) {
  if (d.k <= 16)
    launch_mem<16>(d, mem, n_mem, budget, redge_dev, table, mem_copy, region, res, hdr, opt, status, frontier, st);
  else
    launch_mem<32>(d, mem, n_mem, budget, redge_dev, table, mem_copy, region, res, hdr, opt, status, frontier, st);
  return hipGetLastError();
}

__global__ void fill_i32_kernel(int32_t *p, int n, int32_t v) {
  for (int x = blockIdx.x * blockDim.x + threadIdx.x; x < n; x += gridDim.x * blockDim.x) p[x] = v;
}

hipError_t launch_fill_i32(int32_t *p, int n, int32_t v, hipStream_t st) {
  hipLaunchKernelGGL(fill_i32_kernel, dim3((n + 255) / 256 < 64 ? (n + 255) / 256 : 64), dim3(256), 0, st, p, n, v);
  return hipGetLastError();
}

}  // namespace cfp
