// Search under a memory budget (Sec. 4.4: least Eq. T cost with Eq. M within
// the memory limit, memory quantised into buckets):
//     D[0][s][m] = c[0][s]                                   if mem[0][s] <= m
//     D[i][s][m] = c[i][s] + min_t D[i-1][t][m - mem[i][s]] + R_{e(i)}[t][s]
// with D = +inf where m < mem[i][s]; the answer is min_s D[N-1][s][budget].
// D[i][s][m] is the least cost of a prefix whose memory total is at most m,
// so it does not increase with m.
//
// Product then shift.  A state s with memory shift d = mem[i][s] takes its
// candidates from column m - d, so
//     D[i][s][m] = c[i][s] + P[s][m - d],   P[s][m'] = min_t D[i-1][t][m'] + R[t][s]:
// a step is one min-plus product of the previous rows (buckets x states) with
// the K x K table, followed by a per-state shift of the product along m.
//
// Layout.  The buckets of a search are cut into chunks of 64; one workgroup
// computes one chunk for all states with four compute waves, a loading wave
// and a storing wave (the compute waves issue no global stores, so none of
// their waits for a load ever covers a store).  Compute wave w owns buckets
// 16w .. 16w+15 of its chunk, lane (g, m) = (lane / 16, lane % 16) the bucket
// 16w + m and the K/4 states g K/4 .. g K/4 + K/4 - 1.  The previous row of a
// bucket sits in registers (32 predecessors at a time), and the table entry
// R[t][s] of predecessor t = 16q + j reaches every lane of a row of 16 through
// a DPP row broadcast of lane j of a register that holds R[16q .. 16q+15][s]
// in that row: a candidate is one add with a DPP operand, two candidates one
// three-input minimum.  The tables stream from the L2 cache, each lane loading
// the 16 entries of its row's state, a few items ahead.
// Step i of bucket m reads products at m - d >= m - 16, i.e. of the wave below
// (through a product buffer in LDS) or, for wave 0, of the top 16 buckets of
// the chunk below, which that chunk's storing wave passes through a ring of
// eight slots in device memory together with its offsets.  The loading wave
// fetches the slots and stages the next step's per-state records (and, for
// K <= 64, the step's table) in LDS; the storing wave writes the ring slots,
// the publication counter and the argmin bytes of earlier steps.  Every ring word carries
// the number of its step in its upper half, so no store is ever waited for:
// the chunk above loads a slot ahead of the step that needs it and reloads it
// until every word has the step's number; a chunk waits before
// reusing a slot until the chunk above has consumed it (all waits bounded).
// The chunks of one launch are resident together (the host launches the
// searches in rounds that fit), so the ring stays in the L2 cache.
//
// Arithmetic.  Bucket m carries an exact int64 offset o[m] = min_s D[s][m];
// the row is kept as Q[s][m] = min(D[s][m] - o[m], QCAP) << b with
// QCAP = 2^(31-b) and b index bits, and the packed table words as
// (R << b) | t with R < 2^(31-b), so a candidate Q + R never leaves 32 bits
// and one unsigned minimum yields the value and the lowest argmin.  The best
// candidate of a column with a finite offset is at most R_max < QCAP (through
// the column's minimum state), so capped states never win.
// The new value of state s at bucket m is, relative to the offset
// o[m - dmin] of the least shift dmin over the block's available states,
//     y[s] = c[s] + P[s][m - d] + (o[m - d] - o[m - dmin]),
// where the bracket is >= 0 because o does not increase with m.  A state with
// shift dmin has y < 2^31 + R_max, so y is computed in saturating 32-bit
// arithmetic: the column minimum cm = min_s y[s] is exact, the new offset is
// o[m - dmin] + cm, and a saturated y exceeds cm by more than QCAP.
#include <algorithm>
#include <mutex>

#include "cfp_internal.h"
#include "common.h"

namespace cfp {

constexpr int kMemChunk = 64;        // buckets per workgroup
constexpr int kMemShift = 16;        // largest supported mem entry = halo width = buckets per wave
constexpr int kMemBlocks = 4;        // bucket blocks of 16 per chunk
constexpr int kMemSlots = 8;         // ring slots per chunk
constexpr int kMemFlagStride = 16;   // ints per chunk flag (one 64-byte line each)
constexpr int kMemMaxK = 256;
constexpr int kMemPD = 4;            // table items loaded ahead
// Ring slot of KP states: the top 16 buckets' products of all states, then
// their offsets as two halves, every word tagged with its step.
constexpr int mem_slot_words(int kp) { return 16 * kp + 32; }
constexpr int64_t kOffInf = (int64_t)1 << 62;
constexpr int kSpinLimit = 1 << 20;

enum { MEMF_BAD = 1, MEMF_TIMEOUT = 2 };

template <int KP>
struct MemShape {
  static constexpr int BITS = KP <= 32 ? 5 : KP <= 64 ? 6 : KP <= 128 ? 7 : 8;
  static constexpr bool ALIAS = KP > 128;   // rows kept in the product buffer, single-buffered
  static constexpr int CW = kMemBlocks;     // compute waves, one per bucket block
  static constexpr int THREADS = 64 * (CW + 2);    // and a loading and a storing wave
  static constexpr int SPL = KP / 4;        // states per lane
  static constexpr int TB = KP / 32;        // blocks of 32 predecessors
  static constexpr bool RLDS = KP <= 64;    // tables staged in LDS by the loading wave
  static constexpr int SP = kMemShift + kMemChunk + 1;  // product buffer row stride (words)
  static constexpr int QS = KP + 4;         // row stride of a wave's rows (words)
  static constexpr uint32_t QCAP = 1u << (31 - BITS);
  static constexpr uint32_t MASK = (1u << BITS) - 1u;
  static_assert(SPL % kMemPD == 0 && SPL % 4 == 0 && SPL % 2 == 0, "items and record words per lane");
};

static int mem_kp(int k) { return k <= 32 ? 32 : k <= 64 ? 64 : k <= 96 ? 96 : k <= 128 ? 128 : k <= 192 ? 192 : 256; }
static int mem_bits(int k) { return k <= 32 ? 5 : k <= 64 ? 6 : k <= 128 ? 7 : 8; }

// Per-(search, block) records: cost cst[s] (kSat for an unavailable or
// padding state), shift dsh[s], the least shift dmin over the available
// states; a copy of mem for the traceback; validation of mem, the costs and
// the budget.  One wave per (b, i) row.
__global__ __launch_bounds__(256) void mem_prep_kernel(const int32_t *__restrict__ cost, const uint8_t *__restrict__ mem,
                                                       const int32_t *__restrict__ budget, int N, int K, int KP, int M,
                                                       int B, uint32_t *__restrict__ cst, uint8_t *__restrict__ dsh,
                                                       int32_t *__restrict__ dmin, uint8_t *__restrict__ mem_copy,
                                                       int32_t *__restrict__ mflags) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= B * N) return;
  const int b = row / N;
  const size_t base = (size_t)row * K;
  bool bad = false;
  int dm = kMemShift + 1;
  for (int s = lane; s < KP; s += 64) {
    uint32_t c = kSat;
    int d = 0;
    if (s < K) {
      d = mem[base + s];
      const int32_t cv = cost[base + s];
      mem_copy[base + s] = (uint8_t)d;
      bad |= d >= M || d > kMemShift || cv < 0;
      if (d > kMemShift) d = kMemShift;
      if (cv >= 0 && cv != CFP_COST_INF) {
        c = (uint32_t)cv;
        dm = min(dm, d);
      }
    }
    cst[(size_t)row * KP + s] = c;
    dsh[(size_t)row * KP + s] = (uint8_t)d;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) dm = min(dm, __shfl_xor(dm, o, 64));
  if (lane == 0) dmin[row] = dm > kMemShift ? 0 : dm;  // a block with no available state: every y saturates
  if (lane == 0 && (row % N) == 0 && (budget[b] < 0 || budget[b] >= M)) bad = true;
  if (__any(bad) && lane == 0) atomicOr(&mflags[b], MEMF_BAD);
}

// Packed tables, state-major: rT[e][s][t] = (R[e][t][s] << b) | t.  A padding
// predecessor or state gets ((QCAP - 1) << b) | t: with the capped row value
// QCAP its candidate is the largest value that fits, above every candidate
// through a column's minimum state.  Every R entry is read here, so the range
// check (entries in [0, 2^(31-b))) is made on the way and flagged in the header.
__global__ void mem_pack_rtab_kernel(const int32_t *__restrict__ rtab, int E, int K, int KP, int bits,
                                     uint32_t *__restrict__ rT, int32_t limit, WsHeader *__restrict__ hdr) {
  const size_t total = (size_t)E * KP * KP;
  const uint32_t pad = (((1u << (31 - bits)) - 1u) << bits);
  for (size_t x = blockIdx.x * (size_t)blockDim.x + threadIdx.x; x < total; x += (size_t)gridDim.x * blockDim.x) {
    const int t = (int)(x % KP), s = (int)((x / KP) % KP), e = (int)(x / ((size_t)KP * KP));
    uint32_t v = pad | (uint32_t)t;
    if (s < K && t < K) {
      const int32_t r = rtab[((size_t)e * K + t) * K + s];
      if (r < 0 || r >= limit) hdr->rflag = 1;
      v = ((uint32_t)r << bits) | (uint32_t)t;
    }
    rT[x] = v;
  }
}

struct MemWs {
  uint32_t *cst;       // [B][N][KP]
  uint8_t *dsh;        // [B][N][KP]
  int32_t *dmin;       // [B][N]
  uint32_t *rT;        // [E][KP][KP]
  int32_t *mflags;     // [B]
  int32_t *cons;       // [B][nchunk] (stride kMemFlagStride): last step whose slot a chunk has consumed
  uint64_t *ring;      // [B][nchunk][kMemSlots][mem_slot_words(KP)]: word | step << 32
  int nchunk;
};

struct MemArgs {
  const int32_t *budget;
  MemWs w;
  int N, K, M, B;
  int b0, nb, B8;        // searches b0 .. b0+nb-1 of this launch; grid = nchunk * B8
  uint8_t *table;        // [B][N][K][M]
  SearchResult *res;
  const WsHeader *hdr;
  int64_t *opt;
  int32_t *status;
  int64_t *frontier;     // [B][M] or null
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// a = min(a, ra[j] + q_j) and b = min(b, rb[j] + q_j) for predecessors
// j = J0 .. J0+3 of a row of 16, where r[j] is lane j of r's row (a DPP row
// broadcast): two states at once, so that no instruction needs the result of
// the one before it (a wave alone on its SIMD would otherwise wait for it).
// NOP: the first block reading ra and rb, which waits the two states a DPP
// read of a fresh VALU result needs.
#define CFP_M_ADD(T, R, Q, J) "v_add_u32_dpp " T ", " R ", " Q " row_newbcast:" J " row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
template <int J0, bool NOP>
__device__ __forceinline__ void mcand4x2(uint32_t &a, uint32_t &b, uint32_t ra, uint32_t rb, uint32_t q0, uint32_t q1,
                                         uint32_t q2, uint32_t q3) {
  uint32_t t0, t1, t2, t3;
  asm(".if %[nop]\n s_nop 1\n .endif\n"
      CFP_M_ADD("%[t0]", "%[ra]", "%[q0]", "%[j0]")
      CFP_M_ADD("%[t1]", "%[ra]", "%[q1]", "%[j1]")
      CFP_M_ADD("%[t2]", "%[rb]", "%[q0]", "%[j0]")
      CFP_M_ADD("%[t3]", "%[rb]", "%[q1]", "%[j1]")
      "v_min3_u32 %[a], %[a], %[t0], %[t1]\n"
      "v_min3_u32 %[b], %[b], %[t2], %[t3]\n"
      CFP_M_ADD("%[t0]", "%[ra]", "%[q2]", "%[j2]")
      CFP_M_ADD("%[t1]", "%[ra]", "%[q3]", "%[j3]")
      CFP_M_ADD("%[t2]", "%[rb]", "%[q2]", "%[j2]")
      CFP_M_ADD("%[t3]", "%[rb]", "%[q3]", "%[j3]")
      "v_min3_u32 %[a], %[a], %[t0], %[t1]\n"
      "v_min3_u32 %[b], %[b], %[t2], %[t3]\n"
      : [a] "+v"(a), [b] "+v"(b), [t0] "=&v"(t0), [t1] "=&v"(t1), [t2] "=&v"(t2), [t3] "=&v"(t3)
      : [ra] "v"(ra), [rb] "v"(rb), [q0] "v"(q0), [q1] "v"(q1), [q2] "v"(q2), [q3] "v"(q3), [j0] "i"(J0),
        [j1] "i"(J0 + 1), [j2] "i"(J0 + 2), [j3] "i"(J0 + 3), [nop] "i"(NOP ? 1 : 0));
}
#undef CFP_M_ADD

// Minimum over the four rows of a wave (lanes m, m+16, m+32, m+48); every
// lane gets its bucket's minimum.
__device__ __forceinline__ uint32_t rows_min(uint32_t x) {
  const auto h = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  const uint32_t z = umin(h[0], h[1]);
  const auto q = __builtin_amdgcn_permlane16_swap(z, z, false, false);
  return umin(q[0], q[1]);
}

__device__ __forceinline__ bool spin_until(const int32_t *flag, int target, int &seen) {
  int spins = 0;
  while (seen < target) {
    if (++spins > kSpinLimit) return false;
    __builtin_amdgcn_s_sleep(1);
    seen = __hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  return true;
}

// Work split.  Compute wave w owns bucket block w of the chunk (buckets
// 16w .. 16w+15); its lane (g, m) has bucket 16w + m and the K/4 states of row
// g.  (Two waves per block, each with half of the states, were measured
// slower: the products already keep a SIMD's vector unit busy, and the pair
// costs two more barriers per step.)  Of the two I/O waves one does
// every global load of a step (the chunk below's top products into the halo
// columns, the next steps' tables and records into LDS) and one every global
// store (the chunk's top products to the ring for the chunk above, the argmin
// bytes to the table).  Loads and stores of one wave complete in order, so a
// wave that both stored and loaded would wait for its stores whenever it
// needed a load; the compute waves issue no global stores at all and, when
// the tables fit in LDS (K <= 64), no global loads either.
//
// Barriers of step i (P_i: products of step i, o_i: offsets after step i):
//   compute: products from Q_{i-1} and the table of step i -> P_i      | B
//            shifted products, offset gaps, bucket minima -> Q_i, o_i,
//            argmin bytes of step i (K > 128: the rows overwrite the
//            products, after a second barrier B2)
//   I/O, between the previous step's last barrier and B: halo of step i
//            (slot i of the chunk below: P_i and o_{i-1} of its top
//            buckets), table and records of step i+1, slot i-1 of this
//            chunk (P_{i-1}, o_{i-2}), argmin bytes of step i-2 (K > 128:
//            of step i-1, and slot i between B and B2, before the rows
//            overwrite P_i).
// The edge map and the least shifts are read through restrict-qualified
// arguments, so that their uniform per-step loads are scalar loads.
template <int KP>
__global__ __launch_bounds__(MemShape<KP>::THREADS) void mem_fwd_kernel(MemArgs a, const int32_t *__restrict__ redge,
                                                                        const int32_t *__restrict__ dmin) {
  using S = MemShape<KP>;
  constexpr int BITS = S::BITS, SPL = S::SPL, TB = S::TB, H = kMemShift, C = kMemChunk, SP = S::SP;
  constexpr uint32_t QCAP = S::QCAP;
  constexpr bool ALIAS = S::ALIAS, RLDS = S::RLDS;
  constexpr int CW = S::CW;
  constexpr int FL = ALIAS ? 1 : 2;  // the argmin bytes of step t are written back during step t + FL
  constexpr int NPB = ALIAS ? 1 : 2;
  constexpr int PD = kMemPD;
  constexpr int NBK = kMemBlocks;

  __shared__ uint32_t Pb[NPB][KP][SP];                                         // products (and, ALIAS, rows)
  __shared__ __align__(16) uint32_t Qw[ALIAS ? 1 : NBK][ALIAS ? 1 : 16][ALIAS ? 4 : S::QS];  // rows
  __shared__ int64_t offs[2][H + C];                                           // offsets by step parity
  __shared__ __align__(16) uint8_t argb[2][NBK][KP][16];                       // argmin bytes by step parity
  __shared__ __align__(16) uint32_t rbuf[RLDS ? 2 : 1][RLDS ? KP : 1][RLDS ? KP : 4];  // tables by step parity
  __shared__ __align__(16) uint32_t rcost[2][KP];                             // records by step parity
  __shared__ __align__(16) uint8_t rshift[2][KP];
  __shared__ int rdmin[2];
  __shared__ int s_timeout;
  __shared__ int s_done;    // last step whose halo slot was taken (loading wave -> storing wave)
  __shared__ int s_upcons;  // progress of the chunk above, as last read by the loading wave

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool io = w >= CW;
  const int blk = w;  // compute waves: bucket block
  const int g = lane >> 4, m = lane & 15;
  const int col = H + 16 * blk + m;  // compute waves: this lane's column

  const int bl = blockIdx.x % a.B8, j = blockIdx.x / a.B8;
  if (bl >= a.nb) return;
  const int b = a.b0 + bl;
  const int N = a.N, K = a.K, M = a.M;
  const int m0 = j * C;
  const int bucket = m0 + 16 * blk + m;
  const MemWs &W = a.w;

  if (W.mflags[b] & MEMF_BAD) {  // written by the prep kernel earlier in the stream
    if (a.frontier && !io && g == 0 && bucket < M) a.frontier[(size_t)b * M + bucket] = INT64_MAX;
    if (j == 0 && tid == 0) {
      a.status[b] = CFP_ST_BADINPUT;
      a.opt[b] = INT64_MAX;
      a.res[b].final_state = -1;
      a.res[b].status = CFP_ST_BADINPUT;
      a.res[b].final_m = -1;
    }
    return;
  }
  const int Bb = a.budget[b];
  const int top = min(Bb, M - 1);
  if (m0 > top) return;  // no bucket of this chunk is within the budget
  const bool has_consumer = m0 + C <= top;
  const bool consumer = j > 0;
  const size_t chunk_id = (size_t)b * W.nchunk + j;
  const size_t rowbase = (size_t)b * N;
  const bool vec16 = (M % 16) == 0;
  if (tid == 0) s_timeout = 0;


  if (io) {
    // ------------------------------------------------------------ I/O waves --
    const bool loader = w == CW;
    const size_t lo_id = consumer ? chunk_id - 1 : chunk_id;
    const size_t up_id = has_consumer ? chunk_id + 1 : chunk_id;
    int32_t *my_cons = W.cons + chunk_id * kMemFlagStride;
    const int32_t *up_cons = W.cons + up_id * kMemFlagStride;
    constexpr int SW = mem_slot_words(KP);
    uint64_t *my_ring = W.ring + chunk_id * kMemSlots * SW;
    const uint64_t *lo_ring = W.ring + lo_id * kMemSlots * SW;
    constexpr int HW = KP * 16 / 64;       // product words of a slot per lane
    constexpr int HB = 8;                  // words per lane moved at once (HW is a multiple of 8)
    static_assert(HW % HB == 0, "slot words per lane in whole blocks");
    constexpr int RW = RLDS ? KP * KP / 256 : 1;  // 16-byte table pieces per lane
    bool timeout = false;

    if (loader) {
      u32x4 rv[RW];
      auto load_table = [&](int e) __attribute__((always_inline)) {
        if constexpr (RLDS) {
          const u32x4 *src = (const u32x4 *)(W.rT + (size_t)e * KP * KP);
#pragma unroll
          for (int u = 0; u < RW; ++u) rv[u] = src[lane + 64 * u];
        }
      };
      auto store_table = [&](int par) __attribute__((always_inline)) {
        if constexpr (RLDS) {
#pragma unroll
          for (int u = 0; u < RW; ++u) ((u32x4 *)&rbuf[par][0][0])[lane + 64 * u] = rv[u];
        }
      };
      // records of step t into parity buffer t & 1: KP costs and KP shift bytes,
      // four per lane, and the least shift
      auto stage_records = [&](int t, const u32x4 &c4, uint32_t s4, int dmt) __attribute__((always_inline)) {
        if (lane < KP / 4) {
          *(u32x4 *)&rcost[t & 1][4 * lane] = c4;
          *(uint32_t *)&rshift[t & 1][4 * lane] = s4;
        }
        if (lane == 0) rdmin[t & 1] = dmt;
      };
      auto load_records = [&](int t, u32x4 &c4, uint32_t &s4) __attribute__((always_inline)) {
        if (lane < KP / 4) {
          c4 = *(const u32x4 *)(W.cst + (rowbase + t) * KP + 4 * lane);
          s4 = *(const uint32_t *)(W.dsh + (rowbase + t) * KP + 4 * lane);
        }
      };
      if (N > 1) {  // the table and the records of step 1
        if (RLDS) load_table(redge[1]);
        u32x4 c4 = {};
        uint32_t s4 = 0;
        load_records(1, c4, s4);
        if (RLDS) store_table(1);
        stage_records(1, c4, s4, dmin[rowbase + 1]);
      }
      if (lane == 0) {
        s_done = -1;
        s_upcons = -1;
      }
      __syncthreads();  // step 0 of the compute waves
      for (int i = 1; i < N; ++i) {
        const int par = i & 1, pprev = par ^ 1;
        const int pb = ALIAS ? 0 : par;
        const uint64_t *src = lo_ring + (size_t)(i % kMemSlots) * SW;
        uint64_t hv[HB];
        uint64_t ho = (uint64_t)i << 32;
        auto load_block = [&](int u0) __attribute__((always_inline)) {
#pragma unroll
          for (int u = 0; u < HB; ++u)
            hv[u] = __hip_atomic_load(src + lane + 64 * (u0 + u), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        };
        auto block_fresh = [&]() __attribute__((always_inline)) {
          bool ok = true;
#pragma unroll
          for (int u = 0; u < HB; ++u) ok &= (uint32_t)(hv[u] >> 32) == (uint32_t)i;
          return ok;
        };
        if (consumer) {
          load_block(0);
          if (lane < 32) ho = __hip_atomic_load(src + 16 * KP + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (RLDS && i + 1 < N) load_table(redge[i + 1]);
        u32x4 cpc = {};  // records of step i + 1
        uint32_t spc = 0;
        if (i + 1 < N) load_records(i + 1, cpc, spc);
        const int dmi = i + 1 < N ? dmin[rowbase + i + 1] : 0;
        int upc = -1;
        if (has_consumer) upc = __hip_atomic_load(up_cons, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

        if (consumer) {  // every word of slot i must carry the step's number (bounded reloads)
          for (int u0 = 0; u0 < HW; u0 += HB) {
            if (u0 > 0) load_block(u0);
            bool ok = block_fresh() && (u0 > 0 || (uint32_t)(ho >> 32) == (uint32_t)i);
            if (!__all(ok) && !timeout) {
              int spins = 0;
              do {
                if (++spins > kSpinLimit) {
                  timeout = true;
                  break;
                }
                __builtin_amdgcn_s_sleep(1);
                load_block(u0);
                if (u0 == 0 && lane < 32)
                  ho = __hip_atomic_load(src + 16 * KP + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                ok = block_fresh() && (u0 > 0 || (uint32_t)(ho >> 32) == (uint32_t)i);
              } while (!__all(ok));
            }
#pragma unroll
            for (int u = 0; u < HB; ++u) {
              const int x = lane + 64 * (u0 + u);
              Pb[pb][x >> 4][x & 15] = (uint32_t)hv[u];
            }
          }
          // offset of halo bucket h from its two halves (lanes 2h and 2h+1)
          const uint32_t other = (uint32_t)__shfl_xor((int)(uint32_t)ho, 1, 64);
          if (lane < 32 && (lane & 1) == 0)
            offs[pprev][lane >> 1] = (int64_t)(((uint64_t)other << 32) | (ho & 0xFFFFFFFFull));
          if (lane == 0) s_done = i;  // published by the storing wave
        }
        if (RLDS && i + 1 < N) store_table(par ^ 1);
        if (i + 1 < N) stage_records(i + 1, cpc, spc, dmi);
        if (lane == 0) s_upcons = upc;
        __syncthreads();  // B
        if constexpr (ALIAS) __syncthreads();  // B2
      }
      __syncthreads();  // the last step's rows, offsets and argmin bytes
    } else {
      // Slot of step t: word x < 16 KP is the product of state x / 16 at bucket
      // 48 + x % 16, words 16 KP + 2h and +1 the offset of bucket 48 + h.
      auto store_slot = [&](int t, int pbuf, int opar) __attribute__((always_inline)) {
        uint64_t *dst = my_ring + (size_t)(t % kMemSlots) * SW;
        const uint64_t tag = (uint64_t)t << 32;
#pragma unroll
        for (int u = 0; u < HW; ++u) {
          const int x = lane + 64 * u;
          __hip_atomic_store(dst + x, (uint64_t)Pb[pbuf][x >> 4][H + 48 + (x & 15)] | tag, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
        }
        if (lane < 32) {
          const uint64_t o = (uint64_t)offs[opar][H + 48 + (lane >> 1)];
          __hip_atomic_store(dst + 16 * KP + lane, ((lane & 1) ? (o >> 32) : (o & 0xFFFFFFFFull)) | tag,
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      };
      // Before slot t is reused, the chunk above must have consumed its previous
      // step: the loading wave's last reading of its progress, else polling.
      auto wait_consumed = [&](int t) __attribute__((always_inline)) {
        if (t < kMemSlots || timeout) return;
        int seen = s_upcons;
        if (seen < t - kMemSlots && !spin_until(up_cons, t - kMemSlots, seen)) timeout = true;
      };
      // Argmin bytes of step t (parity buffer t & 1) to the table, the buckets
      // within the budget only.
      auto flush = [&](int t) __attribute__((always_inline)) {
        for (int x = lane; x < NBK * K; x += 64) {
          const int bb = x / K, s = x % K;
          const int lim = top + 1 - (m0 + 16 * bb);
          if (lim <= 0) continue;
          uint8_t *dst = a.table + ((rowbase + t) * K + s) * (size_t)M + m0 + 16 * bb;
          const u32x4 v = *(const u32x4 *)&argb[t & 1][bb][s][0];
          if (vec16 && lim >= 16) {
            *(u32x4 *)dst = v;
          } else {
            const uint8_t *vb = (const uint8_t *)&v;
            for (int q = 0; q < 16 && q < lim; ++q) dst[q] = vb[q];
          }
        }
      };
      int published = -1;
      auto publish = [&]() __attribute__((always_inline)) {
        const int d = s_done;
        if (consumer && d != published) {
          published = d;
          if (lane == 0) __hip_atomic_store(my_cons, d, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      };
      __syncthreads();  // step 0 of the compute waves
      for (int i = 1; i < N; ++i) {
        publish();
        if (!ALIAS && has_consumer && i >= 2) {  // slot i-1: P_{i-1}, o_{i-2}
          wait_consumed(i - 1);
          store_slot(i - 1, (i - 1) & 1, (i - 2) & 1);
        }
        if (i - FL >= 1) flush(i - FL);  // written before the previous step's last barrier
        __syncthreads();  // B
        if constexpr (ALIAS) {  // P_i is overwritten by the rows after B2
          if (has_consumer) {
            wait_consumed(i);
            store_slot(i, 0, (i - 1) & 1);
          }
          __syncthreads();  // B2
        }
      }
      __syncthreads();  // the last step's rows, offsets and argmin bytes
      // the progress, slot N-1 (P_{N-1}, o_{N-2}) and the last steps' argmin bytes
      publish();
      if (!ALIAS && has_consumer && N >= 2) {
        wait_consumed(N - 1);
        store_slot(N - 1, (N - 1) & 1, (N - 2) & 1);
      }
      for (int t = N - FL > 1 ? N - FL : 1; t < N; ++t) flush(t);
    }
    if (timeout) {
      s_timeout = 1;  // read by the reporting wave after the last barrier
      atomicOr(&W.mflags[b], MEMF_TIMEOUT);
    }
    __syncthreads();
    return;
  }

  // -------------------------------------------------------- compute waves --
  const int s0 = g * SPL;  // first state of this lane

  // Rows of the lane's states to LDS: non-ALIAS the block's row buffer
  // [bucket][state], ALIAS the wave's own columns of the product buffer.
  auto store_rows = [&](const uint32_t *q) __attribute__((always_inline)) {
    if constexpr (ALIAS) {
#pragma unroll
      for (int k = 0; k < SPL; ++k) Pb[0][s0 + k][col] = q[k];
    } else {
#pragma unroll
      for (int v = 0; v < SPL / 4; ++v)
        *(u32x4 *)&Qw[blk][m][s0 + 4 * v] = u32x4{q[4 * v], q[4 * v + 1], q[4 * v + 2], q[4 * v + 3]};
    }
  };

  // Normalisation of the lane's values y (kSat = unreachable) against the
  // bucket minimum over all states; returns the new offset relative to `base`.
  uint32_t y[SPL];
  auto normalise = [&](int64_t base) __attribute__((always_inline)) -> int64_t {
    uint32_t x = y[0];
#pragma unroll
    for (int k = 1; k < SPL; ++k) x = umin(x, y[k]);
    const uint32_t cm = rows_min(x);
    const bool feas = cm != kSat && base < kOffInf;
#pragma unroll
    for (int k = 0; k < SPL; ++k) y[k] = (feas ? umin(y[k] - cm, QCAP) : QCAP) << BITS;
    return feas ? base + (int64_t)cm : kOffInf;
  };

  // Step 0: D[0][s][m] = c[0][s] where mem[0][s] <= m (records read directly).
  {
    const u32x4 *cp = (const u32x4 *)(W.cst + rowbase * KP + s0);
    const uint32_t *dp = (const uint32_t *)(W.dsh + rowbase * KP + s0);
#pragma unroll
    for (int v = 0; v < SPL / 4; ++v) {
      const u32x4 c4 = cp[v];
      const uint32_t d4 = dp[v];
      y[4 * v] = bucket >= (int)(d4 & 0xFF) ? c4.x : kSat;
      y[4 * v + 1] = bucket >= (int)((d4 >> 8) & 0xFF) ? c4.y : kSat;
      y[4 * v + 2] = bucket >= (int)((d4 >> 16) & 0xFF) ? c4.z : kSat;
      y[4 * v + 3] = bucket >= (int)(d4 >> 24) ? c4.w : kSat;
    }
    const int64_t o0 = normalise(0);
    store_rows(y);
    if (g == 0) offs[0][col] = o0;
  }
  if (!consumer) {  // below bucket 0: infeasible
    for (int x = tid; x < 2 * H; x += 64 * CW) offs[x / H][x % H] = kOffInf;
    for (int x = tid; x < NPB * KP * H; x += 64 * CW) Pb[x / (KP * H)][(x / H) % KP][x % H] = kSat;
  }
  __syncthreads();

  // Table items: item (tb, k) of a step is the pair of registers holding
  // R[32 tb + 16 h + l][s0 + k] in lane l of row g (h = 0, 1): from the
  // staged table in LDS (K <= 64), else from the cache, PD items ahead
  // across step ends.
  const int l16 = lane & 15;
  auto item_ptr = [&](int e, int tb, int k) __attribute__((always_inline)) {
    return W.rT + ((size_t)e * KP + s0 + k) * KP + 32 * tb + l16;
  };
  u32x2 rr[PD];
  int e_cur = N > 1 ? redge[1] : 0;
  int e_nn = N > 2 ? redge[2] : e_cur;
  if constexpr (!RLDS) {
#pragma unroll
    for (int x = 0; x < PD; ++x) {
      const uint32_t *p = item_ptr(e_cur, x / SPL, x % SPL);  // PD <= SPL: items of block 0
      rr[x] = u32x2{p[0], p[16]};
    }
  }

  // Records of the lane's states for step t: costs, shift bytes (four per
  // word) and the least shift, from the parity buffer t & 1.
  constexpr int RB = ALIAS ? 8 : SPL;  // states whose records are held at once
  uint32_t cr[RB], dr[RB / 4];
  int dm = 0;
  auto read_records = [&](int par, int v0) __attribute__((always_inline)) {
#pragma unroll
    for (int v = 0; v < RB / 4; ++v) {
      const u32x4 c4 = *(const u32x4 *)&rcost[par][s0 + v0 + 4 * v];
      cr[4 * v] = c4.x;
      cr[4 * v + 1] = c4.y;
      cr[4 * v + 2] = c4.z;
      cr[4 * v + 3] = c4.w;
      dr[v] = *(const uint32_t *)&rshift[par][s0 + v0 + 4 * v];
    }
  };

  for (int i = 1; i < N; ++i) {
    const int par = i & 1, pprev = par ^ 1;
    const int pb = ALIAS ? 0 : par;
    const int e_next = e_nn;
    if constexpr (!ALIAS) {  // this step's records: the buffer is restaged after the step's barrier
      read_records(par, 0);
      dm = rdmin[par];
    }
    if constexpr (!RLDS) e_nn = i + 2 < N ? redge[i + 2] : e_next;
    if constexpr (RLDS) {
#pragma unroll
      for (int x = 0; x < PD; ++x) {
        const uint32_t *p = &rbuf[par][s0 + x][l16];
        rr[x] = u32x2{p[0], p[16]};
      }
    }

    // Phase A: products of the block's buckets for the wave's states.
    uint32_t acc[SPL];
#pragma unroll
    for (int k = 0; k < SPL; ++k) acc[k] = kSat;
    for (int tb = 0; tb < TB; ++tb) {
      uint32_t qb[32];
      if constexpr (ALIAS) {
#pragma unroll
        for (int x = 0; x < 32; ++x) qb[x] = Pb[0][32 * tb + x][col];
      } else {
#pragma unroll
        for (int v = 0; v < 8; ++v) {
          const u32x4 q = *(const u32x4 *)&Qw[blk][m][32 * tb + 4 * v];
          qb[4 * v] = q.x;
          qb[4 * v + 1] = q.y;
          qb[4 * v + 2] = q.z;
          qb[4 * v + 3] = q.w;
        }
      }
#pragma unroll
      for (int k = 0; k < SPL; k += 2) {
        const u32x2 ra = rr[k % PD], rb = rr[(k + 1) % PD];
#pragma unroll
        for (int u = 0; u < 2; ++u) {  // the items PD ahead
          const int kk = k + u + PD;
          const bool wrap = kk >= SPL;
          const int tn = wrap ? tb + 1 : tb;
          const int kn = wrap ? kk - SPL : kk;
          if constexpr (RLDS) {
            if (tn < TB) {  // within the step (the next step's table is staged later)
              const uint32_t *p = &rbuf[par][s0 + kn][32 * tn + l16];
              rr[(k + u) % PD] = u32x2{p[0], p[16]};
            }
          } else {
            const bool nstep = wrap && tn >= TB;
            const uint32_t *p = item_ptr(nstep ? e_next : e_cur, nstep ? 0 : tn, kn);
            rr[(k + u) % PD] = u32x2{p[0], p[16]};
          }
        }
        mcand4x2<0, true>(acc[k], acc[k + 1], ra.x, rb.x, qb[0], qb[1], qb[2], qb[3]);
        mcand4x2<4, false>(acc[k], acc[k + 1], ra.x, rb.x, qb[4], qb[5], qb[6], qb[7]);
        mcand4x2<8, false>(acc[k], acc[k + 1], ra.x, rb.x, qb[8], qb[9], qb[10], qb[11]);
        mcand4x2<12, false>(acc[k], acc[k + 1], ra.x, rb.x, qb[12], qb[13], qb[14], qb[15]);
        mcand4x2<0, true>(acc[k], acc[k + 1], ra.y, rb.y, qb[16], qb[17], qb[18], qb[19]);
        mcand4x2<4, false>(acc[k], acc[k + 1], ra.y, rb.y, qb[20], qb[21], qb[22], qb[23]);
        mcand4x2<8, false>(acc[k], acc[k + 1], ra.y, rb.y, qb[24], qb[25], qb[26], qb[27]);
        mcand4x2<12, false>(acc[k], acc[k + 1], ra.y, rb.y, qb[28], qb[29], qb[30], qb[31]);
      }
    }
    e_cur = e_next;
#pragma unroll
    for (int k = 0; k < SPL; ++k) Pb[pb][s0 + k][col] = acc[k];
    __syncthreads();  // B

    // Phase B: the shifted products, their offset gaps, the bucket minimum and
    // the new rows.  The gap o[m - d] - o[m - dmin] of an available state is
    // >= 0, and infinite (saturated) when column m - d is infeasible; an
    // unavailable state has cost kSat, so its gap does not matter.
    const int64_t *O = offs[pprev];
    if constexpr (ALIAS) dm = rdmin[par];
    const int64_t base = O[col - dm];
#pragma unroll
    for (int v0 = 0; v0 < SPL; v0 += 8) {  // eight states at a time (registers)
      if constexpr (ALIAS) read_records(par, v0);
      constexpr int V = ALIAS ? 0 : 1;  // ALIAS: the records of states v0 .. v0+7 are in cr[0..7]
      constexpr int NK = SPL < 8 ? SPL : 8;
      uint32_t pvs[NK];
      int64_t ods[NK];
#pragma unroll
      for (int k = 0; k < NK; ++k) {
        const int kr = V * v0 + k;
        const int d = (int)((dr[kr >> 2] >> (8 * (kr & 3))) & 0xFF);
        pvs[k] = Pb[pb][s0 + v0 + k][col - d];
        ods[k] = O[col - d];
      }
#pragma unroll
      for (int k = 0; k < NK; ++k) {
        const uint64_t gap = (uint64_t)(ods[k] - base);
        const uint32_t dk = gap > (uint64_t)kSat ? kSat : (uint32_t)gap;  // an infinite offset gives a huge gap
        argb[par][blk][s0 + v0 + k][m] = (uint8_t)(pvs[k] & S::MASK);
        y[v0 + k] = sat_add(sat_add(pvs[k] >> BITS, cr[V * v0 + k]), dk);
      }
    }
    const int64_t onew = normalise(base);
    if constexpr (ALIAS) __syncthreads();  // B2: every product read before the rows overwrite them
    store_rows(y);
    if (g == 0) offs[par][col] = onew;
  }
  __syncthreads();  // the last step's rows and offsets (matches the I/O waves')

  const int fin = (N - 1) & 1;  // offsets of the last step
  // Budget frontier: the offset of bucket m is min_s D[N-1][s][m], the least
  // cost with memory total at most m.
  if (a.frontier && g == 0 && bucket < M)
    a.frontier[(size_t)b * M + bucket] = (bucket <= top && offs[fin][col] < kOffInf) ? offs[fin][col] : INT64_MAX;
  __syncthreads();  // the I/O waves' timeout flag

  // The chunk holding the budget bucket reports the search.
  if (Bb >= m0 && Bb < m0 + C && w == 0) {
    const int cb = Bb - m0, wb = cb >> 4, mb = cb & 15;
    uint32_t f = kSat;
    for (int s = lane; s < K; s += 64) {
      uint32_t q;
      if constexpr (ALIAS) q = Pb[0][s][H + cb];
      else q = Qw[wb][mb][s];
      f = umin(f, q | (uint32_t)s);
    }
    f = wave_min(f);
    if (lane == 0) {
      const int64_t o = offs[fin][H + cb];
      const int sf = __hip_atomic_load(&W.mflags[b], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT);
      int st = CFP_ST_OK;
      if (s_timeout || (sf & MEMF_TIMEOUT)) st = CFP_ST_TIMEOUT;
      else if (a.hdr->rflag) st = CFP_ST_BADINPUT;
      else if (o >= kOffInf) st = CFP_ST_INFEASIBLE;
      else if ((f >> BITS) != 0) st = CFP_ST_OVERFLOW;  // the least state of a feasible bucket is 0
      a.status[b] = st;
      a.opt[b] = st == CFP_ST_OK ? o : INT64_MAX;
      a.res[b].final_state = st == CFP_ST_OK ? (int32_t)(f & S::MASK) : -1;
      a.res[b].status = st;
      a.res[b].final_m = Bb;
    }
  }
}

// Plan recovery for the memory variant.  The state is (s, m): the table gives
// the predecessor strategy t = arg[i][s][m] and the budget shrinks by
// mem[i][s].  The chase runs in windows of `win` steps: the argmin rows of the
// window are loaded into LDS for the only buckets it can reach,
// [m - kMemShift*(win-1), m], then one thread follows them.
constexpr int kMemWinMax = 12;
constexpr size_t kMemTbLds = 96 * 1024;

__host__ __device__ constexpr int mem_win_width(int win) { return (kMemShift * (win - 1) + 16 + 15) / 16 * 16; }

static int mem_window(int k) {
  int win = kMemWinMax;
  while (win > 1 && (size_t)win * k * mem_win_width(win) + (size_t)win * k > kMemTbLds) --win;
  return win;
}

constexpr int kMemTbThreads = 1024;  // every 16-byte piece of a window in flight at once
constexpr int kMemTbLoads = 8;       // pieces per thread and pass

__global__ __launch_bounds__(kMemTbThreads) void mem_tb_kernel(int N, int K, int M, int win,
                                                          const uint8_t *__restrict__ table,
                                                          const uint8_t *__restrict__ mem_copy,
                                                          const SearchResult *__restrict__ res,
                                                          int32_t *__restrict__ plan) {
  // window rows are 16-byte aligned copies of [lo16, lo16 + width) of a table row
  extern __shared__ __align__(16) uint8_t wbuf[];  // [win][K][width] then mem rows [win][K]
  __shared__ int cur_s, cur_m;
  const int b = blockIdx.x, tid = threadIdx.x;
  int32_t *pb = plan + (size_t)b * N;
  if (res[b].status != CFP_ST_OK) {
    for (int i = tid; i < N; i += blockDim.x) pb[i] = -1;
    return;
  }
  const int width = mem_win_width(win);
  uint8_t *mrow = wbuf + (size_t)win * K * width;
  const bool vec = (M % 16) == 0;
  if (tid == 0) {
    cur_s = res[b].final_state;
    cur_m = res[b].final_m;
    pb[N - 1] = cur_s;
  }
  __syncthreads();
  for (int i = N - 1; i >= 1;) {
    const int steps = i < win ? i : win;
    const int mtop = cur_m;
    const int lo = mtop - kMemShift * (steps - 1) > 0 ? mtop - kMemShift * (steps - 1) : 0;
    const int lo16 = lo & ~15;
    const int n16 = (mtop - lo16) / 16 + 1;  // 16-byte pieces covering [lo16, mtop]
    if (vec) {
      // all pieces of a pass are loaded before any is stored, so the window
      // costs about one memory latency
      const int total = steps * K * n16;
      for (int x0 = 0; x0 < total; x0 += kMemTbLoads * kMemTbThreads) {
        typedef uint32_t u32x4l __attribute__((ext_vector_type(4)));  // copies stay in registers
        u32x4l v[kMemTbLoads];
#pragma unroll
        for (int u = 0; u < kMemTbLoads; ++u) {
          const int x = x0 + u * kMemTbThreads + tid;
          const int k = x / (K * n16), t = (x / n16) % K, c = x % n16;
          if (x < total)
            v[u] = *(const u32x4l *)&table[(((size_t)b * N + (i - k)) * K + t) * M + lo16 + 16 * c];
        }
#pragma unroll
        for (int u = 0; u < kMemTbLoads; ++u) {
          const int x = x0 + u * kMemTbThreads + tid;
          const int k = x / (K * n16), t = (x / n16) % K, c = x % n16;
          if (x < total) *(u32x4l *)&wbuf[((size_t)k * K + t) * width + 16 * c] = v[u];
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
          if (x < total) wbuf[((size_t)k * K + t) * width + c] = v[u];
        }
      }
    }
    for (int x = tid; x < steps * K; x += blockDim.x)
      mrow[x] = mem_copy[((size_t)b * N + (i - x / K)) * K + x % K];
    __syncthreads();
    if (tid == 0) {
      int s = cur_s, m = mtop;
      for (int k = 0; k < steps; ++k) {
        int t = wbuf[((size_t)k * K + s) * width + (m - lo16)];
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
  const int win = mem_window(k);
  const size_t lds = (size_t)win * k * mem_win_width(win) + (size_t)win * k;
  hipLaunchKernelGGL(mem_tb_kernel, dim3(batch), dim3(kMemTbThreads), lds, st, n, k, n_mem, win, table, mem, res,
                     plan);
  return hipGetLastError();
}

static MemWs carve(uint8_t *region, int n, int k, int batch, int n_mem, int n_tables, size_t *bytes) {
  const int KP = mem_kp(k);
  MemWs w;
  w.nchunk = (n_mem + kMemChunk - 1) / kMemChunk;
  const size_t chunks = (size_t)batch * w.nchunk;
  size_t off = 0;
  w.cst = (uint32_t *)(region + off); off = align_up(off + (size_t)batch * n * KP * 4);
  w.dsh = region + off; off = align_up(off + (size_t)batch * n * KP);
  w.dmin = (int32_t *)(region + off); off = align_up(off + (size_t)batch * n * 4);
  w.rT = (uint32_t *)(region + off); off = align_up(off + (size_t)n_tables * KP * KP * 4);
  w.mflags = (int32_t *)(region + off); off = align_up(off + (size_t)batch * 4);
  w.cons = (int32_t *)(region + off); off = align_up(off + chunks * kMemFlagStride * 4);
  w.ring = (uint64_t *)(region + off); off = align_up(off + chunks * kMemSlots * mem_slot_words(KP) * 8);
  if (bytes) *bytes = off;
  return w;
}

size_t mem_region_bytes(int n, int k, int batch, int n_mem, int n_tables) {
  size_t bytes = 0;
  (void)carve(nullptr, n, k, batch, n_mem, n_tables, &bytes);
  return bytes;
}

// Clears the flags, marks every slot as consumed before step 0 and stamps
// every ring word with an impossible step number, so that nothing a previous
// call left in the workspace is taken for a fresh slot.
__global__ void mem_init_kernel(int32_t *mflags, int nb, int32_t *cons, int nflag, uint64_t *ring, size_t nring) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t x = blockIdx.x * (size_t)blockDim.x + threadIdx.x; x < (size_t)(nb + nflag); x += stride) {
    if (x < (size_t)nb) mflags[x] = 0;
    else cons[x - nb] = -1;
  }
  for (size_t x = blockIdx.x * (size_t)blockDim.x + threadIdx.x; x < nring; x += stride) ring[x] = ~0ull;
}

// Workgroups of one launch that the device holds at once, per XCD: the
// chunks of a search run as a pipeline whose stages wait for each other, so
// every chunk of a launch must be resident together.  Workgroup x runs on XCD
// x mod 8, and the chunks of search b of a launch are workgroups j * B8 + b,
// so they share one XCD and its L2 cache.
template <int KP>
static int mem_xcd_capacity() {
  static std::once_flag once;
  static int cap = 0;
  std::call_once(once, [] {
    int dev = 0, cus = 0, per_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, mem_fwd_kernel<KP>, MemShape<KP>::THREADS, 0) !=
            hipSuccess)
      return;
    cap = (cus / 8) * per_cu;
  });
  return cap;
}

template <int KP>
static hipError_t launch_mem(const cfp_chain_desc &d, const uint8_t *mem, int n_mem, const int32_t *budget,
                             const int32_t *redge_dev, uint8_t *table, uint8_t *mem_copy, uint8_t *region,
                             SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status,
                             int64_t *frontier, hipStream_t st) {
  const int N = d.n_blocks, K = d.k, B = d.batch, E = d.n_tables;
  MemWs w = carve(region, N, K, B, n_mem, E, nullptr);
  const int nflag = B * w.nchunk * kMemFlagStride;
  const size_t nring = (size_t)B * w.nchunk * kMemSlots * mem_slot_words(KP);
  hipLaunchKernelGGL(mem_init_kernel, dim3((unsigned)std::min<size_t>((nring + 255) / 256, 1024)), dim3(256), 0, st,
                     w.mflags, B, w.cons, nflag, w.ring, nring);
  const size_t packed = (size_t)E * KP * KP;
  hipLaunchKernelGGL(mem_pack_rtab_kernel, dim3((unsigned)std::min<size_t>((packed + 255) / 256, 2048)), dim3(256), 0,
                     st, d.rtab, E, K, KP, MemShape<KP>::BITS, w.rT, cfp_r_limit(CFP_V_MEM, K),
                     const_cast<WsHeader *>(hdr));
  hipLaunchKernelGGL(mem_prep_kernel, dim3((B * N + 3) / 4), dim3(256), 0, st, d.cost, mem, budget, N, K, KP, n_mem,
                     B, w.cst, w.dsh, w.dmin, mem_copy, w.mflags);
  // Rounds of searches whose chunks the device holds at once: with per_xcd
  // searches on each of the 8 XCDs, a round takes 8 * per_xcd searches.
  const int cap = mem_xcd_capacity<KP>();
  const int per_xcd = cap / w.nchunk;
  if (per_xcd < 1) return hipErrorInvalidConfiguration;
  const int round = 8 * per_xcd;
  MemArgs a;
  a.budget = budget;
  a.w = w;
  a.N = N;
  a.K = K;
  a.M = n_mem;
  a.B = B;
  a.table = table;
  a.res = res;
  a.hdr = hdr;
  a.opt = opt;
  a.status = status;
  a.frontier = frontier;
  timer_begin(st);
  for (int b0 = 0; b0 < B; b0 += round) {
    a.b0 = b0;
    a.nb = std::min(round, B - b0);
    a.B8 = (a.nb + 7) / 8 * 8;
    timed_launch(mem_fwd_kernel<KP>, dim3(w.nchunk * a.B8), dim3(MemShape<KP>::THREADS), 0, st, a, redge_dev,
                 (const int32_t *)w.dmin);
  }
  timer_end(st);
  return hipGetLastError();
}

bool chain_mem_supported(int k, int n_tables) { return k >= 1 && k <= kMemMaxK && n_tables >= 1; }

int32_t mem_r_limit(int k) { return k >= 1 && k <= kMemMaxK ? (int32_t)(1u << (31 - mem_bits(k))) : 0; }

hipError_t launch_chain_mem_fwd(const cfp_chain_desc &d, const uint8_t *mem, int n_mem, const int32_t *budget,
                                const int32_t *redge_dev, uint8_t *table, uint8_t *mem_copy, uint8_t *region,
                                SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status,
                                int64_t *frontier, hipStream_t st) {
#define CFP_MEM_CASE(KPV) \
  case KPV:               \
    return launch_mem<KPV>(d, mem, n_mem, budget, redge_dev, table, mem_copy, region, res, hdr, opt, status, frontier, st);
  switch (mem_kp(d.k)) {
    CFP_MEM_CASE(32)
    CFP_MEM_CASE(64)
    CFP_MEM_CASE(96)
    CFP_MEM_CASE(128)
    CFP_MEM_CASE(192)
    CFP_MEM_CASE(256)
    default:
      return hipErrorInvalidValue;
  }
#undef CFP_MEM_CASE
}

__global__ void fill_i32_kernel(int32_t *p, int n, int32_t v) {
  for (int x = blockIdx.x * blockDim.x + threadIdx.x; x < n; x += gridDim.x * blockDim.x) p[x] = v;
}

hipError_t launch_fill_i32(int32_t *p, int n, int32_t v, hipStream_t st) {
  hipLaunchKernelGGL(fill_i32_kernel, dim3((n + 255) / 256 < 64 ? (n + 255) / 256 : 64), dim3(256), 0, st, p, n, v);
  return hipGetLastError();
}

}  // namespace cfp
