// Chunk-parallel forward pass of the chain search for 32 < K <= 64 and at most
// 12 resharding tables (Sec. 4.4, Eq. T recurrence), one wave per search.
//
// Parallelism over the chain.  The recurrence is a chain of N-1 dependent
// min-plus steps per search.  Each chain is cut into P chunks that run
// concurrently, using the rank convergence of min-plus products (Maleki,
// Musuvathi and Mytkowicz, "Parallelizing dynamic programming through rank
// convergence", PPoPP 2014): the recurrence started from an arbitrary row
// becomes parallel to the true run (the rows differ by one constant in every
// state) after a few steps, and from then on both choose the same argmins.
//   1. speculative pass, every chunk: chunk p starts at its first row from that
//      row's costs alone, as if the chain began there.  It writes the argmin
//      rows of its steps and, at the end of every quad of 4 rows (a
//      checkpoint), its normalised row and the running sum of its offsets.
//   2. fix-up pass, chunks 1..P-1: chunk p starts again from the last
//      checkpoint row of chunk p-1 and recomputes its steps until its
//      normalised row equals the stored checkpoint row of the same quad,
//      rewriting the argmins on the way.  Equal normalised rows mean every
//      later step of the speculative pass is exactly the true one.
//   3. final pass, per search: sums the offsets of the chunks; if a chunk's
//      fix-up reached its end without meeting a checkpoint (so its successor
//      started from a wrong row), the rest of the chain is rerun sequentially
//      from that chunk's end row, which is the true one.  Then the lowest
//      optimal final state and the optimum.
// The result is the sequential recurrence's bit for bit whatever the inputs;
// only the time depends on how fast the rows converge.
//
// One step of one search in one wave.  Lane s holds the word of state s,
// Q[s] = (value << 6).  Two permlane swaps give four registers C_k whose every
// row of 16 lanes holds row k of the wave (states 16k .. 16k+15), so a DPP row
// broadcast of lane j of C_k hands predecessor t = 16k + j to every lane.  The
// candidate of (t, s) is C_k[j] + RP[t][s] with RP = (R[t][s] << 6) | t packed
// once per call, so one unsigned min gives the value and the lowest argmin.
// A step is 64 adds with a DPP operand and 32 three-input mins per search, a
// minimum over the wave and the normalisation; no other wave is involved.
//
// Normalisation.  The new row is x[s] = (m[s] >> 6) + c[i][s] with m the
// packed minimum; it is normalised by its own minimum d = min_s x[s]:
//     Q_i[s] = min(x[s] - d, qcap) << 6,   qcap = 2^25 - 1,
// and d is added to the search's offset, so the optimum is the sum of the row
// minima.  Since the previous row has minimum 0, m >> 6 <= R_max < 2^24 and
// x < 2^32; a state at the cap is more than R_max above the minimum and is
// beaten through the minimum state, so capping never changes an argmin.  An
// unavailable strategy (cost CFP_COST_INF) and a padding state (s >= K) get
// x = 2^32 - 1 and stay capped.
//
// Work split of a workgroup: 16 waves, each with one search of the same chunk
// (kWG searches per wave in general), so every wave steps through the same
// rows and the same tables.  The packed tables of four consecutive rows
// (4 x 16 KiB) sit in LDS and the next four are staged while these are used
// (double buffer, one barrier per four rows); the rows are cut into blocks of
// 12, the period of the edge map the kernels are specialised for.
#include <algorithm>
#include <atomic>
#include <chrono>
#include <random>

#include "res_common.h"

namespace cfp {

namespace {

// Four packed words as a native vector: copies stay in registers (a struct
// copy of the HIP vector type goes through a private-memory temporary).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWSpec = 0, kWFix = 1, kWRepair = 2;
constexpr int kWU = 12;                 // rows per block (checkpoint spacing)
constexpr int kWWaves = 16;             // waves per workgroup of the speculative pass
constexpr int kWG = 1;                  // searches per wave
constexpr int kWTable16 = 64 * 64 / 4;  // 16-byte chunks of one packed table
constexpr int kWMaxChunks = 64;         // chunks per search (the final pass reads one per lane)
constexpr int kWMinBlocks = 4;          // least blocks of 12 rows per chunk
constexpr uint32_t kWX = 0xFFFFFFFFu;   // x of an unavailable or padding state
constexpr int kWBits = 6;
constexpr uint32_t kWQcap6 = ((1u << 25) - 1u) << kWBits;

struct WaveRec {
  int64_t dfix;   // fix-up pass: offset sum at the meeting checkpoint, or at the chunk end
  int32_t flags;  // speculative pass: bit 0 a negative cost, bit 1 a row with no available strategy
  int32_t conv;   // fix-up pass: quad of the meeting checkpoint, -1 if none
};

struct WaveArgs {
  const int32_t *cost;
  const u32x4 *rpk;     // packed tables [E][16 chunks][64 states] of 4 words
  const int32_t *redge;
  int N, K, E, B, P, CB, nblk, nq;  // nq = quads of 4 rows
  uint8_t *table;       // argmin entries [B][N][K]
  WaveRec *rec;         // [B][P]
  int64_t *dck;         // speculative offset sum (from the chunk's start row) at every checkpoint [B][nq]
  uint32_t *ckrow;      // speculative row at every checkpoint (end of a quad of rows) [B][nq][64]
  uint32_t *endrow;     // fix-up end row of chunks that met no checkpoint [B][P][64]
  uint64_t seq;         // number of this call: a range error in R is flagged as hdr->rseq = seq
};

// Packed tables: word u of chunk c of lane s of table e is (R_e[t][s] << 6) | t
// with t = 4c + u.  Rows t >= K and columns s >= K take row or column K-1: a
// predecessor t >= K holds a capped word, so its candidate exceeds every exact
// one without wrapping, and a state s >= K is padding.
// Every R entry is read here, so the range check of R (entries in [0, limit))
// is made on the way and flagged in the header as the call's number.
__global__ void wave_pack_kernel(const int32_t *__restrict__ rtab, int E, int K, uint32_t *__restrict__ rpk,
                                 int32_t limit, WsHeader *__restrict__ hdr, uint64_t seq) {
  const size_t words = (size_t)E * 64 * 64;
  for (size_t w = blockIdx.x * (size_t)blockDim.x + threadIdx.x; w < words; w += (size_t)gridDim.x * blockDim.x) {
    const int u = (int)(w & 3), s = (int)((w >> 2) & 63), c = (int)((w >> 8) & 15), e = (int)(w >> 12);
    const int t = 4 * c + u;
    const int32_t r = rtab[((size_t)e * K + min(t, K - 1)) * K + min(s, K - 1)];
    if (r < 0 || r >= limit) hdr->rseq = seq;
    rpk[w] = ((uint32_t)r << kWBits) | (uint32_t)t;
  }
}

// Minimum over the 64 lanes of a wave as a scalar: row minima by DPP, then the
// row broadcasts of lanes 15 and 31 fold rows 0..3 into row 3, read at lane 63.
__device__ __forceinline__ uint32_t wave_min64_s(uint32_t x) {
  x = dpp_min<kQuadSwap1>(x);
  x = dpp_min<kQuadSwap2>(x);
  x = dpp_min<kHalfMirror>(x);
  x = dpp_min<kMirror>(x);
  asm("s_nop 1\n"
      "v_min_u32_dpp %0, %0, %0 row_bcast:15 row_mask:0xa bank_mask:0xf\n"
      "s_nop 1\n"
      "v_min_u32_dpp %0, %0, %0 row_bcast:31 row_mask:0xc bank_mask:0xf\n"
      "s_nop 1\n"
      : "+v"(x));
  return __builtin_amdgcn_readlane(x, 63);
}

// Four candidates of predecessors 16k + J0 .. 16k + J0 + 3 for the wave's
// searches: acc = min(acc, C[J0 + v] + w_v) with C the row-broadcast source of
// the search and w the four packed table words.  Written out so that every add
// is one instruction with a DPP operand: the compiler keeps such adds fused in
// short functions but, in the unrolled step, leaves a separate move per add.
// The source registers come from permlane swaps; NOP = the first block after
// them, which waits the two states a DPP read of a fresh VALU result needs.
#define CFP_W_ADD(T, C, W, J) "v_add_u32_dpp " T ", " C ", " W " row_newbcast:" J " row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
template <int J0, bool NOP>
__device__ __forceinline__ void cand4_g2(uint32_t &a0, uint32_t &a1, uint32_t c0, uint32_t c1, const u32x4 &w) {
  uint32_t t0, t1, t2, t3;
  asm(
      ".if %[nop]\n s_nop 2\n .endif\n"
      CFP_W_ADD("%[t0]", "%[c0]", "%[wx]", "%[j0]")
      CFP_W_ADD("%[t1]", "%[c0]", "%[wy]", "%[j1]")
      CFP_W_ADD("%[t2]", "%[c1]", "%[wx]", "%[j0]")
      CFP_W_ADD("%[t3]", "%[c1]", "%[wy]", "%[j1]")
      "v_min3_u32 %[a0], %[a0], %[t0], %[t1]\n"
      "v_min3_u32 %[a1], %[a1], %[t2], %[t3]\n"
      CFP_W_ADD("%[t0]", "%[c0]", "%[wz]", "%[j2]")
      CFP_W_ADD("%[t1]", "%[c0]", "%[ww]", "%[j3]")
      CFP_W_ADD("%[t2]", "%[c1]", "%[wz]", "%[j2]")
      CFP_W_ADD("%[t3]", "%[c1]", "%[ww]", "%[j3]")
      "v_min3_u32 %[a0], %[a0], %[t0], %[t1]\n"
      "v_min3_u32 %[a1], %[a1], %[t2], %[t3]\n"
      : [a0] "+v"(a0), [a1] "+v"(a1), [t0] "=&v"(t0), [t1] "=&v"(t1), [t2] "=&v"(t2), [t3] "=&v"(t3)
      : [c0] "v"(c0), [c1] "v"(c1), [wx] "v"(w.x), [wy] "v"(w.y), [wz] "v"(w.z), [ww] "v"(w.w),
        [j0] "i"(J0), [j1] "i"(J0 + 1), [j2] "i"(J0 + 2), [j3] "i"(J0 + 3), [nop] "i"(NOP ? 1 : 0));
}
template <int J0, bool NOP>
__device__ __forceinline__ void cand4_g1(uint32_t &a0, uint32_t c0, const u32x4 &w) {
  uint32_t t0, t1;
  asm(
      ".if %[nop]\n s_nop 2\n .endif\n"
      CFP_W_ADD("%[t0]", "%[c0]", "%[wx]", "%[j0]")
      CFP_W_ADD("%[t1]", "%[c0]", "%[wy]", "%[j1]")
      "v_min3_u32 %[a0], %[a0], %[t0], %[t1]\n"
      CFP_W_ADD("%[t0]", "%[c0]", "%[wz]", "%[j2]")
      CFP_W_ADD("%[t1]", "%[c0]", "%[ww]", "%[j3]")
      "v_min3_u32 %[a0], %[a0], %[t0], %[t1]\n"
      : [a0] "+v"(a0), [t0] "=&v"(t0), [t1] "=&v"(t1)
      : [c0] "v"(c0), [wx] "v"(w.x), [wy] "v"(w.y), [wz] "v"(w.z), [ww] "v"(w.w),
        [j0] "i"(J0), [j1] "i"(J0 + 1), [j2] "i"(J0 + 2), [j3] "i"(J0 + 3), [nop] "i"(NOP ? 1 : 0));
}
// The first four candidates of a row: a0 is set, not updated.
__device__ __forceinline__ void cand4_g1_first(uint32_t &a0, uint32_t c0, const u32x4 &w) {
  uint32_t t0, t1;
  asm(
      "s_nop 2\n"
      CFP_W_ADD("%[t0]", "%[c0]", "%[wx]", "0")
      CFP_W_ADD("%[t1]", "%[c0]", "%[wy]", "1")
      "v_min_u32 %[a0], %[t0], %[t1]\n"
      CFP_W_ADD("%[t0]", "%[c0]", "%[wz]", "2")
      CFP_W_ADD("%[t1]", "%[c0]", "%[ww]", "3")
      "v_min3_u32 %[a0], %[a0], %[t0], %[t1]\n"
      : [a0] "=&v"(a0), [t0] "=&v"(t0), [t1] "=&v"(t1)
      : [c0] "v"(c0), [wx] "v"(w.x), [wy] "v"(w.y), [wz] "v"(w.z), [ww] "v"(w.w));
}
#undef CFP_W_ADD

template <int NW>
struct WaveSmem {
  static constexpr int CPT = kWTable16 / (64 * NW);  // 16-byte chunks per thread and table
  u32x4 tb[2][4][kWTable16];                          // packed tables of two quads of rows
  uint8_t argb[NW][kWG][kWU][64];                     // argmin bytes of the block's rows, per wave and search
  uint32_t wact[2][NW];                               // fix-up: wave still has an unmet search, by quad parity
};

// State of a wave's searches.
template <int G>
struct WaveChains {
  uint32_t qv[G];      // the lane's word of the current row
  uint64_t dsum[G];    // offset sum since the start row
  uint32_t flags[G];   // bit 0 a negative cost, bit 1 a row with no available strategy
  uint32_t cor[G];     // speculative pass: OR of the lane's costs (bit 31 = a negative cost)
  int conv[G];         // fix-up: quad where the row met the checkpoint, -1 if never
  uint64_t dconv[G];   // fix-up: offset sum at that quad
};

// Runs rows [12*blk0 (+1 for kSpec), min(12*blk1, N)) of the wave's G searches
// bw .. bw+G-1, of which those below B and (for the final pass) the first
// nvalid are real.
//   kSpec:   the start row is row 12*blk0 from its costs alone; checkpoints are
//            written.
//   kRepair: the start row (row 12*blk0 - 1) is start[g].
//   kFix:    as kRepair; at every quad end the row is compared with the
//            speculative checkpoint of the same quad.  A search that has met
//            it stops computing (its later speculative rows are the true ones)
//            and the workgroup stops once all of its searches have met.
template <int NW, int G, int MODE, int EP>
__device__ __forceinline__ void wave_run(const WaveArgs &a, int bw, int nvalid, int blk0, int blk1,
                                         const uint32_t *const *start, WaveSmem<NW> &sm, WaveChains<G> &ch) {
  constexpr int U = kWU, CPT = WaveSmem<NW>::CPT;
  static_assert(G == 1 || G == 2, "one or two searches per wave");
  static_assert(MODE != kWFix || G == 1, "the fix-up carries one search per wave");
  static_assert(CPT == 1 || CPT == 2 || CPT == 4, "1, 2 or 4 chunks per thread and table");
  const int tid = threadIdx.x, lane = tid & 63, wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int N = a.N, K = a.K;
  const int i0 = blk0 * U + (MODE == kWSpec ? 1 : 0);  // first computed row
  const int ilast = min(blk1 * U, N) - 1;              // last row of the run
  const int sl = min(lane, K - 1);

  auto valid = [&](int g) __attribute__((always_inline)) { return g < nvalid && bw + g < a.B; };
  auto srch = [&](int g) __attribute__((always_inline)) { return min(bw + g, a.B - 1); };
  auto edge = [&](int row) __attribute__((always_inline)) { return EP ? row % (EP ? EP : 1) : a.redge[row]; };
  // cost rows of the two searches (wave-uniform bases; a row adds row * K and
  // the lane its state, so the loads take a scalar base and a lane offset)
  const int32_t *cb0 = a.cost + (size_t)srch(0) * N * K;
  const int32_t *cb1 = a.cost + (size_t)srch(G - 1) * N * K;
  uint8_t *tb0 = a.table + (size_t)srch(0) * N * K;
  uint8_t *tb1 = a.table + (size_t)srch(G - 1) * N * K;

  // Memory schedule.  The tables of the next quad are loaded during the first
  // three rows of a quad of four and the costs of the quad after the next in
  // its last row; everything is consumed at a quad's end, after its one wait.  (With stores in flight the wait covers
  // every outstanding load, so a load consumed earlier would stall the row.)
  // Array indices are literals only, so every array stays in registers.
  u32x4 sq[4][4];           // next quad's tables: [row in quad][chunk of this thread]
  // Costs of three consecutive quads, [quad mod 3][row in quad][search]: quad
  // q reads set q mod 3 while set (q+2) mod 3 is loaded.  A block of 12 rows
  // starts at a quad that is 0 mod 3, so every index is a constant.
  uint32_t cs[3][4][2] = {};
#define CFP_QLOAD(V)                                                               \
  {                                                                                \
    const int row = min(qbase + (V), ilast); /* past the end: any in-range row */  \
    const u32x4 *src = a.rpk + (size_t)edge(row) * kWTable16;                      \
    sq[V][0] = src[tid];                                                           \
    if constexpr (CPT >= 2) sq[V][1] = src[tid + 64 * NW];                         \
    if constexpr (CPT == 4) {                                                      \
      sq[V][2] = src[tid + 128 * NW];                                              \
      sq[V][3] = src[tid + 192 * NW];                                              \
    }                                                                              \
  }
#define CFP_CLOAD(V, DST)                                                          \
  {                                                                                \
    const int row = min(cbase + (V), ilast);                                       \
    DST[V][0] = (uint32_t)(cb0 + (size_t)row * K)[sl];                             \
    if constexpr (G == 2) DST[V][1] = (uint32_t)(cb1 + (size_t)row * K)[sl];       \
  }
#define CFP_QSTORE(V)                                                              \
  {                                                                                \
    u32x4 *dst = sm.tb[((qbase + (V)) >> 2) & 1][V] + tid;                         \
    dst[0] = sq[V][0];                                                             \
    if constexpr (CPT >= 2) dst[64 * NW] = sq[V][1];                               \
    if constexpr (CPT == 4) {                                                      \
      dst[128 * NW] = sq[V][2];                                                    \
      dst[192 * NW] = sq[V][3];                                                    \
    }                                                                              \
  }
#define CFP_Q4(M) M(0) M(1) M(2) M(3)

  // Prologue: the first quad (rows from i0) at once, the next quad's loads,
  // and the costs of the two quads after the first.
  {
    int qbase = i0 & ~3, cbase = qbase;
#define CFP_QFIRST(V) /* rows before i0 are staged too, and never read */ \
  CFP_QLOAD(V)                                                             \
  CFP_QSTORE(V)
    CFP_Q4(CFP_QFIRST)
#undef CFP_QFIRST
    qbase += 4;
    CFP_Q4(CFP_QLOAD)
    // the first quad is 0 mod 3 (blocks start at quads 3 blk)
#define CFP_C0(V) CFP_CLOAD(V, cs[0])
#define CFP_C1(V) CFP_CLOAD(V, cs[1])
#define CFP_C2(V) CFP_CLOAD(V, cs[2])
    CFP_Q4(CFP_C0)
    cbase += 4;
    CFP_Q4(CFP_C1)
    cbase += 4;
    CFP_Q4(CFP_C2)
  }

  // Start row.
#pragma unroll
  for (int g = 0; g < G; ++g) {
    ch.flags[g] = 0;
    if (MODE == kWSpec) {
      const uint32_t cv = (uint32_t)((g == 0 ? cb0 : cb1) + (size_t)blk0 * U * K)[sl];
      const bool avail = lane < K && cv != (uint32_t)CFP_COST_INF;
      ch.cor[g] = cv;
      const uint32_t x = avail ? cv : kWX;
      const uint32_t d = wave_min64_s(x);
      if (d == kWX) ch.flags[g] |= 2;
      ch.qv[g] = umin(x - d, kWQcap6 >> kWBits) << kWBits;
      ch.dsum[g] = d;
      if (i0 > ilast && valid(g)) {  // a run of one row: the start row is its checkpoint
        a.ckrow[((size_t)(bw + g) * a.nq + (i0 - 1) / 4) * 64 + lane] = ch.qv[g];
        if (lane == 0) a.dck[(size_t)(bw + g) * a.nq + (i0 - 1) / 4] = (int64_t)ch.dsum[g];
      }
    } else {
      ch.qv[g] = start[g][lane];
      ch.dsum[g] = 0;
    }
    ch.conv[g] = valid(g) ? -1 : 0;  // a missing search counts as met
    ch.dconv[g] = 0;
  }
  int endr[G];  // last row whose argmin bytes are written back
  uint32_t ckv[G] = {};  // fix-up: checkpoint of the current quad
#pragma unroll
  for (int g = 0; g < G; ++g) endr[g] = ilast;
  bool stop = false;
  __syncthreads();  // the first quad's tables

  // Argmin bytes of rows [12 blk + r0, 12 blk + nr) of the wave's searches from
  // LDS to the table: a row of one search is 64 bytes, four 16-byte pieces.
  auto flush = [&](int blk, int nr) __attribute__((always_inline)) {
    const int r0 = (MODE == kWSpec && blk == blk0) ? 1 : 0;  // the start row has no argmin
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (!valid(g)) continue;
      uint8_t *dst = (g == 0 ? tb0 : tb1) + (size_t)blk * U * K;
      const int nrg = MODE == kWFix ? min(nr, endr[g] - blk * U + 1) : nr;
      for (int x = lane + 4 * r0; x < 4 * nrg; x += 64) {  // piece x: row x / 4, bytes 16 (x % 4) ..
        const int r = x >> 2, c = (x & 3) * 16;
        const u32x4 v = *(const u32x4 *)&sm.argb[wid][g][r][c];
        if (K == 64) {
          *(u32x4 *)(dst + (size_t)r * K + c) = v;
        } else {
          const uint8_t *vb = (const uint8_t *)&v;
          for (int q = 0; q < 16 && c + q < K; ++q) dst[(size_t)r * K + c + q] = vb[q];
        }
      }
    }
  };

  constexpr int NPRE = 4;  // table chunks of the next row read ahead
  u32x4 wpre[NPRE];
  // One row; J = row mod 12.  GUARD: the block may end before its 12th row;
  // FIRST: the run's first block, whose rows before i0 are skipped and whose
  // first quad's loads were issued before the loop.
  auto step = [&](auto Jc, auto Gd, auto Fd, int blk) __attribute__((always_inline)) {
    constexpr int J = decltype(Jc)::value, u = J & 3;
    constexpr bool GUARD = decltype(Gd)::value, FIRST = decltype(Fd)::value;
    const int i = blk * U + J;
    if (MODE == kWFix && stop) return;
    if (GUARD && i > ilast) return;
    if (FIRST && i < i0) return;
    if (!FIRST || i >= (i0 & ~3) + 4) {  // the next quad's loads (the first quad's: prologue)
      // rows 0 and 1 at step 0, row 2 at step 1, row 3 at step 2: every load
      // has at least one row of compute before the quad's wait
      const int qbase = (i & ~3) + 4;
      if constexpr (u == 0) {
        CFP_QLOAD(0)
        CFP_QLOAD(1)
      }
      if constexpr (u == 1) CFP_QLOAD(2)
      if constexpr (u == 2) CFP_QLOAD(3)
    }
    if (MODE == kWFix && u == 0) {  // this quad's checkpoint (runs start at a quad)
#pragma unroll
      for (int g = 0; g < G; ++g) ckv[g] = (a.ckrow + ((size_t)srch(g) * a.nq + (i >> 2)) * 64)[lane];
    }
    if (u == 3 && (!FIRST || i >= (i0 & ~3) + 4)) {  // costs two quads ahead, after this quad's table loads
      const int cbase = (i & ~3) + 8;
      constexpr int nset = (J / 4 + 2) % 3;
      if constexpr (nset == 0) { CFP_Q4(CFP_C0) }
      if constexpr (nset == 1) { CFP_Q4(CFP_C1) }
      if constexpr (nset == 2) { CFP_Q4(CFP_C2) }
    }

    // Row-broadcast sources: C_k has row k of the wave in every row.
    uint32_t c0[G], c1[G], c2[G], c3[G], acc[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const auto p = __builtin_amdgcn_permlane16_swap(ch.qv[g], ch.qv[g], false, false);
      const auto lo = __builtin_amdgcn_permlane32_swap(p[0], p[0], false, false);
      const auto hi = __builtin_amdgcn_permlane32_swap(p[1], p[1], false, false);
      c0[g] = lo[0];
      c2[g] = lo[1];
      c1[g] = hi[0];
      c3[g] = hi[1];
      acc[g] = kSat;
    }
    const u32x4 *tb = sm.tb[(i >> 2) & 1][u];
    // With two searches a wave has the registers for all sixteen table chunks
    // of a row; with one (sixteen waves per workgroup) it loads them in two
    // halves, and outside the first block the first half of rows 1..3 of a
    // quad is read during the previous row's normalisation (PRE).
    constexpr int WH = (MODE == kWSpec && G == 2) ? 16 : 8;
    constexpr bool PRE = WH < 16 && !FIRST && u != 0;
    u32x4 w[16];
    // Candidates of every predecessor for the searches X (and Y): two
    // searches share each table chunk read.
#define CFP_CH2(C, cc_) cand4_g2<4 * ((cc_) & 3), ((cc_) & 3) == 0>(acc[0], acc[G - 1], C[0], C[G - 1], w[cc_]);
#define CFP_CH1(X, C, cc_)                                                  \
  if constexpr ((cc_) == 0) cand4_g1_first(acc[X], C[X], w[0]);             \
  else cand4_g1<4 * ((cc_) & 3), ((cc_) & 3) == 0>(acc[X], C[X], w[cc_]);
#define CFP_ROW(CH, ...)                                                                   \
  {                                                                                        \
    if constexpr (PRE) {                                                                   \
      _Pragma("unroll") for (int cc_ = 0; cc_ < NPRE; ++cc_) w[cc_] = wpre[cc_];           \
      _Pragma("unroll") for (int cc_ = NPRE; cc_ < WH; ++cc_) w[cc_] = tb[cc_ * 64 + lane]; \
    } else {                                                                               \
      _Pragma("unroll") for (int cc_ = 0; cc_ < WH; ++cc_) w[cc_] = tb[cc_ * 64 + lane];   \
    }                                                                                      \
    CH(__VA_ARGS__ c0, 0) CH(__VA_ARGS__ c0, 1) CH(__VA_ARGS__ c0, 2) CH(__VA_ARGS__ c0, 3) \
    CH(__VA_ARGS__ c1, 4) CH(__VA_ARGS__ c1, 5) CH(__VA_ARGS__ c1, 6) CH(__VA_ARGS__ c1, 7) \
    if constexpr (WH < 16) {                                                               \
      _Pragma("unroll") for (int cc_ = 8; cc_ < 16; ++cc_) w[cc_] = tb[cc_ * 64 + lane];   \
    }                                                                                      \
    CH(__VA_ARGS__ c2, 8) CH(__VA_ARGS__ c2, 9) CH(__VA_ARGS__ c2, 10) CH(__VA_ARGS__ c2, 11) \
    CH(__VA_ARGS__ c3, 12) CH(__VA_ARGS__ c3, 13) CH(__VA_ARGS__ c3, 14) CH(__VA_ARGS__ c3, 15) \
    if constexpr (WH < 16 && !FIRST && u != 3) {                                           \
      _Pragma("unroll") for (int cc_ = 0; cc_ < NPRE; ++cc_) wpre[cc_] = tb[kWTable16 + cc_ * 64 + lane]; \
    }                                                                                      \
  }
    const bool live = MODE != kWFix || ch.conv[0] < 0;  // (one search per wave in the fix-up)
    if constexpr (G == 2) CFP_ROW(CFP_CH2)
    else if (live) CFP_ROW(CFP_CH1, 0,)
#undef CFP_ROW
#undef CFP_CH1
#undef CFP_CH2

    // New row: add the cost, normalise by the row minimum, record the argmin.
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (MODE == kWFix && !live) continue;
      const uint32_t cv = cs[(J / 4) % 3][u][g];
      const bool avail = lane < K && cv != (uint32_t)CFP_COST_INF;
      if (MODE == kWSpec) {
        ch.cor[g] |= cv;
        // kept in its row: sunk to the end of a block, the OR waits for the
        // latest cost loads behind the block's argmin stores
        asm volatile("" : "+v"(ch.cor[g]));
      }
      const uint32_t x = avail ? (acc[g] >> kWBits) + cv : kWX;
      const uint32_t d = wave_min64_s(x);
      if (MODE == kWSpec && d == kWX) ch.flags[g] |= 2;
      ch.qv[g] = umin(x - d, kWQcap6 >> kWBits) << kWBits;
      ch.dsum[g] += d;
      sm.argb[wid][g][J][lane] = (uint8_t)acc[g];
    }

    // End of a quad: the next quad's tables in place and one barrier, then the
    // checkpoint (speculative pass) and, at the end of a block, the argmin rows
    // (each wave writes back its own searches' bytes with 16-byte stores).  The
    // stores come after the barrier's wait for the staged loads, so that wait
    // does not cover them.
    constexpr bool QEND = u == 3;
    if (QEND || (GUARD && i == ilast)) {
      {
        const int qbase = (i & ~3) + 4;
        CFP_Q4(CFP_QSTORE)
      }
      if (MODE == kWFix) {
        if (ch.conv[0] < 0 && __ballot(ch.qv[0] != ckv[0]) == 0) {
          ch.conv[0] = i >> 2;
          ch.dconv[0] = ch.dsum[0];
          endr[0] = i;
        }
        if (lane == 0) sm.wact[(i >> 2) & 1][wid] = ch.conv[0] < 0 ? 1u : 0u;
      }
      __syncthreads();
      if (MODE == kWFix) {  // every wave reads the same flags: a uniform decision
        const uint32_t f = lane < NW ? sm.wact[(i >> 2) & 1][lane] : 0u;
        stop = __ballot(f != 0) == 0;
        if (stop) {
          flush(blk, J + 1);
          return;
        }
      }
      if (MODE == kWSpec) {
        const int q = i >> 2;
#pragma unroll
        for (int g = 0; g < G; ++g) {
          if (!valid(g)) continue;
          (a.ckrow + ((size_t)(bw + g) * a.nq + q) * 64)[lane] = ch.qv[g];
          if (lane == 0) a.dck[(size_t)(bw + g) * a.nq + q] = (int64_t)ch.dsum[g];
        }
      }
      if (J == U - 1 || (GUARD && i == ilast)) flush(blk, J + 1);
    }
  };
#undef CFP_Q4
#undef CFP_QSTORE
#undef CFP_QLOAD
#undef CFP_CLOAD
#undef CFP_C0
#undef CFP_C1
#undef CFP_C2

  auto block = [&](auto Gd, auto Fd, int blk) __attribute__((always_inline)) {
#define CFP_S(J_) step(std::integral_constant<int, J_>{}, Gd, Fd, blk);
    CFP_S(0) CFP_S(1) CFP_S(2) CFP_S(3) CFP_S(4) CFP_S(5)
    CFP_S(6) CFP_S(7) CFP_S(8) CFP_S(9) CFP_S(10) CFP_S(11)
#undef CFP_S
  };

  const int full_end = min(blk1, N / U);  // blocks with 12 rows
  if (blk0 >= full_end) {  // a single block, not full
    block(std::true_type{}, std::true_type{}, blk0);
    return;
  }
  block(std::false_type{}, std::true_type{}, blk0);
  int blk = blk0 + 1;
  for (; blk < full_end && !(MODE == kWFix && stop); ++blk) block(std::false_type{}, std::false_type{}, blk);
  if (blk < blk1 && !(MODE == kWFix && stop)) block(std::true_type{}, std::false_type{}, blk);
}

// Speculative pass, grid (ceil(B/16), P).
template <int EP>
__global__ __launch_bounds__(64 * kWWaves) void chain_wave_kernel(WaveArgs a) {
  __shared__ __align__(16) WaveSmem<kWWaves> sm;
  const int lane = threadIdx.x & 63, wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int bw = blockIdx.x * kWWaves * kWG + wid * kWG;
  const int p = blockIdx.y;
  const int blk0 = p * a.CB, blk1 = min(blk0 + a.CB, a.nblk);
  WaveChains<kWG> ch;
  wave_run<kWWaves, kWG, kWSpec, EP>(a, bw, kWG, blk0, blk1, nullptr, sm, ch);
#pragma unroll
  for (int g = 0; g < kWG; ++g) {
    if (__ballot((int32_t)ch.cor[g] < 0)) ch.flags[g] |= 1;  // wave-uniform
    if (bw + g >= a.B) continue;
    if (lane == 0) a.rec[(size_t)(bw + g) * a.P + p].flags = (int32_t)ch.flags[g];
  }
}

// Fix-up pass, grid (ceil(B/16), P-1): the sixteen searches of a workgroup
// rerun chunk p >= 1 from the last checkpoint row of chunk p-1 (their true row
// once chunk p-1 has met) until each row equals chunk p's checkpoint at a quad
// end; the tables are staged once per quad for all sixteen, a search that has
// met stops computing, and the workgroup stops when all have met.
template <int EP>
__global__ __launch_bounds__(64 * kWWaves) void chain_wave_fix_kernel(WaveArgs a) {
  __shared__ __align__(16) WaveSmem<kWWaves> sm;
  const int lane = threadIdx.x & 63, wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int bw = blockIdx.x * kWWaves + wid;  // one search per wave
  const int p = blockIdx.y + 1;
  const int blk0 = p * a.CB, blk1 = min(blk0 + a.CB, a.nblk);
  const int i0 = blk0 * kWU;  // a multiple of 4
  const int b = min(bw, a.B - 1);
  const uint32_t *start[1] = {a.ckrow + ((size_t)b * a.nq + (i0 / 4 - 1)) * 64};
  WaveChains<1> ch;
  wave_run<kWWaves, 1, kWFix, EP>(a, bw, 1, blk0, blk1, start, sm, ch);
  if (bw >= a.B) return;
  if (ch.conv[0] < 0) a.endrow[((size_t)bw * a.P + p) * 64 + lane] = ch.qv[0];
  if (lane == 0) {
    WaveRec &r = a.rec[(size_t)bw * a.P + p];
    r.conv = ch.conv[0];
    r.dfix = (int64_t)(ch.conv[0] >= 0 ? ch.dconv[0] : ch.dsum[0]);
  }
}

// Final pass, one workgroup of 4 waves per search (see the top of the file);
// only wave 0 carries the search, the others keep the table staging shared.
constexpr int kWFinalWaves = 4;

template <int EP>
__global__ __launch_bounds__(64 * kWFinalWaves, 1) void chain_wave_final_kernel(WaveArgs a,
                                                                                const WsHeader *__restrict__ hdr,
                                                                                SearchResult *__restrict__ res,
                                                                                int64_t *__restrict__ opt,
                                                                                int32_t *__restrict__ status) {
  __shared__ __align__(16) WaveSmem<kWFinalWaves> sm;
  __shared__ int s_q, s_flags;
  __shared__ int64_t s_dtot;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int b = blockIdx.x, P = a.P;

  if (wid == 0) {
    const bool in = lane < P;
    WaveRec r{};
    if (in) r = a.rec[(size_t)b * P + lane];
    const int endq = (min((lane + 1) * a.CB * kWU, a.N) - 1) >> 2;  // quad of the chunk's last row
    const uint64_t nc = __ballot(in && lane >= 1 && r.conv < 0);
    const int q = nc ? __ffsll((long long)nc) - 1 : P;  // first chunk whose fix-up met no checkpoint
    int64_t delta = 0;
    if (in && lane < q) {
      const int64_t *dk = a.dck + (size_t)b * a.nq;
      delta = lane == 0 ? dk[endq] : r.dfix + dk[endq] - dk[r.conv];
    } else if (lane == q) {
      delta = r.dfix;  // its fix-up started from the true row and ran to the end
    }
    int fl = in ? r.flags : 0;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      delta += __shfl_xor(delta, off, 64);
      fl |= __shfl_xor(fl, off, 64);
    }
    if (lane == 0) {
      s_q = q;
      s_dtot = delta;
      s_flags = fl;
    }
  }
  __syncthreads();
  const int q = s_q;
  uint64_t drep = 0;
  uint32_t qv;
  if (q < P - 1) {
    // Rerun the chain after chunk q from its end row (wave 0; the others stage).
    const uint32_t *start[1] = {a.endrow + ((size_t)b * P + q) * 64};
    WaveChains<1> ch;
    wave_run<kWFinalWaves, 1, kWRepair, EP>(a, b, wid == 0 ? 1 : 0, (q + 1) * a.CB, a.nblk, start, sm, ch);
    qv = ch.qv[0];
    drep = ch.dsum[0];
  } else if (q == P - 1) {
    qv = a.endrow[((size_t)b * P + q) * 64 + lane];
  } else {
    qv = a.ckrow[((size_t)b * a.nq + a.nq - 1) * 64 + lane];
  }
  if (wid != 0) return;
  // The final row has minimum 0: the lowest state at the minimum.
  const uint32_t pk = wave_min(lane < a.K ? (qv | (uint32_t)lane) : kSat);
  if (lane == 0) {
    const int fl = s_flags;
    int st = CFP_ST_OK;
    if ((fl & 1) || hdr->rseq == a.seq) st = CFP_ST_BADINPUT;
    else if (fl & 2) st = CFP_ST_INFEASIBLE;
    else if ((pk >> kWBits) != 0) st = CFP_ST_OVERFLOW;
    status[b] = st;
    opt[b] = st == CFP_ST_OK ? s_dtot + (int64_t)drep : INT64_MAX;
    res[b].final_state = st == CFP_ST_OK ? (int32_t)(pk & 63u) : -1;
    res[b].status = st;
    res[b].final_m = 0;
  }
}

struct WavePlan {
  int P, CB, nblk, nq;
};

WavePlan wave_plan(int n, int k, int e, int batch) {
  WavePlan c{0, 0, 0, 0};
  if (k <= 32 || k > 64 || e > kResTables) return c;
  c.nblk = (n + kWU - 1) / kWU;
  c.nq = (n + 3) / 4;
  const int rows = (batch + kWWaves * kWG - 1) / (kWWaves * kWG);
  int P = std::max(1, 256 / rows);  // one workgroup per compute unit
  P = std::min(P, std::min(kWMaxChunks, c.nblk / kWMinBlocks));
  if (P < 2) return WavePlan{0, 0, 0, 0};
  c.CB = (c.nblk + P - 1) / P;
  c.P = (c.nblk + c.CB - 1) / c.CB;
  return c;
}

template <int EP>
static void launch_wave_passes(const WaveArgs &a, const WsHeader *hdr, SearchResult *res, int64_t *opt,
                               int32_t *status, hipStream_t st) {
  const int rows = (a.B + kWWaves * kWG - 1) / (kWWaves * kWG);
  timer_begin(st);
  timed_launch(chain_wave_kernel<EP>, dim3(rows, a.P), dim3(64 * kWWaves), 0, st, a);
  timer_end(st);
  hipLaunchKernelGGL((chain_wave_fix_kernel<EP>), dim3((a.B + kWWaves - 1) / kWWaves, a.P - 1), dim3(64 * kWWaves), 0,
                     st, a);
  hipLaunchKernelGGL((chain_wave_final_kernel<EP>), dim3(a.B), dim3(64 * kWFinalWaves), 0, st, a, hdr, res, opt,
                     status);
}

// Number of a call, stored as the range flag of a workspace whose header is
// not uploaded.  The word starts as whatever the workspace held, so the
// numbers must not be guessable from stale bytes: the sequence starts at a
// random 64-bit point drawn once per process and every number has its top bit
// set, so no zero word (what an upload writes) and no small or non-negative
// integer left in the workspace ever equals one.
static uint64_t next_call_number() {
  static std::atomic<uint64_t> counter{0};
  static const uint64_t base = [] {
    std::random_device rd;
    uint64_t x = ((uint64_t)rd() << 32) ^ (uint64_t)rd();
    x ^= (uint64_t)std::chrono::steady_clock::now().time_since_epoch().count();
    // SplitMix64 finaliser (Steele, Lea and Flood, OOPSLA 2014)
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
  }();
  return (base + counter.fetch_add(1, std::memory_order_relaxed)) | (1ull << 63);
}

// Period of the edge map if redge[i] == i mod E for all i >= 1 with E
// dividing 12, else 0.
static int wave_edge_period(const int32_t *redge, int n, int e) {
  if (kWU % e != 0) return 0;
  for (int i = 1; i < n; ++i)
    if (redge[i] != i % e) return 0;
  return e;
}

}  // namespace

bool chain_wave_headerless(const cfp_chain_desc &d) {
  return wave_edge_period(d.redge, d.n_blocks, d.n_tables) == 12;
}

bool chain_wave_supported(int n, int k, int e, int batch) { return wave_plan(n, k, e, batch).P >= 2; }

size_t wave_region_bytes(int n, int k, int e, int batch) {
  const WavePlan c = wave_plan(n, k, e, batch);
  if (c.P < 2) return 0;
  size_t off = align_up((size_t)e * 64 * 64 * 4);
  off += align_up((size_t)batch * c.P * sizeof(WaveRec));
  off += align_up((size_t)batch * c.nq * 8);
  off += align_up((size_t)batch * c.nq * 64 * 4);
  off += align_up((size_t)batch * c.P * 64 * 4);
  return off;
}

hipError_t launch_chain_wave(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *region, uint8_t *table,
                             SearchResult *res, const WsHeader *hdr, int64_t *opt, int32_t *status,
                             hipStream_t st) {
  const WavePlan c = wave_plan(d.n_blocks, d.k, d.n_tables, d.batch);
  WaveArgs a;
  a.cost = d.cost;
  a.redge = redge_dev;
  a.N = d.n_blocks;
  a.K = d.k;
  a.E = d.n_tables;
  a.B = d.batch;
  a.P = c.P;
  a.CB = c.CB;
  a.nblk = c.nblk;
  a.nq = c.nq;
  a.table = table;
  size_t off = 0;
  uint32_t *rpk = (uint32_t *)(region + off);
  a.rpk = (const u32x4 *)rpk;
  off += align_up((size_t)d.n_tables * 64 * 64 * 4);
  a.rec = (WaveRec *)(region + off);
  off += align_up((size_t)d.batch * c.P * sizeof(WaveRec));
  a.dck = (int64_t *)(region + off);
  off += align_up((size_t)d.batch * c.nq * 8);
  a.ckrow = (uint32_t *)(region + off);
  off += align_up((size_t)d.batch * c.nq * 64 * 4);
  a.endrow = (uint32_t *)(region + off);
  a.seq = next_call_number();
  hipLaunchKernelGGL(wave_pack_kernel, dim3(std::min(1024, d.n_tables * 16)), dim3(256), 0, st, d.rtab, d.n_tables,
                     d.k, rpk, cfp_r_limit(CFP_V_CHAIN, d.k), const_cast<WsHeader *>(hdr), a.seq);
  if (wave_edge_period(d.redge, d.n_blocks, d.n_tables) == 12) launch_wave_passes<12>(a, hdr, res, opt, status, st);
  else launch_wave_passes<0>(a, hdr, res, opt, status, st);
  return hipGetLastError();
}

}  // namespace cfp
