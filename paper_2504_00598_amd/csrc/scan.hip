// The chain search as a min-plus parallel scan (for long chains).
//
// Block i becomes the transfer matrix T_i[t][s] = R_{e(i)}[t][s] + c[i][s]
// (T_0[t][s] = c[0][s]: block 0 has no incoming edge), so that the forward
// recurrence of Sec. 4.4 is D[i] = D[i-1] (x) T_i with (v (x) T)[s] =
// min_t v[t] + T[t][s], and D[N-1] = 0 (x) T_0 (x) ... (x) T_{N-1}.  The
// min-plus matrix product is associative, so:
//   up-sweep   a tree of min-plus matrix products: level 0 holds the N
//              blocks, level l+1 the products of adjacent pairs of level l (an
//              unpaired last node moves up unchanged);
//   down-sweep the prefix vector entering every node: the root's is 0, a
//              left child inherits its parent's, a right child gets
//              parent (x) left-sibling product;
//   leaves     D[i] = prefix(i) (x) T_i, together with the lowest argmin
//              t of every state, which is the traceback table of the chain.
// Level-0 matrices are never stored: they are formed from R and c on the fly.
//
// Values.  Every stored matrix and vector holds uint32 entries "raw" with a
// per-object minimum mn and an int64 offset tot: true value = raw - mn + tot.
// Entries are clamped at BIG = 2^31 - 1 when read, so the plain 32-bit sums of
// a product never wrap.  Block costs enter as c[i][s] - min_s c[i][s] (BIG for
// an unavailable strategy).  The entries of a product over any run of blocks
// lie within 2 R_max + max_i (max_s c[i][s] - min_s c[i][s]) of its minimum,
// so with R < 2^23 and finite costs of a block within 2^30 of each other no
// entry that can matter reaches BIG and every result is exact; the second
// condition is checked on the device (status BADINPUT otherwise).
#include <type_traits>

#include "cfp_internal.h"
#include "common.h"

namespace cfp {

constexpr uint32_t kBig = 0x7FFFFFFFu;
constexpr int kTile = 128;  // output tile of a product
constexpr int kTk = 16;     // predecessor depth of one LDS stage
constexpr int kMaxLevels = 40;

__host__ __device__ inline int scan_kp(int k) { return (k + kTile - 1) / kTile * kTile; }

struct ScanLayout {
  int nlev;               // number of levels (level 0 = blocks)
  int cnt[kMaxLevels];    // nodes per level
  size_t mat[kMaxLevels]; // offset of the matrices of level l (l >= 1): [B][cnt][KP][KP] uint32
  size_t mn[kMaxLevels];  // [B][cnt] uint32
  size_t tot[kMaxLevels]; // [B][cnt] int64
  size_t pre[kMaxLevels]; // prefix vectors entering each node: [B][cnt][KP] uint32
  size_t ptot[kMaxLevels];// [B][cnt] int64
  size_t cmin;            // [B][N] int32
  size_t flags;           // [B] int32
  size_t bytes;
};

static ScanLayout scan_layout(int n, int k, int batch) {
  ScanLayout S;
  const size_t KP = scan_kp(k);
  S.nlev = 1;
  S.cnt[0] = n;
  while (S.cnt[S.nlev - 1] > 1 && S.nlev < kMaxLevels) {
    S.cnt[S.nlev] = (S.cnt[S.nlev - 1] + 1) / 2;
    ++S.nlev;
  }
  size_t off = 0;
  for (int l = 0; l < S.nlev; ++l) {
    const size_t c = (size_t)batch * S.cnt[l];
    S.mat[l] = off;
    if (l > 0) off = align_up(off + c * KP * KP * 4);
    S.mn[l] = off;
    off = align_up(off + c * 4);
    S.tot[l] = off;
    off = align_up(off + c * 8);
    S.pre[l] = off;
    off = align_up(off + c * KP * 4);
    S.ptot[l] = off;
    off = align_up(off + c * 8);
  }
  S.cmin = off;
  off = align_up(off + (size_t)batch * n * 4);
  S.flags = off;
  off = align_up(off + (size_t)batch * 4);
  S.bytes = off;
  return S;
}

size_t scan_region_bytes(int n, int k, int batch) { return scan_layout(n, k, batch).bytes; }

enum { SCANF_BAD = 1, SCANF_INFEASIBLE = 2 };

// cmin[b][i] = min_s c[b][i][s] over available strategies; validates the costs.
__global__ __launch_bounds__(256) void scan_prep_kernel(const int32_t *__restrict__ cost, int N, int K, int B,
                                                        int32_t *__restrict__ cmin, int32_t *__restrict__ flags) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= B * N) return;
  const int32_t *c = cost + (size_t)row * K;
  int32_t lo = CFP_COST_INF, hi = -1;
  bool neg = false;
  for (int s = lane; s < K; s += 64) {
    const int32_t v = c[s];
    neg |= v < 0;
    if (v != CFP_COST_INF) {
      lo = v < lo ? v : lo;
      hi = v > hi ? v : hi;
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const int32_t l2 = __shfl_xor(lo, off, 64), h2 = __shfl_xor(hi, off, 64);
    lo = l2 < lo ? l2 : lo;
    hi = h2 > hi ? h2 : hi;
  }
  neg = __any(neg);
  if (lane == 0) {
    cmin[row] = lo;
    int f = 0;
    if (neg || (hi >= 0 && (int64_t)hi - lo >= (1 << 30))) f |= SCANF_BAD;
    if (lo == CFP_COST_INF) f |= SCANF_INFEASIBLE;
    if (f) atomicOr(&flags[row / N], f);
  }
}

// Adjusted cost of block i, strategy s (BIG when unavailable or padding).
__device__ __forceinline__ uint32_t cadj(const int32_t *crow, int32_t cm, int s, int K) {
  if (s >= K) return kBig;
  const int32_t v = crow[s];
  return v == CFP_COST_INF ? kBig : (uint32_t)(v - cm);
}

struct ScanArgs {
  int N, K, KP, B, l;             // l: level of the products being formed (>= 1)
  const int32_t *cost, *rtab, *redge;
  const int32_t *cmin;
  const uint32_t *src;            // matrices of level l-1 (l >= 2)
  const uint32_t *src_mn;         // [B][cnt[l-1]]
  uint32_t *dst;                  // matrices of level l
  uint32_t *dst_mn;               // [B][cnt[l]]
  int cnt_src, cnt_dst;
};

// One 128x128 tile of C = A (x) B for the pair (2j, 2j+1) of level l-1.
// 256 threads; thread (ty, tx) owns rows {4ty..4ty+3, 64+4ty..} and columns
// {4tx..4tx+3, 64+4tx..} of the tile: 64 entries, two predecessors per
// update as two adds and one three-input min.
template <bool LEAF, bool FULL>
__global__ __launch_bounds__(256) void scan_gemm_kernel(ScanArgs a) {
  __shared__ __align__(16) uint32_t As[2][kTk][kTile];
  __shared__ __align__(16) uint32_t Bs[2][kTk][kTile];
  __shared__ uint32_t red[4];
  const int tid = threadIdx.x;
  const int tiles = a.KP / kTile;
  const int tile = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  const int tr0 = (tile / tiles) * kTile, tc0 = (tile % tiles) * kTile;
  const int K = a.K, KP = a.KP;
  const int ia = 2 * j, ib = 2 * j + 1;  // operand indices at level l-1

  // operand sources
  const int32_t *Ra = nullptr, *Rb = nullptr, *ca = nullptr, *cb = nullptr;
  int32_t cma = 0, cmb = 0;
  const uint32_t *Am = nullptr, *Bm = nullptr;
  uint32_t mna = 0, mnb = 0;
  if (LEAF) {
    ca = a.cost + ((size_t)b * a.N + ia) * K;
    cb = a.cost + ((size_t)b * a.N + ib) * K;
    cma = a.cmin[(size_t)b * a.N + ia];
    cmb = a.cmin[(size_t)b * a.N + ib];
    Ra = ia == 0 ? nullptr : a.rtab + (size_t)a.redge[ia] * K * K;
    Rb = a.rtab + (size_t)a.redge[ib] * K * K;
  } else {
    Am = a.src + ((size_t)b * a.cnt_src + ia) * KP * KP;
    Bm = a.src + ((size_t)b * a.cnt_src + ib) * KP * KP;
    mna = a.src_mn[(size_t)b * a.cnt_src + ia];
    mnb = a.src_mn[(size_t)b * a.cnt_src + ib];
  }

  // loader mapping: A tile row lr, 8 predecessors from lk; B tile row bk, 8 columns from bc
  const int lr = tid >> 1, lk = (tid & 1) * 8;
  const int bk = tid >> 4, bc = (tid & 15) * 8;
  uint32_t ra[8], rb[8];
  auto load8 = [&](const void *p, uint32_t (&v)[8]) __attribute__((always_inline)) {
    const uint4 x0 = ((const uint4 *)p)[0], x1 = ((const uint4 *)p)[1];
    v[0] = x0.x; v[1] = x0.y; v[2] = x0.z; v[3] = x0.w; v[4] = x1.x; v[5] = x1.y; v[6] = x1.z; v[7] = x1.w;
  };
  auto load = [&](int k0) __attribute__((always_inline)) {
    const int t = tr0 + lr;
    if (FULL) {  // K == KP: no padding, 16-byte aligned rows
      if (LEAF) {
        uint32_t c8[8], r8[8];
        load8(ca + k0 + lk, c8);
        if (Ra != nullptr) load8(Ra + (size_t)t * K + k0 + lk, r8);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const uint32_t cv = (int32_t)c8[q] == CFP_COST_INF ? kBig : c8[q] - (uint32_t)cma;
          ra[q] = umin(cv + (Ra != nullptr ? r8[q] : 0u), kBig);
        }
        load8(Rb + (size_t)(k0 + bk) * K + tc0 + bc, rb);
      } else {
        load8(Am + (size_t)t * KP + k0 + lk, ra);
        load8(Bm + (size_t)(k0 + bk) * KP + tc0 + bc, rb);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          ra[q] = umin(ra[q] - mna, kBig);
          rb[q] = umin(rb[q] - mnb, kBig);
        }
      }
      return;
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int k = k0 + lk + q;
      uint32_t v;
      if (LEAF) {
        const uint32_t cv = cadj(ca, cma, k, K);
        const uint32_t rv = (Ra == nullptr) ? 0u : (t < K && k < K) ? (uint32_t)Ra[(size_t)t * K + k] : kBig;
        v = umin(cv + rv, kBig);
      } else {
        v = umin(Am[(size_t)t * KP + k] - mna, kBig);
      }
      ra[q] = v;
    }
    const int k = k0 + bk;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int s = tc0 + bc + q;
      uint32_t v;
      if (LEAF)
        v = (k < K && s < K) ? (uint32_t)Rb[(size_t)k * K + s] : kBig;
      else
        v = umin(Bm[(size_t)k * KP + s] - mnb, kBig);
      rb[q] = v;
    }
  };
  auto store = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < 8; ++q) As[buf][lk + q][lr] = ra[q];
    *(uint4 *)&Bs[buf][bk][bc] = make_uint4(rb[0], rb[1], rb[2], rb[3]);
    *(uint4 *)&Bs[buf][bk][bc + 4] = make_uint4(rb[4], rb[5], rb[6], rb[7]);
  };

  const int ty = tid >> 4, tx = tid & 15;
  uint32_t acc[8][8];
#pragma unroll
  for (int r = 0; r < 8; ++r)
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[r][c] = kSat;

  const int nst = KP / kTk;
  load(0);
  store(0);
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    const int buf = st & 1;
    if (st + 1 < nst) load((st + 1) * kTk);
#pragma unroll 1  // one predecessor pair per iteration keeps the tile in 128 VGPRs
    for (int kk = 0; kk < kTk; kk += 2) {
      const uint4 a0l = *(const uint4 *)&As[buf][kk][4 * ty], a0h = *(const uint4 *)&As[buf][kk][64 + 4 * ty];
      const uint4 a1l = *(const uint4 *)&As[buf][kk + 1][4 * ty], a1h = *(const uint4 *)&As[buf][kk + 1][64 + 4 * ty];
      const uint4 b0l = *(const uint4 *)&Bs[buf][kk][4 * tx], b0h = *(const uint4 *)&Bs[buf][kk][64 + 4 * tx];
      const uint4 b1l = *(const uint4 *)&Bs[buf][kk + 1][4 * tx], b1h = *(const uint4 *)&Bs[buf][kk + 1][64 + 4 * tx];
      const uint32_t a0[8] = {a0l.x, a0l.y, a0l.z, a0l.w, a0h.x, a0h.y, a0h.z, a0h.w};
      const uint32_t a1[8] = {a1l.x, a1l.y, a1l.z, a1l.w, a1h.x, a1h.y, a1h.z, a1h.w};
      const uint32_t b0[8] = {b0l.x, b0l.y, b0l.z, b0l.w, b0h.x, b0h.y, b0h.z, b0h.w};
      const uint32_t b1[8] = {b1l.x, b1l.y, b1l.z, b1l.w, b1h.x, b1h.y, b1h.z, b1h.w};
#pragma unroll
      for (int r = 0; r < 8; ++r)
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          const uint32_t x = a0[r] + b0[c], y = a1[r] + b1[c];
          acc[r][c] = umin(acc[r][c], umin(x, y));
        }
    }
    if (st + 1 < nst) store(buf ^ 1);
    __syncthreads();
  }

  // epilogue: add the later block's cost (leaf products), clamp, store, tile minimum
  uint32_t *C = a.dst + ((size_t)b * a.cnt_dst + j) * KP * KP;
  uint32_t tmin = kSat;
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const int t = tr0 + (r < 4 ? 4 * ty + r : 64 + 4 * ty + r - 4);
    uint32_t out[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int s = tc0 + (c < 4 ? 4 * tx + c : 64 + 4 * tx + c - 4);
      uint32_t v = acc[r][c];
      if (LEAF) v = sat_add(v, cadj(cb, cmb, s, K));
      v = umin(v, kBig);
      out[c] = v;
      tmin = umin(tmin, v);
    }
    *(uint4 *)&C[(size_t)t * KP + tc0 + 4 * tx] = make_uint4(out[0], out[1], out[2], out[3]);
    *(uint4 *)&C[(size_t)t * KP + tc0 + 64 + 4 * tx] = make_uint4(out[4], out[5], out[6], out[7]);
  }
  tmin = wave_min(tmin);
  if ((tid & 63) == 0) red[tid >> 6] = tmin;
  __syncthreads();
  if (tid == 0) atomicMin(&a.dst_mn[(size_t)b * a.cnt_dst + j], umin(umin(red[0], red[1]), umin(red[2], red[3])));
}

// Level-l nodes: tot = tot(left) + tot(right) + mn for products; an unpaired
// last node is carried (its matrix copied, or formed from its block).
__global__ void scan_tot_kernel(ScanArgs a, const int64_t *__restrict__ src_tot, int64_t *__restrict__ dst_tot) {
  const int x = blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= a.B * a.cnt_dst) return;
  const int b = x / a.cnt_dst, j = x % a.cnt_dst;
  const int ia = 2 * j, ib = 2 * j + 1;
  auto node_tot = [&](int i) -> int64_t {
    if (a.l == 1) return (int64_t)a.cmin[(size_t)b * a.N + i];
    return src_tot[(size_t)b * a.cnt_src + i];
  };
  if (ib < a.cnt_src)
    dst_tot[x] = node_tot(ia) + node_tot(ib) + (int64_t)a.dst_mn[x];
  else
    dst_tot[x] = node_tot(ia);  // carried: tot of the single child, matrix copied with mn = the child's
}

// Copy (or form from its block) the unpaired last node of level l-1 into level l.
__global__ void scan_carry_kernel(ScanArgs a) {
  const int b = blockIdx.y;
  const int j = a.cnt_dst - 1, i = a.cnt_src - 1;
  const size_t n2 = (size_t)a.KP * a.KP;
  uint32_t *C = a.dst + ((size_t)b * a.cnt_dst + j) * n2;
  for (size_t x = (size_t)blockIdx.x * blockDim.x + threadIdx.x; x < n2; x += (size_t)gridDim.x * blockDim.x) {
    const int t = (int)(x / a.KP), s = (int)(x % a.KP);
    uint32_t v;
    if (a.l == 1) {
      const int32_t *c = a.cost + ((size_t)b * a.N + i) * a.K;
      const int32_t cm = a.cmin[(size_t)b * a.N + i];
      const uint32_t rv = i == 0 ? 0u
                                 : (t < a.K && s < a.K) ? (uint32_t)a.rtab[(size_t)a.redge[i] * a.K * a.K + (size_t)t * a.K + s]
                                                        : kBig;
      v = umin(rv + cadj(c, cm, s, a.K), kBig);
    } else {
      v = a.src[((size_t)b * a.cnt_src + i) * n2 + x];
    }
    C[x] = v;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0)
    a.dst_mn[(size_t)b * a.cnt_dst + j] = a.l == 1 ? 0u : a.src_mn[(size_t)b * a.cnt_src + i];
}

__global__ void scan_fill_kernel(uint32_t *p, size_t n, uint32_t v) {
  for (size_t x = (size_t)blockIdx.x * blockDim.x + threadIdx.x; x < n; x += (size_t)gridDim.x * blockDim.x) p[x] = v;
}

struct DownArgs {
  int N, K, KP, B, l;  // level l >= 1: children at level l-1
  const int32_t *cost, *rtab, *redge, *cmin;
  const uint32_t *mat;     // matrices of level l-1 (l-1 >= 1)
  const uint32_t *mat_mn;  // [B][cnt[l-1]]
  const int64_t *mat_tot;
  const uint32_t *pre;     // prefix vectors entering the nodes of level l
  const int64_t *ptot;
  uint32_t *cpre;          // prefix vectors entering the nodes of level l-1
  int64_t *cptot;
  int cnt, ccnt;
};

constexpr int kVmRows = 16;  // matrix rows in flight per thread in vecmat

// v (x) M for one vector and one matrix (a block's transfer matrix when
// the matrices are level 0); returns the minimum of the output in `mn` and
// writes out - mn.  256 threads, KP/256 outputs each.
template <bool TRACK>
__device__ void vecmat(const uint32_t *v, int KP, int K, const uint32_t *Mm, uint32_t mmn, const int32_t *R,
                       bool block0, const int32_t *crow, int32_t cm, uint32_t *out, uint32_t &mn,
                       uint32_t *args_out, uint32_t *red) {
  const int tid = threadIdx.x;
  uint32_t best[2] = {kSat, kSat}, arg[2] = {0, 0};
  // Rows t are taken kVmRows at a time: every load of a batch is issued
  // before any is used (one memory latency per batch rather than per row),
  // from clamped addresses, so that no load sits behind a branch; entries of
  // columns past KP (or past K for R) are never used.
  const int c0 = tid, c1 = tid + 256;
  auto take = [&](int t, uint32_t a0, uint32_t a1) __attribute__((always_inline)) {
    const uint32_t vt = umin(v[t], kBig);
    const uint32_t x0 = vt + a0, x1 = vt + a1;  // both below 2^32
    if (x0 < best[0]) {
      best[0] = x0;
      arg[0] = t;
    }
    if (x1 < best[1]) {
      best[1] = x1;
      arg[1] = t;
    }
  };
  if (Mm) {
    const uint32_t *p0 = Mm + min(c0, KP - 1), *p1 = Mm + min(c1, KP - 1);
    for (int t0 = 0; t0 < KP; t0 += kVmRows) {
      uint32_t m0[kVmRows], m1[kVmRows];
#pragma unroll
      for (int u = 0; u < kVmRows; ++u) {
        m0[u] = p0[(size_t)(t0 + u) * KP];
        m1[u] = p1[(size_t)(t0 + u) * KP];
      }
#pragma unroll
      for (int u = 0; u < kVmRows; ++u) take(t0 + u, umin(m0[u] - mmn, kBig), umin(m1[u] - mmn, kBig));
    }
  } else if (block0) {
    for (int t = 0; t < KP; ++t) take(t, 0u, 0u);
  } else {
    const int32_t *p0 = R + min(c0, K - 1), *p1 = R + min(c1, K - 1);
    const bool k0 = c0 < K, k1 = c1 < K;
    for (int t0 = 0; t0 < KP; t0 += kVmRows) {
      uint32_t m0[kVmRows], m1[kVmRows];
#pragma unroll
      for (int u = 0; u < kVmRows; ++u) {
        const size_t row = (size_t)min(t0 + u, K - 1) * K;
        m0[u] = (uint32_t)p0[row];
        m1[u] = (uint32_t)p1[row];
      }
#pragma unroll
      for (int u = 0; u < kVmRows; ++u) {
        const bool tin = t0 + u < K;
        take(t0 + u, tin && k0 ? m0[u] : kBig, tin && k1 ? m1[u] : kBig);
      }
    }
  }
  uint32_t lmin = kSat;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int s = tid + 256 * h;
    if (s >= KP) continue;
    uint32_t o = umin(best[h], kBig);
    if (!Mm) o = umin(sat_add(o, cadj(crow, cm, s, K)), kBig);  // a block adds its own cost
    best[h] = o;
    lmin = umin(lmin, o);
    if (TRACK) args_out[s] = arg[h];
  }
  lmin = wave_min(lmin);
  if ((tid & 63) == 0) red[tid >> 6] = lmin;
  __syncthreads();
  mn = umin(umin(red[0], red[1]), umin(red[2], red[3]));
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int s = tid + 256 * h;
    if (s < KP) out[s] = best[h] - mn;
  }
  __syncthreads();
}

// Down-sweep one level: node (l, j) hands its prefix to its left child and
// prefix (x) left-child matrix to its right child.
__global__ __launch_bounds__(256) void scan_down_kernel(DownArgs a) {
  extern __shared__ __align__(16) uint32_t sm[];
  __shared__ uint32_t red[4];
  uint32_t *v = sm;  // [KP]
  const int j = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int KP = a.KP;
  const uint32_t *pv = a.pre + ((size_t)b * a.cnt + j) * KP;
  for (int t = tid; t < KP; t += 256) v[t] = pv[t];
  __syncthreads();
  const int64_t ptot = a.ptot[(size_t)b * a.cnt + j];
  const int ia = 2 * j, ib = 2 * j + 1;
  uint32_t *lv = a.cpre + ((size_t)b * a.ccnt + ia) * KP;
  for (int t = tid; t < KP; t += 256) lv[t] = v[t];
  if (tid == 0) a.cptot[(size_t)b * a.ccnt + ia] = ptot;
  if (ib >= a.ccnt) return;
  uint32_t *rv = a.cpre + ((size_t)b * a.ccnt + ib) * KP;
  uint32_t mn;
  int64_t mtot;
  if (a.l == 1) {
    // left child is block ia: its transfer matrix from R and c
    const int32_t *crow = a.cost + ((size_t)b * a.N + ia) * a.K;
    const int32_t cm = a.cmin[(size_t)b * a.N + ia];
    const int32_t *R = ia == 0 ? nullptr : a.rtab + (size_t)a.redge[ia] * a.K * a.K;
    vecmat<false>(v, KP, a.K, nullptr, 0, R, ia == 0, crow, cm, rv, mn, nullptr, red);
    mtot = cm;
  } else {
    const size_t mi = (size_t)b * a.ccnt + ia;
    vecmat<false>(v, KP, a.K, a.mat + mi * KP * KP, a.mat_mn[mi], nullptr, false, nullptr, 0, rv, mn, nullptr, red);
    mtot = a.mat_tot[mi];
  }
  if (tid == 0) a.cptot[(size_t)b * a.ccnt + ib] = ptot + mtot + (int64_t)mn;
}

// Leaves: D[i] = prefix(i) (x) T_i with the argmin table row i; block N-1
// reports the search.
template <typename T>
__global__ __launch_bounds__(256) void scan_leaf_kernel(DownArgs a, T *__restrict__ table,
                                                        const int32_t *__restrict__ flags,
                                                        const WsHeader *__restrict__ hdr, SearchResult *__restrict__ res,
                                                        int64_t *__restrict__ opt, int32_t *__restrict__ status) {
  extern __shared__ __align__(16) uint32_t sm[];
  __shared__ uint32_t red[4];
  const int KP = a.KP, K = a.K;
  uint32_t *v = sm, *out = sm + KP, *args = sm + 2 * KP;
  const int i = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const uint32_t *pv = a.pre + ((size_t)b * a.N + i) * KP;
  for (int t = tid; t < KP; t += 256) v[t] = pv[t];
  __syncthreads();
  const int32_t *crow = a.cost + ((size_t)b * a.N + i) * K;
  const int32_t cm = a.cmin[(size_t)b * a.N + i];
  const int32_t *R = i == 0 ? nullptr : a.rtab + (size_t)a.redge[i] * K * K;
  uint32_t mn;
  vecmat<true>(v, KP, K, nullptr, 0, R, i == 0, crow, cm, out, mn, args, red);
  if (i > 0)
    for (int s = tid; s < K; s += 256) table[((size_t)b * a.N + i) * K + s] = (T)args[s];
  if (i == a.N - 1) {
    // lowest final state of least value
    uint32_t pk = kSat;
    int ps = 0;
    for (int s = tid; s < K; s += 256)
      if (out[s] < pk) {
        pk = out[s];
        ps = s;
      }
    // (value, state) minimum over the block, lowest state on ties
    uint64_t key = ((uint64_t)pk << 32) | (uint32_t)ps;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const uint64_t o = __shfl_xor(key, off, 64);
      key = o < key ? o : key;
    }
    __shared__ uint64_t kred[4];
    if ((tid & 63) == 0) kred[tid >> 6] = key;
    __syncthreads();
    if (tid == 0) {
      uint64_t k = kred[0];
      for (int w = 1; w < 4; ++w) k = kred[w] < k ? kred[w] : k;
      const int f = flags[b];
      int st = CFP_ST_OK;
      if ((f & SCANF_BAD) || hdr->rflag) st = CFP_ST_BADINPUT;
      else if ((f & SCANF_INFEASIBLE) || (uint32_t)(k >> 32) >= kBig) st = CFP_ST_INFEASIBLE;
      const int64_t total = a.ptot[(size_t)b * a.N + i] + (int64_t)cm + (int64_t)mn + (int64_t)(k >> 32);
      status[b] = st;
      opt[b] = st == CFP_ST_OK ? total : INT64_MAX;
      res[b].final_state = st == CFP_ST_OK ? (int32_t)(k & 0xFFFFFFFFu) : -1;
      res[b].status = st;
      res[b].final_m = 0;
    }
  }
}

hipError_t launch_scan(const cfp_chain_desc &d, const int32_t *redge_dev, uint8_t *region, size_t region_bytes,
                       uint8_t *table, int elem, SearchResult *res, const WsHeader *hdr, int64_t *opt,
                       int32_t *status, hipStream_t st) {
  (void)region_bytes;
  const int N = d.n_blocks, K = d.k, B = d.batch, KP = scan_kp(K);
  const ScanLayout S = scan_layout(N, K, B);
  int32_t *cmin = (int32_t *)(region + S.cmin);
  int32_t *flags = (int32_t *)(region + S.flags);
  hipLaunchKernelGGL(scan_fill_kernel, dim3(1), dim3(256), 0, st, (uint32_t *)flags, (size_t)B, 0u);
  hipLaunchKernelGGL(scan_prep_kernel, dim3((B * N + 3) / 4), dim3(256), 0, st, d.cost, N, K, B, cmin, flags);

  // up-sweep
  for (int l = 1; l < S.nlev; ++l) {
    ScanArgs a;
    a.N = N; a.K = K; a.KP = KP; a.B = B; a.l = l;
    a.cost = d.cost; a.rtab = d.rtab; a.redge = redge_dev; a.cmin = cmin;
    a.src = l >= 2 ? (const uint32_t *)(region + S.mat[l - 1]) : nullptr;
    a.src_mn = (const uint32_t *)(region + S.mn[l - 1]);
    a.dst = (uint32_t *)(region + S.mat[l]);
    a.dst_mn = (uint32_t *)(region + S.mn[l]);
    a.cnt_src = S.cnt[l - 1];
    a.cnt_dst = S.cnt[l];
    hipLaunchKernelGGL(scan_fill_kernel, dim3(64), dim3(256), 0, st, a.dst_mn, (size_t)B * S.cnt[l], kSat);
    const int pairs = S.cnt[l - 1] / 2;
    if (pairs > 0) {
      const dim3 grid((KP / kTile) * (KP / kTile), pairs, B);
      // vector loads need unpadded rows and 16-byte aligned inputs
      const bool full = K == KP && ((uintptr_t)d.cost % 16) == 0 && ((uintptr_t)d.rtab % 16) == 0;
      timer_begin(st);
      if (l == 1) {
        if (full) timed_launch(scan_gemm_kernel<true, true>, grid, dim3(256), 0, st, a);
        else timed_launch(scan_gemm_kernel<true, false>, grid, dim3(256), 0, st, a);
      } else {
        if (full) timed_launch(scan_gemm_kernel<false, true>, grid, dim3(256), 0, st, a);
        else timed_launch(scan_gemm_kernel<false, false>, grid, dim3(256), 0, st, a);
      }
      timer_end(st);
    }
    if (S.cnt[l - 1] & 1) hipLaunchKernelGGL(scan_carry_kernel, dim3(64, B), dim3(256), 0, st, a);
    hipLaunchKernelGGL(scan_tot_kernel, dim3((B * S.cnt[l] + 255) / 256), dim3(256), 0, st, a,
                       (const int64_t *)(region + S.tot[l - 1]), (int64_t *)(region + S.tot[l]));
  }

  // down-sweep: the root's prefix is the zero vector
  const int top = S.nlev - 1;
  hipLaunchKernelGGL(scan_fill_kernel, dim3(64), dim3(256), 0, st, (uint32_t *)(region + S.pre[top]),
                     (size_t)B * KP, 0u);
  hipLaunchKernelGGL(scan_fill_kernel, dim3(1), dim3(256), 0, st, (uint32_t *)(region + S.ptot[top]),
                     (size_t)B * 2, 0u);
  for (int l = top; l >= 1; --l) {
    DownArgs a;
    a.N = N; a.K = K; a.KP = KP; a.B = B; a.l = l;
    a.cost = d.cost; a.rtab = d.rtab; a.redge = redge_dev; a.cmin = cmin;
    a.mat = l - 1 >= 1 ? (const uint32_t *)(region + S.mat[l - 1]) : nullptr;
    a.mat_mn = (const uint32_t *)(region + S.mn[l - 1]);
    a.mat_tot = (const int64_t *)(region + S.tot[l - 1]);
    a.pre = (const uint32_t *)(region + S.pre[l]);
    a.ptot = (const int64_t *)(region + S.ptot[l]);
    a.cpre = (uint32_t *)(region + S.pre[l - 1]);
    a.cptot = (int64_t *)(region + S.ptot[l - 1]);
    a.cnt = S.cnt[l];
    a.ccnt = S.cnt[l - 1];
    hipLaunchKernelGGL(scan_down_kernel, dim3(S.cnt[l], B), dim3(256), (size_t)KP * 4, st, a);
  }
  DownArgs a;
  a.N = N; a.K = K; a.KP = KP; a.B = B; a.l = 0;
  a.cost = d.cost; a.rtab = d.rtab; a.redge = redge_dev; a.cmin = cmin;
  a.mat = nullptr; a.mat_mn = nullptr; a.mat_tot = nullptr;
  a.pre = (const uint32_t *)(region + S.pre[0]);
  a.ptot = (const int64_t *)(region + S.ptot[0]);
  a.cpre = nullptr; a.cptot = nullptr;
  a.cnt = N; a.ccnt = 0;
  const size_t lds = (size_t)3 * KP * 4;
  if (elem == 1)
    hipLaunchKernelGGL(scan_leaf_kernel<uint8_t>, dim3(N, B), dim3(256), lds, st, a, table, flags, hdr, res, opt, status);
  else
    hipLaunchKernelGGL(scan_leaf_kernel<uint16_t>, dim3(N, B), dim3(256), lds, st, a, (uint16_t *)table, flags, hdr, res,
                       opt, status);
  return hipGetLastError();
}

}  // namespace cfp
