// HBM-bound passes of the MALT / MALTER step (gfx950):
//   momentum_rowcol   M <- mu1 M + (1-mu1) G, per-tile row and column sums of G^2
//   precond_finalize  l, r EMAs and L = (l+eps)^(-1/8), R = (r+eps)^(-1/8)
//   scale_convert     X0 = bf16(L M R) in the canonical orientation, ||LMR||^2
//                     and (MALTER) ||LGR||^2 partials
//   norm_scalars      s, sigma, nu_t, alpha_t per matrix
//   graft_scalars     ||O||, ||D||, graft and step coefficient per matrix
//   backmap_write     W <- decay W - coef * L O R
// Reductions are two-stage and deterministic: fixed per-tile partials, then a
// fixed-order combine in float64.  No float atomics.
#include "malt_internal.h"

namespace malt {

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

typedef float ew_f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned ew_u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned ew_u32x4 __attribute__((ext_vector_type(4)));

// Load 4 consecutive floats of one row starting at column c (columns >= n
// read 0). STREAM marks data this step reads once (non-temporal load).
// INSIDE: the caller has established that the row allows 16-byte access and
// c + 3 < n, so the load is unconditional.
template <bool STREAM = false, bool INSIDE = false>
__device__ __forceinline__ void load4(const MALT_GLOBAL float* __restrict__ p, int c, int n, bool vec, float v[4]) {
  if (INSIDE || (vec && c + 3 < n)) {
    ew_f32x4 x;
    if (STREAM) x = __builtin_nontemporal_load(reinterpret_cast<const MALT_GLOBAL ew_f32x4*>(p + c));
    else x = *reinterpret_cast<const MALT_GLOBAL ew_f32x4*>(p + c);
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = (c + e < n) ? p[c + e] : 0.f;
  }
}

template <bool INSIDE = false>
__device__ __forceinline__ void store4(MALT_GLOBAL float* __restrict__ p, int c, int n, bool vec, const float v[4]) {
  if (INSIDE || (vec && c + 3 < n)) {
    const ew_f32x4 x = {v[0], v[1], v[2], v[3]};
    *reinterpret_cast<MALT_GLOBAL ew_f32x4*>(p + c) = x;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (c + e < n) p[c + e] = v[e];
  }
}

// One matrix's descriptor fields and caller pointers, as the tile passes use
// them, read in one place before any branch: the compiler then issues them as
// one batch of scalar loads, not a chain of load-and-wait behind each test.
struct EwView {
  int m, n, np, tall;
  bool vec;
  MALT_GLOBAL float* W;
  const MALT_GLOBAL float* G;
  MALT_GLOBAL float* M;
  const MALT_GLOBAL float* Lv;
  const MALT_GLOBAL float* Rv;
  MALT_GLOBAL float* rowpart;
  MALT_GLOBAL float* colpart;
  MALT_GLOBAL float* k2part;
  MALT_GLOBAL bf16_t* X0;
  const MALT_GLOBAL bf16_t* O;   // back-map: the buffer holding the final iterate
  const MALT_GLOBAL double* scal;
};

__device__ __forceinline__ EwView ew_view(const EwArgs& a, int mat) {
  const MatDesc& d = a.desc[mat];
  const PtrPair& p = a.ptrs[mat];
  EwView v;
  v.m = d.m;
  v.n = d.n;
  v.np = d.np;
  v.tall = d.tall;
  v.vec = p.vec != 0;
  v.W = gptr(p.W);
  v.G = gptr(p.G);
  v.M = gptr(d.M);
  v.Lv = gptr(d.Lv);
  v.Rv = gptr(d.Rv);
  v.rowpart = gptr(d.rowpart);
  v.colpart = gptr(d.colpart);
  v.k2part = gptr(d.k2part);
  v.X0 = gptr(d.X[0]);
  v.O = gptr(d.X[a.o_parity]);
  v.scal = gptr(d.scal);
  return v;
}

// ---------------------------------------------------------------------------
// Momentum EMA (Alg. 1/2, momentum line) fused with the per-tile row and
// column sums of G^2 that feed the l, r EMAs (Eq. dp_preconditioner).
// Reads G and M, writes M: 12 bytes per element.
// ---------------------------------------------------------------------------
// Interior tiles (every row and column of the tile inside the matrix, rows
// open to 16-byte access) take INSIDE = true: no bounds test anywhere, so
// each lane's loads form one straight run and are all in flight together.
// (With a bounds branch per row the compiler waited for one row's loads
// before issuing the next row's.)  Edge tiles take the checked path.
template <bool INSIDE>
__device__ __forceinline__ void momentum_tile(const EwArgs& a, const EwView& v, const Tile& t, float (*colsh)[EW_TC]) {
  constexpr int NW = EW_THREADS / 64, RPW = EW_TR / NW;   // 16 waves, 2 rows each
  static_assert(NW * RPW == EW_TR && EW_TC == 256, "one 256-column row segment per wave and row");
  const int m = v.m, n = v.n;
  const bool vec = v.vec;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r0 = t.ti * EW_TR + w * RPW, c = t.tj * EW_TC + lane * 4;
  const MALT_GLOBAL float* __restrict__ G = v.G;
  MALT_GLOBAL float* __restrict__ M = v.M;
  MALT_GLOBAL float* __restrict__ rowpart = v.rowpart;
  MALT_GLOBAL float* __restrict__ colpart = v.colpart;
  float g[RPW][4], mm[RPW][4];
#pragma unroll
  for (int u = 0; u < RPW; ++u) {
    if (INSIDE || r0 + u < m) {
      const size_t off = (size_t)(r0 + u) * n;
      load4<true, INSIDE>(G + off, c, n, vec, g[u]);
      load4<false, INSIDE>(M + off, c, n, vec, mm[u]);
    }
  }
  float cacc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int u = 0; u < RPW; ++u) {
    const int r = r0 + u;
    if (!INSIDE && r >= m) break;   // uniform over the wave
    float racc = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      mm[u][e] = a.mu1 * mm[u][e] + a.one_minus_mu1 * g[u][e];
      const float g2 = g[u][e] * g[u][e];
      racc += g2;
      cacc[e] += g2;
    }
    store4<INSIDE>(M + (size_t)r * n, c, n, vec, mm[u]);
    racc = wave_sum(racc);
    if (lane == 0) rowpart[(size_t)t.tj * m + r] = racc;
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) colsh[w][lane * 4 + e] = cacc[e];
  __syncthreads();
  const int cc = threadIdx.x;
  const int col = t.tj * EW_TC + cc;
  if (cc < EW_TC && (INSIDE || col < n)) {
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < NW; ++k) s += colsh[k][cc];
    colpart[(size_t)t.ti * n + col] = s;
  }
}

__global__ __launch_bounds__(EW_THREADS) void momentum_rowcol_kernel(EwArgs a) {
  __shared__ float colsh[EW_THREADS / 64][EW_TC];
  const Tile t = a.tiles[xcd_remap(blockIdx.x, gridDim.x)];
  const EwView v = ew_view(a, t.mat);
  const bool inside = v.vec & ((t.ti + 1) * EW_TR <= v.m) & ((t.tj + 1) * EW_TC <= v.n);
  if (inside) momentum_tile<true>(a, v, t, colsh);
  else momentum_tile<false>(a, v, t, colsh);
}

// ---------------------------------------------------------------------------
// Row / column EMAs and the diagonal preconditioners.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NTHREADS) void precond_finalize_kernel(EwArgs a) {
  // Tile (mat, 0 = rows | 1 = columns, chunk): FIN_W rows or columns, each
  // summed by FIN_SPLIT threads (every FIN_SPLIT-th partial, in order), the
  // thread sums combined in a fixed order.
  constexpr int SPLIT = NTHREADS / FIN_W;
  static_assert(SPLIT == 4, "pairwise combine of four sums");
  __shared__ double part[SPLIT][FIN_W];
  const Tile t = a.tiles[blockIdx.x];
  const MatDesc& d = a.desc[t.mat];
  const bool rows = t.ti == 0;
  const int len = rows ? d.m : d.n, nparts = rows ? d.k1_ct : d.k1_rt;
  const MALT_GLOBAL float* const src = gptr(rows ? d.rowpart : d.colpart);
  const int g = threadIdx.x / FIN_W, j = threadIdx.x % FIN_W;
  const int i = t.tj * FIN_W + j;
  // Eight partials in flight per thread, still added one by one in order
  // (a column of a 5120-row matrix has 160 partials, 40 per thread).
  double s = 0.0;
  if (i < len) {
    int c = g;
    for (; c + 7 * SPLIT < nparts; c += 8 * SPLIT) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = src[(size_t)(c + u * SPLIT) * len + i];
#pragma unroll
      for (int u = 0; u < 8; ++u) s += (double)v[u];
    }
    for (; c < nparts; c += SPLIT) s += (double)src[(size_t)c * len + i];
  }
  part[g][j] = s;
  __syncthreads();
  if (g != 0 || i >= len) return;
  const double sum = (part[0][j] + part[1][j]) + (part[2][j] + part[3][j]);
  float* const ema = rows ? d.l : d.r;
  float* const inv = rows ? d.Lv : d.Rv;
  const double v = a.mu2 * (double)gptr(ema)[i] + (1.0 - a.mu2) * sum;
  gptr(ema)[i] = (float)v;
  gptr(inv)[i] = a.identity ? 1.f : (float)pow(v + a.eps, -0.125);
}

// ---------------------------------------------------------------------------
// X0 = bf16(L M R) in the canonical orientation over the zero-padded domain,
// plus per-tile sums of (LMR)^2 and, for MALTER, (LGR)^2.
// ---------------------------------------------------------------------------
// Wide matrices: the canonical matrix is W. Tiles of K2W_R padded rows x
// EW_TC padded columns; each wave converts K2W_R / waves consecutive rows, one
// float4 of M (and of G) per lane and row, all loads issued first.
// Interior tiles (INSIDE: all K2W_R rows and EW_TC columns inside W, 16-byte
// rows) load without bounds tests, as in the momentum pass.
template <bool MALTER, bool INSIDE>
__device__ __forceinline__ void scale_convert_wide_tile(const EwView& v, const Tile& t, float (*red)[K2W_THREADS / 64]) {
  constexpr int NW = K2W_THREADS / 64, RPW = K2W_R / NW;
  static_assert(NW * RPW == K2W_R && EW_TC == 256, "whole 256-column row segments per wave");
  const int m = v.m, n = v.n;
  const bool vec = v.vec;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int rw = t.ti * K2W_R + w * RPW, c = t.tj * EW_TC + lane * 4;   // rows < mp, c < np
  const MALT_GLOBAL float* __restrict__ M = v.M;
  const MALT_GLOBAL float* __restrict__ G = v.G;
  const MALT_GLOBAL float* __restrict__ Lv = v.Lv;
  MALT_GLOBAL bf16_t* __restrict__ X0 = v.X0;
  const int ldx = v.np;
  float mm[RPW][4], gg[RPW][4], rv[4];
#pragma unroll
  for (int u = 0; u < RPW; ++u) {
#pragma unroll
    for (int e = 0; e < 4; ++e) mm[u][e] = gg[u][e] = 0.f;
    if (INSIDE || rw + u < m) {
      load4<false, INSIDE>(M + (size_t)(rw + u) * n, c, n, vec, mm[u]);
      if (MALTER) load4<false, INSIDE>(G + (size_t)(rw + u) * n, c, n, vec, gg[u]);
    }
  }
  load4<false, INSIDE>(v.Rv, c, n, true, rv);
  float lv[RPW];   // all read before the first store, which the compiler cannot tell apart from Lv
#pragma unroll
  for (int u = 0; u < RPW; ++u) lv[u] = (INSIDE || rw + u < m) ? Lv[rw + u] : 0.f;
  float s2 = 0.f, q2 = 0.f;
#pragma unroll
  for (int u = 0; u < RPW; ++u) {
    const int r = rw + u;
    const float li = lv[u];
    float x[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[e] = li * mm[u][e] * rv[e];
      s2 += x[e] * x[e];
      if (MALTER) {
        const float y = li * gg[u][e] * rv[e];
        q2 += y * y;
      }
    }
    // X0 is consumed by the next kernel from L2/HBM; streaming store.
    const ew_u32x2 pk = {pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3])};
    __builtin_nontemporal_store(pk, reinterpret_cast<MALT_GLOBAL ew_u32x2*>(X0 + (size_t)r * ldx + c));
  }
  s2 = wave_sum(s2);
  if (MALTER) q2 = wave_sum(q2);
  if (lane == 0) {
    red[0][w] = s2;
    red[1][w] = q2;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float so = 0.f, sq = 0.f;
#pragma unroll
    for (int k = 0; k < NW; ++k) {
      so += red[0][k];
      sq += red[1][k];
    }
    v.k2part[2 * (size_t)t.idx + 0] = so;
    v.k2part[2 * (size_t)t.idx + 1] = sq;
  }
}

template <bool MALTER>
__global__ __launch_bounds__(K2W_THREADS) void scale_convert_wide_kernel(EwArgs a) {
  __shared__ float red[2][K2W_THREADS / 64];
  const Tile t = a.tiles[xcd_remap(blockIdx.x, gridDim.x)];
  const EwView v = ew_view(a, t.mat);
  const bool inside = v.vec & ((t.ti + 1) * K2W_R <= v.m) & ((t.tj + 1) * EW_TC <= v.n);
  if (inside) scale_convert_wide_tile<MALTER, true>(v, t, red);
  else scale_convert_wide_tile<MALTER, false>(v, t, red);
}

// Tall matrices: the canonical matrix is W^T, written through an LDS
// transpose. Tiles cover W-oriented padded rows x cols in K2_T x K2_T blocks;
// one workgroup converts K2_GROUP consecutive tiles, a 64-row band of
// K2_GROUP * 64 W columns of one matrix (a matrix's tiles are listed band by
// band, and every band holds a multiple of K2_GROUP tiles).
// Each thread converts two consecutive W rows of four W columns per tile, so
// it holds, per W column, the two bf16 values of one 32-bit word of the
// canonical row (canonical columns 2p, 2p + 1).  The words go to LDS as
// [canonical row][word], word p of row c rotated to (p + 2 (c / 4) + c % 4)
// mod 32 (tall_word): the 32 lanes of each half-wave hit 32 distinct banks,
// both when writing (16 column groups x 2 row pairs) and when the copy-out
// reads its 16-byte row pieces back as four words.  X0 leaves in 128-byte row
// pieces.
__device__ __forceinline__ int tall_word(int c, int p) { return c * (K2_T / 2) + ((p + 2 * (c >> 2) + (c & 3)) & (K2_T / 2 - 1)); }

// Interior groups (INSIDE: the 64 W rows and TG * 64 W columns inside W,
// 16-byte rows) load without bounds tests, as in the momentum pass.
template <bool MALTER, bool INSIDE>
__device__ __forceinline__ void scale_convert_tall_group(const EwView& v, const Tile& t, uint32_t (*tsh)[K2_T * (K2_T / 2)],
                                                         float (*red)[K2T_THREADS / 64]) {
  constexpr int TG = K2_GROUP;
  constexpr int NW = K2T_THREADS / 64;
  constexpr int NP = K2T_THREADS / 16;         // row pairs per pass: 16 threads x 4 columns span 64 columns
  constexpr int PASSES = K2_T / (2 * NP);      // row-pair passes per tile
  constexpr int WPR = K2_T / 2;                // words per canonical row of a tile
  constexpr int CPR = WPR / 4;                 // 16-byte pieces per canonical row of a tile
  constexpr int ROWS_OUT = K2T_THREADS / CPR;  // canonical rows per copy-out pass
  static_assert(PASSES * 2 * NP == K2_T && K2_T % ROWS_OUT == 0, "tall tile layout");
  static_assert(WPR == 32, "tall_word rotates within 32-word rows");
  const int m = v.m, n = v.n;
  const bool vec = v.vec;
  MALT_GLOBAL bf16_t* __restrict__ X0 = v.X0;
  const int ldx = v.np;                  // canonical row pitch
  const MALT_GLOBAL float* __restrict__ M = v.M;
  const MALT_GLOBAL float* __restrict__ G = v.G;
  const int r0 = t.ti * K2_T, cb = t.tj * K2_T;   // band columns cb .. cb + TG*K2_T
  const int cg = threadIdx.x & 15;                // W columns 4 cg .. 4 cg + 3 of each tile
  const int pp = threadIdx.x >> 4;                // row pair pp + NP * pass

  float Li[PASSES][2];
#pragma unroll
  for (int ps = 0; ps < PASSES; ++ps)
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int r = r0 + 2 * (pp + NP * ps) + u;
      Li[ps][u] = (INSIDE || r < m) ? v.Lv[r] : 0.f;
    }
  float Rv[TG][4];
#pragma unroll
  for (int j = 0; j < TG; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int c = cb + j * K2_T + 4 * cg + e;
      Rv[j][e] = (INSIDE || c < n) ? v.Rv[c] : 0.f;
    }
  float mm[TG][PASSES][2][4], gg[TG][PASSES][2][4];
#pragma unroll
  for (int j = 0; j < TG; ++j)
#pragma unroll
    for (int ps = 0; ps < PASSES; ++ps)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int r = r0 + 2 * (pp + NP * ps) + u;
        const int c = cb + j * K2_T + 4 * cg;
#pragma unroll
        for (int e = 0; e < 4; ++e) mm[j][ps][u][e] = gg[j][ps][u][e] = 0.f;
        if (INSIDE || r < m) {
          load4<false, INSIDE>(M + (size_t)r * n, c, n, vec, mm[j][ps][u]);
          if (MALTER) load4<false, INSIDE>(G + (size_t)r * n, c, n, vec, gg[j][ps][u]);
        }
      }

  float s2[TG], q2[TG];
#pragma unroll
  for (int j = 0; j < TG; ++j) {
    s2[j] = 0.f;
    q2[j] = 0.f;
#pragma unroll
    for (int ps = 0; ps < PASSES; ++ps) {
      const int p = pp + NP * ps;   // word index: W rows 2p, 2p + 1 of the tile
      float x[2][4];
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          x[u][e] = Li[ps][u] * mm[j][ps][u][e] * Rv[j][e];
          s2[j] += x[u][e] * x[u][e];
          if (MALTER) {
            const float y = Li[ps][u] * gg[j][ps][u][e] * Rv[j][e];
            q2[j] += y * y;
          }
        }
#pragma unroll
      for (int e = 0; e < 4; ++e) tsh[j][tall_word(4 * cg + e, p)] = pack_bf16x2(x[0][e], x[1][e]);
    }
  }
  __syncthreads();
  // Copy-out: thread -> (canonical row, 16-byte piece); CPR threads per row.
  const int piece = threadIdx.x % CPR;
#pragma unroll
  for (int j = 0; j < TG; ++j)
#pragma unroll
    for (int rr = threadIdx.x / CPR; rr < K2_T; rr += ROWS_OUT) {
      const ew_u32x4 wv = {tsh[j][tall_word(rr, 4 * piece + 0)], tsh[j][tall_word(rr, 4 * piece + 1)],
                          tsh[j][tall_word(rr, 4 * piece + 2)], tsh[j][tall_word(rr, 4 * piece + 3)]};
      __builtin_nontemporal_store(
          wv, reinterpret_cast<MALT_GLOBAL ew_u32x4*>(X0 + (size_t)(cb + j * K2_T + rr) * ldx + r0 + 8 * piece));
    }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int j = 0; j < TG; ++j) {
    const float sj = wave_sum(s2[j]);
    const float qj = MALTER ? wave_sum(q2[j]) : 0.f;
    if (lane == 0) {
      red[2 * j][w] = sj;
      red[2 * j + 1][w] = qj;
    }
  }
  __syncthreads();
  if (threadIdx.x < TG) {
    const int j = threadIdx.x;
    float so = 0.f, sq = 0.f;
#pragma unroll
    for (int k = 0; k < NW; ++k) {
      so += red[2 * j][k];
      sq += red[2 * j + 1][k];
    }
    v.k2part[2 * (size_t)(t.idx + j) + 0] = so;
    v.k2part[2 * (size_t)(t.idx + j) + 1] = sq;
  }
}


template <bool MALTER>
__global__ __launch_bounds__(K2T_THREADS) void scale_convert_tall_kernel(EwArgs a) {
  __shared__ uint32_t tsh[K2_GROUP][K2_T * (K2_T / 2)];
  __shared__ float red[2 * K2_GROUP][K2T_THREADS / 64];
  const Tile t = a.tiles[xcd_remap(blockIdx.x, gridDim.x) * K2_GROUP];
  const EwView v = ew_view(a, t.mat);
  const bool inside = v.vec & ((t.ti + 1) * K2_T <= v.m) & ((t.tj + K2_GROUP) * K2_T <= v.n);
  if (inside) scale_convert_tall_group<MALTER, true>(v, t, tsh, red);
  else scale_convert_tall_group<MALTER, false>(v, t, tsh, red);
}

// Fixed-order block reduction of count pairs (stride 2) into float64 sums.
__device__ void block_sum_pairs(const float* __restrict__ p, int count, double out[2]) {
  __shared__ double sh[2][4];
  double s0 = 0.0, s1 = 0.0;
  for (int k = threadIdx.x; k < count; k += NTHREADS) {
    s0 += (double)p[2 * (size_t)k];
    s1 += (double)p[2 * (size_t)k + 1];
  }
  s0 = wave_sum_d(s0);
  s1 = wave_sum_d(s1);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane == 0) {
    sh[0][w] = s0;
    sh[1][w] = s1;
  }
  __syncthreads();
  out[0] = (sh[0][0] + sh[0][1]) + (sh[0][2] + sh[0][3]);
  out[1] = (sh[1][0] + sh[1][1]) + (sh[1][2] + sh[1][3]);
}

// ||Mt||_F, sigma = 1/(s+ns_eps), nu_t and alpha_t (Alg. 2; displayed alpha_t).
__global__ __launch_bounds__(NTHREADS) void norm_scalars_kernel(EwArgs a) {
  const MatDesc& d = a.desc[blockIdx.x];
  double sums[2];
  block_sum_pairs(d.k2part, d.k2_tiles, sums);
  if (threadIdx.x != 0) return;
  const double s = sqrt(sums[0]);
  double* sc = d.scal;
  sc[SC_S] = s;
  sc[SC_SIGMA] = 1.0 / (s + a.ns_eps);
  if (a.malter) {
    const double nu = a.mu2 * (double)d.nu[0] + (1.0 - a.mu2) * sums[1];
    d.nu[0] = (float)nu;
    sc[SC_NU] = nu;
    sc[SC_Q] = sums[1];
    sc[SC_ALPHA] = a.bc * s / (sqrt(nu) + a.eps);
  } else {
    sc[SC_NU] = 0.0;
    sc[SC_Q] = 0.0;
    sc[SC_ALPHA] = 1.0;
  }
}

// Condition numbers of diag(l) and diag(r) (the quantity the paper's analysis
// of the diagonal preconditioners plots per layer): the largest entry over the
// smallest, +inf when the smallest is 0, NaN when an entry is NaN.  One
// workgroup per matrix; max and min are exact, so the result does not depend
// on the reduction order.
__device__ __forceinline__ void block_max_min(const MALT_GLOBAL float* __restrict__ x, int len, float* mx_out,
                                              float* mn_out, int* nan_out) {
  __shared__ float sh[2][NTHREADS / 64];
  __shared__ int shn[NTHREADS / 64];
  float mx = 0.f, mn = INFINITY;
  int nan = 0;
  for (int i = threadIdx.x; i < len; i += NTHREADS) {
    const float y = x[i];
    nan |= y != y;
    mx = fmaxf(mx, y);
    mn = fminf(mn, y);
  }
  for (int o = 32; o > 0; o >>= 1) {
    mx = fmaxf(mx, __shfl_xor(mx, o));
    mn = fminf(mn, __shfl_xor(mn, o));
    nan |= __shfl_xor(nan, o);
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane == 0) {
    sh[0][w] = mx;
    sh[1][w] = mn;
    shn[w] = nan;
  }
  __syncthreads();
  mx = sh[0][0];
  mn = sh[1][0];
  nan = shn[0];
#pragma unroll
  for (int k = 1; k < NTHREADS / 64; ++k) {
    mx = fmaxf(mx, sh[0][k]);
    mn = fminf(mn, sh[1][k]);
    nan |= shn[k];
  }
  __syncthreads();   // sh is reused by the next call
  *mx_out = mx;
  *mn_out = mn;
  *nan_out = nan;
}

__global__ __launch_bounds__(NTHREADS) void precond_cond_kernel(const MatDesc* desc, double* out) {
  const MatDesc& d = desc[blockIdx.x];
  float mx[2], mn[2];
  int nan[2];
  block_max_min(gptr(d.l), d.m, &mx[0], &mn[0], &nan[0]);
  block_max_min(gptr(d.r), d.n, &mx[1], &mn[1], &nan[1]);
  if (threadIdx.x < 2) {
    const int v = threadIdx.x;
    double k = mn[v] > 0.f ? (double)mx[v] / (double)mn[v] : INFINITY;
    if (nan[v]) k = NAN;
    gptr(out)[2 * (size_t)blockIdx.x + v] = k;
  }
}

// ||O||, ||D|| = ||L O R|| from the update-tile partials; graft and coefficient.
__global__ __launch_bounds__(NTHREADS) void graft_scalars_kernel(EwArgs a) {
  const MatDesc& d = a.desc[blockIdx.x];
  double sums[2];
  block_sum_pairs(d.gpart, d.upd_tiles, sums);
  if (threadIdx.x != 0) return;
  double* sc = d.scal;
  const double g = sqrt(sums[0]) / (sqrt(sums[1]) + a.eps);
  sc[SC_O2] = sums[0];
  sc[SC_D2] = sums[1];
  sc[SC_GRAFT] = g;
  sc[SC_COEF] = a.lr * sc[SC_ALPHA] * g;
}

// ---------------------------------------------------------------------------
// W <- decay * W - coef * L_i O_ij R_j  (Alg. 1/2, last line; D = L O R).
// O is the bf16 canonical Newton-Schulz output: W-oriented for wide matrices,
// W^T for tall ones (read through an LDS transpose).  Reads W and O, writes
// W: 10 bytes per element.
// ---------------------------------------------------------------------------
// Tall matrices: the tile's O^T block (EW_TC canonical rows = W columns, EW_TR
// canonical columns = W rows) is staged in LDS as 32-bit words, word w holding
// W rows 2w and 2w + 1 of one W column.  bm_word() places word (c, w), with
// c = 4 l + e, in a 64-word segment per (w, e) that holds the 64 values of l
// rotated by 8 e + 2 (w / 4).  Both the fill (each thread: 16 bytes of one
// canonical row, four words) and the read (a wave's two W rows are one word;
// lane l reads W columns 4 l .. 4 l + 3) then hit 32 distinct banks in each
// half-wave.
__device__ __forceinline__ int bm_word(int c, int w) {
  const int l = c >> 2, e = c & 3;
  return w * EW_TC + e * 64 + ((l + 8 * e + 2 * (w >> 2)) & 63);
}

// Instances per orientation (TALL) and per interior tile (INSIDE: all EW_TR
// rows and EW_TC columns inside W, 16-byte rows; no bounds tests, as in the
// momentum pass). Every global load is issued before the tall path's LDS
// staging and its barrier, so W's loads are in flight while O's block makes
// its round trip.
template <bool TALL, bool INSIDE>
__device__ __forceinline__ void backmap_tile(const EwArgs& a, const EwView& v, const Tile& t, uint32_t* osh) {
  constexpr int NW = EW_THREADS / 64, RPW = EW_TR / NW;   // 16 waves, 2 rows each
  static_assert(NW * RPW == EW_TR && EW_TC * EW_TR == EW_THREADS * 8, "tall fill: 8 bf16 per thread");
  static_assert(RPW == 2 && EW_TC == 256, "tall read: one word holds a wave's two rows; 64 lanes x 4 columns");
  const int m = v.m, n = v.n;
  const bool vec = v.vec;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r0 = t.ti * EW_TR, c0 = t.tj * EW_TC, c = c0 + lane * 4;
  const MALT_GLOBAL bf16_t* __restrict__ O = v.O;
  const int ldo = v.np;
  MALT_GLOBAL float* __restrict__ W = v.W;
  const MALT_GLOBAL float* __restrict__ Lv = v.Lv;
  const int rw = r0 + w * RPW;   // this wave's first row
  float wv[RPW][4];
  uint2 pk[RPW];
#pragma unroll
  for (int u = 0; u < RPW; ++u) {
    if (INSIDE || rw + u < m) {
      load4<false, INSIDE>(W + (size_t)(rw + u) * n, c, n, vec, wv[u]);
      if (!TALL) {
        const ew_u32x2 q = __builtin_nontemporal_load(reinterpret_cast<const MALT_GLOBAL ew_u32x2*>(O + (size_t)(rw + u) * ldo + c));
        pk[u] = make_uint2(q.x, q.y);
      }
    }
  }
  ew_u32x4 ob;
  const int cr = threadIdx.x >> 2, q = threadIdx.x & 3;
  if (TALL) {
    // Canonical rows c0 .. c0+255 (W columns), columns r0 .. r0+31 (W rows):
    // four threads per canonical row, 16 bytes (four words) each, inside the
    // padded buffer.
    ob = __builtin_nontemporal_load(reinterpret_cast<const MALT_GLOBAL ew_u32x4*>(O + (size_t)(c0 + cr) * ldo + r0 + q * 8));
  }
  float Rv[4];
  load4<false, INSIDE>(v.Rv, c, n, true, Rv);
  const float coef = (float)v.scal[SC_COEF];
  const float decay = a.decay;
  float lv[RPW];   // all read before the first store, which the compiler cannot tell apart from Lv
#pragma unroll
  for (int u = 0; u < RPW; ++u) lv[u] = (INSIDE || rw + u < m) ? Lv[rw + u] : 0.f;
  uint32_t ow[4];   // tall: W rows rw, rw + 1 at W column c + e
  if (TALL) {
    osh[bm_word(cr, 4 * q + 0)] = ob.x;
    osh[bm_word(cr, 4 * q + 1)] = ob.y;
    osh[bm_word(cr, 4 * q + 2)] = ob.z;
    osh[bm_word(cr, 4 * q + 3)] = ob.w;
    __syncthreads();
#pragma unroll
    for (int e = 0; e < 4; ++e) ow[e] = osh[bm_word(4 * lane + e, w)];
  }
#pragma unroll
  for (int u = 0; u < RPW; ++u) {
    const int r = rw + u;
    if (!INSIDE && r >= m) break;   // uniform over the wave
    const float cl = coef * lv[u];
    float o[4];
    if (!TALL) {
      o[0] = bf16_lo(pk[u].x);
      o[1] = bf16_hi(pk[u].x);
      o[2] = bf16_lo(pk[u].y);
      o[3] = bf16_hi(pk[u].y);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = u == 0 ? bf16_lo(ow[e]) : bf16_hi(ow[e]);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) wv[u][e] = decay * wv[u][e] - cl * o[e] * Rv[e];
    store4<INSIDE>(W + (size_t)r * n, c, n, vec, wv[u]);
  }
}

__global__ __launch_bounds__(EW_THREADS) void backmap_write_kernel(EwArgs a) {
  __shared__ uint32_t osh[EW_TR / 2 * EW_TC];   // tall: O^T block as words (see bm_word)
  const Tile t = a.tiles[xcd_remap(blockIdx.x, gridDim.x)];
  const EwView v = ew_view(a, t.mat);
  const bool inside = v.vec & ((t.ti + 1) * EW_TR <= v.m) & ((t.tj + 1) * EW_TC <= v.n);
  if (v.tall) {
    if (inside) backmap_tile<true, true>(a, v, t, osh);
    else backmap_tile<true, false>(a, v, t, osh);
  } else {
    if (inside) backmap_tile<false, true>(a, v, t, osh);
    else backmap_tile<false, false>(a, v, t, osh);
  }
}

// ---------------------------------------------------------------------------
// Plan plumbing: the pointer table of a step, and zeroing of device buffers
// (a kernel rather than a memset node, so either can sit in a captured graph).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(PTR_CHUNK) void ptr_upload_kernel(PtrUploadArgs a) {
  const int i = threadIdx.x;
  if (i < a.count) {
    // Field by field: PtrPair is 24 bytes, written as three 8-byte words.
    const uint64_t* src = reinterpret_cast<const uint64_t*>(&a.p[i]);
    MALT_GLOBAL uint64_t* dst = reinterpret_cast<MALT_GLOBAL uint64_t*>(gptr(a.dst + i));
    static_assert(sizeof(PtrPair) == 24, "pointer table entry layout");
    dst[0] = src[0];
    dst[1] = src[1];
    dst[2] = src[2];
  }
}

__global__ __launch_bounds__(NTHREADS) void zero_fill_kernel(ew_u32x4* dst, size_t n16, uint8_t* tail, int ntail) {
  const ew_u32x4 z = {0u, 0u, 0u, 0u};
  for (size_t i = (size_t)blockIdx.x * NTHREADS + threadIdx.x; i < n16; i += (size_t)gridDim.x * NTHREADS)
    gptr(dst)[i] = z;
  if (blockIdx.x == 0 && (int)threadIdx.x < ntail) gptr(tail)[threadIdx.x] = 0;
}

hipError_t launch_ptr_upload(const PtrUploadArgs& a, hipStream_t s) {
  if (a.count <= 0 || a.count > PTR_CHUNK) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ptr_upload_kernel, dim3(1), dim3(PTR_CHUNK), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_zero_fill(void* dst, size_t bytes, hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  if (reinterpret_cast<uintptr_t>(dst) % 16 != 0) return hipErrorInvalidValue;
  const size_t n16 = bytes / 16;
  const int ntail = int(bytes % 16);
  const size_t want = (n16 + NTHREADS - 1) / NTHREADS;
  const unsigned grid = unsigned(want < 4096 ? (want > 0 ? want : 1) : 4096);
  hipLaunchKernelGGL(zero_fill_kernel, dim3(grid), dim3(NTHREADS), 0, s, reinterpret_cast<ew_u32x4*>(dst), n16,
                     static_cast<uint8_t*>(dst) + n16 * 16, ntail);
  return hipGetLastError();
}

hipError_t launch_momentum_rowcol(const EwArgs& a, hipStream_t s) {
  if (a.ntiles == 0) return hipSuccess;
  hipLaunchKernelGGL(momentum_rowcol_kernel, dim3(a.ntiles), dim3(EW_THREADS), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_precond_finalize(const EwArgs& a, hipStream_t s) {
  if (a.ntiles == 0) return hipSuccess;
  hipLaunchKernelGGL(precond_finalize_kernel, dim3(a.ntiles), dim3(NTHREADS), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_scale_convert(const EwArgs& a, bool tall, hipStream_t s) {
  if (a.ntiles == 0) return hipSuccess;
  if (!tall) {
    if (a.malter) hipLaunchKernelGGL(scale_convert_wide_kernel<true>, dim3(a.ntiles), dim3(K2W_THREADS), 0, s, a);
    else hipLaunchKernelGGL(scale_convert_wide_kernel<false>, dim3(a.ntiles), dim3(K2W_THREADS), 0, s, a);
    return hipGetLastError();
  }
  if (a.ntiles % K2_GROUP != 0) return hipErrorInvalidValue;   // bands hold whole groups
  const dim3 grid(a.ntiles / K2_GROUP);
  if (a.malter) hipLaunchKernelGGL(scale_convert_tall_kernel<true>, grid, dim3(K2T_THREADS), 0, s, a);
  else hipLaunchKernelGGL(scale_convert_tall_kernel<false>, grid, dim3(K2T_THREADS), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_norm_scalars(const EwArgs& a, int32_t nmat, hipStream_t s) {
  if (nmat == 0) return hipSuccess;
  hipLaunchKernelGGL(norm_scalars_kernel, dim3(nmat), dim3(NTHREADS), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_graft_scalars(const EwArgs& a, int32_t nmat, hipStream_t s) {
  if (nmat == 0) return hipSuccess;
  hipLaunchKernelGGL(graft_scalars_kernel, dim3(nmat), dim3(NTHREADS), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_precond_cond(const MatDesc* desc, int32_t nmat, double* out, hipStream_t s) {
  if (nmat == 0) return hipSuccess;
  hipLaunchKernelGGL(precond_cond_kernel, dim3(nmat), dim3(NTHREADS), 0, s, desc, out);
  return hipGetLastError();
}
hipError_t launch_backmap_write(const EwArgs& a, hipStream_t s) {
  if (a.ntiles == 0) return hipSuccess;
  hipLaunchKernelGGL(backmap_write_kernel, dim3(a.ntiles), dim3(EW_THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace malt
