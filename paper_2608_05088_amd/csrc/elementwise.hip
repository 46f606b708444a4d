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

// Load 4 consecutive floats of one row starting at column c (columns >= n read 0).
__device__ __forceinline__ void load4(const float* __restrict__ p, int c, int n, bool vec, float v[4]) {
  if (vec && c + 3 < n) {
    const float4 x = *reinterpret_cast<const float4*>(p + c);
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = (c + e < n) ? p[c + e] : 0.f;
  }
}

__device__ __forceinline__ void store4(float* __restrict__ p, int c, int n, bool vec, const float v[4]) {
  if (vec && c + 3 < n) {
    *reinterpret_cast<float4*>(p + c) = make_float4(v[0], v[1], v[2], v[3]);
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (c + e < n) p[c + e] = v[e];
  }
}

// ---------------------------------------------------------------------------
// Momentum EMA (Alg. 1/2, momentum line) fused with the per-tile row and
// column sums of G^2 that feed the l, r EMAs (Eq. dp_preconditioner).
// Reads G and M, writes M: 12 bytes per element.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NTHREADS) void momentum_rowcol_kernel(EwArgs a) {
  __shared__ float colsh[4][EW_TC];
  const Tile t = a.tiles[xcd_remap(blockIdx.x, gridDim.x)];
  const MatDesc& d = a.desc[t.mat];
  const int m = d.m, n = d.n;
  const bool vec = a.ptrs[t.mat].vec != 0;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r0 = t.ti * EW_TR, c = t.tj * EW_TC + lane * 4;
  const float* __restrict__ G = a.ptrs[t.mat].G;
  float* __restrict__ M = d.M;
  float cacc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int rr = w; rr < EW_TR; rr += 4) {
    const int r = r0 + rr;
    if (r >= m) break;
    const size_t off = (size_t)r * n;
    float g[4], mm[4];
    load4(G + off, c, n, vec, g);
    load4(M + off, c, n, vec, mm);
    float racc = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      mm[e] = a.mu1 * mm[e] + a.one_minus_mu1 * g[e];
      const float g2 = g[e] * g[e];
      racc += g2;
      cacc[e] += g2;
    }
    store4(M + off, c, n, vec, mm);
    racc = wave_sum(racc);
    if (lane == 0) d.rowpart[(size_t)t.tj * m + r] = racc;
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) colsh[w][lane * 4 + e] = cacc[e];
  __syncthreads();
  const int cc = threadIdx.x;
  const int col = t.tj * EW_TC + cc;
  if (col < n) {
    const float s = (colsh[0][cc] + colsh[1][cc]) + (colsh[2][cc] + colsh[3][cc]);
    d.colpart[(size_t)t.ti * n + col] = s;
  }
}

// ---------------------------------------------------------------------------
// Row / column EMAs and the diagonal preconditioners.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NTHREADS) void precond_finalize_kernel(EwArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  const MatDesc& d = a.desc[t.mat];
  const int i = t.tj * NTHREADS + threadIdx.x;
  if (t.ti == 0) {
    if (i >= d.m) return;
    double s = 0.0;
    for (int c = 0; c < d.k1_ct; ++c) s += (double)d.rowpart[(size_t)c * d.m + i];
    const double lv = a.mu2 * (double)d.l[i] + (1.0 - a.mu2) * s;
    d.l[i] = (float)lv;
    d.Lv[i] = a.identity ? 1.f : (float)pow(lv + a.eps, -0.125);
  } else {
    if (i >= d.n) return;
    double s = 0.0;
    for (int c = 0; c < d.k1_rt; ++c) s += (double)d.colpart[(size_t)c * d.n + i];
    const double rv = a.mu2 * (double)d.r[i] + (1.0 - a.mu2) * s;
    d.r[i] = (float)rv;
    d.Rv[i] = a.identity ? 1.f : (float)pow(rv + a.eps, -0.125);
  }
}

// ---------------------------------------------------------------------------
// X0 = bf16(L M R) in the canonical orientation (W for wide matrices, W^T
// through an LDS transpose for tall ones) over the zero-padded domain, plus
// per-tile sums of (LMR)^2 and, for MALTER, (LGR)^2.  Tiles cover W-oriented
// padded rows x cols in K2_T x K2_T blocks, K2_GROUP tiles per workgroup.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NTHREADS) void scale_convert_kernel(EwArgs a) {
  // One workgroup converts K2_GROUP consecutive tiles: a 64-row band of
  // K2_GROUP * 64 W columns of one matrix (a matrix's tiles are listed band by
  // band, and every band holds a multiple of K2_GROUP tiles).  All loads of the
  // band are issued before any conversion.
  constexpr int TG = K2_GROUP;
  __shared__ bf16_t tsh[TG][K2_T][K2_T + 2];
  __shared__ float red[2 * TG][4];
  const int grp = xcd_remap(blockIdx.x, gridDim.x);
  const Tile t = a.tiles[grp * TG];
  const MatDesc& d = a.desc[t.mat];
  const int m = d.m, n = d.n;
  const bool vec = a.ptrs[t.mat].vec != 0;
  bf16_t* __restrict__ X0 = d.X[0];
  const int ldx = d.np;                  // canonical row pitch
  const float* __restrict__ M = d.M;
  const float* __restrict__ G = a.ptrs[t.mat].G;
  const bool malter = a.malter != 0;
  const int r0 = t.ti * K2_T, cb = t.tj * K2_T;   // band columns cb .. cb + TG*K2_T
  const int cc = (threadIdx.x & 15) * 4;          // 4 columns of each tile
  const int rq = threadIdx.x >> 4;                // rows rq + 16p, p = 0..3

  float Li[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int r = r0 + p * 16 + rq;
    Li[p] = r < m ? d.Lv[r] : 0.f;
  }
  float Rv[TG][4];
#pragma unroll
  for (int j = 0; j < TG; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int c = cb + j * K2_T + cc + e;
      Rv[j][e] = c < n ? d.Rv[c] : 0.f;
    }
  float mm[TG][4][4], gg[TG][4][4];
#pragma unroll
  for (int j = 0; j < TG; ++j)
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int r = r0 + p * 16 + rq;
      const int c = cb + j * K2_T + cc;
#pragma unroll
      for (int e = 0; e < 4; ++e) mm[j][p][e] = gg[j][p][e] = 0.f;
      if (r < m) {
        load4(M + (size_t)r * n, c, n, vec, mm[j][p]);
        if (malter) load4(G + (size_t)r * n, c, n, vec, gg[j][p]);
      }
    }

  float s2[TG], q2[TG];
#pragma unroll
  for (int j = 0; j < TG; ++j) {
    s2[j] = 0.f;
    q2[j] = 0.f;
    const int c0 = cb + j * K2_T;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int rr = p * 16 + rq;
      float x[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[e] = Li[p] * mm[j][p][e] * Rv[j][e];
        s2[j] += x[e] * x[e];
        const float y = Li[p] * gg[j][p][e] * Rv[j][e];   // zero for MALT (gg = 0)
        q2[j] += y * y;
      }
      uint2 pk;
      pk.x = pack_bf16x2(x[0], x[1]);
      pk.y = pack_bf16x2(x[2], x[3]);
      if (!d.tall) {
        *reinterpret_cast<uint2*>(X0 + (size_t)(r0 + rr) * ldx + c0 + cc) = pk;
      } else {
        tsh[j][rr][cc + 0] = (bf16_t)(pk.x & 0xffffu);
        tsh[j][rr][cc + 1] = (bf16_t)(pk.x >> 16);
        tsh[j][rr][cc + 2] = (bf16_t)(pk.y & 0xffffu);
        tsh[j][rr][cc + 3] = (bf16_t)(pk.y >> 16);
      }
    }
  }
  if (d.tall) {
    __syncthreads();
    // Transposed write: thread -> (W column ct, 16-row segment) of each tile.
    const int ct = threadIdx.x >> 2;
    const int seg = (threadIdx.x & 3) * 16;
#pragma unroll
    for (int j = 0; j < TG; ++j) {
      uint32_t wv[8];
#pragma unroll
      for (int k = 0; k < 8; ++k)
        wv[k] = (uint32_t)tsh[j][seg + 2 * k][ct] | ((uint32_t)tsh[j][seg + 2 * k + 1][ct] << 16);
      uint4* dst = reinterpret_cast<uint4*>(X0 + (size_t)(cb + j * K2_T + ct) * ldx + r0 + seg);
      dst[0] = make_uint4(wv[0], wv[1], wv[2], wv[3]);
      dst[1] = make_uint4(wv[4], wv[5], wv[6], wv[7]);
    }
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int j = 0; j < TG; ++j) {
    const float sj = wave_sum(s2[j]);
    const float qj = wave_sum(q2[j]);
    if (lane == 0) {
      red[2 * j][w] = sj;
      red[2 * j + 1][w] = qj;
    }
  }
  __syncthreads();
  if (threadIdx.x < TG) {
    const int j = threadIdx.x;
    d.k2part[2 * (size_t)(t.idx + j) + 0] = (red[2 * j][0] + red[2 * j][1]) + (red[2 * j][2] + red[2 * j][3]);
    d.k2part[2 * (size_t)(t.idx + j) + 1] =
        (red[2 * j + 1][0] + red[2 * j + 1][1]) + (red[2 * j + 1][2] + red[2 * j + 1][3]);
  }
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
__global__ __launch_bounds__(NTHREADS) void backmap_write_kernel(EwArgs a) {
  __shared__ bf16_t osh[EW_TC][EW_TR + 2];   // tall: O^T block, [W col][W row]
  const Tile t = a.tiles[xcd_remap(blockIdx.x, gridDim.x)];
  const MatDesc& d = a.desc[t.mat];
  const int m = d.m, n = d.n;
  const bool vec = a.ptrs[t.mat].vec != 0;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r0 = t.ti * EW_TR, c0 = t.tj * EW_TC, c = c0 + lane * 4;
  const bf16_t* __restrict__ O = d.X[a.o_parity];
  const int ldo = d.np;
  float* __restrict__ W = a.ptrs[t.mat].W;
  const float coef = (float)d.scal[SC_COEF];
  const float decay = a.decay;
  if (d.tall) {
    // Canonical rows c0 .. c0+255 (W columns), columns r0 .. r0+31 (W rows):
    // one 64-byte row segment per thread (inside the padded buffer).
    const uint4* srow = reinterpret_cast<const uint4*>(O + (size_t)(c0 + threadIdx.x) * ldo + r0);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint4 v = srow[q];
      const uint32_t vw[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        osh[threadIdx.x][q * 8 + 2 * k] = (bf16_t)(vw[k] & 0xffffu);
        osh[threadIdx.x][q * 8 + 2 * k + 1] = (bf16_t)(vw[k] >> 16);
      }
    }
    __syncthreads();
  }
  float Rv[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) Rv[e] = (c + e < n) ? d.Rv[c + e] : 0.f;
  for (int rr = w; rr < EW_TR; rr += 4) {
    const int r = r0 + rr;
    if (r >= m) break;
    const float cl = coef * d.Lv[r];
    float wv[4];
    load4(W + (size_t)r * n, c, n, vec, wv);
    float o[4];
    if (!d.tall) {
      const uint2 pk = *reinterpret_cast<const uint2*>(O + (size_t)r * ldo + c);
      o[0] = bf2f((bf16_t)(pk.x & 0xffffu));
      o[1] = bf2f((bf16_t)(pk.x >> 16));
      o[2] = bf2f((bf16_t)(pk.y & 0xffffu));
      o[3] = bf2f((bf16_t)(pk.y >> 16));
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = bf2f(osh[lane * 4 + e][rr]);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) wv[e] = decay * wv[e] - cl * o[e] * Rv[e];
    store4(W + (size_t)r * n, c, n, vec, wv);
  }
}

hipError_t launch_momentum_rowcol(const EwArgs& a, hipStream_t s) {
  if (a.ntiles == 0) return hipSuccess;
  hipLaunchKernelGGL(momentum_rowcol_kernel, dim3(a.ntiles), dim3(NTHREADS), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_precond_finalize(const EwArgs& a, hipStream_t s) {
  if (a.ntiles == 0) return hipSuccess;
  hipLaunchKernelGGL(precond_finalize_kernel, dim3(a.ntiles), dim3(NTHREADS), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_scale_convert(const EwArgs& a, hipStream_t s) {
  if (a.ntiles == 0) return hipSuccess;
  if (a.ntiles % K2_GROUP != 0) return hipErrorInvalidValue;   // bands hold whole groups
  hipLaunchKernelGGL(scale_convert_kernel, dim3(a.ntiles / K2_GROUP), dim3(NTHREADS), 0, s, a);
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
hipError_t launch_backmap_write(const EwArgs& a, hipStream_t s) {
  if (a.ntiles == 0) return hipSuccess;
  hipLaunchKernelGGL(backmap_write_kernel, dim3(a.ntiles), dim3(NTHREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace malt
