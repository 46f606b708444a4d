// Newton-Schulz in fp32 for matrices whose short side m' is at most
// NS_SMALL_MAX (32).
//
// The bf16 matrix-core path pads such a matrix to a 256 x 256 tile, and with
// few singular values its rounding is not averaged away: the quintic is still
// far from converged on the small ones, and it magnifies the bf16 rounding of
// X there. These matrices instead keep X, A and B' in fp32. The work is
// m'^2 n' per product, which the chip does in microseconds.
//
// One iteration is three grouped launches over the small matrices of a step:
//   Gram      each workgroup takes SM_CH_G columns of X and sums X_c X_c^T
//             with v_mfma_f32_32x32x2f32 (the 32 x 32 output is the whole
//             Gram); per-chunk partials go to the workspace
//   Poly      one workgroup per matrix sums the partials in chunk order and
//             forms B' = a I + b A + c A A in fp32
//   Update    one thread per column: X'_c = B' X_c; the last iteration writes
//             O rounded to bf16 (for the back-map) and per-chunk sums of O^2
//             and (L O R)^2 from the rounded values
// Iteration 0 reads X0 = sigma L M R straight from the fp32 momentum, in the
// canonical orientation (rows <= columns).
#include "malt_internal.h"

namespace malt {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int SM_M = NS_SMALL_MAX;     // 32: one MFMA output tile
constexpr int SM_SUB = 256;            // columns staged in LDS at a time
static_assert(SM_CH_U == NTHREADS, "one update column per thread");
static_assert(SM_CH_G % SM_SUB == 0 && SM_SUB % 8 == 0, "Gram chunk layout");

// Canonical X (rows i < mc, columns c < nc; zero elsewhere) at column c for
// rows 0..SM_M-1, from the momentum (first iteration) or the fp32 iterate.
__device__ __forceinline__ float sm_x(const MatDesc& d, bool first, const float* Xs, int i, int c, float sig) {
  if (i >= d.mc || c >= d.nc) return 0.f;
  if (!first) return gptr(Xs)[(size_t)i * d.np + c];
  // canonical (i, c) is W(i, c) for wide and W(c, i) for tall matrices
  if (!d.tall) return sig * gptr(d.Lv)[i] * gptr(d.M)[(size_t)i * d.n + c] * gptr(d.Rv)[c];
  return sig * gptr(d.Lv)[c] * gptr(d.M)[(size_t)c * d.n + i] * gptr(d.Rv)[i];
}

__global__ __launch_bounds__(NTHREADS) void sm_gram_kernel(NsArgs args) {
  const Tile t = args.tiles[blockIdx.x];   // (mat, chunk, -, -)
  const MatDesc& d = args.desc[t.mat];
  __shared__ float tile[SM_M][SM_SUB + 1];
  __shared__ float red[4][SM_M * SM_M];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool first = args.first != 0;
  const float sig = first ? (float)d.scal[SC_SIGMA] : 1.f;
  const float* Xs = d.Xs[args.src];
  f32x16 acc;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.f;
  for (int sub = 0; sub < SM_CH_G / SM_SUB; ++sub) {
    const int c0 = t.ti * SM_CH_G + sub * SM_SUB;
    if (c0 >= d.np) break;   // uniform over the workgroup
    __syncthreads();
    for (int q = tid; q < SM_M * SM_SUB; q += NTHREADS) {
      const int i = q / SM_SUB, c = q % SM_SUB;
      tile[i][c] = sm_x(d, first, Xs, i, c0 + c, sig);
    }
    __syncthreads();
    // A(m, n) += sum_k X(m, k) X(n, k): lane l supplies X(l % 32, k + l / 32)
    // as both operands. Each wave takes a quarter of the staged columns.
    constexpr int PER = SM_SUB / 4;
    for (int k = wave * PER; k < (wave + 1) * PER; k += 2) {
      const float v = tile[lane & 31][k + (lane >> 5)];
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(v, v, acc, 0, 0, 0);
    }
  }
  // acc[4g + e] = A(8g + 4 (lane >> 5) + e, lane & 31); the four waves' sums
  // are combined in a fixed order.
  __syncthreads();
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int r = 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3), c = lane & 31;
    red[wave][r * SM_M + c] = acc[e];
  }
  __syncthreads();
  float* out = d.Ap + (size_t)t.ti * SM_M * SM_M;
  for (int q = tid; q < SM_M * SM_M; q += NTHREADS) out[q] = (red[0][q] + red[1][q]) + (red[2][q] + red[3][q]);
}

__global__ __launch_bounds__(NTHREADS) void sm_poly_kernel(NsArgs args) {
  const MatDesc& d = args.desc[args.tiles[blockIdx.x].mat];
  __shared__ float A[SM_M][SM_M + 1];
  const int tid = threadIdx.x;
  for (int q = tid; q < SM_M * SM_M; q += NTHREADS) {
    float s = 0.f;
    for (int ch = 0; ch < d.sm_gchunks; ++ch) s += d.Ap[(size_t)ch * SM_M * SM_M + q];
    A[q / SM_M][q % SM_M] = s;
  }
  __syncthreads();
  for (int q = tid; q < SM_M * SM_M; q += NTHREADS) {
    const int i = q / SM_M, j = q % SM_M;
    float s2 = 0.f;
#pragma unroll 8
    for (int k = 0; k < SM_M; ++k) s2 += A[i][k] * A[k][j];
    d.Bs[q] = (i == j ? args.a : 0.f) + args.b * A[i][j] + args.c * s2;
  }
}

__global__ __launch_bounds__(NTHREADS) void sm_update_kernel(NsArgs args) {
  const Tile t = args.tiles[blockIdx.x];   // (mat, chunk, -, partial slot)
  const MatDesc& d = args.desc[t.mat];
  __shared__ float B[SM_M][SM_M];
  __shared__ float red[2][NTHREADS / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int q = tid; q < SM_M * SM_M; q += NTHREADS) B[q / SM_M][q % SM_M] = gptr(d.Bs)[q];
  const bool first = args.first != 0;
  const float sig = first ? (float)d.scal[SC_SIGMA] : 1.f;
  const int c = t.ti * SM_CH_U + tid;      // canonical column (< np)
  float x[SM_M];
#pragma unroll
  for (int i = 0; i < SM_M; ++i) x[i] = sm_x(d, first, d.Xs[args.src], i, c, sig);
  __syncthreads();
  float y[SM_M];
#pragma unroll
  for (int i = 0; i < SM_M; ++i) {
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < SM_M; ++j) s += B[i][j] * x[j];
    y[i] = s;
  }
  const int mc = d.mc;
  if (!args.last) {
    MALT_GLOBAL float* Xn = gptr(d.Xs[args.src ^ 1]);
#pragma unroll
    for (int i = 0; i < SM_M; ++i)
      if (i < mc) Xn[(size_t)i * d.np + c] = y[i];
    return;
  }
  // Last iteration: O in bf16 where the back-map reads it, and the norms of
  // the rounded values (canonical row i carries the row factor of W for wide
  // and the column factor for tall matrices).
  MALT_GLOBAL bf16_t* O = gptr(d.X[args.src ^ 1]);
  const MALT_GLOBAL float* const Lm = gptr(d.tall ? d.Rv : d.Lv);
  const MALT_GLOBAL float* const Ln = gptr(d.tall ? d.Lv : d.Rv);
  const float ln = c < d.nc ? Ln[c] : 0.f;
  float o2 = 0.f, d2 = 0.f;
#pragma unroll
  for (int i = 0; i < SM_M; ++i) {
    if (i >= mc) continue;
    const uint32_t pk = pack_bf16x2(y[i], 0.f);
    O[(size_t)i * d.np + c] = (bf16_t)(pk & 0xffffu);
    const float o = bf16_lo(pk);
    if (c < d.nc) {
      const float q = o * o;
      const float lm = Lm[i];
      o2 += q;
      d2 += lm * lm * ln * ln * q;
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    o2 += __shfl_xor(o2, off, 64);
    d2 += __shfl_xor(d2, off, 64);
  }
  if (lane == 0) {
    red[0][wave] = o2;
    red[1][wave] = d2;
  }
  __syncthreads();
  if (tid == 0) {
    float so = 0.f, sd = 0.f;
#pragma unroll
    for (int w = 0; w < NTHREADS / 64; ++w) {
      so += red[0][w];
      sd += red[1][w];
    }
    gptr(d.gpart)[2 * (size_t)t.idx + 0] = so;
    gptr(d.gpart)[2 * (size_t)t.idx + 1] = sd;
  }
}

hipError_t launch_small_ns(const NsArgs& a, hipStream_t s) {
  if (a.ntiles == 0) return hipSuccess;
  if (a.phase == PH_GRAM)
    hipLaunchKernelGGL(sm_gram_kernel, dim3(a.ntiles), dim3(NTHREADS), 0, s, a);
  else if (a.phase == PH_POLY)
    hipLaunchKernelGGL(sm_poly_kernel, dim3(a.ntiles), dim3(NTHREADS), 0, s, a);
  else
    hipLaunchKernelGGL(sm_update_kernel, dim3(a.ntiles), dim3(NTHREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace malt
