// Grouped Newton-Schulz GEMMs on the gfx950 matrix cores (bf16 in, fp32 acc).
//
// Every phase is one launch over all matrices of the step; every workgroup
// computes one 256 x 256 output tile C = P Q^T with P, Q row-major bf16 and
// the contraction index contiguous in both (an "NT" product):
//   Gram:       A = s X X^T            (P = Q = X, symmetric: upper tiles only,
//                                        mirrored on write; s = sigma^2 on the
//                                        first iteration, else 1)
//   Polynomial: B = b A + c A A^T      (A symmetric, so A A = A A^T; upper tiles)
//   Update:     X' = s (a X + B X)     (Q = X^T, the stored transpose; s = sigma
//                                        on the first iteration)
// X is kept in both orientations so that every product reads its operands
// along contiguous rows; the update writes both orientations of X', and on
// the last iteration only the one in W's orientation plus the per-tile sums
// of O^2 and (L O R)^2 used by norm grafting.
//
// Rounding: A, B and X are stored as bf16 (round to nearest even) and the
// same rounded A feeds both terms of B, the same rounded X both terms of X'.
//
// Workgroup: 256 threads = 4 waves in a 2 x 2 arrangement, each wave owning a
// 128 x 128 sub-tile as 4 x 4 blocks of v_mfma_f32_32x32x16_bf16.  K advances
// in steps of 64 through two LDS stages (rows padded to 72 bf16 so that the
// 16-byte fragment reads of 16 consecutive rows hit distinct banks); global
// loads for step k+1 are in flight while step k is multiplied.
#include "malt_internal.h"

namespace malt {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int LDS_STRIDE = NS_BK + 8;                 // bf16 per LDS row
constexpr int STAGE_ELEMS = NS_TILE * LDS_STRIDE;    // one operand, one stage
constexpr int LDS_BYTES = 2 * 2 * STAGE_ELEMS * 2;   // 2 stages x (P, Q) x bf16
constexpr int EPI_F = NS_TILE + 4;                   // fp32 epilogue stage row (floats)
constexpr int EPI_B = NS_TILE + 8;                   // bf16 epilogue stage row
static_assert(64 * EPI_F * 4 + 2 * 64 * EPI_B * 2 <= LDS_BYTES, "epilogue stage exceeds LDS");

__device__ __forceinline__ bf16_t f2bf_rne(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}
__device__ __forceinline__ float bf2f_(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

__device__ __forceinline__ float wsum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__global__ __launch_bounds__(NTHREADS, 1) void ns_gemm_kernel(NsArgs args) {
  extern __shared__ __attribute__((aligned(16))) bf16_t lds[];
  const Tile t = args.tiles[xcd_remap(blockIdx.x, gridDim.x)];
  const MatDesc& d = args.desc[t.mat];
  const int phase = args.phase;
  const int mp = d.mp, np = d.np;

  const bf16_t* P;
  const bf16_t* Q;
  int ldp, ldq, K;
  if (phase == PH_GRAM) {
    P = d.X[args.src]; Q = P; ldp = ldq = np; K = np;
  } else if (phase == PH_POLY) {
    P = d.A; Q = P; ldp = ldq = mp; K = mp;
  } else {
    // Split matrices contract over [B_hi | B_lo] and [X^T | X^T]: K = 2 mp.
    P = d.B; Q = d.XT[args.src]; ldq = mp;
    ldp = d.split ? 2 * mp : mp;
    K = d.split ? 2 * mp : mp;
  }
  const int kwrap = (phase == PH_UPDATE) ? mp : K;   // Q's k index wraps at mp
  const int row0 = t.ti * NS_TILE, col0 = t.tj * NS_TILE;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;

  // Global -> LDS mapping: 8 threads per 64-wide row (16 B each), 32 rows per pass.
  const int lrow = tid >> 3, lchunk = (tid & 7) * 8;
  const bf16_t* gp = P + (size_t)(row0 + lrow) * ldp + lchunk;
  const bf16_t* gq = Q + (size_t)(col0 + lrow) * ldq + lchunk;
  u32x4 rp[8], rq[8];

  // Stage b holds P at lds + 2b*STAGE_ELEMS and Q right after it.

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int frow = lane & 31, fk = (lane >> 5) * 8;
  const int KT = K / NS_BK;
#define NS_GLOAD(k0)                                                                  \
  _Pragma("unroll") for (int p = 0; p < 8; ++p) {                                      \
    rp[p] = *reinterpret_cast<const u32x4*>(gp + (size_t)(32 * p) * ldp + (k0));       \
    rq[p] = *reinterpret_cast<const u32x4*>(gq + (size_t)(32 * p) * ldq +              \
                                            ((k0) >= kwrap ? (k0) - kwrap : (k0)));     \
  }
#define NS_LSTORE(buf)                                                                 \
  _Pragma("unroll") for (int p = 0; p < 8; ++p) {                                      \
    bf16_t* sp = lds + (buf) * 2 * STAGE_ELEMS + (lrow + 32 * p) * LDS_STRIDE + lchunk; \
    *reinterpret_cast<u32x4*>(sp) = rp[p];                                             \
    *reinterpret_cast<u32x4*>(sp + STAGE_ELEMS) = rq[p];                               \
  }
  NS_GLOAD(0);
  NS_LSTORE(0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < KT) { NS_GLOAD((kt + 1) * NS_BK); }
    const bf16_t* bp = lds + cur * 2 * STAGE_ELEMS + (wr * 128 + frow) * LDS_STRIDE + fk;
    const bf16_t* bq = lds + cur * 2 * STAGE_ELEMS + STAGE_ELEMS + (wc * 128 + frow) * LDS_STRIDE + fk;
#pragma unroll
    for (int s = 0; s < NS_BK / 16; ++s) {
      bf16x8 fa[4], fb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        fa[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(bp + i * 32 * LDS_STRIDE + s * 16));
#pragma unroll
      for (int j = 0; j < 4; ++j)
        fb[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(bq + j * 32 * LDS_STRIDE + s * 16));
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < KT) { NS_LSTORE(cur ^ 1); }
    __syncthreads();
  }

#undef NS_GLOAD
#undef NS_LSTORE
  // ---------------------------------------------------------------- epilogue
  // Four rounds; round i stages rows {wr*128 + i*32 + [0,32)} of both wave rows
  // (64 tile rows x 256 cols, fp32) in LDS.  Pass 1 reads 8 consecutive
  // columns per thread, applies the phase's epilogue, writes bf16 rows and
  // keeps the bf16 values in LDS; pass 2 writes the transposed orientation
  // from there.  Local staged row lr maps to tile row (lr >> 5)*128 + i*32 + (lr & 31).
  float* stf = reinterpret_cast<float*>(lds);                                  // [64][EPI_F]
  bf16_t* stb = reinterpret_cast<bf16_t*>(lds) + 2 * 64 * EPI_F;               // [64][EPI_B]
  bf16_t* stl = stb + 64 * EPI_B;                                              // [64][EPI_B] (split lo)
  const bool sym = phase != PH_UPDATE;
  const bool mirror = sym && (t.ti != t.tj);
  const int dst = args.src ^ 1;
  const bool last = args.last != 0;
  const bool wo_is_x = !d.tall;            // W orientation = canonical for wide matrices
  float sc = 1.f;
  if (args.first) {
    const float sig = (float)d.scal[SC_SIGMA];
    sc = (phase == PH_GRAM) ? sig * sig : (phase == PH_UPDATE ? sig : 1.f);
  }
  bf16_t* out_row;       // row-major destination (pitch ldo) or nullptr
  bf16_t* out_tr;        // transposed destination (pitch ldt) or nullptr
  int ldo, ldt;
  // Split B: the low part bf16(v - hi) goes lo_off columns to the right.
  const int lo_off = (phase == PH_POLY && d.split) ? mp : 0;
  if (phase == PH_GRAM || phase == PH_POLY) {
    out_row = (phase == PH_GRAM) ? d.A : d.B;
    out_tr = mirror ? out_row : nullptr;
    ldo = ldt = lo_off ? 2 * mp : mp;
  } else {
    out_row = (!last || wo_is_x) ? d.X[dst] : nullptr;
    out_tr = (!last || !wo_is_x) ? d.XT[dst] : nullptr;
    ldo = np;
    ldt = mp;
  }
  const bf16_t* addend = (phase == PH_POLY) ? d.A : (phase == PH_UPDATE ? d.X[args.src] : nullptr);
  const int lda = (phase == PH_POLY) ? mp : np;
  const float k_add = (phase == PH_POLY) ? args.b : args.a;
  const float k_acc = (phase == PH_POLY) ? args.c : 1.f;
  float o2 = 0.f, d2 = 0.f;

  // Pass-1 mapping: 32 threads per staged row (8 columns each), 8 row groups.
  const int p1c = (tid & 31) * 8, p1r = tid >> 5;
  // Pass-2 mapping: 4 threads per output column (8 rows each), 64 columns per pass.
  const int p2c = tid >> 2, p2s = (tid & 3) * 8;

#pragma unroll
  for (int i = 0; i < 4; ++i) {
    __syncthreads();   // previous round's readers are done with the stage
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int lr = wr * 32 + g * 8 + (lane >> 5) * 4 + e;
          const int lc = wc * 128 + j * 32 + (lane & 31);
          stf[lr * EPI_F + lc] = acc[i][j][4 * g + e];
        }
    __syncthreads();
    // Pass 1: straight orientation.
    for (int k = 0; k < 8; ++k) {
      const int lr = p1r + 8 * k;
      const int R = row0 + (lr >> 5) * 128 + i * 32 + (lr & 31);
      const int C = col0 + p1c;
      const float4 a0 = *reinterpret_cast<const float4*>(stf + lr * EPI_F + p1c);
      const float4 a1 = *reinterpret_cast<const float4*>(stf + lr * EPI_F + p1c + 4);
      float v[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
      if (addend) {
        const uint4 q = *reinterpret_cast<const uint4*>(addend + (size_t)R * lda + C);
        const uint32_t qw[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float av = bf2f_((bf16_t)((qw[e >> 1] >> (16 * (e & 1))) & 0xffffu));
          v[e] = k_add * av + k_acc * v[e];
        }
      }
      uint32_t hw[4], lw[4];
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const float v0 = sc * v[e], v1 = sc * v[e + 1];
        const bf16_t h0 = f2bf_rne(v0), h1 = f2bf_rne(v1);
        hw[e >> 1] = (uint32_t)h0 | ((uint32_t)h1 << 16);
        stb[lr * EPI_B + p1c + e] = h0;
        stb[lr * EPI_B + p1c + e + 1] = h1;
        if (lo_off) {
          const bf16_t l0 = f2bf_rne(v0 - bf2f_(h0)), l1 = f2bf_rne(v1 - bf2f_(h1));
          lw[e >> 1] = (uint32_t)l0 | ((uint32_t)l1 << 16);
          stl[lr * EPI_B + p1c + e] = l0;
          stl[lr * EPI_B + p1c + e + 1] = l1;
        }
        if (last && phase == PH_UPDATE) {
          // Canonical (R, C) is W(R, C) for wide, W(C, R) for tall matrices.
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const int cc = C + e + u;
            if (R < d.mc && cc < d.nc) {
              const float o = bf2f_(u ? h1 : h0);
              const float dv = (d.tall ? d.Rv[R] * d.Lv[cc] : d.Lv[R] * d.Rv[cc]) * o;
              o2 += o * o;
              d2 += dv * dv;
            }
          }
        }
      }
      if (out_row) {
        *reinterpret_cast<uint4*>(out_row + (size_t)R * ldo + C) = make_uint4(hw[0], hw[1], hw[2], hw[3]);
        if (lo_off)
          *reinterpret_cast<uint4*>(out_row + (size_t)R * ldo + lo_off + C) = make_uint4(lw[0], lw[1], lw[2], lw[3]);
      }
    }
    if (out_tr) {
      __syncthreads();
      // Pass 2: transposed orientation, out_tr[C][R .. R+7] for both row bands.
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int lc = p2c + 64 * q;
        const int C = col0 + lc;
#pragma unroll
        for (int band = 0; band < 2; ++band) {
          const int lr0 = band * 32 + p2s;
          const int R = row0 + band * 128 + i * 32 + p2s;
          uint32_t hw[4];
#pragma unroll
          for (int e = 0; e < 8; e += 2)
            hw[e >> 1] = (uint32_t)stb[(lr0 + e) * EPI_B + lc] | ((uint32_t)stb[(lr0 + e + 1) * EPI_B + lc] << 16);
          *reinterpret_cast<uint4*>(out_tr + (size_t)C * ldt + R) = make_uint4(hw[0], hw[1], hw[2], hw[3]);
          if (lo_off) {
#pragma unroll
            for (int e = 0; e < 8; e += 2)
              hw[e >> 1] = (uint32_t)stl[(lr0 + e) * EPI_B + lc] | ((uint32_t)stl[(lr0 + e + 1) * EPI_B + lc] << 16);
            *reinterpret_cast<uint4*>(out_tr + (size_t)C * ldt + lo_off + R) = make_uint4(hw[0], hw[1], hw[2], hw[3]);
          }
        }
      }
    }
  }
  if (phase == PH_UPDATE && last) {
    // Deterministic per-tile sums for the graft norms.
    __syncthreads();
    float* red = stf;
    o2 = wsum(o2);
    d2 = wsum(d2);
    if (lane == 0) {
      red[wave] = o2;
      red[4 + wave] = d2;
    }
    __syncthreads();
    if (tid == 0) {
      d.gpart[2 * (size_t)t.idx + 0] = (red[0] + red[1]) + (red[2] + red[3]);
      d.gpart[2 * (size_t)t.idx + 1] = (red[4] + red[5]) + (red[6] + red[7]);
    }
  }
}

hipError_t launch_ns_gemm(const NsArgs& a, hipStream_t s) {
  if (a.ntiles == 0) return hipSuccess;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&ns_gemm_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, LDS_BYTES);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL(ns_gemm_kernel, dim3(a.ntiles), dim3(NTHREADS), LDS_BYTES, s, a);
  return hipGetLastError();
}

}  // namespace malt
