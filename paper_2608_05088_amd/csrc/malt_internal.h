// Internal device-side structures and kernel launchers of libmalt (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace malt {

// Elementwise tiles (momentum / back-map): EW_TR rows x EW_TC cols per
// EW_THREADS-thread workgroup; each lane owns 4 consecutive columns and each
// wave EW_TR / 16 = 2 rows, whose loads it issues before any arithmetic.
// (A streaming pass runs closest to HBM's rate with few loads in flight per
// wave and no loop per wave.)
constexpr int EW_TR = 32;
constexpr int EW_TC = 256;
constexpr int EW_THREADS = 1024;
// Scale+convert of wide matrices (canonical = W): K2W_R rows x EW_TC cols per
// K2W_THREADS-thread workgroup, one float4 per lane and row, four rows per
// wave (measured against 1-8 rows per wave and 256-1024 threads: within 2%,
// this the fastest).
constexpr int K2W_R = 64;
constexpr int K2W_THREADS = 1024;
// Scale+convert of tall matrices (canonical = W^T, through an LDS transpose):
// K2_T x K2_T tiles; a K2T_THREADS-thread workgroup takes K2_GROUP consecutive
// tiles of one row band (padded W dimensions are multiples of 256, so bands
// hold whole groups).
constexpr int K2_T = 64;
constexpr int K2_GROUP = 2;
constexpr int K2T_THREADS = 512;
// Newton-Schulz output tile and padding unit of the bf16 buffers.
constexpr int NS_TILE = 256;
constexpr int NS_BK = 64;
// Matrices whose short side is at most this carry B = b A + c A^2 as a bf16
// pair (hi, lo = bf16(B - hi)) into the update product: with few singular
// values the rounding of the small m' x m' polynomial is not averaged away.
constexpr int NS_SPLIT_MAX = 128;
// Threads of every workgroup.
constexpr int NTHREADS = 256;
// Preconditioner finalise: rows or columns per workgroup (4 threads each).
constexpr int FIN_W = 64;
// Matrices whose short side is at most this run Newton-Schulz in fp32 (X, A
// and B' kept in fp32): Gram partials over SM_CH_G columns per workgroup,
// updates over SM_CH_U columns (one per thread).
constexpr int NS_SMALL_MAX = 32;
constexpr int SM_CH_G = 4096;
constexpr int SM_CH_U = 256;

typedef uint16_t bf16_t;   // bf16 storage

// Device pointers read from the descriptor tables are generic (flat) to the
// compiler, and flat memory instructions count against lgkmcnt as well as
// vmcnt: every later wait for an LDS read, a scalar load or a cross-lane
// shuffle would then also wait for them. Accesses through gptr() are global.
#define MALT_GLOBAL __attribute__((address_space(1)))
template <class T>
__device__ __forceinline__ MALT_GLOBAL T* gptr(T* p) {
  return (MALT_GLOBAL T*)p;
}

typedef float malt_f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 malt_bf16x2 __attribute__((ext_vector_type(2)));

// Two floats -> two bf16 (round to nearest even; one v_cvt_pk_bf16_f32),
// packed low | high << 16.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const malt_f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, malt_bf16x2));
}
__device__ __forceinline__ float bf16_lo(uint32_t p) { return __uint_as_float(p << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t p) { return __uint_as_float(p & 0xffff0000u); }

// Per-matrix scalar slots (float64) in the workspace.
enum {
  SC_S = 0,       // ||L M R||_F
  SC_SIGMA = 1,   // 1 / (s + ns_eps)
  SC_NU = 2,      // nu_t (MALTER)
  SC_ALPHA = 3,   // alpha_t (1 for MALT)
  SC_O2 = 4,      // ||O||_F^2
  SC_D2 = 5,      // ||L O R||_F^2
  SC_GRAFT = 6,   // ||O|| / (||D|| + eps)
  SC_COEF = 7,    // lr * alpha * graft
  SC_Q = 8,       // ||L G R||_F^2 (MALTER)
  MAT_SCALARS = 16
};

struct MatDesc {
  int32_t m, n;        // W rows, cols
  int32_t mc, nc;      // canonical orientation: mc = min(m,n) rows, nc = max(m,n) cols
  int32_t mp, np;      // canonical dims padded to NS_TILE
  int32_t tall;        // 1 when m > n: canonical = W^T
  int32_t split;       // 1: B stored as [hi | lo] (row pitch 2*mp)
  int32_t k1_ct;       // column tiles of the momentum pass (row partial count)
  int32_t k1_rt;       // row tiles of the momentum pass (column partial count)
  int32_t k2_tiles;    // scale+convert tiles (norm partial count)
  int32_t upd_tiles;   // NS update tiles (graft partial count)
  float* M;
  float* l;
  float* r;
  float* nu;           // nullptr for MALT
  float* Lv;           // m
  float* Rv;           // n
  float* rowpart;      // [k1_ct][m]
  float* colpart;      // [k1_rt][n]
  float* k2part;       // [k2_tiles][2]: sum (LMR)^2, sum (LGR)^2
  float* gpart;        // [upd_tiles][2]: sum O^2, sum (LOR)^2
  bf16_t* X[2];        // canonical mp x np, row-major (double-buffered iterate)
  bf16_t* A;           // mp x mp  (Gram / A)
  bf16_t* B;           // mp x mp, or mp x 2mp [hi | lo] when split (b A + c A^2)
  double* scal;        // MAT_SCALARS
  // fp32 Newton-Schulz (short side <= NS_SMALL_MAX); null otherwise
  int32_t small;       // 1: this matrix takes the fp32 path
  int32_t sm_gchunks;  // Gram partial count
  float* Xs[2];        // canonical mc x np fp32 iterate (row pitch np)
  float* Ap;           // [sm_gchunks][32][32] Gram partials
  float* Bs;           // [32][32] B'
};

// Per-step caller pointers; vec = 1 when W, G and M rows allow 16-byte access.
struct PtrPair {
  float* W;
  const float* G;
  int32_t vec;
  int32_t pad_;
};

// One unit of work of a grouped launch.
//   momentum/back-map: (mat, row tile, col tile, -)
//   preconditioner finalise: (mat, 0 = rows | 1 = cols, chunk, -)
//   scale+convert: (mat, row tile, col tile, partial slot)
//   NS: (mat, tile row, tile col, partial slot), stored in dispatch order:
//       entry b runs on XCD b % 8; mat = -1 pads the shorter XCD runs
//   fp32 NS: Gram (mat, chunk, -, -), polynomial (mat, -, -, -),
//            update (mat, chunk, -, partial slot)
struct Tile {
  int32_t mat, ti, tj, idx;
};

enum { PH_GRAM = 0, PH_POLY = 1, PH_UPDATE = 2 };

struct EwArgs {
  const MatDesc* desc;
  const PtrPair* ptrs;
  const Tile* tiles;
  int32_t ntiles;
  float mu1, one_minus_mu1;
  double mu2, eps;
  double bc;             // sqrt(1 - mu2^t) / (1 - mu1^t + eps)
  double ns_eps;
  double lr;
  float decay;           // 1 - lr * weight_decay
  int32_t malter;
  int32_t identity;
  int32_t o_parity;      // which X buffer holds the final O
};

struct NsArgs {
  const MatDesc* desc;
  const Tile* tiles;
  int32_t ntiles;
  int32_t phase;
  int32_t first;         // iteration 0: apply sigma
  int32_t last;          // final iteration: write O and graft partials
  int32_t src;           // X[src] is the current iterate, X[src ^ 1] receives the next
  float a, b, c;
};

// Per-step pointer table written by a kernel whose arguments carry the
// pointers: the runtime copies kernel arguments at enqueue, so a step needs no
// host staging buffer and never waits for an earlier upload.
constexpr int PTR_CHUNK = 128;
struct PtrUploadArgs {
  PtrPair* dst;
  int32_t count;       // <= PTR_CHUNK
  PtrPair p[PTR_CHUNK];
};

// Launchers (stream-ordered, no synchronisation).
hipError_t launch_ptr_upload(const PtrUploadArgs& a, hipStream_t s);
hipError_t launch_zero_fill(void* dst, size_t bytes, hipStream_t s);   // dst 16-byte aligned
hipError_t launch_momentum_rowcol(const EwArgs& a, hipStream_t s);
hipError_t launch_precond_finalize(const EwArgs& a, hipStream_t s);
hipError_t launch_scale_convert(const EwArgs& a, bool tall, hipStream_t s);
hipError_t launch_norm_scalars(const EwArgs& a, int32_t nmat, hipStream_t s);
hipError_t launch_graft_scalars(const EwArgs& a, int32_t nmat, hipStream_t s);
hipError_t launch_backmap_write(const EwArgs& a, hipStream_t s);
hipError_t launch_precond_cond(const MatDesc* desc, int32_t nmat, double* out, hipStream_t s);
hipError_t ns_gemm_setup();   // once per plan, on the plan's device
hipError_t launch_ns_gemm(const NsArgs& a, hipStream_t s);
hipError_t ns_update_setup();   // the update kernel (ns_update.hip), called by ns_gemm_setup
hipError_t launch_ns_update(const NsArgs& a, hipStream_t s);
hipError_t launch_small_ns(const NsArgs& a, hipStream_t s);

// XCDs of the chip; workgroups are dispatched to them round-robin.
constexpr int NXCD = 8;

// Map a workgroup id to a work index so that the workgroups that land on one
// XCD (dispatched round-robin over 8 XCDs) take a contiguous run of the work
// list; a bijection on [0, n).
__device__ __forceinline__ int xcd_remap(int b, int n) {
  const int q = n >> 3, r = n & 7;
  const int x = b & 7, k = b >> 3;
  return (x < r) ? x * (q + 1) + k : r * (q + 1) + (x - r) * q + k;
}

}  // namespace malt
