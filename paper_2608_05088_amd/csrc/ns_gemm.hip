// Grouped Newton-Schulz GEMMs on the gfx950 matrix cores (bf16 in, fp32 acc).
//
// One Newton-Schulz iteration (Muon's quintic) on the canonical X (mp x np,
// rows <= cols, zero-padded to multiples of 256) is three grouped launches,
// each over every matrix of the step, one 256 x 256 output tile per
// workgroup:
//   Gram        A  = s X X^T                 NT product, symmetric: upper tiles
//                                            only, mirrored on write; s = sigma^2
//                                            on the first iteration, else 1
//   Polynomial  B' = a I + b A + c A A^T     NT product (A is symmetric, so
//                                            A A = A A^T); upper tiles, mirrored
//   Update      X' = s B' X                  NN product; s = sigma on the first
//                                            iteration
// Folding a X into B' = a I + B makes X' a single product: X' needs no
// addend, and every iteration applies one rounded matrix to one rounded X.
// A, B' and X are bf16 (round to nearest even).
//
// Main loop (all three): 8 waves (2 per SIMD), each owning a 128 x 64 sub-tile
// as 32x32 blocks of v_mfma_f32_32x32x16_bf16.  Operand stages of BK k-values
// stream from global memory straight into an LDS ring (global_load_lds,
// 16 bytes per lane), STAGES deep, one barrier per stage; fragments are
// double-buffered in registers so the reads for the next 16-k sub-step are in
// flight while the current one multiplies.
//
// NT operands (rows with k contiguous) use ds_read_b128 fragments from an
// XOR-swizzled [row][k] tile.  The update reads X as a row-major [k][n]
// stage tile and builds the MFMA A operand with ds_read_b64_tr_b16 transposed
// reads; it computes C^T = X^T B' so every lane holds four consecutive output
// columns of one row and stores them straight from registers.
#include <type_traits>

#include "malt_internal.h"

namespace malt {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

#ifndef MALT_NS_BK
#define MALT_NS_BK 64
#endif
#ifndef MALT_NS_STAGES
#define MALT_NS_STAGES 2
#endif
#ifndef MALT_NS_WAVES
#define MALT_NS_WAVES 8
#endif
constexpr int NW = MALT_NS_WAVES;                    // waves per workgroup (4 or 8)
constexpr int WPE = NW / 4;                          // waves per SIMD
constexpr int NT = NW * 64;                          // threads per workgroup
constexpr int BK = MALT_NS_BK;                       // k per pipeline stage
constexpr int STAGES = MALT_NS_STAGES;               // LDS ring depth
constexpr int H = BK / 16;                           // MFMA sub-steps per stage
constexpr int RB = BK * 2;                           // bytes per [row][k] tile row
constexpr int CPR = BK / 8;                          // 16-byte chunks per [row][k] row
constexpr int RPP = 256 / RB;                        // [row][k] rows per 256-byte bank period
constexpr int KN_ROW = NS_TILE * 2;                  // bytes per [k][n] tile row (512)
constexpr int OPER_BYTES = NS_TILE * BK * 2;         // one operand tile of one stage
constexpr int STAGE_BYTES = 2 * OPER_BYTES;
constexpr int RING_BYTES = STAGES * STAGE_BYTES;
constexpr int LOADS = 2 * OPER_BYTES / 1024 / NW;    // 1 KB direct loads per wave per stage
// Epilogues stage a whole bf16 output tile in LDS and write it out in
// 512-byte rows.  A tile written column-wise (each lane: four consecutive rows
// of one column, 8 bytes into one staged row) uses rows padded by 8 bytes, so
// the 32 staged rows of one write land in distinct banks; a tile written
// row-wise (each lane: four consecutive columns) uses rows padded by 64 bytes.
// The update instead stages each wave's sub-tile (128 rows of 64 bf16 when
// NW = 8) in a region of its own, rows padded by 8 bytes, and keeps its
// per-tile norm partials past the NW regions.
constexpr int ST_PITCH_T = NS_TILE * 2 + 8;
constexpr int ST_PITCH_R = NS_TILE * 2 + 64;
constexpr int UPD_PITCH = NS_TILE / (NW / 2) * 2 + 8;
constexpr int UPD_WAVE = NS_TILE / 2 * UPD_PITCH;
constexpr int UPD_RED = NW * UPD_WAVE;
// Off-diagonal Gram/polynomial tiles also go through per-wave regions: the
// sub-tile transposed (TN rows of TM bf16, padded by 8 bytes), then as is (TM
// rows of TN bf16, unpadded, halves swapped on alternate row pairs).
constexpr int SYM_PITCH_T = NS_TILE / 2 * 2 + 8;
constexpr int SYM_WAVE = (NS_TILE / (NW / 2)) * SYM_PITCH_T > (NS_TILE / 2) * (NS_TILE / (NW / 2)) * 2
                             ? (NS_TILE / (NW / 2)) * SYM_PITCH_T
                             : (NS_TILE / 2) * (NS_TILE / (NW / 2)) * 2;
constexpr int UPD_EPI_BYTES = UPD_RED + 2 * NW * 4;
constexpr int SYM_EPI_BYTES = NS_TILE * ST_PITCH_R;
constexpr int EPI_BYTES = UPD_EPI_BYTES > SYM_EPI_BYTES ? UPD_EPI_BYTES : SYM_EPI_BYTES;
constexpr int LDS_BYTES = RING_BYTES > EPI_BYTES ? RING_BYTES : EPI_BYTES;
static_assert(LDS_BYTES <= 160 * 1024, "LDS budget");
static_assert(NW * SYM_WAVE <= LDS_BYTES && UPD_RED + 2 * NW * 4 <= LDS_BYTES, "per-wave epilogue regions");
static_assert(H % 2 == 0, "sub-steps per stage must be even");
static_assert(LOADS * NW * 1024 == 2 * OPER_BYTES, "loads must split evenly over the waves");

// Wave grid 2 x (NW / 2): each wave owns TM x TN of the 256 x 256 tile.
constexpr int TM = NS_TILE / 2, TN = NS_TILE / (NW / 2);

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4_t;
typedef __attribute__((address_space(1))) void gbl_void_t;

__device__ __forceinline__ float bf2f_(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

__device__ __forceinline__ float wsum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Wait until at most n (<= 63) of this wave's vector-memory loads are in flight.
#define MALT_VM_CASE(k) case k: asm volatile("s_waitcnt vmcnt(" #k ")" ::: "memory"); break;
__device__ __forceinline__ void wait_vm(int n) {
  switch (n) {
    MALT_VM_CASE(0) MALT_VM_CASE(1) MALT_VM_CASE(2) MALT_VM_CASE(3) MALT_VM_CASE(4) MALT_VM_CASE(5)
    MALT_VM_CASE(6) MALT_VM_CASE(7) MALT_VM_CASE(8) MALT_VM_CASE(9) MALT_VM_CASE(10) MALT_VM_CASE(11)
    MALT_VM_CASE(12) MALT_VM_CASE(13) MALT_VM_CASE(14) MALT_VM_CASE(15) MALT_VM_CASE(16)
    MALT_VM_CASE(18) MALT_VM_CASE(20) MALT_VM_CASE(24) MALT_VM_CASE(28) MALT_VM_CASE(32)
    MALT_VM_CASE(36) MALT_VM_CASE(40) MALT_VM_CASE(48) MALT_VM_CASE(56)
    default: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
  }
}
#undef MALT_VM_CASE

// Compile-time vmcnt wait (gfx9 s_waitcnt encoding: vmcnt[3:0] and [15:14],
// expcnt and lgkmcnt left at their maxima, i.e. not waited on).
template <int N>
__device__ __forceinline__ void wait_vm_c() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Operands are read through buffer resources (base address in scalar
// registers, unbounded range, raw addressing): the buffer form of the direct
// load moves more bytes per clock into LDS than the flat-address form.
typedef int i32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ i32x4 buf_rsrc(const void* base) {
  const uint64_t b = (uint64_t)(uintptr_t)base;
  i32x4 r;
  r.x = (int)(uint32_t)b;
  r.y = (int)(uint32_t)((b >> 32) & 0xFFFFu);   // stride 0
  r.z = -1;                                      // num_records: no clamping below 4 GB
  r.w = 0x00020000;                              // 32-bit data format, raw access
  return r;
}

// One 16-byte-per-lane direct load into LDS: lane i reads base + soff + voff_i
// and writes lds_addr + 16 i (lds_addr wave-uniform).  Issued from inline
// assembly so the compiler does not track it: it cannot tell the ring slot
// being filled from the slot being read, and before the transposed reads of
// the update it would wait for each stage's loads right after issuing them.
// Completion is ordered by the pipeline's explicit vmcnt waits and barriers;
// m0 carries the LDS address and needs one wait state after its write.
__device__ __forceinline__ void dma16(const i32x4& rsrc, uint32_t voff, uint32_t soff, uint32_t lds_addr) {
  asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
               :
               : "v"(voff), "s"(rsrc), "s"(soff), "{m0}"(lds_addr)
               : "memory");
}

// LDS byte address of a generic pointer into LDS: its low 32 bits (the flat
// LDS aperture keeps the offset there), read as wave-uniform.
__device__ __forceinline__ uint32_t lds_u32(const void* p) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)p);
}

// [row][k] tile (NT operands): 256 rows x BK bf16, CPR 16-byte chunks per row,
// chunk kc stored at kc ^ ((row / RPP) % CPR): the ds_read_b128 fragment reads
// of 16 consecutive rows at one chunk hit 16 distinct 4-bank groups.
__device__ __forceinline__ int swz_rk(int row, int kc) { return row * RB + ((kc ^ ((row / RPP) % CPR)) << 4); }

// [k][n] tile (X in the update): BK rows of 256 bf16 (512 bytes), 16-byte chunk
// c stored at c ^ (4 * (k & 3)): the 16 lanes of one transposed read (four
// rows x 32 contiguous bytes) hit 16 distinct 4-bank groups.
__device__ __forceinline__ int swz_kn(int k, int n) {
  return k * KN_ROW + (((n >> 3) ^ (4 * (k & 3))) << 4) + ((n & 7) << 1);
}

// Software pipeline over KT stages shared by both kernels.
//   issue(kt, i)      the i-th direct load (0 <= i < nl) this wave issues for
//                     stage kt, into slot kt % STAGES
//   read(buf, st, h)  fragment reads of sub-step h of the stage at st into buf
//   mma(buf, after)   the MFMAs of the fragments in buf, calling after(j) once
//                     the j-th of the NMMA has been issued
// nl is the number of loads this wave issues per stage (LOADS, or fewer).
//
// Burst (two slots): at the barrier closing stage kt, stage kt + 1 has landed
// and every wave is done with slot kt % 2, which then receives all of stage
// kt + 2's loads.
// Spread (three or more slots): stage kt + STAGES - 1 is loaded while stage kt
// computes, its nl loads spread over the H sub-steps (nl / H per sub-step, each
// after an equal share of the MFMAs), into the slot stage kt - 1 freed.  The
// loads of STAGES - 2 stages stay in flight across every barrier, and no wave
// issues a burst of loads while its SIMD partner waits for the matrix core.
constexpr int NMMA = (TM / 32) * (TN / 32);   // MFMAs per wave per sub-step
#ifndef MALT_NS_SPREAD
#define MALT_NS_SPREAD (MALT_NS_STAGES >= 3)
#endif
constexpr bool SPREAD = MALT_NS_SPREAD != 0;
static_assert(!SPREAD || STAGES >= 3, "spread loads need two stages of lead");

template <int RPM, class Issue, class Read, class Mma>
__device__ __forceinline__ void pipeline(const int KT, const int nl, char* lds, Issue&& issue, Read&& read,
                                         Mma&& mma) {
  constexpr int PRE = SPREAD ? STAGES - 1 : STAGES;   // stages loaded before the loop
  // Load indices stay compile-time constants (the kernels index register
  // arrays with them); a wave issuing nl < LOADS loads skips indices >= nl.
#pragma unroll
  for (int s = 0; s < PRE; ++s)
    if (s < KT)
#pragma unroll
      for (int i = 0; i < LOADS; ++i)
        if (i < nl) issue(s, i);
  wait_vm(min(PRE - 1, KT - 1) * nl);   // stage 0 has landed
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  read(0, lds, 0);
  // Spread: load i of a stage goes out in sub-step i / PER, after MFMA
  // (i % PER + 1) * GAP - 1; before the last sub-step min(nl, (H-1) PER) of a
  // stage's loads have been issued.
  constexpr int PER = LOADS / H;
  constexpr int GAP = NMMA / PER;
  static_assert(!SPREAD || (LOADS % H == 0 && NMMA % PER == 0), "loads must spread evenly over the MFMAs");
  const int early = min(nl, (H - 1) * PER);
  auto body = [&](const int kt, auto steady_tag) {
    // steady: the stage this iteration loads (burst: kt + 2 at the barrier;
    // spread: kt + STAGES - 1 over the sub-steps) exists.
    constexpr bool steady = decltype(steady_tag)::value;
    const char* st = lds + (kt % STAGES) * STAGE_BYTES;
#pragma unroll
    for (int h = 0; h < H; ++h) {
      const int c = h & 1;
      if (h + 1 < H) {
        read(c ^ 1, st, h + 1);
      } else if (steady || kt + 1 < KT) {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // this wave's reads of stage kt are done
        if constexpr (SPREAD) {
          // In flight after stage kt + 1: whole stages kt + 2 .. kt + STAGES - 2
          // and, when it exists, all but the last sub-step's share of stage
          // kt + STAGES - 1.
          if constexpr (steady) wait_vm((STAGES - 3) * nl + early);
          else wait_vm(max(0, min(kt + STAGES - 2, KT - 1) - (kt + 1)) * nl);
        } else {
          if constexpr (steady) {
            if constexpr (STAGES == 2) wait_vm_c<0>();
            else wait_vm((STAGES - 2) * nl);
          } else {
            wait_vm(min(STAGES - 2, KT - 1 - (kt + 1)) * nl);
          }
        }
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        if constexpr (!SPREAD && steady) {
#pragma unroll
          for (int i = 0; i < LOADS; ++i)
            if (i < nl) issue(kt + STAGES, i);
        }
        read(c ^ 1, lds + ((kt + 1) % STAGES) * STAGE_BYTES, 0);
      }
      mma(c, [&](int j) {
        if constexpr (SPREAD && steady) {
          if ((j + 1) % GAP == 0) {
            const int i = h * PER + j / GAP;
            if (i < nl) issue(kt + STAGES - 1, i);
          }
        }
      });
      // Interleave the sub-step's MFMAs with the fragment reads for the next
      // one, RPM reads after each MFMA, so each read's latency is covered by
      // this wave's own MFMAs (left to itself the scheduler puts the reads
      // after the last MFMA and the next sub-step then waits for them).
#pragma unroll
      for (int j = 0; j < NMMA; ++j) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);     // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, RPM, 0);   // RPM LDS reads
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  constexpr int LEAD = SPREAD ? STAGES - 1 : STAGES;
  int kt = 0;
  for (; kt < KT - LEAD; ++kt) body(kt, std::true_type{});
  for (; kt < KT; ++kt) body(kt, std::false_type{});
}

#ifndef MALT_NS_UPDATE_TU
// ===========================================================================
// Gram and polynomial phases: C = P Q^T, symmetric output, upper tiles.
// ===========================================================================
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(WPE, WPE)))
void ns_gemm_sym_kernel(NsArgs args) {
  constexpr int I = TM / 32, J = TN / 32;    // 32x32 blocks per wave
  constexpr int ROWS_PER_LOAD = 1024 / RB;
  constexpr int LOADS_PER_OPER = NS_TILE / ROWS_PER_LOAD;

  extern __shared__ __attribute__((aligned(16))) char lds[];
  // Every descriptor field the tile needs is read here, before any store, so
  // the uniform loads go through the scalar cache.
  // The work list is in dispatch order (XCD-balanced on the host); entries
  // with mat < 0 pad the shorter XCD runs.
  const Tile t = args.tiles[blockIdx.x];
  if (t.mat < 0) return;
  const MatDesc* __restrict__ d = args.desc + t.mat;
  const int phase = args.phase;
  const int mp = d->mp, np = d->np;
  const bool split = d->split != 0;
  bf16_t* const Am = d->A;
  bf16_t* const Bm = d->B;
  const bf16_t* P = (phase == PH_GRAM) ? d->X[args.src] : Am;
  const float sig = (args.first && phase == PH_GRAM) ? (float)d->scal[SC_SIGMA] : 1.f;
  const int ld = (phase == PH_GRAM) ? np : mp;
  const int K = ld;
  const int row0 = t.ti * NS_TILE, col0 = t.tj * NS_TILE;
  // A diagonal tile's row and column panels are the same rows of P: it loads
  // the row panel only and reads both operands from it.
  const bool diag = t.ti == t.tj;

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // Sub-tile of each wave. On a diagonal tile only the 32 x 32 blocks on or
  // above the block diagonal are computed (the others are their mirrors). The
  // two waves that share a SIMD (waves w and w + 4) then take sub-tiles with
  // 8 + 0, 8 + 0, 7 + 3 and 3 + 7 such blocks, instead of the 3 + 0, 7 + 0,
  // 8 + 3 and 8 + 7 of the plain order, so every matrix core gets a share.
  static_assert(NW != 8 || (TM == 128 && TN == 64), "diagonal sub-tile pairing assumes a 2 x 4 wave grid");
  const int role = (NW == 8 && diag) ? ((0x76540132u >> (4 * wave)) & 0xF) : wave;
  const int wr = role / (NW / 2), wc = role % (NW / 2);

  // Direct-load sources: instruction g < LOADS_PER_OPER covers rows of the
  // tile-row panel, the rest rows of the tile-column panel (both of P); byte
  // offsets into P's buffer (the padded canonical matrix is below 4 GB).
  const i32x4 rsP = buf_rsrc(P);
  uint32_t voff[LOADS];
  int dst_off[LOADS];
#pragma unroll
  for (int q = 0; q < LOADS; ++q) {
    const int g = wave + q * NW;
    const int op = g / LOADS_PER_OPER, qi = g % LOADS_PER_OPER;
    const int row = qi * ROWS_PER_LOAD + lane / CPR;
    const int kc = (lane % CPR) ^ ((row / RPP) % CPR);
    voff[q] = (uint32_t)(((size_t)((op ? col0 : row0) + row) * ld + kc * 8) * 2);
    dst_off[q] = op * OPER_BYTES + qi * 1024;
  }
  int offa[I][H], offb[J][H];
#pragma unroll
  for (int h = 0; h < H; ++h) {
    const int kc = 2 * h + (lane >> 5);
#pragma unroll
    for (int i = 0; i < I; ++i) offa[i][h] = swz_rk(wr * TM + i * 32 + (lane & 31), kc);
#pragma unroll
    for (int j = 0; j < J; ++j) offb[j][h] = (diag ? 0 : OPER_BYTES) + swz_rk(wc * TN + j * 32 + (lane & 31), kc);
  }

  f32x16 acc[I][J];
#pragma unroll
  for (int i = 0; i < I; ++i)
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  bf16x8 fa[2][I], fb[2][J];

  // With 8 waves, g = wave + 8q < LOADS_PER_OPER exactly for q < LOADS / 2:
  // the first half of a wave's loads are row-panel loads.
  static_assert(LOADS_PER_OPER == (LOADS / 2) * NW, "row-panel loads are the first half");
  // Diagonal and off-diagonal tiles run separate copies of the main loop, so
  // the block test exists only on diagonal tiles.
  auto main_loop = [&](auto diag_tag) {
    constexpr bool DIAG = decltype(diag_tag)::value;
    pipeline<1>(
        K / BK, DIAG ? LOADS / 2 : LOADS, lds,
        [&](int kt, int i) {   // diagonal tiles issue the row-panel loads q < LOADS / 2 only
          dma16(rsP, voff[i], (uint32_t)(kt * BK * 2), lds_u32(lds + (kt % STAGES) * STAGE_BYTES + dst_off[i]));
        },
        [&](int buf, const char* st, int h) {
#pragma unroll
          for (int i = 0; i < I; ++i) fa[buf][i] = *reinterpret_cast<const bf16x8*>(st + offa[i][h]);
#pragma unroll
          for (int j = 0; j < J; ++j) fb[buf][j] = *reinterpret_cast<const bf16x8*>(st + offb[j][h]);
        },
        [&](int buf, auto&& after) {
#pragma unroll
          for (int i = 0; i < I; ++i)
#pragma unroll
            for (int j = 0; j < J; ++j) {
              // Diagonal tiles skip the blocks below the block diagonal.
              if (!DIAG || (wr * TM) / 32 + i <= (wc * TN) / 32 + j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[buf][i], fb[buf][j], acc[i][j], 0, 0, 0);
              after(i * J + j);
            }
        });
  };
  if (diag) main_loop(std::true_type{});
  else main_loop(std::false_type{});

  // ---------------------------------------------------------------- epilogue
  // acc[i][j][4g + e] = C(r, c): tile row r = wr*TM + i*32 + 8g + 4*(lane >> 5)
  // + e, tile column c = wc*TN + j*32 + (lane & 31), so each lane holds four
  // consecutive rows of one column.  The final bf16 values are formed in
  // registers; the tile then leaves through LDS twice in whole rows: first
  // transposed (the mirror tile C^T), then as is after a 4 x 4 transpose
  // inside each lane quad. A diagonal tile is its own mirror and leaves once:
  // its staged copy takes the computed blocks transposed and the blocks above
  // the block diagonal as is, so it is symmetric by construction.
  const bool poly = phase == PH_POLY;
  const float sc = sig * sig;
  // Split B': the low part bf16(v - hi) goes mp columns to the right.
  const int lo_off = (poly && split) ? mp : 0;
  bf16_t* const out = poly ? Bm : Am;
  const int ldo = lo_off ? 2 * mp : mp;
  const int rl0 = wr * TM + 4 * (lane >> 5);   // tile row of i = g = e = 0
  const int cl0 = wc * TN + (lane & 31);       // tile column of j = 0

  __syncthreads();   // every wave is done reading the operand ring
  if (poly) {
    // B' = a I + b A + c A A^T takes A(r, c) at each accumulator position.
    // A's tile goes to LDS as 256 rows in the [k][n] layout (direct loads),
    // and each lane reads its four rows of one column with one transposed
    // read per (i, j, g).
    const i32x4 rsA = buf_rsrc(Am);
#pragma unroll
    for (int it = 0; it < NS_TILE * NS_TILE * 2 / (16 * NT); ++it) {
      const int c = tid + NT * it;                // 16-byte chunk of the tile
      const int row = c >> 5, pc = c & 31;        // physical chunk pc holds logical chunk pc ^ 4 (row & 3)
      const int lc = pc ^ (4 * (row & 3));
      dma16(rsA, (uint32_t)(((size_t)(row0 + row) * mp + col0 + lc * 8) * 2), 0u,
            lds_u32(lds + (c - lane) * 16));
    }
    wait_vm_c<0>();
    __syncthreads();
  }
  uint2 hv[I][J][4];
  {
    const int r = (lane & 15) >> 2, q = lane & 3;
#pragma unroll
    for (int i = 0; i < I; ++i)
#pragma unroll
      for (int j = 0; j < J; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * g + e];
          if (poly) {
            const int k0 = rl0 + i * 32 + 8 * g;
            const int n0 = wc * TN + j * 32 + 16 * ((lane >> 4) & 1);
            const i16x4 av = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)(lds + swz_kn(k0 + r, n0 + 4 * q)));
            const int R = row0 + k0, C = col0 + cl0 + j * 32;
#pragma unroll
            for (int e = 0; e < 4; ++e)
              v[e] = args.b * bf2f_((bf16_t)av[e]) + args.c * v[e] + (R + e == C ? args.a : 0.f);
          }
          hv[i][j][g].x = pack_bf16x2(sc * v[0], sc * v[1]);
          hv[i][j][g].y = pack_bf16x2(sc * v[2], sc * v[3]);
          if (lo_off) {
            // Keep the low parts in acc (its values are no longer needed).
            acc[i][j][4 * g + 0] = sc * v[0] - bf16_lo(hv[i][j][g].x);
            acc[i][j][4 * g + 1] = sc * v[1] - bf16_hi(hv[i][j][g].x);
            acc[i][j][4 * g + 2] = sc * v[2] - bf16_lo(hv[i][j][g].y);
            acc[i][j][4 * g + 3] = sc * v[3] - bf16_hi(hv[i][j][g].y);
          }
        }
  }

  // Row-wise copy of accumulator group (i, j, g): a 4 x 4 transpose of
  // 16-bit values inside each lane quad, after which lane p of the quad holds
  // row p of the quad's four rows, its four columns.
  const int p = lane & 3;
  auto quad_rows = [&](int i, int j, int g) {
    const uint32_t A0 = hv[i][j][g].x, B0 = hv[i][j][g].y;   // rows (0,1), (2,3) of column p
    const uint32_t A1 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)A0, 0xB1, 0xF, 0xF, true);   // lane p ^ 1
    const uint32_t B1 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)B0, 0xB1, 0xF, 0xF, true);
    // Even lanes: row 0 (A) / row 2 (B) at columns p, p+1; odd lanes:
    // row 1 / row 3 at columns p-1, p.
    const uint32_t nA = (p & 1) ? ((A1 >> 16) | (A0 & 0xffff0000u)) : ((A0 & 0xffffu) | (A1 << 16));
    const uint32_t nB = (p & 1) ? ((B1 >> 16) | (B0 & 0xffff0000u)) : ((B0 & 0xffffu) | (B1 << 16));
    const uint32_t S = (p < 2) ? nB : nA;
    const uint32_t S2 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)S, 0x4E, 0xF, 0xF, true);   // lane p ^ 2
    return (p < 2) ? make_uint2(nA, S2) : make_uint2(S2, nB);
  };
  // Writes one set of values (hi, or the split low part at column offset
  // off): the transposed staging first, then the row-wise one.
  auto emit = [&](int off) {
    constexpr int CHUNKS = NS_TILE * NS_TILE * 2 / 16;
    __syncthreads();   // LDS free (A's tile read, or the previous copy-out done)
    if constexpr (TM == 128 && TN == 64) {   // the layout below assumes 128 x 64 wave blocks
      if (!diag) {
        // Off-diagonal tile: each wave moves its own TM x TN block through a
        // private LDS region, first transposed (to the mirror tile), then as
        // is.  A wave reads back only what it wrote and LDS operations of one
        // wave stay in order, so no barrier separates the phases.  Outputs are
        // written with streaming stores, as in the update: the next phase
        // reads them from other XCDs.
        char* const wreg = lds + wave * SYM_WAVE;
#pragma unroll
        for (int i = 0; i < I; ++i)
#pragma unroll
          for (int j = 0; j < J; ++j)
#pragma unroll
            for (int g = 0; g < 4; ++g)
              *reinterpret_cast<uint2*>(wreg + ((lane & 31) + j * 32) * SYM_PITCH_T +
                                        (4 * (lane >> 5) + i * 32 + 8 * g) * 2) = hv[i][j][g];
        // Mirror: staged row x (of TM bf16) goes to row col0 + wc*TN + x.
        constexpr int TCH = TM * 2 / 16;
#pragma unroll
        for (int it = 0; it < TN * TCH / 64; ++it) {
          const int q = lane + 64 * it;
          const int r = q / TCH, ch = q % TCH;
          const char* src = wreg + r * SYM_PITCH_T + ch * 16;
          const uint2 lo = *reinterpret_cast<const uint2*>(src);
          const uint2 hi = *reinterpret_cast<const uint2*>(src + 8);
          const u32x4 v = {lo.x, lo.y, hi.x, hi.y};
          __builtin_nontemporal_store(v, reinterpret_cast<MALT_GLOBAL u32x4*>(
                                             gptr(out) + (size_t)(col0 + wc * TN + r) * ldo + off + row0 + wr * TM + ch * 8));
        }
        // As is: 128-byte rows; rows 2 and 3 (mod 4) hold their two 64-byte
        // halves swapped, so the four rows of one quad write land in four
        // distinct 16-bank groups.
#pragma unroll
        for (int i = 0; i < I; ++i)
#pragma unroll
          for (int j = 0; j < J; ++j)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const int r = 4 * (lane >> 5) + i * 32 + 8 * g + p;
              const int hf = j ^ ((r >> 1) & 1);
              *reinterpret_cast<uint2*>(wreg + r * (TN * 2) + hf * 64 + (((lane & 31) >> 2) << 3)) =
                  quad_rows(i, j, g);
            }
        constexpr int DCH = TN * 2 / 16;
#pragma unroll
        for (int it = 0; it < TM * DCH / 64; ++it) {
          const int q = lane + 64 * it;
          const int r = q / DCH, ch = q % DCH;
          const int hf = (ch >> 2) ^ ((r >> 1) & 1);
          const u32x4 v = *reinterpret_cast<const u32x4*>(wreg + r * (TN * 2) + hf * 64 + (ch & 3) * 16);
          __builtin_nontemporal_store(v, reinterpret_cast<MALT_GLOBAL u32x4*>(
                                             gptr(out) + (size_t)(row0 + wr * TM + r) * ldo + off + col0 + wc * TN + ch * 8));
        }
        return;
      }
    }
    // Transposed staging: staged row x is tile column x. A diagonal tile
    // stages only its computed blocks this way (block row <= block column) and
    // stages the blocks above the block diagonal also as is, at the places of
    // their skipped mirrors: the staged tile is then the whole symmetric tile.
#pragma unroll
    for (int i = 0; i < I; ++i)
#pragma unroll
      for (int j = 0; j < J; ++j) {
        const int br = (wr * TM) / 32 + i, bc = (wc * TN) / 32 + j;   // wave-uniform block coordinates
        if (!diag || br <= bc)
#pragma unroll
          for (int g = 0; g < 4; ++g)
            *reinterpret_cast<uint2*>(lds + (cl0 + j * 32) * ST_PITCH_T + (rl0 + i * 32 + 8 * g) * 2) = hv[i][j][g];
        if (diag && br < bc)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int rr = rl0 + i * 32 + 8 * g + p;
            const int cc = wc * TN + j * 32 + ((lane & 31) & ~3);
            *reinterpret_cast<uint2*>(lds + rr * ST_PITCH_T + cc * 2) = quad_rows(i, j, g);
          }
      }
    __syncthreads();
    // Staged row x goes to row col0 + x (the mirror tile; on a diagonal tile,
    // the tile itself).
#pragma unroll 4
    for (int c = tid; c < CHUNKS; c += NT) {
      const int row = c >> 5, ch = c & 31;
      const char* src = lds + row * ST_PITCH_T + ch * 16;
      const uint2 lo = *reinterpret_cast<const uint2*>(src);
      const uint2 hi = *reinterpret_cast<const uint2*>(src + 8);
      const u32x4 v = {lo.x, lo.y, hi.x, hi.y};
      __builtin_nontemporal_store(
          v, reinterpret_cast<MALT_GLOBAL u32x4*>(gptr(out) + (size_t)(col0 + row) * ldo + off + row0 + ch * 8));
    }
    if (diag) return;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < I; ++i)
#pragma unroll
      for (int j = 0; j < J; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int rr = rl0 + i * 32 + 8 * g + p;
          const int cc = wc * TN + j * 32 + ((lane & 31) & ~3);
          *reinterpret_cast<uint2*>(lds + rr * ST_PITCH_R + cc * 2) = quad_rows(i, j, g);
        }
    __syncthreads();
#pragma unroll 4
    for (int c = tid; c < CHUNKS; c += NT) {
      const int row = c >> 5, ch = c & 31;
      __builtin_nontemporal_store(*reinterpret_cast<const u32x4*>(lds + row * ST_PITCH_R + ch * 16),
                                  reinterpret_cast<MALT_GLOBAL u32x4*>(gptr(out) + (size_t)(row0 + row) * ldo + off +
                                                                       col0 + ch * 8));
    }
  };
  emit(0);
  if (lo_off) {
#pragma unroll
    for (int i = 0; i < I; ++i)
#pragma unroll
      for (int j = 0; j < J; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          hv[i][j][g].x = pack_bf16x2(acc[i][j][4 * g + 0], acc[i][j][4 * g + 1]);
          hv[i][j][g].y = pack_bf16x2(acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
        }
    emit(lo_off);
  }
}

#else
// ===========================================================================
// Update phase: X' = s B' X  (NN), computed as C^T = X^T B'^T blocks.
// ===========================================================================
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(WPE, WPE)))
void ns_update_kernel(NsArgs args) {
  constexpr int NB = TM / 32;                // B' fragments (output rows, MFMA B operand)
  constexpr int NA = TN / 32;                // X fragments (output cols, MFMA A operand)
  constexpr int ROWS_PER_LOAD = 1024 / RB;   // B' rows per 1 KB load
  constexpr int LOADS_P = NS_TILE / ROWS_PER_LOAD;
  constexpr int KROWS_PER_LOAD = 1024 / KN_ROW;   // X k-rows per 1 KB load (2)

  extern __shared__ __attribute__((aligned(16))) char lds[];
  // Every descriptor field the tile needs is read here, before any store, so
  // the uniform loads go through the scalar cache.
  // The work list is in dispatch order (XCD-balanced on the host); entries
  // with mat < 0 pad the shorter XCD runs.
  const Tile t = args.tiles[blockIdx.x];
  if (t.mat < 0) return;
  const MatDesc* __restrict__ d = args.desc + t.mat;
  const int mp = d->mp, np = d->np, mc = d->mc, nc = d->nc;
  const bool tall = d->tall != 0;
  // Split matrices contract over [B'_hi | B'_lo] and [X ; X]: K = 2 mp.
  const int ldb = d->split ? 2 * mp : mp;
  const int K = ldb;
  const bf16_t* Bm = d->B;
  const bf16_t* X = d->X[args.src];
  bf16_t* const Xn = d->X[args.src ^ 1];
  const float* const Lv = d->Lv;
  const float* const Rv = d->Rv;
  float* const gpart = d->gpart;
  const float sc = args.first ? (float)d->scal[SC_SIGMA] : 1.f;
  const int row0 = t.ti * NS_TILE, col0 = t.tj * NS_TILE;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave / (NW / 2), wc = wave % (NW / 2);

  // Direct-load sources as byte offsets into the B' and X buffers: load
  // g < LOADS_P covers B' rows, the rest X k-rows of the tile.
  const i32x4 rsB = buf_rsrc(Bm);
  const i32x4 rsX = buf_rsrc(X);
  // With 8 waves, g = wave + 8q < LOADS_P exactly for q < LOADS / 2, so which
  // operand a load reads is known at compile time.
  static_assert(LOADS_P == (LOADS / 2) * NW, "B' loads are the first half");
  uint32_t voff[LOADS];
  int dst_off[LOADS];
#pragma unroll
  for (int q = 0; q < LOADS; ++q) {
    const int g = wave + q * NW;
    if (q < LOADS / 2) {
      const int row = g * ROWS_PER_LOAD + lane / CPR;
      const int kc = (lane % CPR) ^ ((row / RPP) % CPR);
      voff[q] = (uint32_t)(((size_t)(row0 + row) * ldb + kc * 8) * 2);
      dst_off[q] = g * 1024;
    } else {
      const int qi = g - LOADS_P;
      const int k = qi * KROWS_PER_LOAD + lane / 32;
      const int c = (lane % 32) ^ (4 * (k & 3));   // logical 16-byte chunk of this physical slot
      voff[q] = (uint32_t)(((size_t)k * np + col0 + c * 8) * 2);
      dst_off[q] = OPER_BYTES + qi * 1024;
    }
  }
  // B' fragments: rows of the output, k contiguous.
  int offb[NB][H];
#pragma unroll
  for (int h = 0; h < H; ++h)
#pragma unroll
    for (int b = 0; b < NB; ++b) offb[b][h] = swz_rk(wr * TM + b * 32 + (lane & 31), 2 * h + (lane >> 5));
  // X fragments through transposed reads: in each 16-lane group, lane
  // j = q + 4r addresses row k0 + r, columns n0 + 4q .. n0 + 4q + 3; the
  // read hands lane i the four rows of column n0 + i.
  int offx[NA][2];
  {
    const int r = (lane & 15) >> 2, q = lane & 3;
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int r2 = 0; r2 < 2; ++r2) {
        const int k = 8 * (lane >> 5) + 4 * r2 + r;
        const int n = wc * TN + a * 32 + 16 * ((lane >> 4) & 1) + 4 * q;
        offx[a][r2] = OPER_BYTES + swz_kn(k, n);
      }
  }

  f32x16 acc[NA][NB];
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.f;
  bf16x8 fx[2][NA], fb[2][NB];

  pipeline<2>(
      K / BK, LOADS, lds,
      [&](int kt, int q) {   // q < LOADS / 2: B' rows, else X k-rows
        const int k0 = kt * BK;
        const int k0x = k0 >= mp ? k0 - mp : k0;   // X's k wraps for split matrices
        const uint32_t la = lds_u32(lds + (kt % STAGES) * STAGE_BYTES + dst_off[q]);
        if (q < LOADS / 2) dma16(rsB, voff[q], (uint32_t)(k0 * 2), la);
        else dma16(rsX, voff[q], (uint32_t)((size_t)k0x * np * 2), la);
      },
      [&](int buf, const char* st, int h) {
#pragma unroll
        for (int b = 0; b < NB; ++b) fb[buf][b] = *reinterpret_cast<const bf16x8*>(st + offb[b][h]);
#pragma unroll
        for (int a = 0; a < NA; ++a) {
          const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_i16x4_t*)(st + offx[a][0] + h * 16 * KN_ROW));
          const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_i16x4_t*)(st + offx[a][1] + h * 16 * KN_ROW));
          fx[buf][a] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        }
      },
      [&](int buf, auto&& after) {
#pragma unroll
        for (int a = 0; a < NA; ++a)
#pragma unroll
          for (int b = 0; b < NB; ++b) {
            acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fx[buf][a], fb[buf][b], acc[a][b], 0, 0, 0);
            after(a * NB + b);
          }
      });

  // ---------------------------------------------------------------- epilogue
  // acc[a][b][4g + e] = C(m, n + e), m = row0 + wr*TM + b*32 + (lane & 31),
  // n = col0 + wc*TN + a*32 + 8g + 4*(lane >> 5): four consecutive bf16 per
  // lane.  Each wave copies its own TM x TN sub-tile to a private LDS region
  // and writes it out in whole 128-byte row pieces, not as 16-byte pieces of
  // 32 rows.  A wave reads back only what it staged, so no barrier separates
  // the two and each wave leaves the epilogue at its own pace.
  const int ml0 = wr * TM + (lane & 31);          // tile-local row of b = 0
  const int nl0 = wc * TN + 4 * (lane >> 5);      // tile-local column of a = g = 0
  const int sr0 = lane & 31, sc0 = 4 * (lane >> 5);   // the same within the sub-tile
  char* const sto = lds + wave * UPD_WAVE;
  __syncthreads();   // every wave is done reading the operand ring
  float o2 = 0.f, d2 = 0.f;
  if (!args.last) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          uint2 pk;
          pk.x = pack_bf16x2(sc * acc[a][b][4 * g + 0], sc * acc[a][b][4 * g + 1]);
          pk.y = pack_bf16x2(sc * acc[a][b][4 * g + 2], sc * acc[a][b][4 * g + 3]);
          *reinterpret_cast<uint2*>(sto + (sr0 + b * 32) * UPD_PITCH + (sc0 + a * 32 + 8 * g) * 2) = pk;
        }
  } else {
    // Last iteration: also the per-tile sums of O^2 and (L O R)^2, from the
    // rounded O.  Canonical (m, n) is W(m, n) for wide and W(n, m) for tall
    // matrices.
    const float* const Lm = tall ? Rv : Lv;   // factor indexed by the canonical row
    const float* const Ln = tall ? Lv : Rv;   // factor indexed by the canonical column
    // (Lm O Ln)^2 = Lm^2 Ln^2 O^2: four squared row factors per lane, four
    // squared column factors per (a, g).
    float lm2[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int m = row0 + ml0 + b * 32;
      const float l = m < mc ? Lm[m] : 0.f;
      lm2[b] = l * l;
    }
#pragma unroll
    for (int a = 0; a < NA; ++a) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int nl = nl0 + a * 32 + 8 * g;
        const int n = col0 + nl;
        float ln2[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float l = n + e < nc ? Ln[n + e] : 0.f;
          ln2[e] = l * l;
        }
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          const int m = row0 + ml0 + b * 32;
          uint2 pk;
          pk.x = pack_bf16x2(sc * acc[a][b][4 * g + 0], sc * acc[a][b][4 * g + 1]);
          pk.y = pack_bf16x2(sc * acc[a][b][4 * g + 2], sc * acc[a][b][4 * g + 3]);
          *reinterpret_cast<uint2*>(sto + (sr0 + b * 32) * UPD_PITCH + (sc0 + a * 32 + 8 * g) * 2) = pk;
          const float ov[4] = {bf16_lo(pk.x), bf16_hi(pk.x), bf16_lo(pk.y), bf16_hi(pk.y)};
          float rowo = 0.f, rowd = 0.f;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float q = (n + e < nc) ? ov[e] * ov[e] : 0.f;   // zero padding contributes 0 anyway
            rowo += q;
            rowd += ln2[e] * q;
          }
          if (m < mc) {
            o2 += rowo;
            d2 += lm2[b] * rowd;
          }
        }
        asm volatile("" ::: "memory");   // keep the column-factor loads of one (a, g) at a time
      }
    }
  }
  // Copy-out: TM rows x TN/8 chunks of 16 bytes; one store covers 512 / TN
  // rows.  Each chunk is read as two 8-byte halves (rows are 8-byte aligned
  // in the padded copy).  Streaming store: the next kernel reads X' from
  // another XCD's L2 anyway, and the operand panels keep this one.
  constexpr int SCH = TN * 2 / 16;   // chunks per staged row
  static_assert(TM * SCH % 64 == 0, "whole stores per wave");
#pragma unroll
  for (int it = 0; it < TM * SCH / 64; ++it) {
    const int q = lane + 64 * it;
    const int r = q / SCH, ch = q % SCH;
    const char* src = sto + r * UPD_PITCH + ch * 16;
    const uint2 lo = *reinterpret_cast<const uint2*>(src);
    const uint2 hi = *reinterpret_cast<const uint2*>(src + 8);
    const u32x4 v = {lo.x, lo.y, hi.x, hi.y};
    __builtin_nontemporal_store(
        v, reinterpret_cast<MALT_GLOBAL u32x4*>(gptr(Xn) + (size_t)(row0 + wr * TM + r) * np + col0 + wc * TN + ch * 8));
  }
  if (!args.last) return;
  // Deterministic per-tile sums for the graft norms (LDS past the staged sub-tiles).
  float* red = reinterpret_cast<float*>(lds + UPD_RED);
  o2 = wsum(o2);
  d2 = wsum(d2);
  if (lane == 0) {
    red[wave] = o2;
    red[NW + wave] = d2;
  }
  __syncthreads();
  if (tid == 0) {
    float so = 0.f, sd = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      so += red[w];
      sd += red[NW + w];
    }
    gpart[2 * (size_t)t.idx + 0] = so;
    gpart[2 * (size_t)t.idx + 1] = sd;
  }
}

#endif

// Each kernel uses more dynamic LDS than the default limit; the attribute is
// set for the current device (plan set-up calls ns_gemm_setup with the plan's
// device current, so every device a plan runs on has it).
#ifdef MALT_NS_UPDATE_TU
hipError_t ns_update_setup() {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&ns_update_kernel),
                             hipFuncAttributeMaxDynamicSharedMemorySize, LDS_BYTES);
}

hipError_t launch_ns_update(const NsArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(ns_update_kernel, dim3(a.ntiles), dim3(NT), LDS_BYTES, s, a);
  return hipGetLastError();
}
#else
hipError_t ns_gemm_setup() {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&ns_gemm_sym_kernel),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, LDS_BYTES);
  if (e == hipSuccess) e = ns_update_setup();
  return e;
}

hipError_t launch_ns_gemm(const NsArgs& a, hipStream_t s) {
  if (a.ntiles == 0) return hipSuccess;
  if (a.phase == PH_UPDATE) return launch_ns_update(a, s);
  hipLaunchKernelGGL(ns_gemm_sym_kernel, dim3(a.ntiles), dim3(NT), LDS_BYTES, s, a);
  return hipGetLastError();
}
#endif

}  // namespace malt
