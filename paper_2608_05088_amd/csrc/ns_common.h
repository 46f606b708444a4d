// Shared machinery of the grouped Newton-Schulz GEMMs on the gfx950 matrix
// cores (bf16 operands, fp32 accumulation): the tile geometry, operand
// addressing, direct-to-LDS loads and the software pipeline.  The symmetric
// Gram / polynomial kernel (ns_sym.hip) and the update kernel (ns_update.hip)
// each instantiate the pipeline with their own stage geometry (NsGeom).
//
// Every kernel: one 256 x 256 output tile per workgroup of 8 waves (2 per
// SIMD), each wave owning a 128 x 64 sub-tile as 16x16 blocks of
// v_mfma_f32_16x16x32_bf16 (under the chip's power budget this shape sustains
// a higher rate than 32x32x16 with random operands).  Operand stages of BK
// k-values stream from global memory straight into an LDS ring (buffer_load
// ... lds, 16 bytes per lane), STAGES deep, one barrier per stage; fragments
// are double-buffered in registers so the reads for the next 32-k sub-step
// are in flight while the current one multiplies.
//
// NT operands (rows with k contiguous) use ds_read_b128 fragments from an
// XOR-swizzled [row][k] tile.  A [k][n] operand (X in the update) is read with
// ds_read_b64_tr_b16 transposed reads.
#pragma once

#include <type_traits>

#include "malt_internal.h"

namespace malt {
namespace ns {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr int NW = 8;                       // waves per workgroup
constexpr int WPE = NW / 4;                 // waves per SIMD
constexpr int NT = NW * 64;                 // threads per workgroup
constexpr int KN_ROW = NS_TILE * 2;         // bytes per [k][n] tile row (512)
// Wave grid 2 x (NW / 2): each wave owns TM x TN of the 256 x 256 tile.
constexpr int TM = NS_TILE / 2, TN = NS_TILE / (NW / 2);
static_assert(TM == 128 && TN == 64, "the epilogues assume 128 x 64 wave sub-tiles");

// Stage geometry of one kernel's pipeline: BK k-values per stage, a ring of
// STAGES stage slots in LDS, sub-steps of KSUB k-values, one MFMA k-step: 16
// for v_mfma_f32_32x32x16_bf16 (32 x 32 blocks), 32 for
// v_mfma_f32_16x16x32_bf16 (16 x 16 blocks).
template <int BK_, int STAGES_, int KSUB_ = 16>
struct NsGeom {
  static constexpr int BK = BK_;
  static constexpr int STAGES = STAGES_;
  static constexpr int KSUB = KSUB_;
  static constexpr int H = BK / KSUB;                         // MFMA sub-steps per stage
  static constexpr int BLK = KSUB == 16 ? 32 : 16;            // output block edge of one MFMA
  static constexpr int NMMA = (TM / BLK) * (TN / BLK);        // MFMAs per wave per sub-step
  static_assert(KSUB == 16 || KSUB == 32, "the two bf16 MFMA shapes");
  static constexpr int RB = BK * 2;                           // bytes per [row][k] tile row
  static constexpr int CPR = BK / 8;                          // 16-byte chunks per [row][k] row
  static constexpr int RPP = 256 / RB;                        // [row][k] rows per 256-byte bank period
  static constexpr int OPER_BYTES = NS_TILE * BK * 2;         // one operand tile of one stage
  static constexpr int STAGE_BYTES = 2 * OPER_BYTES;
  static constexpr int RING_BYTES = STAGES * STAGE_BYTES;
  static constexpr int LOADS = 2 * OPER_BYTES / 1024 / NW;    // 1 KB direct loads per wave per stage
  // Spread (three or more slots): a stage's loads go out between the MFMAs of
  // the stage STAGES - 1 ahead of it; burst (two slots): all at the barrier.
  static constexpr bool SPREAD = STAGES >= 3;
  static_assert(H % 2 == 0, "sub-steps per stage must be even");
  static_assert(LOADS * NW * 1024 == 2 * OPER_BYTES, "loads must split evenly over the waves");

  // [row][k] tile (NT operands): 256 rows x BK bf16, CPR 16-byte chunks per
  // row, chunk kc stored at kc ^ ((row / RPP) % CPR): the ds_read_b128
  // fragment reads of 16 consecutive rows at one chunk hit 16 distinct 4-bank
  // groups.
  __host__ __device__ static constexpr int swz_rk(int row, int kc) {
    return row * RB + ((kc ^ ((row / RPP) % CPR)) << 4);
  }
};

// [k][n] tile: rows of 256 bf16 (512 bytes), 16-byte chunk c stored at
// swz_chunk<GB>(k, c) = c ^ 4 (k & 3) ^ 2 (bit GB of k): the 16 lanes of one
// transposed read (four rows x 32 contiguous bytes) hit 16 distinct 4-bank
// groups, and the second 16-lane group of a half-wave, whose rows differ from
// the first's in bit GB and whose columns are the same, hits the other 16.
// GB = 3 for the update's X stages (the two groups read k-rows 8 apart), 2
// for the polynomial's A tile (4 apart).
template <int GB>
__host__ __device__ constexpr int swz_chunk(int k, int c) {
  return c ^ (4 * (k & 3)) ^ (2 * ((k >> GB) & 1));
}
template <int GB>
__host__ __device__ constexpr int swz_kn(int k, int n) {
  return k * KN_ROW + (swz_chunk<GB>(k, n >> 3) << 4) + ((n & 7) << 1);
}

// Diagonal tiles of the symmetric products load one operand panel per stage
// (their row and column panels are the same rows), half of a stage of G: the
// same LDS ring holds twice as many of their stages, so they keep three stages
// of loads in flight instead of one (spread between the MFMAs).
template <class G>
struct DiagGeom : G {
  static constexpr int STAGES = 2 * G::STAGES;
  static constexpr int STAGE_BYTES = G::OPER_BYTES;
  static constexpr int RING_BYTES = STAGES * STAGE_BYTES;
  static constexpr int LOADS = G::LOADS / 2;
  static constexpr bool SPREAD = STAGES >= 3;
  static_assert(RING_BYTES == G::RING_BYTES, "a diagonal tile's ring is the same LDS");
};

// The stage geometries of the kernels.
using SymGeom = NsGeom<64, 2, 32>;    // Gram (ns_sym.hip)
using PolyGeom = NsGeom<64, 2, 32>;   // polynomial (ns_sym.hip)
using UpdGeom = NsGeom<64, 2, 32>;   // update (ns_update.hip)

// ---------------------------------------------------------------------------
// Operand addressing of the direct loads, shared by the kernels and the
// host-side bounds check.  A stage's 1 KB loads are numbered g = wave + q NW;
// lane `lane` of load g reads 16 bytes at byte offset voff(g, lane) + soff(kt)
// from its operand buffer (both 64-bit here; the kernels pass them as the
// 32-bit buffer offsets, which the bounds check proves to fit).
// ---------------------------------------------------------------------------

// Gram / polynomial: loads g < LOADS_PER_OPER cover rows of the tile-row
// panel (rows row0 ..), the rest rows of the tile-column panel (col0 ..), both
// of the [row][k] operand P (row pitch ld elements).
template <class G>
struct SymLoads {
  static constexpr int ROWS_PER_LOAD = 1024 / G::RB;
  static constexpr int LOADS_PER_OPER = NS_TILE / ROWS_PER_LOAD;
  static_assert(LOADS_PER_OPER == (G::LOADS / 2) * NW, "row-panel loads are the first half of each wave's");
  __host__ __device__ static constexpr uint64_t voff(int g, int lane, int row0, int col0, int ld) {
    return ((uint64_t)(((g / LOADS_PER_OPER) ? col0 : row0) + (g % LOADS_PER_OPER) * ROWS_PER_LOAD + lane / G::CPR) *
                (uint64_t)ld +
            (uint64_t)(((lane % G::CPR) ^ ((((g % LOADS_PER_OPER) * ROWS_PER_LOAD + lane / G::CPR) / G::RPP) % G::CPR)) *
                       8)) *
           2;
  }
  __host__ __device__ static constexpr uint64_t soff(int kt) { return (uint64_t)kt * G::BK * 2; }
  // LDS destination of load g within a stage slot.
  __host__ __device__ static constexpr int dst(int g) {
    return (g / LOADS_PER_OPER) * G::OPER_BYTES + (g % LOADS_PER_OPER) * 1024;
  }
};

// Polynomial epilogue: A's 256 x 256 output tile (row0, col0) loaded into LDS
// in the [k][n] layout, 16-byte chunk c (0 <= c < 8192) from tile row c / 32.
__host__ __device__ constexpr uint64_t poly_a_tile_off(int c, int row0, int col0, int mp) {
  return ((uint64_t)(row0 + (c >> 5)) * (uint64_t)mp + col0 + (uint64_t)swz_chunk<2>(c >> 5, c & 31) * 8) * 2;
}

// Update: loads g < LOADS_P read rows row0 .. of B' (row pitch ldb, [row][k]),
// the rest k-rows of X (row pitch np, columns col0 .., the [k][n] layout).
// Split matrices contract over [B'_hi | B'_lo] and [X ; X]: X's k wraps at mp.
template <class G>
struct UpdLoads {
  static constexpr int ROWS_PER_LOAD = 1024 / G::RB;      // B' rows per 1 KB load
  static constexpr int LOADS_P = NS_TILE / ROWS_PER_LOAD;
  static constexpr int KROWS_PER_LOAD = 1024 / KN_ROW;    // X k-rows per 1 KB load
  static_assert(LOADS_P == (G::LOADS / 2) * NW, "B' loads are the first half of each wave's");
  __host__ __device__ static constexpr uint64_t voff_b(int g, int lane, int row0, int ldb) {
    return ((uint64_t)(row0 + g * ROWS_PER_LOAD + lane / G::CPR) * (uint64_t)ldb +
            (uint64_t)(((lane % G::CPR) ^ (((g * ROWS_PER_LOAD + lane / G::CPR) / G::RPP) % G::CPR)) * 8)) *
           2;
  }
  __host__ __device__ static constexpr uint64_t voff_x(int g, int lane, int col0, int np) {
    return ((uint64_t)((g - LOADS_P) * KROWS_PER_LOAD + lane / 32) * (uint64_t)np + col0 +
            (uint64_t)swz_chunk<3>((g - LOADS_P) * KROWS_PER_LOAD + lane / 32, lane % 32) * 8) *
           2;
  }
  __host__ __device__ static constexpr uint64_t soff_b(int kt) { return (uint64_t)kt * G::BK * 2; }
  __host__ __device__ static constexpr uint64_t soff_x(int kt, int mp, int np) {
    return (uint64_t)(kt * G::BK >= mp ? kt * G::BK - mp : kt * G::BK) * (uint64_t)np * 2;
  }
  __host__ __device__ static constexpr int dst(int g) {
    return g < LOADS_P ? g * 1024 : G::OPER_BYTES + (g - LOADS_P) * 1024;
  }
};

typedef __attribute__((address_space(3))) i16x4 lds_i16x4_t;

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
// load moves more bytes per clock into LDS than the flat-address form.  The
// per-lane offsets are 32-bit bytes: every operand buffer (a padded canonical
// matrix, at most 2^31 bf16 elements) lies below 4 GiB of its base.
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

// Software pipeline over KT stages.
//   issue(kt, i)      the i-th direct load (0 <= i < nl) this wave issues for
//                     stage kt, into slot kt % STAGES
//   read(buf, st, h)  fragment reads of sub-step h of the stage at st into buf
//   mma(buf, after)   the MFMAs of the fragments in buf, calling after(j) once
//                     the j-th of the NMMA has been issued
//   pre(kt, h, st)    extra work of the kernel at the start of sub-step h of
//                     stage kt (slot st), before the next sub-step's fragment
//                     reads: the registers of those fragments are free here
// nl is the number of loads this wave issues per stage (LOADS, or fewer); RPM
// the LDS fragment reads placed after each MFMA.  LATE (burst only): the
// first LATE of a stage's loads go out from among the MFMAs of the sub-step
// after the barrier instead of before them, so the matrix cores restart
// first; the rest go out right after the barrier.
//
// Burst (two slots): at the barrier closing stage kt, stage kt + 1 has landed
// and every wave is done with slot kt % 2, which then receives all of stage
// kt + 2's loads.
// Spread (three or more slots): stage kt + STAGES - 1 is loaded while stage kt
// computes, its nl loads spread over the H sub-steps (nl / H per sub-step, each
// after an equal share of the MFMAs), into the slot stage kt - 1 freed.  The
// loads of STAGES - 2 stages stay in flight across every barrier, and no wave
// issues a burst of loads while its SIMD partner waits for the matrix core.
template <class G, int RPM, int LATE, class Issue, class Read, class Pre, class Mma>
__device__ __forceinline__ void pipeline(const int KT, const int nl, char* lds, Issue&& issue, Read&& read,
                                         Pre&& pre, Mma&& mma) {
  constexpr int STAGES = G::STAGES, H = G::H, LOADS = G::LOADS, STAGE_BYTES = G::STAGE_BYTES;
  constexpr bool SPREAD = G::SPREAD;
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
  constexpr int NMMA = G::NMMA;
  constexpr int GAP = PER > 0 ? NMMA / PER : 1;
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
      pre(kt, h, st);
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
          for (int i = LATE; i < LOADS; ++i)
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
        if constexpr (!SPREAD && LATE > 0 && steady) {
          // The compiler keeps the loads' order with the fragment reads (the
          // loads are asm with a memory clobber) but may move MFMAs ahead.
          if (h == H - 1 && j < LATE && j < nl) issue(kt + STAGES, j);
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

template <class G, int RPM, class Issue, class Read, class Mma>
__device__ __forceinline__ void pipeline(const int KT, const int nl, char* lds, Issue&& issue, Read&& read,
                                         Mma&& mma) {
  pipeline<G, RPM, 0>(KT, nl, lds, issue, read, [](int, int, const char*) {}, mma);
}

}  // namespace ns
}  // namespace malt
