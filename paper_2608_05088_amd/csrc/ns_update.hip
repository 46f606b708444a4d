// Update phase of Newton-Schulz: X' = s B' X (NN), s = sigma on the first
// iteration, with B' = a I + b A + c A A from the polynomial phase
// (ns_sym.hip).  Computed as C^T = X^T B'^T blocks, so every lane holds four
// consecutive output columns of one row.  X is read as a row-major [k][n]
// stage tile through transposed LDS reads.  The last iteration also writes
// the per-tile sums of O^2 and (L O R)^2 for the grafting norms.
// v_mfma_f32_16x16x32_bf16 on 16 x 16 blocks, in stages of 64 k (two 32-k
// sub-steps) in a two-slot ring.
#include "ns_common.h"

namespace malt {

using namespace ns;

namespace {

using G = UpdGeom;
using L = UpdLoads<G>;
constexpr int BK = G::BK, STAGES = G::STAGES, H = G::H, RB = G::RB, CPR = G::CPR, RPP = G::RPP;
constexpr int OPER_BYTES = G::OPER_BYTES, STAGE_BYTES = G::STAGE_BYTES, LOADS = G::LOADS;
__device__ __forceinline__ int swz_rk(int row, int kc) { return G::swz_rk(row, kc); }

// Epilogue: each wave stages its own TM x TN sub-tile in a region of its own,
// rows padded by 8 bytes, and keeps its per-tile norm partials past the NW
// regions.
constexpr int UPD_PITCH = TN * 2 + 8;
constexpr int UPD_WAVE = TM * UPD_PITCH;
constexpr int UPD_RED = NW * UPD_WAVE;
constexpr int UPD_EPI_BYTES = UPD_RED + 2 * NW * 4;
constexpr int LDS_BYTES = G::RING_BYTES > UPD_EPI_BYTES ? G::RING_BYTES : UPD_EPI_BYTES;
static_assert(LDS_BYTES <= 160 * 1024, "LDS budget");

}  // namespace

// ===========================================================================
// Update phase: X' = s B' X  (NN), computed as C^T = X^T B'^T blocks.
// ===========================================================================
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(WPE, WPE)))
void ns_update_kernel(NsArgs args) {
  constexpr int NB = TM / 16;                // B' fragments (output rows, MFMA B operand)
  constexpr int NA = TN / 16;                // X fragments (output cols, MFMA A operand)

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

  // wave is read as uniform, so each direct load's LDS address (m0) is scalar
  // arithmetic, not a vector add and a readfirstlane per load.
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave / (NW / 2), wc = wave % (NW / 2);

  // Direct-load sources as 32-bit byte offsets into the B' and X buffers
  // (UpdLoads, shared with the host bounds check): load g < LOADS_P covers B'
  // rows, the rest X k-rows of the tile.  With 8 waves, g = wave + 8q < LOADS_P
  // exactly for q < LOADS / 2, so which operand a load reads is known at
  // compile time.
  const i32x4 rsB = buf_rsrc(Bm);
  const i32x4 rsX = buf_rsrc(X);
  uint32_t voff[LOADS];
  int dst_off[LOADS];
#pragma unroll
  for (int q = 0; q < LOADS; ++q) {
    const int g = wave + q * NW;
    voff[q] = (uint32_t)(q < LOADS / 2 ? L::voff_b(g, lane, row0, ldb) : L::voff_x(g, lane, col0, np));
    dst_off[q] = L::dst(g);
  }
  // MFMA operands (16 x 32 and 32 x 16): lane l holds k = 8 (l / 16) .. + 7
  // of row / column l % 16 of its block.
  // B' fragments: rows of the output, k contiguous.  The swizzle repeats
  // every RPP * CPR rows, so block b sits 16 b rows below block 0.
  static_assert(16 % (RPP * CPR) == 0, "16-row blocks keep the swizzle phase");
  int offb[H];
#pragma unroll
  for (int h = 0; h < H; ++h) offb[h] = swz_rk(wr * TM + (lane & 15), 4 * h + (lane >> 4));
  // X fragments through transposed reads: in each 16-lane group, lane
  // j = q + 4r addresses row k0 + r, columns n0 + 4q .. n0 + 4q + 3; the
  // read hands lane i the four rows of column n0 + i.  Group l / 16 reads k
  // rows 8 (l / 16) .. + 7 in two such reads.
  int offx[NA][2];
  {
    const int r = (lane & 15) >> 2, q = lane & 3;
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int r2 = 0; r2 < 2; ++r2) {
        const int k = 8 * (lane >> 4) + 4 * r2 + r;
        const int n = wc * TN + a * 16 + 4 * q;
        offx[a][r2] = OPER_BYTES + swz_kn<3>(k, n);
      }
  }

  f32x4 acc[NA][NB];
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[a][b][e] = 0.f;
  bf16x8 fx[2][NA], fb[2][NB];

  // X stages (from further away) are issued right after each barrier, B'
  // stages (L2-resident panels) from among the MFMAs that follow it.
  pipeline<G, 1, LOADS / 2>(
      K / BK, LOADS, lds,
      [&](int kt, int q) {   // q < LOADS / 2: B' rows, else X k-rows
        const uint32_t la = lds_u32(lds + (kt % STAGES) * STAGE_BYTES + dst_off[q]);
        if (q < LOADS / 2) dma16(rsB, voff[q], (uint32_t)L::soff_b(kt), la);
        else dma16(rsX, voff[q], (uint32_t)L::soff_x(kt, mp, np), la);   // X's k wraps for split matrices
      },
      [&](int buf, const char* st, int h) {
#pragma unroll
        for (int b = 0; b < NB; ++b) fb[buf][b] = *reinterpret_cast<const bf16x8*>(st + offb[h] + b * 16 * RB);
#pragma unroll
        for (int a = 0; a < NA; ++a) {
          const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_i16x4_t*)(st + offx[a][0] + h * 32 * KN_ROW));
          const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_i16x4_t*)(st + offx[a][1] + h * 32 * KN_ROW));
          fx[buf][a] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        }
      },
      [](int, int, const char*) {},
      [&](int buf, auto&& after) {
#pragma unroll
        for (int a = 0; a < NA; ++a)
#pragma unroll
          for (int b = 0; b < NB; ++b) {
            acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fx[buf][a], fb[buf][b], acc[a][b], 0, 0, 0);
            after(a * NB + b);
          }
      });

  // ---------------------------------------------------------------- epilogue
  // acc[a][b][e] = C(m, n + e), m = row0 + wr*TM + b*16 + (lane & 15),
  // n = col0 + wc*TN + a*16 + 4*(lane >> 4): four consecutive bf16 per lane.
  // Each wave copies its own TM x TN sub-tile to a private LDS region and
  // writes it out in whole 128-byte row pieces, not as 8-byte pieces of 16
  // rows.  A wave reads back only what it staged, so no barrier separates
  // the two and each wave leaves the epilogue at its own pace.
  const int ml0 = wr * TM + (lane & 15);          // tile-local row of b = 0
  const int nl0 = wc * TN + 4 * (lane >> 4);      // tile-local column of a = 0
  const int sr0 = lane & 15, sc0 = 4 * (lane >> 4);   // the same within the sub-tile
  char* const sto = lds + wave * UPD_WAVE;
  __syncthreads();   // every wave is done reading the operand ring
  float o2 = 0.f, d2 = 0.f;
  if (!args.last) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int a = 0; a < NA; ++a) {
        uint2 pk;
        pk.x = pack_bf16x2(sc * acc[a][b][0], sc * acc[a][b][1]);
        pk.y = pack_bf16x2(sc * acc[a][b][2], sc * acc[a][b][3]);
        *reinterpret_cast<uint2*>(sto + (sr0 + b * 16) * UPD_PITCH + (sc0 + a * 16) * 2) = pk;
      }
  } else {
    // Last iteration: also the per-tile sums of O^2 and (L O R)^2, from the
    // rounded O.  Canonical (m, n) is W(m, n) for wide and W(n, m) for tall
    // matrices.
    const float* const Lm = tall ? Rv : Lv;   // factor indexed by the canonical row
    const float* const Ln = tall ? Lv : Rv;   // factor indexed by the canonical column
    // (Lm O Ln)^2 = Lm^2 Ln^2 O^2: NB squared row factors per lane, four
    // squared column factors per a.
    float lm2[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int m = row0 + ml0 + b * 16;
      const float l = m < mc ? Lm[m] : 0.f;
      lm2[b] = l * l;
    }
#pragma unroll
    for (int a = 0; a < NA; ++a) {
      {
        const int nl = nl0 + a * 16;
        const int n = col0 + nl;
        float ln2[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float l = n + e < nc ? Ln[n + e] : 0.f;
          ln2[e] = l * l;
        }
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          const int m = row0 + ml0 + b * 16;
          uint2 pk;
          pk.x = pack_bf16x2(sc * acc[a][b][0], sc * acc[a][b][1]);
          pk.y = pack_bf16x2(sc * acc[a][b][2], sc * acc[a][b][3]);
          *reinterpret_cast<uint2*>(sto + (sr0 + b * 16) * UPD_PITCH + (sc0 + a * 16) * 2) = pk;
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
        asm volatile("" ::: "memory");   // keep the column-factor loads of one a at a time
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


// The kernel uses more dynamic LDS than the default limit (set per device by
// ns_gemm_setup at plan set-up).
hipError_t ns_update_setup() {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&ns_update_kernel),
                             hipFuncAttributeMaxDynamicSharedMemorySize, LDS_BYTES);
}

hipError_t launch_ns_update(const NsArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(ns_update_kernel, dim3(a.ntiles), dim3(NT), LDS_BYTES, s, a);
  return hipGetLastError();
}

}  // namespace malt
