// Gram and polynomial phases of Newton-Schulz (Muon's quintic, the Orth step
// of Sec. 3.1) on the canonical X (mp x np, rows <= cols, zero-padded to
// multiples of 256), each one grouped launch over every matrix of the step:
//   Gram        A  = s X X^T                 NT product, symmetric: upper tiles
//                                            only, mirrored on write; s = sigma^2
//                                            on the first iteration, else 1
//   Polynomial  B' = a I + b A + c A A^T     NT product (A is symmetric, so
//                                            A A = A A^T); upper tiles, mirrored
// The update X' = s B' X (ns_update.hip) then needs no addend: a X is folded
// into B', so every iteration applies one rounded matrix to one rounded X.
// A and B' are bf16 (round to nearest even).  One kernel template, one
// instance per phase, each compiled for its own phase only and with its own
// pipeline geometry (both 64-k stages in a two-slot ring: the Gram contracts
// over K = n', up to 80 stages, and gains from the fewer barriers).
#include "ns_common.h"

namespace malt {

using namespace ns;

namespace {

// Epilogue staging.  A diagonal tile stages the whole bf16 tile in LDS and
// writes it out in 512-byte rows: written column-wise (each lane: four
// consecutive rows of one column, 8 bytes into one staged row), rows padded by
// 16 bytes so the 16 staged rows and two row groups of a half-wave's write
// land in distinct banks; written row-wise (each lane: four consecutive
// columns), rows padded by 64 bytes.  Off-diagonal tiles go through per-wave
// regions: the sub-tile transposed (TN rows of TM bf16, padded by 16 bytes),
// then as is (TM rows of TN bf16, unpadded, the 32-byte column units of a row
// rotated by its row pair).
constexpr int ST_PITCH_T = NS_TILE * 2 + 16;
constexpr int ST_PITCH_R = NS_TILE * 2 + 64;
constexpr int SYM_PITCH_T = TM * 2 + 16;
constexpr int SYM_WAVE = TN * SYM_PITCH_T > TM * TN * 2 ? TN * SYM_PITCH_T : TM * TN * 2;
constexpr int SYM_EPI_BYTES = NS_TILE * ST_PITCH_R;
template <class G>
struct SymLds {
  static constexpr int BYTES = G::RING_BYTES > SYM_EPI_BYTES ? G::RING_BYTES : SYM_EPI_BYTES;
  static_assert(BYTES <= 160 * 1024, "LDS budget");
  static_assert(NW * SYM_WAVE <= BYTES, "per-wave epilogue regions");
};

}  // namespace

// ===========================================================================
// Gram and polynomial phases: C = P Q^T, symmetric output, upper tiles.
// ===========================================================================
// G is the stage geometry of the phase's pipeline (SymGeom for the Gram,
// PolyGeom for the polynomial), PHASE the phase.
template <class G, int PHASE>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(WPE, WPE)))
void ns_gemm_sym_kernel(NsArgs args) {
  constexpr int I = TM / 16, J = TN / 16;    // 16x16 blocks per wave
  static_assert(G::KSUB == 32, "v_mfma_f32_16x16x32_bf16 sub-steps");

  extern __shared__ __attribute__((aligned(16))) char lds[];
  // Every descriptor field the tile needs is read here, before any store, so
  // the uniform loads go through the scalar cache.
  // The work list is in dispatch order (XCD-balanced on the host); entries
  // with mat < 0 pad the shorter XCD runs.
  const Tile t = args.tiles[blockIdx.x];
  if (t.mat < 0) return;
  const MatDesc* __restrict__ d = args.desc + t.mat;
  constexpr int phase = PHASE;
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

  // Polynomial with c != 0: B' = c (A A^T + (b/c) A) + a I, the (b/c) A term
  // added to the accumulators inside the main loop (below).  With c = 0 the
  // epilogue reloads A's tile instead.
  const bool fuse = phase == PH_POLY && args.c != 0.f;
  const float beta = fuse ? args.b / args.c : 0.f;

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // Sub-tile of each wave. On a diagonal tile only the 16 x 16 blocks on or
  // above the block diagonal are computed (the others are their mirrors). The
  // two waves that share a SIMD (waves w and w + 4) then take sub-tiles with
  // 32 + 0, 32 + 0, 26 + 10 and 10 + 26 such blocks, instead of the 10 + 0,
  // 26 + 0, 32 + 10 and 32 + 26 of the plain order, so every matrix core gets
  // a share.
  const int role = diag ? ((0x76540132u >> (4 * wave)) & 0xF) : wave;
  const int wr = role / (NW / 2), wc = role % (NW / 2);

  f32x4 acc[I][J];
#pragma unroll
  for (int i = 0; i < I; ++i)
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[i][j][e] = 0.f;
  const i32x4 rsP = buf_rsrc(P);

  // Off-diagonal tiles and the four block patterns of diagonal tiles run
  // separate copies of the main loop, so no copy tests blocks at run time, and
  // each tile kind has its own ring geometry: G for off-diagonal tiles,
  // DiagGeom<SymGeom> (64-k stages of the row panel alone, four in the ring)
  // for diagonal ones.
  auto main_loop = [&](auto diag_tag, auto d_tag) {
    constexpr bool DIAG = decltype(diag_tag)::value;
    // Diagonal tiles compute block (i, j) of the wave's sub-tile when
    // i <= j + D, D = (wc TN - wr TM) / 16: a compile-time pattern per wave,
    // so the skipped MFMAs cost no branch.
    constexpr int D = decltype(d_tag)::value;
    using PG = std::conditional_t<DIAG, DiagGeom<SymGeom>, G>;
    using PL = SymLoads<std::conditional_t<DIAG, SymGeom, G>>;
    constexpr int H = PG::H, NL = PG::LOADS;
    // Direct-load sources: load g < LOADS_PER_OPER covers rows of the tile-row
    // panel, the rest rows of the tile-column panel (both of P); 32-bit byte
    // offsets into P's buffer (SymLoads, shared with the host bounds check).
    // With 8 waves, g = wave + 8q < LOADS_PER_OPER exactly for q < LOADS / 2:
    // the first half of a wave's loads are row-panel loads (SymLoads asserts
    // it), and a diagonal tile issues those only.
    uint32_t voff[NL];
    int dst_off[NL];
#pragma unroll
    for (int q = 0; q < NL; ++q) {
      const int g = wave + q * NW;
      voff[q] = (uint32_t)PL::voff(g, lane, row0, col0, ld);
      dst_off[q] = PL::dst(g);
    }
    // MFMA operands: lane l holds k = 8 (l / 16) .. + 7 of row l % 16 of its
    // block; a sub-step of 32 k spans chunks 4h .. 4h + 3.  The swizzle
    // repeats every RPP * CPR rows, so block i sits 16 i rows below block 0.
    static_assert(16 % (PG::RPP * PG::CPR) == 0, "16-row blocks keep the swizzle phase");
    int offa[H], offb[H];
#pragma unroll
    for (int h = 0; h < H; ++h) {
      const int kc = 4 * h + (lane >> 4);
      offa[h] = PG::swz_rk(wr * TM + (lane & 15), kc);
      offb[h] = (DIAG ? 0 : PG::OPER_BYTES) + PG::swz_rk(wc * TN + (lane & 15), kc);
    }
    // The (b/c) A term of the polynomial.  A is symmetric, so the entry
    // A(r, c) of accumulator position (r, c) is k = r of the tile-column
    // panel's row c: the stage holding k = row0 + wr TM .. + 63 has block rows
    // 0..3 of the wave's sub-tile, the next stage block rows 4..7, and each
    // lane's four consecutive rows of one column are 8 contiguous bytes.  The
    // first stage is read in its first sub-step and the second in its second,
    // each before the next sub-step's fragment reads, whose registers are
    // still free there.
    static_assert(PG::BK == 64 && 4 * 16 == PG::BK, "four block rows per stage");
    const int kta = fuse ? (row0 + wr * TM) / PG::BK : -2;
    auto add_a = [&](auto s_tag, const char* st) {
      constexpr int S = decltype(s_tag)::value;
      // Offsets formed here from a copy of the lane id the compiler cannot
      // hoist: the main loop has no registers to keep them in.
      int l = lane;
      asm volatile("" : "+v"(l));
      // Two block rows at a time (16 registers of values).
#pragma unroll
      for (int i0 = 0; i0 < 4; i0 += 2) {
        uint2 w[2][J];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const int ao = (DIAG ? 0 : PG::OPER_BYTES) + wc * TN * PG::RB +
                         PG::swz_rk(l & 15, 2 * (i0 + i) + (l >> 5)) + ((l >> 4) & 1) * 8;
#pragma unroll
          for (int j = 0; j < J; ++j) w[i][j] = *reinterpret_cast<const uint2*>(st + ao + j * 16 * PG::RB);
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < J; ++j)
            if (!DIAG || 4 * S + i0 + i <= j + D) {
              f32x4& a = acc[4 * S + i0 + i][j];
              a[0] = fmaf(beta, __uint_as_float(w[i][j].x << 16), a[0]);
              a[1] = fmaf(beta, __uint_as_float(w[i][j].x & 0xffff0000u), a[1]);
              a[2] = fmaf(beta, __uint_as_float(w[i][j].y << 16), a[2]);
              a[3] = fmaf(beta, __uint_as_float(w[i][j].y & 0xffff0000u), a[3]);
            }
      }
    };
    bf16x8 fa[2][I], fb[2][J];
    // Burst stages (off-diagonal tiles) issue all their loads among the MFMAs
    // after the barrier.
    pipeline<PG, 1, PG::LOADS>(
        K / PG::BK, NL, lds,
        [&](int kt, int i) {
          dma16(rsP, voff[i], (uint32_t)PL::soff(kt),
                lds_u32(lds + (kt % PG::STAGES) * PG::STAGE_BYTES + dst_off[i]));
        },
        [&](int buf, const char* st, int h) {
#pragma unroll
          for (int i = 0; i < I; ++i) fa[buf][i] = *reinterpret_cast<const bf16x8*>(st + offa[h] + i * 16 * PG::RB);
#pragma unroll
          for (int j = 0; j < J; ++j) fb[buf][j] = *reinterpret_cast<const bf16x8*>(st + offb[h] + j * 16 * PG::RB);
        },
        [&](int kt, int h, const char* st) {
          if constexpr (PHASE == PH_POLY && !(DIAG && D < 0)) {
            // One test per sub-step: nested tests of the stage would make
            // the compiler copy the accumulators between branches.
            if (h == 0 && kt == kta) add_a(std::integral_constant<int, 0>{}, st);
            if (h == 1 && kt == kta + 1) add_a(std::integral_constant<int, 1>{}, st);
          }
        },
        [&](int buf, auto&& after) {
#pragma unroll
          for (int i = 0; i < I; ++i)
#pragma unroll
            for (int j = 0; j < J; ++j) {
              // Diagonal tiles skip the blocks below the block diagonal.
              if (!DIAG || i <= j + D)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[buf][i], fb[buf][j], acc[i][j], 0, 0, 0);
              after(i * J + j);
            }
        });
  };
  if (!diag) {
    main_loop(std::false_type{}, std::integral_constant<int, 0>{});
  } else {
    static_assert(TM == 2 * TN && TM / 16 == 8, "the four block patterns of a diagonal tile");
    // d = -8, -4: no block; 0: the upper triangle; 4: all but the 6 blocks of
    // the lower-left corner; 8, 12: every block.
    const int d = (wc * TN - wr * TM) / 16;
    if (d < 0) main_loop(std::true_type{}, std::integral_constant<int, -8>{});
    else if (d == 0) main_loop(std::true_type{}, std::integral_constant<int, 0>{});
    else if (d == 4) main_loop(std::true_type{}, std::integral_constant<int, 4>{});
    else main_loop(std::true_type{}, std::integral_constant<int, 8>{});
  }

  // ---------------------------------------------------------------- epilogue
  // acc[i][j][e] = C(r, c): tile row r = wr*TM + i*16 + 4*(lane >> 4) + e,
  // tile column c = wc*TN + j*16 + (lane & 15), so each lane holds four
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
  const int rl0 = wr * TM + 4 * (lane >> 4);   // tile row of i = e = 0
  const int cl0 = wc * TN + (lane & 15);       // tile column of j = 0

  __syncthreads();   // every wave is done reading the operand ring
  if (poly && !fuse) {
    // c = 0: B' = a I + b A + c A A^T takes A(r, c) at each accumulator
    // position. A's tile goes to LDS as 256 rows in the [k][n] layout (direct
    // loads), and each lane reads its four rows of one column with one
    // transposed read per (i, j).
    const i32x4 rsA = buf_rsrc(Am);
#pragma unroll
    for (int it = 0; it < NS_TILE * NS_TILE * 2 / (16 * NT); ++it) {
      const int c = tid + NT * it;   // 16-byte chunk of the tile; physical chunk c & 31 of
                                     // row c >> 5 holds logical chunk (c & 31) ^ 4 (row & 3)
      dma16(rsA, (uint32_t)poly_a_tile_off(c, row0, col0, mp), 0u, lds_u32(lds + (c - lane) * 16));
    }
    wait_vm_c<0>();
    __syncthreads();
  }
  uint2 hv[I][J];
  {
    const int r = (lane & 15) >> 2, q = lane & 3;
#pragma unroll
    for (int i = 0; i < I; ++i)
#pragma unroll
      for (int j = 0; j < J; ++j) {
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[i][j][e];
        if (poly) {
          const int k0 = rl0 + i * 16;
          const int R = row0 + k0, C = col0 + cl0 + j * 16;
          if (fuse) {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = args.c * v[e] + (R + e == C ? args.a : 0.f);
          } else {
            // In each 16-lane group (one row group, sixteen columns) lane
            // q + 4r addresses row k0 + r, columns n0 + 4q .. n0 + 4q + 3.
            const int n0 = wc * TN + j * 16;
            const i16x4 av =
                __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)(lds + swz_kn<2>(k0 + r, n0 + 4 * q)));
#pragma unroll
            for (int e = 0; e < 4; ++e)
              v[e] = args.b * bf2f_((bf16_t)av[e]) + args.c * v[e] + (R + e == C ? args.a : 0.f);
          }
        }
        hv[i][j].x = pack_bf16x2(sc * v[0], sc * v[1]);
        hv[i][j].y = pack_bf16x2(sc * v[2], sc * v[3]);
        if (lo_off) {
          // Keep the low parts in acc (its values are no longer needed).
          acc[i][j][0] = sc * v[0] - bf16_lo(hv[i][j].x);
          acc[i][j][1] = sc * v[1] - bf16_hi(hv[i][j].x);
          acc[i][j][2] = sc * v[2] - bf16_lo(hv[i][j].y);
          acc[i][j][3] = sc * v[3] - bf16_hi(hv[i][j].y);
        }
      }
  }

  // Row-wise copy of accumulator group (i, j, g): a 4 x 4 transpose of
  // 16-bit values inside each lane quad, after which lane p of the quad holds
  // row p of the quad's four rows, its four columns.
  const int p = lane & 3;
  auto quad_rows = [&](int i, int j) {
    const uint32_t A0 = hv[i][j].x, B0 = hv[i][j].y;   // rows (0,1), (2,3) of column p
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
            *reinterpret_cast<uint2*>(wreg + ((lane & 15) + j * 16) * SYM_PITCH_T + (4 * (lane >> 4) + i * 16) * 2) =
                hv[i][j];
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
        // As is: 128-byte rows of four 32-byte column units (j); unit j of
        // row r sits at j ^ ((r >> 1) & 3), so the eight rows and four quads
        // of a half-wave's write land in distinct banks.
#pragma unroll
        for (int i = 0; i < I; ++i)
#pragma unroll
          for (int j = 0; j < J; ++j) {
            const int r = 4 * (lane >> 4) + i * 16 + p;
            const int u = j ^ ((r >> 1) & 3);
            *reinterpret_cast<uint2*>(wreg + r * (TN * 2) + u * 32 + (((lane & 15) >> 2) << 3)) = quad_rows(i, j);
          }
        constexpr int DCH = TN * 2 / 16;
#pragma unroll
        for (int it = 0; it < TM * DCH / 64; ++it) {
          const int q = lane + 64 * it;
          const int r = q / DCH, ch = q % DCH;
          const int u = (ch >> 1) ^ ((r >> 1) & 3);
          const u32x4 v = *reinterpret_cast<const u32x4*>(wreg + r * (TN * 2) + u * 32 + (ch & 1) * 16);
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
        const int br = (wr * TM) / 16 + i, bc = (wc * TN) / 16 + j;   // wave-uniform block coordinates
        if (!diag || br <= bc)
          *reinterpret_cast<uint2*>(lds + (cl0 + j * 16) * ST_PITCH_T + (rl0 + i * 16) * 2) = hv[i][j];
        if (diag && br < bc) {
          const int rr = rl0 + i * 16 + p;
          const int cc = wc * TN + j * 16 + ((lane & 15) & ~3);
          *reinterpret_cast<uint2*>(lds + rr * ST_PITCH_T + cc * 2) = quad_rows(i, j);
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
      for (int j = 0; j < J; ++j) {
        const int rr = rl0 + i * 16 + p;
        const int cc = wc * TN + j * 16 + ((lane & 15) & ~3);
        *reinterpret_cast<uint2*>(lds + rr * ST_PITCH_R + cc * 2) = quad_rows(i, j);
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
      for (int j = 0; j < J; ++j) {
        hv[i][j].x = pack_bf16x2(acc[i][j][0], acc[i][j][1]);
        hv[i][j].y = pack_bf16x2(acc[i][j][2], acc[i][j][3]);
      }
    emit(lo_off);
  }
}


// The kernels use more dynamic LDS than the default limit; the attribute is
// set for the current device (plan set-up calls ns_gemm_setup with the plan's
// device current, so every device a plan runs on has it).
hipError_t ns_gemm_setup() {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&ns_gemm_sym_kernel<SymGeom, PH_GRAM>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, SymLds<SymGeom>::BYTES);
  if (e == hipSuccess)
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(&ns_gemm_sym_kernel<PolyGeom, PH_POLY>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, SymLds<PolyGeom>::BYTES);
  if (e == hipSuccess) e = ns_update_setup();
  return e;
}

hipError_t launch_ns_gemm(const NsArgs& a, hipStream_t s) {
  if (a.ntiles == 0) return hipSuccess;
  if (a.phase == PH_UPDATE) return launch_ns_update(a, s);
  if (a.phase == PH_GRAM)
    hipLaunchKernelGGL((ns_gemm_sym_kernel<SymGeom, PH_GRAM>), dim3(a.ntiles), dim3(NT), SymLds<SymGeom>::BYTES, s,
                       a);
  else
    hipLaunchKernelGGL((ns_gemm_sym_kernel<PolyGeom, PH_POLY>), dim3(a.ntiles), dim3(NT), SymLds<PolyGeom>::BYTES, s,
                       a);
  return hipGetLastError();
}

}  // namespace malt
