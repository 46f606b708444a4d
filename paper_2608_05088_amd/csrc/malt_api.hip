// Host runtime of libmalt: argument validation, the per-plan layout of the
// caller's state and workspace buffers, grouped work lists, and the launch
// sequence of one MALT / MALTER step (Algorithms 1 and 2).
#include <math.h>
#include <stdarg.h>
#include <stddef.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/libmalt.h"
#include "malt_internal.h"
#include "ns_common.h"

using namespace malt;

namespace {

thread_local std::string g_last_error;

malt_status_t fail(malt_status_t st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
malt_status_t fail(malt_status_t st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

malt_status_t hip_fail(hipError_t e, const char* what) {
  return fail(MALT_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr int64_t kMaxDim = int64_t(1) << 20;        // rows or cols
constexpr int64_t kMaxShort = 32768;                   // min(rows, cols): NS Gram side
constexpr int64_t kMaxElems = (int64_t(1) << 31) - 1;  // rows * cols

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t pad_to(int64_t a, int64_t b) { return cdiv(a, b) * b; }
inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

struct MatPlan {
  int64_t m, n, mc, nc, mp, np;
  bool tall, split, small;
  int64_t sm_gchunks;                  // fp32 path: Gram partials
  int64_t k1_ct, k1_rt, k2_tr, k2_tc, k2_tiles, upd_tiles, sym_tiles;
  // offsets
  int64_t st_M, st_l, st_r, st_nu;     // floats from state base
  size_t ws_scal, ws_Lv, ws_Rv, ws_rowpart, ws_colpart, ws_k2part, ws_gpart;
  size_t ws_X[2], ws_A, ws_B;
  size_t ws_Xs[2], ws_Ap, ws_Bs;       // fp32 path only
  // algorithmic cost
  double ns_flops_sym_per_iter;        // 3 mc^2 nc + mc^3 (symmetric minimum)
};

struct Layout {
  std::vector<MatPlan> mats;
  size_t state_bytes = 0, ws_bytes = 0;
  size_t ws_desc = 0, ws_ptrs = 0;
  size_t ws_t_ew = 0, ws_t_fin = 0, ws_t_k2 = 0, ws_t_gram = 0, ws_t_poly = 0, ws_t_upd = 0;
  size_t ws_t_smg = 0, ws_t_smp = 0, ws_t_smu = 0;
  int64_t n_ew = 0, n_fin = 0, n_k2 = 0, n_sym = 0, n_upd = 0;
  int64_t n_k2w = 0;   // scale+convert tiles of wide matrices, listed before those of tall ones
  int64_t n_gram = 0, n_poly = 0, n_updd = 0;   // dispatch-ordered NS lists (padded)
  int64_t n_smg = 0, n_smp = 0, n_smu = 0;   // fp32 Newton-Schulz lists
};

malt_status_t check_shapes(const malt_shape_t* shapes, int32_t n) {
  if (n < 1) return fail(MALT_ERR_INVALID_ARG, "matrix count must be >= 1 (got %d)", n);
  if (!shapes) return fail(MALT_ERR_INVALID_ARG, "shapes is NULL");
  for (int32_t i = 0; i < n; ++i) {
    const int64_t m = shapes[i].rows, c = shapes[i].cols;
    if (m < 1 || c < 1) return fail(MALT_ERR_SHAPE, "matrix %d: rows/cols must be >= 1 (got %lld x %lld)",
                                    i, (long long)m, (long long)c);
    // The Newton-Schulz buffers are addressed with 32-bit byte offsets: the
    // canonical matrix padded to multiples of 256 must stay below 2^31 elements.
    if (m > kMaxDim || c > kMaxDim || std::min(m, c) > kMaxShort || m * c > kMaxElems ||
        pad_to(m, 256) * pad_to(c, 256) > kMaxElems)
      return fail(MALT_ERR_SHAPE, "matrix %d: %lld x %lld exceeds the supported size "
                  "(dims <= 2^20, min dim <= 32768, elements (padded to multiples of 256) < 2^31)", i,
                  (long long)m, (long long)c);
  }
  return MALT_OK;
}

// Order of matrices in the grouped work lists: larger Newton-Schulz cost first.
std::vector<int32_t> cost_order(const Layout& L) {
  std::vector<int32_t> ord(L.mats.size());
  for (size_t i = 0; i < ord.size(); ++i) ord[i] = int32_t(i);
  std::stable_sort(ord.begin(), ord.end(), [&](int32_t a, int32_t b) {
    return L.mats[a].ns_flops_sym_per_iter > L.mats[b].ns_flops_sym_per_iter;
  });
  return ord;
}

// Newton-Schulz work lists in dispatch order. Workgroup b runs on XCD
// b % NXCD and takes entry b, so the k-th tile of XCD x's run sits at
// NXCD * k + x; shorter runs are padded with mat = -1.
//
// The runs are filled matrix by matrix, largest first, each matrix going to
// the run with the least work so far (cost: 64-k pipeline stages per tile plus
// a fixed cost). Every XCD gets the same work and a mix of shapes, and a
// matrix's tiles, which share operand panels, stay together in one XCD's L2.
// A matrix holding more than 1/16 of the launch is first cut into contiguous
// pieces of at most that size, so a single large matrix still spreads over
// all XCDs.
std::vector<Tile> xcd_order(const std::vector<Tile>& list, const std::vector<double>& cost) {
  const size_t n = list.size();
  if (n == 0) return {};
  double total = 0.0;
  for (double c : cost) total += c;
  const double limit = total / (2 * NXCD);
  struct Item { size_t lo, hi; double c; };
  std::vector<Item> items;
  for (size_t lo = 0; lo < n;) {   // the list holds each matrix's tiles contiguously
    size_t hi = lo;
    double c = 0.0;
    while (hi < n && list[hi].mat == list[lo].mat) c += cost[hi++];
    // Cut [lo, hi) into `pieces` contiguous ranges of about equal cost.
    const int pieces = std::max(1, int(std::ceil(c / limit)));
    double acc = 0.0;
    size_t a = lo;
    int cut = 1;
    double pc = 0.0;
    for (size_t k = lo; k < hi; ++k) {
      acc += cost[k];
      pc += cost[k];
      if (cut < pieces && acc >= c * cut / pieces) {
        items.push_back({a, k + 1, pc});
        a = k + 1;
        pc = 0.0;
        ++cut;
      }
    }
    if (a < hi) items.push_back({a, hi, pc});
    lo = hi;
  }
  std::stable_sort(items.begin(), items.end(), [](const Item& x, const Item& y) { return x.c > y.c; });
  std::vector<size_t> runs[NXCD];
  double load[NXCD] = {0.0};
  for (const Item& it : items) {
    int best = 0;
    for (int x = 1; x < NXCD; ++x)
      if (load[x] < load[best]) best = x;
    for (size_t k = it.lo; k < it.hi; ++k) runs[best].push_back(k);
    load[best] += it.c;
  }
  size_t longest = 0;
  for (int x = 0; x < NXCD; ++x) longest = std::max(longest, runs[x].size());
  std::vector<Tile> out(NXCD * longest, Tile{-1, 0, 0, 0});
  for (int x = 0; x < NXCD; ++x)
    for (size_t k = 0; k < runs[x].size(); ++k) out[NXCD * k + x] = list[runs[x][k]];
  return out;
}

// Gram, polynomial and update lists in dispatch order (the Gram and the
// polynomial share tiles but not costs: K is n' for one and m' for the other).
void ns_dispatch_lists(const Layout& L, const std::vector<Tile>& sym, const std::vector<Tile>& upd,
                       std::vector<Tile>& gram, std::vector<Tile>& poly, std::vector<Tile>& upd_d) {
  constexpr double kTileFixed = 1.5;   // prologue + epilogue, in stages
  std::vector<double> cg(sym.size()), cp(sym.size()), cu(upd.size());
  for (size_t k = 0; k < sym.size(); ++k) {
    const MatPlan& q = L.mats[sym[k].mat];
    // A diagonal tile loads one operand panel instead of two.
    const double f = sym[k].ti == sym[k].tj ? 0.75 : 1.0;
    cg[k] = f * double(q.np) / NS_BK + kTileFixed;
    cp[k] = f * double(q.mp) / NS_BK + kTileFixed;
  }
  for (size_t k = 0; k < upd.size(); ++k) {
    const MatPlan& q = L.mats[upd[k].mat];
    cu[k] = double(q.split ? 2 * q.mp : q.mp) / NS_BK + kTileFixed;
  }
  gram = xcd_order(sym, cg);
  poly = xcd_order(sym, cp);
  upd_d = xcd_order(upd, cu);
}

void build_tiles(const Layout& L, std::vector<Tile>& ew, std::vector<Tile>& fin, std::vector<Tile>& k2,
                 std::vector<Tile>& sym, std::vector<Tile>& upd, std::vector<Tile>& smg, std::vector<Tile>& smp,
                 std::vector<Tile>& smu) {
  const std::vector<int32_t> ord = cost_order(L);
  for (int32_t i : ord) {
    const MatPlan& q = L.mats[i];
    for (int32_t ti = 0; ti < q.k1_rt; ++ti)
      for (int32_t tj = 0; tj < q.k1_ct; ++tj) ew.push_back({i, ti, tj, 0});
    for (int32_t c = 0; c < cdiv(q.m, FIN_W); ++c) fin.push_back({i, 0, c, 0});
    for (int32_t c = 0; c < cdiv(q.n, FIN_W); ++c) fin.push_back({i, 1, c, 0});
    if (q.small) {
      for (int32_t c = 0; c < q.sm_gchunks; ++c) smg.push_back({i, c, 0, 0});
      smp.push_back({i, 0, 0, 0});
      for (int32_t c = 0; c < q.upd_tiles; ++c) smu.push_back({i, c, 0, c});
      continue;
    }
    const int32_t T = int32_t(q.mp / NS_TILE), TN = int32_t(q.np / NS_TILE);
    int32_t idx = 0;
    for (int32_t ti = 0; ti < T; ++ti)
      for (int32_t tj = ti; tj < T; ++tj) sym.push_back({i, ti, tj, idx++});
    idx = 0;
    for (int32_t tj = 0; tj < TN; ++tj)       // column panel major: neighbours share X^T panels
      for (int32_t ti = 0; ti < T; ++ti) upd.push_back({i, ti, tj, idx++});
  }
  // Scale+convert: the wide matrices' tiles, then the tall ones' (two kernels).
  for (int pass = 0; pass < 2; ++pass)
    for (int32_t i : ord) {
      const MatPlan& q = L.mats[i];
      if (q.tall != (pass == 1)) continue;
      int32_t idx = 0;
      for (int32_t ti = 0; ti < q.k2_tr; ++ti)
        for (int32_t tj = 0; tj < q.k2_tc; ++tj) k2.push_back({i, ti, tj, idx++});
    }
}


Layout make_layout(const malt_shape_t* shapes, int32_t n, malt_variant_t variant) {
  Layout L;
  L.mats.resize(n);
  // State: [M... | l... | r... | nu...], float32, unpadded.
  int64_t fo = 0;
  for (int32_t i = 0; i < n; ++i) { L.mats[i].st_M = fo; fo += shapes[i].rows * shapes[i].cols; }
  for (int32_t i = 0; i < n; ++i) { L.mats[i].st_l = fo; fo += shapes[i].rows; }
  for (int32_t i = 0; i < n; ++i) { L.mats[i].st_r = fo; fo += shapes[i].cols; }
  for (int32_t i = 0; i < n; ++i) {
    if (variant == MALT_VARIANT_MALTER) { L.mats[i].st_nu = fo; fo += 1; } else { L.mats[i].st_nu = -1; }
  }
  L.state_bytes = size_t(fo) * 4;

  for (int32_t i = 0; i < n; ++i) {
    MatPlan& p = L.mats[i];
    p.m = shapes[i].rows; p.n = shapes[i].cols;
    p.tall = p.m > p.n;
    p.mc = std::min(p.m, p.n); p.nc = std::max(p.m, p.n);
    p.mp = pad_to(p.mc, NS_TILE); p.np = pad_to(p.nc, NS_TILE);
    p.small = p.mc <= NS_SMALL_MAX;
    p.split = !p.small && p.mc <= NS_SPLIT_MAX;
    p.sm_gchunks = p.small ? cdiv(p.np, SM_CH_G) : 0;
    p.k1_ct = cdiv(p.n, EW_TC); p.k1_rt = cdiv(p.m, EW_TR);
    // Scale+convert tiles over the padded W-oriented domain.
    if (p.tall) { p.k2_tr = p.np / K2_T; p.k2_tc = p.mp / K2_T; }
    else { p.k2_tr = p.mp / K2W_R; p.k2_tc = p.np / EW_TC; }
    p.k2_tiles = p.k2_tr * p.k2_tc;
    const int64_t T = p.mp / NS_TILE;
    // fp32 path: no matrix-core tiles; the update's partial slots are its
    // column chunks.
    p.sym_tiles = p.small ? 0 : T * (T + 1) / 2;
    p.upd_tiles = p.small ? p.np / SM_CH_U : T * (p.np / NS_TILE);
    p.ns_flops_sym_per_iter = 3.0 * double(p.mc) * p.mc * p.nc + double(p.mc) * p.mc * p.mc;
    L.n_ew += p.k1_rt * p.k1_ct;
    L.n_fin += cdiv(p.m, FIN_W) + cdiv(p.n, FIN_W);
    L.n_k2 += p.k2_tiles;
    if (!p.tall) L.n_k2w += p.k2_tiles;
    if (p.small) {
      L.n_smg += p.sm_gchunks;
      L.n_smp += 1;
      L.n_smu += p.upd_tiles;
    } else {
      L.n_sym += p.sym_tiles;
      L.n_upd += p.upd_tiles;
    }
  }
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t o = off; off = align256(off + bytes); return o; };
  L.ws_desc = take(sizeof(MatDesc) * n);
  L.ws_ptrs = take(sizeof(PtrPair) * n);
  L.ws_t_ew = take(sizeof(Tile) * L.n_ew);
  L.ws_t_fin = take(sizeof(Tile) * L.n_fin);
  L.ws_t_k2 = take(sizeof(Tile) * L.n_k2);
  {
    // The padded lengths of the dispatch-ordered lists depend on the costs.
    std::vector<Tile> ew, fin, k2, sym, upd, smg, smp, smu, gram, poly, updd;
    build_tiles(L, ew, fin, k2, sym, upd, smg, smp, smu);
    ns_dispatch_lists(L, sym, upd, gram, poly, updd);
    L.n_gram = int64_t(gram.size());
    L.n_poly = int64_t(poly.size());
    L.n_updd = int64_t(updd.size());
  }
  L.ws_t_gram = take(sizeof(Tile) * L.n_gram);
  L.ws_t_poly = take(sizeof(Tile) * L.n_poly);
  L.ws_t_upd = take(sizeof(Tile) * L.n_updd);
  L.ws_t_smg = take(sizeof(Tile) * L.n_smg);
  L.ws_t_smp = take(sizeof(Tile) * L.n_smp);
  L.ws_t_smu = take(sizeof(Tile) * L.n_smu);
  for (int32_t i = 0; i < n; ++i) {
    MatPlan& p = L.mats[i];
    p.ws_scal = take(sizeof(double) * MAT_SCALARS);
    p.ws_Lv = take(4 * p.m);
    p.ws_Rv = take(4 * p.n);
    p.ws_rowpart = take(4 * size_t(p.k1_ct) * p.m);
    p.ws_colpart = take(4 * size_t(p.k1_rt) * p.n);
    p.ws_k2part = take(8 * size_t(p.k2_tiles));
    p.ws_gpart = take(8 * size_t(p.upd_tiles));
    for (int b = 0; b < 2; ++b) p.ws_X[b] = take(2 * size_t(p.mp) * p.np);
    p.ws_A = take(2 * size_t(p.mp) * p.mp);
    p.ws_B = take(2 * size_t(p.mp) * p.mp * (p.split ? 2 : 1));
    if (p.small) {
      for (int b = 0; b < 2; ++b) p.ws_Xs[b] = take(4 * size_t(p.mc) * p.np);
      p.ws_Ap = take(4 * size_t(p.sm_gchunks) * NS_SMALL_MAX * NS_SMALL_MAX);
      p.ws_Bs = take(4 * size_t(NS_SMALL_MAX) * NS_SMALL_MAX);
    } else {
      p.ws_Xs[0] = p.ws_Xs[1] = p.ws_Ap = p.ws_Bs = 0;
    }
  }
  L.ws_bytes = off;
  return L;
}

bool ranges_overlap(uintptr_t a0, size_t an, uintptr_t b0, size_t bn) {
  return a0 < b0 + bn && b0 < a0 + an;
}

}  // namespace

// The workspace of plans made by malt_init_state_scratch, for callers that
// cannot allocate device memory.  Every device the library runs on holds its
// own copy until the process ends.  In host code `scratch` names a host-side
// stand-in: the device address comes from hipGetSymbolAddress, fetched once per
// device (with that device current) and kept in g_scratch_ptr.
static __device__ __align__(256) unsigned char scratch[MALT_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};
uint64_t g_scratch_gen[kMaxDevices] = {};

// The current device's scratch address and a new generation for it: a plan
// holding an older generation has lost the array to the newer plan.
malt_status_t scratch_claim(int* dev, char** ptr, uint64_t* gen) {
  hipError_t e = hipGetDevice(dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (*dev < 0 || *dev >= kMaxDevices) return fail(MALT_ERR_INVALID_ARG, "device %d out of range", *dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[*dev]) {
    void* a = nullptr;
    e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!a || reinterpret_cast<uintptr_t>(a) % 256 != 0)
      return fail(MALT_ERR_HIP, "static scratch array has no usable device address");
    g_scratch_ptr[*dev] = static_cast<char*>(a);
  }
  *ptr = g_scratch_ptr[*dev];
  *gen = ++g_scratch_gen[*dev];
  return MALT_OK;
}

bool scratch_current(int dev, uint64_t gen) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  return dev >= 0 && dev < kMaxDevices && g_scratch_gen[dev] == gen;
}

}  // namespace

struct malt_plan {
  Layout L;
  malt_variant_t variant;
  int32_t n = 0;
  std::vector<malt_shape_t> shapes;
  char* state = nullptr;
  char* ws = nullptr;
  int64_t t = 0;
  // pointer table last written to the workspace (compared on every step)
  std::vector<PtrPair> cur_ptrs;
  bool ptrs_valid = false;
  // workspace in the library's static scratch array of device `device`,
  // valid while that device's scratch generation still equals scratch_gen
  bool scratch = false;
  int device = -1;
  uint64_t scratch_gen = 0;
  // profiling
  bool prof = false;
  struct EvSet { std::vector<hipEvent_t> ev; std::vector<int> phase; };
  std::vector<EvSet> pending;
  std::vector<hipEvent_t> free_events;
  double prof_ms[MALT_NUM_PHASES] = {0};
  int64_t prof_launches[MALT_NUM_PHASES] = {0};
  int32_t last_ns_steps = 5;
};

namespace {

hipEvent_t get_event(malt_plan* p) {
  if (!p->free_events.empty()) {
    hipEvent_t e = p->free_events.back();
    p->free_events.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

hipError_t drain_profile(malt_plan* p) {
  for (auto& s : p->pending) {
    if (s.ev.empty()) continue;
    hipError_t e = hipEventSynchronize(s.ev.back());
    if (e != hipSuccess) return e;
    for (size_t k = 1; k < s.ev.size(); ++k) {
      float ms = 0.f;
      e = hipEventElapsedTime(&ms, s.ev[k - 1], s.ev[k]);
      if (e != hipSuccess) return e;
      p->prof_ms[s.phase[k - 1]] += ms;
      p->prof_launches[s.phase[k - 1]] += 1;
    }
    for (hipEvent_t ev : s.ev) p->free_events.push_back(ev);
  }
  p->pending.clear();
  return hipSuccess;
}

malt_status_t check_hparams(const malt_hparams_t* hp) {
  if (!hp) return fail(MALT_ERR_INVALID_ARG, "hparams is NULL");
  if (!(hp->lr >= 0.0) || !isfinite(hp->lr)) return fail(MALT_ERR_INVALID_ARG, "lr must be finite and >= 0");
  if (!(hp->mu1 >= 0.0 && hp->mu1 < 1.0)) return fail(MALT_ERR_INVALID_ARG, "mu1 must be in [0, 1)");
  if (!(hp->mu2 >= 0.0 && hp->mu2 < 1.0)) return fail(MALT_ERR_INVALID_ARG, "mu2 must be in [0, 1)");
  if (!(hp->eps > 0.0) || !isfinite(hp->eps)) return fail(MALT_ERR_INVALID_ARG, "eps must be finite and > 0");
  if (!(hp->weight_decay >= 0.0) || !isfinite(hp->weight_decay))
    return fail(MALT_ERR_INVALID_ARG, "weight_decay must be finite and >= 0");
  if (hp->ns_steps < 1 || hp->ns_steps > 64) return fail(MALT_ERR_INVALID_ARG, "ns_steps must be in [1, 64]");
  if (!isfinite(hp->ns_a) || !isfinite(hp->ns_b) || !isfinite(hp->ns_c))
    return fail(MALT_ERR_INVALID_ARG, "Newton-Schulz coefficients must be finite");
  if (!(hp->ns_eps >= 0.0) || !isfinite(hp->ns_eps)) return fail(MALT_ERR_INVALID_ARG, "ns_eps must be finite and >= 0");
  return MALT_OK;
}

void fill_desc(const malt_plan* p, std::vector<MatDesc>& D) {
  D.resize(p->n);
  for (int32_t i = 0; i < p->n; ++i) {
    const MatPlan& q = p->L.mats[i];
    MatDesc& d = D[i];
    memset(&d, 0, sizeof(d));
    d.m = int32_t(q.m); d.n = int32_t(q.n);
    d.mc = int32_t(q.mc); d.nc = int32_t(q.nc);
    d.mp = int32_t(q.mp); d.np = int32_t(q.np);
    d.tall = q.tall ? 1 : 0;
    d.split = q.split ? 1 : 0;
    d.k1_ct = int32_t(q.k1_ct); d.k1_rt = int32_t(q.k1_rt);
    d.k2_tiles = int32_t(q.k2_tiles); d.upd_tiles = int32_t(q.upd_tiles);
    float* st = reinterpret_cast<float*>(p->state);
    d.M = st + q.st_M; d.l = st + q.st_l; d.r = st + q.st_r;
    d.nu = q.st_nu >= 0 ? st + q.st_nu : nullptr;
    char* w = p->ws;
    d.Lv = reinterpret_cast<float*>(w + q.ws_Lv);
    d.Rv = reinterpret_cast<float*>(w + q.ws_Rv);
    d.rowpart = reinterpret_cast<float*>(w + q.ws_rowpart);
    d.colpart = reinterpret_cast<float*>(w + q.ws_colpart);
    d.k2part = reinterpret_cast<float*>(w + q.ws_k2part);
    d.gpart = reinterpret_cast<float*>(w + q.ws_gpart);
    for (int b = 0; b < 2; ++b) d.X[b] = reinterpret_cast<bf16_t*>(w + q.ws_X[b]);
    d.A = reinterpret_cast<bf16_t*>(w + q.ws_A);
    d.B = reinterpret_cast<bf16_t*>(w + q.ws_B);
    d.scal = reinterpret_cast<double*>(w + q.ws_scal);
    d.small = q.small ? 1 : 0;
    d.sm_gchunks = int32_t(q.sm_gchunks);
    for (int b = 0; b < 2; ++b) d.Xs[b] = q.small ? reinterpret_cast<float*>(w + q.ws_Xs[b]) : nullptr;
    d.Ap = q.small ? reinterpret_cast<float*>(w + q.ws_Ap) : nullptr;
    d.Bs = q.small ? reinterpret_cast<float*>(w + q.ws_Bs) : nullptr;
  }
}

malt_status_t check_init_args(const malt_shape_t* shapes, int32_t n, malt_variant_t variant, void* state_mem,
                              int32_t from_existing, int64_t step) {
  if (variant != MALT_VARIANT_MALT && variant != MALT_VARIANT_MALTER)
    return fail(MALT_ERR_INVALID_ARG, "unknown variant %d", int(variant));
  malt_status_t st = check_shapes(shapes, n);
  if (st != MALT_OK) return st;
  if (!state_mem) return fail(MALT_ERR_INVALID_ARG, "state pointer is NULL");
  if (reinterpret_cast<uintptr_t>(state_mem) % 16 != 0)
    return fail(MALT_ERR_ALIGNMENT, "state_mem must be 16-byte aligned");
  if (from_existing != 0 && from_existing != 1) return fail(MALT_ERR_INVALID_ARG, "from_existing must be 0 or 1");
  if (from_existing && step < 0) return fail(MALT_ERR_INVALID_ARG, "step must be >= 0");
  return MALT_OK;
}

// Lays the plan over state_mem and ws (p->L already set): uploads the
// descriptor table and work lists, zeroes the workspace (and the state unless
// resuming), and synchronises the stream.  Allocates no device or pinned host
// memory.
malt_status_t init_plan(malt_plan* p, const malt_shape_t* shapes, int32_t n, malt_variant_t variant,
                        void* state_mem, char* ws, int32_t from_existing, int64_t step, void* stream) {
  if (ranges_overlap(reinterpret_cast<uintptr_t>(state_mem), p->L.state_bytes, reinterpret_cast<uintptr_t>(ws),
                     p->L.ws_bytes))
    return fail(MALT_ERR_ALIAS, "state and workspace buffers overlap");
  // Device work starts here, after every argument check.
  hipError_t e = ns_gemm_setup();
  if (e != hipSuccess) return hip_fail(e, "setting the Newton-Schulz kernels' LDS limit");
  p->variant = variant;
  p->n = n;
  p->shapes.assign(shapes, shapes + n);
  p->state = static_cast<char*>(state_mem);
  p->ws = ws;
  p->t = from_existing ? step : 0;
  hipStream_t s = static_cast<hipStream_t>(stream);

  std::vector<MatDesc> D;
  fill_desc(p, D);
  std::vector<Tile> ew, fin, k2, sym, upd, smg, smp, smu;
  build_tiles(p->L, ew, fin, k2, sym, upd, smg, smp, smu);
  std::vector<Tile> gram, poly, updd;
  ns_dispatch_lists(p->L, sym, upd, gram, poly, updd);

  // Every table in one host image of the workspace head.
  const size_t head = p->L.ws_t_smu + sizeof(Tile) * smu.size();
  std::vector<char> h(head, 0);
  char* hc = h.data();
  memcpy(hc + p->L.ws_desc, D.data(), sizeof(MatDesc) * n);
  memcpy(hc + p->L.ws_t_ew, ew.data(), sizeof(Tile) * ew.size());
  memcpy(hc + p->L.ws_t_fin, fin.data(), sizeof(Tile) * fin.size());
  memcpy(hc + p->L.ws_t_k2, k2.data(), sizeof(Tile) * k2.size());
  memcpy(hc + p->L.ws_t_gram, gram.data(), sizeof(Tile) * gram.size());
  memcpy(hc + p->L.ws_t_poly, poly.data(), sizeof(Tile) * poly.size());
  memcpy(hc + p->L.ws_t_upd, updd.data(), sizeof(Tile) * updd.size());
  memcpy(hc + p->L.ws_t_smg, smg.data(), sizeof(Tile) * smg.size());
  memcpy(hc + p->L.ws_t_smp, smp.data(), sizeof(Tile) * smp.size());
  memcpy(hc + p->L.ws_t_smu, smu.data(), sizeof(Tile) * smu.size());

  e = launch_zero_fill(p->ws, p->L.ws_bytes, s);
  if (e == hipSuccess) e = hipMemcpyAsync(p->ws, hc, head, hipMemcpyHostToDevice, s);
  if (e == hipSuccess && !from_existing) e = launch_zero_fill(p->state, p->L.state_bytes, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "uploading plan tables");
  p->cur_ptrs.assign(n, PtrPair{nullptr, nullptr, 0, 0});
  return MALT_OK;
}


// ---------------------------------------------------------------------------
// Host-side bounds check of the work lists (no device work).  For every entry
// of every list it derives, with the kernels' own address functions where the
// kernels compute offsets (ns_common.h), the byte ranges the kernel can touch
// and checks them against the buffer each lies in.
// ---------------------------------------------------------------------------
struct BoundsCheck {
  const Layout& L;
  int64_t shrink = 0;
  int64_t checked = 0;
  malt_status_t st = MALT_OK;

  // [lo, hi) inside a buffer of `size` bytes (minus shrink unless exact);
  // off32: the range is addressed with 32-bit offsets from the buffer's base.
  bool range(const char* kernel, const char* buf, const Tile& t, uint64_t lo, uint64_t hi, uint64_t size,
             bool off32 = false, bool exact = false) {
    ++checked;
    const uint64_t lim = exact ? size : size > uint64_t(shrink) ? size - uint64_t(shrink) : 0;
    if (lo <= hi && hi <= lim && (!off32 || hi <= (uint64_t(1) << 32))) return true;
    st = fail(MALT_ERR_BOUNDS, "%s: matrix %d tile (%d, %d, %d): %s bytes [%llu, %llu) outside [0, %llu)%s", kernel,
              t.mat, t.ti, t.tj, t.idx, buf, (unsigned long long)lo, (unsigned long long)hi,
              (unsigned long long)lim, off32 && hi > (uint64_t(1) << 32) ? " or beyond 32-bit offsets" : "");
    return false;
  }
  // The same for the elementwise kernels' buffers, which shrink leaves alone:
  // it tests the Newton-Schulz buffers, read with hardware range checks off.
  bool erange(const char* kernel, const char* buf, const Tile& t, uint64_t lo, uint64_t hi, uint64_t size) {
    return range(kernel, buf, t, lo, hi, size, false, true);
  }
  bool cond(bool ok, const char* kernel, const Tile& t, const char* what) {
    ++checked;
    if (ok) return true;
    st = fail(MALT_ERR_BOUNDS, "%s: entry (mat %d, %d, %d, %d): %s", kernel, t.mat, t.ti, t.tj, t.idx, what);
    return false;
  }
  bool mat_ok(const char* kernel, const Tile& t) {
    return cond(t.mat >= 0 && size_t(t.mat) < L.mats.size(), kernel, t, "matrix index out of range");
  }
};

malt_status_t check_bounds(const Layout& L, int64_t shrink, int64_t* checked) {
  using UL = ns::UpdLoads<ns::UpdGeom>;
  constexpr int NW = ns::NW, LANES = 64;
  BoundsCheck B{L, shrink};
  std::vector<Tile> ew, fin, k2, sym, upd, smg, smp, smu, gram, poly, updd;
  build_tiles(L, ew, fin, k2, sym, upd, smg, smp, smu);
  ns_dispatch_lists(L, sym, upd, gram, poly, updd);
  const uint64_t u2 = 2, u4 = 4;

  // Workspace regions lie inside the workspace, in order, without overlap.
  {
    const Tile none{-1, 0, 0, 0};
    uint64_t end = L.ws_t_smu + sizeof(Tile) * smu.size();
    for (const MatPlan& q : L.mats) {
      const std::pair<size_t, uint64_t> regions[] = {
          {q.ws_scal, 8 * MAT_SCALARS}, {q.ws_Lv, 4 * q.m}, {q.ws_Rv, 4 * q.n},
          {q.ws_rowpart, 4 * uint64_t(q.k1_ct) * q.m}, {q.ws_colpart, 4 * uint64_t(q.k1_rt) * q.n},
          {q.ws_k2part, 8 * uint64_t(q.k2_tiles)}, {q.ws_gpart, 8 * uint64_t(q.upd_tiles)},
          {q.ws_X[0], 2 * uint64_t(q.mp) * q.np}, {q.ws_X[1], 2 * uint64_t(q.mp) * q.np},
          {q.ws_A, 2 * uint64_t(q.mp) * q.mp}, {q.ws_B, 2 * uint64_t(q.mp) * q.mp * (q.split ? 2 : 1)}};
      for (const auto& r : regions) {
        if (!B.cond(r.first >= end, "layout", none, "workspace regions overlap")) return B.st;
        end = r.first + r.second;
      }
      if (q.small) {
        const std::pair<size_t, uint64_t> sm[] = {{q.ws_Xs[0], 4 * uint64_t(q.mc) * q.np},
                                                  {q.ws_Xs[1], 4 * uint64_t(q.mc) * q.np},
                                                  {q.ws_Ap, 4 * uint64_t(q.sm_gchunks) * NS_SMALL_MAX * NS_SMALL_MAX},
                                                  {q.ws_Bs, 4 * uint64_t(NS_SMALL_MAX) * NS_SMALL_MAX}};
        for (const auto& r : sm) {
          if (!B.cond(r.first >= end, "layout", none, "workspace regions overlap")) return B.st;
          end = r.first + r.second;
        }
      }
    }
    if (!B.range("layout", "workspace", none, 0, end, L.ws_bytes, false, true)) return B.st;
  }

  // Momentum (row / column partials) and back-map (W, G, M guarded by r < m
  // and c < n in the kernels; O read inside the padded canonical buffer).
  for (const Tile& t : ew) {
    if (!B.mat_ok("momentum/back-map", t)) return B.st;
    const MatPlan& q = L.mats[t.mat];
    if (!B.cond(t.ti >= 0 && t.ti < q.k1_rt && t.tj >= 0 && t.tj < q.k1_ct, "momentum/back-map", t,
                "tile outside the matrix's tile grid"))
      return B.st;
    const uint64_t r0 = uint64_t(t.ti) * EW_TR, c0 = uint64_t(t.tj) * EW_TC;
    const uint64_t r1 = std::min<uint64_t>(r0 + EW_TR, q.m), c1 = std::min<uint64_t>(c0 + EW_TC, q.n);
    if (!B.cond(r0 < uint64_t(q.m) && c0 < uint64_t(q.n), "momentum/back-map", t, "tile origin outside W")) return B.st;
    if (!B.erange("momentum", "row partials", t, u4 * (t.tj * uint64_t(q.m) + r0), u4 * (t.tj * uint64_t(q.m) + r1),
                 u4 * q.k1_ct * q.m) ||
        !B.erange("momentum", "column partials", t, u4 * (t.ti * uint64_t(q.n) + c0),
                 u4 * (t.ti * uint64_t(q.n) + c1), u4 * q.k1_rt * q.n))
      return B.st;
    const uint64_t osz = u2 * q.mp * q.np;
    if (q.tall) {   // canonical rows c0 .. c0+255, columns r0 .. r0+31
      if (!B.erange("back-map", "O (tall)", t, u2 * (c0 * q.np + r0), u2 * ((c0 + EW_TC - 1) * q.np + r0 + EW_TR), osz))
        return B.st;
    } else {        // rows r0 .. r1-1, columns c0 .. c0+255
      if (!B.erange("back-map", "O (wide)", t, u2 * (r0 * q.np + c0), u2 * ((r1 - 1) * q.np + c0 + EW_TC), osz))
        return B.st;
    }
  }
  // Preconditioner finalise: chunks of FIN_W rows or columns.
  for (const Tile& t : fin) {
    if (!B.mat_ok("precond_finalize", t)) return B.st;
    const MatPlan& q = L.mats[t.mat];
    const int64_t len = t.ti == 0 ? q.m : q.n;
    if (!B.cond((t.ti == 0 || t.ti == 1) && t.tj >= 0 && int64_t(t.tj) * FIN_W < len, "precond_finalize", t,
                "chunk outside the rows / columns"))
      return B.st;
  }
  // Scale+convert: X0 over the padded canonical domain; norm partial slots.
  for (size_t k = 0; k < k2.size(); ++k) {
    const Tile& t = k2[k];
    if (!B.mat_ok("scale_convert", t)) return B.st;
    const MatPlan& q = L.mats[t.mat];
    const bool tall_list = int64_t(k) >= L.n_k2w;
    if (!B.cond(q.tall == tall_list && t.ti >= 0 && t.ti < q.k2_tr && t.tj >= 0 && t.tj < q.k2_tc, "scale_convert",
                t, "tile outside the grid or in the other kernel's list"))
      return B.st;
    const uint64_t xsz = u2 * q.mp * q.np;
    if (!tall_list) {
      const uint64_t r0 = uint64_t(t.ti) * K2W_R, c0 = uint64_t(t.tj) * EW_TC;
      if (!B.erange("scale_convert_wide", "X0", t, u2 * (r0 * q.np + c0), u2 * ((r0 + K2W_R - 1) * q.np + c0 + EW_TC),
                   xsz) ||
          !B.erange("scale_convert_wide", "norm partials", t, 8 * uint64_t(t.idx), 8 * uint64_t(t.idx) + 8,
                   8 * uint64_t(q.k2_tiles)))
        return B.st;
    } else if ((k - L.n_k2w) % K2_GROUP == 0) {
      // A workgroup takes K2_GROUP consecutive entries: one band of one matrix.
      for (int j = 1; j < K2_GROUP; ++j) {
        const bool in = k + j < k2.size();
        if (!B.cond(in && k2[k + j].mat == t.mat && k2[k + j].ti == t.ti && k2[k + j].tj == t.tj + j &&
                        k2[k + j].idx == t.idx + j,
                    "scale_convert_tall", t, "group entries are not consecutive tiles of one band"))
          return B.st;
      }
      const uint64_t r0 = uint64_t(t.ti) * K2_T, cb = uint64_t(t.tj) * K2_T;   // W rows, W columns
      if (!B.erange("scale_convert_tall", "X0", t, u2 * (cb * q.np + r0),
                   u2 * ((cb + K2_GROUP * K2_T - 1) * q.np + r0 + K2_T), xsz) ||
          !B.erange("scale_convert_tall", "norm partials", t, 8 * uint64_t(t.idx),
                   8 * (uint64_t(t.idx) + K2_GROUP), 8 * uint64_t(q.k2_tiles)))
        return B.st;
    }
  }
  if (!B.cond((L.n_k2 - L.n_k2w) % K2_GROUP == 0, "scale_convert_tall", Tile{-1, 0, 0, 0},
              "tall tile count is not a multiple of the group"))
    return B.st;

  // Newton-Schulz Gram and polynomial: direct loads of both panels over the
  // whole contraction, the polynomial's reload of A's tile, and the stores of
  // the tile and its mirror.
  for (int phase = 0; phase < 2; ++phase) {
    const std::vector<Tile>& list = phase == 0 ? gram : poly;
    const char* kname = phase == 0 ? "ns_gram" : "ns_poly";
    if (!B.cond(list.size() % NXCD == 0, kname, Tile{-1, 0, 0, 0}, "dispatch list not a multiple of the XCDs"))
      return B.st;
    for (const Tile& t : list) {
      if (t.mat < 0) continue;   // padding: the workgroup returns at once
      if (!B.mat_ok(kname, t)) return B.st;
      const MatPlan& q = L.mats[t.mat];
      const int T = int(q.mp / NS_TILE);
      if (!B.cond(!q.small && t.ti >= 0 && t.ti <= t.tj && t.tj < T, kname, t, "not an upper tile of the matrix"))
        return B.st;
      const int row0 = t.ti * NS_TILE, col0 = t.tj * NS_TILE;
      const int ld = phase == 0 ? int(q.np) : int(q.mp);
      const uint64_t psz = u2 * q.mp * ld;   // X[src] (Gram) or A (polynomial)
      const bool diag = t.ti == t.tj;
      // The Gram's and the polynomial's pipeline geometries.
      auto panel_span = [&](auto geom) -> uint64_t {
        using G = decltype(geom);
        using SL = ns::SymLoads<G>;
        const int KT = ld / G::BK;
        const int nloads = (diag ? G::LOADS / 2 : G::LOADS) * NW;   // g = wave + NW q
        uint64_t vmax = 0;
        for (int g = 0; g < nloads; ++g)
          for (int lane = 0; lane < LANES; ++lane) vmax = std::max(vmax, SL::voff(g, lane, row0, col0, ld));
        return vmax + SL::soff(KT - 1) + 16;
      };
      // A diagonal tile loads its row panel with the Gram geometry's load map.
      const uint64_t span = diag ? panel_span(ns::SymGeom{}) : phase == 0 ? panel_span(ns::SymGeom{})
                                                                           : panel_span(ns::PolyGeom{});
      if (!B.range(kname, phase == 0 ? "X panels" : "A panels", t, 0, span, psz, true)) return B.st;
      if (phase == 1) {
        uint64_t amax = 0;
        for (int c = 0; c < NS_TILE * NS_TILE * 2 / 16; ++c)
          amax = std::max(amax, ns::poly_a_tile_off(c, row0, col0, int(q.mp)));
        if (!B.range(kname, "A tile", t, 0, amax + 16, u2 * q.mp * q.mp, true)) return B.st;
      }
      const uint64_t ldo = (phase == 1 && q.split) ? 2 * q.mp : q.mp;
      const uint64_t off = (phase == 1 && q.split) ? q.mp : 0;   // the low part of a split B'
      const uint64_t far = uint64_t(std::max(row0, col0)) + NS_TILE;
      if (!B.range(kname, phase == 0 ? "A (tile and mirror)" : "B' (tile and mirror)", t,
                   u2 * (uint64_t(std::min(row0, col0)) * ldo), u2 * ((far - 1) * ldo + off + far), u2 * q.mp * ldo))
        return B.st;
    }
  }
  // Newton-Schulz update: B' rows and X k-rows over the contraction (X's k
  // wraps at mp for split matrices), the X' tile, the graft partial slot.
  if (!B.cond(updd.size() % NXCD == 0, "ns_update", Tile{-1, 0, 0, 0}, "dispatch list not a multiple of the XCDs"))
    return B.st;
  for (const Tile& t : updd) {
    if (t.mat < 0) continue;
    if (!B.mat_ok("ns_update", t)) return B.st;
    const MatPlan& q = L.mats[t.mat];
    if (!B.cond(!q.small && t.ti >= 0 && t.ti < q.mp / NS_TILE && t.tj >= 0 && t.tj < q.np / NS_TILE &&
                    t.idx >= 0 && t.idx < q.upd_tiles,
                "ns_update", t, "tile outside the matrix or partial slot out of range"))
      return B.st;
    const int row0 = t.ti * NS_TILE, col0 = t.tj * NS_TILE;
    const int ldb = int(q.split ? 2 * q.mp : q.mp);
    const int KT = ldb / ns::UpdGeom::BK;
    uint64_t bmax = 0, xmax = 0, sxmax = 0;
    for (int g = 0; g < ns::UpdGeom::LOADS * NW; ++g)
      for (int lane = 0; lane < LANES; ++lane) {
        if (g < UL::LOADS_P) bmax = std::max(bmax, UL::voff_b(g, lane, row0, ldb));
        else xmax = std::max(xmax, UL::voff_x(g, lane, col0, int(q.np)));
      }
    for (int kt = 0; kt < KT; ++kt) sxmax = std::max(sxmax, UL::soff_x(kt, int(q.mp), int(q.np)));
    if (!B.range("ns_update", "B' rows", t, 0, bmax + UL::soff_b(KT - 1) + 16, u2 * q.mp * ldb, true) ||
        !B.range("ns_update", "X k-rows", t, 0, xmax + sxmax + 16, u2 * q.mp * q.np, true) ||
        !B.range("ns_update", "X' tile", t, u2 * (uint64_t(row0) * q.np + col0),
                 u2 * (uint64_t(row0 + NS_TILE - 1) * q.np + col0 + NS_TILE), u2 * q.mp * q.np) ||
        !B.range("ns_update", "graft partials", t, 8 * uint64_t(t.idx), 8 * uint64_t(t.idx) + 8,
                 8 * uint64_t(q.upd_tiles)))
      return B.st;
  }
  // fp32 Newton-Schulz of short sides <= 32: chunk and partial-slot indices.
  for (const Tile& t : smg) {
    if (!B.mat_ok("sm_gram", t)) return B.st;
    const MatPlan& q = L.mats[t.mat];
    if (!B.cond(q.small && t.ti >= 0 && t.ti < q.sm_gchunks && int64_t(t.ti) * SM_CH_G < q.np, "sm_gram", t,
                "chunk out of range"))
      return B.st;
  }
  for (const Tile& t : smp) {
    if (!B.mat_ok("sm_poly", t)) return B.st;
    if (!B.cond(L.mats[t.mat].small, "sm_poly", t, "matrix is not on the fp32 path")) return B.st;
  }
  for (const Tile& t : smu) {
    if (!B.mat_ok("sm_update", t)) return B.st;
    const MatPlan& q = L.mats[t.mat];
    if (!B.cond(q.small && t.ti >= 0 && int64_t(t.ti + 1) * SM_CH_U <= q.np && t.idx >= 0 && t.idx < q.upd_tiles,
                "sm_update", t, "chunk or partial slot out of range"))
      return B.st;
  }
  *checked = B.checked;
  return MALT_OK;
}

}  // namespace

extern "C" {

void malt_hparams_default(malt_hparams_t* hp) {
  if (!hp) return;
  hp->lr = 1.3e-3;
  hp->mu1 = 0.95;
  hp->mu2 = 0.99;
  hp->eps = 1e-8;
  hp->weight_decay = 0.0;
  hp->ns_steps = 5;
  hp->ns_a = 3.4445;
  hp->ns_b = -4.7750;
  hp->ns_c = 2.0315;
  hp->ns_eps = 1e-7;
  hp->precond_identity = 0;
}

malt_status_t malt_state_size(const malt_shape_t* shapes, int32_t n, malt_variant_t variant,
                              size_t* state_bytes, size_t* workspace_bytes) {
  if (variant != MALT_VARIANT_MALT && variant != MALT_VARIANT_MALTER)
    return fail(MALT_ERR_INVALID_ARG, "unknown variant %d", int(variant));
  if (!state_bytes || !workspace_bytes) return fail(MALT_ERR_INVALID_ARG, "output pointer is NULL");
  malt_status_t st = check_shapes(shapes, n);
  if (st != MALT_OK) return st;
  const Layout L = make_layout(shapes, n, variant);
  *state_bytes = L.state_bytes;
  *workspace_bytes = L.ws_bytes;
  return MALT_OK;
}

malt_status_t malt_init_state(malt_plan_t** out, const malt_shape_t* shapes, int32_t n,
                              malt_variant_t variant, void* state_mem, void* workspace_mem,
                              int32_t from_existing, int64_t step, void* stream) {
  if (!out) return fail(MALT_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  malt_status_t st = check_init_args(shapes, n, variant, state_mem, from_existing, step);
  if (st != MALT_OK) return st;
  if (!workspace_mem) return fail(MALT_ERR_INVALID_ARG, "workspace pointer is NULL");
  if (reinterpret_cast<uintptr_t>(workspace_mem) % 256 != 0)
    return fail(MALT_ERR_ALIGNMENT, "workspace_mem must be 256-byte aligned");
  malt_plan* p = new malt_plan();
  p->L = make_layout(shapes, n, variant);
  st = init_plan(p, shapes, n, variant, state_mem, static_cast<char*>(workspace_mem), from_existing, step, stream);
  if (st != MALT_OK) { delete p; return st; }
  *out = p;
  return MALT_OK;
}

malt_status_t malt_init_state_scratch(malt_plan_t** out, const malt_shape_t* shapes, int32_t n,
                                      malt_variant_t variant, void* state_mem, int32_t from_existing,
                                      int64_t step, void* stream) {
  if (!out) return fail(MALT_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  malt_status_t st = check_init_args(shapes, n, variant, state_mem, from_existing, step);
  if (st != MALT_OK) return st;
  Layout L = make_layout(shapes, n, variant);
  if (L.ws_bytes > MALT_SCRATCH_BYTES)
    return fail(MALT_ERR_SCRATCH_SIZE, "these shapes need a %zu-byte workspace; the static scratch holds %llu bytes "
                "(use malt_init_state with a caller-allocated workspace)", L.ws_bytes,
                (unsigned long long)MALT_SCRATCH_BYTES);
  int dev = -1;
  char* ws = nullptr;
  uint64_t gen = 0;
  st = scratch_claim(&dev, &ws, &gen);
  if (st != MALT_OK) return st;
  malt_plan* p = new malt_plan();
  p->L = std::move(L);
  p->scratch = true;
  p->device = dev;
  p->scratch_gen = gen;
  st = init_plan(p, shapes, n, variant, state_mem, ws, from_existing, step, stream);
  if (st != MALT_OK) { delete p; return st; }
  *out = p;
  return MALT_OK;
}

malt_status_t malt_step(malt_plan_t* p, float* const* params, const float* const* grads,
                        const malt_shape_t* shapes, int32_t n, const malt_hparams_t* hp, void* stream) {
  if (!p) return fail(MALT_ERR_INVALID_ARG, "plan is NULL");
  if (!params || !grads) return fail(MALT_ERR_INVALID_ARG, "params or grads is NULL");
  malt_status_t st = check_hparams(hp);
  if (st != MALT_OK) return st;
  if (n != p->n || !shapes) return fail(MALT_ERR_STATE_MISMATCH, "matrix count %d differs from the plan's %d", n, p->n);
  for (int32_t i = 0; i < n; ++i)
    if (shapes[i].rows != p->shapes[i].rows || shapes[i].cols != p->shapes[i].cols)
      return fail(MALT_ERR_STATE_MISMATCH, "matrix %d: shape %lld x %lld differs from the plan's %lld x %lld", i,
                  (long long)shapes[i].rows, (long long)shapes[i].cols, (long long)p->shapes[i].rows,
                  (long long)p->shapes[i].cols);
  // Pointer checks (host-side, before any enqueue).
  bool changed = !p->ptrs_valid;
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(p->state), w0 = reinterpret_cast<uintptr_t>(p->ws);
  for (int32_t i = 0; i < n; ++i) {
    const uintptr_t W = reinterpret_cast<uintptr_t>(params[i]), G = reinterpret_cast<uintptr_t>(grads[i]);
    if (!W || !G) return fail(MALT_ERR_INVALID_ARG, "matrix %d: NULL param or grad", i);
    if (W % 4 || G % 4) return fail(MALT_ERR_ALIGNMENT, "matrix %d: param/grad not 4-byte aligned", i);
    const size_t bytes = size_t(p->shapes[i].rows) * p->shapes[i].cols * 4;
    if (ranges_overlap(W, bytes, G, bytes)) return fail(MALT_ERR_ALIAS, "matrix %d: param and grad overlap", i);
    if (ranges_overlap(W, bytes, s0, p->L.state_bytes) || ranges_overlap(G, bytes, s0, p->L.state_bytes) ||
        ranges_overlap(W, bytes, w0, p->L.ws_bytes) || ranges_overlap(G, bytes, w0, p->L.ws_bytes))
      return fail(MALT_ERR_ALIAS, "matrix %d: param/grad overlaps the state or workspace", i);
    if (p->cur_ptrs[i].W != params[i] || p->cur_ptrs[i].G != grads[i]) changed = true;
  }
  if (changed && n > 1) {
    // Parameters are updated in place: they must not overlap one another.
    std::vector<std::pair<uintptr_t, size_t>> rs(n);
    for (int32_t i = 0; i < n; ++i)
      rs[i] = {reinterpret_cast<uintptr_t>(params[i]), size_t(p->shapes[i].rows) * p->shapes[i].cols * 4};
    std::sort(rs.begin(), rs.end());
    for (int32_t i = 1; i < n; ++i)
      if (rs[i - 1].first + rs[i - 1].second > rs[i].first)
        return fail(MALT_ERR_ALIAS, "two parameter matrices overlap");
  }

  if (p->scratch && !scratch_current(p->device, p->scratch_gen))
    return fail(MALT_ERR_STATE_MISMATCH, "the static scratch of device %d now belongs to a newer plan; "
                "this plan's workspace is gone", p->device);

  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (changed) {
    // The new table travels in the arguments of small copy kernels, which the
    // runtime captures at enqueue: nothing on the host waits.
    PtrUploadArgs up;
    up.count = 0;
    std::vector<PtrPair> next(n);
    for (int32_t i = 0; i < n; ++i) {
      // The vectorised elementwise path needs 16-byte aligned rows of W, G and M.
      const MatPlan& q = p->L.mats[i];
      const uintptr_t M = reinterpret_cast<uintptr_t>(p->state) + 4 * size_t(q.st_M);
      next[i].W = params[i];
      next[i].G = grads[i];
      next[i].vec = (q.n % 4 == 0) && (reinterpret_cast<uintptr_t>(params[i]) % 16 == 0) &&
                    (reinterpret_cast<uintptr_t>(grads[i]) % 16 == 0) && (M % 16 == 0);
      next[i].pad_ = 0;
    }
    PtrPair* dst = reinterpret_cast<PtrPair*>(p->ws + p->L.ws_ptrs);
    e = hipSuccess;
    for (int32_t i0 = 0; i0 < n && e == hipSuccess; i0 += PTR_CHUNK) {
      up.dst = dst + i0;
      up.count = std::min<int32_t>(PTR_CHUNK, n - i0);
      memcpy(up.p, next.data() + i0, sizeof(PtrPair) * up.count);
      e = launch_ptr_upload(up, s);
    }
    if (e != hipSuccess) { p->ptrs_valid = false; return hip_fail(e, "uploading pointer table"); }
    p->cur_ptrs = next;
    p->ptrs_valid = true;
  }

  const int64_t t = p->t + 1;
  EwArgs ea;
  ea.desc = reinterpret_cast<const MatDesc*>(p->ws + p->L.ws_desc);
  ea.ptrs = reinterpret_cast<const PtrPair*>(p->ws + p->L.ws_ptrs);
  ea.tiles = nullptr;
  ea.ntiles = 0;
  ea.mu1 = float(hp->mu1);
  ea.one_minus_mu1 = float(1.0 - hp->mu1);
  ea.mu2 = hp->mu2;
  ea.eps = hp->eps;
  ea.bc = sqrt(1.0 - pow(hp->mu2, double(t))) / (1.0 - pow(hp->mu1, double(t)) + hp->eps);
  ea.ns_eps = hp->ns_eps;
  ea.lr = hp->lr;
  ea.decay = float(1.0 - hp->lr * hp->weight_decay);
  ea.malter = p->variant == MALT_VARIANT_MALTER;
  ea.identity = hp->precond_identity != 0;
  ea.o_parity = hp->ns_steps & 1;

  malt_plan::EvSet evs;
  auto mark = [&](int phase) -> hipError_t {
    if (!p->prof) return hipSuccess;
    hipEvent_t ev = get_event(p);
    if (!ev) return hipErrorOutOfMemory;
    evs.ev.push_back(ev);
    evs.phase.push_back(phase);
    return hipEventRecord(ev, s);
  };
  auto tiles_at = [&](size_t off) { return reinterpret_cast<const Tile*>(p->ws + off); };

#define MALT_LAUNCH(phase, call)                            \
  do {                                                      \
    if ((e = mark(phase)) != hipSuccess) goto hip_error;    \
    if ((e = (call)) != hipSuccess) goto hip_error;         \
  } while (0)
  {
    ea.tiles = tiles_at(p->L.ws_t_ew); ea.ntiles = int32_t(p->L.n_ew);
    MALT_LAUNCH(0, launch_momentum_rowcol(ea, s));
    ea.tiles = tiles_at(p->L.ws_t_fin); ea.ntiles = int32_t(p->L.n_fin);
    MALT_LAUNCH(1, launch_precond_finalize(ea, s));
    if (p->L.n_k2w > 0) {
      ea.tiles = tiles_at(p->L.ws_t_k2); ea.ntiles = int32_t(p->L.n_k2w);
      MALT_LAUNCH(2, launch_scale_convert(ea, false, s));
    }
    if (p->L.n_k2 > p->L.n_k2w) {
      ea.tiles = tiles_at(p->L.ws_t_k2) + p->L.n_k2w; ea.ntiles = int32_t(p->L.n_k2 - p->L.n_k2w);
      MALT_LAUNCH(2, launch_scale_convert(ea, true, s));
    }
    MALT_LAUNCH(3, launch_norm_scalars(ea, n, s));
    NsArgs na;
    na.desc = ea.desc;
    na.a = float(hp->ns_a); na.b = float(hp->ns_b); na.c = float(hp->ns_c);
    for (int32_t it = 0; it < hp->ns_steps; ++it) {
      na.first = it == 0;
      na.last = it == hp->ns_steps - 1;
      na.src = it & 1;
      if (p->L.n_sym > 0) {   // matrix-core path
        na.tiles = tiles_at(p->L.ws_t_gram); na.ntiles = int32_t(p->L.n_gram);
        na.phase = PH_GRAM;
        MALT_LAUNCH(4, launch_ns_gemm(na, s));
        na.tiles = tiles_at(p->L.ws_t_poly); na.ntiles = int32_t(p->L.n_poly);
        na.phase = PH_POLY;
        MALT_LAUNCH(5, launch_ns_gemm(na, s));
        na.tiles = tiles_at(p->L.ws_t_upd); na.ntiles = int32_t(p->L.n_updd);
        na.phase = PH_UPDATE;
        MALT_LAUNCH(6, launch_ns_gemm(na, s));
      }
      if (p->L.n_smp > 0) {   // fp32 path of the small matrices
        na.tiles = tiles_at(p->L.ws_t_smg); na.ntiles = int32_t(p->L.n_smg);
        na.phase = PH_GRAM;
        MALT_LAUNCH(4, launch_small_ns(na, s));
        na.tiles = tiles_at(p->L.ws_t_smp); na.ntiles = int32_t(p->L.n_smp);
        na.phase = PH_POLY;
        MALT_LAUNCH(5, launch_small_ns(na, s));
        na.tiles = tiles_at(p->L.ws_t_smu); na.ntiles = int32_t(p->L.n_smu);
        na.phase = PH_UPDATE;
        MALT_LAUNCH(6, launch_small_ns(na, s));
      }
    }
    MALT_LAUNCH(7, launch_graft_scalars(ea, n, s));
    ea.tiles = tiles_at(p->L.ws_t_ew); ea.ntiles = int32_t(p->L.n_ew);
    MALT_LAUNCH(8, launch_backmap_write(ea, s));
    if ((e = mark(-1)) != hipSuccess) goto hip_error;
  }
#undef MALT_LAUNCH
  if (p->prof) {
    p->pending.push_back(std::move(evs));
    if (p->pending.size() > 256) {
      e = drain_profile(p);
      if (e != hipSuccess) return hip_fail(e, "reading profile events");
    }
  }
  p->last_ns_steps = hp->ns_steps;
  p->t = t;
  return MALT_OK;
hip_error:
  for (hipEvent_t ev : evs.ev) p->free_events.push_back(ev);
  return hip_fail(e, "launching step kernels");
}

malt_status_t malt_check_bounds(const malt_shape_t* shapes, int32_t n, malt_variant_t variant, int64_t shrink_bytes,
                                int64_t* ranges_checked) {
  if (variant != MALT_VARIANT_MALT && variant != MALT_VARIANT_MALTER)
    return fail(MALT_ERR_INVALID_ARG, "unknown variant %d", int(variant));
  if (!ranges_checked) return fail(MALT_ERR_INVALID_ARG, "ranges_checked is NULL");
  if (shrink_bytes < 0) return fail(MALT_ERR_INVALID_ARG, "shrink_bytes must be >= 0");
  *ranges_checked = 0;
  malt_status_t st = check_shapes(shapes, n);
  if (st != MALT_OK) return st;
  const Layout L = make_layout(shapes, n, variant);
  return check_bounds(L, shrink_bytes, ranges_checked);
}

malt_status_t malt_state_layout(const malt_plan_t* p, int32_t i, malt_state_layout_t* out) {
  if (!p || !out) return fail(MALT_ERR_INVALID_ARG, "NULL argument");
  if (i < 0 || i >= p->n) return fail(MALT_ERR_INVALID_ARG, "matrix index %d out of range", i);
  const MatPlan& q = p->L.mats[i];
  out->M = q.st_M; out->l = q.st_l; out->r = q.st_r; out->nu = q.st_nu;
  return MALT_OK;
}

malt_status_t malt_debug_layout(const malt_plan_t* p, int32_t i, malt_debug_layout_t* out) {
  if (!p || !out) return fail(MALT_ERR_INVALID_ARG, "NULL argument");
  if (i < 0 || i >= p->n) return fail(MALT_ERR_INVALID_ARG, "matrix index %d out of range", i);
  const MatPlan& q = p->L.mats[i];
  const int par = p->last_ns_steps & 1;
  out->Lv = int64_t(q.ws_Lv);
  out->Rv = int64_t(q.ws_Rv);
  out->O = int64_t(q.ws_X[par]);
  out->X0 = int64_t(q.ws_X[0]);
  out->O_pitch = q.np;
  out->O_transposed = q.tall ? 1 : 0;
  out->scalars = int64_t(q.ws_scal);
  out->A = q.small ? 0 : int64_t(q.ws_A);
  out->B = q.small ? 0 : int64_t(q.ws_B);
  out->AB_pitch = q.small ? 0 : q.mp;
  out->B_split = q.split ? 1 : 0;
  return MALT_OK;
}

malt_status_t malt_precond_condition(const malt_plan_t* p, double* out, void* stream) {
  if (!p || !out) return fail(MALT_ERR_INVALID_ARG, "NULL argument");
  const uintptr_t o = reinterpret_cast<uintptr_t>(out);
  if (o % 8) return fail(MALT_ERR_ALIGNMENT, "out is not 8-byte aligned");
  const size_t bytes = 16 * size_t(p->n);
  if (ranges_overlap(o, bytes, reinterpret_cast<uintptr_t>(p->state), p->L.state_bytes) ||
      ranges_overlap(o, bytes, reinterpret_cast<uintptr_t>(p->ws), p->L.ws_bytes))
    return fail(MALT_ERR_ALIAS, "out overlaps the state or workspace");
  if (p->scratch && !scratch_current(p->device, p->scratch_gen))
    return fail(MALT_ERR_STATE_MISMATCH, "the static scratch of device %d now belongs to a newer plan; "
                "this plan's workspace is gone", p->device);
  const hipError_t e = launch_precond_cond(reinterpret_cast<const MatDesc*>(p->ws + p->L.ws_desc), p->n, out,
                                           static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MALT_OK : hip_fail(e, "launching the condition-number kernel");
}

int64_t malt_plan_step(const malt_plan_t* p) { return p ? p->t : -1; }

malt_status_t malt_profile_enable(malt_plan_t* p, int32_t enable) {
  if (!p) return fail(MALT_ERR_INVALID_ARG, "plan is NULL");
  p->prof = enable != 0;
  return MALT_OK;
}

malt_status_t malt_profile_read(malt_plan_t* p, malt_profile_t* out, int32_t reset) {
  if (!p || !out) return fail(MALT_ERR_INVALID_ARG, "NULL argument");
  hipError_t e = drain_profile(p);
  if (e != hipSuccess) return hip_fail(e, "reading profile events");
  memset(out, 0, sizeof(*out));
  for (int k = 0; k < MALT_NUM_PHASES; ++k) {
    out->ms[k] = p->prof_ms[k];
    out->launches[k] = p->prof_launches[k];
  }
  // Algorithmic bytes / flops of one step (float32 = 4 B, bf16 = 2 B).
  const bool malter = p->variant == MALT_VARIANT_MALTER;
  for (const MatPlan& q : p->L.mats) {
    const double el = double(q.m) * q.n, mn = double(q.m + q.n);
    out->bytes[0] += 12.0 * el + 4.0 * mn;                      // G, M in; M out; row/col partials
    out->bytes[1] += 8.0 * mn + 4.0 * mn;                       // l, r in/out, L, R out
    out->bytes[2] += (malter ? 8.0 : 4.0) * el + 2.0 * el;      // M (+G) in; bf16 X0 out
    out->bytes[8] += 10.0 * el;                                 // W, O in; W out
    const int steps = p->last_ns_steps;
    out->flops[4] += steps * double(q.mc) * q.mc * q.nc;            // X X^T, one triangle
    out->flops[5] += steps * double(q.mc) * q.mc * q.mc;            // A A, one triangle
    out->flops[6] += steps * 2.0 * double(q.mc) * q.mc * q.nc;      // B X (once, also when split)
  }
  if (reset) {
    memset(p->prof_ms, 0, sizeof(p->prof_ms));
    memset(p->prof_launches, 0, sizeof(p->prof_launches));
  }
  return MALT_OK;
}

void malt_destroy_state(malt_plan_t* p) {
  if (!p) return;
  (void)drain_profile(p);
  for (hipEvent_t ev : p->free_events) (void)hipEventDestroy(ev);
  delete p;
}

const char* malt_status_string(malt_status_t s) {
  switch (s) {
    case MALT_OK: return "MALT_OK";
    case MALT_ERR_INVALID_ARG: return "MALT_ERR_INVALID_ARG";
    case MALT_ERR_SHAPE: return "MALT_ERR_SHAPE";
    case MALT_ERR_ALIGNMENT: return "MALT_ERR_ALIGNMENT";
    case MALT_ERR_STATE_MISMATCH: return "MALT_ERR_STATE_MISMATCH";
    case MALT_ERR_HIP: return "MALT_ERR_HIP";
    case MALT_ERR_ALIAS: return "MALT_ERR_ALIAS";
    case MALT_ERR_SCRATCH_SIZE: return "MALT_ERR_SCRATCH_SIZE";
    case MALT_ERR_BOUNDS: return "MALT_ERR_BOUNDS";
  }
  return "MALT_ERR_UNKNOWN";
}

const char* malt_last_error(void) { return g_last_error.c_str(); }

const char* malt_version(void) { return "libmalt 0.1 (gfx950)"; }

}  // extern "C"
