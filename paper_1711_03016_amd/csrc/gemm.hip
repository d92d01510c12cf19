// Host side of the dense-layer products: choice of the tile configuration for
// a given problem, and the launch.
#include <algorithm>
#include <cstdlib>

#include "gemm_kernel.hpp"

namespace dlvm {

namespace {

// Compute units of an MI355X and per-compute-unit rates the planner assumes:
// matrix-core flops per clock (float32, bf16) and L2 bytes per clock.
constexpr int kComputeUnits = 256;
constexpr double kRateF32 = 256.0;
constexpr double kRateBF16 = 4096.0;
constexpr double kL2BytesPerClock = 64.0;

// Tile configurations with the fraction of the matrix-core rate each sustains
// when not starved, for float32 and for bf16 operands (measured on large
// products). Configurations 0-5 are the register-staged kernel
// (gemm_kernel.hpp), 10-13, 16 and 17 the bf16 kernel with direct-to-LDS loads
// (gemm_async.hpp; 18 with two k-groups of waves), 14-15 the four-wave bf16
// kernel (gemm_xl.hpp).
struct TileShape {
  int cfg;
  int bm, bn;
  double eff_f32, eff_bf16;
  bool async;
  int kseg;  // register-staged kernel: 128-byte k-segments per pipeline stage
};
constexpr TileShape kTiles[] = {
    {0, 128, 128, 0.8, 0.55, false, 1},  {1, 64, 64, 0.6, 0.3, false, 2},
    {2, 128, 32, 0.6, 0.3, false, 2},    {3, 32, 32, 0.5, 0.25, false, 4},
    {4, 64, 64, 0.65, 0.2, false, 2},    {5, 32, 32, 0.5, 0.25, false, 8},
    {10, 256, 256, 0.0, 0.9, true, 0},   {11, 256, 128, 0.0, 0.63, true, 0},
    {12, 128, 128, 0.0, 0.54, true, 0},  {13, 256, 256, 0.0, 0.88, true, 0},
    {14, 256, 256, 0.0, 0.89, true, 0},  {15, 256, 256, 0.0, 0.85, true, 0},
    {16, 64, 128, 0.0, 0.5, true, 0},    {17, 128, 128, 0.0, 0.54, true, 0},
    {18, 64, 128, 0.0, 0.55, true, 0},   {19, 128, 128, 0.0, 0.56, true, 0}};

// The register-staged kernel has one stage of loads in flight: a stage costs
// at least one load round trip (measured on small float32 products).
constexpr double kStageCycles = 3500.0;

// Fixed cost of one round of tiles (first loads, epilogue) and of the extra
// launch of a split reduction, in clock cycles; HBM bytes per clock.
constexpr double kTileFixed = 4000.0;
constexpr double kLaunch = 9600.0;
constexpr double kHbmBytesPerClock = 2000.0;
constexpr int kMaxSplits = 16;
constexpr int64_t kMinChunk = 256;  // k per slice at least (a multiple of every k-tile)

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool aligned16(const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15u) == 0; }

// The direct-to-LDS kernel moves whole 16-byte chunks: bf16 operands with
// 16-byte aligned bases, leading dimensions and contraction extent; its
// epilogue moves 8 consecutive outputs at a time (16-byte aligned output rows,
// saved activation and residual).
bool phases_ok(const GemmDesc& d, int vw) {
  return d.A2 == nullptr || (aligned16(d.A2) && d.lda2 % vw == 0 && d.K1 % vw == 0);
}

// A contraction in two phases (a second source A2 for k in [K1, K)). Told by
// the phase split as well as by A2, so a plan description, whose bases are
// null, plans such a product as the call does.
bool two_phase(const GemmDesc& d) { return d.A2 != nullptr || (d.K1 > 0 && d.K1 < d.K); }

bool async_ok(const GemmDesc& d) {
  return d.dtype == BF16 && aligned16(d.A) && aligned16(d.B) && d.lda % 8 == 0 &&
         d.ldb % 8 == 0 && d.K % 8 == 0 && d.ldc % 8 == 0 && aligned16(d.C) &&
         aligned16(d.aux) && aligned16(d.residual) && aligned16(d.bias) && phases_ok(d, 8);
}

// Extent in bytes of a row-major operand of `rows` rows of `cols` elements at
// stride `ld`.
int64_t extent_bytes(int64_t rows, int64_t cols, int64_t ld, int64_t es) {
  return ((rows - 1) * ld + cols) * es;
}

// Operand rows and columns of a product (A is M x K or K x M, B is N x K or K x N).
void operand_dims(const GemmDesc& d, int64_t& ar, int64_t& ac, int64_t& br, int64_t& bc) {
  const bool ak = d.layout != Layout::TN, bk = d.layout == Layout::NT;
  ar = ak ? d.M : d.K; ac = ak ? d.K : d.M;
  br = bk ? d.N : d.K; bc = bk ? d.K : d.N;
}

// The buffer-descriptor kernel addresses its operands with 32-bit byte
// offsets: every offset it forms (up to one tile past either extent) must stay
// below 2^31.
bool xl_ok(const GemmDesc& d) {
  if (!async_ok(d) || two_phase(d)) return false;
  int64_t ar, ac, br, bc;
  operand_dims(d, ar, ac, br, bc);
  const int64_t lim = int64_t(1) << 31;
  return (ar + 256) * d.lda * 2 + 512 < lim && (br + 256) * d.ldb * 2 + 512 < lim &&
         ac <= d.lda && bc <= d.ldb;
}

// The same for the k-slices of a two-phase (forward) product, each of which
// reads one phase: A's M x K1 block (stride lda), A2's M x (K - K1) block
// (stride lda2) and B.
bool xl_phases_ok(const GemmDesc& d) {
  if (!async_ok(d) || !two_phase(d) || d.layout != Layout::NN) return false;
  const int64_t lim = int64_t(1) << 31;
  return (d.M + 256) * d.lda * 2 + 512 < lim && (d.M + 256) * d.lda2 * 2 + 512 < lim &&
         (d.K + 256) * d.ldb * 2 + 512 < lim && d.K1 <= d.lda && d.K - d.K1 <= d.lda2 &&
         d.N <= d.ldb;
}

// k per slice when K is split `splits` ways (a multiple of 64, so every
// slice but the last is whole k-tiles for every kernel).
int64_t slice_k(int64_t K, int splits) { return ceil_div(ceil_div(K, splits), 64) * 64; }

// Clock cycles one configuration needs: rounds of tiles over the compute
// units, each tile bound by its matrix-core work or its operand traffic, plus
// the reduction of a split product.
double estimate(const GemmDesc& d, const TileShape& t, int splits) {
  const int64_t tiles = ceil_div(d.M, t.bm) * ceil_div(d.N, t.bn);
  const int64_t kc = splits > 1 ? slice_k(d.K, splits) : d.K;
  const int64_t slices = ceil_div(d.K, kc);
  const double es = d.dtype == F32 ? 4.0 : 2.0;
  const double eff = d.dtype == F32 ? t.eff_f32 : t.eff_bf16;
  const double rate = (d.dtype == F32 ? kRateF32 : kRateBF16) * eff;
  const double flops = 2.0 * t.bm * t.bn * double(kc);
  const double bytes = double(t.bm + t.bn) * double(kc) * es;
  double per_tile = std::max(flops / rate, bytes / kL2BytesPerClock);
  if (!t.async && d.dtype == BF16) {  // (the float32 choices were measured without it)
    const int64_t kstage = int64_t(t.kseg) * 64;
    per_tile = std::max(per_tile, double(ceil_div(kc, kstage)) * kStageCycles);
  }
  per_tile += kTileFixed;
  double c = double(ceil_div(tiles * slices, kComputeUnits)) * per_tile;
  if (slices > 1) c += kLaunch + double(slices + 1) * double(d.M) * double(d.N) * 4.0 / kHbmBytesPerClock;
  return c;
}

// Float32 elements the partials of a `splits`-way split of product d take.
int64_t split_need(const GemmDesc& d, int splits) {
  const int64_t nv = d.nvec > 0 ? d.nvec : d.N;
  return static_cast<int64_t>(splits) * (d.M * d.ldc + nv);
}

}  // namespace

// Tile configuration forced through the environment variable
// DLVM_GEMM_CONFIG (for tests and tuning), or -1. A forced configuration that
// cannot run the product is ignored.
int env_int(const char* name) {
  const char* v = std::getenv(name);
  if (v == nullptr || *v == 0) return -1;
  char* end = nullptr;
  const long c = std::strtol(v, &end, 10);
  return (end != nullptr && *end == 0) ? static_cast<int>(c) : -1;
}
// Inside a tuning scope (one library call) the two variables are read once,
// at its start, not once per product.
thread_local int t_depth = 0;
thread_local bool t_loaded = false;
thread_local int t_config = -1, t_splits = -1;

void load_tuning() {
  if (t_depth > 0 && t_loaded) return;
  t_config = env_int("DLVM_GEMM_CONFIG");
  t_splits = env_int("DLVM_GEMM_SPLITS");
  t_loaded = t_depth > 0;
}

int forced_config() {
  load_tuning();
  return t_config;
}

// Number of k-slices forced through DLVM_GEMM_SPLITS (for tests and tuning)
// on products the caller lets split with their epilogue, or -1.
int forced_splits() {
  load_tuning();
  return t_splits;
}

void tuning_scope_begin() {
  if (t_depth++ == 0) t_loaded = false;
}
void tuning_scope_end() { --t_depth; }

namespace {

// The configuration and split (only products wrt the weights, TN, with
// scratch for the partials) that the estimate prefers. `assume_aligned`
// ignores the operands' addresses (for sizing scratch before they exist).
GemmPlan choose(const GemmDesc& d, bool assume_aligned, int64_t capacity, int forced,
                int fsplits) {
  const bool can_async = assume_aligned ? (d.dtype == BF16 && d.lda % 8 == 0 && d.ldb % 8 == 0 &&
                                           d.K % 8 == 0 && d.ldc % 8 == 0 &&
                                           (!two_phase(d) || (d.lda2 % 8 == 0 && d.K1 % 8 == 0)))
                                        : async_ok(d);
  const TileShape* best = nullptr;
  int best_s = 1;
  double best_t = 0.0;
  for (const TileShape& t : kTiles) {
    if (t.cfg == 2 && d.N > 32) continue;  // the narrow tile only for narrow outputs
    if (t.cfg == 5 && forced != 5) continue;
    if (t.async && !can_async) continue;
    if (t.async && d.dtype == F32) continue;
    // Measured: where the direct-to-LDS kernels can run a bf16 product, the
    // register-staged 64 x 64 and 128 x 128 tiles are never faster (with one
    // workgroup per compute unit they cannot hide their load latency).
    if (can_async && (t.cfg == 0 || t.cfg == 1 || t.cfg == 4) && forced != t.cfg) continue;
    if ((t.cfg == 14 || t.cfg == 15) && !xl_ok(d)) continue;
    // The direct-to-LDS tiles load one-phase products through buffer
    // descriptors: operand extents below 2^31 bytes.
    if (t.async && !two_phase(d) && !xl_ok(d)) continue;
    // Measured on 16384 x 4096 x 4096: the four-wave kernel is the faster
    // one for the forward layout only; 15 runs only when forced.
    if (t.cfg == 14 && d.layout != Layout::NN && forced != 14) continue;
    if (t.cfg == 15 && forced != 15) continue;
    if (t.cfg == 16 && (d.layout == Layout::TN || forced != 16)) continue;
    if (t.cfg == 17 && forced != 17) continue;
    // The k-group tile: products whose caller asks for k-slices (the steps
    // of a recurrence, whose few output tiles are split over k to fill the
    // CUs). Measured on the 1024 x 1024 x 2048 cell and 1024 x 1024 x 1024
    // recurrent products, two slices on this tile against four on the
    // 128 x 128 tile: 17.3 against 16.9 us and 11.6 against 15.7 us. On the
    // 4096 x 1024 products of a whole batch it gains nothing over 16 in the
    // step, and a 64-deep contraction is slower.
    if (t.cfg == 19 && forced != 19) continue;
    if (t.cfg == 18 && (d.layout == Layout::TN ||
                        (forced != 18 && !(d.split_epilogue && d.splits_hint > 0))))
      continue;
    if (forced >= 0 && t.cfg != forced) continue;
    for (int sp = 1; sp <= kMaxSplits; sp *= 2) {
      // a two-phase product's slices must not straddle its phase boundary,
      // and on the direct-to-LDS tiles they load through descriptors
      if (sp > 1 && two_phase(d) && d.K1 % slice_k(d.K, sp) != 0) continue;
      if (sp > 1 && two_phase(d) && t.async && !assume_aligned && !xl_phases_ok(d)) continue;
      const bool forcing = fsplits > 0 && d.split_epilogue;  // (overrides the caller's split)
      if (!forcing && d.splits_hint > 0 && split_need(d, d.splits_hint) <= capacity) {
        // the caller's split (a multiple of 64 k per slice, whole slices)
        if (sp != d.splits_hint && !(sp == 1 && d.splits_hint == 1)) {
          if (sp > d.splits_hint) break;
          continue;
        }
      } else if (sp > 1) {
        if ((d.layout != Layout::TN && !d.split_epilogue) || capacity <= 0) break;
        if (slice_k(d.K, sp) < kMinChunk || ceil_div(d.K, slice_k(d.K, sp)) < sp) break;
        if (split_need(d, sp) > capacity) break;
      }
      if (forcing && sp != fsplits) continue;
      const double e = estimate(d, t, sp);
      if (best == nullptr || e < best_t * 0.97) {  // prefer earlier (larger) tiles, fewer splits
        best = &t;
        best_s = sp;
        best_t = e;
      }
    }
  }
  // Measured on 4096 x 1024 outputs (K 784 and 1024): where the 128 x 128
  // direct-to-LDS tile gives at most one tile per CU, the 64 x 128 tile (two
  // workgroups per CU, each running while the other waits on its loads) is
  // faster, even where it costs the paired adjoint launch. Only products
  // the planner keeps whole of their own accord (no split asked for by the
  // caller, no second phase).
  if (best != nullptr && best->cfg == 12 && best_s == 1 && forced < 0 && can_async &&
      d.layout != Layout::TN && !two_phase(d) && d.splits_hint == 0 &&
      ceil_div(d.M, 128) * ceil_div(d.N, 128) <= kComputeUnits) {
    for (const TileShape& t : kTiles)
      if (t.cfg == 16) best = &t;
  }
  // A product w.r.t. the weights split into k-slices that fill the CUs once:
  // the 128 x 128 tile of two k-groups of waves, same slices.
  if (best != nullptr && best->cfg == 12 && best_s > 1 && forced < 0 && fsplits < 0 &&
      can_async && d.layout == Layout::TN && !two_phase(d) && d.splits_hint == 0 &&
      ceil_div(d.M, 128) * ceil_div(d.N, 128) * best_s <= kComputeUnits) {
    for (const TileShape& t : kTiles)
      if (t.cfg == 19) best = &t;
  }
  if (best == nullptr) {  // a forced configuration or split that cannot run is ignored
    if (forced >= 0 || fsplits > 0) return choose(d, assume_aligned, capacity, -1, -1);
    best = &kTiles[3];      // (not reached: the 32 x 32 tile runs every product unsplit)
    best_s = 1;
  }
  GemmPlan pl{};
  pl.cfg = best->cfg;
  pl.bm = best->bm;
  pl.bn = best->bn;
  pl.tiles_m = static_cast<int>(ceil_div(d.M, pl.bm));
  pl.tiles_n = static_cast<int>(ceil_div(d.N, pl.bn));
  pl.k_chunk = best_s > 1 ? slice_k(d.K, best_s) : d.K;
  pl.splits = static_cast<int>(ceil_div(d.K, pl.k_chunk));
  return pl;
}

}  // namespace

int64_t chain_partials(const GemmPlan& pl) {
  // wavefronts of a tile (waves along M x N) of the register-staged configurations
  const int waves = (pl.cfg == 3 || pl.cfg == 5) ? 1 : 4;
  return static_cast<int64_t>(pl.tiles_m) * pl.tiles_n * waves;
}

GemmPlan plan_gemm(const GemmDesc& d) {
  return choose(d, false, d.split_ws != nullptr ? d.split_ws_elems : 0, forced_config(),
                forced_splits());
}

bool mask_ok(const GemmDesc& d, const GemmPlan& pl) {
  if (d.dtype != BF16 || d.out_dtype != BF16 || d.act != ACT_RELU) return false;
  if ((pl.cfg != 10 && pl.cfg != 16) || pl.splits != 1 || two_phase(d) || d.chain_epilogue)
    return false;
  return d.layout == Layout::NN || (d.layout == Layout::NT && d.residual == nullptr);
}

int64_t mask_bytes(int64_t M, int64_t N) {
  // one bit per element of whole tiles: 256 x 256 (config 10) or 64 x 128 (16)
  return std::max(ceil_div(M, 256) * ceil_div(N, 256) * 8192, ceil_div(M, 64) * ceil_div(N, 128) * 1024);
}

int64_t split_ws_elems(const GemmDesc& d) {
  if (d.layout != Layout::TN && !d.split_epilogue) return 0;
  const GemmPlan pl = choose(d, true, int64_t(1) << 40, forced_config(), forced_splits());
  return pl.splits > 1 ? split_need(d, pl.splits) : 0;
}

namespace {

// Whether 16-byte loads are legal for each operand of the register-staged
// kernel. 16-byte loads need 16-byte aligned rows (ld a multiple of the vector
// width). Along k a chunk must lie entirely inside or outside [0, K) (k
// padding would reach every output); along m or n a chunk that starts inside
// the extent stays inside its row, and its elements past the extent only reach
// outputs that are not stored.
void vector_ok(const GemmDesc& d, bool& va, bool& vb) {
  const int vw = d.dtype == F32 ? 4 : 8;
  va = aligned16(d.A) && d.lda % vw == 0;
  vb = aligned16(d.B) && d.ldb % vw == 0;
  switch (d.layout) {
    case Layout::NN: va = va && d.K % vw == 0; break;
    case Layout::NT: va = va && d.K % vw == 0; vb = vb && d.K % vw == 0; break;
    case Layout::TN: break;
  }
  // Two phases: every chunk along k inside or outside each phase's extent,
  // and 16-byte rows of A2.
  if (d.A2 != nullptr) {
    va = va && phases_ok(d, vw);
    if (d.layout != Layout::NN) vb = vb && d.K1 % vw == 0;
  }
}

// Whether a launch loads its operands through buffer descriptors (and needs
// their extents below 2^31 bytes): the bf16 direct-to-LDS and four-wave
// kernels, for one-phase products.
bool buffer_loads(const GemmDesc& d, const GemmPlan& pl) {
  if (two_phase(d) && pl.splits <= 1) return false;  // (unsplit: computed addresses)
  for (const TileShape& t : kTiles)
    if (t.cfg == pl.cfg) return t.async;
  return false;
}

gemm::Params make_params(const GemmDesc& d, const GemmPlan& pl) {
  gemm::Params p;
  p.M = d.M; p.N = d.N; p.K = d.K;
  p.A = d.A; p.lda = d.lda; p.B = d.B; p.ldb = d.ldb; p.C = d.C; p.ldc = d.ldc;
  p.bias = d.bias; p.aux = d.aux; p.residual = d.residual; p.colsum = d.colsum;
  p.alpha = d.alpha; p.act = d.act;
  p.tiles_m = pl.tiles_m; p.tiles_n = pl.tiles_n;
  p.nvec = d.nvec > 0 ? d.nvec : d.N;
  p.splits = pl.splits;
  p.k_chunk = pl.k_chunk;
  p.A2 = d.A2;
  p.lda2 = d.A2 != nullptr ? d.lda2 : 0;
  p.K1 = d.A2 != nullptr ? d.K1 : d.K;
  p.res_pre = d.res_pre ? 1 : 0;
  p.C2 = d.chain_epilogue ? d.C2 : nullptr;
  p.partials = d.chain_epilogue ? d.partials : nullptr;
  p.inv_n = d.inv_n;
  p.mask = d.mask;
  if (pl.splits > 1) {
    p.C = d.split_ws;                  // partial products, then partial column sums
    p.c_split = d.M * d.ldc;
    p.colsum = d.colsum != nullptr ? d.split_ws + pl.splits * p.c_split : nullptr;
    p.cs_split = p.nvec;
    if (d.layout != Layout::TN) {  // slices are raw products (the epilogue follows the sum)
      p.bias = p.aux = p.residual = nullptr;
      p.act = ACT_NONE;
      p.alpha = 1.0f;
      p.res_pre = 0;
    }
  } else {
    p.c_split = p.cs_split = 0;
  }
  // Extents for the buffer-descriptor loads (the planner runs these kernels
  // only where xl_ok holds; launch_gemm refuses them otherwise).
  p.a2_bytes = 0;
  if (buffer_loads(d, pl) && two_phase(d)) {  // k-slices of a two-phase forward product
    p.a_bytes = static_cast<uint32_t>(extent_bytes(d.M, d.K1, d.lda, 2));
    p.a2_bytes = static_cast<uint32_t>(extent_bytes(d.M, d.K - d.K1, d.lda2, 2));
    p.b_bytes = static_cast<uint32_t>(extent_bytes(d.K, d.N, d.ldb, 2));
  } else if (buffer_loads(d, pl)) {
    int64_t ar, ac, br, bc;
    operand_dims(d, ar, ac, br, bc);
    p.a_bytes = static_cast<uint32_t>(extent_bytes(ar, ac, d.lda, 2));
    p.b_bytes = static_cast<uint32_t>(extent_bytes(br, bc, d.ldb, 2));
  } else {
    p.a_bytes = p.b_bytes = 0;
  }
  return p;
}

unsigned grid_of(const GemmPlan& pl) {
  return static_cast<unsigned>(static_cast<int64_t>(pl.tiles_m) * pl.tiles_n * pl.splits);
}

}  // namespace

hipError_t launch_gemm(const GemmDesc& d, const GemmPlan& pl, hipStream_t s) {
  bool va, vb;
  vector_ok(d, va, vb);
  if (d.mask != nullptr && (!mask_ok(d, pl) || !aligned16(d.mask))) return hipErrorInvalidValue;
  if (buffer_loads(d, pl) && !(two_phase(d) ? xl_phases_ok(d) : xl_ok(d)))
    return hipErrorInvalidValue;
  const gemm::Params p = make_params(d, pl);
  const unsigned grid = grid_of(pl);
  const int out = pl.splits > 1 ? F32 : d.out_dtype;  // split slices: float32 partials
  switch (d.layout) {
    case Layout::NN: return gemm::launch_nn(p, d.dtype, out, pl.cfg, grid, va, vb, s);
    case Layout::NT: return gemm::launch_nt(p, d.dtype, out, pl.cfg, grid, va, vb, s);
    case Layout::TN: return gemm::launch_tn(p, d.dtype, pl.cfg, grid, va, vb, s);
  }
  return hipErrorInvalidValue;
}

bool pairable(const GemmDesc& tn, const GemmPlan& ptn, const GemmDesc& nt, const GemmPlan& pnt) {
  if (tn.layout != Layout::TN || nt.layout != Layout::NT || tn.dtype != nt.dtype) return false;
  if (ptn.cfg != pnt.cfg || !gemm::pair_config(tn.dtype, ptn.cfg)) return false;
  if ((buffer_loads(tn, ptn) && !xl_ok(tn)) || (buffer_loads(nt, pnt) && !xl_ok(nt))) return false;
  if (ptn.cfg < 10) {  // register-staged: 16-byte loads for all four operands
    bool a1, b1, a2, b2;
    vector_ok(tn, a1, b1);
    vector_ok(nt, a2, b2);
    if (!(a1 && b1 && a2 && b2)) return false;
  }
  return int64_t(grid_of(ptn)) + int64_t(grid_of(pnt)) < (int64_t(1) << 31);
}

hipError_t launch_gemm_pair(const GemmDesc& tn, const GemmPlan& ptn, const GemmDesc& nt,
                            const GemmPlan& pnt, hipStream_t s) {
  if (tn.mask != nullptr) return hipErrorInvalidValue;
  if ((buffer_loads(tn, ptn) && !xl_ok(tn)) || (buffer_loads(nt, pnt) && !xl_ok(nt)))
    return hipErrorInvalidValue;
  if (nt.mask != nullptr && (!mask_ok(nt, pnt) || !aligned16(nt.mask))) return hipErrorInvalidValue;
  const gemm::Params p1 = make_params(tn, ptn), p2 = make_params(nt, pnt);
  const unsigned n1 = grid_of(ptn);
  return gemm::launch_pair(p1, p2, static_cast<int>(n1), n1 + grid_of(pnt), tn.dtype,
                           nt.out_dtype, ptn.cfg, s);
}

}  // namespace dlvm
