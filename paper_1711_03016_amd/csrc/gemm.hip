// Host side of the dense-layer products: choice of the tile configuration for
// a given problem, and the launch.
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
// when not starved. Configurations 0-4 are the register-staged kernel
// (gemm_kernel.hpp), 10-13 the bf16 kernel with direct-to-LDS loads
// (gemm_async.hpp).
struct TileShape {
  int cfg;
  int bm, bn;
  double eff;
  bool async;
};
constexpr TileShape kTiles[] = {
    {0, 128, 128, 0.8, false}, {1, 64, 64, 0.6, false},   {2, 128, 32, 0.6, false},
    {3, 32, 32, 0.5, false},   {4, 64, 64, 0.65, false},  {5, 32, 32, 0.5, false},  {10, 256, 256, 0.9, true},
    {11, 256, 128, 0.7, true}, {12, 128, 128, 0.84, true}, {13, 256, 256, 0.85, true}};

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool aligned16(const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15u) == 0; }

// The direct-to-LDS kernel moves whole 16-byte chunks: bf16 operands with
// 16-byte aligned bases, leading dimensions and contraction extent; its
// epilogue moves 8 consecutive outputs at a time (16-byte aligned output rows,
// saved activation and residual).
bool async_ok(const GemmDesc& d) {
  return d.dtype == BF16 && aligned16(d.A) && aligned16(d.B) && d.lda % 8 == 0 &&
         d.ldb % 8 == 0 && d.K % 8 == 0 && d.ldc % 8 == 0 && aligned16(d.C) &&
         aligned16(d.aux) && aligned16(d.residual) && aligned16(d.bias);
}

// Clock cycles one configuration needs: rounds of tiles over the compute
// units, each tile bound by its matrix-core work or its operand traffic.
double estimate(const GemmDesc& d, const TileShape& t) {
  const int64_t tiles = ceil_div(d.M, t.bm) * ceil_div(d.N, t.bn);
  const double es = d.dtype == F32 ? 4.0 : 2.0;
  const double rate = (d.dtype == F32 ? kRateF32 : kRateBF16) * t.eff;
  const double flops = 2.0 * t.bm * t.bn * double(d.K);
  const double bytes = double(t.bm + t.bn) * double(d.K) * es;
  const double per_tile = std::max(flops / rate, bytes / kL2BytesPerClock);
  return double(ceil_div(tiles, kComputeUnits)) * per_tile;
}

}  // namespace

// Tile configuration forced through the environment variable
// DLVM_GEMM_CONFIG (for tests and tuning), or -1. A forced configuration that
// cannot run the product is ignored.
int forced_config() {
  const char* v = std::getenv("DLVM_GEMM_CONFIG");
  if (v == nullptr || *v == 0) return -1;
  char* end = nullptr;
  const long c = std::strtol(v, &end, 10);
  return (end != nullptr && *end == 0) ? static_cast<int>(c) : -1;
}

GemmPlan plan_gemm(const GemmDesc& d) {
  const bool can_async = async_ok(d);
  const int forced = forced_config();
  const TileShape* best = nullptr;
  double best_t = 0.0;
  for (const TileShape& t : kTiles) {
    if (t.cfg == 2 && d.N > 32) continue;  // the narrow tile only for narrow outputs
    if (t.cfg == 5 && forced != 5) continue;
    if (t.async && !can_async) continue;
    if (t.cfg == forced) {
      best = &t;
      break;
    }
    const double e = estimate(d, t);
    if (best == nullptr || e < best_t * 0.97) {  // prefer earlier (larger) tiles on near ties
      best = &t;
      best_t = e;
    }
  }
  GemmPlan pl{};
  pl.cfg = best->cfg;
  pl.bm = best->bm;
  pl.bn = best->bn;
  pl.tiles_m = static_cast<int>(ceil_div(d.M, pl.bm));
  pl.tiles_n = static_cast<int>(ceil_div(d.N, pl.bn));
  return pl;
}

hipError_t launch_gemm(const GemmDesc& d, const GemmPlan& pl, hipStream_t s) {
  const int vw = d.dtype == F32 ? 4 : 8;
  // 16-byte loads need 16-byte aligned rows (ld a multiple of the vector
  // width). Along k a chunk must lie entirely inside or outside [0, K) (k
  // padding would reach every output); along m or n a chunk that starts inside
  // the extent stays inside its row, and its elements past the extent only
  // reach outputs that are not stored.
  bool va = aligned16(d.A) && d.lda % vw == 0;
  bool vb = aligned16(d.B) && d.ldb % vw == 0;
  switch (d.layout) {
    case Layout::NN: va = va && d.K % vw == 0; break;
    case Layout::NT: va = va && d.K % vw == 0; vb = vb && d.K % vw == 0; break;
    case Layout::TN: break;
  }
  gemm::Params p;
  p.M = d.M; p.N = d.N; p.K = d.K;
  p.A = d.A; p.lda = d.lda; p.B = d.B; p.ldb = d.ldb; p.C = d.C; p.ldc = d.ldc;
  p.bias = d.bias; p.aux = d.aux; p.residual = d.residual; p.colsum = d.colsum;
  p.alpha = d.alpha; p.act = d.act;
  p.tiles_m = pl.tiles_m; p.tiles_n = pl.tiles_n;
  p.nvec = d.nvec > 0 ? d.nvec : d.N;
  const unsigned grid = static_cast<unsigned>(static_cast<int64_t>(pl.tiles_m) * pl.tiles_n);
  switch (d.layout) {
    case Layout::NN: return gemm::launch_nn(p, d.dtype, d.out_dtype, pl.cfg, grid, va, vb, s);
    case Layout::NT: return gemm::launch_nt(p, d.dtype, d.out_dtype, pl.cfg, grid, va, vb, s);
    case Layout::TN: return gemm::launch_tn(p, d.dtype, pl.cfg, grid, va, vb, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace dlvm
