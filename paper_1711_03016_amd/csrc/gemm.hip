// Host side of the dense-layer products: choice of the tile configuration for
// a given problem, and the launch.
#include "gemm_kernel.hpp"

namespace dlvm {

namespace {

// Compute units of an MI355X and per-compute-unit rates the planner assumes:
// matrix-core flops per clock (float32, bf16) and L2 bytes per clock.
constexpr int kComputeUnits = 256;
constexpr double kRateF32 = 256.0;
constexpr double kRateBF16 = 4096.0;
constexpr double kL2BytesPerClock = 64.0;

// Tile configurations of the kernel template (see gemm_kernel.hpp) with the
// fraction of the matrix-core rate each sustains when not starved.
struct TileShape {
  int bm, bn;
  double eff;
};
constexpr TileShape kTiles[5] = {
    {128, 128, 0.8}, {64, 64, 0.6}, {128, 32, 0.6}, {32, 32, 0.5}, {64, 64, 0.65}};

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool aligned16(const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15u) == 0; }

// Clock cycles one configuration needs: rounds of tiles over the compute
// units, each tile bound by its matrix-core work or its operand traffic.
double estimate(const GemmDesc& d, int cfg) {
  const TileShape& t = kTiles[cfg];
  const int64_t tiles = ceil_div(d.M, t.bm) * ceil_div(d.N, t.bn);
  const double es = d.dtype == F32 ? 4.0 : 2.0;
  const double rate = (d.dtype == F32 ? kRateF32 : kRateBF16) * t.eff;
  const double flops = 2.0 * t.bm * t.bn * double(d.K);
  const double bytes = double(t.bm + t.bn) * double(d.K) * es;
  const double per_tile = std::max(flops / rate, bytes / kL2BytesPerClock);
  return double(ceil_div(tiles, kComputeUnits)) * per_tile;
}

}  // namespace

GemmPlan plan_gemm(const GemmDesc& d) {
  int best = 0;
  double best_t = 0.0;
  for (int cfg = 0; cfg < 5; ++cfg) {
    if (cfg == 2 && d.N > 32) continue;  // the narrow tile only for narrow outputs
    const double t = estimate(d, cfg);
    if (cfg == 0 || t < best_t * 0.97) {  // prefer earlier (larger) tiles on near ties
      best = cfg;
      best_t = t;
    }
  }
  GemmPlan pl{};
  pl.cfg = best;
  pl.bm = kTiles[best].bm;
  pl.bn = kTiles[best].bn;
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
