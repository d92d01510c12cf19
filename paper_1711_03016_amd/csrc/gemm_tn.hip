// Instantiations of the dense-layer product for the TN layout (adjoint with respect to the
// weights: float32 dW plus the bias-gradient column sums).
#include "gemm_xl.hpp"

namespace dlvm {
namespace gemm {

hipError_t launch_tn(const Params& p, int dtype, int cfg, unsigned grid, bool va, bool vb,
                     hipStream_t s) {
  if (dtype == F32) return launch_vec<float, float, false, false, EPI_DW>(p, cfg, grid, va, vb, s);
  if (cfg >= kAsyncFirst) return launch_bf16<float, false, false, EPI_DW>(p, cfg, grid, s);
  return launch_vec<bf16_t, float, false, false, EPI_DW>(p, cfg, grid, va, vb, s);
}

}  // namespace gemm
}  // namespace dlvm
