// Instantiations of the dense-layer product for the NT layout (adjoint with respect to the layer
// input: activation-derivative epilogue).
#include "gemm_xl.hpp"

namespace dlvm {
namespace gemm {

hipError_t launch_nt(const Params& p, int dtype, int out_dtype, int cfg, unsigned grid, bool va,
                     bool vb, hipStream_t s) {
  if (dtype == F32) return launch_vec<float, float, true, true, EPI_DACT>(p, cfg, grid, va, vb, s);
  if (cfg >= kAsyncFirst) {
    if (out_dtype == F32) return launch_bf16<float, true, true, EPI_DACT>(p, cfg, grid, s);
    return launch_bf16<bf16_t, true, true, EPI_DACT>(p, cfg, grid, s);
  }
  if (out_dtype == F32) return launch_vec<bf16_t, float, true, true, EPI_DACT>(p, cfg, grid, va, vb, s);
  return launch_vec<bf16_t, bf16_t, true, true, EPI_DACT>(p, cfg, grid, va, vb, s);
}

}  // namespace gemm
}  // namespace dlvm
