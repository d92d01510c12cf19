// Instantiations of the dense-layer product for the NN layout (forward products: bias + activation
// epilogue).
#include "gemm_xl.hpp"

namespace dlvm {
namespace gemm {

hipError_t launch_nn(const Params& p, int dtype, int out_dtype, int cfg, unsigned grid, bool va,
                     bool vb, hipStream_t s) {
  if (p.A2 != nullptr) {  // a two-phase contraction: the kernels that choose A per k-tile
    if (dtype == F32)
      return launch_vec<float, float, true, false, EPI_STORE, true>(p, cfg, grid, va, vb, s);
    if (cfg >= kAsyncFirst) {
      if (out_dtype == F32) return launch_async<float, true, false, EPI_STORE, true>(p, cfg, grid, s);
      return launch_async<bf16_t, true, false, EPI_STORE, true>(p, cfg, grid, s);
    }
    if (out_dtype == F32)
      return launch_vec<bf16_t, float, true, false, EPI_STORE, true>(p, cfg, grid, va, vb, s);
    return launch_vec<bf16_t, bf16_t, true, false, EPI_STORE, true>(p, cfg, grid, va, vb, s);
  }
  if (p.partials != nullptr) {  // the eight-operator chain in the epilogue (float32)
    if (dtype != F32 || p.splits > 1) return hipErrorInvalidValue;
    return launch_vec<float, float, true, false, EPI_CHAIN>(p, cfg, grid, va, vb, s);
  }
  if (dtype == F32) return launch_vec<float, float, true, false, EPI_STORE>(p, cfg, grid, va, vb, s);
  if (cfg >= kAsyncFirst) {
    if (out_dtype == F32) return launch_bf16<float, true, false, EPI_STORE>(p, cfg, grid, s);
    return launch_bf16<bf16_t, true, false, EPI_STORE>(p, cfg, grid, s);
  }
  if (out_dtype == F32) return launch_vec<bf16_t, float, true, false, EPI_STORE>(p, cfg, grid, va, vb, s);
  return launch_vec<bf16_t, bf16_t, true, false, EPI_STORE>(p, cfg, grid, va, vb, s);
}

}  // namespace gemm
}  // namespace dlvm
