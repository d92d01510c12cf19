// Instantiations of the paired launch of a layer's two adjoint products (TN
// wrt the weights, NT wrt the input): register-staged configurations 0 and 3,
// direct-to-LDS configurations 10 and 12.
#include "gemm_xl.hpp"

namespace dlvm {
namespace gemm {

bool pair_config(int dtype, int cfg) {
  if (dtype == F32) return cfg == 0 || cfg == 3;
  return cfg == 3 || cfg == 10 || cfg == 12;
}

namespace {

template <typename T, typename TO2>
hipError_t launch_reg_pair(const Params& p1, const Params& p2, int n1, unsigned grid, int cfg,
                           hipStream_t s) {
  if (cfg == 0)
    launch_kernel((dlvm_gemm_pair_kernel<T, TO2, 128, 128, 2, 2, 1, 1>), dim3(grid), dim3(256), s,
                  p1, p2, n1);
  else
    launch_kernel((dlvm_gemm_pair_kernel<T, TO2, 32, 32, 1, 1, 4, 4>), dim3(grid), dim3(256), s,
                  p1, p2, n1);
  return hipGetLastError();
}

template <typename TO2>
hipError_t launch_async_pair(const Params& p1, const Params& p2, int n1, unsigned grid, int cfg,
                             hipStream_t s) {
  if (cfg == 10)
    launch_kernel((dlvm_gemm_async_pair_kernel<TO2, 256, 256, 64, 2, 4, 2>), dim3(grid),
                  dim3(512), s, p1, p2, n1);
  else
    launch_kernel((dlvm_gemm_async_pair_kernel<TO2, 128, 128, 64, 2, 2, 4>), dim3(grid),
                  dim3(256), s, p1, p2, n1);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_pair(const Params& p1, const Params& p2, int n1, unsigned grid, int dtype,
                       int out_dtype2, int cfg, hipStream_t s) {
  if (dtype == F32) return launch_reg_pair<float, float>(p1, p2, n1, grid, cfg, s);
  if (cfg >= kAsyncFirst) {
    if (out_dtype2 == F32) return launch_async_pair<float>(p1, p2, n1, grid, cfg, s);
    return launch_async_pair<bf16_t>(p1, p2, n1, grid, cfg, s);
  }
  if (out_dtype2 == F32) return launch_reg_pair<bf16_t, float>(p1, p2, n1, grid, cfg, s);
  return launch_reg_pair<bf16_t, bf16_t>(p1, p2, n1, grid, cfg, s);
}

}  // namespace gemm
}  // namespace dlvm
