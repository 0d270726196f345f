// Router scores r = h W_r^T (+ bias), Section 3.2: the launch (the tile code and its
// description are in router_impl.h).
#include "router_impl.h"

namespace rfx {
namespace {

template <int TM, int EB, int KSPLIT, int PF>
__global__ __launch_bounds__(64 * KSPLIT) void router_mfma_kernel(const uint16_t* __restrict__ h,
                                                                 const float* __restrict__ w,
                                                                 const float* __restrict__ bias,
                                                                 float* __restrict__ logits, int T,
                                                                 int d, int E) {
  router_tile<TM, EB, KSPLIT, PF>(blockIdx.x, blockIdx.y, h, w, bias, logits, T, d, E);
}

}  // namespace

int launch_router(const uint16_t* h, const float* w, const float* bias, float* logits, int T,
                  int d, int E, hipStream_t s) {
  // A workgroup's loads all pass through one CU, so tiles are sized to spread the
  // traffic over many CUs: small T uses 16 x 16 tiles with K split over 16 waves;
  // large T uses 64 x 64 tiles so each W_r fragment feeds 4 token blocks.
  if (T >= 4096) {
    hipLaunchKernelGGL((router_mfma_kernel<64, 4, 4, 2>), dim3((T + 63) / 64, (E + 63) / 64),
                       dim3(256), 0, s, h, w, bias, logits, T, d, E);
  } else if (d % (RT_TK * 16) == 0) {
    hipLaunchKernelGGL((router_mfma_kernel<16, 1, 16, 4>), dim3((T + 15) / 16, (E + 15) / 16),
                       dim3(1024), 0, s, h, w, bias, logits, T, d, E);
  } else {
    hipLaunchKernelGGL((router_mfma_kernel<16, 1, 4, 4>), dim3((T + 15) / 16, (E + 15) / 16),
                       dim3(256), 0, s, h, w, bias, logits, T, d, E);
  }
  return launch_status();
}

}  // namespace rfx
