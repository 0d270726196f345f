// Router scores and the REFLEX counts in one launch (Sections 3.2, 4.2, 4.3).  The
// two are independent, so the first B workgroups compute the counts of one sequence
// each while the rest compute score tiles; the counts' long dependent chain then
// overlaps the score tiles instead of following them.  Used for the small-T router
// shape (16 x 16 tiles, 16 waves), whose LDS use leaves room for the count code's.
#include "budget_impl.h"
#include "router_impl.h"

namespace rfx {
namespace {

template <int TM, int EB, int KSPLIT, int PF>
__global__ __launch_bounds__(64 * KSPLIT) void front_kernel(
    const uint16_t* __restrict__ h, const float* __restrict__ w, const float* __restrict__ bias,
    float* __restrict__ logits, int T, int d, int E, int gx, const int32_t* __restrict__ block_idx,
    const uint8_t* __restrict__ masked, const int8_t* __restrict__ hist_len,
    const float* __restrict__ c1, const float* __restrict__ c2,
    const int32_t* __restrict__ seq_offsets, const int32_t* __restrict__ active_block, int B,
    BudgetConsts p, int32_t* __restrict__ k_out, int32_t* __restrict__ zero_word) {
  const int b = blockIdx.x;
  if (zero_word != nullptr && b == 0 && threadIdx.x == 0) *zero_word = 0;
  if (b < B) {
    budget_sequence<64 * KSPLIT>(b, block_idx, masked, hist_len, c1, c2, seq_offsets, active_block,
                                 T, p, k_out, nullptr, nullptr);
    return;
  }
  const int r = b - B;
  router_tile<TM, EB, KSPLIT, PF>(r % gx, r / gx, h, w, bias, logits, T, d, E);
}

}  // namespace

bool front_fits(int T, int d) { return T < 4096 && d % (RT_TK * 16) == 0; }

int launch_front(const uint16_t* h, const float* w, const float* bias, float* logits, int T, int d,
                 int E, const int32_t* block_idx, const uint8_t* masked, const int8_t* hist_len,
                 const float* c1, const float* c2, const int32_t* seq_offsets,
                 const int32_t* active_block, int B, const reflex_alloc_params& prm, int32_t* k_out,
                 hipStream_t s, int32_t* zero_word) {
  // One 1024-thread workgroup fits a CU: with more workgroups than CUs the last ones
  // wait for a CU to free up and the launch takes two rounds.  32-token score tiles
  // halve the grid where 16-token tiles would overflow it.
  const int gy = (E + 15) / 16;
  if (B + ((T + 15) / 16) * gy > device_cus()) {
    const int gx = (T + 31) / 32;
    hipLaunchKernelGGL((front_kernel<32, 1, 16, 4>), dim3(B + gx * gy), dim3(1024), 0, s, h, w,
                       bias, logits, T, d, E, gx, block_idx, masked, hist_len, c1, c2,
                       seq_offsets, active_block, B, budget_consts(prm), k_out, zero_word);
    return launch_status();
  }
  const int gx = (T + 15) / 16;
  hipLaunchKernelGGL((front_kernel<16, 1, 16, 4>), dim3(B + gx * gy), dim3(1024), 0, s, h, w, bias,
                     logits, T, d, E, gx, block_idx, masked, hist_len, c1, c2, seq_offsets,
                     active_block, B, budget_consts(prm), k_out, zero_word);
  return launch_status();
}

}  // namespace rfx
