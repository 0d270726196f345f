// Router scores and the REFLEX counts in one launch (Sections 3.2, 4.2, 4.3).  The
// two are independent, so the first B workgroups compute the counts of one sequence
// each while the rest compute split-K partial score tiles (router_split_tile); the
// counts' long dependent chain then overlaps the score tiles instead of following
// them.  The route kernel adds the partials of each score.
#include "budget_impl.h"
#include "router_impl.h"

namespace rfx {
namespace {

__global__ __launch_bounds__(RS_THREADS) void front_kernel(
    const uint16_t* __restrict__ h, const float* __restrict__ w, float* __restrict__ parts, int T,
    int d, int E, int gy, int n_slices, const int32_t* __restrict__ block_idx,
    const uint8_t* __restrict__ masked, const int8_t* __restrict__ hist_len,
    const float* __restrict__ c1, const float* __restrict__ c2,
    const int32_t* __restrict__ seq_offsets, const int32_t* __restrict__ active_block, int B,
    BudgetConsts p, int32_t* __restrict__ k_out, int32_t* __restrict__ zero_word) {
  const int b = blockIdx.x;
  if (zero_word != nullptr && b == 0 && threadIdx.x == 0) *zero_word = 0;
  if (b < B) {
    budget_sequence<RS_THREADS>(b, block_idx, masked, hist_len, c1, c2, seq_offsets, active_block,
                                T, p, k_out, nullptr, nullptr);
    return;
  }
  // score tiles: K slice fastest, then expert block, then token block
  const int r = b - B;
  const int ks = r % n_slices, rest = r / n_slices;
  router_split_tile(rest / gy, rest % gy, ks, h, w, parts, T, d, E);
}

}  // namespace

bool front_fits(int T, int d) { return T < 4096 && d % RS_KS == 0; }

int front_slices(int d) { return d / RS_KS; }

int launch_front(const uint16_t* h, const float* w, float* parts, int T, int d, int E,
                 const int32_t* block_idx, const uint8_t* masked, const int8_t* hist_len,
                 const float* c1, const float* c2, const int32_t* seq_offsets,
                 const int32_t* active_block, int B, const reflex_alloc_params& prm, int32_t* k_out,
                 hipStream_t s, int32_t* zero_word) {
  const int gx = (T + RS_TM - 1) / RS_TM, gy = (E + RS_TE - 1) / RS_TE, ns = front_slices(d);
  hipLaunchKernelGGL(front_kernel, dim3(B + gx * gy * ns), dim3(RS_THREADS), 0, s, h, w, parts, T,
                     d, E, gy, ns, block_idx, masked, hist_len, c1, c2, seq_offsets, active_block,
                     B, budget_consts(prm), k_out, zero_word);
  return launch_status();
}

}  // namespace rfx
