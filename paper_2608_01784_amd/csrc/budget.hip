// Per-token expert counts of one denoising forward (the device code and its
// description are in budget_impl.h), the constant fill and the count scan.
#include "budget_impl.h"

namespace rfx {
namespace {

constexpr int BG_KERNEL_THREADS = 1024;

__global__ __launch_bounds__(BG_KERNEL_THREADS) void budget_kernel(
    const int32_t* __restrict__ block_idx, const uint8_t* __restrict__ masked,
    const int8_t* __restrict__ hist_len, const float* __restrict__ c1,
    const float* __restrict__ c2, const int32_t* __restrict__ seq_offsets,
    const int32_t* __restrict__ active_block, int T, BudgetConsts p,
    int32_t* __restrict__ k_out, int32_t* __restrict__ pairs_out, double* __restrict__ fps_out) {
  budget_sequence<BG_KERNEL_THREADS>(blockIdx.x, block_idx, masked, hist_len, c1, c2, seq_offsets,
                                     active_block, T, p, k_out, pairs_out, fps_out);
}

__global__ void fill_i32_kernel(int32_t* dst, int32_t v, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = v;
}

// Exclusive prefix sum of the clamped counts: pair_offsets[0..T], P = pair_offsets[T].
// One workgroup walks the counts in slices of 4096 carrying the running total.
__global__ __launch_bounds__(1024) void count_scan_kernel(const int32_t* __restrict__ k, int T,
                                                          int k_max,
                                                          int32_t* __restrict__ pair_offsets,
                                                          int32_t* __restrict__ pairs_out) {
  __shared__ int s_wave[16];
  __shared__ int s_carry;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (tid == 0) s_carry = 0;
  __syncthreads();
  for (int base = 0; base < T; base += 4096) {
    int v[4];
    int sum = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = base + tid * 4 + j;
      v[j] = i < T ? clamp_count(k[i], k_max) : 0;
      sum += v[j];
    }
    const int incl = wave_inclusive_scan_i32(sum, lane);
    if (lane == 63) s_wave[wv] = incl;
    __syncthreads();
    int wave_off = 0;
    for (int x = 0; x < wv; ++x) wave_off += s_wave[x];
    int run = s_carry + wave_off + incl - sum;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = base + tid * 4 + j;
      if (i < T) pair_offsets[i] = run;
      run += v[j];
    }
    __syncthreads();
    if (tid == 1023) s_carry = run;
    __syncthreads();
  }
  if (tid == 0) {
    pair_offsets[T] = s_carry;
    if (pairs_out) pairs_out[0] = s_carry;
  }
}

}  // namespace

int launch_fill_i32(int32_t* dst, int32_t value, int n, hipStream_t s) {
  if (n <= 0) return REFLEX_OK;
  hipLaunchKernelGGL(fill_i32_kernel, dim3((n + 255) / 256), dim3(256), 0, s, dst, value, n);
  return launch_status();
}

int launch_budget(const int32_t* block_idx, const uint8_t* masked, const int8_t* hist_len,
                  const float* c1, const float* c2, const int32_t* seq_offsets,
                  const int32_t* active_block, int B, int T, const reflex_alloc_params& prm,
                  int32_t* k_out, int32_t* pairs_out, double* fps_out, hipStream_t s) {
  const BudgetConsts p = budget_consts(prm);
  if (pairs_out != nullptr) {
    const int rc = launch_fill_i32(pairs_out, 0, 1, s);
    if (rc != REFLEX_OK) return rc;
  }
  hipLaunchKernelGGL(budget_kernel, dim3(B), dim3(BG_KERNEL_THREADS), 0, s, block_idx, masked,
                     hist_len, c1, c2, seq_offsets, active_block, T, p, k_out, pairs_out, fps_out);
  return launch_status();
}

int launch_count_scan(const int32_t* k, int T, int k_max, int32_t* pair_offsets,
                      int32_t* pairs_out, hipStream_t s) {
  hipLaunchKernelGGL(count_scan_kernel, dim3(1), dim3(1024), 0, s, k, T, k_max, pair_offsets,
                     pairs_out);
  return launch_status();
}

}  // namespace rfx
