// Decoding state between denoising forwards (Section 3.1, Eq. (1)).
//
// One workgroup per sequence.  Pass 1 counts the masked active-block positions
// whose confidence reaches theta, finds the most confident of them (for the
// optional progress guard: highest confidence, then lowest position, as one
// 64-bit key) and the sequence's last block.  Pass 2 commits, shifts the
// confidence history of every position that was masked, and counts what is
// left; the sequence advances to its next block when its active block is empty.
#include "common.h"

namespace rfx {
namespace {

constexpr int ST_THREADS = 256;
constexpr int ST_WAVES = ST_THREADS / kWave;

__device__ __forceinline__ int wave_max_i32(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const int w = __shfl_xor(v, o, kWave);
    v = w > v ? w : v;
  }
  return v;
}

__global__ __launch_bounds__(ST_THREADS) void advance_state_kernel(
    const float* __restrict__ conf_t, const int32_t* __restrict__ block_idx,
    const int32_t* __restrict__ seq_offsets, int T, float theta, int min_commit,
    uint8_t* __restrict__ masked, int8_t* __restrict__ hist_len, float* __restrict__ c1,
    float* __restrict__ c2, int32_t* __restrict__ active_block, int32_t* __restrict__ remaining) {
  __shared__ int s_cnt[ST_WAVES], s_last[ST_WAVES], s_left[ST_WAVES], s_rem[ST_WAVES];
  __shared__ uint64_t s_best[ST_WAVES];
  const int s = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  int lo = seq_offsets[s], hi = seq_offsets[s + 1];
  lo = lo < 0 ? 0 : (lo > T ? T : lo);
  hi = hi < lo ? lo : (hi > T ? T : hi);
  const int a = active_block[s];

  int n_commit = 0, last = a;
  uint64_t best = 0;
  for (int i = lo + tid; i < hi; i += ST_THREADS) {
    const int b = block_idx[i];
    last = b > last ? b : last;
    if (masked[i] != 0 && b == a) {
      const float c = conf_t[i];
      n_commit += c >= theta ? 1 : 0;
      const uint64_t key = (static_cast<uint64_t>(f32_order_key(c)) << 32) |
                           (0xffffffffu - static_cast<uint32_t>(i));
      best = key > best ? key : best;
    }
  }
  n_commit = wave_sum_i32(n_commit);
  last = wave_max_i32(last);
  best = wave_max_u64(best);
  if (lane == 0) {
    s_cnt[wv] = n_commit;
    s_last[wv] = last;
    s_best[wv] = best;
  }
  __syncthreads();
  n_commit = 0;
  last = a;
  best = 0;
#pragma unroll
  for (int x = 0; x < ST_WAVES; ++x) {
    n_commit += s_cnt[x];
    last = s_last[x] > last ? s_last[x] : last;
    best = s_best[x] > best ? s_best[x] : best;
  }
  // progress guard: commit the most confident masked active position when none
  // reaches theta (best == 0: the active block has no masked position)
  const bool guard = min_commit != 0 && n_commit == 0 && best != 0;
  const int g = guard ? static_cast<int>(0xffffffffu - static_cast<uint32_t>(best & 0xffffffffu)) : -1;

  int left = 0, rem = 0;
  for (int i = lo + tid; i < hi; i += ST_THREADS) {
    if (masked[i] == 0) continue;
    const int b = block_idx[i];
    const float c = conf_t[i];
    c2[i] = c1[i];
    c1[i] = c;
    const int hl = hist_len[i];
    hist_len[i] = static_cast<int8_t>(hl + 1 < 2 ? hl + 1 : 2);
    if (b == a && (c >= theta || i == g)) {
      masked[i] = 0;
    } else {
      ++rem;
      left += b == a ? 1 : 0;
    }
  }
  left = wave_sum_i32(left);
  rem = wave_sum_i32(rem);
  if (lane == 0) {
    s_left[wv] = left;
    s_rem[wv] = rem;
  }
  __syncthreads();
  if (tid == 0) {
    int l = 0, r = 0;
#pragma unroll
    for (int x = 0; x < ST_WAVES; ++x) {
      l += s_left[x];
      r += s_rem[x];
    }
    if (l == 0 && a < last) active_block[s] = a + 1;
    if (remaining != nullptr) remaining[s] = r;
  }
}

}  // namespace

int launch_advance_state(const float* conf_t, const int32_t* block_idx, const int32_t* seq_offsets,
                         int B, int T, float theta, int min_commit, uint8_t* masked,
                         int8_t* hist_len, float* c1, float* c2, int32_t* active_block,
                         int32_t* remaining, hipStream_t s) {
  hipLaunchKernelGGL(advance_state_kernel, dim3(B), dim3(ST_THREADS), 0, s, conf_t, block_idx,
                     seq_offsets, T, theta, min_commit, masked, hist_len, c1, c2, active_block,
                     remaining);
  return launch_status();
}

}  // namespace rfx
