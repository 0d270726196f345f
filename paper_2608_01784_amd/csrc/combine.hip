// Weighted combine of Eq. (2): out_i = sum_{e in T_i} alpha_{i,e} E_e(h_i), plus the
// always-on shared expert and optional residual streams, accumulated in fp32 in
// the token's rank order and rounded to bf16 once.
//
// One workgroup per token; each thread owns 8 consecutive hidden elements
// (16-byte loads and stores), so every expert row is read once, coalesced.
#include "common.h"

namespace rfx {
namespace {

__device__ __forceinline__ void add_bf16x8(float* acc, uint4 v, float w) {
  const uint32_t x[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    acc[2 * j] = __builtin_fmaf(w, __uint_as_float(x[j] << 16), acc[2 * j]);
    acc[2 * j + 1] = __builtin_fmaf(w, __uint_as_float(x[j] & 0xffff0000u), acc[2 * j + 1]);
  }
}

// CB: expert rows in flight per batch.  16 keep a token's rows in one batch on the small
// layers; from T = 4096 up, 8 (fewer registers, more workgroups resident per CU) are
// faster (16-layer stack layer: 35.1 against 42.1 us; LLaDA-MoE layer: 7.4 against 7.1).
template <int CB>
__global__ __launch_bounds__(256) void combine_kernel(
    const uint16_t* __restrict__ y, const int32_t* __restrict__ pair_offsets,
    const int32_t* __restrict__ pair_to_sorted, const float* __restrict__ pair_weight,
    const uint16_t* __restrict__ shared_y, const uint16_t* __restrict__ res_a,
    const uint16_t* __restrict__ res_b, int d, int cap, uint16_t* __restrict__ out) {
  const int i = blockIdx.x;
  int p0 = pair_offsets[i], p1 = pair_offsets[i + 1];
  p0 = p0 < 0 ? 0 : (p0 > cap ? cap : p0);
  p1 = p1 < p0 ? p0 : (p1 > cap ? cap : p1);
  const size_t tok_off = static_cast<size_t>(i) * d;
  // the token's pair rows and weights, lane j of every wave holding pair p0 + j (one
  // vector load each instead of a scalar load per pair ahead of its row load); a
  // forward's count is at most REFLEX_MAX_K <= 64
  const int lane = threadIdx.x & 63, np = p1 - p0;
  int prow = 0;
  float pw = 0.0f;
  if (lane < np) {
    prow = pair_to_sorted[p0 + lane];
    prow = prow < 0 ? 0 : (prow >= cap ? cap - 1 : prow);
    pw = pair_weight[p0 + lane];
  }
  for (int v = threadIdx.x * 8; v < d; v += 256 * 8) {
    // the token's own rows (shared expert, residuals) are loaded first, so they are in
    // flight with the expert rows; they are still added after them, in the same order
    const uint4 zero = make_uint4(0, 0, 0, 0);
    const uint4 sv = shared_y ? *reinterpret_cast<const uint4*>(shared_y + tok_off + v) : zero;
    const uint4 av = res_a ? *reinterpret_cast<const uint4*>(res_a + tok_off + v) : zero;
    const uint4 bv = res_b ? *reinterpret_cast<const uint4*>(res_b + tok_off + v) : zero;
    float acc[8] = {};
    if (np > kWave) {          // (more pairs than lanes: only through reflex_combine)
      for (int p = p0; p < p1; ++p) {
        int row = pair_to_sorted[p];
        row = row < 0 ? 0 : (row >= cap ? cap - 1 : row);
        add_bf16x8(acc, *reinterpret_cast<const uint4*>(y + static_cast<size_t>(row) * d + v),
                   pair_weight[p]);
      }
    }
    for (int q = 0; q < (np > kWave ? 0 : np); q += CB) {
      uint4 r[CB];
#pragma unroll
      for (int u = 0; u < CB; ++u) {     // past the count: the last row again, not added
        const int row = __builtin_amdgcn_readlane(prow, min(q + u, np - 1));
        r[u] = *reinterpret_cast<const uint4*>(y + static_cast<size_t>(row) * d + v);
      }
#pragma unroll
      for (int u = 0; u < CB; ++u)
        if (q + u < np)
          add_bf16x8(acc, r[u], __int_as_float(__builtin_amdgcn_readlane(__float_as_int(pw), q + u)));
    }
    if (shared_y) add_bf16x8(acc, sv, 1.0f);
    if (res_a) add_bf16x8(acc, av, 1.0f);
    if (res_b) add_bf16x8(acc, bv, 1.0f);
    uint4 o;
    o.x = pack_bf16x2(acc[0], acc[1]);
    o.y = pack_bf16x2(acc[2], acc[3]);
    o.z = pack_bf16x2(acc[4], acc[5]);
    o.w = pack_bf16x2(acc[6], acc[7]);
    *reinterpret_cast<uint4*>(out + tok_off + v) = o;
  }
}

}  // namespace

int launch_combine(const uint16_t* y_sorted, const int32_t* pair_offsets,
                   const int32_t* pair_to_sorted, const float* pair_weight,
                   const uint16_t* shared_y, const uint16_t* res_a, const uint16_t* res_b, int T,
                   int d, int cap, uint16_t* out, hipStream_t s) {
  if (T >= 4096)
    hipLaunchKernelGGL(combine_kernel<8>, dim3(T), dim3(256), 0, s, y_sorted, pair_offsets,
                       pair_to_sorted, pair_weight, shared_y, res_a, res_b, d, cap, out);
  else
    hipLaunchKernelGGL(combine_kernel<16>, dim3(T), dim3(256), 0, s, y_sorted, pair_offsets,
                       pair_to_sorted, pair_weight, shared_y, res_a, res_b, d, cap, out);
  return launch_status();
}

}  // namespace rfx
