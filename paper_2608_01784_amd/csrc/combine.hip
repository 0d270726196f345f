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

// Expert-output rows are read with the non-temporal hint when what the combine streams
// (the P expert rows, the token's own rows: residuals and shared expert, and the output)
// is larger than the 256 MB Infinity Cache: every expert row is read once, and read
// without the hint the rows evict the lines of the other streams.  Below that size the
// down GEMM has just written the rows into the cache and the plain loads hit there.
// Kernel durations traced in one process, identical output: skewed layer (656 MB) 130.3
// -> 109.3 us; 16-layer stack layer with its two residual streams (276 MB) 51.2 -> 50.1
// us; with the hint where the streams fit: stack layer without residuals (209 MB) 35.4
// -> 36.2 us, LLaDA2.0-mini with residuals (152 MB) 28.3 -> 30.3 us.
constexpr size_t kStreamBytes = size_t(256) << 20;

typedef unsigned int u32x4_nt __attribute__((ext_vector_type(4)));

template <bool STREAM>
__device__ __forceinline__ uint4 load_row(const uint16_t* p) {
  if constexpr (STREAM) {
    const u32x4_nt q = __builtin_nontemporal_load(reinterpret_cast<const u32x4_nt*>(p));
    return make_uint4(q.x, q.y, q.z, q.w);
  } else {
    return *reinterpret_cast<const uint4*>(p);
  }
}

// One token's output row (the body of the kernel below).  CB: expert rows in flight per
// batch.  16 keep a token's rows in one batch on the small layers; from T = 4096 up, 8
// (fewer registers, more workgroups resident per CU) are faster (16-layer stack layer:
// 35.1 against 42.1 us; LLaDA-MoE layer: 7.4 against 7.1).  A batch loads only the rows
// the token has (the branch is uniform: one token per workgroup); loading the last row
// again in the unused slots cost L2 requests for nothing (traced in one process: stack
// layer with its residuals 52.6 -> 44.4 us, skewed layer 110.4 -> 105.3 us, LLaDA2.0-mini
// 28.8 -> 27.0 us; batches of 2 or 4 rows with the extra loads were in between).
template <int CB, bool STREAM>
__device__ __forceinline__ void combine_token(
    int i, int p0, int p1, const uint16_t* __restrict__ y,
    const int32_t* __restrict__ pair_to_sorted, const float* __restrict__ pair_weight,
    const uint16_t* __restrict__ shared_y, const uint16_t* __restrict__ res_a,
    const uint16_t* __restrict__ res_b, int d, int cap, uint16_t* __restrict__ out) {
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
        add_bf16x8(acc, load_row<STREAM>(y + static_cast<size_t>(row) * d + v), pair_weight[p]);
      }
    }
    for (int q = 0; q < (np > kWave ? 0 : np); q += CB) {
      uint4 r[CB];
#pragma unroll
      for (int u = 0; u < CB; ++u) {
        r[u] = zero;
        if (q + u < np) {
          const int row = __builtin_amdgcn_readlane(prow, q + u);
          r[u] = load_row<STREAM>(y + static_cast<size_t>(row) * d + v);
        }
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

// One workgroup per token (the grid is the T tokens, so pair_offsets[gridDim.x] is the
// pair count; it is loaded with the token's own offsets, so the choice of load costs no
// extra round trip).  own: the output row and the token's own input rows.
template <int CB>
__global__ __launch_bounds__(256) void combine_kernel(
    const uint16_t* __restrict__ y, const int32_t* __restrict__ pair_offsets,
    const int32_t* __restrict__ pair_to_sorted, const float* __restrict__ pair_weight,
    const uint16_t* __restrict__ shared_y, const uint16_t* __restrict__ res_a,
    const uint16_t* __restrict__ res_b, int d, int cap, uint16_t* __restrict__ out) {
  const int i = blockIdx.x;
  const int p0 = pair_offsets[i], p1 = pair_offsets[i + 1];
  int P = pair_offsets[gridDim.x];
  P = P < 0 ? 0 : (P > cap ? cap : P);
  const size_t own = 1 + (shared_y != nullptr) + (res_a != nullptr) + (res_b != nullptr);
  const size_t rows = static_cast<size_t>(P) + own * gridDim.x;
  if (rows * d * sizeof(uint16_t) > kStreamBytes)
    combine_token<CB, true>(i, p0, p1, y, pair_to_sorted, pair_weight, shared_y, res_a, res_b, d,
                            cap, out);
  else
    combine_token<CB, false>(i, p0, p1, y, pair_to_sorted, pair_weight, shared_y, res_a, res_b, d,
                             cap, out);
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
