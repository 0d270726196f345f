// Router scores r = h W_r^T (+ bias), Section 3.2.
//
// h is bf16 (widened exactly to fp32), W_r is fp32; every product is formed and
// accumulated in fp32 with fused multiply-adds.  Each workgroup computes a
// 64-token x 64-expert tile, staging 32-wide K slices of both operands in LDS.
#include "common.h"

namespace rfx {
namespace {

constexpr int RT_TM = 64;   // tokens per tile
constexpr int RT_TE = 64;   // experts per tile
constexpr int RT_TK = 32;   // K slice

__global__ __launch_bounds__(256) void router_kernel(const uint16_t* __restrict__ h,
                                                     const float* __restrict__ w,
                                                     const float* __restrict__ bias,
                                                     float* __restrict__ logits, int T, int d,
                                                     int E) {
  __shared__ float hs[RT_TK][RT_TM + 4];
  __shared__ float wsm[RT_TK][RT_TE + 4];
  const int tid = threadIdx.x;
  const int t0 = blockIdx.x * RT_TM;
  const int e0 = blockIdx.y * RT_TE;
  const int tx = tid & 15, ty = tid >> 4;     // 16 x 16 threads, 4 x 4 outputs each

  // loader coordinates: 64 rows x 32 k = 256 threads x 8 consecutive k
  const int lrow = tid >> 2, lk = (tid & 3) * 8;
  const int tok = t0 + lrow, ex = e0 + lrow;
  const bool tok_ok = tok < T, ex_ok = ex < E;
  const uint16_t* hp = h + static_cast<size_t>(tok_ok ? tok : 0) * d + lk;
  const float* wp = w + static_cast<size_t>(ex_ok ? ex : 0) * d + lk;

  float acc[4][4] = {};
  for (int k0 = 0; k0 < d; k0 += RT_TK) {
    uint4 hv = tok_ok ? *reinterpret_cast<const uint4*>(hp + k0) : make_uint4(0, 0, 0, 0);
    float4 wa = ex_ok ? *reinterpret_cast<const float4*>(wp + k0) : make_float4(0, 0, 0, 0);
    float4 wb = ex_ok ? *reinterpret_cast<const float4*>(wp + k0 + 4) : make_float4(0, 0, 0, 0);
    const uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      hs[lk + 2 * j][lrow] = __uint_as_float(hw[j] << 16);
      hs[lk + 2 * j + 1][lrow] = __uint_as_float(hw[j] & 0xffff0000u);
    }
    wsm[lk + 0][lrow] = wa.x; wsm[lk + 1][lrow] = wa.y; wsm[lk + 2][lrow] = wa.z; wsm[lk + 3][lrow] = wa.w;
    wsm[lk + 4][lrow] = wb.x; wsm[lk + 5][lrow] = wb.y; wsm[lk + 6][lrow] = wb.z; wsm[lk + 7][lrow] = wb.w;
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < RT_TK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = hs[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = wsm[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = t0 + ty * 4 + i;
    if (t >= T) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = e0 + tx * 4 + j;
      if (e < E) logits[static_cast<size_t>(t) * E + e] = acc[i][j] + (bias ? bias[e] : 0.0f);
    }
  }
}

}  // namespace

int launch_router(const uint16_t* h, const float* w, const float* bias, float* logits, int T,
                  int d, int E, hipStream_t s) {
  dim3 grid((T + RT_TM - 1) / RT_TM, (E + RT_TE - 1) / RT_TE);
  hipLaunchKernelGGL(router_kernel, grid, dim3(256), 0, s, h, w, bias, logits, T, d, E);
  return launch_status();
}

}  // namespace rfx
