#pragma once
// Router scores r = h W_r^T (+ bias), Section 3.2, on bf16 MFMA (device code,
// shared by the router kernel and the fused router + budget kernel).
//
// h is bf16 and W_r is fp32.  Each fp32 weight is split exactly into three bf16
// terms by truncation: hi = w with the low 16 bits cleared, mid = (w - hi) likewise,
// lo = w - hi - mid (at most 8 significant bits left, so exact in bf16).  Every
// product of a bf16 h with a bf16 term is exact in fp32, so three
// v_mfma_f32_16x16x32_bf16 per K step give h . w with fp32 accumulation only.
//
// The contraction is short (E x d per token) and the layer's token count can be
// small, so parallelism comes from splitting K: a workgroup owns TM tokens x 16 EB
// experts and its KSPLIT waves each take 1/KSPLIT of d.  Every lane loads exactly the
// operand fragments it feeds to the MFMA (2 x 8 bytes of h, 4 x 2 x 16 bytes of W_r
// per 32-wide K step) and splits its own weights in registers, so the K loop has no
// LDS traffic and no barrier; a wave issues the loads of PF steps before using any.
// The partial tiles are summed through LDS in a fixed wave order, so the result is
// deterministic.
//   TM = 16, EB = 1, KSPLIT = 16 (small T): one 16 x 16 block per wave
//   TM = 64, EB = 4, KSPLIT = 4  (large T): 4 token blocks x 4 expert blocks per
//                                           wave (each W_r fragment feeds 4 blocks)
#include "common.h"

namespace rfx {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int RT_TK = 32;        // K per MFMA step

__device__ __forceinline__ void split3x8(const float4& lo4, const float4& hi4, bf16x8_t& t0,
                                         bf16x8_t& t1, bf16x8_t& t2) {
  const float v[8] = {lo4.x, lo4.y, lo4.z, lo4.w, hi4.x, hi4.y, hi4.z, hi4.w};
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t uh = __float_as_uint(v[j]) & 0xffff0000u;
    const float r1 = v[j] - __uint_as_float(uh);
    const uint32_t um = __float_as_uint(r1) & 0xffff0000u;
    const float r2 = r1 - __uint_as_float(um);
    t0[j] = __builtin_bit_cast(__bf16, static_cast<uint16_t>(uh >> 16));
    t1[j] = __builtin_bit_cast(__bf16, static_cast<uint16_t>(um >> 16));
    t2[j] = __builtin_bit_cast(__bf16, static_cast<uint16_t>(__float_as_uint(r2) >> 16));
  }
}

// One workgroup's tile (token block bx, expert block by) of the scores.
template <int TM, int EB, int KSPLIT, int PF>
__device__ __forceinline__ void router_tile(int bx, int by, const uint16_t* __restrict__ h,
                                            const float* __restrict__ w,
                                            const float* __restrict__ bias,
                                            float* __restrict__ logits, int T, int d, int E) {
  constexpr int TB = TM / 16;                      // token blocks per wave
  constexpr int RT_TE = 16 * EB;                   // experts per workgroup
  constexpr int NT = 64 * KSPLIT;
  __shared__ float part[KSPLIT][TM * 16 * EB];     // per-wave partial tiles
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int t0 = bx * TM, e0 = by * RT_TE;
  const int kq = d / KSPLIT;                       // this wave's K range (multiple of 32)
  const int kbeg = wv * kq;

  // fragment coordinates: row (lane % 16) of a 16-block.  The MFMA only needs A and
  // B to use the same K order, so lane group g = lane / 16 holds the 8 K values
  // {4g..4g+3, 16+4g..16+4g+3} of each 32-wide step: one 16-byte load per operand
  // half then covers 64 contiguous bytes of a W_r row across the 4 groups.
  const int frow = lane & 15, fk = (lane >> 4) * 4;
  const uint16_t* ap[TB];
  bool a_ok[TB];
#pragma unroll
  for (int b = 0; b < TB; ++b) {
    const int t = t0 + 16 * b + frow;
    a_ok[b] = t < T;
    ap[b] = h + static_cast<size_t>(a_ok[b] ? t : 0) * d + kbeg + fk;
  }
  const float* wp[EB];
  bool w_ok[EB];
#pragma unroll
  for (int c = 0; c < EB; ++c) {
    const int e = e0 + 16 * c + frow;
    w_ok[c] = e < E;
    wp[c] = w + static_cast<size_t>(w_ok[c] ? e : 0) * d + kbeg + fk;
  }

  f32x4_t acc[TB][EB];
#pragma unroll
  for (int b = 0; b < TB; ++b)
#pragma unroll
    for (int c = 0; c < EB; ++c) acc[b][c] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // PF K steps per round: every load of the round is issued before any is used
  for (int k0 = 0; k0 < kq; k0 += PF * RT_TK) {
    uint4 av[PF][TB];
    float4 wlo[PF][EB], whi[PF][EB];
#pragma unroll
    for (int q = 0; q < PF; ++q) {
      const int k = k0 + q * RT_TK;
      const bool in = k < kq;
#pragma unroll
      for (int b = 0; b < TB; ++b) {
        uint2 lo = make_uint2(0, 0), hi = lo;
        if (in && a_ok[b]) {
          lo = *reinterpret_cast<const uint2*>(ap[b] + k);
          hi = *reinterpret_cast<const uint2*>(ap[b] + k + 16);
        }
        av[q][b] = make_uint4(lo.x, lo.y, hi.x, hi.y);
      }
#pragma unroll
      for (int c = 0; c < EB; ++c) {
        const bool ok = in && w_ok[c];
        wlo[q][c] = ok ? *reinterpret_cast<const float4*>(wp[c] + k) : make_float4(0, 0, 0, 0);
        whi[q][c] = ok ? *reinterpret_cast<const float4*>(wp[c] + k + 16) : make_float4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int q = 0; q < PF; ++q) {
#pragma unroll
      for (int c = 0; c < EB; ++c) {
        bf16x8_t w0, w1, w2;
        split3x8(wlo[q][c], whi[q][c], w0, w1, w2);
#pragma unroll
        for (int b = 0; b < TB; ++b) {
          const bf16x8_t a = __builtin_bit_cast(bf16x8_t, av[q][b]);
          acc[b][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, w0, acc[b][c], 0, 0, 0);
          acc[b][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, w1, acc[b][c], 0, 0, 0);
          acc[b][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, w2, acc[b][c], 0, 0, 0);
        }
      }
    }
  }
  // accumulator: lane l, register r -> token row 4 (l/16) + r, expert column l % 16
#pragma unroll
  for (int b = 0; b < TB; ++b)
#pragma unroll
    for (int c = 0; c < EB; ++c)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        part[wv][(16 * b + 4 * (lane >> 4) + r) * RT_TE + 16 * c + (lane & 15)] = acc[b][c][r];
  __syncthreads();
  for (int x = tid; x < TM * RT_TE; x += NT) {
    const int t = t0 + x / RT_TE, e = e0 + x % RT_TE;
    if (t < T && e < E) {
      float s = part[0][x];
#pragma unroll
      for (int q = 1; q < KSPLIT; ++q) s += part[q][x];
      logits[static_cast<size_t>(t) * E + e] = s + (bias ? bias[e] : 0.0f);
    }
  }
}

}  // namespace
}  // namespace rfx
