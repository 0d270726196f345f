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

// ---- split-K partial tiles (the fused router + budget launch) ----
// The small-T router's cost is bytes through each CU: a workgroup that owns TM tokens
// x 16 experts over the whole of d moves (2 TM + 4 x 16) d bytes, and the fp32 W_r
// block is re-read by every token tile.  Here a workgroup owns 32 tokens x 64 experts
// over one 256-wide slice of d (80 KB: 16 KB of h, 64 KB of W_r) and writes the fp32
// partial scores of its slice; the consumer adds the d / 256 partials of a score in
// slice order (and the bias), so the result is deterministic.  16 waves: wave (c, q)
// takes experts 16c..16c+15 and K [64q, 64q+64) of the slice for both token blocks,
// loading its own W_r fragments (lane group g holds the 8 contiguous K values 8g..8g+7
// of each 32-wide step in both operands); the slice's h rows are staged once in LDS by
// one global_load_lds_dwordx4 copy per wave (two whole 512-byte rows), 16-byte chunk c
// of row r in slot c ^ (r % 16) so the 16 rows a 16-lane phase reads hit distinct
// banks.  The four K quarters are summed through LDS in a fixed order.
constexpr int RS_TM = 32;        // tokens per tile
constexpr int RS_TE = 64;        // experts per tile
constexpr int RS_KS = 256;       // K slice per tile (and per partial)
constexpr int RS_THREADS = 1024;

__device__ __forceinline__ void rs_dma(const void* src, void* dst) {
  __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
}

__device__ __forceinline__ void router_split_tile(int bx, int by, int ks,
                                                  const uint16_t* __restrict__ h,
                                                  const float* __restrict__ w,
                                                  float* __restrict__ parts, int T, int d, int E) {
  __shared__ __attribute__((aligned(16))) uint16_t s_h[RS_TM * RS_KS];
  __shared__ float s_red[4][RS_TM * RS_TE];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int t0 = bx * RS_TM, e0 = by * RS_TE, k0 = ks * RS_KS;
  const int c = wv >> 2, q = wv & 3, frow = lane & 15, g = lane >> 4;

  // this wave's W_r fragments: expert e0 + 16c + frow, K k0 + 64q + 32j + 8g .. +7
  const int e = e0 + 16 * c + frow;
  const float* wp = w + static_cast<size_t>(e < E ? e : E - 1) * d + k0 + 64 * q + 8 * g;
  float4 wf[2][2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    wf[j][0] = *reinterpret_cast<const float4*>(wp + 32 * j);
    wf[j][1] = *reinterpret_cast<const float4*>(wp + 32 * j + 4);
  }
  // rows 2 wv, 2 wv + 1 of the h slice (rows past T repeat row T-1; their scores are
  // not stored): lane L fills slot L % 32 of row 2 wv + L / 32
  {
    const int r = 2 * wv + (lane >> 5), chunk = (lane & 31) ^ (r & 15);
    const int t = min(t0 + r, T - 1);
    rs_dma(h + static_cast<size_t>(t) * d + k0 + 8 * chunk, s_h + 2 * wv * RS_KS);
  }
  __builtin_amdgcn_s_waitcnt(0x0f70);     // vmcnt(0): this wave's copy and loads landed
  __syncthreads();

  f32x4_t acc[2];
#pragma unroll
  for (int b = 0; b < 2; ++b) acc[b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    bf16x8_t w0, w1, w2;
    split3x8(wf[j][0], wf[j][1], w0, w1, w2);
    const int kc = (64 * q + 32 * j) / 8 + g;     // the lane's logical 16-byte chunk
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int r = 16 * b + frow;
      const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(s_h + r * RS_KS + 8 * (kc ^ (r & 15)));
      acc[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, w0, acc[b], 0, 0, 0);
      acc[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, w1, acc[b], 0, 0, 0);
      acc[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, w2, acc[b], 0, 0, 0);
    }
  }
  // accumulator: lane l, register i -> token row 16 b + 4 (l/16) + i, expert 16 c + l % 16
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      s_red[q][(16 * b + 4 * g + i) * RS_TE + 16 * c + frow] = acc[b][i];
  __syncthreads();
  for (int x = tid; x < RS_TM * RS_TE; x += RS_THREADS) {
    const int t = t0 + x / RS_TE, ee = e0 + x % RS_TE;
    if (t < T && ee < E)
      parts[static_cast<size_t>(ks) * T * E + static_cast<size_t>(t) * E + ee] =
          ((s_red[0][x] + s_red[1][x]) + s_red[2][x]) + s_red[3][x];
  }
}

}  // namespace
}  // namespace rfx
