// Router scores r = h W_r^T (+ bias), Section 3.2, on bf16 MFMA.
//
// h is bf16 and W_r is fp32.  Each fp32 weight is split exactly into three bf16
// terms by truncation: hi = w with the low 16 bits cleared, mid = (w - hi) likewise,
// lo = w - hi - mid (at most 8 significant bits left, so exact in bf16).  Every
// product of a bf16 h with a bf16 term is exact in fp32, so three
// v_mfma_f32_16x16x32_bf16 per K step give h . w with fp32 accumulation only.
//
// Workgroup tile: TM tokens x 64 experts, 4 waves.  The 64 x 32 slice of W_r for
// each K step is loaded once per workgroup, split, and staged in LDS (double
// buffered); h fragments are loaded straight from global memory.
//   TM = 16: wave w computes the 16 tokens x experts 16w..16w+15   (small T)
//   TM = 64: wave w computes tokens 16w..16w+15 x all 64 experts   (large T)
#include "common.h"

namespace rfx {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int RT_TE = 64;        // experts per workgroup
constexpr int RT_TK = 32;        // K per MFMA step: an LDS row is 64 bytes (4 chunks of 16)

// Chunk c of expert row e is stored at slot c ^ ((e / 4) % 4): the 64 four-byte LDS
// banks then see 16 distinct 16-byte groups both for a fragment read (16 rows, one
// chunk) and for the staging writes (4 rows x 4 chunks).
__device__ __forceinline__ int bs_index(int row, int chunk) {
  return row * RT_TK + ((chunk ^ ((row >> 2) & 3)) << 3);
}

__device__ __forceinline__ void split3(float w, uint16_t& hi, uint16_t& mid, uint16_t& lo) {
  const uint32_t u = __float_as_uint(w);
  const uint32_t uh = u & 0xffff0000u;
  const float r1 = w - __uint_as_float(uh);
  const uint32_t um = __float_as_uint(r1) & 0xffff0000u;
  const float r2 = r1 - __uint_as_float(um);
  hi = static_cast<uint16_t>(uh >> 16);
  mid = static_cast<uint16_t>(um >> 16);
  lo = static_cast<uint16_t>(__float_as_uint(r2) >> 16);
}

template <int TM>
__global__ __launch_bounds__(256) void router_mfma_kernel(const uint16_t* __restrict__ h,
                                                          const float* __restrict__ w,
                                                          const float* __restrict__ bias,
                                                          float* __restrict__ logits, int T, int d,
                                                          int E) {
  constexpr int NB = TM == 16 ? 1 : 4;      // 16 x 16 accumulators per wave
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][3][RT_TE * RT_TK];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int t0 = blockIdx.x * TM, e0 = blockIdx.y * RT_TE;

  // W staging: thread -> expert tid/4, k chunk (tid%4)*8
  const int se = tid >> 2, sk = (tid & 3) * 8;
  const bool se_ok = e0 + se < E;
  const float* wsrc = w + static_cast<size_t>(se_ok ? e0 + se : 0) * d + sk;
  float4 wa, wb;
  auto load_w = [&](int k0) {
    if (se_ok) {
      wa = *reinterpret_cast<const float4*>(wsrc + k0);
      wb = *reinterpret_cast<const float4*>(wsrc + k0 + 4);
    } else {
      wa = make_float4(0, 0, 0, 0);
      wb = wa;
    }
  };
  auto store_w = [&](int buf) {
    const float v[8] = {wa.x, wa.y, wa.z, wa.w, wb.x, wb.y, wb.z, wb.w};
    uint16_t t[3][8];
#pragma unroll
    for (int j = 0; j < 8; ++j) split3(v[j], t[0][j], t[1][j], t[2][j]);
#pragma unroll
    for (int x = 0; x < 3; ++x) {
      uint4 pk;
      pk.x = t[x][0] | (uint32_t(t[x][1]) << 16);
      pk.y = t[x][2] | (uint32_t(t[x][3]) << 16);
      pk.z = t[x][4] | (uint32_t(t[x][5]) << 16);
      pk.w = t[x][6] | (uint32_t(t[x][7]) << 16);
      *reinterpret_cast<uint4*>(&Bs[buf][x][bs_index(se, sk >> 3)]) = pk;
    }
  };

  // A fragments: lane holds token row (lane % 16) of its 16-token block, k (lane/16)*8..+8
  const int tok_base = TM == 16 ? t0 : t0 + 16 * wv;
  const int arow = lane & 15, ak = (lane >> 4) * 8;
  const int tok = tok_base + arow;
  const bool tok_ok = tok < T;
  const uint16_t* asrc = h + static_cast<size_t>(tok_ok ? tok : 0) * d + ak;
  uint4 afrag;
  auto load_a = [&](int k0) {
    afrag = tok_ok ? *reinterpret_cast<const uint4*>(asrc + k0) : make_uint4(0, 0, 0, 0);
  };

  f32x4_t acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) acc[b] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int nk = d / RT_TK;
  load_w(0);
  load_a(0);
  store_w(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    const bf16x8_t a = __builtin_bit_cast(bf16x8_t, afrag);
    if (kt + 1 < nk) {
      load_w((kt + 1) * RT_TK);
      load_a((kt + 1) * RT_TK);
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int erow = (TM == 16 ? 16 * wv : 16 * b) + (lane & 15);
#pragma unroll
      for (int x = 0; x < 3; ++x) {
        const bf16x8_t bf = *reinterpret_cast<const bf16x8_t*>(&Bs[buf][x][bs_index(erow, ak >> 3)]);
        acc[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bf, acc[b], 0, 0, 0);
      }
    }
    if (kt + 1 < nk) store_w(buf ^ 1);
    __syncthreads();
  }
  // accumulator: lane l, register r -> token row 4 (l/16) + r, expert column l % 16
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int e = e0 + (TM == 16 ? 16 * wv : 16 * b) + (lane & 15);
    if (e >= E) continue;
    const float be = bias ? bias[e] : 0.0f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = tok_base + 4 * (lane >> 4) + r;
      if (t < T) logits[static_cast<size_t>(t) * E + e] = acc[b][r] + be;
    }
  }
}

}  // namespace

int launch_router(const uint16_t* h, const float* w, const float* bias, float* logits, int T,
                  int d, int E, hipStream_t s) {
  const int ne = (E + RT_TE - 1) / RT_TE;
  if (T >= 4096) {
    hipLaunchKernelGGL(router_mfma_kernel<64>, dim3((T + 63) / 64, ne), dim3(256), 0, s, h, w, bias,
                       logits, T, d, E);
  } else {
    hipLaunchKernelGGL(router_mfma_kernel<16>, dim3((T + 15) / 16, ne), dim3(256), 0, s, h, w, bias,
                       logits, T, d, E);
  }
  return launch_status();
}

}  // namespace rfx
