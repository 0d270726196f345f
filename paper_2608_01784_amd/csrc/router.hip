// Router scores r = h W_r^T (+ bias), Section 3.2: the launch (the tile code and its
// description are in router_impl.h).
#include "router_impl.h"

namespace rfx {
namespace {

template <int TM, int EB, int KSPLIT, int PF>
__global__ __launch_bounds__(64 * KSPLIT) void router_mfma_kernel(const uint16_t* __restrict__ h,
                                                                 const float* __restrict__ w,
                                                                 const float* __restrict__ bias,
                                                                 float* __restrict__ logits, int T,
                                                                 int d, int E,
                                                                 int32_t* __restrict__ zero_word) {
  if (zero_word != nullptr && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *zero_word = 0;
  router_tile<TM, EB, KSPLIT, PF>(blockIdx.x, blockIdx.y, h, w, bias, logits, T, d, E);
}

// Large T: a workgroup owns TM tokens x 64 experts over the whole of d, 64-wide K
// steps staged in LDS by global_load_lds_dwordx4 copies (whole 128-byte row segments,
// so every line the copies touch is used in full) through a ring of S slices.  Wave w
// takes experts 16w..16w+15 for all TM tokens: it splits only its own weights, and
// each split weight fragment feeds TM/16 token blocks.  Lane group g of a fragment
// holds the 8 contiguous K values 8g..8g+7 of a 32-wide MFMA step in both operands.
// LDS rows: h rows of 64 bf16 (128 B, 8 chunks of 16 B, chunk c of row r in slot
// c ^ ((r / 2) % 8)); W rows of 64 fp32 (256 B, 16 chunks, chunk c in slot c ^ (r % 16)),
// so the 16 rows one 16-lane phase reads hit distinct banks.
constexpr int RB_BK = 64;
constexpr int RB_TE = 64;
constexpr int RB_THREADS = 256;

// One wave's 1 KB copy, 16 bytes per lane, global -> LDS; out of line of the kernel's
// lambda so that the host-side pass of the templated kernel stays valid.
__device__ __forceinline__ void rb_dma(const void* src, void* dst) {
  __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
}

// s_waitcnt vmcnt(N) (gfx9 encoding: vmcnt in bits [3:0] and [15:14]; expcnt and
// lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void rb_waitcnt_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0f70);
}

// Wait for this wave's copies of the oldest slice in flight, leaving those of the
// `pending` younger slices (each OPS copies) outstanding.
template <int OPS, int S>
__device__ __forceinline__ void rb_wait(int pending) {
  switch (pending) {
    case 0: rb_waitcnt_vm<0>(); break;
    case 1: rb_waitcnt_vm<(S > 2 ? OPS : 0)>(); break;
    default: rb_waitcnt_vm<(S > 3 ? 2 * OPS : 0)>(); break;
  }
}

template <int TM, int S>
__global__ __launch_bounds__(RB_THREADS) void router_big_kernel(const uint16_t* __restrict__ h,
                                                                const float* __restrict__ w,
                                                                const float* __restrict__ bias,
                                                                float* __restrict__ logits, int T,
                                                                int d, int E,
                                                                int32_t* __restrict__ zero_word,
                                                                int n_slices) {
  // n_slices > 1: this workgroup covers d columns [ks kd, ks kd + kd), kd = d / n_slices,
  // ks = blockIdx.z, and writes the partial scores (no bias) to logits + ks T E
  constexpr int TB = TM / 16;                          // token blocks per wave
  constexpr int H_ELEMS = TM * RB_BK;                  // bf16 per h slice
  constexpr int W_ELEMS = RB_TE * RB_BK;               // fp32 per W slice
  constexpr int H_OPS = TM / 8 / 4;                    // 1 KB copies per wave (8 h rows each)
  constexpr int W_OPS = RB_TE / 4 / 4;                 // (4 W rows each)
  static_assert(S >= 2 && S <= 4, "ring depth");
  __shared__ __attribute__((aligned(16))) uint16_t s_h[S][H_ELEMS];
  __shared__ __attribute__((aligned(16))) float s_w[S][W_ELEMS];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int t0 = blockIdx.x * TM, e0 = blockIdx.y * RB_TE;
  const int kd = d / n_slices, kbase = blockIdx.z * kd;
  const int nk = kd / RB_BK;
  if (zero_word != nullptr && blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0 && tid == 0)
    *zero_word = 0;

  // copy sources: lane L of an h op fills row 8q + L/8, slot L%8; of a W op row 4q + L/16,
  // slot L%16; rows past T or E repeat the last valid row (their results are not stored)
  const uint16_t* hp[H_OPS];
  const float* wp[W_OPS];
#pragma unroll
  for (int j = 0; j < H_OPS; ++j) {
    const int q = wv * H_OPS + j, r = 8 * q + lane / 8;
    const int c = (lane % 8) ^ ((r / 2) % 8);
    const int t = min(t0 + r, T - 1);
    hp[j] = h + static_cast<size_t>(t) * d + kbase + c * 8;
  }
#pragma unroll
  for (int j = 0; j < W_OPS; ++j) {
    const int q = wv * W_OPS + j, r = 4 * q + lane / 16;
    const int c = (lane % 16) ^ (r % 16);
    const int e = min(e0 + r, E - 1);
    wp[j] = w + static_cast<size_t>(e) * d + kbase + c * 4;
  }
  auto issue = [&](int kt) {
    const int buf = kt % S, k0 = kt * RB_BK;
#pragma unroll
    for (int j = 0; j < H_OPS; ++j)
      rb_dma(hp[j] + k0, &s_h[buf][(wv * H_OPS + j) * 512]);
#pragma unroll
    for (int j = 0; j < W_OPS; ++j)
      rb_dma(wp[j] + k0, &s_w[buf][(wv * W_OPS + j) * 256]);
  };

  const int frow = lane & 15, g = lane >> 4;
  f32x4_t acc[TB];
#pragma unroll
  for (int b = 0; b < TB; ++b) acc[b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (int k = 0; k < S - 1 && k < nk; ++k) issue(k);
  for (int kt = 0; kt < nk; ++kt) {
    rb_wait<H_OPS + W_OPS, S>(min(S - 2, nk - 1 - kt));   // this wave's copies of slice kt
    __builtin_amdgcn_s_waitcnt(0xc07f);            // lgkmcnt(0)
    asm volatile("s_barrier" ::: "memory");        // slice kt complete; slice kt-1 released
    // Every LDS read of slice kt is issued before the copies of the slice S - 1 ahead:
    // the compiler cannot tell a copy's LDS destination from the slot being read, so a
    // read placed after a copy would wait for that copy to land (18.8 -> 16.9 us on the
    // 16-layer stack's router, measured; identical output).
    const uint16_t* H = s_h[kt % S];
    const float* W = s_w[kt % S];
    const int wr = 16 * wv + frow;                 // this wave's expert row
    float4 lo4[RB_BK / 32], hi4[RB_BK / 32];
    bf16x8_t a[RB_BK / 32][TB];
#pragma unroll
    for (int s32 = 0; s32 < RB_BK / 32; ++s32) {
      // W: K chunk pair (8 s32 + 2g, +1) of 4 fp32 each; h: 16-byte chunk 4 s32 + g
      const int wc = 8 * s32 + 2 * g;
      lo4[s32] = *reinterpret_cast<const float4*>(W + wr * RB_BK + ((wc ^ (wr % 16)) * 4));
      hi4[s32] = *reinterpret_cast<const float4*>(W + wr * RB_BK + (((wc + 1) ^ (wr % 16)) * 4));
#pragma unroll
      for (int b = 0; b < TB; ++b) {
        const int hr = 16 * b + frow, hc = 4 * s32 + g;
        a[s32][b] = *reinterpret_cast<const bf16x8_t*>(H + hr * RB_BK + ((hc ^ ((hr / 2) % 8)) * 8));
      }
    }
    if (kt + S - 1 < nk) issue(kt + S - 1);
    // the three split terms in turn over all token blocks: each accumulator still adds
    // hi, mid, lo of one 32-wide step in that order, TB MFMAs apart instead of one
#pragma unroll
    for (int s32 = 0; s32 < RB_BK / 32; ++s32) {
      bf16x8_t bt[3];
      split3x8(lo4[s32], hi4[s32], bt[0], bt[1], bt[2]);
#pragma unroll
      for (int t = 0; t < 3; ++t)
#pragma unroll
        for (int b = 0; b < TB; ++b)
          acc[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[s32][b], bt[t], acc[b], 0, 0, 0);
    }
  }
  // accumulator: lane l, register r -> token row 4 (l/16) + r, expert column l % 16
  const int e = e0 + 16 * wv + (lane & 15);
  if (e < E) {
    const float be = (bias && n_slices == 1) ? bias[e] : 0.0f;
    float* out = logits + static_cast<size_t>(blockIdx.z) * T * E;
#pragma unroll
    for (int b = 0; b < TB; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = t0 + 16 * b + 4 * (lane >> 4) + r;
        if (t < T) out[static_cast<size_t>(t) * E + e] = acc[b][r] + be;
      }
  }
}

}  // namespace

// K slices of the split-K router for T >= 4096 (1: finished scores).  The 128-token x
// 64-expert LDS-staged tiles re-read neither operand much (h once per 64 experts, W_r
// once per 128 tokens), so where they are too few to fill the GPU the K range is split
// instead of shrinking the tiles: up to ~512 workgroups (two fit a CU), slices of at
// least 256 columns.
int router_slices(int T, int d, int E) {
  if (T < 4096 || d % RB_BK != 0) return 1;
  const long tiles = static_cast<long>((T + 127) / 128) * ((E + RB_TE - 1) / RB_TE);
  int ns = 1;
  while (tiles * ns * 2 <= 512 && d % (2 * ns * 256) == 0) ns *= 2;
  return ns;
}

int launch_router(const uint16_t* h, const float* w, const float* bias, float* logits, int T,
                  int d, int E, hipStream_t s, int32_t* zero_word, int n_slices) {
  // A workgroup's loads all pass through one CU, so tiles are sized to spread the
  // traffic over many CUs: small T uses 16 x 16 tiles with K split over 16 waves.  For
  // T >= 4096 the split-K path (n_slices > 1, partial scores for the caller to add) runs
  // 128 x 64 tiles over a slice of d each.  With finished scores requested: 128 x 64
  // tiles where that gives 512 or more (T = 16384, E = 256), else 32 x 64 tiles (T = 4096,
  // E = 256: 33 us against 39 us for 64 x 64 register tiles), and with at most 64 experts
  // the register kernel with 32-token tiles and K split over 8 waves (T = 8192, E = 64:
  // 29 us against 34 us and 38 us for the LDS kernel and 64 x 64 register tiles; all
  // measured).
  if (n_slices > 1) {
    hipLaunchKernelGGL((router_big_kernel<128, 2>),
                       dim3((T + 127) / 128, (E + RB_TE - 1) / RB_TE, n_slices), dim3(RB_THREADS), 0,
                       s, h, w, bias, logits, T, d, E, zero_word, n_slices);
    return launch_status();
  }
  const long big_tiles = static_cast<long>((T + 127) / 128) * ((E + RB_TE - 1) / RB_TE);
  if (big_tiles >= 512) {
    hipLaunchKernelGGL((router_big_kernel<128, 2>), dim3((T + 127) / 128, (E + RB_TE - 1) / RB_TE),
                       dim3(RB_THREADS), 0, s, h, w, bias, logits, T, d, E, zero_word, 1);
  } else if (T >= 4096 && E <= 64 && d % (RT_TK * 8) == 0) {
    hipLaunchKernelGGL((router_mfma_kernel<32, 4, 8, 2>), dim3((T + 31) / 32, (E + 63) / 64),
                       dim3(512), 0, s, h, w, bias, logits, T, d, E, zero_word);
  } else if (T >= 4096) {
    hipLaunchKernelGGL((router_big_kernel<32, 2>), dim3((T + 31) / 32, (E + RB_TE - 1) / RB_TE),
                       dim3(RB_THREADS), 0, s, h, w, bias, logits, T, d, E, zero_word, 1);
  } else if (d % (RT_TK * 16) == 0) {
    hipLaunchKernelGGL((router_mfma_kernel<16, 1, 16, 4>), dim3((T + 15) / 16, (E + 15) / 16),
                       dim3(1024), 0, s, h, w, bias, logits, T, d, E, zero_word);
  } else {
    hipLaunchKernelGGL((router_mfma_kernel<16, 1, 4, 4>), dim3((T + 15) / 16, (E + 15) / 16),
                       dim3(256), 0, s, h, w, bias, logits, T, d, E, zero_word);
  }
  return launch_status();
}

}  // namespace rfx
