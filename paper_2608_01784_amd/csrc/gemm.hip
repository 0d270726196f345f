// SwiGLU experts over expert-sorted rows on bf16 MFMA (gfx950).
//
// Expert e (Eq. (2)) is E_e(x) = W_down[e] (SiLU(W_gate[e] x) * (W_up[e] x)), the
// two input projections and one output projection counted in Appendix A.  Two
// grouped GEMMs do the work, both "NT" (both operands K-contiguous):
//   up:   act[j, :] = SiLU(x_j W_gate[e]^T) * (x_j W_up[e]^T),  x_j = h[sorted_token[j]]
//   down: y[j, :]   = act[j, :] W_down[e]^T
// Rows of one expert are contiguous after the permutation; a device-side plan
// cuts each expert's rows into 128-row M tiles, so the grid never depends on the
// (device-resident) per-expert counts: workgroups past the last tile exit.
//
// Tile: 128 (M) x 128 (B rows) x 64 (K), 4 waves in 2 x 2, each wave 64 x 64 as
// 2 x 2 v_mfma_f32_32x32x16_bf16 tiles, fp32 accumulators.  Operands are staged
// through LDS with double buffering (rows padded to 144 bytes).  In the up GEMM
// the 128 B rows are 64 gate rows and the 64 matching up rows, so gate and up of
// the same output column land in the same lane and register, and SiLU(g) * u is
// formed in registers before the single bf16 rounding of the activation.
#include "common.h"

namespace rfx {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int GM_BM = 128;
constexpr int GM_BK = 64;
constexpr int GM_LDS = GM_BK + 8;          // padded row, in bf16 elements (144 bytes)
constexpr int GM_THREADS = 256;
constexpr int GM_UP_BN = 64;               // activation columns per up-GEMM tile
constexpr int GM_DOWN_BN = 128;            // output columns per down-GEMM tile

struct TileRange {
  int row0, row_end, expert;
};

// M tile -> (expert, first row, end row).  Routed mode searches the per-expert tile
// prefix; dense mode (one expert over rows 0..M-1) has dense_M >= 0.
// Rows are clamped to [0, out_rows) so inconsistent offsets can never index outside
// the row buffers.
__device__ __forceinline__ bool tile_range(int m_tile, const int32_t* __restrict__ tile_off,
                                           const int32_t* __restrict__ expert_offsets, int E,
                                           int dense_M, int out_rows, TileRange& tr) {
  if (dense_M >= 0) {
    tr.row0 = m_tile * GM_BM;
    tr.row_end = dense_M;
    tr.expert = 0;
    return tr.row0 < dense_M;
  }
  if (m_tile >= tile_off[E]) return false;
  int lo = 0, hi = E - 1;               // largest e with tile_off[e] <= m_tile
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (tile_off[mid] <= m_tile) lo = mid; else hi = mid - 1;
  }
  tr.expert = lo;
  tr.row0 = expert_offsets[lo] + (m_tile - tile_off[lo]) * GM_BM;
  tr.row_end = expert_offsets[lo + 1] < out_rows ? expert_offsets[lo + 1] : out_rows;
  return tr.row0 >= 0 && tr.row0 < tr.row_end;
}

// UP = true : act = SiLU(X Wg^T) * (X Wu^T);  UP = false: y = act Wd^T.
template <bool UP>
__global__ __launch_bounds__(GM_THREADS, 2) void swiglu_gemm_kernel(
    const uint16_t* __restrict__ x,            // UP: h [T, K]; DOWN: act [rows, K]
    const int32_t* __restrict__ gather,        // UP: sorted_token or NULL (identity)
    const int32_t* __restrict__ tile_off, const int32_t* __restrict__ expert_offsets, int E,
    int dense_M, const uint16_t* __restrict__ w0,   // UP: W_gate; DOWN: W_down
    const uint16_t* __restrict__ w1,                // UP: W_up
    size_t w_expert_stride, int K, int N_out, int x_rows, int out_rows,
    uint16_t* __restrict__ out) {
  __shared__ __attribute__((aligned(16))) uint16_t As[2][GM_BM * GM_LDS];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][GM_BM * GM_LDS];

  constexpr int BN = UP ? GM_UP_BN : GM_DOWN_BN;
  const int n_tiles = N_out / BN;
  const int m_tile = blockIdx.x / n_tiles;
  const int n0 = (blockIdx.x % n_tiles) * BN;
  TileRange tr;
  if (!tile_range(m_tile, tile_off, expert_offsets, E, dense_M, out_rows, tr)) return;

  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int wm = wv >> 1, wn = wv & 1;

  // loader: 4 x 16-byte vectors of A and of B per thread; row (tid >> 3) + 32 j,
  // column chunk (tid & 7) * 8
  const int lcol = (tid & 7) * 8;
  const uint16_t* a_src[4];
  const uint16_t* b_src[4];
  bool a_ok[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = (tid >> 3) + 32 * j;
    const int grow = tr.row0 + r;
    a_ok[j] = grow < tr.row_end;
    int src_row = a_ok[j] ? grow : tr.row0;
    if (UP && gather != nullptr) {
      src_row = gather[src_row];
      src_row = src_row < 0 ? 0 : (src_row >= x_rows ? x_rows - 1 : src_row);
    }
    a_src[j] = x + static_cast<size_t>(src_row) * K + lcol;
    const uint16_t* wbase;
    int wrow;
    if (UP) {
      wbase = (r < 64 ? w0 : w1) + tr.expert * w_expert_stride;
      wrow = n0 + (r & 63);
    } else {
      wbase = w0 + tr.expert * w_expert_stride;
      wrow = n0 + r;
    }
    b_src[j] = wbase + static_cast<size_t>(wrow) * K + lcol;
  }

  uint4 ra[4], rb[4];
  auto load_global = [&](int k0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      ra[j] = a_ok[j] ? *reinterpret_cast<const uint4*>(a_src[j] + k0) : make_uint4(0, 0, 0, 0);
      rb[j] = *reinterpret_cast<const uint4*>(b_src[j] + k0);
    }
  };
  auto store_lds = [&](int buf) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = (tid >> 3) + 32 * j;
      *reinterpret_cast<uint4*>(&As[buf][r * GM_LDS + lcol]) = ra[j];
      *reinterpret_cast<uint4*>(&Bs[buf][r * GM_LDS + lcol]) = rb[j];
    }
  };

  // B sub-tile rows of this wave: UP -> gate rows wn*32.., up rows 64 + wn*32..;
  // DOWN -> rows wn*64 and wn*64 + 32
  const int b_row[2] = {UP ? wn * 32 : wn * 64, UP ? 64 + wn * 32 : wn * 64 + 32};
  const int a_row[2] = {wm * 64, wm * 64 + 32};
  const int frag_row = lane & 31, frag_k = (lane >> 5) * 8;

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nk = K / GM_BK;
  load_global(0);
  store_lds(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load_global((kt + 1) * GM_BK);
#pragma unroll
    for (int kk = 0; kk < GM_BK / 16; ++kk) {
      bf16x8_t af[2], bfr[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        af[i] = *reinterpret_cast<const bf16x8_t*>(
            &As[buf][(a_row[i] + frag_row) * GM_LDS + kk * 16 + frag_k]);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8_t*>(
            &Bs[buf][(b_row[j] + frag_row) * GM_LDS + kk * 16 + frag_k]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) store_lds(buf ^ 1);
    __syncthreads();
  }

  // epilogue: acc lane l, register r holds row 8 (r/4) + 4 (l/32) + r%4, column l%32
  const int col = lane & 31;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int mrow = a_row[i] + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      const int grow = tr.row0 + mrow;
      if (grow >= tr.row_end) continue;
      uint16_t* orow = out + static_cast<size_t>(grow) * N_out + n0;
      if (UP) {
        const float g = acc[i][0][r], u = acc[i][1][r];
        const float a = g / (1.0f + expf(-g)) * u;
        orow[wn * 32 + col] = f32_to_bf16(a);
      } else {
        orow[wn * 64 + col] = f32_to_bf16(acc[i][0][r]);
        orow[wn * 64 + 32 + col] = f32_to_bf16(acc[i][1][r]);
      }
    }
  }
}

// Per-expert M-tile prefix: tile_off[e] = sum_{e' < e} ceil(n_e' / 128), tile_off[E] = total.
__global__ __launch_bounds__(256) void tile_plan_kernel(const int32_t* __restrict__ expert_offsets,
                                                        int E, int32_t* __restrict__ tile_off) {
  __shared__ int s_wave[4];
  const int e = threadIdx.x, lane = e & 63, wv = e >> 6;
  int n = 0;
  if (e < E) {
    n = expert_offsets[e + 1] - expert_offsets[e];
    n = n < 0 ? 0 : (n + GM_BM - 1) / GM_BM;
  }
  const int incl = wave_inclusive_scan_i32(n, lane);
  if (lane == 63) s_wave[wv] = incl;
  __syncthreads();
  int base = incl - n;
  for (int x = 0; x < wv; ++x) base += s_wave[x];
  if (e < E) {
    tile_off[e] = base;
    if (e == E - 1) tile_off[E] = base + n;
  }
}

int max_m_tiles(int cap, int E) {
  long long t = (static_cast<long long>(cap) + GM_BM - 1) / GM_BM + E;
  if (t > cap) t = cap;
  return static_cast<int>(t < 1 ? 1 : t);
}

}  // namespace

size_t swiglu_ws_bytes(int pair_capacity, int E, int f) {
  return align_up(sizeof(int32_t) * (E + 1)) +
         align_up(static_cast<size_t>(pair_capacity) * f * sizeof(uint16_t));
}

size_t swiglu_dense_ws_bytes(int M, int f) {
  return align_up(static_cast<size_t>(M) * f * sizeof(uint16_t));
}

int launch_swiglu_plan(const int32_t* expert_offsets, int E, void* ws, hipStream_t s) {
  hipLaunchKernelGGL(tile_plan_kernel, dim3(1), dim3(256), 0, s, expert_offsets, E,
                     static_cast<int32_t*>(ws));
  return launch_status();
}

static uint16_t* routed_act(void* ws, int E) {
  return reinterpret_cast<uint16_t*>(static_cast<char*>(ws) + align_up(sizeof(int32_t) * (E + 1)));
}

int launch_swiglu_up(const uint16_t* h, const int32_t* sorted_token, const int32_t* expert_offsets,
                     const uint16_t* wg, const uint16_t* wu, int T, int E, int d, int f, int cap,
                     void* ws, hipStream_t s) {
  if (cap <= 0) return REFLEX_OK;
  const int32_t* tile_off = static_cast<const int32_t*>(ws);
  const int mt = max_m_tiles(cap, E);
  hipLaunchKernelGGL(swiglu_gemm_kernel<true>, dim3(mt * (f / GM_UP_BN)), dim3(GM_THREADS), 0, s,
                     h, sorted_token, tile_off, expert_offsets, E, -1, wg, wu,
                     static_cast<size_t>(f) * d, d, f, T, cap, routed_act(ws, E));
  return launch_status();
}

int launch_swiglu_down(const int32_t* expert_offsets, const uint16_t* wd, int E, int d, int f,
                       int cap, uint16_t* y_sorted, void* ws, hipStream_t s) {
  if (cap <= 0) return REFLEX_OK;
  const int32_t* tile_off = static_cast<const int32_t*>(ws);
  const int mt = max_m_tiles(cap, E);
  hipLaunchKernelGGL(swiglu_gemm_kernel<false>, dim3(mt * (d / GM_DOWN_BN)), dim3(GM_THREADS), 0,
                     s, routed_act(ws, E), nullptr, tile_off, expert_offsets, E, -1, wd, nullptr,
                     static_cast<size_t>(d) * f, f, d, cap, cap, y_sorted);
  return launch_status();
}

int launch_swiglu_routed(const uint16_t* h, const int32_t* sorted_token,
                         const int32_t* expert_offsets, const uint16_t* wg, const uint16_t* wu,
                         const uint16_t* wd, int T, int E, int d, int f, int cap,
                         uint16_t* y_sorted, void* ws, hipStream_t s) {
  if (cap <= 0) return REFLEX_OK;
  int rc = launch_swiglu_plan(expert_offsets, E, ws, s);
  if (rc == REFLEX_OK) rc = launch_swiglu_up(h, sorted_token, expert_offsets, wg, wu, T, E, d, f, cap, ws, s);
  if (rc == REFLEX_OK) rc = launch_swiglu_down(expert_offsets, wd, E, d, f, cap, y_sorted, ws, s);
  return rc;
}

int launch_swiglu_dense(const uint16_t* x, const uint16_t* wg, const uint16_t* wu,
                        const uint16_t* wd, int M, int d, int f, uint16_t* y, void* ws,
                        hipStream_t s) {
  if (M <= 0) return REFLEX_OK;
  uint16_t* act = static_cast<uint16_t*>(ws);
  const int mt = (M + GM_BM - 1) / GM_BM;
  hipLaunchKernelGGL(swiglu_gemm_kernel<true>, dim3(mt * (f / GM_UP_BN)), dim3(GM_THREADS), 0, s,
                     x, nullptr, nullptr, nullptr, 1, M, wg, wu, size_t(0), d, f, M, M, act);
  hipLaunchKernelGGL(swiglu_gemm_kernel<false>, dim3(mt * (d / GM_DOWN_BN)), dim3(GM_THREADS), 0,
                     s, act, nullptr, nullptr, nullptr, 1, M, wd, nullptr, size_t(0), f, d, M, M, y);
  return launch_status();
}

}  // namespace rfx
