// Internal helpers shared by the gfx950 kernels of libreflex (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "reflex.h"

#define RFX_DEVICE __device__ __forceinline__

namespace rfx {

constexpr int kWave = 64;
constexpr int kGemmBM = 128;   // M tile (rows) of the grouped SwiGLU GEMM

// ---- bf16 <-> fp32 ------------------------------------------------------------------
RFX_DEVICE float bf16_to_f32(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }

// Round to nearest, ties to even, with the hardware conversion (v_cvt_pk_bf16_f32).
// Inputs here are finite.
typedef float rfx_f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 rfx_bf16x2 __attribute__((ext_vector_type(2)));

RFX_DEVICE uint32_t pack_bf16x2(float lo, float hi) {
  const rfx_f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, rfx_bf16x2));
}

RFX_DEVICE uint16_t f32_to_bf16(float f) { return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f)); }

// ---- wave64 reductions ----------------------------------------------------------------
// Built from DPP lane moves within 16-lane rows and the row swaps of v_permlane16_swap /
// v_permlane32_swap, all VALU: no LDS round trip per step, as a shuffle through
// ds_bpermute would take.  Every step pairs lanes symmetrically, so an all-reduce leaves
// the bit-identical result in every lane (floating-point sums included).
template <int CTRL>
RFX_DEVICE uint32_t dpp_u32(uint32_t v) {     // a lane move that has a source in every lane
  return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), CTRL, 0xf, 0xf, false));
}
constexpr int kDppXor1 = 0xB1;          // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;          // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;   // lane i <-> 7 - i within 8 lanes
constexpr int kDppMirror = 0x140;       // lane i <-> 15 - i within a row

// The value of the lane in the partner row (rows 0<->1, 2<->3) and in the partner half
// (lanes 0-31 <-> 32-63).  With both operands x, permlane16_swap returns rows
// (x0, x0, x2, x2) and (x1, x1, x3, x3): the lane's own row in one, the partner's in the
// other; a symmetric combine of the two needs not know which.
RFX_DEVICE void rows_swap16(uint32_t x, uint32_t& a, uint32_t& b) {
  const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  a = r[0];
  b = r[1];
}
RFX_DEVICE void rows_swap32(uint32_t x, uint32_t& a, uint32_t& b) {
  const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  a = r[0];
  b = r[1];
}

RFX_DEVICE int wave_sum_i32(int v) {
  uint32_t x = static_cast<uint32_t>(v), a, b;
  x += dpp_u32<kDppXor1>(x);
  x += dpp_u32<kDppXor2>(x);
  x += dpp_u32<kDppHalfMirror>(x);
  x += dpp_u32<kDppMirror>(x);
  rows_swap16(x, a, b);
  x = a + b;
  rows_swap32(x, a, b);
  return static_cast<int>(a + b);
}

RFX_DEVICE float wave_sum_f32(float v) {
  uint32_t a, b;
  v += __uint_as_float(dpp_u32<kDppXor1>(__float_as_uint(v)));
  v += __uint_as_float(dpp_u32<kDppXor2>(__float_as_uint(v)));
  v += __uint_as_float(dpp_u32<kDppHalfMirror>(__float_as_uint(v)));
  v += __uint_as_float(dpp_u32<kDppMirror>(__float_as_uint(v)));
  rows_swap16(__float_as_uint(v), a, b);
  v = __uint_as_float(a) + __uint_as_float(b);
  rows_swap32(__float_as_uint(v), a, b);
  return __uint_as_float(a) + __uint_as_float(b);
}

template <int CTRL>
RFX_DEVICE uint64_t max_dpp_u64(uint64_t v) {
  const uint64_t w = (static_cast<uint64_t>(dpp_u32<CTRL>(static_cast<uint32_t>(v >> 32))) << 32) |
                     dpp_u32<CTRL>(static_cast<uint32_t>(v));
  return w > v ? w : v;
}

RFX_DEVICE uint64_t wave_max_u64(uint64_t v) {
  v = max_dpp_u64<kDppXor1>(v);
  v = max_dpp_u64<kDppXor2>(v);
  v = max_dpp_u64<kDppHalfMirror>(v);
  v = max_dpp_u64<kDppMirror>(v);
  uint32_t a_lo, b_lo, a_hi, b_hi;
  rows_swap16(static_cast<uint32_t>(v), a_lo, b_lo);
  rows_swap16(static_cast<uint32_t>(v >> 32), a_hi, b_hi);
  uint64_t a = (static_cast<uint64_t>(a_hi) << 32) | a_lo, b = (static_cast<uint64_t>(b_hi) << 32) | b_lo;
  v = a > b ? a : b;
  rows_swap32(static_cast<uint32_t>(v), a_lo, b_lo);
  rows_swap32(static_cast<uint32_t>(v >> 32), a_hi, b_hi);
  a = (static_cast<uint64_t>(a_hi) << 32) | a_lo;
  b = (static_cast<uint64_t>(b_hi) << 32) | b_lo;
  return a > b ? a : b;
}

RFX_DEVICE uint32_t wave_max_u32(uint32_t v) {
  uint32_t a, b;
  v = max(v, dpp_u32<kDppXor1>(v));
  v = max(v, dpp_u32<kDppXor2>(v));
  v = max(v, dpp_u32<kDppHalfMirror>(v));
  v = max(v, dpp_u32<kDppMirror>(v));
  rows_swap16(v, a, b);
  v = max(a, b);
  rows_swap32(v, a, b);
  return max(a, b);
}

// Inclusive prefix sum across the 64 lanes of a wave: shifts by 1, 2, 4, 8 within each
// 16-lane row (lanes with no source add 0), then the last lane of row 0 added to row 1
// and of row 2 to row 3 (row_bcast:15), then lane 31 added to rows 2 and 3 (row_bcast:31).
RFX_DEVICE int wave_inclusive_scan_i32(int v, int /*lane*/) {
  int x = v;
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);   // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);   // row_bcast:15, rows 1, 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);   // row_bcast:31, rows 2, 3
  return x;
}

// Order-preserving map of fp32 to uint32 (larger float -> larger key), with
// -0.0 folded onto +0.0 so equal values tie.
RFX_DEVICE uint32_t f32_order_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

RFX_DEVICE float f32_from_order_key(uint32_t k) {
  uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
  return __uint_as_float(u);
}

RFX_DEVICE int clamp_count(int k, int k_max) { return k < 0 ? 0 : (k > k_max ? k_max : k); }

}  // namespace rfx

// ---- launch wrappers (host side, one per kernel family) ---------------------------------
// Each returns REFLEX_OK or REFLEX_ERR_LAUNCH.  Arguments are already validated.
namespace rfx {

// zero_word (nullable): set to 0 by the launch (the counter the fused route kernel that
// follows in the same forward expects to find at zero).  n_slices > 1 (only a value of
// router_slices(T, d, E)): logits receives n_slices fp32 partial score arrays [T, E]
// without the bias, slice s covering d columns [s d/n, (s+1) d/n); a score is the
// partials added in slice order, plus the bias.
int router_slices(int T, int d, int E);
int launch_router(const uint16_t* h, const float* w, const float* bias, float* logits, int T,
                  int d, int E, hipStream_t s, int32_t* zero_word = nullptr, int n_slices = 1);

// pairs_out may be NULL (the fused forward takes P from the count scan instead).
int launch_budget(const int32_t* block_idx, const uint8_t* masked, const int8_t* hist_len,
                  const float* c1, const float* c2, const int32_t* seq_offsets,
                  const int32_t* active_block, int B, int T, const reflex_alloc_params& p,
                  int32_t* k_out, int32_t* pairs_out, double* fps_out, hipStream_t s);

int launch_fill_i32(int32_t* dst, int32_t value, int n, hipStream_t s);

// Router scores and REFLEX counts in one launch; only for shapes where front_fits().
// The scores come out as front_slices(d) fp32 partials without the bias, parts[s][T][E]
// (slice s covers d columns [256 s, 256 s + 256)); a score is the partials added in
// slice order, plus the bias.
bool front_fits(int T, int d);
int front_slices(int d);
int launch_front(const uint16_t* h, const float* w, float* parts, int T, int d, int E,
                 const int32_t* block_idx, const uint8_t* masked, const int8_t* hist_len,
                 const float* c1, const float* c2, const int32_t* seq_offsets,
                 const int32_t* active_block, int B, const reflex_alloc_params& p, int32_t* k_out,
                 hipStream_t s, int32_t* zero_word = nullptr);

// One forward's commitment and state bookkeeping, one workgroup per sequence.
int launch_advance_state(const float* conf_t, const int32_t* block_idx, const int32_t* seq_offsets,
                         int B, int T, float theta, int min_commit, uint8_t* masked,
                         int8_t* hist_len, float* c1, float* c2, int32_t* active_block,
                         int32_t* remaining, hipStream_t s);

int launch_count_scan(const int32_t* k, int T, int k_max, int32_t* pair_offsets,
                      int32_t* pairs_out, hipStream_t s);

// Score-derived counts (REFLEX_RULE_TOP_P / REFLEX_RULE_THRESHOLD); pairs_out nullable.
int launch_count_rule(const float* logits, int T, int E, int rule, float threshold, int k_min,
                      int k_max, int32_t* k_out, int32_t* pairs_out, hipStream_t s);

int launch_topk(const float* logits, const int32_t* k, int T, int E, int k_max, int norm_topk,
                const int32_t* pair_offsets, int32_t* pair_expert, float* pair_weight,
                hipStream_t s);

// Pair offsets + TopK, and the permutation:
//  - route_fused_sorts(T, E): inside this launch, given hist (route_hist_bytes(T, E) of
//    scratch) and `done`, a device word the preceding launch set to zero;
//  - route_block_sorts(T, E): given hist and done NULL, this launch ranks the pairs in
//    their 16-token blocks (counts expert-major in hist) and launch_block_sort finishes;
//  - otherwise hist and done NULL, and launch_permute follows.
// pairs_out nullable.  The scores are n_parts partials part_stride floats apart, added
// in order, plus bias (nullable); n_parts = 1 with bias NULL reads finished scores.
// logits_out (nullable) receives the finished scores.
bool route_fused_sorts(int T, int E);
bool route_block_sorts(int T, int E);
size_t route_hist_bytes(int T, int E);
int launch_block_sort(const int32_t* pair_offsets, const int32_t* pair_expert, int T, int E,
                      int cap, int32_t* hist, int32_t* expert_offsets, int32_t* sorted_token,
                      int32_t* pair_to_sorted, int32_t* gemm_tile_off, hipStream_t s);
int launch_route_fused(const float* logits, int n_parts, size_t part_stride, const float* bias,
                       float* logits_out, const int32_t* k, int T, int E, int k_max,
                       int norm_topk, int32_t* pair_offsets, int32_t* pair_expert,
                       float* pair_weight, int32_t* pairs_out, int32_t* done, int32_t* hist,
                       int32_t* expert_offsets, int32_t* sorted_token, int32_t* pair_to_sorted,
                       int32_t* gemm_tile_off, hipStream_t s);

size_t permute_ws_bytes(int pair_capacity, int E);
// gemm_tile_off (nullable): also write the grouped GEMM's per-expert M-tile prefix.
int launch_permute(const int32_t* pair_offsets, const int32_t* pair_expert, const int32_t* pairs,
                   int T, int E, int pair_capacity, int32_t* expert_offsets,
                   int32_t* sorted_token, int32_t* pair_to_sorted, void* ws,
                   int32_t* gemm_tile_off, hipStream_t s);

size_t swiglu_ws_bytes(int pair_capacity, int E, int f);
// Routed experts: rows grouped by expert_offsets, inputs gathered through sorted_token.
int launch_swiglu_routed(const uint16_t* h, const int32_t* sorted_token,
                         const int32_t* expert_offsets, const uint16_t* wg, const uint16_t* wu,
                         const uint16_t* wd, int T, int E, int d, int f, int pair_capacity,
                         uint16_t* y_sorted, void* ws, hipStream_t s);
// The same in three steps: per-expert M-tile plan, gate/up GEMM, down GEMM.
int launch_swiglu_plan(const int32_t* expert_offsets, int E, void* ws, hipStream_t s);
int launch_swiglu_up(const uint16_t* h, const int32_t* sorted_token, const int32_t* expert_offsets,
                     const uint16_t* wg, const uint16_t* wu, int T, int E, int d, int f, int cap,
                     void* ws, hipStream_t s);
int launch_swiglu_down(const int32_t* expert_offsets, const uint16_t* wd, int E, int d, int f,
                       int cap, uint16_t* y_sorted, void* ws, hipStream_t s);
// One dense expert over rows 0..M-1 of x (the always-on shared expert).
size_t swiglu_dense_ws_bytes(int M, int f);
int launch_swiglu_dense(const uint16_t* x, const uint16_t* wg, const uint16_t* wu,
                        const uint16_t* wd, int M, int d, int f, uint16_t* y, void* ws,
                        hipStream_t s);

int launch_combine(const uint16_t* y_sorted, const int32_t* pair_offsets,
                   const int32_t* pair_to_sorted, const float* pair_weight,
                   const uint16_t* shared_y, const uint16_t* res_a, const uint16_t* res_b,
                   int T, int d, int pair_capacity, uint16_t* out, hipStream_t s);

inline int launch_status() {
  return hipGetLastError() == hipSuccess ? REFLEX_OK : REFLEX_ERR_LAUNCH;
}

inline size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

// Compute units of the current device, read once per process (256 on MI355X).
inline int device_cus() {
  static int cus = 0;
  if (cus == 0) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
      cus = n;
    else
      cus = 256;
  }
  return cus;
}

}  // namespace rfx
