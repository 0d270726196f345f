// Per-token expert counts of one denoising forward: Refinement-Role Budgeting
// (Section 4.2, Eq. (5)) followed by Frontier-Guided Expert Reallocation
// (Section 4.3, Eqs. (6)-(9)) and the count bounds of Eq. (3).
//
// One workgroup per sequence.  The ranking key of every candidate (a masked
// active-block token with confidence history) is evaluated in fp64 with the
// same operation order as the defining formulas; floating-point contraction is
// disabled in this file so no fused multiply-add changes a rounding.  A token's
// rank is the number of candidates that precede it under (key descending,
// token index ascending), counted against LDS-staged slices of 2048 tokens, so
// sequences of any length work; the common case (<= 2048 tokens) is one slice.
#include "common.h"

#pragma clang fp contract(off)

namespace rfx {
namespace {

constexpr int BG_THREADS = 256;
constexpr int BG_PER_THREAD = 8;
constexpr int BG_CHUNK = BG_THREADS * BG_PER_THREAD;

struct BudgetConsts {
  double q, theta, w, v_ref, tau;
  int k_base, delta_role, delta_cur, k_min, k_max, signal;
};

__device__ __forceinline__ double logistic(double x) { return 1.0 / (1.0 + exp(-x)); }

// Ranking key of one candidate token (hist >= 1).  Out of line: it is called from
// several unrolled loops and would otherwise be inlined (with its three exp calls)
// at every one of them.
__device__ __attribute__((noinline)) double rank_key(const BudgetConsts& p, float c1f, float c2f,
                                                   int hist) {
  const double c1 = static_cast<double>(c1f), c2 = static_cast<double>(c2f);
  const double w = p.w;
  double v_bar, c_hat;
  if (hist >= 2) {
    const double v = c1 - c2;
    v_bar = fmin(fmax(v, -w / 2.0), w / 2.0);
    c_hat = fmin(fmax(c1 + v_bar, 0.0), 1.0);
  } else {               // one observation: zero velocity, forecast = c^{t-1}
    v_bar = 0.0;
    c_hat = c1;
  }
  const double F = logistic((c_hat - p.theta + w) / p.tau) * logistic((p.theta - c_hat) / p.tau);
  const double P = hist >= 2 ? logistic((p.v_ref - v_bar) / p.tau) : 1.0;
  switch (p.signal) {
    case REFLEX_SIGNAL_FRONTIER: return F;
    case REFLEX_SIGNAL_PROGRESS: return P;
    case REFLEX_SIGNAL_CONFIDENCE: return c1;
    case REFLEX_SIGNAL_UNCERTAINTY: return 1.0 - c1;
    default: return F * P;
  }
}

__device__ __forceinline__ int block_sum(int v, int* red) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  v = wave_sum_i32(v);
  __syncthreads();
  if (lane == 0) red[wv] = v;
  __syncthreads();
  int s = 0;
#pragma unroll
  for (int i = 0; i < BG_THREADS / kWave; ++i) s += red[i];
  return s;
}

__global__ __launch_bounds__(BG_THREADS) void budget_kernel(
    const int32_t* __restrict__ block_idx, const uint8_t* __restrict__ masked,
    const int8_t* __restrict__ hist_len, const float* __restrict__ c1,
    const float* __restrict__ c2, const int32_t* __restrict__ seq_offsets,
    const int32_t* __restrict__ active_block, int T, BudgetConsts p,
    int32_t* __restrict__ k_out, int32_t* __restrict__ pairs_out, double* __restrict__ fps_out) {
  __shared__ double s_key[BG_CHUNK];
  __shared__ int s_idx[BG_CHUNK];
  __shared__ int s_cnt;
  __shared__ int s_red[BG_THREADS / kWave];

  const int s = blockIdx.x;
  int lo = seq_offsets[s], hi = seq_offsets[s + 1];
  lo = lo < 0 ? 0 : (lo > T ? T : lo);
  hi = hi < lo ? lo : (hi > T ? T : hi);
  const int a = active_block[s];
  const int k_cur = p.k_base + p.delta_role;
  const int tid = threadIdx.x;

  // own tokens of one slice: candidate flag (masked, in the active block, with
  // confidence history), its ranking key, and the RRB count H(|b - a|) (Eq. (5))
  double key[BG_PER_THREAD];
  int rank[BG_PER_THREAD], kr[BG_PER_THREAD];
  bool cand[BG_PER_THREAD];
  auto load_slice = [&](int c0) {
#pragma unroll
    for (int r = 0; r < BG_PER_THREAD; ++r) {
      const int i = c0 + r * BG_THREADS + tid;
      cand[r] = false;
      key[r] = 0.0;
      rank[r] = 0;
      kr[r] = 0;
      if (i < hi) {
        // every field is loaded up front (one round of memory latency)
        const int b = block_idx[i];
        const bool msk = masked[i] != 0;
        const int hl = hist_len[i];
        const float x1 = c1[i], x2 = c2[i];
        const bool in_j = msk && b == a;
        const int dist = b > a ? b - a : a - b;
        kr[r] = in_j ? k_cur
                     : (dist <= 1 ? p.k_base + p.delta_role
                                  : (dist == 2 ? p.k_base : p.k_base - p.delta_role));
        cand[r] = in_j && hl >= 1;
        if (cand[r]) key[r] = rank_key(p, x1, x2, hl);
      }
    }
  };

  // m = |J'|, the number of ranked tokens of this sequence
  const bool single = hi - lo <= BG_CHUNK;      // uniform: one slice holds the sequence
  int mine = 0;
  if (single) {
    load_slice(lo);
#pragma unroll
    for (int r = 0; r < BG_PER_THREAD; ++r) mine += cand[r] ? 1 : 0;
  } else {
    for (int i = lo + tid; i < hi; i += BG_THREADS)
      mine += (masked[i] != 0 && block_idx[i] == a && hist_len[i] >= 1) ? 1 : 0;
  }
  const int m = block_sum(mine, s_red);
  const int n_q = static_cast<int>(floor(p.q * static_cast<double>(m)));

  int total = 0;
  for (int c0 = lo; c0 < hi; c0 += BG_CHUNK) {
    if (!single) load_slice(c0);
    if (m > 0) {
      for (int d0 = lo; d0 < hi; d0 += BG_CHUNK) {
        // stage the candidates of slice d0 (slot order is irrelevant to the count)
        if (tid == 0) s_cnt = 0;
        __syncthreads();
#pragma unroll
        for (int r = 0; r < BG_PER_THREAD; ++r) {
          const int j = d0 + r * BG_THREADS + tid;
          bool cj;
          double kj;
          if (d0 == c0) {
            cj = cand[r];
            kj = key[r];
          } else {
            cj = j < hi && masked[j] != 0 && block_idx[j] == a && hist_len[j] >= 1;
            kj = cj ? rank_key(p, c1[j], c2[j], hist_len[j]) : 0.0;
          }
          if (cj) {
            const int slot = atomicAdd(&s_cnt, 1);
            s_key[slot] = kj;
            s_idx[slot] = j;
          }
        }
        __syncthreads();
        const int cnt = s_cnt;
#pragma unroll
        for (int r = 0; r < BG_PER_THREAD; ++r) {
          if (!cand[r]) continue;
          const int i = c0 + r * BG_THREADS + tid;
          int before = 0;
          for (int x = 0; x < cnt; ++x) {
            const double kx = s_key[x];
            before += (kx > key[r] || (kx == key[r] && s_idx[x] < i)) ? 1 : 0;
          }
          rank[r] += before;
        }
        __syncthreads();
      }
    }
#pragma unroll
    for (int r = 0; r < BG_PER_THREAD; ++r) {
      const int i = c0 + r * BG_THREADS + tid;
      if (i >= hi) continue;
      int k = kr[r];
      if (cand[r]) {      // Eq. (9): high / middle / low group by rank
        if (rank[r] < n_q) k = k_cur + p.delta_cur;
        else if (rank[r] >= m - n_q) k = k_cur - p.delta_cur;
      }
      k = k < p.k_min ? p.k_min : (k > p.k_max ? p.k_max : k);
      k_out[i] = k;
      total += k;
      if (fps_out) fps_out[i] = cand[r] ? key[r] : __longlong_as_double(0x7ff8000000000000ll);
    }
  }
  if (pairs_out) {        // uniform
    total = block_sum(total, s_red);
    if (tid == 0 && total != 0) atomicAdd(pairs_out, total);
  }
}

__global__ void fill_i32_kernel(int32_t* dst, int32_t v, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = v;
}

// Exclusive prefix sum of the clamped counts: pair_offsets[0..T], P = pair_offsets[T].
// One workgroup walks the counts in slices of 4096 carrying the running total.
__global__ __launch_bounds__(1024) void count_scan_kernel(const int32_t* __restrict__ k, int T,
                                                          int k_max,
                                                          int32_t* __restrict__ pair_offsets,
                                                          int32_t* __restrict__ pairs_out) {
  __shared__ int s_wave[16];
  __shared__ int s_carry;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (tid == 0) s_carry = 0;
  __syncthreads();
  for (int base = 0; base < T; base += 4096) {
    int v[4];
    int sum = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = base + tid * 4 + j;
      v[j] = i < T ? clamp_count(k[i], k_max) : 0;
      sum += v[j];
    }
    const int incl = wave_inclusive_scan_i32(sum, lane);
    if (lane == 63) s_wave[wv] = incl;
    __syncthreads();
    int wave_off = 0;
    for (int x = 0; x < wv; ++x) wave_off += s_wave[x];
    int run = s_carry + wave_off + incl - sum;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = base + tid * 4 + j;
      if (i < T) pair_offsets[i] = run;
      run += v[j];
    }
    __syncthreads();
    if (tid == 1023) s_carry = run;
    __syncthreads();
  }
  if (tid == 0) {
    pair_offsets[T] = s_carry;
    if (pairs_out) pairs_out[0] = s_carry;
  }
}

}  // namespace

int launch_fill_i32(int32_t* dst, int32_t value, int n, hipStream_t s) {
  if (n <= 0) return REFLEX_OK;
  hipLaunchKernelGGL(fill_i32_kernel, dim3((n + 255) / 256), dim3(256), 0, s, dst, value, n);
  return launch_status();
}

int launch_budget(const int32_t* block_idx, const uint8_t* masked, const int8_t* hist_len,
                  const float* c1, const float* c2, const int32_t* seq_offsets,
                  const int32_t* active_block, int B, int T, const reflex_alloc_params& prm,
                  int32_t* k_out, int32_t* pairs_out, double* fps_out, hipStream_t s) {
  BudgetConsts p;
  p.q = prm.q; p.theta = prm.theta; p.w = prm.w_cf; p.v_ref = prm.v_ref; p.tau = prm.tau;
  p.k_base = prm.k_base; p.delta_role = prm.delta_role; p.delta_cur = prm.delta_cur;
  p.k_min = prm.k_min; p.k_max = prm.k_max; p.signal = prm.signal;
  if (pairs_out != nullptr) {
    const int rc = launch_fill_i32(pairs_out, 0, 1, s);
    if (rc != REFLEX_OK) return rc;
  }
  hipLaunchKernelGGL(budget_kernel, dim3(B), dim3(BG_THREADS), 0, s, block_idx, masked, hist_len,
                     c1, c2, seq_offsets, active_block, T, p, k_out, pairs_out, fps_out);
  return launch_status();
}

int launch_count_scan(const int32_t* k, int T, int k_max, int32_t* pair_offsets,
                      int32_t* pairs_out, hipStream_t s) {
  hipLaunchKernelGGL(count_scan_kernel, dim3(1), dim3(1024), 0, s, k, T, k_max, pair_offsets,
                     pairs_out);
  return launch_status();
}

}  // namespace rfx
