#pragma once
// Per-token expert counts of one denoising forward: Refinement-Role Budgeting
// (Section 4.2, Eq. (5)) followed by Frontier-Guided Expert Reallocation
// (Section 4.3, Eqs. (6)-(9)) and the count bounds of Eq. (3).
//
// Device code shared by the budget kernel and the fused router + budget kernel.
//
// One workgroup per sequence.  The ranking key of every candidate (a masked
// active-block token with confidence history) is evaluated in fp64 with the
// same operation order as the defining formulas; floating-point contraction is
// disabled in the key's code so no fused multiply-add changes a rounding.  A token's
// rank is the number of candidates that precede it under (key descending,
// token index ascending), counted against LDS-staged slices of 2048 tokens, so
// sequences of any length work; the common case (<= 2048 tokens) is one slice.
#include "common.h"

namespace rfx {
namespace {

constexpr int BG_CHUNK = 2048;       // tokens staged per slice

struct BudgetConsts {
  double q, theta, w, v_ref, tau;
  int k_base, delta_role, delta_cur, k_min, k_max, signal;
};

inline BudgetConsts budget_consts(const reflex_alloc_params& prm) {
  BudgetConsts p;
  p.q = prm.q; p.theta = prm.theta; p.w = prm.w_cf; p.v_ref = prm.v_ref; p.tau = prm.tau;
  p.k_base = prm.k_base; p.delta_role = prm.delta_role; p.delta_cur = prm.delta_cur;
  p.k_min = prm.k_min; p.k_max = prm.k_max; p.signal = prm.signal;
  return p;
}

__device__ __forceinline__ double logistic(double x) {
#pragma clang fp contract(off)
  return 1.0 / (1.0 + exp(-x));
}

// Ranking key of one candidate token (hist >= 1).
__device__ __forceinline__ double rank_key(const BudgetConsts& p, float c1f, float c2f, int hist) {
#pragma clang fp contract(off)
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

// Sum over aligned groups of N lanes (N a power of two up to 16), every lane of a group
// receiving its group's sum: the symmetric DPP steps of wave_sum_i32 that stay inside
// the group.
template <int N>
__device__ __forceinline__ int lane_group_sum(int v) {
  uint32_t x = static_cast<uint32_t>(v);
  if (N >= 2) x += dpp_u32<kDppXor1>(x);
  if (N >= 4) x += dpp_u32<kDppXor2>(x);
  if (N >= 8) x += dpp_u32<kDppHalfMirror>(x);
  if (N >= 16) x += dpp_u32<kDppMirror>(x);
  return static_cast<int>(x);
}

template <int NT>
__device__ __forceinline__ int block_sum(int v, int* red) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  v = wave_sum_i32(v);
  __syncthreads();
  if (lane == 0) red[wv] = v;
  __syncthreads();
  int s = 0;
#pragma unroll
  for (int i = 0; i < NT / kWave; ++i) s += red[i];
  return s;
}

// Counts of sequence s by a workgroup of NT threads.
template <int NT>
__device__ __forceinline__ void budget_sequence(
    int s, const int32_t* __restrict__ block_idx, const uint8_t* __restrict__ masked,
    const int8_t* __restrict__ hist_len, const float* __restrict__ c1,
    const float* __restrict__ c2, const int32_t* __restrict__ seq_offsets,
    const int32_t* __restrict__ active_block, int T, const BudgetConsts& p,
    int32_t* __restrict__ k_out, int32_t* __restrict__ pairs_out, double* __restrict__ fps_out) {
  constexpr int BG_THREADS = NT;
  constexpr int BG_PER_THREAD = BG_CHUNK / NT;
  constexpr int NW = BG_THREADS / kWave;
  __shared__ double s_key[BG_CHUNK];
  __shared__ int s_idx[BG_CHUNK];
  __shared__ int s_off[BG_PER_THREAD * NW + 1];
  __shared__ int s_red[NW];

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
  const int m = block_sum<NT>(mine, s_red);
  const int n_q = static_cast<int>(floor(p.q * static_cast<double>(m)));

  int total = 0;
  for (int c0 = lo; c0 < hi; c0 += BG_CHUNK) {
    if (!single) load_slice(c0);
    if (m > 0) {
      for (int d0 = lo; d0 < hi; d0 += BG_CHUNK) {
        // stage the candidates of slice d0 in token order: slot = candidates of
        // earlier (r, wave) groups + earlier lanes of this wave (ballot counts)
        const int lane = tid & 63, wv = tid >> 6;
        bool cj[BG_PER_THREAD];
        double kj[BG_PER_THREAD];
        int slot[BG_PER_THREAD];
#pragma unroll
        for (int r = 0; r < BG_PER_THREAD; ++r) {
          const int j = d0 + r * BG_THREADS + tid;
          if (d0 == c0) {
            cj[r] = cand[r];
            kj[r] = key[r];
          } else {
            cj[r] = j < hi && masked[j] != 0 && block_idx[j] == a && hist_len[j] >= 1;
            kj[r] = cj[r] ? rank_key(p, c1[j], c2[j], hist_len[j]) : 0.0;
          }
          const uint64_t bal = __ballot(cj[r]);
          slot[r] = __popcll(bal & ((1ull << lane) - 1));
          if (lane == 0) s_off[r * NW + wv] = __popcll(bal);
        }
        __syncthreads();
        static_assert(BG_PER_THREAD * NW <= kWave, "one wave scans the group counts");
        if (wv == 0) {           // exclusive prefix over the (r, wave) groups
          const int c = lane < BG_PER_THREAD * NW ? s_off[lane] : 0;
          const int incl = wave_inclusive_scan_i32(c, lane);
          if (lane < BG_PER_THREAD * NW) s_off[lane] = incl - c;
          if (lane == kWave - 1) s_off[BG_PER_THREAD * NW] = incl;
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < BG_PER_THREAD; ++r) {
          slot[r] += s_off[r * NW + wv];
          if (cj[r]) {
            s_key[slot[r]] = kj[r];
            s_idx[slot[r]] = d0 + r * BG_THREADS + tid;
          }
        }
        const int cnt = s_off[BG_PER_THREAD * NW];
        __syncthreads();
        if (d0 == c0 && cnt <= kWave) {
          // the candidates rank themselves: LPX lanes per staged candidate x each count
          // the candidates among every LPX-th one that precede x (key descending, token
          // ascending), and a DPP sum over the LPX lanes gives x's rank within the slice
          constexpr int LPX = BG_THREADS / kWave;
          static_assert(LPX >= 1 && LPX <= 16 && (LPX & (LPX - 1)) == 0, "lanes per candidate");
          const int x = tid / LPX, yq = tid % LPX;
          int before = 0;
          if (x < cnt) {
            const double kx = s_key[x];
            const int ix = s_idx[x];
#pragma unroll
            for (int u = 0; u < kWave / LPX; ++u) {
              const int y = yq + LPX * u;
              if (y < cnt) {
                const double ky = s_key[y];
                const int iy = s_idx[y];
                before += (ky > kx || (ky == kx && iy < ix)) ? 1 : 0;
              }
            }
          }
          before = lane_group_sum<LPX>(before);
          __syncthreads();                              // every read of s_idx done
          if (x < cnt && yq == 0) s_idx[x] = before;    // slot -> rank within the slice
          __syncthreads();
#pragma unroll
          for (int r = 0; r < BG_PER_THREAD; ++r)
            if (cand[r]) rank[r] += s_idx[slot[r]];
        } else {
#pragma unroll
          for (int r = 0; r < BG_PER_THREAD; ++r) {
            if (!cand[r]) continue;
            const int i = c0 + r * BG_THREADS + tid;
            int before = 0;
#pragma unroll 4
            for (int x = 0; x < cnt; ++x) {
              const double kx = s_key[x];
              before += (kx > key[r] || (kx == key[r] && s_idx[x] < i)) ? 1 : 0;
            }
            rank[r] += before;
          }
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
    total = block_sum<NT>(total, s_red);
    if (tid == 0 && total != 0) atomicAdd(pairs_out, total);
  }
}

}  // namespace
}  // namespace rfx
