// Variable-count TopK with routing weights (Section 3.2, Eq. (2)) and the
// expert-sorted permutation of the selected expert-token pairs.
#include "common.h"

namespace rfx {
namespace {

// ------------------------------------------------------------------------------------
// TopK: one wave per token.  Lane l holds experts l, l+64, l+128, l+192 as 32-bit
// order-preserving keys of their scores; k_i rounds of a wave-wide max pick the
// experts in rank order.
// ------------------------------------------------------------------------------------
constexpr int TK_WAVES = 4;

// TopK of one token by one wave, in two parts so that the logit loads can be issued
// early: topk_load reads the token's scores (lane l: experts l, l+64, ... over NX
// slots of 64), topk_select writes the first ki experts in rank order and their
// weights at pair_expert / pair_weight [o, o + ki) and returns the lane's expert (-1
// past ki).  Ranking is by score, ties to the lower expert index.  Each round takes the
// wave maximum of the lanes' largest remaining 32-bit order keys; a ballot names the
// lane holding it, and equal keys in several lanes go to the lowest expert index.
// Lanes past E hold key 0, below every finite score's key.
template <int NX>
struct TopkRow {
  uint32_t key[NX];
  float val[NX];
};

// A score may arrive as n_parts partials part_stride floats apart (the split-K router
// tiles of the fused router + budget launch): they are added in order, then the bias
// (nullable).  n_parts = 1 with no bias reads finished scores.
template <int NX>
__device__ __forceinline__ TopkRow<NX> topk_load(const float* __restrict__ row, int E,
                                                 int n_parts = 1, size_t part_stride = 0,
                                                 const float* __restrict__ bias = nullptr) {
  const int lane = threadIdx.x & 63;
  TopkRow<NX> r;
  // unconditional loads (lanes past E read expert E-1 and discard it), all in flight
  // together rather than one guarded load and wait at a time
  float v[NX];
#pragma unroll
  for (int j = 0; j < NX; ++j) {
    const int e = lane + kWave * j;
    v[j] = row[e < E ? e : E - 1];
  }
  if (n_parts > 1) {
    constexpr int PB = 8 / NX > 0 ? 8 / NX : 1;     // partials per batch: 8 loads in flight
    for (int s0 = 1; s0 < n_parts; s0 += PB) {
      float pv[PB][NX];
#pragma unroll
      for (int u = 0; u < PB; ++u)
#pragma unroll
        for (int j = 0; j < NX; ++j) {
          const int e = lane + kWave * j, sp = min(s0 + u, n_parts - 1);
          pv[u][j] = row[static_cast<size_t>(sp) * part_stride + (e < E ? e : E - 1)];
        }
#pragma unroll
      for (int u = 0; u < PB; ++u)
#pragma unroll
        for (int j = 0; j < NX; ++j)
          if (s0 + u < n_parts) v[j] += pv[u][j];
    }
  }
  if (bias != nullptr) {
#pragma unroll
    for (int j = 0; j < NX; ++j) {
      const int e = lane + kWave * j;
      v[j] += bias[e < E ? e : E - 1];
    }
  }
#pragma unroll
  for (int j = 0; j < NX; ++j) {
    const bool ok = lane + kWave * j < E;
    r.val[j] = ok ? v[j] : 0.0f;
    r.key[j] = ok ? f32_order_key(v[j]) : 0u;
  }
  return r;
}

template <int NX>
__device__ __forceinline__ int topk_select(const TopkRow<NX>& r, int ki, int E, int norm_topk,
                                           int o, int32_t* __restrict__ pair_expert,
                                           float* __restrict__ pair_weight) {
  const int lane = threadIdx.x & 63;
  // The lane's own keys, sorted once into descending order (equal keys: lower slot,
  // i.e. lower expert, first), so that a round compares only the lanes' heads: the
  // wave maximum of the heads is the round's best key, and the lane holding it pops
  // its head.  A lane's head is its largest remaining key and, among equal ones, its
  // lowest expert, so the lowest expert among the heads equal to the maximum is the
  // lowest expert of the whole token with that key.
  // (the slots of the sorted keys are packed 2 bits each, position x at bits 2x)
  uint32_t key[NX];
  uint32_t slots = 0;
#pragma unroll
  for (int x = 0; x < NX; ++x) {
    key[x] = r.key[x];
    slots |= static_cast<uint32_t>(x) << (2 * x);
  }
#pragma unroll
  for (int a = 1; a < NX; ++a)          // insertion sort, fully unrolled (registers)
#pragma unroll
    for (int b = a; b > 0; --b) {
      const bool sw = key[b] > key[b - 1];     // strictly greater: ties keep slot order
      const uint32_t k0 = key[b - 1], k1 = key[b];
      key[b - 1] = sw ? k1 : k0;
      key[b] = sw ? k0 : k1;
      const uint32_t s0 = (slots >> (2 * (b - 1))) & 3u, s1 = (slots >> (2 * b)) & 3u;
      const uint32_t swapped = (slots & ~(15u << (2 * (b - 1)))) | (s1 << (2 * (b - 1))) | (s0 << (2 * b));
      slots = sw ? swapped : slots;
    }
  int my_e = 0;
  uint32_t my_key = 0u, top_key = 0u;
  for (int j = 0; j < ki; ++j) {
    const uint32_t best = wave_max_u32(key[0]);
    const uint64_t m = __ballot(key[0] == best);
    int wl = __builtin_ctzll(m);
    if (__builtin_popcountll(m) > 1) {
      // equal heads in several lanes (rare): the lowest expert index among them, as
      // the wave maximum of the complemented indices
      const uint32_t c =
          key[0] == best ? ~static_cast<uint32_t>(lane + kWave * static_cast<int>(slots & 3u)) : 0u;
      wl = static_cast<int>(~wave_max_u32(c)) & (kWave - 1);
    }
    const int e = wl + kWave * static_cast<int>(__builtin_amdgcn_readlane(slots, wl) & 3u);
    if (lane == wl) {                     // the winner pops its head
#pragma unroll
      for (int x = 0; x + 1 < NX; ++x) key[x] = key[x + 1];
      key[NX - 1] = 0u;
      slots >>= 2;
    }
    if (lane == j) { my_e = e; my_key = best; }
    if (j == 0) top_key = best;
  }
  const float my_r = f32_from_order_key(my_key), rmax = f32_from_order_key(top_key);
  float den;
  if (norm_topk) {
    den = wave_sum_f32(lane < ki ? expf(my_r - rmax) : 0.0f);
  } else {
    float part = 0.0f;
#pragma unroll
    for (int j = 0; j < NX; ++j)
      if (lane + kWave * j < E) part += expf(f32_from_order_key(r.key[j]) - rmax);
    den = wave_sum_f32(part);
  }
  if (lane < ki) {
    pair_expert[o + lane] = my_e;
    pair_weight[o + lane] = expf(my_r - rmax) / den;
  }
  return lane < ki ? my_e : -1;
}

// Slots of 64 experts per lane for E experts.
inline int topk_slots(int E) { return (E + kWave - 1) / kWave; }

template <int NX>
__global__ __launch_bounds__(TK_WAVES * kWave) void topk_kernel(
    const float* __restrict__ logits, const int32_t* __restrict__ k, int T, int E, int k_max,
    int norm_topk, const int32_t* __restrict__ pair_offsets, int32_t* __restrict__ pair_expert,
    float* __restrict__ pair_weight) {
  const int i = blockIdx.x * TK_WAVES + (threadIdx.x >> 6);
  if (i >= T) return;
  const int ki = clamp_count(k[i], k_max);
  if (ki == 0) return;
  topk_select<NX>(topk_load<NX>(logits + static_cast<size_t>(i) * E, E), ki, E, norm_topk, pair_offsets[i],
              pair_expert, pair_weight);
}

// ------------------------------------------------------------------------------------
// Score-derived counts (Appendix B).  One wave per token: lane l holds experts l,
// l+64, l+128, l+192; the routing mass exp(r_e - r_max) / sum_e' exp(r_e' - r_max)
// is evaluated in fp64.  Top-p walks the experts in TopK order (the same 64-bit keys
// as the TopK kernel), adding their mass in that order until it reaches p; at most
// k_max steps are needed, since longer prefixes are clamped to k_max anyway.
// ------------------------------------------------------------------------------------
__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__global__ __launch_bounds__(TK_WAVES * kWave) void count_rule_kernel(
    const float* __restrict__ logits, int T, int E, int rule, double thr, int k_min, int k_max,
    int32_t* __restrict__ k_out, int32_t* __restrict__ pairs_out) {
  const int lane = threadIdx.x & 63;
  const int i = blockIdx.x * TK_WAVES + (threadIdx.x >> 6);
  if (i >= T) return;
  const float* row = logits + static_cast<size_t>(i) * E;
  uint64_t key[4];
  float val[4];
  uint64_t best = 0;
  float v[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {     // unconditional loads, all in flight together
    const int e = lane + kWave * j;
    v[j] = row[e < E ? e : E - 1];
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = lane + kWave * j;
    val[j] = e < E ? v[j] : 0.0f;
    key[j] = e < E ? (static_cast<uint64_t>(f32_order_key(val[j])) << 32) | (0xffffu - e) : 0;
    best = key[j] > best ? key[j] : best;
  }
  best = wave_max_u64(best);
  const double rmax = static_cast<double>(f32_from_order_key(static_cast<uint32_t>(best >> 32)));
  double ex[4];
  double part = 0.0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    ex[j] = lane + kWave * j < E ? exp(static_cast<double>(val[j]) - rmax) : 0.0;
    part += ex[j];
  }
  const double den = wave_sum_f64(part);
  int n;
  if (rule == REFLEX_RULE_THRESHOLD) {
    int c = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) c += (lane + kWave * j < E && ex[j] / den > thr) ? 1 : 0;
    n = wave_sum_i32(c);
  } else {
    n = k_max;
    double cum = 0.0;
    for (int j = 0; j < k_max; ++j) {
      uint64_t b = key[0];
#pragma unroll
      for (int x = 1; x < 4; ++x) b = key[x] > b ? key[x] : b;
      b = wave_max_u64(b);
      const int e = 0xffff - static_cast<int>(b & 0xffffu);
      const int slot = e >> 6;
      double mine = 0.0;
#pragma unroll
      for (int x = 0; x < 4; ++x) mine = x == slot ? ex[x] : mine;
      const double m = __shfl(mine, e & 63, kWave);
#pragma unroll
      for (int x = 0; x < 4; ++x)        // consume the winner (static indices: registers)
        key[x] = ((e & 63) == lane && x == slot) ? 0 : key[x];
      cum += m / den;
      if (cum >= thr) {
        n = j + 1;
        break;
      }
    }
  }
  const int k = n < k_min ? k_min : (n > k_max ? k_max : n);
  if (lane == 0) {
    k_out[i] = k;
    if (pairs_out != nullptr && k != 0) atomicAdd(pairs_out, k);
  }
}

// ------------------------------------------------------------------------------------
// Permutation: stable counting sort of the token-major pair list by expert.
//   1. per 1024-pair tile, an LDS histogram over experts
//   2. one workgroup turns the [tile][expert] counts into start rows, expert-major
//      then tile-minor, writes expert_offsets and (optionally) the grouped GEMM's
//      per-expert M-tile prefix
//   3. per tile: an LDS table of each pair's owning token, then 256-pair steps in
//      which each wave finds the lanes holding the same expert with eight ballots
//      (one per bit of the expert id) and ranks them by lane; the waves of a step
//      are ordered through LDS counts, so rows follow pair order within each expert
//      (i.e. token order).
// ------------------------------------------------------------------------------------
constexpr int PM_TILE = 1024;
constexpr int PM_THREADS = 256;
constexpr int PM_STEPS = PM_TILE / PM_THREADS;
constexpr int PM_SCAN_THREADS = 1024;

__device__ __forceinline__ int pair_count(const int32_t* pairs, int cap) {
  int P = *pairs;
  return P < 0 ? 0 : (P > cap ? cap : P);
}

__global__ __launch_bounds__(PM_THREADS) void perm_hist_kernel(const int32_t* __restrict__ pair_expert,
                                                               const int32_t* __restrict__ pairs,
                                                               int cap, int E,
                                                               int32_t* __restrict__ hist) {
  __shared__ int cnt[REFLEX_MAX_EXPERTS];
  const int P = pair_count(pairs, cap);
  const int t = blockIdx.x, tid = threadIdx.x;
  for (int e = tid; e < E; e += PM_THREADS) cnt[e] = 0;
  __syncthreads();
  const int begin = t * PM_TILE;
#pragma unroll
  for (int j = 0; j < PM_STEPS; ++j) {
    const int p = begin + j * PM_THREADS + tid;
    if (p < P) {
      int e = pair_expert[p];
      e = e < 0 ? 0 : (e >= E ? E - 1 : e);
      atomicAdd(&cnt[e], 1);
    }
  }
  __syncthreads();
  for (int e = tid; e < E; e += PM_THREADS) hist[static_cast<size_t>(t) * E + e] = cnt[e];
}

// 1024 threads: group q = tid / 256 owns a contiguous quarter of the tiles, thread
// e = tid % 256 one expert.  Group sums give expert totals; group 0 scans them into
// expert_offsets (and the grouped GEMM's per-expert M-tile prefix); each group then
// rewrites its tiles' counts as start rows (expert base + earlier groups + earlier
// tiles of the group).
__global__ __launch_bounds__(PM_SCAN_THREADS) void perm_scan_kernel(
    int32_t* __restrict__ hist, int n_tiles, int E, int32_t* __restrict__ expert_offsets,
    int32_t* __restrict__ gemm_tile_off) {
  __shared__ int s_part[4][REFLEX_MAX_EXPERTS];
  __shared__ int s_base[REFLEX_MAX_EXPERTS];
  __shared__ int s_wave[8];
  const int tid = threadIdx.x, q = tid >> 8, e = tid & 255, lane = tid & 63, wv = tid >> 6;
  const int per = (n_tiles + 3) / 4;
  const int tb = q * per, te = min(n_tiles, tb + per);
  int n = 0;
  if (e < E) {
#pragma unroll 8
    for (int t = tb; t < te; ++t) n += hist[static_cast<size_t>(t) * E + e];   // 8 loads in flight
  }
  s_part[q][e] = n;
  __syncthreads();
  int tot = 0, incl = 0, tiles = 0, tincl = 0;
  if (q == 0) {            // waves 0..3
    tot = e < E ? s_part[0][e] + s_part[1][e] + s_part[2][e] + s_part[3][e] : 0;
    tiles = (tot + kGemmBM - 1) / kGemmBM;
    incl = wave_inclusive_scan_i32(tot, lane);
    tincl = wave_inclusive_scan_i32(tiles, lane);
    if (lane == 63) {
      s_wave[wv] = incl;
      s_wave[4 + wv] = tincl;
    }
  }
  __syncthreads();
  if (q == 0) {
    int off = 0, toff = 0;
    for (int x = 0; x < wv; ++x) {
      off += s_wave[x];
      toff += s_wave[4 + x];
    }
    const int base = off + incl - tot;
    s_base[e] = base;
    if (e < E) {
      expert_offsets[e] = base;
      if (e == E - 1) expert_offsets[E] = base + tot;
      if (gemm_tile_off != nullptr) {
        gemm_tile_off[e] = toff + tincl - tiles;
        if (e == E - 1) gemm_tile_off[E] = toff + tincl;
      }
    }
  }
  __syncthreads();
  if (e < E) {
    int run = s_base[e];
    for (int qq = 0; qq < q; ++qq) run += s_part[qq][e];
    // start rows of the group's tiles, in batches of 8 whose counts are loaded together
    for (int t0 = tb; t0 < te; t0 += 8) {
      int c[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {       // unconditional loads (clamped), then selects
        const int tt = t0 + j < te ? t0 + j : te - 1;
        c[j] = hist[static_cast<size_t>(tt) * E + e];
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) c[j] = t0 + j < te ? c[j] : 0;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (t0 + j < te) hist[static_cast<size_t>(t0 + j) * E + e] = run;
        run += c[j];
      }
    }
  }
}

// The tokens that own pairs pa and pb: the largest i in [0, T) with off[i] <= p (off is
// the nondecreasing pair-offset scan), for both at once, by the whole workgroup.  Each
// round samples 256 evenly spaced entries of the current range in one load per thread
// and keeps the bracket the count of samples <= p points to: two rounds of dependent
// loads for up to 65536 tokens instead of a 16-step binary search by one thread.
__device__ __forceinline__ void owner_tokens(const int32_t* __restrict__ off, int T, int pa,
                                             int pb, int* s_out) {
  int lo_a = 0, n_a = T, lo_b = 0, n_b = T;      // candidate ranges [lo, lo + n)
  while (n_a > 1 || n_b > 1) {                   // uniform across the workgroup
    const int st_a = (n_a + PM_THREADS - 1) / PM_THREADS, st_b = (n_b + PM_THREADS - 1) / PM_THREADS;
    const int ia = threadIdx.x * st_a, ib = threadIdx.x * st_b;
    const bool fa = ia < n_a && off[lo_a + ia] <= pa;
    const bool fb = ib < n_b && off[lo_b + ib] <= pb;
    const int ca = __syncthreads_count(fa), cb = __syncthreads_count(fb);
    const int ka = ca > 0 ? ca - 1 : 0, kb = cb > 0 ? cb - 1 : 0;   // last sample <= p
    lo_a += ka * st_a;
    n_a = min(st_a, n_a - ka * st_a);
    lo_b += kb * st_b;
    n_b = min(st_b, n_b - kb * st_b);
  }
  if (threadIdx.x == 0) {
    s_out[0] = lo_a;
    s_out[1] = lo_b;
  }
}

__global__ __launch_bounds__(PM_THREADS) void perm_scatter_kernel(
    const int32_t* __restrict__ pair_offsets, const int32_t* __restrict__ pair_expert,
    const int32_t* __restrict__ pairs, int T, int cap, int E, const int32_t* __restrict__ start,
    int32_t* __restrict__ sorted_token, int32_t* __restrict__ pair_to_sorted) {
  __shared__ int run[REFLEX_MAX_EXPERTS];
  __shared__ int wcnt[PM_THREADS / kWave][REFLEX_MAX_EXPERTS];
  __shared__ int owner[PM_TILE];
  __shared__ int s_tok[2];
  const int P = pair_count(pairs, cap);
  const int t = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int begin = t * PM_TILE;
  if (begin >= P) return;
  const int end = min(begin + PM_TILE, P);
  for (int e = tid; e < E; e += PM_THREADS) {
    run[e] = start[static_cast<size_t>(t) * E + e];
#pragma unroll
    for (int w = 0; w < PM_THREADS / kWave; ++w) wcnt[w][e] = 0;
  }
  owner_tokens(pair_offsets, T, begin, end - 1, s_tok);
  __syncthreads();
  // owning token of every pair of the tile
  for (int i = s_tok[0] + tid; i <= s_tok[1]; i += PM_THREADS) {
    const int p0 = max(pair_offsets[i], begin), p1 = min(pair_offsets[i + 1], end);
    for (int p = p0; p < p1; ++p) owner[p - begin] = i;
  }
  __syncthreads();
  const uint64_t lt_mask = (1ull << lane) - 1ull;
  for (int j = 0; j < PM_STEPS; ++j) {
    const int p = begin + j * PM_THREADS + tid;
    const bool valid = p < end;
    int e = 0, tok = 0;
    if (valid) {
      e = pair_expert[p];
      e = e < 0 ? 0 : (e >= E ? E - 1 : e);
      tok = owner[p - begin];
    }
    uint64_t same = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool bit = (e >> b) & 1;
      const uint64_t m = __ballot(bit);
      same &= bit ? m : ~m;
    }
    const int local = __popcll(same & lt_mask);
    if (valid && local == 0) wcnt[wv][e] = __popcll(same);
    __syncthreads();
    if (valid) {
      int pos = run[e] + local;
      for (int w = 0; w < wv; ++w) pos += wcnt[w][e];
      sorted_token[pos] = tok;
      pair_to_sorted[p] = pos;
    }
    __syncthreads();
    for (int x = tid; x < E; x += PM_THREADS) {
      int add = 0;
#pragma unroll
      for (int w = 0; w < PM_THREADS / kWave; ++w) {
        add += wcnt[w][x];
        wcnt[w][x] = 0;
      }
      run[x] += add;
    }
    __syncthreads();
    if (begin + (j + 1) * PM_THREADS >= end) break;   // uniform across the workgroup
  }
}

// Small pair lists (capacity <= PS_MAX_CAP): the whole permutation in one
// 1024-thread workgroup, with every pair's owning token in an LDS table: LDS
// histogram, expert scan (+ GEMM tile plan), then 1024-pair steps ranked exactly as
// in the per-tile scatter above, carrying each expert's running row across steps.
// Saves two launches and their gaps where the list is short.
constexpr int PS_THREADS = 1024;
constexpr int PS_WAVES = PS_THREADS / kWave;
constexpr int PS_MAX_CAP = 16384;

__device__ __forceinline__ void perm_small_run(
    const int32_t* __restrict__ pair_offsets, const int32_t* __restrict__ pair_expert,
    const int32_t* __restrict__ pairs, int T, int cap, int E, int32_t* __restrict__ expert_offsets,
    int32_t* __restrict__ sorted_token, int32_t* __restrict__ pair_to_sorted,
    int32_t* __restrict__ gemm_tile_off) {
  __shared__ int owner[PS_MAX_CAP];
  __shared__ uint8_t pexp[PS_MAX_CAP];           // each pair's expert (E <= 256)
  __shared__ int cnt[REFLEX_MAX_EXPERTS], run[REFLEX_MAX_EXPERTS];
  __shared__ int wcnt[PS_WAVES][REFLEX_MAX_EXPERTS];
  __shared__ int s_wave[8];
  const int P = pair_count(pairs, cap);
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  for (int x = tid; x < PS_WAVES * REFLEX_MAX_EXPERTS; x += PS_THREADS) (&wcnt[0][0])[x] = 0;
  for (int e = tid; e < REFLEX_MAX_EXPERTS; e += PS_THREADS) cnt[e] = 0;
  __syncthreads();
  for (int t = tid; t < T; t += PS_THREADS) {
    const int p0 = max(pair_offsets[t], 0), p1 = min(pair_offsets[t + 1], P);
    for (int p = p0; p < p1; ++p) owner[p] = t;
  }
  for (int p = tid; p < P; p += PS_THREADS) {
    int e = pair_expert[p];
    e = e < 0 ? 0 : (e >= E ? E - 1 : e);
    pexp[p] = static_cast<uint8_t>(e);
    atomicAdd(&cnt[e], 1);
  }
  __syncthreads();
  // expert scan (waves 0..3, one expert per thread) and the GEMM's M-tile prefix
  int n = 0, incl = 0, tiles = 0, tincl = 0;
  if (tid < REFLEX_MAX_EXPERTS) {
    n = tid < E ? cnt[tid] : 0;
    tiles = (n + kGemmBM - 1) / kGemmBM;
    incl = wave_inclusive_scan_i32(n, lane);
    tincl = wave_inclusive_scan_i32(tiles, lane);
    if (lane == 63) {
      s_wave[wv] = incl;
      s_wave[4 + wv] = tincl;
    }
  }
  __syncthreads();
  if (tid < E) {
    int off = 0, toff = 0;
    for (int x = 0; x < wv; ++x) {
      off += s_wave[x];
      toff += s_wave[4 + x];
    }
    const int base = off + incl - n;
    run[tid] = base;
    expert_offsets[tid] = base;
    if (tid == E - 1) expert_offsets[E] = base + n;
    if (gemm_tile_off != nullptr) {
      gemm_tile_off[tid] = toff + tincl - tiles;
      if (tid == E - 1) gemm_tile_off[E] = toff + tincl;
    }
  }
  __syncthreads();
  const uint64_t lt_mask = (1ull << lane) - 1ull;
  for (int c = 0; c < P; c += PS_THREADS) {      // uniform across the workgroup
    const int p = c + tid;
    const bool valid = p < P;
    int e = 0, tok = 0;
    if (valid) {
      e = pexp[p];
      tok = owner[p];
    }
    uint64_t same = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool bit = (e >> b) & 1;
      const uint64_t m = __ballot(bit);
      same &= bit ? m : ~m;
    }
    const int local = __popcll(same & lt_mask);
    if (valid && local == 0) wcnt[wv][e] = __popcll(same);
    __syncthreads();
    if (valid) {
      int pos = run[e] + local;
#pragma unroll
      for (int w = 0; w < PS_WAVES; ++w) pos += w < wv ? wcnt[w][e] : 0;
      sorted_token[pos] = tok;
      pair_to_sorted[p] = pos;
    }
    __syncthreads();
    for (int x = tid; x < E; x += PS_THREADS) {
      int add = 0;
#pragma unroll
      for (int w = 0; w < PS_WAVES; ++w) {
        add += wcnt[w][x];
        wcnt[w][x] = 0;
      }
      run[x] += add;
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(PS_THREADS) void perm_small_kernel(
    const int32_t* __restrict__ pair_offsets, const int32_t* __restrict__ pair_expert,
    const int32_t* __restrict__ pairs, int T, int cap, int E, int32_t* __restrict__ expert_offsets,
    int32_t* __restrict__ sorted_token, int32_t* __restrict__ pair_to_sorted,
    int32_t* __restrict__ gemm_tile_off) {
  perm_small_run(pair_offsets, pair_expert, pairs, T, cap, E, expert_offsets, sorted_token,
                 pair_to_sorted, gemm_tile_off);
}

// ------------------------------------------------------------------------------------
// Pair offsets, TopK and (for small layers) the permutation in one launch.  Workgroup
// b owns tokens 16 b .. 16 b + 15, one wave each: it sums the counts of all earlier
// tokens itself (no separate scan launch), scans its own 16, writes pair_offsets and
// runs TopK.  With `done` given, it also ranks each of its pairs among the workgroup's
// pairs of the same expert (an LDS bit mask of the tokens that chose each expert),
// keeps (token, rank) in pair_to_sorted and its per-expert counts in hist[b][.]; the
// workgroup that finishes last (agent-scope acquire-release counter, so every other
// workgroup's pairs are visible to it) turns hist into per-(workgroup, expert) start
// rows, writes expert_offsets and the GEMM tile plan, and scatters every pair to
//   expert_offsets[e] + start[b][e] + rank,
// the same stable (expert, token) order as the permutation kernels.  It then resets the
// counter to zero, which is where the launch before this one left it.
// ------------------------------------------------------------------------------------
constexpr int RF_WAVES = 16;
constexpr int RF_HIST_MAX = 16384;       // workgroups x experts held in LDS by the last one

// SORT: this launch sorts the pairs (its last workgroup, above).  Without it the kernel
// holds none of that step's LDS tables, so two workgroups fit a CU instead of one.
template <int NX, bool SORT>
__global__ __launch_bounds__(RF_WAVES * kWave) void route_fused_kernel(
    const float* __restrict__ logits, int n_parts, size_t part_stride,
    const float* __restrict__ bias, float* __restrict__ logits_out,
    const int32_t* __restrict__ k, int T, int E, int k_max,
    int norm_topk, int32_t* __restrict__ pair_offsets, int32_t* __restrict__ pair_expert,
    float* __restrict__ pair_weight, int32_t* __restrict__ pairs_out, int32_t* __restrict__ done,
    int32_t* __restrict__ hist, int32_t* __restrict__ expert_offsets,
    int32_t* __restrict__ sorted_token, int32_t* __restrict__ pair_to_sorted,
    int32_t* __restrict__ gemm_tile_off) {
  __shared__ int s_before[RF_WAVES], s_cnt[RF_WAVES];
  __shared__ uint32_t s_mask[REFLEX_MAX_EXPERTS];
  __shared__ int s_last;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int t0 = blockIdx.x * RF_WAVES;
  for (int e = tid; e < REFLEX_MAX_EXPERTS; e += RF_WAVES * kWave) s_mask[e] = 0;
  const int i = t0 + wv;
  // this token's scores are loaded first: their latency overlaps the count prefix
  const TopkRow<NX> row = topk_load<NX>(logits + static_cast<size_t>(i < T ? i : T - 1) * E, E,
                                        n_parts, part_stride, bias);
  if (logits_out != nullptr && i < T) {
#pragma unroll
    for (int j = 0; j < NX; ++j)
      if (lane + kWave * j < E) logits_out[static_cast<size_t>(i) * E + lane + kWave * j] = row.val[j];
  }
  int part = 0;     // (unrolled so that several count loads are in flight at once)
#pragma unroll 8
  for (int t = tid; t < t0; t += RF_WAVES * kWave) part += clamp_count(k[t], k_max);
  part = wave_sum_i32(part);
  const int ki = i < T ? clamp_count(k[i], k_max) : 0;
  if (lane == 0) {
    s_before[wv] = part;
    s_cnt[wv] = ki;
  }
  __syncthreads();
  int base = 0, off = 0, blk = 0;
#pragma unroll
  for (int w = 0; w < RF_WAVES; ++w) {
    base += s_before[w];
    off += w < wv ? s_cnt[w] : 0;
    blk += s_cnt[w];
  }
  off += base;
  if (i < T && lane == 0) pair_offsets[i] = off;
  if (blockIdx.x == gridDim.x - 1 && tid == 0) {     // the last block closes the list
    pair_offsets[T] = base + blk;
    if (pairs_out) pairs_out[0] = base + blk;
  }
  int my_e = -1;
  if (ki > 0) my_e = topk_select<NX>(row, ki, E, norm_topk, off, pair_expert, pair_weight);
  if (hist == nullptr) return;     // the permutation launches sort the pairs
  if (my_e >= 0) atomicOr(&s_mask[my_e], 1u << wv);
  __syncthreads();
  if (my_e >= 0)       // (token, rank among this workgroup's tokens that chose my_e)
    pair_to_sorted[off + lane] = (i << 5) | __popc(s_mask[my_e] & ((1u << wv) - 1u));
  if (!SORT) {     // the block-sort launches finish: counts expert-major
    for (int e = tid; e < E; e += RF_WAVES * kWave)
      hist[static_cast<size_t>(e) * gridDim.x + blockIdx.x] = __popc(s_mask[e]);
    return;
  }
  for (int e = tid; e < E; e += RF_WAVES * kWave)
    hist[static_cast<size_t>(blockIdx.x) * E + e] = __popc(s_mask[e]);
  if constexpr (SORT) {
  // every wave's stores acknowledged (vmcnt 0, i.e. in this XCD's L2) before the
  // barrier, so the counter's agent-scope release by thread 0 writes them all back
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (tid == 0)
    s_last = __hip_atomic_fetch_add(done, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT) ==
             static_cast<int>(gridDim.x) - 1;
  __syncthreads();
  if (!s_last) return;

  // ---- the last workgroup: start rows and the scatter ----
  constexpr int RF_BATCH = 8;                       // pairs per thread per scatter pass
  constexpr int RF_PASS = RF_BATCH * RF_WAVES * kWave;
  __shared__ int s_tab[RF_HIST_MAX];
  __shared__ int s_part[RF_WAVES][REFLEX_MAX_EXPERTS];
  __shared__ int s_eo[REFLEX_MAX_EXPERTS];
  __shared__ int s_wave[8];
  constexpr int RF_THREADS = RF_WAVES * kWave;
  constexpr int RF_TAB_PT = RF_HIST_MAX / RF_THREADS;     // table words per thread, at most
  const int G = gridDim.x, n_tab = G * E;
  // the whole table's loads in flight at once (a uniform branch skips the unused
  // slices), then the pair count's, then one wait
  int hv[RF_TAB_PT];
#pragma unroll
  for (int j = 0; j < RF_TAB_PT; ++j)
    if (j * RF_THREADS < n_tab) hv[j] = hist[min(tid + j * RF_THREADS, n_tab - 1)];
  const int P = pair_offsets[T];
#pragma unroll
  for (int j = 0; j < RF_TAB_PT; ++j)
    if (j * RF_THREADS < n_tab && tid + j * RF_THREADS < n_tab) s_tab[tid + j * RF_THREADS] = hv[j];
  // the first pass's scatter inputs do not depend on the start rows: their loads go
  // out now and their latency hides behind the scans (a barrier does not wait for them)
  int v[RF_BATCH], ev[RF_BATCH];
  auto load_pass = [&](int p0) {
#pragma unroll
    for (int j = 0; j < RF_BATCH; ++j) {
      const int p = p0 + j * RF_WAVES * kWave + tid;
      const int q = p < P ? p : 0;     // (P >= 1 here: the loads stay inside the pair list)
      v[j] = pair_to_sorted[q];
      ev[j] = pair_expert[q];
    }
  };
  if (P > 0) load_pass(0);
  __syncthreads();
  // start[w][e] = sum of column e above row w.  Wave q owns rows [q rpw, (q+1) rpw) and
  // lane l experts l, l+64, ...: a row's experts lie in consecutive words (no bank
  // conflicts).  Pass 1: per-wave column sums; pass 2: exclusive walk down the rows
  // from the sum of the waves above.
  const int rpw = (G + RF_WAVES - 1) / RF_WAVES;
  const int w_lo = wv * rpw, w_hi = min(G, w_lo + rpw);
  for (int e = lane; e < E; e += kWave) {
    int sum = 0;
    for (int w = w_lo; w < w_hi; ++w) sum += s_tab[w * E + e];
    s_part[wv][e] = sum;
  }
  __syncthreads();
  for (int e = lane; e < E; e += kWave) {
    int run = 0;
    for (int q = 0; q < wv; ++q) run += s_part[q][e];
    for (int w = w_lo; w < w_hi; ++w) {
      const int c = s_tab[w * E + e];
      s_tab[w * E + e] = run;
      run += c;
    }
    if (wv == RF_WAVES - 1) s_eo[e] = run;     // the last wave's walk ends at the total
  }
  __syncthreads();
  const int tot = tid < E ? s_eo[tid] : 0;
  int incl = 0, tiles = 0, tincl = 0;
  if (tid < REFLEX_MAX_EXPERTS) {
    tiles = (tot + kGemmBM - 1) / kGemmBM;
    incl = wave_inclusive_scan_i32(tot, lane);
    tincl = wave_inclusive_scan_i32(tiles, lane);
    if (lane == 63) {
      s_wave[wv] = incl;
      s_wave[4 + wv] = tincl;
    }
  }
  __syncthreads();
  if (tid < E) {
    int eoff = 0, toff = 0;
    for (int x = 0; x < wv; ++x) {
      eoff += s_wave[x];
      toff += s_wave[4 + x];
    }
    const int ebase = eoff + incl - tot;
    s_eo[tid] = ebase;
    expert_offsets[tid] = ebase;
    if (tid == E - 1) expert_offsets[E] = ebase + tot;
    gemm_tile_off[tid] = toff + tincl - tiles;
    if (tid == E - 1) gemm_tile_off[E] = toff + tincl;
  }
  __syncthreads();
  // the scatter: pair p of workgroup w's token t with rank r in its expert e goes to
  // expert_offsets[e] + start[w][e] + r
  for (int p0 = 0; p0 < P; p0 += RF_PASS) {
    if (p0 > 0) load_pass(p0);
#pragma unroll
    for (int j = 0; j < RF_BATCH; ++j) {
      const int p = p0 + j * RF_WAVES * kWave + tid;
      if (p >= P) continue;
      const int e = ev[j] < 0 ? 0 : (ev[j] >= E ? E - 1 : ev[j]);
      const int t = v[j] >> 5, w = t / RF_WAVES;
      const int pos = s_eo[e] + s_tab[w * E + e] + (v[j] & 31);
      sorted_token[pos] = t;
      pair_to_sorted[p] = pos;
    }
  }
  if (tid == 0) __hip_atomic_store(done, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// ------------------------------------------------------------------------------------
// Block sort (layers above RF_HIST_MAX counts): the route launch has ranked every pair
// among its 16-token block's pairs of the same expert (pair_to_sorted = token << 5 |
// rank) and written the blocks' per-expert counts expert-major, cnt[e][b].  Two
// launches finish the stable (expert, token) order, with no workgroup walking every
// pair and no cross-workgroup wait:
//   column scan: workgroup e turns row e of cnt into start rows (the pairs of expert e
//   in earlier blocks), in place, and writes the expert's total to tot[e];
//   scatter: every workgroup scans the E totals into expert bases (workgroup 0 also
//   writes them as expert_offsets, with the GEMM tile plan) and sends each pair of its
//   block b to base[e] + start[e][b] + rank.
// ------------------------------------------------------------------------------------
constexpr int BS_THREADS = 1024;
constexpr long BS_MAX_COUNTS = 1L << 20;   // (block, expert) counts the block sort takes

__global__ __launch_bounds__(BS_THREADS) void block_colscan_kernel(int32_t* __restrict__ cnt,
                                                                   int G,
                                                                   int32_t* __restrict__ tot) {
  __shared__ int s_wave[BS_THREADS / kWave];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  int32_t* row = cnt + static_cast<size_t>(blockIdx.x) * G;
  int run = 0;     // pairs of this expert in the blocks before the current chunk
  for (int b0 = 0; b0 < G; b0 += BS_THREADS) {     // uniform across the workgroup
    const int b = b0 + tid;
    const int c = b < G ? row[b] : 0;
    const int incl = wave_inclusive_scan_i32(c, lane);
    if (lane == 63) s_wave[wv] = incl;
    __syncthreads();
    int before = run, chunk = 0;
#pragma unroll
    for (int w = 0; w < BS_THREADS / kWave; ++w) {
      before += w < wv ? s_wave[w] : 0;
      chunk += s_wave[w];
    }
    if (b < G) row[b] = before + incl - c;
    run += chunk;
    __syncthreads();     // s_wave is rewritten by the next chunk
  }
  if (tid == 0) tot[blockIdx.x] = run;
}

__global__ __launch_bounds__(256) void block_scatter_kernel(
    const int32_t* __restrict__ pair_offsets, const int32_t* __restrict__ pair_expert, int T,
    int cap, int E, int G, const int32_t* __restrict__ start, const int32_t* __restrict__ tot,
    int32_t* __restrict__ expert_offsets, int32_t* __restrict__ gemm_tile_off,
    int32_t* __restrict__ sorted_token, int32_t* __restrict__ pair_to_sorted) {
  __shared__ int s_base[REFLEX_MAX_EXPERTS];
  __shared__ int s_wave[8];
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int t0 = b * RF_WAVES, t1 = min(T, t0 + RF_WAVES);
  int p0 = pair_offsets[t0], p1 = pair_offsets[t1];
  // expert bases: exclusive scan of the totals (thread e holds expert e), then this
  // block's start row added
  const int n = tid < E ? tot[tid] : 0;
  const int st = tid < E ? start[static_cast<size_t>(tid) * G + b] : 0;
  const int incl = wave_inclusive_scan_i32(n, lane);
  const int tiles = (n + kGemmBM - 1) / kGemmBM;
  const int tincl = b == 0 ? wave_inclusive_scan_i32(tiles, lane) : 0;
  if (lane == 63) {
    s_wave[wv] = incl;
    s_wave[4 + wv] = tincl;
  }
  __syncthreads();
  if (tid < E) {
    int eoff = 0, toff = 0;
    for (int x = 0; x < wv; ++x) {
      eoff += s_wave[x];
      toff += s_wave[4 + x];
    }
    const int base = eoff + incl - n;
    s_base[tid] = base + st;
    if (b == 0) {
      expert_offsets[tid] = base;
      if (tid == E - 1) expert_offsets[E] = base + n;
      gemm_tile_off[tid] = toff + tincl - tiles;
      if (tid == E - 1) gemm_tile_off[E] = toff + tincl;
    }
  }
  p0 = p0 < 0 ? 0 : (p0 > cap ? cap : p0);
  p1 = p1 < p0 ? p0 : (p1 > cap ? cap : p1);
  __syncthreads();
  for (int p = p0 + tid; p < p1; p += 256) {
    const int v = pair_to_sorted[p];
    int e = pair_expert[p];
    e = e < 0 ? 0 : (e >= E ? E - 1 : e);
    int pos = s_base[e] + (v & 31);
    pos = pos < 0 ? 0 : (pos >= cap ? cap - 1 : pos);
    sorted_token[pos] = v >> 5;
    pair_to_sorted[p] = pos;
  }
}

}  // namespace

int launch_count_rule(const float* logits, int T, int E, int rule, float threshold, int k_min,
                      int k_max, int32_t* k_out, int32_t* pairs_out, hipStream_t s) {
  if (pairs_out != nullptr) {
    const int rc = launch_fill_i32(pairs_out, 0, 1, s);
    if (rc != REFLEX_OK) return rc;
  }
  hipLaunchKernelGGL(count_rule_kernel, dim3((T + TK_WAVES - 1) / TK_WAVES), dim3(TK_WAVES * kWave),
                     0, s, logits, T, E, rule, static_cast<double>(threshold), k_min, k_max, k_out,
                     pairs_out);
  return launch_status();
}

int launch_topk(const float* logits, const int32_t* k, int T, int E, int k_max, int norm_topk,
                const int32_t* pair_offsets, int32_t* pair_expert, float* pair_weight,
                hipStream_t s) {
  const dim3 grid((T + TK_WAVES - 1) / TK_WAVES), block(TK_WAVES * kWave);
  switch (topk_slots(E)) {
    case 1: hipLaunchKernelGGL(topk_kernel<1>, grid, block, 0, s, logits, k, T, E, k_max, norm_topk,
                               pair_offsets, pair_expert, pair_weight); break;
    case 2: hipLaunchKernelGGL(topk_kernel<2>, grid, block, 0, s, logits, k, T, E, k_max, norm_topk,
                               pair_offsets, pair_expert, pair_weight); break;
    case 3: hipLaunchKernelGGL(topk_kernel<3>, grid, block, 0, s, logits, k, T, E, k_max, norm_topk,
                               pair_offsets, pair_expert, pair_weight); break;
    default: hipLaunchKernelGGL(topk_kernel<4>, grid, block, 0, s, logits, k, T, E, k_max, norm_topk,
                                pair_offsets, pair_expert, pair_weight); break;
  }
  return launch_status();
}

bool route_fused_sorts(int T, int E) {
  return static_cast<long>((T + RF_WAVES - 1) / RF_WAVES) * E <= RF_HIST_MAX;
}

bool route_block_sorts(int T, int E) {
  const long n = static_cast<long>((T + RF_WAVES - 1) / RF_WAVES) * E;
  return n > RF_HIST_MAX && n <= BS_MAX_COUNTS;
}

size_t route_hist_bytes(int T, int E) {     // the counts, and the block sort's E totals
  return align_up((static_cast<size_t>((T + RF_WAVES - 1) / RF_WAVES) + 1) * E * sizeof(int32_t));
}

int launch_block_sort(const int32_t* pair_offsets, const int32_t* pair_expert, int T, int E,
                      int cap, int32_t* hist, int32_t* expert_offsets, int32_t* sorted_token,
                      int32_t* pair_to_sorted, int32_t* gemm_tile_off, hipStream_t s) {
  if (T <= 0) return REFLEX_OK;
  const int G = (T + RF_WAVES - 1) / RF_WAVES;
  int32_t* tot = hist + static_cast<size_t>(G) * E;
  hipLaunchKernelGGL(block_colscan_kernel, dim3(E), dim3(BS_THREADS), 0, s, hist, G, tot);
  hipLaunchKernelGGL(block_scatter_kernel, dim3(G), dim3(256), 0, s, pair_offsets, pair_expert, T,
                     cap, E, G, hist, tot, expert_offsets, gemm_tile_off, sorted_token,
                     pair_to_sorted);
  return launch_status();
}

int launch_route_fused(const float* logits, int n_parts, size_t part_stride, const float* bias,
                       float* logits_out, const int32_t* k, int T, int E, int k_max,
                       int norm_topk, int32_t* pair_offsets, int32_t* pair_expert,
                       float* pair_weight, int32_t* pairs_out, int32_t* done, int32_t* hist,
                       int32_t* expert_offsets, int32_t* sorted_token, int32_t* pair_to_sorted,
                       int32_t* gemm_tile_off, hipStream_t s) {
  const bool sort = done != nullptr;
  auto kernel = sort ? route_fused_kernel<4, true> : route_fused_kernel<4, false>;
  switch (topk_slots(E)) {
    case 1: kernel = sort ? route_fused_kernel<1, true> : route_fused_kernel<1, false>; break;
    case 2: kernel = sort ? route_fused_kernel<2, true> : route_fused_kernel<2, false>; break;
    case 3: kernel = sort ? route_fused_kernel<3, true> : route_fused_kernel<3, false>; break;
    default: break;
  }
  hipLaunchKernelGGL(kernel, dim3((T + RF_WAVES - 1) / RF_WAVES), dim3(RF_WAVES * kWave), 0, s, logits,
                     n_parts, part_stride, bias, logits_out, k, T, E, k_max, norm_topk, pair_offsets, pair_expert, pair_weight, pairs_out, done,
                     hist, expert_offsets, sorted_token, pair_to_sorted, gemm_tile_off);
  return launch_status();
}

static int perm_tiles(int cap) { return cap <= 0 ? 1 : (cap + PM_TILE - 1) / PM_TILE; }

size_t permute_ws_bytes(int pair_capacity, int E) {
  return align_up(static_cast<size_t>(perm_tiles(pair_capacity)) * E * sizeof(int32_t));
}

int launch_permute(const int32_t* pair_offsets, const int32_t* pair_expert, const int32_t* pairs,
                   int T, int E, int cap, int32_t* expert_offsets, int32_t* sorted_token,
                   int32_t* pair_to_sorted, void* ws, int32_t* gemm_tile_off, hipStream_t s) {
  if (cap <= PS_MAX_CAP) {
    hipLaunchKernelGGL(perm_small_kernel, dim3(1), dim3(PS_THREADS), 0, s, pair_offsets, pair_expert,
                       pairs, T, cap, E, expert_offsets, sorted_token, pair_to_sorted, gemm_tile_off);
    return launch_status();
  }
  const int n_tiles = perm_tiles(cap);
  int32_t* hist = static_cast<int32_t*>(ws);
  hipLaunchKernelGGL(perm_hist_kernel, dim3(n_tiles), dim3(PM_THREADS), 0, s, pair_expert, pairs,
                     cap, E, hist);
  hipLaunchKernelGGL(perm_scan_kernel, dim3(1), dim3(PM_SCAN_THREADS), 0, s, hist, n_tiles, E,
                     expert_offsets, gemm_tile_off);
  hipLaunchKernelGGL(perm_scatter_kernel, dim3(n_tiles), dim3(PM_THREADS), 0, s, pair_offsets,
                     pair_expert, pairs, T, cap, E, hist, sorted_token, pair_to_sorted);
  return launch_status();
}

}  // namespace rfx
