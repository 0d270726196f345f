// SwiGLU experts over expert-sorted rows on bf16 MFMA (gfx950).
//
// Expert e (Eq. (2)) is E_e(x) = W_down[e] (SiLU(W_gate[e] x) * (W_up[e] x)), the
// two input projections and one output projection counted in Appendix A.  Two
// grouped GEMMs do the work, both "NT" (both operands K-contiguous):
//   up:   act[j, :] = SiLU(x_j W_gate[e]^T) * (x_j W_up[e]^T),  x_j = h[sorted_token[j]]
//   down: y[j, :]   = act[j, :] W_down[e]^T
// Rows of one expert are contiguous after the permutation; a device-side plan
// (tile_off) cuts each expert's rows into 128-row M tiles, so no launch shape
// depends on the device-resident per-expert counts.
//
// Two kernels, chosen per launch from the pair capacity: 256-row tiles where the MFMAs
// bound the launch (below), and 128-row tiles where streaming the weights does:
// tile 128 (M) x GM_BROWS (256 weight rows) x 64 (K) on v_mfma_f32_32x32x16_bf16
// with fp32 accumulators: 4 compute waves in 2 x 2, each 64 x 128, plus 4 waves
// that only issue the global->LDS copies (one of each kind per SIMD), so a wave
// waiting for room in the memory queue never holds up the matrix cores.
// In the up GEMM the first half of the weight rows are gate rows and the second
// half the matching up rows, so gate and up of one output column meet in the same
// lane and register and SiLU(g) * u is formed before the single bf16 rounding of
// the activation.  A partial last N tile clamps its weight rows and skips the
// stores past N.
//
// Data movement: operands go from global memory straight into LDS with
// global_load_lds_dwordx4 (16 bytes per lane, no register staging) through a ring
// of GM_STAGES K-slices, so GM_STAGES-1 slices are in flight while one is multiplied.
// Rows are 128 bytes (8 chunks of 16 bytes) with chunk c of row r stored in slot
// c ^ ((r / 2) % 8).  The LDS has 64 four-byte banks and serves a 16-byte read
// for 16 lanes at a time, i.e. 16 rows of one fragment: their (row parity, slot)
// pairs are all distinct, so fragment reads are conflict-free, while a wave's DMA
// still writes 1 KB (8 whole rows) contiguously.
//
// Scheduling: a persistent grid (one workgroup per CU) walks a flattened
// sequence of (tile, K-slice) steps, so prefetching continues across tile
// boundaries.  Tiles are dealt to the 8 XCDs in contiguous runs (workgroup b
// runs on XCD b % 8), so one expert's tiles share that XCD's L2.  Within an
// expert the N tiles of one M tile are adjacent, so the workgroups of an XCD
// working at the same time share each gathered input slice and each weight slice.
#include <type_traits>

#include "common.h"

namespace rfx {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

#ifndef RFX_GEMM_BROWS
#define RFX_GEMM_BROWS 256
#endif
#ifndef RFX_GEMM_STAGES
#define RFX_GEMM_STAGES 3
#endif
#ifndef RFX_GEMM_BK
#define RFX_GEMM_BK 64
#endif
#ifndef RFX_GEMM_NINNER
#define RFX_GEMM_NINNER 1
#endif
constexpr int GM_BK = RFX_GEMM_BK;         // K per pipeline step: 64 or 32
constexpr int GM_BROWS = RFX_GEMM_BROWS;   // weight (B) rows per tile: 128 or 256
constexpr int GM_UP_BN = GM_BROWS / 2;     // activation columns per up-GEMM tile (gate + up rows)
constexpr int GM_DOWN_BN = GM_BROWS;       // output columns per down-GEMM tile
constexpr int GM_B_ELEMS = GM_BROWS * GM_BK;   // B slice
constexpr int GM_XCDS = 8;
#ifndef RFX_GEMM_CW
#define RFX_GEMM_CW 4
#endif
constexpr int GM_CW = RFX_GEMM_CW;         // compute waves: 2 (M) x GM_WN (N)
constexpr int GM_WN = GM_CW / 2;
constexpr int GM_NT = GM_BROWS / (32 * GM_WN);   // 32-wide B sub-tiles per compute wave
static_assert(GM_CW == 4 || GM_CW == 8, "compute waves");
// LDS rows are BK bf16 = CH chunks of 16 bytes; one DMA op (a wave, 64 lanes x 16
// bytes = 1 KB) fills ROWS_PER_OP whole rows.  Chunk c of row r sits in slot
// c ^ ((r / RG) % CH), RG = 16 / CH: the 16 rows one 16-lane group reads cover all
// 64 four-byte banks exactly once.
constexpr int GM_CH = GM_BK / 8;
constexpr int GM_ROWS_PER_OP = 64 / GM_CH;
constexpr int GM_RG = 16 / GM_CH;
constexpr int GM_BM = kGemmBM;
constexpr int GM_THREADS = 64 * (GM_CW + 4);   // compute waves + 4 loading waves
constexpr int GM_STAGES = RFX_GEMM_STAGES;
constexpr int GM_A_ELEMS = GM_BM * GM_BK;
constexpr int GM_STAGE_ELEMS = GM_A_ELEMS + GM_B_ELEMS;
constexpr int GM_A_OPS = GM_BM / GM_ROWS_PER_OP / 4;      // DMA ops per loading wave per step for A
constexpr int GM_B_OPS = GM_BROWS / GM_ROWS_PER_OP / 4;   // ... and for B
constexpr int GM_OPS = GM_A_OPS + GM_B_OPS;
constexpr size_t GM_LDS = size_t(GM_STAGES) * GM_STAGE_ELEMS * sizeof(uint16_t);
static_assert(GM_BK == 32 || GM_BK == 64, "BK");

struct Tile {
  int expert, row0, row_end, n0;
};

// Logical tile L -> tile.  Routed: experts in order, within an expert the M tile
// outer and the N tile inner (or the reverse when RFX_GEMM_NINNER is 0).  Dense:
// one expert over rows 0..dense_M-1.  tile_off and expert_offsets are the kernel's
// LDS copies; the expert is found in one round: every lane tests up to 4 experts
// and the wave counts those whose first tile lies at or before L (tile_off is
// nondecreasing, so that count minus one is the expert).  L is wave-uniform.
template <int BM, int BN>
__device__ __forceinline__ Tile decode_tile(int L, const int32_t* tile_off,
                                            const int32_t* expert_offsets, int E, int dense_M,
                                            int n_tiles, int out_rows) {
  Tile t;
  if (dense_M >= 0) {
    const int mt = (dense_M + BM - 1) / BM;
    t.expert = 0;
    t.n0 = (L / mt) * BN;
    t.row0 = (L % mt) * BM;
    t.row_end = dense_M;
    return t;
  }
  const int lane = threadIdx.x & 63;
  int cnt = 0;
#pragma unroll
  for (int q = 0; q < REFLEX_MAX_EXPERTS / 64; ++q) {
    const int e = lane + 64 * q;
    cnt += (e < E && tile_off[e] * n_tiles <= L) ? 1 : 0;
  }
  int lo = wave_sum_i32(cnt) - 1;
  lo = lo < 0 ? 0 : lo;
  const int local = L - tile_off[lo] * n_tiles;
  t.expert = lo;
#if RFX_GEMM_NINNER
  t.n0 = (local % n_tiles) * BN;
  t.row0 = expert_offsets[lo] + (local / n_tiles) * BM;
#else
  const int mt = tile_off[lo + 1] - tile_off[lo];
  t.n0 = (local / mt) * BN;
  t.row0 = expert_offsets[lo] + (local % mt) * BM;
#endif
  const int re = expert_offsets[lo + 1];
  t.row_end = re < out_rows ? re : out_rows;
  if (t.row0 < 0 || t.row0 >= t.row_end) t.row_end = t.row0;   // inconsistent offsets: no rows
  return t;
}

// s_waitcnt vmcnt(N) with expcnt and lgkmcnt left at their maxima (gfx9 encoding:
// vmcnt in bits [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8]).
template <int N>
__device__ __forceinline__ void waitcnt_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0f70);
}

// Each step issues OPS vector-memory ops per loading wave; let the ops of `pending`
// later steps stay outstanding.  Ops complete in issue order, so anything issued
// after them (epilogue stores) only makes the wait longer, never too short.
template <int OPS, int STAGES>
__device__ __forceinline__ void wait_steps(int pending) {
  static_assert(STAGES >= 2 && STAGES <= 6, "stage count");
  switch (pending) {
    case 0: waitcnt_vm<0>(); break;
    case 1: waitcnt_vm<(STAGES > 2 ? OPS : 0)>(); break;
    case 2: waitcnt_vm<(STAGES > 3 ? 2 * OPS : 0)>(); break;
    case 3: waitcnt_vm<(STAGES > 4 ? 3 * OPS : 0)>(); break;
    default: waitcnt_vm<(STAGES > 5 ? 4 * OPS : 0)>(); break;
  }
}

// Cache policy of the copies: sc0 (work-group scope).  Each copied line is read once
// per workgroup, so nothing is gained from keeping it in the CU's vector L1; measured
// 1-2 % less grouped-GEMM time on the tall-tile layers than the default policy (the
// non-temporal hint, which lets L2 drop the lines early, was 35-40 % slower: the
// weight lines it evicts are the ones the other M tiles of the expert read next).
constexpr int kDmaPolicy = 1;

// One wave's 1 KB copy: 16 bytes per lane from `src` straight into LDS at `dst`
// (the wave-uniform base; lane L lands at dst + 16 L bytes).  Kept out of line of
// the kernel's lambdas so that the host-side pass of the kernel stays valid.
__device__ __forceinline__ void lds_dma(const uint16_t* src, uint16_t* dst) {
  __builtin_amdgcn_global_load_lds(src, dst, 16, 0, kDmaPolicy);
}

// Workgroup barrier without the release/acquire fences of __syncthreads(): those
// would drain every outstanding vector-memory op (the in-flight LDS-DMA slices
// included) at each step.  The explicit vmcnt wait before it already makes this
// wave's DMA writes complete; lgkmcnt(0) makes this wave's earlier LDS reads
// complete before any wave refills the slice they read; the memory clobber keeps
// the compiler from moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Epilogue of one compute wave: its 64 x (32 NT) accumulator block (2 x NT MFMA
// tiles, weights as the A operand) to bf16 rows of `out`.  Lane l, register r holds
// output row l % 32 (a pair row) and column 8 (r/4) + 4 (l/32) + r%4 of its 32 x 32
// block.  Stored as it lies, one instruction would write 8 bytes to each of 32 rows;
// instead each 32 x 32 bf16 block goes through the wave's staging buffer in LDS and
// comes back with 4 lanes per row, so each store instruction writes 16 rows of 64
// contiguous bytes (a quarter of the write requests).  UP: sub-tiles j and j + NT/2
// hold gate and up of the same columns and the stored value is SiLU(g) u.  Rows at
// or past the tile's row_end are skipped; N is a multiple of 64, so a group of 8
// columns is wholly inside a partial last N tile or wholly past it.
//
// The staging accesses are inline assembly: the compiler cannot tell that the buffer
// does not alias the ring the direct-to-LDS copies write, and would wait for the next
// slice's copies (issued before the epilogue) before touching it.
constexpr int ST_LD = 40;                 // staging row pitch (elements): 80 B, 16 B aligned
constexpr int ST_ELEMS = 32 * ST_LD;      // one wave's staging buffer
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

template <bool UP, int NT>
__device__ __forceinline__ void store_wave_tile(const f32x16_t (&acc)[2][NT], const Tile& t,
                                                int row_in_tile, int col0, int N_out,
                                                uint16_t* __restrict__ out, uint16_t* stage) {
  const int lane = threadIdx.x & 63;
  // LDS byte offsets: a generic pointer to LDS carries the offset in its low 32 bits
  const uint32_t base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(stage));
  const uint32_t wr = base + ((lane & 31) * ST_LD + 4 * (lane >> 5)) * 2;
  const uint32_t rd = base + ((lane >> 2) * ST_LD + 8 * (lane & 3)) * 2;
  constexpr int NB = UP ? NT / 2 : NT;     // 32-column output blocks per 32 rows
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int rbase = t.row0 + row_in_tile + 32 * i + (lane >> 2);
#pragma unroll
    for (int jb = 0; jb < NB; ++jb) {
      u32x2_t v[4];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float a4[4];
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          if (UP) {     // SiLU(g) u = g u / (1 + e^-g), e^x = 2^(x log2 e)
            const float gg = acc[i][jb][4 * g + h], uu = acc[i][jb + NT / 2][4 * g + h];
            const float en = __builtin_amdgcn_exp2f(gg * -1.4426950408889634f);
            a4[h] = gg * __builtin_amdgcn_rcpf(1.0f + en) * uu;
          } else {
            a4[h] = acc[i][jb][4 * g + h];
          }
        }
        v[g] = u32x2_t{pack_bf16x2(a4[0], a4[1]), pack_bf16x2(a4[2], a4[3])};
      }
      u32x4_t r0, r1;
      // write the block (row l%32, columns 8g + 4(l/32) ..+3), read rows l/4 and
      // 16 + l/4 (columns 8 (l%4) ..+7); the wait ends the reads before the next
      // block overwrites the buffer
      asm volatile(
          "ds_write_b64 %2, %4\n\t"
          "ds_write_b64 %2, %5 offset:16\n\t"
          "ds_write_b64 %2, %6 offset:32\n\t"
          "ds_write_b64 %2, %7 offset:48\n\t"
          "ds_read_b128 %0, %3\n\t"
          "ds_read_b128 %1, %3 offset:1280\n\t"
          "s_waitcnt lgkmcnt(0)"
          : "=&v"(r0), "=&v"(r1)
          : "v"(wr), "v"(rd), "v"(v[0]), "v"(v[1]), "v"(v[2]), "v"(v[3])
          : "memory");
      const int col = t.n0 + col0 + 32 * jb + 8 * (lane & 3);
      if (col < N_out) {
        if (rbase < t.row_end)
          *reinterpret_cast<u32x4_t*>(out + static_cast<size_t>(rbase) * N_out + col) = r0;
        if (rbase + 16 < t.row_end)
          *reinterpret_cast<u32x4_t*>(out + static_cast<size_t>(rbase + 16) * N_out + col) = r1;
      }
    }
  }
}

static_assert(GM_LDS + 8 * (REFLEX_MAX_EXPERTS + 1) + GM_CW * ST_ELEMS * 2 <= 160 * 1024,
              "128-row ring + staging");

// One 32 x 32 output block of a wave: rows row_base + (0..31), columns col_base +
// (0..31); UP: SiLU(g) u from the gate and up accumulators.  Same lane layout and LDS
// staging as store_wave_tile (one store instruction writes 16 rows of 64 bytes).
template <bool UP>
__device__ __forceinline__ void store_block(const f32x16_t& g, const f32x16_t& u, int row_base,
                                            int col_base, int row_end, int N_out,
                                            uint16_t* __restrict__ out, uint16_t* stage) {
  const int lane = threadIdx.x & 63;
  const uint32_t base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(stage));
  const uint32_t wr = base + ((lane & 31) * ST_LD + 4 * (lane >> 5)) * 2;
  const uint32_t rd = base + ((lane >> 2) * ST_LD + 8 * (lane & 3)) * 2;
  u32x2_t v[4];
#pragma unroll
  for (int gi = 0; gi < 4; ++gi) {
    float a4[4];
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      if (UP) {
        const float gg = g[4 * gi + h], uu = u[4 * gi + h];
        const float en = __builtin_amdgcn_exp2f(gg * -1.4426950408889634f);
        a4[h] = gg * __builtin_amdgcn_rcpf(1.0f + en) * uu;
      } else {
        a4[h] = g[4 * gi + h];
      }
    }
    v[gi] = u32x2_t{pack_bf16x2(a4[0], a4[1]), pack_bf16x2(a4[2], a4[3])};
  }
  u32x4_t r0, r1;
  asm volatile(
      "ds_write_b64 %2, %4\n\t"
      "ds_write_b64 %2, %5 offset:16\n\t"
      "ds_write_b64 %2, %6 offset:32\n\t"
      "ds_write_b64 %2, %7 offset:48\n\t"
      "ds_read_b128 %0, %3\n\t"
      "ds_read_b128 %1, %3 offset:1280\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(r0), "=&v"(r1)
      : "v"(wr), "v"(rd), "v"(v[0]), "v"(v[1]), "v"(v[2]), "v"(v[3])
      : "memory");
  const int rbase = row_base + (lane >> 2);
  const int col = col_base + 8 * (lane & 3);
  if (col < N_out) {
    if (rbase < row_end) *reinterpret_cast<u32x4_t*>(out + static_cast<size_t>(rbase) * N_out + col) = r0;
    if (rbase + 16 < row_end)
      *reinterpret_cast<u32x4_t*>(out + static_cast<size_t>(rbase + 16) * N_out + col) = r1;
  }
}


// UP = true : act = SiLU(X Wg^T) * (X Wu^T);  UP = false: y = act Wd^T.
template <bool UP>
__global__ __launch_bounds__(GM_THREADS) void swiglu_gemm_kernel(
    const uint16_t* __restrict__ x,            // UP: h [T, K]; DOWN: act [rows, K]
    const int32_t* __restrict__ gather,        // UP: sorted_token or NULL (identity)
    const int32_t* __restrict__ tile_off, const int32_t* __restrict__ expert_offsets, int E,
    int dense_M, const uint16_t* __restrict__ w0,   // UP: W_gate; DOWN: W_down
    const uint16_t* __restrict__ w1,                // UP: W_up
    size_t w_expert_stride, int K, int N_out, int x_rows, int out_rows,
    uint16_t* __restrict__ out) {
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  constexpr int BN = UP ? GM_UP_BN : GM_DOWN_BN;
  const int n_tiles = (N_out + BN - 1) / BN;     // the last N tile may be partial
  // the tile plan and expert row offsets, copied to LDS once for the tile decodes
  __shared__ int s_tile_off[REFLEX_MAX_EXPERTS + 1], s_eo[REFLEX_MAX_EXPERTS + 1];
  __shared__ __attribute__((aligned(16))) uint16_t s_stage[GM_CW][ST_ELEMS];
  if (dense_M < 0) {
    for (int e = threadIdx.x; e <= E; e += blockDim.x) {
      s_tile_off[e] = tile_off[e];
      s_eo[e] = expert_offsets[e];
    }
    __syncthreads();
  }
  const int total = dense_M >= 0 ? ((dense_M + GM_BM - 1) / GM_BM) * n_tiles : s_tile_off[E] * n_tiles;

  // this workgroup's tiles: a contiguous run per XCD, strided over the XCD's workgroups
  const int xcd = blockIdx.x % GM_XCDS;
  const int per_xcd = gridDim.x / GM_XCDS;
  const int j0 = blockIdx.x / GM_XCDS;
  const int chunk = (total + GM_XCDS - 1) / GM_XCDS;
  const int l_begin = xcd * chunk + j0;
  const int l_end = min(total, (xcd + 1) * chunk);
  if (l_begin >= l_end) return;
  const int n_my = (l_end - l_begin + per_xcd - 1) / per_xcd;
  const int nk = K / GM_BK;
  const int n_steps = n_my * nk;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool producer = wave >= GM_CW;
  const int wv = producer ? wave - GM_CW : wave;   // index among the loading / computing waves
  const int wm = wv / GM_WN, wn = wv % GM_WN;

  if (producer) {
    // ---- loading waves: run GM_STAGES-1 steps ahead of the multiply ----
    // op q of a wave fills rows R0 = ROWS_PER_OP q' .. (q' the op's global row-group
    // index); lane L writes row r = R0 + L / CH, slot L % CH, which must hold
    // logical chunk c = (L % CH) ^ ((r / RG) % CH).
    auto lane_row = [&](int q) { return q * GM_ROWS_PER_OP + lane / GM_CH; };
    auto lane_chunk = [&](int q) {
      return ((lane % GM_CH) ^ ((lane_row(q) / GM_RG) % GM_CH)) * 8;
    };
    const uint16_t* a_ptr[GM_A_OPS];
    const uint16_t* b_ptr[GM_B_OPS];
    int ld_tile = -1;
    // K rotation of the tile being loaded, (2 m + n + 5 e) mod nk for M tile m of expert
    // e and N tile n (5 e in the up GEMM only): the tiles sharing an input-row slice
    // request it a step apart (as in the 256-row kernel below; 6 % less GEMM time on the
    // LLaDA-MoE layer, measured), and the tiles of different experts that stream weights
    // at the same time start at different K slices.  With a weight row of 4 KB (d = 2048)
    // and one M tile per expert, n alone gives the 256 concurrent tiles 8 distinct 128-byte
    // offsets within their rows; spread over all 32, the LLaDA-MoE up GEMM took 103
    // against 125 us (traced in one process, the same in three separate runs; the down
    // GEMM, whose 2 KB rows already spread, was 1-2 % slower with it, 10 % slower with 8 e).
    int ld_rot = 0;
    auto setup_loader = [&](int tile_i) {
      const Tile t = decode_tile<GM_BM, BN>(l_begin + tile_i * per_xcd, s_tile_off, s_eo, E, dense_M,
                                     n_tiles, out_rows);
      const int rows_valid = t.row_end - t.row0;
      ld_rot = (2 * ((t.row0 - (dense_M >= 0 ? 0 : s_eo[t.expert])) / GM_BM) + t.n0 / BN +
                (UP ? 5 * t.expert : 0)) % nk;
#pragma unroll
      for (int j = 0; j < GM_A_OPS; ++j) {
        const int r = lane_row(GM_A_OPS * wv + j);
        int src = t.row0 + (r < rows_valid ? r : 0);     // rows past the expert reuse row0
        if (rows_valid <= 0) src = 0;
        if (UP && gather != nullptr) {
          src = gather[src];
          src = src < 0 ? 0 : (src >= x_rows ? x_rows - 1 : src);
        }
        a_ptr[j] = x + static_cast<size_t>(src) * K + lane_chunk(GM_A_OPS * wv + j);
      }
#pragma unroll
      for (int j = 0; j < GM_B_OPS; ++j) {
        const int r = lane_row(GM_B_OPS * wv + j);
        const uint16_t* wb;
        int wr;
        if (UP) {     // rows [0, BROWS/2): gate rows n0 + r; the rest: up rows n0 + r - BROWS/2
          wb = (r < GM_BROWS / 2 ? w0 : w1) + t.expert * w_expert_stride;
          wr = t.n0 + (r < GM_BROWS / 2 ? r : r - GM_BROWS / 2);
        } else {
          wb = w0 + t.expert * w_expert_stride;
          wr = t.n0 + r;
        }
        wr = wr < N_out ? wr : N_out - 1;     // partial last N tile: columns past N are not stored
        b_ptr[j] = wb + static_cast<size_t>(wr) * K + lane_chunk(GM_B_OPS * wv + j);
      }
    };
    auto issue = [&](int step) {
      const int tile_i = step / nk, kt = step - tile_i * nk;
      if (tile_i != ld_tile) {
        setup_loader(tile_i);
        ld_tile = tile_i;
      }
      uint16_t* As = smem + (step % GM_STAGES) * GM_STAGE_ELEMS;
      uint16_t* Bs = As + GM_A_ELEMS;
      int kr = kt + ld_rot;
      kr = kr >= nk ? kr - nk : kr;
      const int k0 = kr * GM_BK;
#pragma unroll
      for (int j = 0; j < GM_A_OPS; ++j) lds_dma(a_ptr[j] + k0, As + (GM_A_OPS * wv + j) * 512);
#pragma unroll
      for (int j = 0; j < GM_B_OPS; ++j) lds_dma(b_ptr[j] + k0, Bs + (GM_B_OPS * wv + j) * 512);
    };
    for (int s = 0; s < GM_STAGES - 1 && s < n_steps; ++s) issue(s);
    for (int s = 0; s < n_steps; ++s) {
      wait_steps<GM_OPS, GM_STAGES>(min(GM_STAGES - 2, n_steps - 1 - s));
      lds_barrier();       // slice s visible to all waves; slice s-1 no longer read
      if (s + GM_STAGES - 1 < n_steps) issue(s + GM_STAGES - 1);
    }
    return;
  }

  // ---- compute waves ----
  // B sub-tiles of this wave (32 rows each).  UP: the first GM_NT/2 are gate rows
  // wn*BROWS/4 + 32j, the rest the matching up rows (+ BROWS/2), so sub-tile j and
  // j + GM_NT/2 hold gate and up of the same output columns.  DOWN: wn*BROWS/2 + 32j.
  int b_row[GM_NT];
#pragma unroll
  for (int j = 0; j < GM_NT; ++j)
    b_row[j] = UP ? (j < GM_NT / 2 ? wn * (GM_BROWS / 2 / GM_WN) + 32 * j
                                   : GM_BROWS / 2 + wn * (GM_BROWS / 2 / GM_WN) + 32 * (j - GM_NT / 2))
                  : wn * (GM_BROWS / GM_WN) + 32 * j;
  const int a_row[2] = {wm * 64, wm * 64 + 32};
  // fragment rows are 32-aligned bases + (lane % 32): (row / RG) % CH from lane % 32
  const int frow = lane & 31, fsel = lane >> 5, fx = (frow / GM_RG) % GM_CH;
  f32x16_t acc[2][GM_NT];
  int s = 0;        // flattened step over (tile, K slice), in step with the loading waves
  for (int tile_i = 0; tile_i < n_my; ++tile_i) {
    // a wave's second 32-row block past the expert's last row is skipped: fewer
    // MFMAs, and less power drawn, on the partly filled tiles of experts with few rows
    const Tile tt = decode_tile<GM_BM, BN>(l_begin + tile_i * per_xcd, s_tile_off, s_eo, E, dense_M,
                                           n_tiles, out_rows);
    const bool blk1 = tt.row0 + wm * 64 + 32 < tt.row_end;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < GM_NT; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
    for (int kt = 0; kt < nk; ++kt, ++s) {
      lds_barrier();       // slice s visible to all waves; slice s-1 no longer read
      const uint16_t* As = smem + (s % GM_STAGES) * GM_STAGE_ELEMS;
      const uint16_t* Bs = As + GM_A_ELEMS;
      // 16-wide K sub-steps; the fragments of sub-step kk+1 are read from LDS into
      // the other register set before the MFMAs of kk are issued, so the LDS latency
      // hides behind them (only the first read after the barrier is exposed)
      bf16x8_t af[2][2], bfr[2][GM_NT];
      auto load = [&](int kk, int buf) {
        const int slot = ((2 * kk + fsel) ^ fx) * 8;
#pragma unroll
        for (int i = 0; i < 2; ++i)
          af[buf][i] = *reinterpret_cast<const bf16x8_t*>(As + (a_row[i] + frow) * GM_BK + slot);
#pragma unroll
        for (int j = 0; j < GM_NT; ++j)
          bfr[buf][j] = *reinterpret_cast<const bf16x8_t*>(Bs + (b_row[j] + frow) * GM_BK + slot);
      };
      // (the instruction scheduler is told the order: reads of kk+1, then MFMAs of kk)
      constexpr int kReads = 2 + GM_NT;
      load(0, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);      // LDS reads
#pragma unroll
      for (int kk = 0; kk < GM_BK / 16; ++kk) {
        if (kk + 1 < GM_BK / 16) {
          load(kk + 1, (kk + 1) & 1);
          __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);
        }
        // weights as the MFMA's A operand: the accumulator is the transposed tile,
        // so each lane ends up holding 4 consecutive output columns of one row
        if (blk1) {
#pragma unroll
          for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < GM_NT; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[kk & 1][j], af[kk & 1][i],
                                                                  acc[i][j], 0, 0, 0);
        } else {
#pragma unroll
          for (int j = 0; j < GM_NT; ++j)
            acc[0][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[kk & 1][j], af[kk & 1][0],
                                                                acc[0][j], 0, 0, 0);
        }
      }
    }
    const Tile t = decode_tile<GM_BM, BN>(l_begin + tile_i * per_xcd, s_tile_off, s_eo, E, dense_M,
                                          n_tiles, out_rows);
    store_wave_tile<UP, GM_NT>(acc, t, wm * 64,
                               UP ? wn * (GM_BROWS / 2 / GM_WN) : wn * (GM_BROWS / GM_WN), N_out, out,
                               s_stage[wv]);
  }
}

// ---- tall tiles: 256 rows x 256 weight rows, 8 waves that all load and multiply ----
//
// For experts with many rows the MFMAs, not the weight stream, are the bound.  Two
// waves share each SIMD.  The waves form 2 (pair rows) x 4 (weight rows): wave
// (wm, wn) multiplies pair rows 128 wm .. 128 wm + 127 (four 32-row blocks) by 64
// weight rows (UP: the 32 gate rows and the 32 matching up rows of activation columns
// n0 + 32 wn ..; DOWN: weight rows 64 wn ..).  Waves w and w + 4 share a SIMD, so each
// SIMD holds one wave of each row half: an expert's last tile, whose rows end early,
// shortens the MFMA stream of all four SIMDs alike (row blocks past the expert's end
// are skipped), instead of idling some SIMDs while the others run a full tile.  The K
// loop is instantiated per count of active row blocks, so the common full tile runs
// straight-line code with no per-block branches.  Every wave issues its share of the
// global->LDS copies of the next input-row slice and of the weight slice two steps
// ahead into the ring slots the previous step has just released, one copy between
// every two MFMAs of the first two K sub-steps: issued all at once after the barrier,
// the 64 copies of a step queue up in the texture path and stall both waves of each
// SIMD until they drain.  The M tile is 256 rows, so per expert the tiles are
// ceil(n_e / 256), counted at start.
#ifndef RFX_TALL_MIN_ROWS
#define RFX_TALL_MIN_ROWS 512
#endif
constexpr int TL_BM = 2 * kGemmBM;
constexpr int TL_BK = 64;
constexpr int TL_WAVES = 8;
constexpr int TL_THREADS = 64 * TL_WAVES;
constexpr int TL_MI = 4;                         // 32-row pair blocks per wave
constexpr int TL_NJ = 2;                         // 32-row weight blocks per wave
constexpr int TL_CH = TL_BK / 8;
constexpr int TL_ROWS_PER_OP = 64 / TL_CH;
constexpr int TL_RG = 16 / TL_CH;
constexpr int TL_A_ELEMS = TL_BM * TL_BK;        // one input-row slice (32 KB)
constexpr int TL_B_ELEMS = GM_BROWS * TL_BK;     // one weight slice (32 KB)
constexpr int TL_A_SLOTS = 2;                    // input rows: one slice ahead
constexpr int TL_B_SLOTS = 3;                    // weights: two slices ahead
constexpr int TL_A_OPS = TL_BM / TL_ROWS_PER_OP / TL_WAVES;   // DMA ops per wave per step
constexpr int TL_B_OPS = GM_BROWS / TL_ROWS_PER_OP / TL_WAVES;
constexpr size_t TL_LDS =
    size_t(TL_A_SLOTS * TL_A_ELEMS + TL_B_SLOTS * TL_B_ELEMS) * sizeof(uint16_t);
static_assert(GM_BROWS == 256, "tall tiles: four wave columns of 64 weight rows");
static_assert(TL_A_OPS == 4 && TL_B_OPS == 4, "copy interleave: four of each per wave and step");
static_assert(TL_LDS <= 160 * 1024, "tall LDS rings");
static_assert(TL_WAVES * ST_ELEMS <= TL_A_ELEMS, "the epilogue staging fits in an input-row slot");
static_assert(3 * (REFLEX_MAX_EXPERTS + 1) * 4 <= TL_A_ELEMS * 2, "start-up scratch in the ring");
#if !RFX_GEMM_NINNER
#error "the 256-row kernel decodes tiles with the N tile inner"
#endif

template <bool UP>
__global__ __launch_bounds__(TL_THREADS) void swiglu_gemm_tall_kernel(
    const uint16_t* __restrict__ x, const int32_t* __restrict__ gather,
    const int32_t* __restrict__ expert_offsets, int E, const uint16_t* __restrict__ w0,
    const uint16_t* __restrict__ w1, size_t w_expert_stride, int K, int N_out, int x_rows,
    int out_rows, uint16_t* __restrict__ out) {
  // The whole 160 KB of LDS holds the two rings: input-row slices in slots 0-1, weight
  // slices in the three slots after them.  The weight lines mostly come from HBM (the
  // input rows mostly hit in L2), so they are copied two K steps ahead and the copies of
  // the next weight slice stay in flight across each step's barrier.  The tile tables
  // live in registers, and the epilogue stages its stores in the input-row slot the
  // tile's last K step has read.
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  uint16_t* const a_ring = smem;
  uint16_t* const b_ring = smem + TL_A_SLOTS * TL_A_ELEMS;
  constexpr int BN = UP ? GM_UP_BN : GM_DOWN_BN;
  const int n_tiles = (N_out + BN - 1) / BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // ---- expert row offsets and the per-expert prefix of 256-row tiles, computed in LDS
  // (scratch: the rings are empty until the first copies) and kept in registers: lane l
  // holds the entries of experts l, l + 64, l + 128, l + 192
  int toff_r[4], eo_r[4], eo_E, m_total;
  {
    int* s_eo = reinterpret_cast<int*>(smem);
    int* s_toff = s_eo + (REFLEX_MAX_EXPERTS + 1);
    int* s_part = s_toff + (REFLEX_MAX_EXPERTS + 1);
    for (int e = tid; e <= E; e += TL_THREADS) s_eo[e] = expert_offsets[e];
    __syncthreads();
    int n = 0;
    if (tid < E) {
      n = s_eo[tid + 1] - s_eo[tid];
      n = n < 0 ? 0 : (n + TL_BM - 1) / TL_BM;
    }
    const int incl = wave_inclusive_scan_i32(n, lane);
    if (lane == 63) s_part[wave] = incl;
    __syncthreads();
    int base = incl - n;
    for (int q = 0; q < wave; ++q) base += s_part[q];
    if (tid <= E) s_toff[tid] = base;       // tid == E: the total
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = lane + 64 * q;
      toff_r[q] = e < E ? s_toff[e] : 0;
      eo_r[q] = e < E ? s_eo[e] : 0;
    }
    eo_E = __builtin_amdgcn_readfirstlane(s_eo[E]);
    m_total = __builtin_amdgcn_readfirstlane(s_toff[E]);
    __syncthreads();     // all scratch reads done before the first copies land
  }
  // entry e (< 256) of a per-lane table, uniform e
  auto table_at = [&](const int (&r)[4], int e) {
    const int q = e >> 6;
    const int v = q == 0 ? r[0] : (q == 1 ? r[1] : (q == 2 ? r[2] : r[3]));
    return __builtin_amdgcn_readlane(v, e & 63);
  };
  // Logical tile L -> tile: experts in order, the M tile outer and the N tile inner; the
  // expert is found in one round (the wave counts the experts whose first tile lies at or
  // before L).  rot: the tile's K rotation (below).
  struct TT {
    int expert, row0, row_end, n0, rot;
  };
  const int nk = K / TL_BK;
  auto decode = [&](int L) {
    TT t;
    int cnt = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) cnt += (lane + 64 * q < E && toff_r[q] * n_tiles <= L) ? 1 : 0;
    int lo = wave_sum_i32(cnt) - 1;
    lo = __builtin_amdgcn_readfirstlane(lo < 0 ? 0 : lo);
    const int local = L - table_at(toff_r, lo) * n_tiles;
    const int er0 = table_at(eo_r, lo);
    const int er1 = lo + 1 < E ? table_at(eo_r, lo + 1) : eo_E;
    t.expert = lo;
    t.n0 = (local % n_tiles) * BN;
    const int m = local / n_tiles;
    t.row0 = er0 + m * TL_BM;
    t.row_end = er1 < out_rows ? er1 : out_rows;
    if (t.row0 < 0 || t.row0 >= t.row_end) t.row_end = t.row0;   // inconsistent offsets: no rows
    // K rotation: tile (M tile m of its expert, N tile n) walks its K slices starting at
    // slice n mod nk (down) or (n mod 2) mod nk (up).  The tiles sharing an input-row slice
    // (same m) then request it a step apart instead of all at once (5 % less GEMM time on
    // the 16-layer stack, 3 % on the skewed layer, against no rotation), while the M tiles
    // sharing a weight slice (same n) read it in the same step, so it comes from HBM once
    // for all of them (1 % less time than a rotation of 2 m + n, which spread them two
    // steps apart).  In the up GEMM the 8 N tiles sharing a gathered-row slice stay within
    // two steps, so fewer of its lines leave L2 before the last of them reads it (1 % less
    // up-GEMM time than n mod nk; the same in the down GEMM made it 2-4 % slower).  All
    // traced in one process.  Only the order of the fp32 sums over K changes.
    t.rot = (UP ? (t.n0 / BN) % 2 : t.n0 / BN) % nk;
    return t;
  };
  const int total = m_total * n_tiles;
  const int xcd = blockIdx.x % GM_XCDS;
  const int per_xcd = gridDim.x / GM_XCDS;
  const int j0 = blockIdx.x / GM_XCDS;
  const int chunk = (total + GM_XCDS - 1) / GM_XCDS;
  const int l_begin = xcd * chunk + j0;
  const int l_end = min(total, (xcd + 1) * chunk);
  if (l_begin >= l_end) return;
  const int n_my = (l_end - l_begin + per_xcd - 1) / per_xcd;
  const int wm = wave >> 2, wn = wave & 3;

  // ---- copies: op q of the step fills rows ROWS_PER_OP q ..; lane L writes row
  // r = ROWS_PER_OP q + L / CH at slot L % CH, holding chunk (L % CH) ^ ((r / RG) % CH)
  auto lane_row = [&](int q) { return q * TL_ROWS_PER_OP + lane / TL_CH; };
  auto lane_chunk = [&](int q) { return ((lane % TL_CH) ^ ((lane_row(q) / TL_RG) % TL_CH)) * 8; };
  constexpr int CP_OPS = TL_A_OPS;     // copies of each operand per wave and step
  // The copies are buffer loads into LDS.  Input rows go through a resource of the
  // operand's size, and a copy that is skipped (wholly past the expert's last row) gets
  // an offset past that size, which the hardware's range check turns into no memory
  // access, so the step has no branch: a branch splits the step into several basic
  // blocks, and the instruction order pinned below then holds only within each (16-layer
  // stack and skewed layer: 2-3 % less GEMM time than a branch around each copy,
  // identical output; traced in one process).  Weight rows go through a resource of the
  // wave's 32 rows of the tile: with global_load_lds copies the compiler made each
  // sub-step's MFMAs wait for all of the step's LDS reads, not only their own (2-3 %
  // less GEMM time with the buffer form).  Copy sources are 32-bit element offsets (the
  // host keeps the tall kernel to input operands of fewer than 2^30 elements).
  //
  // Input-row loader: its tile and K slice, rotation, the copies that hold rows of its
  // tile, and copy j's offset into x.
  int a_tile = 0, a_k = 0, a_rot = 0, a_ops = CP_OPS;
  uint32_t a_off[CP_OPS];
  auto setup_a = [&](int tile_i) {
    const TT t = decode(l_begin + tile_i * per_xcd);
    const int rows_valid = t.row_end - t.row0;
    // Input-row copy q holds rows ROWS_PER_OP q ..; copies wholly past the expert's last
    // row are not issued.  The multiply reads whole 32-row blocks, but only up to the
    // block holding the last row, and every copy with a row of that block is issued, so
    // no row it reads is skipped (16-layer stack and skewed layer: 1-2 % less GEMM time,
    // identical output; traced in one process).
    int n = (rows_valid + TL_ROWS_PER_OP - 1) / TL_ROWS_PER_OP - CP_OPS * wave;
    n = n < 0 ? 0 : (n > CP_OPS ? CP_OPS : n);
    a_ops = __builtin_amdgcn_readfirstlane(n);
    a_rot = t.rot;
#pragma unroll
    for (int j = 0; j < CP_OPS; ++j) {
      const int r = lane_row(CP_OPS * wave + j);
      int src = t.row0 + (r < rows_valid ? r : 0);     // rows past the expert reuse row0
      if (rows_valid <= 0) src = 0;
      if (UP && gather != nullptr) {
        src = gather[src];
        src = src < 0 ? 0 : (src >= x_rows ? x_rows - 1 : src);
      }
      a_off[j] = static_cast<uint32_t>(src) * static_cast<uint32_t>(K) +
                 static_cast<uint32_t>(lane_chunk(CP_OPS * wave + j));
    }
  };
  // Weight loader: its tile and K slice, rotation, and the address of the wave's 32
  // weight rows: tile rows 32 wave .. (UP: 32 (wave % 4) .. of the gate (waves 0-3) or up
  // (waves 4-7) rows).  N is a multiple of 64 and the rows start at a multiple of 32, so
  // in a partial last N tile they are all valid or all past N; past N they are replaced
  // by the last 32 rows (the columns past N are not stored).  Copies j and j + 2 are 16
  // rows apart and share the chunk swizzle: copy j reads 16 K (j / 2) + b_off[j % 2].
  int b_tile = 0, b_k = 0, b_rot = 0;
  uint32_t b_lo = 0, b_hi = 0;
  uint32_t b_off[2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
    b_off[j] = static_cast<uint32_t>(lane_row(j) * K) +
               static_cast<uint32_t>(lane_chunk(CP_OPS * wave + j));
  auto setup_b = [&](int tile_i) {
    const TT t = decode(l_begin + tile_i * per_xcd);
    b_rot = t.rot;
    int wr0 = t.n0 + 32 * (UP ? (wave & 3) : wave);
    wr0 = wr0 + 32 <= N_out ? wr0 : N_out - 32;
    const uint16_t* wm_base = (UP && wave >= 4 ? w1 : w0) + t.expert * w_expert_stride;
    const uint64_t b_addr = reinterpret_cast<uint64_t>(wm_base + static_cast<size_t>(wr0) * K);
    b_lo = static_cast<uint32_t>(b_addr);
    b_hi = static_cast<uint32_t>(b_addr >> 32);
  };
  // The K offset of a loader's next slice; then it advances (past the workgroup's last
  // tile it stays on its last slice, so the issue never branches and every source
  // address stays in bounds).
  auto a_next = [&]() {
    if (a_k == nk) {
      if (a_tile + 1 < n_my) {
        ++a_tile;
        a_k = 0;
        setup_a(a_tile);
      } else {
        a_k = nk - 1;
      }
    }
    int kr = a_k + a_rot;
    kr = kr >= nk ? kr - nk : kr;
    ++a_k;
    return kr * TL_BK;
  };
  auto b_next = [&]() {
    if (b_k == nk) {
      if (b_tile + 1 < n_my) {
        ++b_tile;
        b_k = 0;
        setup_b(b_tile);
      } else {
        b_k = nk - 1;
      }
    }
    int kr = b_k + b_rot;
    kr = kr >= nk ? kr - nk : kr;
    ++b_k;
    return kr * TL_BK;
  };
  const __amdgpu_buffer_rsrc_t x_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(x), static_cast<short>(0),
      static_cast<int>(static_cast<uint32_t>(x_rows) * static_cast<uint32_t>(K) * 2u), 0x00020000);
  auto dma_a = [&](int j, uint16_t* As_, int k0_) {
    const uint32_t voff = j < a_ops ? (a_off[j] + static_cast<uint32_t>(k0_)) * 2u : 0x80000000u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        x_rsrc, (__attribute__((address_space(3))) void*)(As_ + (CP_OPS * wave + j) * 512), 16,
        voff, 0, 0, kDmaPolicy);
  };
  auto dma_b = [&](int j, uint16_t* Bs_, int k0_) {
    // the resource is rebuilt from wave-uniform halves at each use, so that it always
    // lives in scalar registers (held across the loop it could end up in vector
    // registers, and each copy would then become a loop over the distinct values)
    const uint64_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b_lo)));
    const uint64_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b_hi)));
    const __amdgpu_buffer_rsrc_t b_rsrc = __builtin_amdgcn_make_buffer_rsrc(
        reinterpret_cast<void*>(lo | (hi << 32)), static_cast<short>(0), 64 * K, 0x00020000);
    const uint32_t voff = (b_off[j % 2] + static_cast<uint32_t>(k0_ + 16 * (j / 2) * K)) * 2u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        b_rsrc, (__attribute__((address_space(3))) void*)(Bs_ + (CP_OPS * wave + j) * 512), 16,
        voff, 0, 0, kDmaPolicy);
  };
  // ---- multiply: pair blocks 128 wm + 32 i, weight blocks b_row[j]
  const int b_row[TL_NJ] = {UP ? 32 * wn : 64 * wn, UP ? GM_BROWS / 2 + 32 * wn : 64 * wn + 32};
  const int frow = lane & 31, fsel = lane >> 5, fx = (frow / TL_RG) % TL_CH;
  f32x16_t acc[TL_MI][TL_NJ];
  // prologue: input-row slice 0 and weight slices 0 and 1
  setup_a(0);
  setup_b(0);
  {
    const int ka = a_next();
#pragma unroll
    for (int j = 0; j < CP_OPS; ++j) dma_a(j, a_ring, ka);
#pragma unroll
    for (int q = 0; q < TL_B_SLOTS - 1; ++q) {
      const int kb = b_next();
#pragma unroll
      for (int j = 0; j < CP_OPS; ++j) dma_b(j, b_ring + q * TL_B_ELEMS, kb);
    }
  }
  int s = 0;     // K steps so far (the rings' slot counter)
  // The K loop of one tile with NB active pair blocks (0: this wave only copies).  The
  // MFMAs of each slice's last 16-wide sub-step run after the next step's barrier, from
  // fragments read before it, so they overlap the LDS reads of the next slice's first
  // sub-step instead of every SIMD waiting for those reads after each barrier (16-layer
  // stack and skewed layer: 3-4 % less GEMM time, identical output; traced in one
  // process).  The fragments stay in the second register buffer across the barrier.
  auto k_loop = [&](auto nb_c) {
    constexpr int NB = decltype(nb_c)::value;
    constexpr int kReads = NB + TL_NJ, kMfmas = NB * TL_NJ;
    constexpr int kPer = kMfmas / CP_OPS > 0 ? kMfmas / CP_OPS : 1;
    bf16x8_t af[2][TL_MI], bfr[2][TL_NJ];
    // weights as the MFMA's A operand: the accumulator is the transposed tile, so each
    // lane ends up holding 4 consecutive output columns of one row
    auto mfmas = [&](int buf) {
#pragma unroll
      for (int i = 0; i < NB; ++i)
#pragma unroll
        for (int j = 0; j < TL_NJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[buf][j], af[buf][i], acc[i][j],
                                                              0, 0, 0);
    };
    // a copy after every kPer MFMAs: the copies drain at the rate the texture path takes
    // them while the matrix cores keep busy
    auto interleave_copies = [&]() {
#pragma unroll
      for (int q = 0; q < CP_OPS; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, kPer, 0);
        __builtin_amdgcn_sched_group_barrier(0x010, 1, 0);
      }
    };
    // One K step.  FIRST: the tile's first, with no deferred MFMAs of a previous slice;
    // it follows the previous tile's output stores, which need not complete in order with
    // the copies, so it waits for all of its wave's ops.
    auto step = [&](auto first_c) {
      constexpr bool FIRST = decltype(first_c)::value;
      const int ka = a_next();
      const int kb = b_next();
      // Input-row slice s and weight slice s have landed (issued one and two steps ago;
      // the ops issued after them are the next weight slice's) and are visible to all
      // waves; the slots of the slices the previous step read are free.
      if constexpr (FIRST)
        waitcnt_vm<0>();
      else
        waitcnt_vm<TL_B_OPS>();
      lds_barrier();
      // Raised issue priority from the barrier through the deferred MFMAs and the first
      // copies: the SIMD's two waves leave the barrier together, and the one served first
      // gets its MFMAs going while the other's LDS reads are in flight (16-layer stack:
      // 1.1 / 1.5 % less up / down GEMM time, skewed layer 0.2 / 0.5 %; traced in one
      // process.  Raised around every MFMA group instead: 1.3 % slower).
      __builtin_amdgcn_s_setprio(1);
      uint16_t* An = a_ring + ((s + 1) % TL_A_SLOTS) * TL_A_ELEMS;
      uint16_t* Bn = b_ring + ((s + TL_B_SLOTS - 1) % TL_B_SLOTS) * TL_B_ELEMS;
      if constexpr (NB == 0) {
#pragma unroll
        for (int j = 0; j < CP_OPS; ++j) dma_a(j, An, ka);
#pragma unroll
        for (int j = 0; j < CP_OPS; ++j) dma_b(j, Bn, kb);
        __builtin_amdgcn_s_setprio(0);
      } else {
        const uint16_t* As = a_ring + (s % TL_A_SLOTS) * TL_A_ELEMS;
        const uint16_t* Bs = b_ring + (s % TL_B_SLOTS) * TL_B_ELEMS;
        auto load = [&](int kk, int buf) {
          const int slot = ((2 * kk + fsel) ^ fx) * 8;
#pragma unroll
          for (int i = 0; i < NB; ++i)
            af[buf][i] =
                *reinterpret_cast<const bf16x8_t*>(As + (128 * wm + 32 * i + frow) * TL_BK + slot);
#pragma unroll
          for (int j = 0; j < TL_NJ; ++j)
            bfr[buf][j] = *reinterpret_cast<const bf16x8_t*>(Bs + (b_row[j] + frow) * TL_BK + slot);
        };
        // (the instruction scheduler is told the order: reads of kk+1, then MFMAs of kk)
        load(0, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);
        if constexpr (!FIRST) {
          mfmas(1);     // the previous slice's last sub-step
#pragma unroll
          for (int j = 0; j < CP_OPS; ++j) dma_a(j, An, ka);
          interleave_copies();
        }
        __builtin_amdgcn_s_setprio(0);
#pragma unroll
        for (int kk = 0; kk < TL_BK / 16 - 1; ++kk) {
          load(kk + 1, (kk + 1) & 1);
          __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);
          mfmas(kk & 1);
          if (FIRST ? kk == 0 : false) {
#pragma unroll
            for (int j = 0; j < CP_OPS; ++j) dma_a(j, An, ka);
          }
          if (FIRST ? kk == 1 : kk == 0) {
#pragma unroll
            for (int j = 0; j < CP_OPS; ++j) dma_b(j, Bn, kb);
          }
          if (FIRST ? kk < 2 : kk < 1)
            interleave_copies();
          else
            __builtin_amdgcn_sched_group_barrier(0x008, kMfmas, 0);
        }
      }
    };
    step(std::true_type{});
    ++s;
    for (int kt = 1; kt < nk; ++kt, ++s) step(std::false_type{});
    if constexpr (NB > 0) mfmas(1);     // the last slice's last sub-step
  };
  for (int tile_i = 0; tile_i < n_my; ++tile_i) {
    const TT t = decode(l_begin + tile_i * per_xcd);
    // pair blocks of this wave's 128 rows that hold pairs (wave-uniform)
    int rows = t.row_end - t.row0 - 128 * wm;
    rows = rows < 0 ? 0 : (rows > 128 ? 128 : rows);
    const int nb = __builtin_amdgcn_readfirstlane((rows + 31) >> 5);
#pragma unroll
    for (int i = 0; i < TL_MI; ++i)
#pragma unroll
      for (int j = 0; j < TL_NJ; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
    switch (nb) {
      case 4: k_loop(std::integral_constant<int, 4>{}); break;
      case 3: k_loop(std::integral_constant<int, 3>{}); break;
      case 2: k_loop(std::integral_constant<int, 2>{}); break;
      case 1: k_loop(std::integral_constant<int, 1>{}); break;
      default: k_loop(std::integral_constant<int, 0>{}); break;
    }
    // every wave has read the tile's last input-row slice: its slot takes the staging
    // (the next tile's first step refills it only after its own barrier)
    lds_barrier();
    uint16_t* stage = a_ring + ((s + 1) % TL_A_SLOTS) * TL_A_ELEMS + wave * ST_ELEMS;
#pragma unroll
    for (int i = 0; i < TL_MI; ++i) {
      if (i < nb) {
        const int rb = t.row0 + 128 * wm + 32 * i;
        if (UP) {
          store_block<true>(acc[i][0], acc[i][1], rb, t.n0 + 32 * wn, t.row_end, N_out, out, stage);
        } else {
#pragma unroll
          for (int j = 0; j < TL_NJ; ++j)
            store_block<false>(acc[i][j], acc[i][j], rb, t.n0 + 64 * wn + 32 * j, t.row_end, N_out,
                               out, stage);
        }
      }
    }
  }
  waitcnt_vm<0>();     // the last (unused) copies land before the workgroup's LDS is released
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

// One persistent workgroup per CU (the LDS ring admits one per CU), rounded up to
// a multiple of the XCD count.
int persistent_grid() {
  const int cus = device_cus();
  return (cus + GM_XCDS - 1) / GM_XCDS * GM_XCDS;
}

template <bool UP>
int launch_gemm(const uint16_t* x, const int32_t* gather, const int32_t* tile_off,
                const int32_t* eo, int E, int dense_M, const uint16_t* w0, const uint16_t* w1,
                size_t stride, int K, int N, int x_rows, int out_rows, uint16_t* out, hipStream_t s) {
  static bool attr_set = false;
  if (!attr_set) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(&swiglu_gemm_kernel<UP>),
                            hipFuncAttributeMaxDynamicSharedMemorySize,
                            static_cast<int>(GM_LDS)) != hipSuccess)
      return REFLEX_ERR_LAUNCH;
    attr_set = true;
  }
  hipLaunchKernelGGL(swiglu_gemm_kernel<UP>, dim3(persistent_grid()), dim3(GM_THREADS), GM_LDS, s,
                     x, gather, tile_off, eo, E, dense_M, w0, w1, stride, K, N, x_rows, out_rows, out);
  return launch_status();
}

// Tall tiles where an expert would average RFX_TALL_MIN_ROWS rows or more at full
// pair capacity (the MFMAs, not the weight stream, bound such launches).
// The tall kernel reads its input rows through a buffer resource with 32-bit byte
// offsets, so its input operand must hold fewer than 2^30 elements.
bool use_tall(int cap, int E, int x_rows, int K) {
  return RFX_TALL_MIN_ROWS > 0 && E > 0 && cap / E >= RFX_TALL_MIN_ROWS &&
         static_cast<size_t>(x_rows) * static_cast<size_t>(K) < (size_t(1) << 30);
}

template <bool UP>
int launch_gemm_tall(const uint16_t* x, const int32_t* gather, const int32_t* eo, int E,
                     const uint16_t* w0, const uint16_t* w1, size_t stride, int K, int N, int x_rows,
                     int out_rows, uint16_t* out, hipStream_t s) {
  static bool attr_set = false;
  if (!attr_set) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(&swiglu_gemm_tall_kernel<UP>),
                            hipFuncAttributeMaxDynamicSharedMemorySize,
                            static_cast<int>(TL_LDS)) != hipSuccess)
      return REFLEX_ERR_LAUNCH;
    attr_set = true;
  }
  hipLaunchKernelGGL(swiglu_gemm_tall_kernel<UP>, dim3(persistent_grid()), dim3(TL_THREADS), TL_LDS,
                     s, x, gather, eo, E, w0, w1, stride, K, N, x_rows, out_rows, out);
  return launch_status();
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
  if (use_tall(cap, E, T, d))
    return launch_gemm_tall<true>(h, sorted_token, expert_offsets, E, wg, wu,
                                  static_cast<size_t>(f) * d, d, f, T, cap, routed_act(ws, E), s);
  return launch_gemm<true>(h, sorted_token, static_cast<const int32_t*>(ws), expert_offsets, E, -1,
                           wg, wu, static_cast<size_t>(f) * d, d, f, T, cap, routed_act(ws, E), s);
}

int launch_swiglu_down(const int32_t* expert_offsets, const uint16_t* wd, int E, int d, int f,
                       int cap, uint16_t* y_sorted, void* ws, hipStream_t s) {
  if (cap <= 0) return REFLEX_OK;
  if (use_tall(cap, E, cap, f))
    return launch_gemm_tall<false>(routed_act(ws, E), nullptr, expert_offsets, E, wd, nullptr,
                                   static_cast<size_t>(d) * f, f, d, cap, cap, y_sorted, s);
  return launch_gemm<false>(routed_act(ws, E), nullptr, static_cast<const int32_t*>(ws),
                            expert_offsets, E, -1, wd, nullptr, static_cast<size_t>(d) * f, f, d,
                            cap, cap, y_sorted, s);
}

int launch_swiglu_routed(const uint16_t* h, const int32_t* sorted_token,
                         const int32_t* expert_offsets, const uint16_t* wg, const uint16_t* wu,
                         const uint16_t* wd, int T, int E, int d, int f, int cap,
                         uint16_t* y_sorted, void* ws, hipStream_t s) {
  if (cap <= 0) return REFLEX_OK;
  int rc = launch_swiglu_plan(expert_offsets, E, ws, s);
  if (rc == REFLEX_OK)
    rc = launch_swiglu_up(h, sorted_token, expert_offsets, wg, wu, T, E, d, f, cap, ws, s);
  if (rc == REFLEX_OK)
    rc = launch_swiglu_down(expert_offsets, wd, E, d, f, cap, y_sorted, ws, s);
  return rc;
}

int launch_swiglu_dense(const uint16_t* x, const uint16_t* wg, const uint16_t* wu,
                        const uint16_t* wd, int M, int d, int f, uint16_t* y, void* ws,
                        hipStream_t s) {
  if (M <= 0) return REFLEX_OK;
  uint16_t* act = static_cast<uint16_t*>(ws);
  int rc = launch_gemm<true>(x, nullptr, nullptr, nullptr, 1, M, wg, wu, 0, d, f, M, M, act, s);
  if (rc == REFLEX_OK)
    rc = launch_gemm<false>(act, nullptr, nullptr, nullptr, 1, M, wd, nullptr, 0, f, d, M, M, y, s);
  return rc;
}

}  // namespace rfx
