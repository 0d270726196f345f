/*
 * reflex.h - C ABI of the REFLEX variable-K MoE layer for MI355X (gfx950).
 *
 * The layer is the MoE feed-forward block of a diffusion language model's
 * denoising forward in which each token i gets its own expert count k_i
 * (Section 3.2, Eq. (2)), chosen per forward by Refinement-Role Budgeting
 * (Section 4.2, Eq. (5)) and Frontier-Guided Expert Reallocation with the
 * Frontier-Progress Score (Section 4.3, Eqs. (6)-(9)), subject to the count
 * bounds of Eq. (3).
 *
 * Conventions shared by every entry point
 *  - All array arguments are DEVICE pointers owned by the caller; the library
 *    never allocates, frees or retains them.  Struct arguments
 *    (reflex_alloc_params, reflex_moe_args) are HOST pointers, read during the
 *    call only.
 *  - bf16 data is passed as uint16_t bit patterns.  Matrices are row-major and
 *    dense (leading dimension = row length).
 *  - `stream` is a hipStream_t passed as void* (NULL = default stream).  Work is
 *    enqueued asynchronously; nothing is read back to the host and no call
 *    synchronises.  Calls keep no state between them and may be made from several
 *    threads; the lasting resources are a second stream per device (non-blocking,
 *    default priority, created on first use) on which reflex_moe_forward runs the
 *    shared expert beside the routing, ordered against `stream` by events from a
 *    per-device pool (created on first use, reused by later calls), and the device
 *    scratch of reflex_moe_forward_noalloc.
 *  - Arguments are validated on the host before anything is launched; on error
 *    nothing is launched and a negative status is returned.  No C++ exception
 *    crosses the ABI.
 *  - T = 0 (no tokens) is valid and enqueues nothing.
 *  - Alignment (REFLEX_ERR_SHAPE otherwise): bf16 matrices (h, expert weights,
 *    y_sorted, shared_y, residuals, out), the fp32 router weight and workspaces
 *    must be 16-byte aligned (the kernels move them in 16-byte vectors); every
 *    other pointer needs the natural alignment of its element type.
 *  - Content preconditions that cannot be checked without reading device memory
 *    (seq_offsets non-decreasing from 0 to T, block_idx >= 0, hist_len in
 *    {0,1,2}, finite logits, expert_offsets consistent with the pair count) are
 *    the caller's.  Kernels never index outside the buffers whose sizes the
 *    arguments state, whatever those contents are: counts are clamped to
 *    [0, k_max] before they size anything.
 */
#ifndef REFLEX_H
#define REFLEX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------------ */
#define REFLEX_OK                 0
#define REFLEX_ERR_NULL         (-1)  /* a required pointer is NULL                        */
#define REFLEX_ERR_SHAPE        (-2)  /* a size is out of range or not a supported multiple */
#define REFLEX_ERR_PARAM        (-3)  /* a hyper-parameter is out of range or not finite    */
#define REFLEX_ERR_WORKSPACE    (-4)  /* workspace or pair capacity too small               */
#define REFLEX_ERR_LAUNCH       (-5)  /* the HIP runtime reported a launch error            */
#define REFLEX_ERR_UNSUPPORTED  (-6)  /* a valid request this build does not implement      */

/* ---- limits ------------------------------------------------------------------ */
#define REFLEX_MAX_EXPERTS  256       /* E <= 256                                        */
#define REFLEX_MAX_K        32        /* k_max <= min(E, 32)                             */
#define REFLEX_D_MULTIPLE   128       /* hidden size d must be a multiple of this        */
#define REFLEX_F_MULTIPLE   64        /* expert widths f, f_shared must be multiples     */
#define REFLEX_MAX_DIM      16384     /* d, f, f_shared <= this                          */
#define REFLEX_MAX_TOKENS   (1 << 24) /* T <= this                                       */

/* Ranking key of the active-block reallocation (Section 4.3; Appendix C). */
#define REFLEX_SIGNAL_FPS          0  /* S = F * P, Eq. (8)                    */
#define REFLEX_SIGNAL_FRONTIER     1  /* F alone, Eq. (6)                      */
#define REFLEX_SIGNAL_PROGRESS     2  /* P alone, Eq. (7)                      */
#define REFLEX_SIGNAL_CONFIDENCE   3  /* lagged confidence c^{t-1}             */
#define REFLEX_SIGNAL_UNCERTAINTY  4  /* 1 - c^{t-1}                           */

/*
 * Allocation hyper-parameters (Eqs. (3), (5)-(9); defaults in Section 5.1:
 * k_base 8, delta_role 4, delta_cur 2, q 0.25, theta 0.9, w_cf 0.30 or 0.25,
 * v_ref 0.01, tau 0.05).  Real values are float32 and are widened exactly to
 * fp64 inside the kernels.
 * Valid: 0 <= k_min <= k_max <= REFLEX_MAX_K; k_base, delta_role, delta_cur >= 0;
 * 0 < q <= 0.5; tau > 0; w_cf > 0; theta, v_ref finite; signal in 0..4.
 */
typedef struct {
  int32_t k_base;      /* K_base: nominal count (Eq. (5))                            */
  int32_t delta_role;  /* delta_role: role offset (Eq. (5)); K_cur = k_base+delta_role */
  int32_t delta_cur;   /* delta_cur: reallocation offset (Eq. (9))                  */
  int32_t k_min;       /* K_min: lower count bound (Eq. (3)), applied as a clamp     */
  int32_t k_max;       /* K_max: upper count bound (Eq. (3)), applied as a clamp     */
  float   q;           /* outer-group fraction; groups have floor(q*m) members      */
  float   theta;       /* commitment threshold theta                                */
  float   w_cf;        /* commitment-frontier width w_cf                            */
  float   v_ref;       /* velocity reference v_ref                                  */
  float   tau;         /* gate temperature tau                                      */
  int32_t signal;      /* REFLEX_SIGNAL_*                                           */
} reflex_alloc_params;

/*
 * The paper's settings as ready-made parameters (host only, no GPU work):
 * Section 5.1 defaults with the given count bounds and frontier width, and the
 * ablation variants of Section 5.3 and Appendix C:
 *  REFLEX_PRESET_FULL         RRB + FGER with the Frontier-Progress Score
 *  REFLEX_PRESET_RRB_ONLY     delta_cur = 0 (no reallocation inside the active block)
 *  REFLEX_PRESET_FGER_ONLY    delta_role = 0 (every role keeps k_base)
 *  REFLEX_PRESET_FRONTIER_ONLY, _PROGRESS_ONLY, _CONFIDENCE_ONLY, _UNCERTAINTY_ONLY
 *                             the full method ranking by one signal (REFLEX_SIGNAL_*)
 *  k_min, k_max   count bounds (e.g. 2, 12); w_cf 0.30 (LLaDA-MoE) or 0.25 (LLaDA2.0-mini)
 * Errors: NULL out; unknown preset (REFLEX_ERR_PARAM); the result failing the
 * validity rules above (REFLEX_ERR_PARAM).
 */
#define REFLEX_PRESET_FULL              0
#define REFLEX_PRESET_RRB_ONLY          1
#define REFLEX_PRESET_FGER_ONLY         2
#define REFLEX_PRESET_FRONTIER_ONLY     3
#define REFLEX_PRESET_PROGRESS_ONLY     4
#define REFLEX_PRESET_CONFIDENCE_ONLY   5
#define REFLEX_PRESET_UNCERTAINTY_ONLY  6
int reflex_alloc_preset(int preset, int k_min, int k_max, float w_cf, reflex_alloc_params* out);

/* ---- introspection ---------------------------------------------------------- */
int         reflex_version(void);               /* 100 * major + minor                */
const char* reflex_status_string(int status);   /* static string, never NULL          */
size_t      reflex_sizeof_alloc_params(void);   /* sizeof(reflex_alloc_params)        */
size_t      reflex_sizeof_moe_args(void);       /* sizeof(reflex_moe_args)            */

/* ---- workspace sizes ----------------------------------------------------------
 * Bytes of device scratch the entry points below need; 0 on invalid sizes.
 * reflex_workspace_size covers reflex_moe_forward and is also large enough for
 * reflex_permute and reflex_grouped_swiglu with pair_capacity = T * k_max. */
size_t reflex_workspace_size(int T, int E, int d, int f, int f_shared, int k_max);
size_t reflex_permute_workspace_size(int pair_capacity, int E);

/*
 * Where reflex_moe_forward (and _timed, _noalloc) leaves the routing of a forward in its
 * workspace, for inspection once the stream has completed (tests, debugging): byte
 * offset of `field` in a workspace sized by reflex_workspace_size with the same
 * arguments (k_max = the forward's pair-capacity count kcap).  The arrays are those of
 * reflex_topk_variable (pair_offsets [T+1], pair_expert and pair_weight [T * kcap]) and
 * reflex_permute (expert_offsets [E+1], sorted_token and pair_to_sorted [T * kcap]),
 * holding the forward's P selected expert-token pairs (Section 3.2).  The layout is
 * internal to this library version.  Returns (size_t)-1 for invalid sizes or field.
 */
#define REFLEX_WS_PAIR_OFFSETS    0
#define REFLEX_WS_PAIR_EXPERT     1
#define REFLEX_WS_PAIR_WEIGHT     2
#define REFLEX_WS_EXPERT_OFFSETS  3
#define REFLEX_WS_SORTED_TOKEN    4
#define REFLEX_WS_PAIR_TO_SORTED  5
size_t reflex_workspace_offset(int T, int E, int d, int f, int f_shared, int k_max, int field);
size_t reflex_swiglu_workspace_size(int pair_capacity, int E, int f);

/*
 * Router scores r_{i,e} = sum_k h[i,k] * w_router[e,k] (+ bias[e])  (Section 3.2).
 *  h        [T, d]  bf16   token representations
 *  w_router [E, d]  fp32   router weight (nn.Linear layout)
 *  bias     [E]     fp32   optional per-expert offset, NULL for none
 *  logits   [T, E]  fp32   output; products of the bf16 input and the fp32 weight
 *                          are accumulated in fp32 (max row error ~1e-6 relative)
 * Errors: NULL h/w_router/logits; T, d or E out of range (d % 128, 1 <= E <= 256).
 */
int reflex_router_logits(const uint16_t* h, const float* w_router, const float* bias,
                         float* logits, int T, int d, int E, void* stream);

/*
 * Per-token expert counts for one denoising forward (the allocator Pi of Eq. (3)).
 * For every sequence s (tokens seq_offsets[s] .. seq_offsets[s+1]-1, active block
 * active_block[s]):
 *   1. RRB prior k_i = H(|b(i) - a_s|)  (Eq. (5)); prompt tokens have b = 0.
 *   2. J = masked tokens of the active block (Section 3.1).  Tokens of J with
 *      hist_len >= 1 are ranked by the key `params->signal` selects, in fp64,
 *      descending, ties to the lower token index; the first floor(q*m) get
 *      K_cur + delta_cur, the last floor(q*m) get K_cur - delta_cur, the rest
 *      K_cur (Eq. (9)).  Tokens of J with no history keep K_cur.
 *      Forecast (Section 4.3): hist 2: v = c1 - c2 clipped to +-w_cf/2,
 *      c_hat = clip(c1 + v, 0, 1); hist 1: v = 0, c_hat = c1, P = 1.
 *   3. Every count is clamped to [k_min, k_max].
 *  block_idx   [T] int32   b(i) >= 0
 *  masked      [T] uint8   nonzero = position still [MASK]
 *  hist_len    [T] int8    number of confidence observations available (0..2)
 *  conf_prev1  [T] fp32    c^{t-1};  conf_prev2 [T] fp32  c^{t-2}
 *  seq_offsets [B+1] int32 token ranges, non-decreasing, 0 .. T
 *  active_block[B] int32   a_s >= 1
 *  params      host pointer
 *  k_out       [T] int32   output counts
 *  pairs_out   [1] int32   output sum_i k_i
 *  fps_out     [T] fp64    optional: the ranking key of every ranked token, NaN
 *                          for tokens that are not ranked; NULL to skip
 * Errors: NULL required pointers; T > 0 with B < 1; invalid params.
 */
int reflex_assign_budget(const int32_t* block_idx, const uint8_t* masked, const int8_t* hist_len,
                         const float* conf_prev1, const float* conf_prev2,
                         const int32_t* seq_offsets, const int32_t* active_block, int B, int T,
                         const reflex_alloc_params* params, int32_t* k_out, int32_t* pairs_out,
                         double* fps_out, void* stream);

/*
 * Decoding state after one denoising forward (Section 3.1, Eq. (1)), per sequence:
 * the masked positions of the active block whose confidence reaches theta are
 * committed (with min_commit = 1, a forward that would commit none commits the
 * most confident one, lowest position on ties); every position that was masked
 * records the forward's confidence (conf_prev2 <- conf_prev1, conf_prev1 <- conf_t,
 * hist_len <- min(hist_len + 1, 2)); a sequence whose active block has no masked
 * position left moves to its next block, if it has one.
 *  conf_t       [T] fp32  confidences of this forward (read at masked positions)
 *  block_idx    [T] int32, seq_offsets [B+1] int32   as in reflex_assign_budget
 *  theta        commitment threshold in (0, 1]
 *  masked, hist_len, conf_prev1, conf_prev2 [T], active_block [B]   updated in place
 *  remaining    [B] int32 output: masked positions left per sequence, or NULL
 * Errors: NULL required pointers; T > 0 with B < 1; theta outside (0, 1] or
 * min_commit not 0/1 (REFLEX_ERR_PARAM).
 */
int reflex_advance_state(const float* conf_t, const int32_t* block_idx, const int32_t* seq_offsets,
                         int B, int T, float theta, int min_commit, uint8_t* masked,
                         int8_t* hist_len, float* conf_prev1, float* conf_prev2,
                         int32_t* active_block, int32_t* remaining, void* stream);

/*
 * Counts derived from the router scores alone: the score-threshold rules the
 * paper compares against (Appendix B).  Routing mass is the softmax of a token's
 * scores over all E experts, evaluated in fp64.
 *  rule = REFLEX_RULE_TOP_P:     k_i = the smallest n such that the n best experts
 *                                (logit descending, index ascending) hold routing
 *                                mass >= threshold (summed in that order);
 *  rule = REFLEX_RULE_THRESHOLD: k_i = the number of experts with routing mass
 *                                > threshold;
 * then k_i = min(max(k_i, k_min), k_max).
 *  logits    [T, E] fp32
 *  threshold p in (0, 1] for Top-p; tau in [0, 1) for the threshold rule (a float,
 *            widened exactly to fp64)
 *  k_out     [T] int32 output counts
 *  pairs_out [1] int32 output sum_i k_i, or NULL
 * Errors: NULL logits / k_out; unknown rule or threshold out of range
 * (REFLEX_ERR_PARAM); k_min < 0, k_min > k_max or k_max > min(E, 32) (REFLEX_ERR_SHAPE).
 */
#define REFLEX_RULE_BUDGET     0   /* Refinement-Role Budgeting + FGER (Sections 4.2-4.3) */
#define REFLEX_RULE_TOP_P      1   /* Top-p over routing mass (Appendix B)                */
#define REFLEX_RULE_THRESHOLD  2   /* Expert-Threshold Routing (Appendix B)               */
int reflex_count_rule(const float* logits, int T, int E, int rule, float threshold, int k_min,
                      int k_max, int32_t* k_out, int32_t* pairs_out, void* stream);

/*
 * Variable-count TopK and routing weights (Section 3.2, Eq. (2)).
 * Token i keeps its min(max(k[i],0), k_max) best experts in the order (logit
 * descending, expert index ascending; -0.0 == +0.0).  Pairs are written
 * token-major, in rank order, at pair_offsets[i] ... pair_offsets[i+1]-1.
 *  logits       [T, E] fp32
 *  k            [T]    int32   counts (clamped as above)
 *  norm_topk    1: alpha = softmax over the selected experts (sums to 1);
 *               0: alpha = the full softmax probability over all E experts
 *  pair_offsets [T+1]  int32   output exclusive prefix sum of the counts
 *  pair_expert  [pair_capacity] int32  output expert of each pair
 *  pair_weight  [pair_capacity] fp32   output alpha of each pair
 *  pair_capacity must be >= T * k_max (REFLEX_ERR_WORKSPACE otherwise).
 * Errors: NULL pointers; k_max < 0 or > min(E, 32); norm_topk not 0/1.
 */
int reflex_topk_variable(const float* logits, const int32_t* k, int T, int E, int k_max,
                         int norm_topk, int32_t* pair_offsets, int32_t* pair_expert,
                         float* pair_weight, int32_t pair_capacity, void* stream);

/*
 * Group the selected expert-token pairs by expert.  The pairs are those of
 * Section 3.2: token i contributes one pair per selected expert, P = sum_i k_i in
 * all, and each pair is one row of the routed experts' work in Eq. (2).  A stable
 * counting sort of the token-major pair list by expert orders the rows by
 * (expert, token), so every expert's rows are contiguous for its GEMM.
 *  pair_offsets [T+1] int32, pair_expert [P] int32   from reflex_topk_variable
 *  pairs        [1]   int32  device P (clamped to pair_capacity)
 *  expert_offsets [E+1] int32  output: rows of expert e are
 *                              expert_offsets[e] .. expert_offsets[e+1]-1
 *  sorted_token [pair_capacity] int32  output: token of each expert-sorted row
 *  pair_to_sorted [pair_capacity] int32 output: expert-sorted row of each pair
 *  ws, ws_bytes  scratch of >= reflex_permute_workspace_size(pair_capacity, E)
 * Errors: NULL pointers; E out of range; workspace too small.
 */
int reflex_permute(const int32_t* pair_offsets, const int32_t* pair_expert, const int32_t* pairs,
                   int T, int E, int32_t pair_capacity, int32_t* expert_offsets,
                   int32_t* sorted_token, int32_t* pair_to_sorted, void* ws, size_t ws_bytes,
                   void* stream);

/*
 * SwiGLU experts on expert-sorted rows (the expert E_e of Eq. (2); two input and
 * one output projection as counted in Appendix A, Eq. (10)):
 *   for each row j of expert e, x = h[sorted_token[j]],
 *   y_sorted[j] = W_down[e] (SiLU(W_gate[e] x) * (W_up[e] x)).
 * Both projections run on bf16 MFMA with fp32 accumulation; the activation
 * SiLU(g)*u is rounded to bf16 once, y once.
 *  h        [T, d] bf16;  w_gate, w_up [E, f, d] bf16;  w_down [E, d, f] bf16
 *  y_sorted [pair_capacity, d] bf16 output (rows >= expert_offsets[E] untouched)
 *  ws       scratch of >= reflex_swiglu_workspace_size(pair_capacity, E, f)
 * Errors: NULL pointers; d % 128 or f % 64 nonzero; workspace too small.
 */
int reflex_grouped_swiglu(const uint16_t* h, const int32_t* sorted_token,
                          const int32_t* expert_offsets, const uint16_t* w_gate,
                          const uint16_t* w_up, const uint16_t* w_down, int T, int E, int d,
                          int f, int32_t pair_capacity, uint16_t* y_sorted, void* ws,
                          size_t ws_bytes, void* stream);

/*
 * Weighted combine (Eq. (2)): out[i] = sum over the pairs j of token i, in rank
 * order, of pair_weight[j] * y_sorted[pair_to_sorted[j]], plus shared_y[i] when
 * given; accumulated in fp32 and rounded to bf16 once.
 *  y_sorted [pair_capacity, d] bf16; pair_offsets [T+1];
 *  pair_to_sorted, pair_weight [pair_capacity]  (pair indices and rows are clamped
 *                          to [0, pair_capacity) before use)
 *  shared_y [T, d] bf16 optional (always-on shared expert, weight 1)
 *  out      [T, d] bf16 output
 * Errors: NULL pointers; d % 128 nonzero; pair_capacity < 0.
 */
int reflex_combine(const uint16_t* y_sorted, const int32_t* pair_offsets,
                   const int32_t* pair_to_sorted, const float* pair_weight,
                   const uint16_t* shared_y, int T, int d, int32_t pair_capacity, uint16_t* out,
                   void* stream);

/*
 * The whole layer on one stream, no host synchronisation: router -> counts ->
 * TopK -> permutation -> SwiGLU experts -> combine (+ shared expert, + residuals).
 * Count source, first match wins:
 *   k_in != NULL   reuse counts computed earlier in the same forward (the paper
 *                  shares k_i across MoE layers, Section 3.3);
 *   uniform_k > 0  default fixed token-choice routing, k_i = uniform_k;
 *   k_rule = REFLEX_RULE_TOP_P / REFLEX_RULE_THRESHOLD
 *                  reflex_count_rule on this layer's scores with k_threshold and the
 *                  bounds params.k_min, params.k_max;
 *   otherwise      reflex_assign_budget with `params` and the token state.
 * Pair capacity is T * kcap with kcap = uniform_k if uniform_k > 0, else params.k_max;
 * counts (k_in included) are clamped to [0, kcap].  `params` is validated only when
 * uniform_k <= 0.
 */
typedef struct {
  int32_t T, d, E, f;
  int32_t f_shared;        /* width of the always-on shared expert, 0 = none           */
  int32_t norm_topk;       /* as in reflex_topk_variable                               */
  int32_t uniform_k;       /* > 0: fixed count for every token                         */
  int32_t B;               /* number of sequences (budget path)                         */
  int32_t k_rule;          /* REFLEX_RULE_*; 0 = the REFLEX budget                      */
  float   k_threshold;     /* p or tau of the score-derived rules                       */
  const uint16_t *h;                         /* [T, d]                                   */
  const uint16_t *w_gate, *w_up, *w_down;    /* [E, f, d], [E, f, d], [E, d, f]          */
  const uint16_t *ws_gate, *ws_up, *ws_down; /* shared [fs, d], [fs, d], [d, fs] or NULL  */
  const float    *w_router, *router_bias;    /* [E, d], [E] or NULL                      */
  const int32_t  *block_idx, *seq_offsets, *active_block;  /* budget path only           */
  const uint8_t  *masked;
  const int8_t   *hist_len;
  const float    *conf_prev1, *conf_prev2;
  const int32_t  *k_in;                      /* [T] or NULL                              */
  const uint16_t *residual_a, *residual_b;   /* [T, d] bf16 added before rounding, or NULL */
  reflex_alloc_params params;
  uint16_t *out;                             /* [T, d] bf16                              */
  int32_t  *k_out;                           /* [T] counts used, or NULL                 */
  int32_t  *pairs_out;                       /* [1] P, or NULL                           */
  float    *logits_out;                      /* [T, E] router scores (bias added), or NULL */
} reflex_moe_args;

/* ws: >= reflex_workspace_size(T, E, d, f, f_shared, kcap) bytes, 256-byte aligned. */
int reflex_moe_forward(const reflex_moe_args* args, void* ws, size_t ws_bytes, void* stream);

/*
 * reflex_moe_forward for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the same work
 * on the same kernels, with the workspace taken from a scratch array the library holds
 * on each device (REFLEX_NOALLOC_SCRATCH_BYTES, reserved when the library is loaded on
 * that device and held until the process ends).  The call allocates nothing: no
 * hipMalloc / hipFree, no stream or event creation (the shared expert runs on `stream`,
 * not on a side stream).  The caller still passes every input and output in `args`.
 * Layers whose reflex_workspace_size(T, E, d, f, f_shared, kcap) exceeds
 * REFLEX_NOALLOC_SCRATCH_BYTES are rejected with REFLEX_ERR_WORKSPACE before anything
 * is launched (96 MiB holds, e.g., one LLaDA-MoE-shaped layer of T = 1024 tokens,
 * d 2048, E 64, f 1024, k_max 12).  Every call on a device shares that device's scratch
 * and leaves its contents behind (nothing in it needs to start zeroed): calls whose
 * work overlaps on one device (other streams, other threads) race on it and must be
 * serialised by the caller.
 * Errors: as reflex_moe_forward; REFLEX_ERR_LAUNCH if the scratch cannot be located.
 */
#define REFLEX_NOALLOC_SCRATCH_BYTES (96u << 20)
int reflex_moe_forward_noalloc(const reflex_moe_args* args, void* stream);

/*
 * reflex_moe_forward with timing marks, for benchmarks: identical work, plus
 * hipEventRecord(stage_events[i], stream) at each stage boundary:
 *   0 start, 1 router done (for layers with T < 4096 on the REFLEX budget path one
 *   launch computes the counts and the scores as d/256 partial sums, which step 3 adds
 *   with the bias), 2 counts done (budget / rule / uniform fill / reuse),
 *   3 count scan + TopK done, 4 permutation + GEMM tile plan done,
 *   5 gate/up GEMM done, 6 down GEMM done, 7 shared expert done, 8 combine done.
 * stage_events: host array of REFLEX_N_STAGE_EVENTS hipEvent_t handles created by
 * the caller (hipEventCreate); the library only records them.
 * Errors: as reflex_moe_forward; NULL stage_events or a NULL entry;
 * n_stage_events != REFLEX_N_STAGE_EVENTS (REFLEX_ERR_SHAPE).
 */
#define REFLEX_N_STAGE_EVENTS 9
int reflex_moe_forward_timed(const reflex_moe_args* args, void* ws, size_t ws_bytes, void* stream,
                             void* const* stage_events, int n_stage_events);

#ifdef __cplusplus
}
#endif
#endif /* REFLEX_H */
