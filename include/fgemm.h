/*
 * fgemm.h — C ABI of the MI355X (gfx950) fused GEMM + epilogue library.
 *
 * Two operations are exported:
 *
 *  1. fgemm: y = tail(x·Wᵀ + b), a dense GEMM whose post-GEMM ("tail") ops run
 *     inside the GEMM kernel on the fp32 accumulators, so the matmul result is
 *     read once and the result written once (paper §IV-B, the four techniques
 *     found in the generated GEMM + tail-ops kernels: layer-wise fusion,
 *     mixed-precision execution with fp32 accumulation and post-processing,
 *     single-pass reductions, partitioning without cross-block reductions).
 *     The tail is a chain of up to FG_MAX_OPS elementwise ops (scale, add,
 *     ReLU, GELU-tanh, SiLU, clamp, Mish, LeakyReLU — the pointwise
 *     vocabulary of Table III) optionally followed by one row reduction:
 *     LogSumExp over the N columns of each row, or GroupNorm over contiguous
 *     channel groups (Table III: Scale + LSE, Swish + GroupNorm), and then a
 *     second chain of up to FG_MAX_OPS elementwise ops applied to the
 *     reduction's result (Table III: LSE → Mish, GroupNorm → Swish → Mul →
 *     Swish, GroupNorm → LeakyReLU → Sum).
 *
 *  2. moe_grouped_ffn: one MoE expert-FFN step of a gpt-oss-20b-like layer
 *     (paper §IV-A: the MoE decode path and its "MoE finalize" kernel,
 *     Table I; §V: optimising the whole MoE-MLP block jointly): top-k routing
 *     over router logits, a stable token permutation by expert, the grouped
 *     gate/up GEMM with a clamped-SwiGLU epilogue, the grouped down GEMM
 *     (unweighted fp32 outputs per routed slot, in token order), and the
 *     finalize, which weights each slot by its routing weight and sums them.
 *
 * Conventions shared by every entry point
 *  - All tensors are row-major and dense. W follows the nn.Linear layout
 *    [N, K], so both GEMM operands are contiguous along K.
 *  - Every device buffer is owned by the caller. The library never allocates
 *    device memory, never synchronises the stream and keeps no pointer after a
 *    call returns. Work is enqueued on `stream` (a hipStream_t passed as
 *    void*; NULL is the default stream) and runs asynchronously.
 *  - Every argument is validated before anything is enqueued. On any error
 *    nothing is launched and a status other than FG_OK is returned;
 *    fg_last_error() then holds a one-line description (per thread).
 *    Launch failures reported by the HIP runtime map to FG_ERR_HIP.
 *  - Device pointers must be 16-byte aligned. Scalars marked "host" are read
 *    on the host; everything else is a device pointer.
 *  - No C++ exception crosses this interface.
 */
#ifndef FGEMM_H
#define FGEMM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FG_OK = 0,
  FG_ERR_INVALID_ARG = 1,   /* null pointer, bad shape, bad enum value */
  FG_ERR_UNSUPPORTED = 2,   /* valid request the library has no kernel for */
  FG_ERR_ALIGNMENT = 3,     /* pointer or leading dimension not aligned */
  FG_ERR_WORKSPACE = 4,     /* workspace missing or smaller than required */
  FG_ERR_HIP = 5            /* the HIP runtime reported a launch error */
} fg_status;

typedef enum { FG_F32 = 0, FG_BF16 = 1, FG_E4M3 = 2 } fg_dtype;

/* Elementwise tail ops, applied in order to z = x·Wᵀ (+ b), in fp32. */
typedef enum {
  FG_OP_SCALE = 0,      /* z·a */
  FG_OP_ADD = 1,        /* z + a */
  FG_OP_RELU = 2,       /* max(z, 0) */
  FG_OP_GELU_TANH = 3,  /* ½z(1 + tanh(√(2/π)(z + 0.044715 z³))) */
  FG_OP_SILU = 4,       /* z/(1 + e^−z) */
  FG_OP_CLAMP = 5,      /* min(max(z, a), b); requires a ≤ b */
  FG_OP_MISH = 6,       /* z·tanh(ln(1 + e^z))  (Mish, Table III) */
  FG_OP_LEAKY_RELU = 7  /* z for z ≥ 0, a·z otherwise (LeakyReLU, Table III) */
} fg_op_kind;

typedef struct {
  int32_t kind;         /* fg_op_kind */
  float a;
  float b;
} fg_op;

typedef enum {
  FG_RED_NONE = 0,
  FG_RED_LOGSUMEXP_ROW = 1, /* out[m] = log Σ_n exp(t[m,n]); out is fp32 [M] */
  FG_RED_GROUPNORM = 2      /* per row, over gn_groups contiguous channel
                               groups: (t − μ)/√(σ² + eps)·γ[n] + β[n], σ²
                               biased; out is [M, N] */
} fg_reduction;

#define FG_MAX_OPS 8

typedef struct {
  int32_t has_bias;         /* 1: add bias[N] (fp32) before the ops */
  int32_t n_ops;            /* 0 .. FG_MAX_OPS */
  fg_op ops[FG_MAX_OPS];
  int32_t reduction;        /* fg_reduction */
  int32_t gn_groups;        /* GroupNorm only: N must be a multiple */
  float gn_eps;             /* GroupNorm only: ≥ 0 */
  int32_t n_post_ops;       /* 0 .. FG_MAX_OPS; non-zero only with a reduction */
  fg_op post_ops[FG_MAX_OPS]; /* applied in order to the reduction's result:
                               per element after GroupNorm, per row value
                               after LogSumExp */
} fg_epilogue;

typedef struct fg_plan fg_plan; /* opaque, host memory, immutable once built */

/*
 * fgemm_plan — validate a problem and choose its kernel (host only; makes no
 * HIP call, so it can run without a GPU).
 *   plan     out: receives a new plan, to be released with fgemm_destroy.
 *   M, N, K  x is [M, K], W is [N, K], output [M, N] (or [M] for LSE).
 *            M = 0 is a valid empty problem (fgemm_run enqueues nothing);
 *            K = 0 gives z = b. Each must be < 2^31.
 *   in_dtype FG_F32, FG_BF16 or FG_E4M3 for both x and W. K must be a
 *            multiple of 4 (f32), 8 (bf16) or 16 (e4m3) so that rows stay
 *            16-byte aligned (FG_ERR_ALIGNMENT otherwise), and a row of x or
 *            W may hold at most 4 MiB (K·element size; FG_ERR_UNSUPPORTED
 *            beyond, since tile operands use 32-bit offsets). FG_E4M3 is the W8A8
 *            form: OCP e4m3fn codes with one fp32 scale per row of x and per
 *            row of W, run with fgemm_run_scaled; the fp8 MFMA accumulates in
 *            fp32 and z = (Σ_k qx·qw)·sx[m]·sw[n] + b before the tail (each
 *            128-value dot product is summed below fp32 precision: measured
 *            within 2.4e-5 of the sum of its |products| on Gaussian data, up
 *            to 2.6e-4 when one product dominates).
 *   out_dtype FG_F32 or FG_BF16; LogSumExp requires FG_F32. N must be a
 *            multiple of 4 (f32 out) or 8 (bf16 out) (FG_ERR_ALIGNMENT).
 *   epi      the tail (copied into the plan; the caller keeps ownership).
 *            GroupNorm accepts any gn_groups that divides N. Groups of
 *            16, 32, 64 or 128 channels (and 256 with bf16 inputs) are
 *            normalised inside the GEMM launch; other widths take a second
 *            launch, and the workspace then holds the fp32 values before
 *            the normalisation (M·N·4 bytes).
 */
fg_status fgemm_plan(fg_plan **plan, int64_t M, int64_t N, int64_t K,
                     int32_t in_dtype, int32_t out_dtype, const fg_epilogue *epi);

/* Bytes of device workspace fgemm_run needs: the LogSumExp per-tile
 * (max, Σexp) pairs, or the fp32 pre-normalisation values of a GroupNorm
 * that takes a second launch, and, when the plan splits K across
 * workgroups, one arrival counter per output tile plus an fp32 partial tile
 * per slice. 0 when none applies, and for a NULL plan. */
size_t fgemm_workspace_bytes(const fg_plan *plan);

/*
 * fgemm_run — enqueue y = tail(x·Wᵀ + b) on `stream`.
 *   A      [M, K] in_dtype.      W      [N, K] in_dtype (both may be NULL when K = 0).
 *   bias   [N] fp32, required iff epi.has_bias (else ignored, may be NULL).
 *   gamma, beta  [N] fp32, required iff GroupNorm (else ignored).
 *   out    [M, N] out_dtype, or [M] fp32 for LogSumExp; must not overlap A,
 *          W, bias, gamma, beta or the workspace.
 *   workspace, ws_bytes  device scratch of at least fgemm_workspace_bytes;
 *          may be NULL when that is 0. Contents on entry are ignored: the
 *          split-K arrival counters carry a per-run epoch, so values left by
 *          other runs or by other users of the memory are recognised as
 *          stale. Runs that overlap in time must not share a workspace.
 * Re-entrant: one plan may be run concurrently on several streams provided
 * each run has its own output and workspace.
 */
fg_status fgemm_run(const fg_plan *plan, const void *A, const void *W,
                    const float *bias, const float *gamma, const float *beta,
                    void *out, void *workspace, size_t ws_bytes, void *stream);

/*
 * fgemm_run_scaled — fgemm_run with per-row scales, required for FG_E4M3
 * plans (and ignored, may be NULL, for f32 / bf16 plans):
 *   a_scale  [M] fp32: x[m, k] = codes_x[m, k]·a_scale[m];
 *   w_scale  [N] fp32: W[n, k] = codes_w[n, k]·w_scale[n];
 * every other argument as for fgemm_run (A and W are the uint8 codes).
 * FG_ERR_INVALID_ARG for an e4m3 plan without both scales; fgemm_run on an
 * e4m3 plan returns the same status.
 */
fg_status fgemm_run_scaled(const fg_plan *plan, const void *A, const void *W,
                           const float *a_scale, const float *w_scale,
                           const float *bias, const float *gamma, const float *beta,
                           void *out, void *workspace, size_t ws_bytes, void *stream);

void fgemm_destroy(fg_plan *plan);

/* Kernel choice of a plan, for tests and reports: tile rows and columns,
 * workgroups per launch, launches per run, and K slices (1 unless the plan
 * splits K across workgroups). Returns FG_ERR_INVALID_ARG for a NULL plan.
 * Any output pointer may be NULL. */
fg_status fgemm_plan_info(const fg_plan *plan, int32_t *tile_m, int32_t *tile_n,
                          int64_t *workgroups, int32_t *launches, int32_t *k_slices);

/* ---------------------------------------------------------------------- */
/* MoE expert FFN                                                         */

typedef struct {
  int64_t T;                /* tokens (0 allowed: only expert_offsets is
                               written, all zeros) */
  int64_t H;                /* hidden size; multiple of 64 */
  int64_t I;                /* expert intermediate size; multiple of 64 */
  int32_t E;                /* experts, 1 .. 256 */
  int32_t top_k;            /* experts per token, 1 .. min(E, 8) */
  int32_t w_dtype;          /* FG_BF16, or FG_E4M3 (W8A8: tokens and the
                               intermediate are quantised per row on the fly) */
  float swiglu_alpha;       /* σ(α·gate); gpt-oss uses 1.702 */
  float swiglu_limit;       /* gate ≤ limit, −limit ≤ up ≤ limit; 7.0 */
  int32_t gateup_interleaved; /* 0: rows [0, I) gate, [I, 2I) up;
                                 1: even rows gate, odd rows up */
} moe_desc;

/* Device workspace moe_grouped_ffn needs for `d` (the permuted
 * intermediate, per-slot outputs, routing scratch, quantised activations).
 * 0 if d is NULL or invalid. */
size_t moe_workspace_bytes(const moe_desc *d);

/*
 * moe_grouped_ffn — enqueue one MoE expert-FFN step on `stream`.
 *   tokens         [T, H] bf16.
 *   router_logits  [T, E] fp32.
 *   w_gateup       [E, 2I, H] bf16, or e4m3 codes (one byte each).
 *   w_down         [E, H, I] bf16, or e4m3 codes.
 *   s_gateup       [E, 2I] fp32 per-row weight scales (e4m3 only, else NULL).
 *   s_down         [E, H] fp32 per-row weight scales (e4m3 only, else NULL).
 *   out            [T, H] bf16: out[t] = Σ_j w[t,j]·FFN_{idx[t,j]}(tokens[t]);
 *                  no output or workspace may overlap an input or each other.
 *   topk_idx       [T, top_k] int32 out: selected experts, logits descending,
 *                  ties to the lower expert index (a NaN logit ranks as −∞).
 *   topk_w         [T, top_k] fp32 out: softmax over the selected logits.
 *   perm           [T·top_k] int32 out: slot ids p = t·top_k + j sorted by
 *                  (expert, p) — stable, hence unique.
 *   expert_offsets [E + 1] int32 out: exclusive prefix of the per-expert
 *                  slot counts; expert e owns perm[offsets[e] .. offsets[e+1]).
 *   workspace, ws_bytes  at least moe_workspace_bytes(d).
 * Nothing is copied back to the host: the per-expert counts stay on the
 * device and the grouped GEMMs read them there. Arithmetic: fp32
 * accumulation (with e4m3 weights each 128-value dot product of the matrix
 * cores is summed below fp32 precision: measured within 2.4e-5 of the sum of
 * its |products| on Gaussian data, up to 2.6e-4 when one product dominates);
 * h (the SwiGLU output) is stored as bf16 (and, with e4m3
 * weights, quantised per row to e4m3); the per-slot down outputs stay fp32
 * and out is rounded once to bf16 after the weighted sum over j in
 * ascending order, so results are bit-identical from call to call.
 */
fg_status moe_grouped_ffn(const moe_desc *d, const void *tokens,
                          const float *router_logits, const void *w_gateup,
                          const void *w_down, const float *s_gateup,
                          const float *s_down, void *out, int32_t *topk_idx,
                          float *topk_w, int32_t *perm, int32_t *expert_offsets,
                          void *workspace, size_t ws_bytes, void *stream);

/*
 * moe_grouped_ffn_noalloc — moe_grouped_ffn for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops
 * and harnesses that forbid allocation. Same arguments, semantics and
 * results as moe_grouped_ffn, without workspace arguments: the workspace is
 * a static device array of moe_noalloc_scratch_bytes() bytes (64 MiB) inside
 * the library, one per GPU the library runs on, held until the process ends.
 * The call itself allocates nothing (the array's address is looked up once
 * per device on the first call there). Problems whose
 * moe_workspace_bytes(d) exceeds the array are rejected with
 * FG_ERR_UNSUPPORTED (at H = I = 2880, E = 32, top-4: up to about 970
 * tokens with bf16 weights, 790 with e4m3). All calls on one GPU share its
 * array: calls that overlap in time there (other streams or threads) race
 * and must be serialised by the caller. Every other error as for
 * moe_grouped_ffn; FG_ERR_HIP if the device or the array's address cannot
 * be queried.
 */
fg_status moe_grouped_ffn_noalloc(const moe_desc *d, const void *tokens,
                                  const float *router_logits, const void *w_gateup,
                                  const void *w_down, const float *s_gateup,
                                  const float *s_down, void *out, int32_t *topk_idx,
                                  float *topk_w, int32_t *perm, int32_t *expert_offsets,
                                  void *stream);

/* Bytes of the static scratch moe_grouped_ffn_noalloc uses on each GPU. */
size_t moe_noalloc_scratch_bytes(void);

/*
 * moe_finalize — the MoE finalize step on its own (paper §IV-A, the "MoE
 * finalize" kernel of Table I; moe_grouped_ffn's last launch is the same
 * kernel reading fp32 unweighted slot outputs and applying the weights):
 *   out[t, :] = Σ_{j = 0 .. top_k−1} y_slot[t·top_k + j, :]
 * summed in fp32 in ascending j, rounded once to bf16 (nearest even).
 *   y_slot  [T·top_k, H] bf16, row t·top_k + j = token t's j-th routed slot,
 *           already multiplied by its routing weight (caller-owned, device).
 *   out     [T, H] bf16 (caller-owned, device); must not overlap y_slot.
 *   T ≥ 0 (0: nothing is enqueued), 1 ≤ top_k ≤ 8, H a multiple of 8.
 * FG_ERR_INVALID_ARG for bad sizes or NULL pointers, FG_ERR_ALIGNMENT for H
 * not a multiple of 8 or pointers not 16-byte aligned; nothing is enqueued
 * on error.
 */
fg_status moe_finalize(const void *y_slot, void *out, int64_t T, int64_t H,
                       int32_t top_k, void *stream);

/*
 * add_rmsnorm — fused residual add + RMSNorm (paper §IV-A, "Fused Add +
 * RMSNorm" in Table I), for each of the T rows of H channels:
 *   s = x + residual  (fp32; exact for bf16 inputs)
 *   residual ← bf16(s)                                   (in place)
 *   out = bf16(s / sqrt(mean_h s² + eps) · weight)        (s before rounding)
 *   x [T, H] bf16; residual [T, H] bf16, read and overwritten; weight [H]
 *   bf16; out [T, H] bf16. All caller-owned device memory; out must not
 *   overlap x or residual. T ≥ 0 (0: nothing is enqueued); H a multiple of
 *   8 and at most 4096; eps finite and ≥ 0 (gpt-oss uses 1e-5).
 * FG_ERR_INVALID_ARG for bad sizes, eps or NULL pointers, FG_ERR_ALIGNMENT
 * for H not a multiple of 8 or pointers not 16-byte aligned,
 * FG_ERR_UNSUPPORTED for H above 4096; nothing is enqueued on error.
 */
fg_status add_rmsnorm(const void *x, void *residual, const void *weight,
                      void *out, int64_t T, int64_t H, float eps, void *stream);

/*
 * bias_rope_kv_update — QKV bias + rotary position embedding + paged KV-cache
 * write of one decode step (paper §IV-A, "Bias + RoPE + KV update" in
 * Table I). Each of the T tokens is the newest token of its own sequence, at
 * position positions[t]:
 *   s = qkv[t] + bias (fp32), split into n_q_heads query, n_kv_heads key and
 *   n_kv_heads value heads of head_dim values, in that order;
 *   query and key heads are rotated (RoFormer's rotary embedding): pair i of
 *   a head, (a, b), becomes (a·cos φ − b·sin φ, a·sin φ + b·cos φ) with
 *   φ = pos·rope_base^(−2i/head_dim); pairs are (i, i + head_dim/2) or, with
 *   `interleaved`, (2i, 2i + 1). The angle and its sine and cosine are taken
 *   in fp64, the rotation in fp32;
 *   q_out[t, h, :] = bf16(rotated query head h);
 *   kv_cache[blk, 0, h, r, :] = bf16(rotated key head h) and
 *   kv_cache[blk, 1, h, r, :] = bf16(value head h), with
 *   blk = block_table[t·max_blocks + pos / block_size], r = pos % block_size.
 * A token whose position is negative or at least max_blocks·block_size, or
 * whose block id lies outside [0, num_blocks), writes nothing to the cache
 * (its q_out row is still written). Two tokens of one call must not map to
 * the same cache row (their writes would race).
 *   qkv          [T, (n_q_heads + 2·n_kv_heads)·head_dim] bf16.
 *   bias         [(n_q_heads + 2·n_kv_heads)·head_dim] bf16, or NULL (no bias).
 *   positions    [T] int32.   block_table [T, max_blocks] int32.
 *   q_out        [T, n_q_heads, head_dim] bf16; must not overlap qkv.
 *   kv_cache     [num_blocks, 2, n_kv_heads, block_size, head_dim] bf16, read
 *                nowhere, written only in the rows above.
 * All caller-owned device memory; bf16 pointers 16-byte aligned, int32
 * pointers 4-byte aligned. FG_ERR_INVALID_ARG for a NULL desc or pointer
 * (bias excepted), bad sizes or a non-finite / non-positive base;
 * FG_ERR_ALIGNMENT for misaligned pointers or head_dim not a multiple of 16;
 * FG_ERR_UNSUPPORTED for head_dim above 256. T = 0 enqueues nothing.
 */
typedef struct {
  int64_t T;                /* decode tokens (one per sequence), 0 .. 2^31 − 1 */
  int32_t n_q_heads;        /* ≥ 1 */
  int32_t n_kv_heads;       /* ≥ 1 */
  int32_t head_dim;         /* multiple of 16, 16 .. 256 */
  int32_t block_size;       /* tokens per cache block, ≥ 1 */
  int32_t max_blocks;       /* entries per block_table row, ≥ 1 */
  int64_t num_blocks;       /* blocks in kv_cache, ≥ 1 */
  float rope_base;          /* θ base, finite and > 0 (gpt-oss: 150000) */
  int32_t interleaved;      /* 0: pairs (i, i + head_dim/2); 1: (2i, 2i + 1) */
} rope_desc;

fg_status bias_rope_kv_update(const rope_desc *d, const void *qkv, const void *bias,
                              const int32_t *positions, const int32_t *block_table,
                              void *q_out, void *kv_cache, void *stream);

/*
 * fg_quantize_rows_e4m3 — the W8A8 path's activation quantiser as a
 * standalone call: for each of `rows` rows of `cols` bf16 values,
 * s = amax/448 (1 for an all-zero row) and q = e4m3fn(v/s) with
 * round-to-nearest-even and saturation to ±448; both decisions in fp32.
 *   x [rows, cols] bf16; q [rows, cols] uint8 codes out; s [rows] fp32 out.
 *   cols must be a multiple of 8.
 */
fg_status fg_quantize_rows_e4m3(const void *x, int64_t rows, int64_t cols,
                                uint8_t *q, float *s, void *stream);

/*
 * Launch trace, for benchmarks and measurement tools. fg_trace_begin opens a
 * trace on the calling thread: from then on, the i-th kernel launch that any
 * entry point makes on this thread (i < capacity; later launches are not
 * traced) records one HIP event right before and one right after the
 * launch, on the launch's stream. fg_trace_end closes the trace and returns
 * the number of launches traced. fg_trace_read(i, ms, kernel) then waits
 * for launch i's second event and gives the time between its two events in
 * milliseconds, and the kernel's symbol name as the HIP runtime reports it
 * (valid until the next trace); either output may be NULL. The events are
 * created by the library on first use and kept for the thread's later
 * traces. While a trace is open, event records are enqueued beside every
 * launch, so a trace must not be open during graph capture and the timings
 * of untraced runs are the reference for throughput.
 * FG_ERR_INVALID_ARG for a capacity outside 1 .. 2^20, a read while the
 * trace is open or an index outside the traced launches; FG_ERR_HIP if the
 * runtime fails to create, wait for or time an event.
 */
fg_status fg_trace_begin(int32_t capacity);
int32_t fg_trace_end(void);
fg_status fg_trace_read(int32_t i, float *ms, const char **kernel);

/* Static description of a status code. */
const char *fg_status_str(fg_status s);

/* Description of the last error returned on the calling thread ("" if none). */
const char *fg_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FGEMM_H */
