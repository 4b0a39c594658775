/*
 * laga.h — C ABI of one rank's share of LAGA (Latent All-Gather Attention).
 *
 * After the latent all-gather (Alg. 1 step 3) a rank holds, for the whole
 * gathered sequence, the compressed latent c_kv [B,S,d_c] and the shared RoPE
 * key k_pe [B,S,d_rope]; after the head-scatter (Alg. 1 step 2) it holds the
 * queries q [B,S,H,d_nope+d_rope] of its H heads, and it owns the head shard
 * W_kv_b [d_c, H*(d_nope+d_v)] of the up-projection. This library computes:
 *
 *   laga_reconstruct_kv : Alg. 1 step 4 — kv = c_kv @ W_kv_b (per-head K_nope, V)
 *   laga_attn_fwd       : Alg. 1 step 5 — causal softmax attention with
 *                         K_h = [K_nope,h || k_pe] (k_pe broadcast to all heads,
 *                         property P2 of Section 2.1) and V_h; also returns the
 *                         per-row log-sum-exp that the backward reuses
 *   laga_attn_bwd       : the per-rank backward (Section 5.2 covers the
 *                         collectives around it): dq, the head-shard partials
 *                         dc_kv and dk_pe, and the W_kv_b shard gradient dW
 *   laga_out_proj_fwd/_bwd : Alg. 1 step 7, the output projection W_o after the
 *                         out all-to-all, and its backward
 *
 * Layouts (all row-major, contiguous, device memory, 16-byte aligned):
 *   c_kv   [B, S, d_c]                     element dtype
 *   k_pe   [B, S, d_rope]                  element dtype
 *   q      [B, S, H, d_nope + d_rope]      element dtype; q_nope first, then q_rope
 *   w_kv_b [d_c, H * (d_nope + d_v)]       element dtype; head h owns the column
 *                                          block [h*(d_nope+d_v), (h+1)*(d_nope+d_v)),
 *                                          K_nope columns first, then V
 *   kv     [B, S, H, d_nope + d_v]         element dtype (= [B*S, H*(d_nope+d_v)])
 *   out    [B, S, H, d_v]                  element dtype
 *   lse    [B, H, S]                       fp32, natural-log log-sum-exp of each row
 *   dout   [B, S, H, d_v]                  element dtype
 *   dq     [B, S, H, d_nope + d_rope]      element dtype
 *   dc_kv  [B, S, d_c]                     fp32 (partial sum over this head shard)
 *   dk_pe  [B, S, d_rope]                  fp32 (partial sum over this head shard)
 *   dw_kv_b[d_c, H * (d_nope + d_v)]       fp32 (the full gradient of this shard)
 *
 * Conventions:
 *   - Ownership: the caller owns every buffer, including the workspace; the
 *     library allocates and frees nothing and keeps no state between calls.
 *   - Asynchrony: work is enqueued on `stream` (a hipStream_t passed as void*,
 *     NULL = the default stream); calls return without synchronising.
 *   - Validation happens on the host before any launch; on error nothing is
 *     launched and no output is touched. Asynchronous device faults surface at
 *     the caller's next synchronisation. No exception crosses the ABI.
 *   - Every output is overwritten, never accumulated into.
 *   - dc_kv and dk_pe are partial sums over this rank's heads; across ranks
 *     they are completed by the reduce-scatter that is the backward of the
 *     latent all-gather (Section 5.2), so they are returned in fp32 to be summed
 *     before any rounding to the element dtype.
 *   - Causal means key j is visible to query i iff j <= i (0-based positions in
 *     the gathered sequence, S_q == S_k). Non-causal attends to every key.
 *   - Supported head dims: (d_nope, d_rope, d_v) = (128, 64, 128) — DeepSeek-V3 —,
 *     (64, 32, 64) and (32, 16, 32); d_c a multiple of 32 up to 1024; S >= 1;
 *     B >= 1; H >= 1. Anything else returns LAGA_ERR_UNSUPPORTED. Each width is a
 *     compile-time kernel instance (the tile shapes follow from it); the
 *     DeepSeek-V3 widths have the tuned bf16 kernels, the others the generic ones.
 *   - Kernels index inside a tensor with 32-bit element offsets: B*S*H*W, with
 *     W = d_nope + max(d_rope, d_v) + max(d_nope, d_v), B*S*d_c, B*S, and
 *     16*d_c*H*(d_nope + d_v) must each stay below 2^31, else
 *     LAGA_ERR_UNSUPPORTED (and laga_workspace_bytes() returns 0). Memory,
 *     not this limit, bounds S first for the backward with dq_mode FROM_STORE:
 *     its dS^T store holds B*H*S*S/2 bf16 values (dq_mode RECOMPUTE has none).
 *   - Results do not depend on H: every per-head output (kv columns, out, lse,
 *     dq, dw_kv_b columns) of a head is bit-identical whichever head shard it is
 *     computed in; repeated calls are bit-identical.
 */
#ifndef LAGA_H_
#define LAGA_H_

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__) || defined(__clang__)
#define LAGA_API __attribute__((visibility("default")))
#else
#define LAGA_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

#define LAGA_ABI_VERSION 3

typedef enum {
  LAGA_OK = 0,
  LAGA_ERR_NULL = 1,        /* a required pointer (or the problem) is NULL */
  LAGA_ERR_SHAPE = 2,       /* a dimension is <= 0 or sizes are inconsistent */
  LAGA_ERR_UNSUPPORTED = 3, /* dims/dtype/mode/size the library has no kernel for */
  LAGA_ERR_ALIGN = 4,       /* a pointer is not 16-byte aligned */
  LAGA_ERR_WORKSPACE = 5,   /* workspace smaller than laga_workspace_bytes() */
  LAGA_ERR_DEVICE = 6,      /* the HIP runtime reported an error at launch */
  LAGA_ERR_SCRATCH = 7      /* laga_attn_bwd_noalloc: workspace need above its fixed array */
} laga_status_t;

typedef enum { LAGA_DTYPE_BF16 = 0, LAGA_DTYPE_FP32 = 1 } laga_dtype_t;

/* Where attention gets its per-head K_nope/V from.
 * MATERIALIZED: from `kv`, written beforehand by laga_reconstruct_kv.
 * FUSED: rebuilt tile by tile on chip from c_kv and w_kv_b; no per-head K/V
 *        tensor is ever written to HBM by the forward. */
typedef enum { LAGA_KV_MATERIALIZED = 0, LAGA_KV_FUSED = 1 } laga_kv_mode_t;

typedef enum { LAGA_OP_FWD = 0, LAGA_OP_BWD = 1, LAGA_OP_PROLOGUE_BWD = 2 } laga_op_t;

/* How the backward gets dq = scale * dZ K (dZ = P * (dP - delta), the score gradient).
 * FROM_STORE: the key-stationary pass that forms dZ for dK also writes it (bf16) to a
 *        store in the workspace, and the dq pass is a product over that store. This
 *        is the fastest path, but the store holds B*H*S*S/2 values (about 4.3 GB at
 *        S = 16384, H = 16). Only bf16 with 192/128-wide heads has it; other problems
 *        recompute (below) whatever this field says.
 * RECOMPUTE: no buffer of S*S size anywhere (workspace linear in S): the dq pass is
 *        query-stationary and recomputes the scores and dP for its queries, which costs
 *        the Q K^T and dO V^T products a second time. Every output equals FROM_STORE's
 *        exactly for bf16 with 192/128-wide heads (the same products, exp2 arguments,
 *        roundings and key order); elsewhere dq may differ in fp32 summation order. */
typedef enum { LAGA_DQ_FROM_STORE = 0, LAGA_DQ_RECOMPUTE = 1 } laga_dq_mode_t;

typedef struct {
  int64_t batch;       /* B */
  int64_t seq_len;     /* S: gathered sequence length */
  int64_t n_heads;     /* H: heads of THIS rank's shard */
  int64_t d_c;         /* latent width (d_kv) */
  int64_t d_nope;      /* per-head no-RoPE q/k width */
  int64_t d_rope;      /* shared RoPE band width */
  int64_t d_v;         /* per-head value width */
  float softmax_scale; /* multiplies q.k; the paper's 1/sqrt(d) with d = d_nope + d_rope */
  int32_t causal;      /* 1: causal mask, 0: none */
  int32_t dtype;       /* laga_dtype_t: element type of all non-fp32 tensors */
  int32_t kv_mode;     /* laga_kv_mode_t */
  int32_t deterministic; /* 1: asks for bitwise-reproducible results. Every kernel of
                            this library is deterministic (no floating-point atomics),
                            so 0 is accepted and changes nothing */
  int32_t dq_mode;     /* laga_dq_mode_t */
} laga_problem_t;

/* Alg. 1 step 4: kv[b,t,:] = c_kv[b,t,:] @ w_kv_b, stored [B,S,H,d_nope+d_v].
 * Accumulates in fp32 over d_c in ascending order; bf16 outputs are rounded to
 * nearest-even. */
LAGA_API laga_status_t laga_reconstruct_kv(const laga_problem_t* p, const void* c_kv,
                                  const void* w_kv_b, void* kv, void* stream);

/* Alg. 1 step 5 for the H heads of the shard: out and lse.
 * kv is required (non-NULL) for MATERIALIZED and ignored for FUSED, which
 * instead reads c_kv and w_kv_b. k_pe is shared by all heads. The workspace
 * must hold laga_workspace_bytes(p, LAGA_OP_FWD) bytes (may be 0 / NULL). */
LAGA_API laga_status_t laga_attn_fwd(const laga_problem_t* p, const void* q,
                            const void* c_kv, const void* k_pe,
                            const void* w_kv_b, const void* kv, void* out,
                            float* lse, void* workspace, size_t workspace_bytes,
                            void* stream);

/* Backward of laga_reconstruct_kv + laga_attn_fwd given dout:
 *   dq = dL/dq (element dtype); dc_kv = dL/dc_kv and dk_pe = dL/dk_pe summed
 *   over this shard's heads (fp32); dw_kv_b = dL/dW_kv_b (fp32). All overwritten.
 *   Deterministic: no floating-point atomics are used.
 * out and lse are the forward's outputs. kv is required for MATERIALIZED; for
 * FUSED it may be NULL and K/V are rebuilt into the workspace. */
LAGA_API laga_status_t laga_attn_bwd(const laga_problem_t* p, const void* q,
                            const void* c_kv, const void* k_pe,
                            const void* w_kv_b, const void* kv, const void* out,
                            const float* lse, const void* dout, void* dq,
                            float* dc_kv, float* dk_pe, float* dw_kv_b,
                            void* workspace, size_t workspace_bytes,
                            void* stream);

/* The backward in its stages; laga_attn_bwd runs all four in this order on one
 * stream. A caller may run them itself (same arguments and workspace for every
 * stage) to put other work between them or to time them one by one:
 *   LAGA_BWD_PREPARE  per-row delta = sum(dout * out) (and the K/V rebuild of
 *                     the FUSED mode when kv is NULL)
 *   LAGA_BWD_DKDV     key-stationary attention backward: dK, dV of every key
 *                     (bf16 with 192/128-wide heads and dq_mode FROM_STORE: also
 *                     stores dS^T of every causal pair, bf16, in the workspace)
 *   LAGA_BWD_DQ       attention backward for dq (with the store: the product
 *                     K^T dS^T over it; otherwise a query-stationary pass that
 *                     recomputes the scores)
 *   LAGA_BWD_FINISH   dk_pe head sum, dc_kv and dw_kv_b up-projection GEMMs
 * Each stage reads what the previous ones left in the workspace. */
typedef enum {
  LAGA_BWD_PREPARE = 0,
  LAGA_BWD_DKDV = 1,
  LAGA_BWD_DQ = 2,
  LAGA_BWD_FINISH = 3
} laga_bwd_stage_t;

LAGA_API laga_status_t laga_attn_bwd_stage(int stage, const laga_problem_t* p,
                                           const void* q, const void* c_kv,
                                           const void* k_pe, const void* w_kv_b,
                                           const void* kv, const void* out,
                                           const float* lse, const void* dout,
                                           void* dq, float* dc_kv, float* dk_pe,
                                           float* dw_kv_b, void* workspace,
                                           size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): laga_attn_bwd without a workspace
 * argument. Same arguments, results and stream semantics as laga_attn_bwd; its
 * workspace is a static device array of LAGA_NOALLOC_SCRATCH_BYTES that the library
 * holds on each GPU it runs on until the process ends (the entry point itself calls no
 * allocator). Limits and behaviour:
 *   - a problem whose laga_workspace_bytes(p, LAGA_OP_BWD) exceeds the array returns
 *     LAGA_ERR_SCRATCH before any launch (e.g. bf16 V3 heads, H = 16: S up to 2048
 *     with dq_mode RECOMPUTE, up to 1024 with FROM_STORE);
 *   - the array belongs to the current device; `stream` (NULL: the default stream) must
 *     be a stream of that device, else LAGA_ERR_DEVICE;
 *   - every call on one GPU uses the same array, and a call leaves its contents behind:
 *     calls that can overlap on one GPU (on different streams, or from different host
 *     threads without ordering) race and must not be issued. */
#define LAGA_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
LAGA_API laga_status_t laga_attn_bwd_noalloc(const laga_problem_t* p, const void* q,
                                             const void* c_kv, const void* k_pe,
                                             const void* w_kv_b, const void* kv, const void* out,
                                             const float* lse, const void* dout, void* dq,
                                             float* dc_kv, float* dk_pe, float* dw_kv_b,
                                             void* stream);

/* ---- Producers around the latent all-gather ---------------------------------
 * The per-token steps that make this block's inputs and consume its gradients
 * (Alg. 1 step 1's latent normalisation; the decoupled RoPE of Section 2.1,
 * property P2, and Section 5.3). Token t of the sequence axis sits at position
 * p = position_offset + t (0 for the gathered sequence; a rank's chunk of S/P
 * tokens starts at r*S/P). R(p) rotates each pair (2i, 2i+1) of a d_rope-wide
 * band counter-clockwise by p * rope_base^(-2i/d_rope):
 * (x0, x1) -> (x0 cos - x1 sin, x0 sin + x1 cos). The problem must be valid as
 * for the attention calls; its softmax_scale, causal and kv_mode are not used. */
typedef struct {
  float eps;               /* added to the mean square, >= 0 (e.g. 1e-6) */
  float rope_base;         /* rotary base, > 1 (e.g. 10000) */
  int64_t position_offset; /* position of token 0, 0 <= offset, offset + S < 2^53 */
} laga_prologue_t;

/* Forward, per token (b, t):
 *   rstd[b,t]  = 1 / sqrt(mean_j latent_raw[b,t,j]^2 + eps)               fp32 [B,S]
 *   c_kv[b,t,j] = latent_raw[b,t,j] * rstd[b,t] * gamma[j]  (gamma NULL: 1) [B,S,d_c]
 *   k_pe[b,t,:] = R(p) kpe_raw[b,t,:]                                      [B,S,d_rope]
 *   q[b,t,h,d_nope:] = R(p) q[b,t,h,d_nope:] for every head, IN PLACE; the
 *                      q_nope columns are left untouched; q may be NULL.
 * latent_raw [B,S,d_c], gamma [d_c], kpe_raw [B,S,d_rope] and q [B,S,H,d_nope+
 * d_rope] are in the element dtype, as are c_kv and k_pe. Statistics in fp32.
 * No workspace. Errors: LAGA_ERR_NULL (problem, cfg or a required pointer),
 * LAGA_ERR_SHAPE (eps < 0, rope_base <= 1, offset out of range, or the problem),
 * LAGA_ERR_ALIGN, LAGA_ERR_UNSUPPORTED (dims as for the attention calls). */
LAGA_API laga_status_t laga_prologue_fwd(const laga_problem_t* p, const laga_prologue_t* cfg,
                                         const void* latent_raw, const void* gamma,
                                         const void* kpe_raw, void* q, void* c_kv,
                                         void* k_pe, float* rstd, void* stream);

/* Backward of laga_prologue_fwd, given the complete fp32 gradients dc_kv [B,S,d_c]
 * and dk_pe [B,S,d_rope] (on one rank with every head: laga_attn_bwd's; across
 * ranks: after the reduce-scatter of Section 5.2) and dq:
 *   d_latent_raw = rstd * (g - y * mean_j(g y)),  y = rstd * latent_raw,
 *                  g = gamma * dc_kv (gamma NULL: dc_kv)                 fp32 [B,S,d_c]
 *   d_gamma[j]   = sum over (b, t) of dc_kv[b,t,j] * y[b,t,j], in a fixed order
 *                  (bitwise repeatable)           fp32 [d_c]; required iff gamma given
 *   d_kpe_raw    = R(p)^T dk_pe                                        fp32 [B,S,d_rope]
 *   dq[b,t,h,d_nope:] = R(p)^T dq[b,t,h,d_nope:], IN PLACE (element dtype); may be NULL.
 * rstd is the forward's. With gamma the workspace must hold
 * laga_workspace_bytes(p, LAGA_OP_PROLOGUE_BWD) bytes (partial sums of d_gamma);
 * without, it may be NULL. Errors as for the forward, plus LAGA_ERR_WORKSPACE. */
LAGA_API laga_status_t laga_prologue_bwd(const laga_problem_t* p, const laga_prologue_t* cfg,
                                         const void* latent_raw, const void* gamma,
                                         const float* rstd, const float* dc_kv,
                                         const float* dk_pe, void* dq, float* d_latent_raw,
                                         float* d_kpe_raw, float* d_gamma, void* workspace,
                                         size_t workspace_bytes, void* stream);

/* ---- Consumer of the block: the output projection (Alg. 1 step 7) -------------
 * After the out all-to-all (Alg. 1 step 6) a rank holds the attention output of every
 * head for its tokens; step 7 returns W_o(reshape(out)):
 *   out  [T, n_heads, d_v]    element dtype (head-major: feature f = h * d_v + e)
 *   w_o  [F, d_model]         element dtype, F = n_heads * d_v (in x out)
 *   y    [T, d_model]         element dtype:  y = reshape(out) @ w_o
 * and its backward given dy [T, d_model] (element dtype):
 *   d_out [T, n_heads, d_v]   element dtype:  d_out = dy @ w_o^T
 *   dw_o  [F, d_model]        fp32:           dw_o = reshape(out)^T @ dy (over all T tokens,
 *                             in a fixed order: bitwise repeatable)
 * fp32 accumulation throughout. T is whatever rows the caller has: a rank's S/P tokens
 * after the all-to-all, or B*S on one rank. Validation as for the attention calls: NULL
 * problem or pointer -> LAGA_ERR_NULL; a non-positive size -> LAGA_ERR_SHAPE; F or d_model
 * not a multiple of 16, an unknown dtype, reserved != 0, or T*F, T*d_model or F*d_model
 * not below 2^31 -> LAGA_ERR_UNSUPPORTED; misaligned -> LAGA_ERR_ALIGN; workspace smaller
 * than laga_out_proj_workspace_bytes() -> LAGA_ERR_WORKSPACE. */
typedef struct {
  int64_t tokens;  /* T */
  int64_t n_heads; /* every head of the layer */
  int64_t d_v;
  int64_t d_model; /* D */
  int32_t dtype;   /* laga_dtype_t */
  int32_t reserved; /* must be 0 */
} laga_out_proj_t;

LAGA_API laga_status_t laga_out_proj_fwd(const laga_out_proj_t* p, const void* out, const void* w_o,
                                         void* y, void* stream);
LAGA_API laga_status_t laga_out_proj_bwd(const laga_out_proj_t* p, const void* out, const void* w_o,
                                         const void* dy, void* d_out, float* dw_o, void* workspace,
                                         size_t workspace_bytes, void* stream);
/* Workspace of laga_out_proj_bwd (partial sums of dw_o over token ranges); 0 if none is
 * needed or p is invalid. */
LAGA_API size_t laga_out_proj_workspace_bytes(const laga_out_proj_t* p);

/* Workspace bytes that op (laga_op_t) needs for problem p; 0 if none or if p
 * is invalid (check with the entry point itself for the error code). For the
 * backward in bf16 with 192/128-wide heads and dq_mode FROM_STORE this includes the
 * dS^T store: 2 * B * H * 512 * T * (T + 1) bytes with the causal mask
 * (2 * B * H * 1024 * T^2 without), T = ceil(S / 32) -- about 4.3 GB at S = 16384,
 * H = 16. With dq_mode RECOMPUTE the backward workspace is linear in S. */
LAGA_API size_t laga_workspace_bytes(const laga_problem_t* p, int op);

/* Static, never-NULL description of a status code. */
LAGA_API const char* laga_status_string(laga_status_t s);

/* LAGA_ABI_VERSION of the built library. */
LAGA_API int laga_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* LAGA_H_ */
