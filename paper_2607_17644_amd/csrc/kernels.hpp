// Host-side launchers of the gfx950 kernels (all enqueue on the given stream).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include "common.hpp"

namespace laga {

// Per-row backward statistics (delta, lse2) are stored with rows padded to a
// multiple of this many queries, so query tiles can be fetched whole.
constexpr int kRowPad = 64;

// Tokens per split of the dW reduction over tokens: a function of the token count only
// (never of the head count), so each dW column is bit-identical whatever head shard
// computes it. 2048 for long sequences, down to 512 for short ones (enough workgroups).
int dw_split_tokens(int tokens);
size_t dw_split_count(int tokens);
// Splits of the dc_kv GEMM's contraction (over the shard's heads x 256), chosen so that
// the launch has enough workgroups; dc_kv sums over heads, so no bit-identity across
// head shards is asked of it. Partials of both GEMMs share one workspace buffer.
int dc_split_count(int tokens, int d_c, int K);
size_t gemm_partial_elems(int tokens, int d_c, int K);

template <typename T>
hipError_t launch_reconstruct(const T* c, const T* w, T* kv, int M, int N, int K, hipStream_t st);
// dkv_lo (may be NULL): low bf16 halves of dKV, so that dKV = dkv + dkv_lo to ~16 bits.
// partial: workspace of gemm_partial_elems floats (used when the contraction is split).
template <typename T>
hipError_t launch_dc(const T* dkv, const T* dkv_lo, const T* w, float* dc, float* partial, int M, int N, int K,
                     hipStream_t st);
template <typename T>
hipError_t launch_dw(const T* c, const T* dkv, const T* dkv_lo, float* dw, float* partial, int M, int N, int K,
                     hipStream_t st);

// Plain GEMMs of the output projection (Alg. 1 step 7) on the same kernels:
//   gemm_nt: c[M][N] = a[M][K] @ w^T, w stored [N][K]; element-dtype output
//   gemm_tn: c[M][N] = a^T @ b, a stored [K][M], b [K][N]; fp32 output, contraction split
//            into nsplit ranges (partial: nsplit * M * N floats when nsplit > 1) summed in
//            ascending order
template <typename T>
hipError_t launch_gemm_nt(const T* a, const T* w, T* c, int M, int N, int K, hipStream_t st);
template <typename T>
hipError_t launch_gemm_tn(const T* a, const T* b, float* c, float* partial, int M, int N, int K, int nsplit,
                          hipStream_t st);
// contraction splits gemm_tn is given for an M x N output over K (element size esize):
// enough workgroups for the GPU, each split at least 512 indices; a function of the shape only
int gemm_tn_splits(int M, int N, int K, int esize);

struct AttnFwdArgs {
  const void* q;      // [B,S,H,DN+DR]
  const void* k_pe;   // [B,S,DR]
  const void* kv;     // [B,S,H,DN+DV] (materialised path)
  const void* c_kv;   // [B,S,d_c]     (fused path)
  const void* w;      // [d_c, H*(DN+DV)] W_kv_b (fused path)
  void* out;          // [B,S,H,DV]
  float* lse;         // [B,H,S]
  int B, S, H, d_c;
  float scale;
  int causal;
};

// Online softmax of the forward kernels: the running reference max is only raised
// when a new score exceeds it by more than this (log2 units), so unnormalised
// probabilities stay <= 2^kRescaleLog2 and the O^T rescale is rare.
constexpr float kRescaleLog2 = 8.f;

template <typename T, int DN, int DR, int DV>
hipError_t launch_attn_fwd(const AttnFwdArgs& a, hipStream_t st);

// Fused forward: K/V rebuilt tile by tile from c_kv; w_t_ws receives W_kv_b^T in the
// MFMA fragment order (H*(DN+DV) x d_c elements) first. d_c <= kFusedMaxDc.
constexpr int kFusedMaxDc = 512;
// W_kv_b^T (w [K = d_c, N]) in MFMA A-fragment order with the rows of each 32-row block
// in the order pi (bits 2 and 3 swapped), for the backward's on-chip K/V rebuilds: the
// fragment of row block cb and contraction step ks is the 512 elements at
// (cb * (K / 16) + ks) * 512, lane l = 32 g + n holding row 32 cb + pi(n), elements
// 16 ks + 8 g .. + 7.
template <typename T>
hipError_t launch_frag_w_pi(const T* w, T* w_t, int K, int N, hipStream_t st);
template <typename T, int DN, int DR, int DV>
hipError_t launch_attn_fwd_fused(const AttnFwdArgs& a, void* w_t_ws, hipStream_t st);

struct AttnBwdArgs {
  const void* q;
  const void* k_pe;
  const void* kv;    // [B,S,H,DN+DV]
  const void* out;
  const void* dout;
  const float* lse;
  void* dq;          // [B,S,H,DN+DR]
  float* dk_pe;      // [B,S,DR] fp32
  float* delta;      // workspace [B*H][S_pad]
  float* lse2;       // workspace [B*H][S_pad]: lse * log2(e)
  int S_pad;         // S rounded up to kRowPad
  void* dkv;         // workspace [B,S,H,DN+DV]
  void* dkv_lo;      // workspace [B,S,H,DN+DV], bf16 only: dKV - bf16(dKV) rounded to bf16
  float* dkpe_h;     // workspace [B,S,H,DR]
  void* ds;          // workspace: dS^T store (bf16 path with 192/128-wide heads), else unused
  const void* c_kv;  // [B,S,d_c]: with w_t, the latent K/V are rebuilt from (kv unused)
  const void* w_t;   // W_kv_b^T [H*(DN+DV), d_c] (workspace), or NULL: K/V read from kv
  int d_c;
  int B, S, H;
  float scale;
  int causal;
};

namespace bwd { struct BwdParams; }
template <typename T, int DN, int DR, int DV>
hipError_t launch_bwd_dq(bwd::BwdParams P, int B, hipStream_t st);
// the generic key-stationary dK/dV kernel (attn_bwd_kv.hip)
template <typename T, int DN, int DR, int DV>
hipError_t launch_dkdv_generic(bwd::BwdParams P, int B, hipStream_t st);

// stage 0: delta; 1: dK/dV (into dkv, dkpe_h); 2: dQ; 3: dk_pe head sum.
// (dc_kv / dW are the GEMMs above.)
template <typename T, int DN, int DR, int DV>
hipError_t launch_attn_bwd(const AttnBwdArgs& a, int stage, hipStream_t st);

// Producers around the latent all-gather (latent normalisation, decoupled RoPE).
struct PrologueArgs {
  const void* latent_raw;  // [B,S,d_c] element dtype
  const void* gamma;       // [d_c] element dtype, or NULL
  const void* kpe_raw;     // forward: [B,S,d_rope]
  void* q;                 // forward: q, backward: dq ([B,S,H,d_qk]); rope band rotated in place; or NULL
  void* c_kv;              // forward output [B,S,d_c]
  void* k_pe;              // forward output [B,S,d_rope]
  float* rstd;             // forward output [B,S]
  const float* rstd_in;    // backward input [B,S]
  const float* dc_kv;      // backward input [B,S,d_c]
  const float* dk_pe;      // backward input [B,S,d_rope]
  float* d_latent;         // backward output [B,S,d_c]
  float* d_kpe;            // backward output [B,S,d_rope]
  float* d_gamma;          // backward output [d_c] (with gamma)
  float* partial;          // backward workspace [prologue_bwd_rows + prologue_sum_groups][d_c] (with gamma), else NULL
  int B, S, H, d_c, d_nope, d_rope, d_qk;
  int64_t position_offset;
  float eps;
  double log2_base;
};
// rows of d_gamma partial sums the backward writes for `tokens` tokens
int prologue_bwd_rows(long long tokens);
// row groups of the fixed-order column sum of those rows
int prologue_sum_groups(long long tokens);
template <typename T>
hipError_t launch_prologue_fwd(const PrologueArgs& a, hipStream_t st);
template <typename T>
hipError_t launch_prologue_bwd(const PrologueArgs& a, hipStream_t st);

}  // namespace laga
