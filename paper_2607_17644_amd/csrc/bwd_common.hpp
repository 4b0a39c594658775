// Declarations shared by the backward kernels (attn_bwd.hip, attn_bwd_dq.hip).
#pragma once
#include "common.hpp"

namespace laga {
namespace bwd {

// LDS row pitch (elements) of a tile read both with 16-byte row fragments and
// with transposing reads: for 16-bit types the pitch in dwords is chosen
// = 12, 28, 36 or 52 (mod 64) so that neither access pattern has bank
// conflicts; fp32 rows are padded to stay 32-byte aligned.
template <typename T>
constexpr int lds_pitch(int cols) {
  if (sizeof(T) == 4) return cols + 8;
  for (int pad = 8; pad < 136; pad += 16) {
    const int dw = ((cols + pad) / 2) % 64;
    if (dw == 12 || dw == 28 || dw == 36 || dw == 52) return cols + pad;
  }
  return cols + 8;
}

constexpr int round32(int x) { return (x + 31) / 32 * 32; }

struct BwdParams {
  const void* q;
  const void* k_pe;
  const void* kv;
  const void* dout;
  const float* lse;
  const float* delta;  // [B*H][S_pad]
  const float* lse2;   // [B*H][S_pad], lse * log2(e)
  int S_pad;
  void* dq;
  void* dkv;       // [B,S,H,DN+DV] element dtype
  void* dkv_lo;    // [B,S,H,DN+DV] bf16 low halves (bf16 only; else unused)
  float* dkpe_h;   // [B,S,H,DR] fp32
  int S, H, n_blocks;
  float scale, scale_log2;
  int causal;
  // dS^T store (bf16 path with 192/128-wide heads): written by the key-stationary
  // pass, read by the dQ pass; see ds_tile_offset. ds_T = ceil(S / 32).
  void* ds;
  int ds_T;
  // K/V rebuilt on chip (kv_mode FUSED, bf16 with 192/128-wide heads): kv is unused and
  // each key's K_nope / V rows come from c_kv [B,S,d_c] and w_t = W_kv_b^T [H*(DN+DV), d_c]
  const void* c_kv;
  const void* w_t;
  int d_c;
};

// dS^T store layout: for every (b, h) and query tile t of 32 rows, the keys that tile
// sees (32 (t + 1) with the causal mask, 32 T without) as rows of 32 bf16 values, one
// per query of the tile (key-major, 64-byte rows). Keys past S hold zeros. Within a row,
// query 8j + 4g + e (j < 4, g < 2, e < 4) sits at position 16g + 4j + e: the 16 queries
// one lane of the dK/dV kernel holds in its accumulator (column layout of the 32x32
// MFMA) are contiguous, so it writes them as two 16-byte stores.
__host__ __device__ constexpr int ds_query_of_position(int pos) {
  return 8 * ((pos >> 2) & 3) + 4 * (pos >> 4) + (pos & 3);
}
__host__ __device__ inline size_t ds_head_elems(int T, int causal) {
  return causal ? (size_t)512 * T * (T + 1) : (size_t)1024 * T * T;
}
__host__ __device__ inline size_t ds_tile_offset(int T, int causal, int bh, int t) {
  return (size_t)bh * ds_head_elems(T, causal) + (causal ? (size_t)512 * t * (t + 1) : (size_t)1024 * T * t);
}
__host__ __device__ inline int ds_tile_keys(int T, int causal, int t) { return causal ? 32 * (t + 1) : 32 * T; }

template <typename T> struct BwdTiles;
template <> struct BwdTiles<bf16> { static constexpr int BQ = 32, BC = 64, WPH_KV = 4, WPH_Q = 4; };
template <> struct BwdTiles<float> { static constexpr int BQ = 32, BC = 32, WPH_KV = 4, WPH_Q = 4; };


}  // namespace bwd
}  // namespace laga
