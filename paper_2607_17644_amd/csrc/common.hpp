// Device helpers shared by the gfx950 kernels: element types, 8-element MFMA
// fragments, the 32x32 MFMA wrappers, LDS fragment reads and bf16 rounding.
//
// Fragment convention (all kernels): a 32x32 output block contracted over 16
// indices uses one "fragment" of 8 elements per lane for each operand. Lane l
// serves row/column (l % 32) of its operand and the contraction indices of
// half g = l / 32. For bf16 that is one v_mfma_f32_32x32x16_bf16; for fp32 it
// is eight v_mfma_f32_32x32x2_f32, the t-th taking element t of each fragment.
// The 16 accumulators of a lane hold the output column (l % 32) at rows
// (r / 4) * 8 + g * 4 + (r % 4), r = 0..15.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace laga {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(8 * sizeof(float)))) float f32x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(short)))) short i16x4;

template <typename T> struct FragOf;
template <> struct FragOf<bf16> { using type = bf16x8; using half = bf16x4; };
template <> struct FragOf<float> { using type = f32x8; using half = f32x4; };
template <typename T> using frag_t = typename FragOf<T>::type;

__device__ __forceinline__ void mma(f32x16& acc, const bf16x8& a, const bf16x8& b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma(f32x16& acc, const f32x8& a, const f32x8& b) {
#pragma unroll
  for (int t = 0; t < 8; ++t) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[t], b[t], acc, 0, 0, 0);
}

template <typename T> __device__ __forceinline__ T to_elem(float x);
template <> __device__ __forceinline__ bf16 to_elem<bf16>(float x) { return (bf16)x; }  // RNE
template <> __device__ __forceinline__ float to_elem<float>(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }
__device__ __forceinline__ float to_f32(float x) { return x; }

// 16-byte vector of elements used for global<->LDS staging (8 bf16 or 4 fp32).
typedef __attribute__((__vector_size__(16))) int chunk16;
template <typename T> struct Elems16 { static constexpr int n = 16 / sizeof(T); };

// Fragment of 8 contiguous elements from LDS (row-major, contraction along the row).
template <typename T>
__device__ __forceinline__ frag_t<T> lds_frag(const T* p) {
  return *reinterpret_cast<const frag_t<T>*>(p);
}

// Fragment whose 8 contraction indices run down a column of a row-major LDS
// tile X (pitch in elements): lane l returns X[ra + e][c] for e = 0..3 and
// X[rb + e][c] for e = 0..3, with c = c0 + (l % 32). ra and rb are per lane
// (they may depend on l / 32). For bf16 this uses ds_read_b64_tr_b16: each
// 16-lane group reads a 4 x 16 block, lane s of the group pointing at row
// (r + s / 4) and columns (4 * (s % 4)) .. +3 of the group's 16 columns.
template <typename T> struct TrRead;
template <> struct TrRead<bf16> {
  static __device__ __forceinline__ bf16x8 get(const bf16* X, int pitch, int ra, int rb, int c0) {
    const int l = threadIdx.x & 63;
    const int s = l & 15;
    const int col = c0 + 16 * ((l >> 4) & 1) + 4 * (s & 3);
    typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
    const bf16* pa = X + (ra + (s >> 2)) * pitch + col;
    const bf16* pb = X + (rb + (s >> 2)) * pitch + col;
    bf16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(pa));
    bf16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(pb));
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  }
};
template <> struct TrRead<float> {
  static __device__ __forceinline__ f32x8 get(const float* X, int pitch, int ra, int rb, int c0) {
    const int c = c0 + (threadIdx.x & 31);
    f32x8 f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[e] = X[(ra + e) * pitch + c];
      f[4 + e] = X[(rb + e) * pitch + c];
    }
    return f;
  }
};

// Accumulator rows r -> 8-element fragment used as the next MFMA's operand:
// rows 8*half .. 8*half+7 of the 16, i.e. for the 16 contraction indices
// 16*kk .. 16*kk+15 covered by accumulator block (kk / 2), half = kk % 2, the
// lane supplies indices {g*4 + e, 8 + g*4 + e} (e = 0..3) of that group of 16.
// Operands read with TrRead(ra = 16*kk + 4*g, rb = ra + 8) match this order.
template <typename T>
__device__ __forceinline__ frag_t<T> acc_to_frag(const f32x16& acc, int half) {
  frag_t<T> f;
#pragma unroll
  for (int e = 0; e < 8; ++e) f[e] = to_elem<T>(acc[8 * half + e]);
  return f;
}

__device__ __forceinline__ float wave_xor32_max(float x) {
  return fmaxf(x, __shfl_xor(x, 32));
}
__device__ __forceinline__ float wave_xor32_sum(float x) {
  return x + __shfl_xor(x, 32);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// Direct global -> LDS copy of 16 bytes per lane (gfx950 global_load_lds_dwordx4):
// lane l's 16 bytes from `g` land at LDS address lds + 16 * l, where `lds` must be
// the same for every lane of the wave. Tracked by vmcnt like any global load.
__device__ __forceinline__ void g2lds16(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(g, lds, 16, 0, 0);
}

// Wait until all of this wave's outstanding vector-memory loads (including direct
// global -> LDS copies) have completed.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0); }

// Zero value of a 16-byte staging chunk.
__device__ __forceinline__ chunk16 zero_chunk() { chunk16 z = {0, 0, 0, 0}; return z; }

// XCD-aware ordering of a 1-D grid: the hardware deals consecutive workgroup
// ids round-robin over the 8 XCDs; this returns a "logical" id such that each
// XCD receives a contiguous range of logical ids (so work that shares data —
// same head, same tiles — lands on the same XCD and its L2). Needs n % 8 == 0
// to be a permutation; otherwise returns id unchanged.
__device__ __forceinline__ int xcd_remap(int id, int n) {
  constexpr int kXcd = 8;
  if (n % kXcd) return id;
  return (id % kXcd) * (n / kXcd) + id / kXcd;
}

}  // namespace laga
