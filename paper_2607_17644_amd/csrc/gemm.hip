// MFMA GEMMs of the up-projection and its backward (gfx950).
//
//   reconstruct : kv[B*S, H*(d_nope+d_v)] = c_kv[B*S, d_c] @ W_kv_b     (Alg. 1 step 4)
//   dc          : dc_kv[B*S, d_c] = dKV[B*S, H*(d_nope+d_v)] @ W_kv_b^T   (fp32 out)
//   dW          : dW[d_c, H*(d_nope+d_v)] = c_kv^T @ dKV  (split over tokens,
//                 fixed-order reduction: deterministic)
//
// One kernel template covers all three: each operand is either "k-contiguous"
// (stored [rows][K]) or "k-strided" (stored [K][rows]); both are staged into
// LDS as stored and strided operands are read back with transposing LDS reads,
// so there is no transpose pass anywhere. The output tile is computed as
// C^T = B^T A^T block by block, which puts 4 consecutive output columns in each
// lane's accumulators for vectorised stores.
//
// Per output element the contraction runs over K in ascending 16-wide steps
// (one MFMA each) with fp32 accumulation; tile shapes and the dW token split do
// not depend on N, so a column of the output is bit-identical whatever N (the
// number of heads) is. (dc_kv's contraction runs over the heads and may be split
// into partials summed in a fixed order.)
#include "common.hpp"
#include "kernels.hpp"

namespace laga {

namespace {

constexpr int kThreads = 256;

template <typename T, bool KSTRIDED, int ROWS, int BK>
struct OperandTile {
  static constexpr int E = Elems16<T>::n;                      // elements per 16-byte chunk
  // k-contiguous rows: +8 elements keeps 16-byte fragment reads conflict-free and
  // fp32 rows 32-byte aligned; k-strided rows: +32 bytes for the transposing reads.
  static constexpr int PITCH = KSTRIDED ? ROWS + 32 / (int)sizeof(T) : BK + 8;
  static constexpr int LDS_ELEMS = KSTRIDED ? BK * PITCH : ROWS * PITCH;
  static constexpr int CHUNKS = ROWS * BK / E;
  static constexpr int PER_THREAD = CHUNKS / kThreads;
  static_assert(CHUNKS % kThreads == 0, "tile must split evenly over the workgroup");

  chunk16 reg[PER_THREAD];

  // Global -> registers. rows [r0, r_end) valid, k [k0, k_end) valid; zero fill outside.
  __device__ __forceinline__ void load(const T* __restrict__ g, int ld, int r0, int r_end, int k0, int k_end) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int c = tid + i * kThreads;
      int r, k;
      if (!KSTRIDED) { r = c / (BK / E); k = (c % (BK / E)) * E; }
      else { k = c / (ROWS / E); r = (c % (ROWS / E)) * E; }
      const int gr = r0 + r, gk = k0 + k;
      const bool ok = (gr < r_end) && (gk < k_end);
      const T* src = KSTRIDED ? g + (size_t)gk * ld + gr : g + (size_t)gr * ld + gk;
      reg[i] = ok ? *reinterpret_cast<const chunk16*>(src) : zero_chunk();
    }
  }
  __device__ __forceinline__ void store(T* s) const {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int c = tid + i * kThreads;
      int r, k;
      if (!KSTRIDED) { r = c / (BK / E); k = (c % (BK / E)) * E; }
      else { k = c / (ROWS / E); r = (c % (ROWS / E)) * E; }
      T* dst = KSTRIDED ? s + k * PITCH + r : s + r * PITCH + k;
      *reinterpret_cast<chunk16*>(dst) = reg[i];
    }
  }
  // Fragment for the 32-row block starting at rb, contraction step ks.
  static __device__ __forceinline__ frag_t<T> frag(const T* s, int rb, int ks) {
    const int l = threadIdx.x & 63, g = l >> 5;
    if (!KSTRIDED) return lds_frag<T>(s + (rb + (l & 31)) * PITCH + ks * 16 + 8 * g);
    const int ra = ks * 16 + 8 * g;
    return TrRead<T>::get(s, PITCH, ra, ra + 4, rb);
  }
};

template <typename TO>
__device__ __forceinline__ void store4(TO* p, float a, float b, float c, float d);
template <>
__device__ __forceinline__ void store4<float>(float* p, float a, float b, float c, float d) {
  f32x4 v = {a, b, c, d};
  *reinterpret_cast<f32x4*>(p) = v;
}
template <>
__device__ __forceinline__ void store4<bf16>(bf16* p, float a, float b, float c, float d) {
  bf16x4 v = {(bf16)a, (bf16)b, (bf16)c, (bf16)d};
  *reinterpret_cast<bf16x4*>(p) = v;
}

// C (+ blockIdx.z * split_stride) [M][N] = A[M][K-range] B[K-range][N]
// SPLIT = 1: A is the sum of two arrays A + A2 of the same layout; SPLIT = 2: B = B + B2.
// (A value held as a bf16 pair hi + lo keeps ~16 significant bits through a bf16 MFMA;
// per k-step the hi product is accumulated before the lo product.)
template <typename T, typename TO, bool A_KS, bool B_KS, int BM, int BN, int BK, int SPLIT>
__global__ __launch_bounds__(kThreads) void gemm_kernel(
    const T* __restrict__ A, const T* __restrict__ B, const T* __restrict__ X2, TO* __restrict__ C,
    int M, int N, int K, int lda, int ldb, int ldc, int k_chunk, long long split_stride) {
  using TA = OperandTile<T, A_KS, BM, BK>;
  using TB = OperandTile<T, B_KS, BN, BK>;
  constexpr int WM = BM / 64, WN = BN / 64;  // 32x32 blocks per wave along m and n
  constexpr int A2_ELEMS = SPLIT == 1 ? TA::LDS_ELEMS : 1;
  constexpr int B2_ELEMS = SPLIT == 2 ? TB::LDS_ELEMS : 1;
  __shared__ __attribute__((aligned(16))) T sA[TA::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) T sB[TB::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) T sA2[A2_ELEMS];
  __shared__ __attribute__((aligned(16))) T sB2[B2_ELEMS];

  const int n_tiles = (N + BN - 1) / BN;
  const int m_tiles = (M + BM - 1) / BM;
  const int lin = xcd_remap(blockIdx.x, n_tiles * m_tiles);
  const int tn = lin % n_tiles, tm = lin / n_tiles;
  const int m0 = tm * BM, n0 = tn * BN;
  const int kb = blockIdx.z * k_chunk;
  const int ke = min(K, kb + k_chunk);

  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63, g = l >> 5;
  const int wm = wave & 1, wn = wave >> 1;

  f32x16 acc[WN][WM];
#pragma unroll
  for (int j = 0; j < WN; ++j)
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[j][i][r] = 0.f;

  TA ta, ta2; TB tb, tb2;
  auto load = [&](int k0) {
    ta.load(A, lda, m0, M, k0, ke);
    tb.load(B, ldb, n0, N, k0, ke);
    if (SPLIT == 1) ta2.load(X2, lda, m0, M, k0, ke);
    if (SPLIT == 2) tb2.load(X2, ldb, n0, N, k0, ke);
  };
  auto store = [&]() {
    ta.store(sA); tb.store(sB);
    if (SPLIT == 1) ta2.store(sA2);
    if (SPLIT == 2) tb2.store(sB2);
  };
  load(kb);
  store();
  __syncthreads();
  for (int k0 = kb; k0 < ke; k0 += BK) {
    const bool more = k0 + BK < ke;
    if (more) load(k0 + BK);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      frag_t<T> fa[WM], fb[WN];
#pragma unroll
      for (int i = 0; i < WM; ++i) fa[i] = TA::frag(sA, (wm * WM + i) * 32, ks);
#pragma unroll
      for (int j = 0; j < WN; ++j) fb[j] = TB::frag(sB, (wn * WN + j) * 32, ks);
      if (SPLIT == 0) {
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
          for (int i = 0; i < WM; ++i) mma(acc[j][i], fb[j], fa[i]);
      } else if (SPLIT == 1) {
        frag_t<T> fa2[WM];
#pragma unroll
        for (int i = 0; i < WM; ++i) fa2[i] = TA::frag(sA2, (wm * WM + i) * 32, ks);
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
          for (int i = 0; i < WM; ++i) { mma(acc[j][i], fb[j], fa[i]); mma(acc[j][i], fb[j], fa2[i]); }
      } else {
        frag_t<T> fb2[WN];
#pragma unroll
        for (int j = 0; j < WN; ++j) fb2[j] = TB::frag(sB2, (wn * WN + j) * 32, ks);
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
          for (int i = 0; i < WM; ++i) { mma(acc[j][i], fb[j], fa[i]); mma(acc[j][i], fb2[j], fa[i]); }
      }
    }
    __syncthreads();
    if (more) { store(); __syncthreads(); }
  }

  TO* Cz = C + blockIdx.z * split_stride;
#pragma unroll
  for (int j = 0; j < WN; ++j)
#pragma unroll
    for (int i = 0; i < WM; ++i) {
      const int m = m0 + (wm * WM + i) * 32 + (l & 31);
      if (m >= M) continue;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int n = n0 + (wn * WN + j) * 32 + rr * 8 + g * 4;
        if (n < N)
          store4<TO>(Cz + (size_t)m * ldc + n, acc[j][i][4 * rr], acc[j][i][4 * rr + 1],
                     acc[j][i][4 * rr + 2], acc[j][i][4 * rr + 3]);
      }
    }
}

// dst[i] = sum_{s < nsplit} src[s * stride + i], in ascending s (float4 granularity).
__global__ __launch_bounds__(256) void split_reduce_kernel(const float* __restrict__ src, float* __restrict__ dst,
                                                           long long n4, int nsplit, long long stride) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  f32x4 s = reinterpret_cast<const f32x4*>(src)[i];
  for (int k = 1; k < nsplit; ++k) {
    f32x4 v = reinterpret_cast<const f32x4*>(src + k * stride)[i];
    s += v;
  }
  reinterpret_cast<f32x4*>(dst)[i] = s;
}

template <typename T> struct GemmCfg;
template <> struct GemmCfg<bf16> { static constexpr int BM = 128, BN = 128, BK = 32; };
template <> struct GemmCfg<float> { static constexpr int BM = 64, BN = 64, BK = 16; };

inline int grid_tiles(int M, int N, int BM, int BN) { return ((M + BM - 1) / BM) * ((N + BN - 1) / BN); }

}  // namespace

template <typename T>
hipError_t launch_reconstruct(const T* c, const T* w, T* kv, int M, int N, int K, hipStream_t st) {
  using G = GemmCfg<T>;
  dim3 grid(grid_tiles(M, N, G::BM, G::BN), 1, 1);
  gemm_kernel<T, T, false, true, G::BM, G::BN, G::BK, 0><<<grid, kThreads, 0, st>>>(
      c, w, nullptr, kv, M, N, K, /*lda=*/K, /*ldb=*/N, /*ldc=*/N, /*k_chunk=*/K, 0);
  return hipGetLastError();
}

namespace {
constexpr int kMinGemmBlocks = 512;  // workgroups wanted per GEMM launch (256 CUs)
}  // namespace

int dw_split_tokens(int tokens) {
  int s = 2048;
  while (s > 512 && (tokens + s - 1) / s < 4) s /= 2;
  return s;
}
size_t dw_split_count(int tokens) {
  const int s = dw_split_tokens(tokens);
  return (size_t)((tokens + s - 1) / s);
}
int dc_split_count(int tokens, int d_c, int K) {
  const int tiles = grid_tiles(tokens, d_c, GemmCfg<bf16>::BM, GemmCfg<bf16>::BN);
  const int max_split = K / 256;  // at least one head (256 contraction indices) per split
  int n = (kMinGemmBlocks + tiles - 1) / tiles;
  return n < 1 ? 1 : (n > max_split ? max_split : n);
}
size_t gemm_partial_elems(int tokens, int d_c, int K) {
  const size_t dw = dw_split_count(tokens) > 1 ? dw_split_count(tokens) * (size_t)d_c * K : 0;
  const int ndc = dc_split_count(tokens, d_c, K);
  const size_t dc = ndc > 1 ? (size_t)ndc * tokens * d_c : 0;
  return dw > dc ? dw : dc;
}

template <typename T>
hipError_t launch_dc(const T* dkv, const T* dkv_lo, const T* w, float* dc, float* partial, int M, int N, int K,
                     hipStream_t st) {
  // dc[M=tokens][N=d_c] = (dKV + dKV_lo)[M][K=H*dkvh] @ W^T ; W stored [N][K] (k-contiguous).
  // With a split contraction each split writes its partial and a fixed-order reduce sums them.
  using G = GemmCfg<T>;
  const int nsplit = sizeof(T) == 2 ? dc_split_count(M, N, K) : 1;
  const int k_chunk = (K / nsplit + G::BK - 1) / G::BK * G::BK;
  const int nz = (K + k_chunk - 1) / k_chunk;
  float* target = nz == 1 ? dc : partial;
  dim3 grid(grid_tiles(M, N, G::BM, G::BN), 1, nz);
  if (dkv_lo)
    gemm_kernel<T, float, false, false, G::BM, G::BN, G::BK, 1><<<grid, kThreads, 0, st>>>(
        dkv, w, dkv_lo, target, M, N, K, K, K, N, k_chunk, (long long)M * N);
  else
    gemm_kernel<T, float, false, false, G::BM, G::BN, G::BK, 0><<<grid, kThreads, 0, st>>>(
        dkv, w, nullptr, target, M, N, K, K, K, N, k_chunk, (long long)M * N);
  if (nz > 1) {
    const long long n4 = (long long)M * N / 4;
    split_reduce_kernel<<<(unsigned)((n4 + 255) / 256), 256, 0, st>>>(partial, dc, n4, nz, (long long)M * N);
  }
  return hipGetLastError();
}

template <typename T>
hipError_t launch_dw(const T* c, const T* dkv, const T* dkv_lo, float* dw, float* partial, int M, int N, int K,
                     hipStream_t st) {
  // dW[M=d_c][N=H*dkvh] = c^T @ (dKV + dKV_lo); c stored [K=tokens][M] and dKV [K][N]: both k-strided.
  using G = GemmCfg<T>;
  const int split = dw_split_tokens(K);
  const int nsplit = (int)dw_split_count(K);
  float* target = nsplit == 1 ? dw : partial;
  dim3 grid(grid_tiles(M, N, G::BM, G::BN), 1, nsplit);
  if (dkv_lo)
    gemm_kernel<T, float, true, true, G::BM, G::BN, G::BK, 2><<<grid, kThreads, 0, st>>>(
        c, dkv, dkv_lo, target, M, N, K, M, N, N, split, (long long)M * N);
  else
    gemm_kernel<T, float, true, true, G::BM, G::BN, G::BK, 0><<<grid, kThreads, 0, st>>>(
        c, dkv, nullptr, target, M, N, K, M, N, N, split, (long long)M * N);
  if (nsplit > 1) {
    const long long n4 = (long long)M * N / 4;
    split_reduce_kernel<<<(unsigned)((n4 + 255) / 256), 256, 0, st>>>(partial, dw, n4, nsplit, (long long)M * N);
  }
  return hipGetLastError();
}

template hipError_t launch_reconstruct<bf16>(const bf16*, const bf16*, bf16*, int, int, int, hipStream_t);
template hipError_t launch_reconstruct<float>(const float*, const float*, float*, int, int, int, hipStream_t);
template hipError_t launch_dc<bf16>(const bf16*, const bf16*, const bf16*, float*, float*, int, int, int, hipStream_t);
template hipError_t launch_dc<float>(const float*, const float*, const float*, float*, float*, int, int, int,
                                     hipStream_t);
template hipError_t launch_dw<bf16>(const bf16*, const bf16*, const bf16*, float*, float*, int, int, int, hipStream_t);
template hipError_t launch_dw<float>(const float*, const float*, const float*, float*, float*, int, int, int,
                                     hipStream_t);

}  // namespace laga
