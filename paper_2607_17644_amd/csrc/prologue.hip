// Per-token producers on either side of the latent all-gather, forward and backward:
// the latent normalisation of Alg. 1 step 1 (weight-optional RMS form) and the
// decoupled rotary embedding of the shared k_pe band and of every head's q_rope band
// (Section 2.1, property P2; Section 5.3). HBM-bound: each element is read and
// written once, one wave per token.
//
// Rotation of pair i (elements 2i, 2i+1 of a band d_rope wide) at position p: by the
// angle p * base^(-2i/d_rope), counter-clockwise ((x0, x1) -> (x0 c - x1 s, x0 s + x1 c));
// the backward applies the transpose. The angle is formed and reduced modulo 2 pi in
// double precision, then its sine and cosine are taken in single precision on the
// reduced angle (|a| <= pi), so positions far beyond 2^24 keep full accuracy.
#include <math.h>
#include <stdint.h>

#include "kernels.hpp"

namespace laga {
namespace {

constexpr int kWaves = 4;         // waves per workgroup
constexpr int kBwdTokPerWave = 4;  // tokens per wave in the backward (d_gamma partial rows)
constexpr int kMaxChunks = 2;      // 8-element chunks of the latent row per lane: d_c <= 1024

template <typename T> struct V8;
template <> struct V8<bf16> {
  static __device__ __forceinline__ void load(const bf16* p, float (&v)[8]) {
    const bf16x8 x = *reinterpret_cast<const bf16x8*>(p);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (float)x[e];
  }
  static __device__ __forceinline__ void store(bf16* p, const float (&v)[8]) {
    bf16x8 x;
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = (bf16)v[e];  // round to nearest even
    *reinterpret_cast<bf16x8*>(p) = x;
  }
};
template <> struct V8<float> {
  static __device__ __forceinline__ void load(const float* p, float (&v)[8]) {
    const f32x4 a = *reinterpret_cast<const f32x4*>(p), b = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) { v[e] = a[e]; v[4 + e] = b[e]; }
  }
  static __device__ __forceinline__ void store(float* p, const float (&v)[8]) {
    f32x4 a, b;
#pragma unroll
    for (int e = 0; e < 4; ++e) { a[e] = v[e]; b[e] = v[4 + e]; }
    *reinterpret_cast<f32x4*>(p) = a;
    *reinterpret_cast<f32x4*>(p + 4) = b;
  }
};

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

// cos / sin of the four pairs 4j..4j+3 of a band at position pos
__device__ __forceinline__ void rope_cs(int64_t pos, int j, int d_rope, double log2_base, float (&c)[4],
                                        float (&s)[4]) {
  constexpr double kTwoPi = 6.283185307179586476925286766559;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int i = 4 * j + k;
    const double freq = exp2(-(2.0 * i / d_rope) * log2_base);
    double a = (double)pos * freq;
    a -= kTwoPi * rint(a / kTwoPi);
    sincosf((float)a, &s[k], &c[k]);
  }
}

// rotate the 8 elements (4 pairs) at p in place; sgn = +1 forward, -1 transpose
template <typename T>
__device__ __forceinline__ void rotate8(T* p, const float (&c)[4], const float (&s)[4], float sgn) {
  float v[8];
  V8<T>::load(p, v);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float x0 = v[2 * k], x1 = v[2 * k + 1], sk = sgn * s[k];
    v[2 * k] = x0 * c[k] - x1 * sk;
    v[2 * k + 1] = x0 * sk + x1 * c[k];
  }
  V8<T>::store(p, v);
}

template <typename Tin, typename Tout>
__device__ __forceinline__ void rotate8_to(const Tin* src, Tout* dst, const float (&c)[4], const float (&s)[4],
                                           float sgn) {
  float v[8];
  V8<Tin>::load(src, v);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float x0 = v[2 * k], x1 = v[2 * k + 1], sk = sgn * s[k];
    v[2 * k] = x0 * c[k] - x1 * sk;
    v[2 * k + 1] = x0 * sk + x1 * c[k];
  }
  V8<Tout>::store(dst, v);
}

// The q_rope bands of one token: lane l owns pair chunk j = l % cpr of heads
// l / cpr, l / cpr + 64 / cpr, ... (cpr = d_rope / 8 divides 64).
template <typename T>
__device__ __forceinline__ void rotate_q_bands(T* qrow, int H, int d_nope, int d_qk, int cpr, int l,
                                               const float (&c)[4], const float (&s)[4], float sgn) {
  const int j = l % cpr;
  for (int h = l / cpr; h < H; h += 64 / cpr) rotate8(qrow + (size_t)h * d_qk + d_nope + 8 * j, c, s, sgn);
}

template <typename T>
__global__ __launch_bounds__(64 * kWaves) void prologue_fwd_kernel(PrologueArgs a) {
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int64_t tok = (int64_t)blockIdx.x * kWaves + wave;
  if (tok >= (int64_t)a.B * a.S) return;  // wave-uniform; the kernel has no barrier
  const int64_t pos = a.position_offset + tok % a.S;
  const int nch = a.d_c / 8;

  // normalisation: mean square over the row, in fp32
  const T* x = (const T*)a.latent_raw + tok * a.d_c;
  float v[kMaxChunks][8];
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < kMaxChunks; ++k) {
    const int ch = l + 64 * k;
    if (ch < nch) {
      V8<T>::load(x + 8 * ch, v[k]);
#pragma unroll
      for (int e = 0; e < 8; ++e) ss = __builtin_fmaf(v[k][e], v[k][e], ss);
    }
  }
  ss = wave_sum(ss);
  const float r = 1.f / sqrtf(ss / (float)a.d_c + a.eps);
  T* c = (T*)a.c_kv + tok * a.d_c;
#pragma unroll
  for (int k = 0; k < kMaxChunks; ++k) {
    const int ch = l + 64 * k;
    if (ch < nch) {
      float g[8];
      if (a.gamma) V8<T>::load((const T*)a.gamma + 8 * ch, g);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[k][e] = a.gamma ? (v[k][e] * r) * g[e] : v[k][e] * r;
      V8<T>::store(c + 8 * ch, v[k]);
    }
  }
  if (l == 0) a.rstd[tok] = r;

  // rotary embedding of k_pe and of every head's q_rope band
  const int cpr = a.d_rope / 8;
  float cs[4], sn[4];
  rope_cs(pos, l % cpr, a.d_rope, a.log2_base, cs, sn);
  if (l < cpr)
    rotate8_to((const T*)a.kpe_raw + tok * a.d_rope + 8 * l, (T*)a.k_pe + tok * a.d_rope + 8 * l, cs, sn, 1.f);
  if (a.q) rotate_q_bands((T*)a.q + tok * a.H * a.d_qk, a.H, a.d_nope, a.d_qk, cpr, l, cs, sn, 1.f);
}

// Backward. One wave handles kBwdTokPerWave consecutive tokens; the workgroup writes
// one partial row of d_gamma (its tokens, summed in a fixed order) to `partial`.
template <typename T>
__global__ __launch_bounds__(64 * kWaves) void prologue_bwd_kernel(PrologueArgs a) {
  __shared__ float sg[kWaves][1024];
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int64_t ntok = (int64_t)a.B * a.S;
  const int nch = a.d_c / 8;
  const int cpr = a.d_rope / 8;
  float gacc[kMaxChunks][8];
#pragma unroll
  for (int k = 0; k < kMaxChunks; ++k)
#pragma unroll
    for (int e = 0; e < 8; ++e) gacc[k][e] = 0.f;

  for (int i = 0; i < kBwdTokPerWave; ++i) {
    const int64_t tok = ((int64_t)blockIdx.x * kWaves + wave) * kBwdTokPerWave + i;
    if (tok >= ntok) break;  // wave-uniform
    const int64_t pos = a.position_offset + tok % a.S;
    const T* x = (const T*)a.latent_raw + tok * a.d_c;
    const float* dc = a.dc_kv + tok * a.d_c;
    const float r = a.rstd_in[tok];
    float y[kMaxChunks][8], g[kMaxChunks][8];
    float sgy = 0.f;
#pragma unroll
    for (int k = 0; k < kMaxChunks; ++k) {
      const int ch = l + 64 * k;
      if (ch < nch) {
        float d[8];
        V8<T>::load(x + 8 * ch, y[k]);
        V8<float>::load(dc + 8 * ch, d);
        float gm[8];
        if (a.gamma) V8<T>::load((const T*)a.gamma + 8 * ch, gm);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          y[k][e] *= r;
          g[k][e] = a.gamma ? gm[e] * d[e] : d[e];
          sgy = __builtin_fmaf(g[k][e], y[k][e], sgy);
          gacc[k][e] = __builtin_fmaf(d[e], y[k][e], gacc[k][e]);
        }
      }
    }
    const float m = wave_sum(sgy) / (float)a.d_c;
    float* dx = a.d_latent + tok * a.d_c;
#pragma unroll
    for (int k = 0; k < kMaxChunks; ++k) {
      const int ch = l + 64 * k;
      if (ch < nch) {
        float o[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = r * (g[k][e] - y[k][e] * m);
        V8<float>::store(dx + 8 * ch, o);
      }
    }
    float cs[4], sn[4];
    rope_cs(pos, l % cpr, a.d_rope, a.log2_base, cs, sn);
    if (l < cpr)
      rotate8_to(a.dk_pe + tok * a.d_rope + 8 * l, a.d_kpe + tok * a.d_rope + 8 * l, cs, sn, -1.f);
    if (a.q) rotate_q_bands((T*)a.q + tok * a.H * a.d_qk, a.H, a.d_nope, a.d_qk, cpr, l, cs, sn, -1.f);
  }
  if (!a.partial) return;  // workgroup-uniform: no barrier below is skipped by a subset
#pragma unroll
  for (int k = 0; k < kMaxChunks; ++k) {
    const int ch = l + 64 * k;
    if (ch < nch)
#pragma unroll
      for (int e = 0; e < 8; ++e) sg[wave][8 * ch + e] = gacc[k][e];
  }
  __syncthreads();
  // waves in ascending order (tokens in ascending order inside each wave)
  float* row = a.partial + (size_t)blockIdx.x * a.d_c;
  for (int j = threadIdx.x; j < a.d_c; j += 64 * kWaves) {
    float t = sg[0][j];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) t += sg[w][j];
    row[j] = t;
  }
}

// Column sums of a [rows][cols] partial buffer in a fixed order, in two launches: row
// group g (rows [g*rows/G, (g+1)*rows/G), ascending) of a 64-column block per wave,
// then the G group sums of each column, ascending. One lane per column.
constexpr int kSumGroups = 64;
__global__ __launch_bounds__(64) void column_sum_kernel(const float* __restrict__ src, float* __restrict__ dst,
                                                        int rows, int cols, int groups) {
  const int j = blockIdx.x * 64 + threadIdx.x;
  if (j >= cols) return;
  const int g = blockIdx.y;
  const int r0 = (int)((long long)rows * g / groups), r1 = (int)((long long)rows * (g + 1) / groups);
  float t = 0.f;
  for (int r = r0; r < r1; ++r) t += src[(size_t)r * cols + j];
  dst[(size_t)g * cols + j] = t;
}

}  // namespace

int prologue_bwd_rows(long long tokens) {
  const long long per = (long long)kWaves * kBwdTokPerWave;
  return (int)((tokens + per - 1) / per);
}

int prologue_sum_groups(long long tokens) {
  const int rows = prologue_bwd_rows(tokens);
  return rows < kSumGroups ? rows : kSumGroups;
}

template <typename T>
hipError_t launch_prologue_fwd(const PrologueArgs& a, hipStream_t st) {
  const long long tok = (long long)a.B * a.S;
  prologue_fwd_kernel<T><<<(unsigned)((tok + kWaves - 1) / kWaves), 64 * kWaves, 0, st>>>(a);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_prologue_bwd(const PrologueArgs& a, hipStream_t st) {
  const long long tok = (long long)a.B * a.S;
  const int rows = prologue_bwd_rows(tok);
  prologue_bwd_kernel<T><<<(unsigned)rows, 64 * kWaves, 0, st>>>(a);
  if (a.partial) {
    // partial holds the rows, then the group sums
    const int G = prologue_sum_groups(tok);
    float* gsum = a.partial + (size_t)rows * a.d_c;
    column_sum_kernel<<<dim3((a.d_c + 63) / 64, G), 64, 0, st>>>(a.partial, gsum, rows, a.d_c, G);
    column_sum_kernel<<<dim3((a.d_c + 63) / 64, 1), 64, 0, st>>>(gsum, a.d_gamma, G, a.d_c, 1);
  }
  return hipGetLastError();
}

template hipError_t launch_prologue_fwd<bf16>(const PrologueArgs&, hipStream_t);
template hipError_t launch_prologue_fwd<float>(const PrologueArgs&, hipStream_t);
template hipError_t launch_prologue_bwd<bf16>(const PrologueArgs&, hipStream_t);
template hipError_t launch_prologue_bwd<float>(const PrologueArgs&, hipStream_t);

}  // namespace laga
