// Causal MLA flash-attention forward (Alg. 1 step 5), bf16 with 128/64/128-wide
// heads, materialised K/V: the production kernel of that configuration. The generic
// kernels (other shapes, fp32, the fused latent->LDS variant) are in attn_fwd.hip;
// the arithmetic here is the same as theirs, step for step, so every variant gives
// the same bits.
//
// A workgroup of WPH waves owns 32 * WPH consecutive queries of one head at one
// workgroup per CU; wave w serves 32 of them, a lane one query (everything is
// computed transposed: S^T = K Q^T, O^T += V^T P^T; see attn_fwd.hip). Key tiles of
// BC keys stream through a two-stage LDS ring of direct global->LDS loads:
//   K = [K_nope || k_pe] rows at a pitch of 25 16-byte chunks (odd: the 32x32
//       row-fragment reads of S^T = K Q^T are conflict-free);
//   V rows at a pitch of 20 chunks (20 % 8 == 4: the transposing reads of
//       O^T += V^T P^T are conflict-free).
// Padded tiles keep every LDS read at a per-lane base address plus a constant, so no
// registers go to per-read addresses and the compiler can read fragments ahead of the
// MFMAs. Key tiles entirely after a wave's last query are skipped (a wave-uniform
// branch); with the causal mask that is the upper triangle of the workgroup's
// diagonal block.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace laga {

namespace {

struct FwdPadParams {
  const void* q;
  const void* k_pe;
  const void* kv;
  void* out;
  float* lse;
  int S, H, n_qblocks;
  float scale_log2;  // softmax_scale * log2(e)
  int causal;
};

template <int DN, int DR, int DV, int BC, int WPH>
__global__ __launch_bounds__(64 * WPH, 1) void attn_fwd_pad_kernel(FwdPadParams P) {
  using T = bf16;
  constexpr int DQK = DN + DR, DKVH = DN + DV, NW = WPH, BR = 32 * WPH;
  constexpr int KCPR = DQK / 8, NCPR = DN / 8, VCPR = DV / 8;
  constexpr int KP = KCPR + 1, VP = VCPR + 4;
  static_assert(KP % 2 == 1 && VP % 8 == 4 && BC % 32 == 0, "conflict-free pitches, whole 32-key blocks");
  constexpr int KCH = pad_chunks(BC, KP), VCH = pad_chunks(BC, VP);
  // two ring stages as distinct LDS objects (the reads of one stage are then not
  // made to wait for the direct loads into the other)
  __shared__ __attribute__((aligned(16))) T sK0[KCH * 8], sK1[KCH * 8];
  __shared__ __attribute__((aligned(16))) T sV0[VCH * 8], sV1[VCH * 8];

  const T* __restrict__ q = (const T*)P.q;
  const T* __restrict__ kpe = (const T*)P.k_pe;
  const T* __restrict__ kv = (const T*)P.kv;
  const int S = P.S, H = P.H;

  const int total = P.n_qblocks * H * gridDim.y;
  const int lin = xcd_remap(blockIdx.x + gridDim.x * blockIdx.y, total);
  const int qb = P.n_qblocks - 1 - lin % P.n_qblocks;  // heavy first
  const int bh = lin / P.n_qblocks;
  const int b = bh / H, h = bh % H;

  const int tid = threadIdx.x, wave = tid >> 6, l = tid & 63, n = l & 31, g = l >> 5;
  const int q0 = qb * BR + wave * 32;
  const int my_q = q0 + n;
  const int kend = P.causal ? min(S, (qb + 1) * BR) : S;
  // last key tile this wave needs (all later ones are fully masked for it)
  const int wave_kend = P.causal ? min(kend, q0 + 32) : kend;

  frag_t<T> qf[DQK / 16];
  {
    const bool ok = my_q < S;
    const T* qrow = q + ((size_t)(b * S + (ok ? my_q : 0)) * H + h) * DQK;
#pragma unroll
    for (int ks = 0; ks < DQK / 16; ++ks) {
      qf[ks] = *reinterpret_cast<const frag_t<T>*>(qrow + ks * 16 + 8 * g);
      if (!ok) qf[ks] = frag_t<T>{};
    }
  }
  f32x16 oacc[DV / 32];
#pragma unroll
  for (int i = 0; i < DV / 32; ++i) oacc[i] = f32x16{};
  float m = -INFINITY, lsum = 0.f;

  auto fill = [&](T* dk, T* dv, int kt) {
    // key rows past S are clamped to S-1 (valid memory) and masked below
    pad_fill_chunks<T, BC, KCPR, KP, NW>(dk, wave, l, [&](int r, int c) {
      const size_t row = (size_t)(b * S + min(kt + r, S - 1));
      return c < NCPR ? kv + (row * H + h) * DKVH + c * 8 : kpe + row * DR + (c - NCPR) * 8;
    });
    pad_fill<T, BC, VCPR, VP, NW>(dv, wave, l, [&](int r) {
      return kv + ((size_t)(b * S + min(kt + r, S - 1)) * H + h) * DKVH + DN;
    });
  };

  const int ntiles = (kend + BC - 1) / BC;
  fill(sK0, sV0, 0);
  auto step = [&](auto stage, int it) {
    constexpr int ST = decltype(stage)::value;
    const int kt = it * BC;
    wait_vmem();      // this wave's loads of tile `it` have landed
    __syncthreads();  // ... and everyone's; the other stage is free
    if (it + 1 < ntiles) {
      if constexpr (ST == 0) fill(sK1, sV1, kt + BC);
      else fill(sK0, sV0, kt + BC);
    }
    if (kt >= wave_kend) return;  // wave-uniform: every key of the tile is masked for this wave
    const T* tk = ST == 0 ? sK0 : sK1;
    const T* tv = ST == 0 ? sV0 : sV1;

    f32x16 sacc[BC / 32];
#pragma unroll
    for (int kb = 0; kb < BC / 32; ++kb) {
      sacc[kb] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < DQK / 16; ++ks) mma(sacc[kb], pad_frag<KP>(tk, kb * 32 + n, 2 * ks + g), qf[ks]);
    }
    const bool need_mask = (P.causal && kt + BC - 1 > q0) || (kt + BC > S);
    const int klim = P.causal ? min(S, my_q + 1) : S;  // live keys: key < klim
    if (need_mask) {
#pragma unroll
      for (int kb = 0; kb < BC / 32; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kt + kb * 32 + (r >> 2) * 8 + g * 4 + (r & 3);
          sacc[kb][r] = key < klim ? sacc[kb][r] : -INFINITY;
        }
    }
    float mraw = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < BC / 32; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mraw = fmaxf(mraw, sacc[kb][r]);
    mraw = wave_xor32_max(mraw);
    const float m_new = fmaxf(m, mraw * P.scale_log2);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = fast_exp2(m - m_use);
    float ps = 0.f;
#pragma unroll
    for (int kb = 0; kb < BC / 32; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = fast_exp2(__builtin_fmaf(sacc[kb][r], P.scale_log2, -m_use));
        sacc[kb][r] = p;
        ps += p;
      }
    lsum = lsum * alpha + ps;
    m = m_new;
    if (__ballot(alpha != 1.f)) {
#pragma unroll
      for (int i = 0; i < DV / 32; ++i) oacc[i] *= alpha;
    }
    frag_t<T> pf[BC / 16];
#pragma unroll
    for (int kk = 0; kk < BC / 16; ++kk) pf[kk] = acc_to_frag<T>(sacc[kk >> 1], kk & 1);
#pragma unroll
    for (int db = 0; db < DV / 32; ++db)
#pragma unroll
      for (int kk = 0; kk < BC / 16; ++kk) {
        const int ra = kk * 16 + 4 * g;
        mma(oacc[db], pad_tr_frag<VP>(tv, ra, ra + 8, db * 32), pf[kk]);
      }
  };
  for (int it = 0; it < ntiles; it += 2) {
    step(std::integral_constant<int, 0>{}, it);
    if (it + 1 < ntiles) step(std::integral_constant<int, 1>{}, it + 1);
  }

  if (my_q >= S) return;
  const float ltot = wave_xor32_sum(lsum);
  const float inv = 1.f / ltot;
  T* orow = (T*)P.out + ((size_t)(b * S + my_q) * H + h) * DV;
#pragma unroll
  for (int db = 0; db < DV / 32; ++db)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      bf16x4 v;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = to_elem<T>(oacc[db][4 * rr + e] * inv);
      *reinterpret_cast<bf16x4*>(orow + db * 32 + rr * 8 + g * 4) = v;
    }
  if (g == 0) P.lse[(size_t)(b * H + h) * S + my_q] = (m + fast_log2(ltot)) * 0.69314718055994530942f;
}

}  // namespace

hipError_t launch_attn_fwd_pad(const AttnFwdArgs& a, hipStream_t st) {
  constexpr int DN = 128, DR = 64, DV = 128, BC = 64, WPH = 8, BR = 32 * WPH;
  FwdPadParams P;
  P.q = a.q; P.k_pe = a.k_pe; P.kv = a.kv; P.out = a.out; P.lse = a.lse;
  P.S = a.S; P.H = a.H;
  P.n_qblocks = (a.S + BR - 1) / BR;
  P.scale_log2 = a.scale * 1.4426950408889634f;
  P.causal = a.causal;
  attn_fwd_pad_kernel<DN, DR, DV, BC, WPH><<<dim3(P.n_qblocks * a.H, a.B, 1), 64 * WPH, 0, st>>>(P);
  return hipGetLastError();
}

}  // namespace laga
