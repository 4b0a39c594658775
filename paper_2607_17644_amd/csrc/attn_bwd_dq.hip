// Query-stationary dQ pass of the attention backward (gfx950); see attn_bwd.hip for
// the whole backward. Built with MFMA results kept in VGPRs (the dZ arithmetic on
// the dP accumulators then needs no AGPR<->VGPR copies).
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "bwd_common.hpp"

namespace laga {

using namespace bwd;

namespace {

// ------------------------------------------------------------------ dQ
template <typename T, int DN, int DR, int DV, int BC, int WPH>
__global__ __launch_bounds__(64 * WPH) void dq_kernel(BwdParams P) {
  constexpr int DQK = DN + DR, DKVH = DN + DV, DQK32 = round32(DQK);
  constexpr int NT = 64 * WPH, BR = 32 * WPH, E = Elems16<T>::n;
  constexpr int PK = lds_pitch<T>(DQK32), PV = lds_pitch<T>(DV);
  constexpr int KCH = DQK / E, VCH = DV / E;
  constexpr int TILE_CHUNKS = BC * (KCH + VCH);
  constexpr int PER_THREAD = (TILE_CHUNKS + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) T sK[BC * PK];
  __shared__ __attribute__((aligned(16))) T sV[BC * PV];

  const T* __restrict__ q = (const T*)P.q;
  const T* __restrict__ kpe = (const T*)P.k_pe;
  const T* __restrict__ kv = (const T*)P.kv;
  const T* __restrict__ dout = (const T*)P.dout;
  const int S = P.S, H = P.H;

  const int total = P.n_blocks * H * gridDim.y;
  const int lin = xcd_remap(blockIdx.x + gridDim.x * blockIdx.y, total);
  const int qblk = P.n_blocks - 1 - lin % P.n_blocks;  // heavy first
  const int bh = lin / P.n_blocks;
  const int b = bh / H, h = bh % H;

  const int tid = threadIdx.x, wave = tid >> 6, l = tid & 63, n = l & 31, g = l >> 5;
  const int q0 = qblk * BR + wave * 32;
  const int my_q = q0 + n;
  const int wg_qend = min(S, (qblk + 1) * BR);
  const int kend = P.causal ? wg_qend : S;

  if (DQK32 > DQK)
    for (int i = tid; i < BC * (DQK32 - DQK); i += NT)
      sK[(i / (DQK32 - DQK)) * PK + DQK + i % (DQK32 - DQK)] = to_elem<T>(0.f);

  frag_t<T> qf[DQK / 16], of[DV / 16];
  float lse2 = 0.f, dlt = 0.f;
  {
    const bool ok = my_q < S;
    const size_t base = (size_t)(b * S + (ok ? my_q : 0)) * H + h;
#pragma unroll
    for (int ks = 0; ks < DQK / 16; ++ks) {
      if (ok) qf[ks] = *reinterpret_cast<const frag_t<T>*>(q + base * DQK + ks * 16 + 8 * g);
      else
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[ks][e] = to_elem<T>(0.f);
    }
#pragma unroll
    for (int ks = 0; ks < DV / 16; ++ks) {
      if (ok) of[ks] = *reinterpret_cast<const frag_t<T>*>(dout + base * DV + ks * 16 + 8 * g);
      else
#pragma unroll
        for (int e = 0; e < 8; ++e) of[ks][e] = to_elem<T>(0.f);
    }
    if (ok) {
      lse2 = P.lse2[(size_t)(b * H + h) * P.S_pad + my_q];
      dlt = P.delta[(size_t)(b * H + h) * P.S_pad + my_q];
    }
  }

  f32x16 dqa[DQK32 / 32];
#pragma unroll
  for (int i = 0; i < DQK32 / 32; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) dqa[i][r] = 0.f;

  chunk16 stage[PER_THREAD];
  auto load_tile = [&](int kt) {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int c = tid + i * NT;
      stage[i] = zero_chunk();
      if (c < TILE_CHUNKS) {
        const int row = c / (KCH + VCH), j = c % (KCH + VCH);
        const int key = kt + row;
        if (key < S) {
          const size_t r = (size_t)(b * S + key);
          const T* src = j < DN / E ? kv + (r * H + h) * DKVH + j * E
                       : j < KCH    ? kpe + r * DR + (j - DN / E) * E
                                    : kv + (r * H + h) * DKVH + DN + (j - KCH) * E;
          stage[i] = *reinterpret_cast<const chunk16*>(src);
        }
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int c = tid + i * NT;
      if (c < TILE_CHUNKS) {
        const int row = c / (KCH + VCH), j = c % (KCH + VCH);
        T* dst = j < KCH ? sK + row * PK + j * E : sV + row * PV + (j - KCH) * E;
        *reinterpret_cast<chunk16*>(dst) = stage[i];
      }
    }
  };

  load_tile(0);
  for (int kt = 0; kt < kend; kt += BC) {
    __syncthreads();
    store_tile();
    __syncthreads();
    if (kt + BC < kend) load_tile(kt + BC);

    const bool active = q0 < S && (!P.causal || kt <= q0 + 31);
    if (!active) continue;
    const bool need_mask = (P.causal && kt + BC - 1 > q0) || (kt + BC > S);

    f32x16 sa[BC / 32], dp[BC / 32];
#pragma unroll
    for (int kb = 0; kb < BC / 32; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) { sa[kb][r] = 0.f; dp[kb][r] = 0.f; }
#pragma unroll
      for (int ks = 0; ks < DQK / 16; ++ks)
        mma(sa[kb], lds_frag<T>(sK + (kb * 32 + n) * PK + ks * 16 + 8 * g), qf[ks]);
#pragma unroll
      for (int ks = 0; ks < DV / 16; ++ks)
        mma(dp[kb], lds_frag<T>(sV + (kb * 32 + n) * PV + ks * 16 + 8 * g), of[ks]);
    }
#pragma unroll
    for (int kb = 0; kb < BC / 32; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float p = fast_exp2(sa[kb][r] * P.scale_log2 - lse2);
        if (need_mask) {
          const int key = kt + kb * 32 + (r >> 2) * 8 + g * 4 + (r & 3);
          if (key >= S || (P.causal && key > my_q)) p = 0.f;
        }
        dp[kb][r] = p * (dp[kb][r] - dlt);
      }
#pragma unroll
    for (int kk = 0; kk < BC / 16; ++kk) {
      const frag_t<T> zf = acc_to_frag<T>(dp[kk >> 1], kk & 1);
      const int ra = kk * 16 + 4 * g;
#pragma unroll
      for (int db = 0; db < DQK32 / 32; ++db) mma(dqa[db], TrRead<T>::get(sK, PK, ra, ra + 8, db * 32), zf);
    }
  }

  if (my_q >= S) return;
  T* dqr = (T*)P.dq + ((size_t)(b * S + my_q) * H + h) * DQK;
#pragma unroll
  for (int db = 0; db < DQK32 / 32; ++db)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int d = db * 32 + rr * 8 + g * 4;
      if (d < DQK) {
        typename FragOf<T>::half v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = to_elem<T>(dqa[db][4 * rr + e] * P.scale);
        *reinterpret_cast<typename FragOf<T>::half*>(dqr + d) = v;
      }
    }
}


// Query-stationary dQ, bf16 with 192/128-wide heads: key tiles (K = [K_nope || k_pe]
// as one 192-wide swizzled tile, V as a 128-wide one) stream through a two-stage
// LDS ring of direct global->LDS loads; one barrier per tile; no per-wave branch
// around the MFMAs (tiles entirely after a wave's queries run fully masked).
template <int DN, int DR, int DV, int BC, int WPH>
__global__ __launch_bounds__(64 * WPH, 2) void dq_ring_kernel(BwdParams P) {
  using T = bf16;
  constexpr int DQK = DN + DR, DKVH = DN + DV, NW = WPH, BR = 32 * WPH;
  constexpr int KCPR = DQK / 8, VCPR = DV / 8, NCPR = DN / 8;
  static_assert(KCPR == 24 && VCPR == 16, "swizzles are defined for 192/128-wide rows");
  // two ring stages as distinct LDS objects (so the compiler does not make the reads
  // of one stage wait for the direct loads into the other)
  __shared__ __attribute__((aligned(16))) T sK0[BC * DQK], sK1[BC * DQK];
  __shared__ __attribute__((aligned(16))) T sV0[BC * DV], sV1[BC * DV];
  // the workgroup's dO rows stay in LDS (B operand of dP^T = V dO^T), which keeps
  // the per-lane state small enough for two waves per SIMD
  __shared__ __attribute__((aligned(16))) T sDO[BR * DV];

  const T* __restrict__ q = (const T*)P.q;
  const T* __restrict__ kpe = (const T*)P.k_pe;
  const T* __restrict__ kv = (const T*)P.kv;
  const T* __restrict__ dout = (const T*)P.dout;
  const int S = P.S, H = P.H;

  const int total = P.n_blocks * H * gridDim.y;
  const int lin = xcd_remap(blockIdx.x + gridDim.x * blockIdx.y, total);
  const int qblk = P.n_blocks - 1 - lin % P.n_blocks;
  const int bh = lin / P.n_blocks;
  const int b = bh / H, h = bh % H;

  const int tid = threadIdx.x, wave = tid >> 6, l = tid & 63, n = l & 31, g = l >> 5;
  const int q0 = qblk * BR + wave * 32;
  const int my_q = q0 + n;
  const int kend = P.causal ? min(S, (qblk + 1) * BR) : S;

  frag_t<T> qf[DQK / 16];
  float lse2, dlt;
  {
    const bool ok = my_q < S;
    const size_t base = (size_t)(b * S + (ok ? my_q : 0)) * H + h;
#pragma unroll
    for (int ks = 0; ks < DQK / 16; ++ks) {
      qf[ks] = *reinterpret_cast<const frag_t<T>*>(q + base * DQK + ks * 16 + 8 * g);
      if (!ok) qf[ks] = frag_t<T>{};
    }
    // dO rows of the workgroup's queries (rows past S clamped; their dq is not stored)
    swz_fill<T, BR, VCPR, NW>(sDO, wave, l, [&](int r) {
      return dout + ((size_t)(b * S + min(qblk * BR + r, S - 1)) * H + h) * DV;
    });
    const size_t hr = (size_t)(b * H + h) * P.S_pad + (ok ? my_q : 0);
    lse2 = P.lse2[hr];
    dlt = P.delta[hr];
  }

  f32x16 dqa[DQK / 32];
#pragma unroll
  for (int i = 0; i < DQK / 32; ++i) dqa[i] = f32x16{};

  auto fill = [&](T* dk, T* dv, int kt) {
    swz_fill_chunks<T, BC, KCPR, NW>(dk, wave, l, [&](int r, int c) {
      const size_t row = (size_t)(b * S + min(kt + r, S - 1));
      return c < NCPR ? kv + (row * H + h) * DKVH + c * 8 : kpe + row * DR + (c - NCPR) * 8;
    });
    swz_fill<T, BC, VCPR, NW>(dv, wave, l, [&](int r) {
      return kv + ((size_t)(b * S + min(kt + r, S - 1)) * H + h) * DKVH + DN;
    });
  };

  const int ntiles = (kend + BC - 1) / BC;
  fill(sK0, sV0, 0);
  auto step = [&](auto stage, int it) {
    constexpr int ST = decltype(stage)::value;
    const int kt = it * BC;
    wait_vmem();      // this wave's loads of tile `it` (and, the first time, of dO) have landed
    __syncthreads();  // ... and everyone's; the other stage is free
    if (it + 1 < ntiles) {
      if constexpr (ST == 0) fill(sK1, sV1, kt + BC);
      else fill(sK0, sV0, kt + BC);
    }
    const T* tk = ST == 0 ? sK0 : sK1;
    const T* tv = ST == 0 ? sV0 : sV1;

    f32x16 sa[BC / 32], dp[BC / 32];
#pragma unroll
    for (int kb = 0; kb < BC / 32; ++kb) {
      sa[kb] = f32x16{};
      dp[kb] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < DQK / 16; ++ks) mma(sa[kb], swz_frag<T, KCPR>(tk, kb * 32 + n, 2 * ks + g), qf[ks]);
#pragma unroll
      for (int ks = 0; ks < DV / 16; ++ks)
        mma(dp[kb], swz_frag<T, VCPR>(tv, kb * 32 + n, 2 * ks + g), swz_frag<T, VCPR>(sDO, wave * 32 + n, 2 * ks + g));
    }
    const bool need_mask = (P.causal && kt + BC - 1 > q0) || (kt + BC > S);
#pragma unroll
    for (int kb = 0; kb < BC / 32; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float p = fast_exp2(__builtin_fmaf(sa[kb][r], P.scale_log2, -lse2));
        if (need_mask) {
          const int key = kt + kb * 32 + (r >> 2) * 8 + g * 4 + (r & 3);
          if (key >= S || (P.causal && key > my_q)) p = 0.f;
        }
        dp[kb][r] = p * (dp[kb][r] - dlt);
      }
#pragma unroll
    for (int kk = 0; kk < BC / 16; ++kk) {
      const frag_t<T> zf = acc_to_frag<T>(dp[kk >> 1], kk & 1);
      const int ra = kk * 16 + 4 * g;
#pragma unroll
      for (int db = 0; db < DQK / 32; ++db) mma(dqa[db], swz_tr_frag<KCPR>(tk, ra, ra + 8, db * 32), zf);
    }
  };
  for (int it = 0; it < ntiles; it += 2) {
    step(std::integral_constant<int, 0>{}, it);
    if (it + 1 < ntiles) step(std::integral_constant<int, 1>{}, it + 1);
  }

  if (my_q >= S) return;
  T* dqr = (T*)P.dq + ((size_t)(b * S + my_q) * H + h) * DQK;
#pragma unroll
  for (int db = 0; db < DQK / 32; ++db)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      bf16x4 v;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = to_elem<T>(dqa[db][4 * rr + e] * P.scale);
      *reinterpret_cast<bf16x4*>(dqr + db * 32 + rr * 8 + g * 4) = v;
    }
}

}  // namespace

template <typename T, int DN, int DR, int DV>
hipError_t launch_bwd_dq(bwd::BwdParams P, int B, hipStream_t st) {
  using Tl = BwdTiles<T>;
  constexpr int BR = 32 * Tl::WPH_Q;
  P.n_blocks = (P.S + BR - 1) / BR;
  if constexpr (sizeof(T) == 2 && DN + DR == 192 && DV == 128)
    dq_ring_kernel<DN, DR, DV, 32, Tl::WPH_Q><<<dim3(P.n_blocks * P.H, B), 64 * Tl::WPH_Q, 0, st>>>(P);
  else
    dq_kernel<T, DN, DR, DV, Tl::BC, Tl::WPH_Q><<<dim3(P.n_blocks * P.H, B), 64 * Tl::WPH_Q, 0, st>>>(P);
  return hipGetLastError();
}

#define LAGA_INST_DQ(T, DN, DR, DV) template hipError_t launch_bwd_dq<T, DN, DR, DV>(bwd::BwdParams, int, hipStream_t);
LAGA_INST_DQ(bf16, 128, 64, 128)
LAGA_INST_DQ(float, 128, 64, 128)
LAGA_INST_DQ(bf16, 32, 16, 32)
LAGA_INST_DQ(float, 32, 16, 32)

}  // namespace laga
