// Generic key-stationary dK / dV kernel of the attention backward (the element types
// and head widths without a tuned kernel: fp32, and bf16 at head widths other than
// 192/128). Its own source file because it is compiled with the MFMA results in VGPRs
// (no AGPR<->VGPR copies around the softmax arithmetic on the accumulators, and the
// fp32 instance at 192/128-wide heads fits its 320 resident registers without spills),
// a choice that makes the tuned bf16 kernel of attn_bwd.hip spill.
//
// P = softmax(scale * Q K^T) is recomputed from the saved row log-sum-exp; per key
// block: dV = P^T dO, dP = dO V^T, dZ = P * (dP - delta), dK = scale dZ^T Q (the
// key-side half of the backward; dQ is the query-stationary pass of attn_bwd_dq.hip).
#include <type_traits>

// direct global->LDS copies issued as inline assembly (exact LDS-read waits; the ring
// orders the copies with explicit waits and barriers)
#define LAGA_LDS_DMA_ASM 1
#include "common.hpp"
#include "kernels.hpp"
#include "bwd_common.hpp"

namespace laga {

using namespace bwd;

namespace {

// ------------------------------------------------------------------ dK, dV
template <typename T, int DN, int DR, int DV, int BQ, int WPH>
__global__ __launch_bounds__(64 * WPH) void dkdv_kernel(BwdParams P) {
  constexpr int DQK = DN + DR, DKVH = DN + DV, DQK32 = round32(DQK);
  constexpr int BK = 32 * WPH, E = Elems16<T>::n;
  constexpr int PQ = lds_pitch<T>(DQK32), PO = lds_pitch<T>(DV);
  constexpr int QCH = DQK / E, OCH = DV / E;  // chunks per row
  static_assert(QCH <= 64 && OCH <= 64 && BQ % 4 == 0 && BQ <= 32, "one copy instruction per row");
  // two stages of [Q tile | dO tile | lse2 | delta], filled by direct global->LDS copies
  // while the other stage is consumed (no registers held for the staging)
  __shared__ __attribute__((aligned(16))) T sQb[2][BQ * PQ];
  __shared__ __attribute__((aligned(16))) T sOb[2][BQ * PO];
  __shared__ __attribute__((aligned(16))) float sLD[2][2 * BQ];

  const T* __restrict__ q = (const T*)P.q;
  const T* __restrict__ kpe = (const T*)P.k_pe;
  const T* __restrict__ kv = (const T*)P.kv;
  const T* __restrict__ dout = (const T*)P.dout;
  const int S = P.S, H = P.H;

  const int total = P.n_blocks * H * gridDim.y;
  const int lin = xcd_remap(blockIdx.x + gridDim.x * blockIdx.y, total);
  const int kb = lin % P.n_blocks;  // ascending: the first key blocks see the most queries
  const int bh = lin / P.n_blocks;
  const int b = bh / H, h = bh % H;

  const int tid = threadIdx.x, wave = tid >> 6, l = tid & 63, n = l & 31, g = l >> 5;
  const int k0 = kb * BK + wave * 32;  // first key of this wave
  const int my_k = k0 + n;

  // zero the padding columns [DQK, DQK32) of both stages once: transposing reads of Q^T
  // blocks touch them
  if (DQK32 > DQK)
    for (int i = tid; i < 2 * BQ * (DQK32 - DQK); i += 64 * WPH) {
      const int st = i / (BQ * (DQK32 - DQK)), j = i % (BQ * (DQK32 - DQK));
      sQb[st][(j / (DQK32 - DQK)) * PQ + DQK + j % (DQK32 - DQK)] = to_elem<T>(0.f);
    }

  // this lane's key and value rows (B operands of S = Q K^T and dP = dO V^T)
  frag_t<T> kf[DQK / 16], vf[DV / 16];
  {
    const bool ok = my_k < S;
    const size_t row = (size_t)(b * S + (ok ? my_k : 0));
    const T* kvr = kv + (row * H + h) * DKVH;
#pragma unroll
    for (int ks = 0; ks < DQK / 16; ++ks) {
      const T* src = ks < DN / 16 ? kvr + ks * 16 + 8 * g : kpe + row * DR + (ks - DN / 16) * 16 + 8 * g;
      if (ok) kf[ks] = *reinterpret_cast<const frag_t<T>*>(src);
      else
#pragma unroll
        for (int e = 0; e < 8; ++e) kf[ks][e] = to_elem<T>(0.f);
    }
#pragma unroll
    for (int ks = 0; ks < DV / 16; ++ks) {
      if (ok) vf[ks] = *reinterpret_cast<const frag_t<T>*>(kvr + DN + ks * 16 + 8 * g);
      else
#pragma unroll
        for (int e = 0; e < 8; ++e) vf[ks][e] = to_elem<T>(0.f);
    }
  }

  f32x16 dk[DQK32 / 32], dv[DV / 32];
#pragma unroll
  for (int i = 0; i < DQK32 / 32; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk[i][r] = 0.f;
#pragma unroll
  for (int i = 0; i < DV / 32; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) dv[i][r] = 0.f;

  // Stage st <- query tile qt: row r of the 2*BQ Q and dO rows is one copy instruction
  // of wave r % WPH (lane l copies chunk l of the row); rows past S are zero-filled by
  // LDS stores. lse2 and delta rows are padded to S_pad (a multiple of 64 >= S), so their
  // BQ entries are copied whole by the last wave: lanes [0, BQ/4) lse2, [BQ/4, BQ/2) delta.
  const size_t ld_row = (size_t)(b * H + h) * P.S_pad;
  auto fill = [&](int st, int qt) {
    for (int r = wave; r < 2 * BQ; r += WPH) {
      const bool isq = r < BQ;
      const int row = isq ? r : r - BQ, qi = qt + row;
      T* dst = isq ? &sQb[st][row * PQ] : &sOb[st][row * PO];
      if (l < (isq ? QCH : OCH)) {
        if (qi < S) {
          const size_t base = (size_t)(b * S + qi) * H + h;
          g2lds16(isq ? q + base * DQK + l * E : dout + base * DV + l * E, dst);
        } else {
          *reinterpret_cast<chunk16*>(dst + l * E) = zero_chunk();
        }
      }
    }
    if (wave == WPH - 1 && l < BQ / 2) {
      const float* src = l < BQ / 4 ? P.lse2 + ld_row + qt + 4 * l : P.delta + ld_row + qt + 4 * (l - BQ / 4);
      g2lds16(src, &sLD[st][0]);
    }
  };

  const int qt_begin = P.causal ? (kb * BK) / BQ * BQ : 0;
  fill(0, qt_begin);
  int st = 0;
  for (int qt = qt_begin; qt < S; qt += BQ, st ^= 1) {
    wait_vmem();      // this wave's copies of tile qt have landed
    __syncthreads();  // every wave's copies and zero stores of stage st are visible; stage st^1
                      // is no longer read
    if (qt + BQ < S) fill(st ^ 1, qt + BQ);
    const T* sQ = sQb[st];
    const T* sO = sOb[st];
    const float* sL = sLD[st];
    const float* sD = sLD[st] + BQ;

    const bool active = k0 < S && (!P.causal || qt + BQ - 1 >= k0);
    if (!active) continue;
    const bool need_mask = (P.causal && qt < k0 + 31) || (qt + BQ > S);

    f32x16 sa[BQ / 32], dp[BQ / 32];
#pragma unroll
    for (int qb = 0; qb < BQ / 32; ++qb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) { sa[qb][r] = 0.f; dp[qb][r] = 0.f; }
#pragma unroll
      for (int ks = 0; ks < DQK / 16; ++ks)
        mma(sa[qb], lds_frag<T>(sQ + (qb * 32 + n) * PQ + ks * 16 + 8 * g), kf[ks]);
#pragma unroll
      for (int ks = 0; ks < DV / 16; ++ks)
        mma(dp[qb], lds_frag<T>(sO + (qb * 32 + n) * PO + ks * 16 + 8 * g), vf[ks]);
    }
    // P and dZ (in place): rows = queries qt + qb*32 + (r/4)*8 + g*4 + r%4, column = my key
#pragma unroll
    for (int qb = 0; qb < BQ / 32; ++qb)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int qrow = qb * 32 + rr * 8 + g * 4;
        const f32x4 lq = *reinterpret_cast<const f32x4*>(sL + qrow);
        const f32x4 dq = *reinterpret_cast<const f32x4*>(sD + qrow);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = rr * 4 + e;
          float p = fast_exp2(sa[qb][r] * P.scale_log2 - lq[e]);
          if (need_mask) {
            const int qi = qt + qrow + e;
            if (qi >= S || (P.causal && my_k > qi)) p = 0.f;
          }
          sa[qb][r] = p;
          dp[qb][r] = p * (dp[qb][r] - dq[e]);
        }
      }
#pragma unroll
    for (int kk = 0; kk < BQ / 16; ++kk) {
      const frag_t<T> pf = acc_to_frag<T>(sa[kk >> 1], kk & 1);
      const frag_t<T> zf = acc_to_frag<T>(dp[kk >> 1], kk & 1);
      const int ra = kk * 16 + 4 * g;
#pragma unroll
      for (int db = 0; db < DV / 32; ++db) mma(dv[db], TrRead<T>::get(sO, PO, ra, ra + 8, db * 32), pf);
#pragma unroll
      for (int db = 0; db < DQK32 / 32; ++db) mma(dk[db], TrRead<T>::get(sQ, PQ, ra, ra + 8, db * 32), zf);
    }
  }

  if (my_k >= S) return;
  const size_t row = (size_t)(b * S + my_k) * H + h;
  T* dkvr = (T*)P.dkv + row * DKVH;
  T* dkvl = (T*)P.dkv_lo + row * DKVH;
  float* dper = P.dkpe_h + row * DR;
  // dKV as hi (+ lo for bf16): lo = bf16(x - hi) carries the next 8 bits for the GEMMs
  auto put4 = [&](int col, float a0, float a1, float a2, float a3) {
    typename FragOf<T>::half hi = {to_elem<T>(a0), to_elem<T>(a1), to_elem<T>(a2), to_elem<T>(a3)};
    *reinterpret_cast<typename FragOf<T>::half*>(dkvr + col) = hi;
    if (sizeof(T) == 2) {
      typename FragOf<T>::half lo = {to_elem<T>(a0 - to_f32(hi[0])), to_elem<T>(a1 - to_f32(hi[1])),
                                     to_elem<T>(a2 - to_f32(hi[2])), to_elem<T>(a3 - to_f32(hi[3]))};
      *reinterpret_cast<typename FragOf<T>::half*>(dkvl + col) = lo;
    }
  };
#pragma unroll
  for (int db = 0; db < DQK32 / 32; ++db)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int d = db * 32 + rr * 8 + g * 4;
      const float a0 = dk[db][4 * rr] * P.scale, a1 = dk[db][4 * rr + 1] * P.scale;
      const float a2 = dk[db][4 * rr + 2] * P.scale, a3 = dk[db][4 * rr + 3] * P.scale;
      if (d < DN) {
        put4(d, a0, a1, a2, a3);
      } else if (d < DQK) {
        f32x4 v = {a0, a1, a2, a3};
        *reinterpret_cast<f32x4*>(dper + (d - DN)) = v;
      }
    }
#pragma unroll
  for (int db = 0; db < DV / 32; ++db)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr)
      put4(DN + db * 32 + rr * 8 + g * 4, dv[db][4 * rr], dv[db][4 * rr + 1], dv[db][4 * rr + 2], dv[db][4 * rr + 3]);
}

}  // namespace

template <typename T, int DN, int DR, int DV>
hipError_t launch_dkdv_generic(BwdParams P, int B, hipStream_t st) {
  using Tl = BwdTiles<T>;
  constexpr int BK = 32 * Tl::WPH_KV;
  P.n_blocks = (P.S + BK - 1) / BK;
  dkdv_kernel<T, DN, DR, DV, Tl::BQ, Tl::WPH_KV><<<dim3(P.n_blocks * P.H, B), 64 * Tl::WPH_KV, 0, st>>>(P);
  return hipGetLastError();
}

#define LAGA_INST_DKDV(T, DN, DR, DV) \
  template hipError_t launch_dkdv_generic<T, DN, DR, DV>(BwdParams, int, hipStream_t);
LAGA_INST_DKDV(float, 128, 64, 128)  // bf16 at these widths runs dkdv32_kernel
LAGA_INST_DKDV(bf16, 32, 16, 32)
LAGA_INST_DKDV(float, 32, 16, 32)
LAGA_INST_DKDV(bf16, 64, 32, 64)
LAGA_INST_DKDV(float, 64, 32, 64)

}  // namespace laga
