// Backward of the per-rank LAGA attention block (gfx950). Given dO, with
// P = softmax(scale * Q K^T) recomputed from the saved row log-sum-exp:
//   delta_i = sum_e dO_ie O_ie
//   dV = P^T dO,  dP = dO V^T,  dZ = P * (dP - delta),
//   dQ = scale dZ K,  dK = scale dZ^T Q
// and K_h = [K_nope,h || k_pe] (k_pe shared by every head), so dk_pe sums the
// k_pe columns of dK_h over the shard's heads, while dK_nope,h and dV_h form
// the head's block of dKV, which the up-projection backward turns into dc_kv
// and dW (gemm.hip).
//
// Kernels (all deterministic: no floating-point atomics anywhere):
//   delta_kernel   one thread per (token, head)
//   dkdv_kernel    key-stationary: a workgroup owns 32*WPH keys of one head and
//                  sweeps the query tiles at or after them; lane <-> key layout
//                  (S = Q K^T with K in registers), so P and dZ feed the
//                  dV^T += dO^T P and dK^T += Q^T dZ products directly from the
//                  accumulators, with dO^T / Q^T read by transposing LDS reads
//   dq_kernel      query-stationary: a workgroup owns 32*WPH queries of one
//                  head and sweeps the key tiles up to the diagonal; lane <->
//                  query layout (S^T = K Q^T), dQ^T += K^T dZ^T with K^T read by
//                  transposing LDS reads; it recomputes S and dP (the price of
//                  not accumulating dQ with atomics)
//   dkpe_kernel    dk_pe = sum over heads (ascending) of the per-head k_pe parts
#include "common.hpp"
#include "kernels.hpp"

namespace laga {

namespace {

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
};

// delta[b,h,t] = sum_e dout[b,t,h,e] * out[b,t,h,e]. One wave per token: the token's
// [H, DV] rows of out and dout are contiguous, lanes read consecutive 16-byte chunks,
// and the DV/E lanes that share a head finish the sum with xor shuffles.
// Also writes lse2 = lse * log2(e); delta and lse2 rows are [B*H][S_pad] with
// S_pad = S rounded up to kRowPad, the pad entries zeroed (tiles of the
// key-stationary kernel are fetched whole).
template <typename T, int DV>
__global__ __launch_bounds__(256) void delta_kernel(const T* __restrict__ out, const T* __restrict__ dout,
                                                    const float* __restrict__ lse, float* __restrict__ delta,
                                                    float* __restrict__ lse2, int S, int S_pad, int H, int BS) {
  constexpr int E = Elems16<T>::n, CPH = DV / E;  // chunks per head (a power of two dividing 64)
  static_assert(64 % CPH == 0, "heads must tile the wave");
  const int tok = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int l = threadIdx.x & 63;
  if (tok >= BS) return;
  const int nch = H * CPH;
  const T* o = out + (size_t)tok * H * DV;
  const T* d = dout + (size_t)tok * H * DV;
  const int b = tok / S, t = tok % S;
  for (int c0 = 0; c0 < nch; c0 += 64) {  // wave-uniform trip count
    const int c = c0 + l;
    float acc = 0.f;
    if (c < nch) {
      chunk16 va = *reinterpret_cast<const chunk16*>(o + (size_t)c * E);
      chunk16 vb = *reinterpret_cast<const chunk16*>(d + (size_t)c * E);
      const T* pa = reinterpret_cast<const T*>(&va);
      const T* pb = reinterpret_cast<const T*>(&vb);
#pragma unroll
      for (int e = 0; e < E; ++e) acc += to_f32(pa[e]) * to_f32(pb[e]);
    }
#pragma unroll
    for (int m = 1; m < CPH; m <<= 1) acc += __shfl_xor(acc, m);
    if (c < nch && (c % CPH) == 0) {
      const int h = c / CPH;
      const size_t o = (size_t)(b * H + h) * S_pad + t;
      delta[o] = acc;
      lse2[o] = lse[(size_t)(b * H + h) * S + t] * 1.4426950408889634f;
      if (t == S - 1)
        for (int tp = S; tp < S_pad; ++tp) { delta[o + tp - t] = 0.f; lse2[o + tp - t] = 0.f; }
    }
  }
}

// ------------------------------------------------------------------ dK, dV
template <typename T, int DN, int DR, int DV, int BQ, int WPH>
__global__ __launch_bounds__(64 * WPH) void dkdv_kernel(BwdParams P) {
  constexpr int DQK = DN + DR, DKVH = DN + DV, DQK32 = round32(DQK);
  constexpr int NT = 64 * WPH, BK = 32 * WPH, E = Elems16<T>::n;
  constexpr int PQ = lds_pitch<T>(DQK32), PO = lds_pitch<T>(DV);
  constexpr int QCH = DQK / E, OCH = DV / E;                 // chunks per row
  constexpr int TILE_CHUNKS = BQ * (QCH + OCH);
  constexpr int PER_THREAD = (TILE_CHUNKS + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) T sQ[BQ * PQ];
  __shared__ __attribute__((aligned(16))) T sO[BQ * PO];
  __shared__ __attribute__((aligned(16))) float sL[BQ];
  __shared__ __attribute__((aligned(16))) float sD[BQ];

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

  // zero the padding columns [DQK, DQK32) once: transposing reads of Q^T blocks touch them
  if (DQK32 > DQK)
    for (int i = tid; i < BQ * (DQK32 - DQK); i += NT)
      sQ[(i / (DQK32 - DQK)) * PQ + DQK + i % (DQK32 - DQK)] = to_elem<T>(0.f);

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

  chunk16 stage[PER_THREAD];
  float st_l = 0.f, st_d = 0.f;
  auto load_tile = [&](int qt) {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int c = tid + i * NT;
      stage[i] = zero_chunk();
      if (c < TILE_CHUNKS) {
        const int row = c / (QCH + OCH), j = c % (QCH + OCH);
        const int qi = qt + row;
        if (qi < S) {
          const size_t base = (size_t)(b * S + qi) * H + h;
          stage[i] = j < QCH ? *reinterpret_cast<const chunk16*>(q + base * DQK + j * E)
                             : *reinterpret_cast<const chunk16*>(dout + base * DV + (j - QCH) * E);
        }
      }
    }
    if (tid < BQ) {
      const int qi = qt + tid;
      st_l = qi < S ? P.lse2[(size_t)(b * H + h) * P.S_pad + qi] : 0.f;
      st_d = qi < S ? P.delta[(size_t)(b * H + h) * P.S_pad + qi] : 0.f;
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int c = tid + i * NT;
      if (c < TILE_CHUNKS) {
        const int row = c / (QCH + OCH), j = c % (QCH + OCH);
        T* dst = j < QCH ? sQ + row * PQ + j * E : sO + row * PO + (j - QCH) * E;
        *reinterpret_cast<chunk16*>(dst) = stage[i];
      }
    }
    if (tid < BQ) { sL[tid] = st_l; sD[tid] = st_d; }
  };

  const int qt_begin = P.causal ? (kb * BK) / BQ * BQ : 0;
  load_tile(qt_begin);
  for (int qt = qt_begin; qt < S; qt += BQ) {
    __syncthreads();
    store_tile();
    __syncthreads();
    if (qt + BQ < S) load_tile(qt + BQ);

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


// Key-stationary backward, bf16 with 192/128-wide heads: the query tiles (Q, dO and
// the per-row lse2 / delta) stream through a two-stage LDS ring filled by direct
// global->LDS loads into swizzled, unpadded tiles, so no registers are spent on
// staging and one barrier per tile suffices. Math as in dkdv_kernel.
template <int DN, int DR, int DV, int WPH>
__global__ __launch_bounds__(64 * WPH) void dkdv_ring_kernel(BwdParams P) {
  using T = bf16;
  constexpr int DQK = DN + DR, DKVH = DN + DV, BQ = 32, NW = WPH, BK = 32 * WPH;
  constexpr int QCPR = DQK / 8, OCPR = DV / 8;  // 16-byte chunks per row
  static_assert(QCPR == 24 && OCPR == 16, "swizzles are defined for 192/128-wide rows");
  __shared__ __attribute__((aligned(16))) T sQ[2][BQ * DQK];
  __shared__ __attribute__((aligned(16))) T sO[2][BQ * DV];
  __shared__ __attribute__((aligned(16))) float sLD[2][2 * BQ];  // lse2 then delta

  const T* __restrict__ q = (const T*)P.q;
  const T* __restrict__ kpe = (const T*)P.k_pe;
  const T* __restrict__ kv = (const T*)P.kv;
  const T* __restrict__ dout = (const T*)P.dout;
  const int S = P.S, H = P.H;

  const int total = P.n_blocks * H * gridDim.y;
  const int lin = xcd_remap(blockIdx.x + gridDim.x * blockIdx.y, total);
  const int kb = lin % P.n_blocks;
  const int bh = lin / P.n_blocks;
  const int b = bh / H, h = bh % H;

  const int tid = threadIdx.x, wave = tid >> 6, l = tid & 63, n = l & 31, g = l >> 5;
  const int k0 = kb * BK + wave * 32;
  const int my_k = k0 + n;

  frag_t<T> kf[DQK / 16], vf[DV / 16];
  {
    const bool ok = my_k < S;
    const size_t row = (size_t)(b * S + (ok ? my_k : 0));
    const T* kvr = kv + (row * H + h) * DKVH;
#pragma unroll
    for (int ks = 0; ks < DQK / 16; ++ks) {
      const T* src = ks < DN / 16 ? kvr + ks * 16 + 8 * g : kpe + row * DR + (ks - DN / 16) * 16 + 8 * g;
      kf[ks] = *reinterpret_cast<const frag_t<T>*>(src);
      if (!ok) kf[ks] = frag_t<T>{};
    }
#pragma unroll
    for (int ks = 0; ks < DV / 16; ++ks) {
      vf[ks] = *reinterpret_cast<const frag_t<T>*>(kvr + DN + ks * 16 + 8 * g);
      if (!ok) vf[ks] = frag_t<T>{};
    }
  }

  f32x16 dk[DQK / 32], dv[DV / 32];
#pragma unroll
  for (int i = 0; i < DQK / 32; ++i) dk[i] = f32x16{};
#pragma unroll
  for (int i = 0; i < DV / 32; ++i) dv[i] = f32x16{};

  const size_t hrow = (size_t)(b * H + h) * P.S_pad;
  auto fill = [&](int stage, int qt) {
    // rows past S are clamped to S-1 (valid memory); their P is masked to zero
    swz_fill<T, BQ, QCPR, NW>(sQ[stage], wave, l, [&](int r) {
      const int qi = min(qt + r, S - 1);
      return q + ((size_t)(b * S + qi) * H + h) * DQK;
    });
    swz_fill<T, BQ, OCPR, NW>(sO[stage], wave, l, [&](int r) {
      const int qi = min(qt + r, S - 1);
      return dout + ((size_t)(b * S + qi) * H + h) * DV;
    });
    if (wave == NW - 1 && l < 2 * BQ / 4) {  // 8 chunks of lse2, then 8 of delta (padded rows)
      const float* src = l < BQ / 4 ? P.lse2 + hrow + qt + 4 * l : P.delta + hrow + qt + 4 * (l - BQ / 4);
      g2lds16(src, &sLD[stage][0]);
    }
  };

  const int qt_begin = P.causal ? (kb * BK) / BQ * BQ : 0;
  fill(0, qt_begin);
  int it = 0;
  for (int qt = qt_begin; qt < S; qt += BQ, ++it) {
    const int st = it & 1;
    wait_vmem();      // this wave's part of tile `it` has landed
    __syncthreads();  // all parts landed; everyone is done with the other stage
    if (qt + BQ < S) fill(st ^ 1, qt + BQ);

    // waves whose keys all lie after this tile's queries run it fully masked (P = 0):
    // keeping the loop body free of per-wave branches keeps the accumulators in place
    const bool need_mask = (P.causal && qt < k0 + 31) || (qt + BQ > S);
    const T* tq = sQ[st];
    const T* to = sO[st];

    f32x16 sa{}, dp{};
#pragma unroll
    for (int ks = 0; ks < DQK / 16; ++ks) mma(sa, swz_frag<T, QCPR>(tq, n, 2 * ks + g), kf[ks]);
#pragma unroll
    for (int ks = 0; ks < DV / 16; ++ks) mma(dp, swz_frag<T, OCPR>(to, n, 2 * ks + g), vf[ks]);
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int qrow = rr * 8 + g * 4;
      const f32x4 lq = *reinterpret_cast<const f32x4*>(&sLD[st][qrow]);
      const f32x4 dq = *reinterpret_cast<const f32x4*>(&sLD[st][BQ + qrow]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = rr * 4 + e;
        float p = fast_exp2(sa[r] * P.scale_log2 - lq[e]);
        if (need_mask) {
          const int qi = qt + qrow + e;
          if (qi >= S || (P.causal && my_k > qi)) p = 0.f;
        }
        sa[r] = p;
        dp[r] = p * (dp[r] - dq[e]);
      }
    }
#pragma unroll
    for (int kk = 0; kk < BQ / 16; ++kk) {
      const frag_t<T> pf = acc_to_frag<T>(sa, kk);
      const frag_t<T> zf = acc_to_frag<T>(dp, kk);
      const int ra = kk * 16 + 4 * g;
#pragma unroll
      for (int db = 0; db < DV / 32; ++db) mma(dv[db], swz_tr_frag<OCPR>(to, ra, ra + 8, db * 32), pf);
#pragma unroll
      for (int db = 0; db < DQK / 32; ++db) mma(dk[db], swz_tr_frag<QCPR>(tq, ra, ra + 8, db * 32), zf);
    }
  }

  if (my_k >= S) return;
  const size_t row = (size_t)(b * S + my_k) * H + h;
  T* dkvr = (T*)P.dkv + row * DKVH;
  T* dkvl = (T*)P.dkv_lo + row * DKVH;
  float* dper = P.dkpe_h + row * DR;
  auto put4 = [&](int col, float a0, float a1, float a2, float a3) {
    bf16x4 hi = {to_elem<T>(a0), to_elem<T>(a1), to_elem<T>(a2), to_elem<T>(a3)};
    bf16x4 lo = {to_elem<T>(a0 - to_f32(hi[0])), to_elem<T>(a1 - to_f32(hi[1])), to_elem<T>(a2 - to_f32(hi[2])),
                 to_elem<T>(a3 - to_f32(hi[3]))};
    *reinterpret_cast<bf16x4*>(dkvr + col) = hi;
    *reinterpret_cast<bf16x4*>(dkvl + col) = lo;
  };
#pragma unroll
  for (int db = 0; db < DQK / 32; ++db)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int d = db * 32 + rr * 8 + g * 4;
      const float a0 = dk[db][4 * rr] * P.scale, a1 = dk[db][4 * rr + 1] * P.scale;
      const float a2 = dk[db][4 * rr + 2] * P.scale, a3 = dk[db][4 * rr + 3] * P.scale;
      if (d < DN) {
        put4(d, a0, a1, a2, a3);
      } else {
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

// dk_pe[b,t,:] = sum_{h ascending} dkpe_h[b,t,h,:]   (one thread per 4 outputs, fp32)
template <int DR>
__global__ __launch_bounds__(256) void dkpe_kernel(const float* __restrict__ part, float* __restrict__ dkpe, int H,
                                                   int n4) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= n4) return;
  const int bt = i / (DR / 4), c = (i % (DR / 4)) * 4;
  const float* src = part + (size_t)bt * H * DR + c;
  f32x4 s = *reinterpret_cast<const f32x4*>(src);
  for (int h = 1; h < H; ++h) s += *reinterpret_cast<const f32x4*>(src + (size_t)h * DR);
  *reinterpret_cast<f32x4*>(dkpe + (size_t)bt * DR + c) = s;
}

template <typename T> struct BwdTiles;
template <> struct BwdTiles<bf16> { static constexpr int BQ = 32, BC = 64, WPH_KV = 4, WPH_Q = 4; };
template <> struct BwdTiles<float> { static constexpr int BQ = 32, BC = 32, WPH_KV = 4, WPH_Q = 4; };

}  // namespace

template <typename T, int DN, int DR, int DV>
hipError_t launch_attn_bwd(const AttnBwdArgs& a, int stage, hipStream_t st) {
  using Tl = BwdTiles<T>;
  BwdParams P;
  P.q = a.q; P.k_pe = a.k_pe; P.kv = a.kv; P.dout = a.dout; P.lse = a.lse; P.delta = a.delta;
  P.lse2 = a.lse2; P.S_pad = a.S_pad;
  P.dq = a.dq; P.dkv = a.dkv; P.dkv_lo = a.dkv_lo; P.dkpe_h = a.dkpe_h;
  P.S = a.S; P.H = a.H; P.scale = a.scale; P.scale_log2 = a.scale * 1.4426950408889634f; P.causal = a.causal;
  if (stage == 0) {
    const int BS = a.B * a.S;
    delta_kernel<T, DV><<<(BS + 3) / 4, 256, 0, st>>>((const T*)a.out, (const T*)a.dout, a.lse, a.delta, a.lse2,
                                                      a.S, a.S_pad, a.H, BS);
  } else if (stage == 1) {
    constexpr int BK = 32 * Tl::WPH_KV;
    P.n_blocks = (a.S + BK - 1) / BK;
    if constexpr (sizeof(T) == 2 && DN + DR == 192 && DV == 128)
      dkdv_ring_kernel<DN, DR, DV, Tl::WPH_KV><<<dim3(P.n_blocks * a.H, a.B), 64 * Tl::WPH_KV, 0, st>>>(P);
    else
      dkdv_kernel<T, DN, DR, DV, Tl::BQ, Tl::WPH_KV><<<dim3(P.n_blocks * a.H, a.B), 64 * Tl::WPH_KV, 0, st>>>(P);
  } else if (stage == 2) {
    constexpr int BR = 32 * Tl::WPH_Q;
    P.n_blocks = (a.S + BR - 1) / BR;
    dq_kernel<T, DN, DR, DV, Tl::BC, Tl::WPH_Q><<<dim3(P.n_blocks * a.H, a.B), 64 * Tl::WPH_Q, 0, st>>>(P);
  } else {
    const int n4 = a.B * a.S * DR / 4;
    dkpe_kernel<DR><<<(n4 + 255) / 256, 256, 0, st>>>(a.dkpe_h, a.dk_pe, a.H, n4);
  }
  return hipGetLastError();
}

#define LAGA_INST_BWD(T, DN, DR, DV) template hipError_t launch_attn_bwd<T, DN, DR, DV>(const AttnBwdArgs&, int, hipStream_t);
LAGA_INST_BWD(bf16, 128, 64, 128)
LAGA_INST_BWD(float, 128, 64, 128)
LAGA_INST_BWD(bf16, 32, 16, 32)
LAGA_INST_BWD(float, 32, 16, 32)

}  // namespace laga
