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
#include <type_traits>

// direct global->LDS copies issued as inline assembly (exact LDS-read waits; the
// rings order the copies with explicit waits and barriers)
#define LAGA_LDS_DMA_ASM 1
#include "common.hpp"
#include "kernels.hpp"
#include "bwd_common.hpp"

namespace laga {

using namespace bwd;

namespace {

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


// Key-stationary backward with 16 keys per wave on the 16x16x32 MFMA: the per-wave
// state (K and V rows 40 registers, dK^T / dV^T accumulators 80) is half that of
// the 32-key layout, so two waves share each SIMD and hide each other's latencies.
// (Measured alternatives at S = 16384, this kernel 3.2-3.3 ms: 32 keys per wave on the
// 32x32x16 MFMA at one wave per SIMD, 4.5 ms as a plain loop and 3.1-3.3 ms software-
// pipelined with every LDS read at an immediate offset; a pair of waves splitting 32
// keys into a K role and a V role, 3.1 ms. Those two read fewer LDS bytes per pair,
// but in the whole step the other kernels then ran slower by as much, the board being
// at its power limit.)
// A workgroup of WPH waves owns 16 * WPH keys of one head; query tiles of 32 rows
// (Q, dO, and lse2 / delta of the rows) stream through a two-stage LDS ring of direct
// global->LDS loads into padded tiles (pitch = row + 2 chunks: conflict-free for both
// 16x16 read patterns, and every read is a per-lane base address plus a constant).
//   S = Q K^T, dP = dO V^T: A = Q / dO rows (16-byte row fragments), B = the lane's
//       key / value row; accumulator: lane <-> key, 4 queries per 16-query block.
//   dV^T += dO^T P, dK^T += Q^T dZ: the contraction over the tile's 32 queries takes
//       P / dZ straight from the accumulators in the order {4G..4G+3, 16+4G..16+4G+3}
//       (G = lane / 16), matched by two transposing 4-row reads of dO / Q.
// Alongside, dS^T = dZ (bf16) is stored for the dQ pass.
template <int DN, int DR, int DV, int WPH, int NS>
__global__ __launch_bounds__(64 * WPH) void dkdv16_kernel(BwdParams P) {
  using T = bf16;
  constexpr int DQK = DN + DR, DKVH = DN + DV, BQ = 32, NW = WPH, BK = 16 * WPH;
  constexpr int QCPR = DQK / 8, OCPR = DV / 8;
  static_assert(QCPR % 4 == 0 && OCPR % 4 == 0, "padded pitches assume rows of whole 64-byte groups");
  static_assert(NS == 2, "two-stage ring (the waits are full vmcnt waits)");
  constexpr int QP = QCPR + 2, OP = OCPR + 2;  // pitches in chunks, P % 4 == 2
  constexpr int NQI = pad_chunks(BQ, QP) / 64, NOI = pad_chunks(BQ, OP) / 64;
  static_assert(NQI * 64 == BQ * QP && NOI * 64 == BQ * OP, "tiles are whole load instructions");
  // ring stages as distinct LDS objects (so the compiler does not make the reads of one
  // stage wait for the direct loads into another); unused stages are not allocated
  __shared__ __attribute__((aligned(16))) T sQ0[NQI * 512], sQ1[NQI * 512], sQ2[NQI * 512], sQ3[NQI * 512];
  __shared__ __attribute__((aligned(16))) T sO0[NOI * 512], sO1[NOI * 512], sO2[NOI * 512], sO3[NOI * 512];
  // lse2 of the tile's rows, then delta (the load instruction covers 1 KB; lanes 16..63
  // repeat lanes 0..15)
  __shared__ __attribute__((aligned(16))) float sL0[256], sL1[256], sL2[256], sL3[256];

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

  const int tid = threadIdx.x, l = tid & 63, j = l & 15, G = l >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) & (NW - 1);  // uniform, known < NW
  const int k0 = kb * BK + wave * 16;
  const int my_k = k0 + j;

  bf16x8 kf[DQK / 32], vf[DV / 32];
  {
    const bool ok = my_k < S;
    const size_t row = (size_t)(b * S + (ok ? my_k : 0));
    const T* kvr = kv + (row * H + h) * DKVH;
#pragma unroll
    for (int ks = 0; ks < DQK / 32; ++ks) {
      const int d = ks * 32 + G * 8;
      const T* src = d < DN ? kvr + d : kpe + row * DR + (d - DN);
      kf[ks] = *reinterpret_cast<const bf16x8*>(src);
      if (!ok) kf[ks] = bf16x8{};
    }
#pragma unroll
    for (int ks = 0; ks < DV / 32; ++ks) {
      vf[ks] = *reinterpret_cast<const bf16x8*>(kvr + DN + ks * 32 + G * 8);
      if (!ok) vf[ks] = bf16x8{};
    }
  }

  f32x4 dk[DQK / 16], dv[DV / 16];
#pragma unroll
  for (int i = 0; i < DQK / 16; ++i) dk[i] = f32x4{};
#pragma unroll
  for (int i = 0; i < DV / 16; ++i) dv[i] = f32x4{};

  // Loads of a tile: Q chunks (instruction js of NQI goes to wave js % NW), dO chunks
  // likewise, and the lse2 / delta rows in one instruction of wave NW - 1. Each lane
  // keeps its source pointer for the tile at query 0, and a tile adds qt rows (one
  // 64-bit add); which instructions a wave issues is fixed, so the dispatch is a few
  // scalar compares. A tile crossing the end of the data (rows past S, clamped to
  // S - 1; their P is masked) takes a slower path.
  constexpr int KQ = (NQI + NW - 1) / NW, KO = (NOI + NW - 1) / NW;
  auto q_chunk = [&](int js, int rmax) {  // element offset of this lane's Q chunk from row 0
    const int p = js * 64 + l, r = min(p / QP, rmax), c = p % QP;
    return r * H * DQK + (c < QCPR ? c : 0) * 8;
  };
  auto o_chunk = [&](int js, int rmax) {
    const int p = js * 64 + l, r = min(p / OP, rmax), c = p % OP;
    return r * H * DV + (c < OCPR ? c : 0) * 8;
  };
  const size_t hrow0 = (size_t)(b * S) * H + h;  // row (b, 0, h)
  const T* qlane[KQ];
  const T* olane[KO];
#pragma unroll
  for (int k = 0; k < KQ; ++k) qlane[k] = q + hrow0 * DQK + q_chunk(wave + k * NW, BQ - 1);
#pragma unroll
  for (int k = 0; k < KO; ++k) olane[k] = dout + hrow0 * DV + o_chunk(wave + k * NW, BQ - 1);
  const float* llane = (j < 8 ? P.lse2 : P.delta) + (size_t)(b * H + h) * P.S_pad + 4 * (j & 7);

  auto fill = [&](T* tq, T* to, float* tl, int qt) {
    const size_t qstep = (size_t)qt * H;
    if (qt + BQ <= S) {
#pragma unroll
      for (int k = 0; k < KQ; ++k)
        if (wave + k * NW < NQI) g2lds16(qlane[k] + qstep * DQK, tq + (wave + k * NW) * 512);
#pragma unroll
      for (int k = 0; k < KO; ++k)
        if (wave + k * NW < NOI) g2lds16(olane[k] + qstep * DV, to + (wave + k * NW) * 512);
    } else {
      const T* qb = q + (hrow0 + qstep) * DQK;
      const T* ob = dout + (hrow0 + qstep) * DV;
#pragma unroll
      for (int k = 0; k < KQ; ++k)
        if (wave + k * NW < NQI) g2lds16(qb + q_chunk(wave + k * NW, S - 1 - qt), tq + (wave + k * NW) * 512);
#pragma unroll
      for (int k = 0; k < KO; ++k)
        if (wave + k * NW < NOI) g2lds16(ob + o_chunk(wave + k * NW, S - 1 - qt), to + (wave + k * NW) * 512);
    }
    if (wave == NW - 1) g2lds16(llane + qt, tl);
  };

  // dS^T of a tile for the dQ pass: key my_k's row of 32 queries; the lane holds
  // queries {4G..4G+3} and {16+4G..16+4G+3}. Only the keys the tile sees are stored.
  // The store of tile i is issued right after the barrier of tile i + 1, so its
  // latency hides behind a whole tile. dsl: this key's row in query tile 0.
  T* const dsl = (T*)P.ds + ds_tile_offset(P.ds_T, P.causal, bh, 0) + (size_t)my_k * BQ;
  bf16x8 zs{};
  int ts = -1;
  auto store_ds = [&]() {
    if (ts >= 0 && my_k < ds_tile_keys(P.ds_T, P.causal, ts)) {
      T* dsr = dsl + (P.causal ? (size_t)512 * ts * (ts + 1) : (size_t)1024 * P.ds_T * ts);
      *reinterpret_cast<bf16x4*>(dsr + 4 * G) = __builtin_shufflevector(zs, zs, 0, 1, 2, 3);
      *reinterpret_cast<bf16x4*>(dsr + 16 + 4 * G) = __builtin_shufflevector(zs, zs, 4, 5, 6, 7);
    }
  };

  // live (query, key) pairs of this lane's key: q_lo <= query < q_lo + q_span (none
  // for keys past S), tested with one unsigned compare
  const int q_lo = P.causal ? my_k : 0;
  const unsigned q_span = my_k < S ? (unsigned)(S - q_lo) : 0u;

  const int qt_begin = P.causal ? (kb * BK) / BQ * BQ : 0;
  const int ntiles = (S - qt_begin + BQ - 1) / BQ;
  auto stage_q = [&](auto st) -> T* {
    constexpr int X = decltype(st)::value;
    return X == 0 ? sQ0 : X == 1 ? sQ1 : X == 2 ? sQ2 : sQ3;
  };
  auto stage_o = [&](auto st) -> T* {
    constexpr int X = decltype(st)::value;
    return X == 0 ? sO0 : X == 1 ? sO1 : X == 2 ? sO2 : sO3;
  };
  auto stage_l = [&](auto st) -> float* {
    constexpr int X = decltype(st)::value;
    return X == 0 ? sL0 : X == 1 ? sL1 : X == 2 ? sL2 : sL3;
  };
  {
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    fill(stage_q(I0{}), stage_o(I0{}), stage_l(I0{}), qt_begin);
    if (NS > 2 && ntiles > 1) fill(stage_q(I1{}), stage_o(I1{}), stage_l(I1{}), qt_begin + BQ);
    if (NS > 3 && ntiles > 2) fill(stage_q(I2{}), stage_o(I2{}), stage_l(I2{}), qt_begin + 2 * BQ);
  }
  auto step = [&](auto stage, int it) {
    constexpr int ST = decltype(stage)::value;
    using NX = std::integral_constant<int, (ST + NS - 1) % NS>;
    const int qt = qt_begin + it * BQ;
    // this wave's loads of tile `it` have landed: in the steady state exactly the
    // NS - 2 later tiles' loads may still be in flight
    wait_vmem();
    __syncthreads();  // ... and everyone's; the stage filled next (read at it - 1) is free
    store_ds();       // tile it - 1
    if (it + NS - 1 < ntiles) fill(stage_q(NX{}), stage_o(NX{}), stage_l(NX{}), qt + (NS - 1) * BQ);
    const T* tq = stage_q(stage);
    const T* to = stage_o(stage);
    const float* tld = stage_l(stage);
    // masked: queries past S, keys past S (their dS is stored as zeros) and, causally,
    // keys after the query
    const bool need_mask = (P.causal && qt < k0 + 15) || (qt + BQ > S) || (k0 + 16 > S);

    f32x4 sa[2], dp[2];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      sa[qb] = f32x4{};
      dp[qb] = f32x4{};
#pragma unroll
      for (int ks = 0; ks < DQK / 32; ++ks) mma16(sa[qb], pad_frag<QP>(tq, qb * 16 + j, 4 * ks + G), kf[ks]);
#pragma unroll
      for (int ks = 0; ks < DV / 32; ++ks) mma16(dp[qb], pad_frag<OP>(to, qb * 16 + j, 4 * ks + G), vf[ks]);
    }
    if (need_mask) {
      asm volatile("");  // keep the branch: the common unmasked tile runs no mask code
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          sa[qb][e] = (unsigned)(qt + qb * 16 + G * 4 + e - q_lo) < q_span ? sa[qb][e] : -INFINITY;
    }
    bf16x8 pf, zf;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      const int qrow = qb * 16 + G * 4;
      const f32x4 lq = *reinterpret_cast<const f32x4*>(tld + qrow);
      const f32x4 dq = *reinterpret_cast<const f32x4*>(tld + BQ + qrow);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float p = fast_exp2(__builtin_fmaf(sa[qb][e], P.scale_log2, -lq[e]));
        pf[qb * 4 + e] = to_elem<T>(p);
        zf[qb * 4 + e] = to_elem<T>(p * (dp[qb][e] - dq[e]));
      }
    }
    zs = zf;
    ts = qt / BQ;
    const int ra = 4 * G, rb = 16 + 4 * G;
#pragma unroll
    for (int db = 0; db < DV / 16; ++db) mma16(dv[db], pad_tr_frag16<OP>(to, ra, rb, db * 16), pf);
#pragma unroll
    for (int db = 0; db < DQK / 16; ++db) mma16(dk[db], pad_tr_frag16<QP>(tq, ra, rb, db * 16), zf);
  };
  for (int it = 0; it < ntiles; it += NS) {
    step(std::integral_constant<int, 0>{}, it);
    if (it + 1 < ntiles) step(std::integral_constant<int, 1 % NS>{}, it + 1);
    if (NS > 2 && it + 2 < ntiles) step(std::integral_constant<int, 2 % NS>{}, it + 2);
    if (NS > 3 && it + 3 < ntiles) step(std::integral_constant<int, 3 % NS>{}, it + 3);
  }
  store_ds();  // the last tile

  if (my_k >= S) return;
  const size_t row = (size_t)(b * S + my_k) * H + h;
  T* dkvr = (T*)P.dkv + row * DKVH;
  T* dkvl = (T*)P.dkv_lo + row * DKVH;
  float* dper = P.dkpe_h + row * DR;
  auto put4 = [&](int col, const f32x4& a, float sc) {
    bf16x4 hi, lo;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float x = a[e] * sc;
      hi[e] = to_elem<T>(x);
      lo[e] = to_elem<T>(x - to_f32(hi[e]));
    }
    *reinterpret_cast<bf16x4*>(dkvr + col) = hi;
    *reinterpret_cast<bf16x4*>(dkvl + col) = lo;
  };
#pragma unroll
  for (int db = 0; db < DQK / 16; ++db) {
    const int d = db * 16 + G * 4;
    if (d < DN) {
      put4(d, dk[db], P.scale);
    } else {
      f32x4 v = dk[db] * P.scale;
      *reinterpret_cast<f32x4*>(dper + (d - DN)) = v;
    }
  }
#pragma unroll
  for (int db = 0; db < DV / 16; ++db) put4(DN + db * 16 + G * 4, dv[db], 1.f);
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

}  // namespace

template <typename T, int DN, int DR, int DV>
hipError_t launch_attn_bwd(const AttnBwdArgs& a, int stage, hipStream_t st) {
  using Tl = BwdTiles<T>;
  BwdParams P;
  P.q = a.q; P.k_pe = a.k_pe; P.kv = a.kv; P.dout = a.dout; P.lse = a.lse; P.delta = a.delta;
  P.lse2 = a.lse2; P.S_pad = a.S_pad;
  P.dq = a.dq; P.dkv = a.dkv; P.dkv_lo = a.dkv_lo; P.dkpe_h = a.dkpe_h;
  P.S = a.S; P.H = a.H; P.scale = a.scale; P.scale_log2 = a.scale * 1.4426950408889634f; P.causal = a.causal;
  P.ds = a.ds; P.ds_T = (a.S + 31) / 32;
  if (stage == 0) {
    const int BS = a.B * a.S;
    delta_kernel<T, DV><<<(BS + 3) / 4, 256, 0, st>>>((const T*)a.out, (const T*)a.dout, a.lse, a.delta, a.lse2,
                                                      a.S, a.S_pad, a.H, BS);
  } else if (stage == 1) {
    if constexpr (sizeof(T) == 2 && DN + DR == 192 && DV == 128) {
      // two stages: three and four measured 25 % and 17 % slower at S = 16384 (the
      // loads are mostly cache hits that one tile of compute covers; more stages cost
      // code size and scalar registers)
      constexpr int WPH16 = 8, BK = 16 * WPH16, NS = 2;
      P.n_blocks = (a.S + BK - 1) / BK;
      dkdv16_kernel<DN, DR, DV, WPH16, NS><<<dim3(P.n_blocks * a.H, a.B), 64 * WPH16, 0, st>>>(P);
    } else {
      constexpr int BK = 32 * Tl::WPH_KV;
      P.n_blocks = (a.S + BK - 1) / BK;
      dkdv_kernel<T, DN, DR, DV, Tl::BQ, Tl::WPH_KV><<<dim3(P.n_blocks * a.H, a.B), 64 * Tl::WPH_KV, 0, st>>>(P);
    }
  } else if (stage == 2) {
    return launch_bwd_dq<T, DN, DR, DV>(P, a.B, st);
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
