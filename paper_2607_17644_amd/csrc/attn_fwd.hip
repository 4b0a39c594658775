// Causal MLA flash-attention forward for one rank's head shard (Alg. 1 step 5),
// with the per-head K/V either read from the materialised kv (Alg. 1 step 4
// done beforehand) or rebuilt tile by tile on chip from the latent (fused).
//
// Work decomposition: a workgroup owns G heads x (32 * WPH) queries; wave w
// serves head (w / WPH) and 32 consecutive queries. Key tiles of BC keys are
// staged in LDS: per head K_nope [BC, DN] and V [BC, DV], plus ONE k_pe tile
// [BC, DR] that every head of the workgroup reads (k_pe is shared by all heads,
// property P2 of Section 2.1).
//
// Everything is computed transposed so that a lane owns one query:
//   S^T = K Q^T    (A = K tile rows from LDS, B = the wave's queries in registers)
//   O^T += V^T P^T (A = V tile read with transposing LDS reads, B = P from the
//                   S^T accumulators, no data movement)
// The accumulator of S^T gives lane l the 16 keys (r/4)*8 + g*4 + r%4 of query
// l % 32 (g = l / 32), so the row max / row sum of the online softmax are
// in-lane reductions plus one exchange between lane halves, and the rescale of
// O^T (also lane-per-query) needs no shuffles at all. Softmax runs in base 2
// with log2(e) folded into the scale; lse is returned in natural log.
#include <type_traits>

// direct global->LDS copies issued as inline assembly: LDS reads then get exact waits
// (every ring here orders its copies with an explicit vmcnt wait and a barrier)
#define LAGA_LDS_DMA_ASM 1
#include "common.hpp"
#include "kernels.hpp"

namespace laga {

namespace {

template <typename T, int DN, int DR, int DV, int BC, int WPH, int G, bool FUSED>
struct FwdCfg {
  static constexpr int DQK = DN + DR;
  static constexpr int DKVH = DN + DV;
  static constexpr int NT = 64 * WPH * G;  // threads
  static constexpr int BR = 32 * WPH;      // queries per head per workgroup
  static constexpr int E = Elems16<T>::n;
  static constexpr int PK = DN + 8;   // K_nope pitch (16-byte fragment reads)
  static constexpr int PP = DR + 8;   // k_pe pitch
  static constexpr int PV = DV + 32 / (int)sizeof(T);  // V pitch (transposing reads)
  static constexpr int LDS_K = G * BC * PK;
  static constexpr int LDS_P = BC * PP;
  static constexpr int LDS_V = G * BC * PV;
  static constexpr int ROW_CHUNKS = (G * DKVH + DR) / E;  // 16-byte chunks per key row
  static constexpr int TILE_CHUNKS = BC * ROW_CHUNKS;
  static constexpr int PER_THREAD = (TILE_CHUNKS + NT - 1) / NT;
  static_assert(DN % 16 == 0 && DR % 16 == 0 && DV % 32 == 0 && BC % 32 == 0, "tile shape");
};

struct FwdParams {
  const void* q;
  const void* k_pe;
  const void* kv;
  void* out;
  float* lse;
  int S, H, n_qblocks, n_hgroups;
  float scale_log2;  // softmax_scale * log2(e)
  int causal;
};

// One key tile of the online-softmax forward for one wave (32 queries, one head):
// S^T = K Q^T from the LDS K_nope / k_pe tiles, masked base-2 softmax update of
// (m, lsum, O^T), then O^T += V^T P^T with V^T read by transposing LDS reads.
template <typename T, int DN, int DR, int DV, int BC>
__device__ __forceinline__ void fwd_tile(const T* sKh, int PK, const T* sP, int PP, const T* sVh, int PV,
                                         const frag_t<T> (&qf)[(DN + DR) / 16], f32x16 (&oacc)[DV / 32], float& m,
                                         float& lsum, int kt, int q0, int my_q, int S, float scale_log2, int causal,
                                         bool head_ok) {
  constexpr int DQK = DN + DR;
  const int l = threadIdx.x & 63, n = l & 31, g = l >> 5;
  const bool active = head_ok && q0 < S && (!causal || kt <= q0 + 31);
  if (!active) return;

  f32x16 sacc[BC / 32];
#pragma unroll
  for (int kb = 0; kb < BC / 32; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) sacc[kb][r] = 0.f;
#pragma unroll
  for (int ks = 0; ks < DQK / 16; ++ks)
#pragma unroll
    for (int kb = 0; kb < BC / 32; ++kb) {
      const frag_t<T> a = ks < DN / 16
          ? lds_frag<T>(sKh + (kb * 32 + n) * PK + ks * 16 + 8 * g)
          : lds_frag<T>(sP + (kb * 32 + n) * PP + (ks - DN / 16) * 16 + 8 * g);
      mma(sacc[kb], a, qf[ks]);
    }

  // mask (only tiles crossing the diagonal or the end), running max on the raw scores
  // (scale > 0), p = exp2(s * scale_log2 - m) as one FMA + v_exp_f32, O rescaled only
  // when some lane's max moved: the same arithmetic, in the same order, as the ring
  // kernel, so the two forward kernels agree bit for bit
  const bool need_mask = (causal && kt + BC - 1 > q0) || (kt + BC > S);
  if (need_mask) {
    asm volatile("");  // keep the branch (see the ring kernel)
    // live keys: key < klim, i.e. accumulator row (r/4)*8 + r%4 + 32 kb < klim - kt - 4 g
    const int lim = (causal ? min(S, my_q + 1) : S) - kt - 4 * g;
#pragma unroll
    for (int kb = 0; kb < BC / 32; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        sacc[kb][r] = kb * 32 + (r >> 2) * 8 + (r & 3) < lim ? sacc[kb][r] : -INFINITY;
  }
  float mraw = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < BC / 32; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) mraw = fmaxf(mraw, sacc[kb][r]);
  mraw = wave_xor32_max(mraw);
  const float m_new = fmaxf(m, mraw * scale_log2);
  // lazy rescale: the reference max m moves only when a score exceeds it by more
  // than 2^kRescaleLog2 (until then p <= 2^kRescaleLog2), so O^T is rarely rescaled;
  // the normalised result is the same
  const bool bump = m_new > m + kRescaleLog2;
  const float m_ref = bump ? m_new : m;
  const float alpha = bump ? fast_exp2(m - m_new) : 1.f;
  const float m_use = m_ref == -INFINITY ? 0.f : m_ref;
  float ps = 0.f;
#pragma unroll
  for (int kb = 0; kb < BC / 32; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float p = fast_exp2(__builtin_fmaf(sacc[kb][r], scale_log2, -m_use));
      sacc[kb][r] = p;
      ps += p;
    }
  lsum = lsum * alpha + ps;
  m = m_ref;
  if (__ballot(bump)) {
#pragma unroll
    for (int i = 0; i < DV / 32; ++i) oacc[i] *= alpha;
  }

  frag_t<T> pf[BC / 16];
#pragma unroll
  for (int kk = 0; kk < BC / 16; ++kk) pf[kk] = acc_to_frag<T>(sacc[kk >> 1], kk & 1);
#pragma unroll
  for (int kk = 0; kk < BC / 16; ++kk)
#pragma unroll
    for (int db = 0; db < DV / 32; ++db) {
      const int ra = kk * 16 + 4 * g;
      const frag_t<T> a = TrRead<T>::get(sVh, PV, ra, ra + 8, db * 32);
      mma(oacc[db], a, pf[kk]);
    }
}

template <typename T, int DN, int DR, int DV, int BC, int WPH, int G, bool FUSED>
__global__ __launch_bounds__(64 * WPH * G)
void attn_fwd_kernel(FwdParams P) {
  using C = FwdCfg<T, DN, DR, DV, BC, WPH, G, FUSED>;
  constexpr int DQK = C::DQK, DKVH = C::DKVH, E = C::E;
  __shared__ __attribute__((aligned(16))) T sK[C::LDS_K];
  __shared__ __attribute__((aligned(16))) T sP[C::LDS_P];
  __shared__ __attribute__((aligned(16))) T sV[C::LDS_V];

  const T* __restrict__ q = (const T*)P.q;
  const T* __restrict__ kpe = (const T*)P.k_pe;
  const T* __restrict__ kv = (const T*)P.kv;
  const int S = P.S, H = P.H;

  // heavy-first, head-major ordering; each XCD gets a contiguous range of heads
  const int total = P.n_qblocks * P.n_hgroups * gridDim.y;
  const int lin = xcd_remap(blockIdx.x + gridDim.x * blockIdx.y, total);
  const int qb = P.n_qblocks - 1 - lin % P.n_qblocks;
  const int hgb = lin / P.n_qblocks;
  const int b = hgb / P.n_hgroups;
  const int h0 = (hgb % P.n_hgroups) * G;

  const int tid = threadIdx.x, wave = tid >> 6, l = tid & 63, n = l & 31, g = l >> 5;
  const int hh = wave / WPH;
  const int h = h0 + hh;
  const bool head_ok = h < H;
  const int q0 = qb * C::BR + (wave % WPH) * 32;  // first query of this wave
  const int my_q = q0 + n;
  const int wg_qend = min(S, (qb + 1) * C::BR);
  const int kend = P.causal ? wg_qend : S;

  // queries of this lane (B operand of S^T = K Q^T)
  frag_t<T> qf[DQK / 16];
  {
    const bool ok = head_ok && my_q < S;
    const T* qrow = q + ((size_t)(b * S + (ok ? my_q : 0)) * H + (ok ? h : 0)) * DQK;
#pragma unroll
    for (int ks = 0; ks < DQK / 16; ++ks) {
      if (ok) qf[ks] = *reinterpret_cast<const frag_t<T>*>(qrow + ks * 16 + 8 * g);
      else
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[ks][e] = to_elem<T>(0.f);
    }
  }

  f32x16 oacc[DV / 32];
#pragma unroll
  for (int i = 0; i < DV / 32; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[i][r] = 0.f;
  float m = -INFINITY, lsum = 0.f;

  // ---- staging of one key tile: global -> registers -> LDS
  chunk16 stage[C::PER_THREAD];
  auto load_tile = [&](int kt) {
#pragma unroll
    for (int i = 0; i < C::PER_THREAD; ++i) {
      const int c = tid + i * C::NT;
      stage[i] = zero_chunk();
      if (c < C::TILE_CHUNKS) {
        const int row = c / C::ROW_CHUNKS, j = c % C::ROW_CHUNKS;
        const int key = kt + row;
        if (key < S) {
          if (j < G * DKVH / E) {
            const int hj = j / (DKVH / E);
            if (h0 + hj < H)
              stage[i] = *reinterpret_cast<const chunk16*>(
                  kv + ((size_t)(b * S + key) * H + h0) * DKVH + (size_t)j * E);
          } else {
            stage[i] = *reinterpret_cast<const chunk16*>(kpe + (size_t)(b * S + key) * DR +
                                                         (j - G * DKVH / E) * E);
          }
        }
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < C::PER_THREAD; ++i) {
      const int c = tid + i * C::NT;
      if (c < C::TILE_CHUNKS) {
        const int row = c / C::ROW_CHUNKS, j = c % C::ROW_CHUNKS;
        T* dst;
        if (j < G * DKVH / E) {
          const int hj = j / (DKVH / E), e = (j % (DKVH / E)) * E;
          dst = e < DN ? sK + (hj * BC + row) * C::PK + e : sV + (hj * BC + row) * C::PV + (e - DN);
        } else {
          dst = sP + row * C::PP + (j - G * DKVH / E) * E;
        }
        *reinterpret_cast<chunk16*>(dst) = stage[i];
      }
    }
  };

  const T* sKh = sK + hh * BC * C::PK;
  const T* sVh = sV + hh * BC * C::PV;

  load_tile(0);
  for (int kt = 0; kt < kend; kt += BC) {
    __syncthreads();  // previous tile fully consumed
    store_tile();
    __syncthreads();
    if (kt + BC < kend) load_tile(kt + BC);  // prefetch overlaps the math below

    fwd_tile<T, DN, DR, DV, BC>(sKh, C::PK, sP, C::PP, sVh, C::PV, qf, oacc, m, lsum, kt, q0, my_q, S,
                                P.scale_log2, P.causal, head_ok);
  }

  if (!head_ok || my_q >= S) return;
  const float ltot = wave_xor32_sum(lsum);
  const float inv = 1.f / ltot;
  T* orow = (T*)P.out + ((size_t)(b * S + my_q) * H + h) * DV;
#pragma unroll
  for (int db = 0; db < DV / 32; ++db)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      typename FragOf<T>::half v;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = to_elem<T>(oacc[db][4 * rr + e] * inv);
      *reinterpret_cast<typename FragOf<T>::half*>(orow + db * 32 + rr * 8 + g * 4) = v;
    }
  if (g == 0) P.lse[(size_t)(b * H + h) * S + my_q] = (m + fast_log2(ltot)) * 0.69314718055994530942f;
}


// ------------------------------------------------------------------ ring variant
// bf16 forward for 128-wide K_nope / V and 64-wide k_pe. Key tiles stream through a
// two-stage LDS ring filled by direct global->LDS loads into swizzled, unpadded
// tiles (no staging registers, one barrier per tile). There is no per-wave branch
// around the MFMAs: a wave whose queries all precede a tile runs it fully masked
// (p = 0, m and O unchanged). Softmax details: the running max is taken on the raw
// scores (scale > 0), p = exp2(s * scale_log2 - m) is one FMA and one v_exp_f32,
// and O^T is rescaled only when some lane's running max moved.
// G heads per workgroup (WPH / G waves each, 32 * WPH / G queries per head): each key tile
// stages one K_nope and one V tile per head and ONE k_pe tile that every head's waves read
// (k_pe is shared by all heads, property P2 of Section 2.1).
template <int DN, int DR, int DV, int BC, int WPH, int G>
__global__ __launch_bounds__(64 * WPH) void attn_fwd_ring_kernel(FwdParams P) {
  using T = bf16;
  constexpr int DQK = DN + DR, DKVH = DN + DV, NW = WPH, WH = WPH / G, BR = 32 * WH;
  constexpr int KCPR = DN / 8, PCPR = DR / 8, VCPR = DV / 8;
  static_assert(KCPR == 16 && PCPR == 8 && VCPR == 16, "swizzles are defined for 128/64/128-wide rows");
  static_assert(WPH % G == 0, "whole waves per head");
  // two ring stages as distinct LDS objects: the compiler then sees that the direct
  // loads into one stage cannot alias the reads of the other and does not wait for
  // them (the explicit wait + barrier at the top of each tile orders the stages)
  __shared__ __attribute__((aligned(16))) T sK0[G * BC * DN], sK1[G * BC * DN];
  __shared__ __attribute__((aligned(16))) T sP0[BC * DR], sP1[BC * DR];
  __shared__ __attribute__((aligned(16))) T sV0[G * BC * DV], sV1[G * BC * DV];

  const T* __restrict__ q = (const T*)P.q;
  const T* __restrict__ kpe = (const T*)P.k_pe;
  const T* __restrict__ kv = (const T*)P.kv;
  const int S = P.S, H = P.H;

  const int total = P.n_qblocks * P.n_hgroups * gridDim.y;
  const int lin = xcd_remap(blockIdx.x + gridDim.x * blockIdx.y, total);
  const int qb = P.n_qblocks - 1 - lin % P.n_qblocks;
  const int bhg = lin / P.n_qblocks;
  const int b = bhg / P.n_hgroups, h0 = (bhg % P.n_hgroups) * G;

  const int tid = threadIdx.x, l = tid & 63, n = l & 31, g = l >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hh = wave / WH;   // this wave's head within the group
  const int h = min(h0 + hh, H - 1);
  const bool head_ok = h0 + hh < H;
  const int q0 = qb * BR + (wave % WH) * 32;
  const int my_q = q0 + n;
  const int kend = P.causal ? min(S, (qb + 1) * BR) : S;

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

  // key rows past S are clamped to S-1 (valid memory) and masked below
  SwzRowFill<T, BC, KCPR, NW> kfill, vfill;
  SwzRowFill<T, BC, PCPR, NW> pfill;
  kfill.init(wave, l, H * DKVH);
  vfill.init(wave, l, H * DKVH);
  pfill.init(wave, l, DR);
  auto fill_rows = [&](T* dk, T* dp, T* dv, int kt, int rows) {
#pragma unroll
    for (int gi = 0; gi < G; ++gi) {
      const T* kvb = kv + ((size_t)(b * S + kt) * H + min(h0 + gi, H - 1)) * DKVH;
      kfill.fill(dk + gi * BC * DN, wave, l, kvb, H * DKVH, rows);
      vfill.fill(dv + gi * BC * DV, wave, l, kvb + DN, H * DKVH, rows);
    }
    pfill.fill(dp, wave, l, kpe + (size_t)(b * S + kt) * DR, DR, rows);
  };
  // one branch per tile: whole tiles (all but possibly the last) take the copies with no
  // per-instruction row test
  auto fill = [&](T* dk, T* dp, T* dv, int kt) {
    if (S - kt >= BC) fill_rows(dk, dp, dv, kt, BC);
    else fill_rows(dk, dp, dv, kt, S - kt);
  };

  const int ntiles = (kend + BC - 1) / BC;
  fill(sK0, sP0, sV0, 0);
  auto step = [&](auto stage, int it) {
    constexpr int ST = decltype(stage)::value;
    const int kt = it * BC;
    wait_vmem();      // this wave's loads of tile `it` have landed
    __syncthreads();  // ... and everyone's; the other stage is free
    if (it + 1 < ntiles) {
      if constexpr (ST == 0) fill(sK1, sP1, sV1, kt + BC);
      else fill(sK0, sP0, sV0, kt + BC);
    }
    if (P.causal && kt > q0 + 31) return;  // wave-uniform: every key of the tile is masked for this wave
    const T* tk = (ST == 0 ? sK0 : sK1) + hh * BC * DN;
    const T* tp = ST == 0 ? sP0 : sP1;
    const T* tv = (ST == 0 ? sV0 : sV1) + hh * BC * DV;

    // S^T = K Q^T: product i takes contraction step ks = i / KB of key block kb = i % KB
    // (consecutive products go to different accumulators); its K fragment is read from
    // LDS PF products ahead into a ring of PF + 1 registers (the order of the reads and
    // products is pinned, so the compiler cannot trade the prefetch for registers).
    constexpr int KB = BC / 32, NSP = KB * (DQK / 16), PF = 3;
    auto k_frag = [&](int i) {
      const int ks = i / KB, kb = i % KB;
      return ks < DN / 16 ? swz_frag<T, KCPR>(tk, kb * 32 + n, 2 * ks + g)
                          : swz_frag<T, PCPR>(tp, kb * 32 + n, 2 * (ks - DN / 16) + g);
    };
    f32x16 sacc[KB];
    {
      frag_t<T> ab[PF + 1];
#pragma unroll
      for (int i = 0; i < PF; ++i) ab[i] = k_frag(i);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < NSP; ++i) {
        if (i + PF < NSP) ab[(i + PF) % (PF + 1)] = k_frag(i + PF);
        const int ks = i / KB, kb = i % KB;
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ab[i % (PF + 1)], qf[ks], ks == 0 ? f32x16{} : sacc[kb],
                                                          0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    const bool need_mask = (P.causal && kt + BC - 1 > q0) || (kt + BC > S);
    if (need_mask) {
      // the empty volatile statement keeps this a real branch (if-converted, the mask
      // would cost every tile two VALU operations per score)
      asm volatile("");
      // live keys: key < klim, i.e. accumulator row (r/4)*8 + r%4 + 32 kb < klim - kt - 4 g
      const int lim = (P.causal ? min(S, my_q + 1) : S) - kt - 4 * g;
#pragma unroll
      for (int kb = 0; kb < BC / 32; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          sacc[kb][r] = kb * 32 + (r >> 2) * 8 + (r & 3) < lim ? sacc[kb][r] : -INFINITY;
    }
    float mraw = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < BC / 32; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mraw = fmaxf(mraw, sacc[kb][r]);
    mraw = wave_xor32_max(mraw);
    const float m_new = fmaxf(m, mraw * P.scale_log2);
    // lazy rescale: the reference max m moves only when a score exceeds it by more
    // than 2^kRescaleLog2 (until then p <= 2^kRescaleLog2), so O^T is rarely rescaled;
    // the normalised result is the same
    const bool bump = m_new > m + kRescaleLog2;
    const float m_ref = bump ? m_new : m;
    const float alpha = bump ? fast_exp2(m - m_new) : 1.f;
    const float m_use = m_ref == -INFINITY ? 0.f : m_ref;
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
    m = m_ref;
    if (__ballot(bump)) {
#pragma unroll
      for (int i = 0; i < DV / 32; ++i) oacc[i] *= alpha;
    }
    frag_t<T> pf[BC / 16];
#pragma unroll
    for (int kk = 0; kk < BC / 16; ++kk) pf[kk] = acc_to_frag<T>(sacc[kk >> 1], kk & 1);
    // key chunks outer, value blocks inner: consecutive MFMAs accumulate into different
    // blocks of O^T, so none waits for the result of the one issued just before it (each
    // block still sums its key chunks in ascending order); V fragments prefetched as K's
    constexpr int NDB = DV / 32, NPV = (BC / 16) * NDB;
    auto v_frag = [&](int i) {
      const int kk = i / NDB, db = i % NDB, ra = kk * 16 + 4 * g;
      return swz_tr_frag<VCPR>(tv, ra, ra + 8, db * 32);
    };
    {
      frag_t<T> vb[PF + 1];
#pragma unroll
      for (int i = 0; i < PF; ++i) vb[i] = v_frag(i);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < NPV; ++i) {
        if (i + PF < NPV) vb[(i + PF) % (PF + 1)] = v_frag(i + PF);
        mma(oacc[i % NDB], vb[i % (PF + 1)], pf[i / NDB]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };
  for (int it = 0; it < ntiles; it += 2) {
    step(std::integral_constant<int, 0>{}, it);
    if (it + 1 < ntiles) step(std::integral_constant<int, 1>{}, it + 1);
  }

  if (!head_ok || my_q >= S) return;
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

// ------------------------------------------------------------------ fused variant
// No per-head K/V tensor exists in HBM. For each key tile the latent rows
// c_kv[kt : kt+BC, :] are copied straight into LDS (direct global->LDS loads, one
// row per wave instruction and 64-chunk segment), and the head's K_nope / V tile is
// rebuilt on chip as KV^T = W_h^T c^T: the A operand is the transposed weight
// (w_t [H*(DN+DV), d_c], read from global / L2), the B operand the LDS latent rows.
// Shape, operand roles and contraction order (ascending 16-wide steps over d_c from
// a zero accumulator) are those of the up-projection GEMM, and the result is rounded
// to the element type the same way, so the rebuilt tile equals the materialised kv
// bit for bit. The attention part is fwd_tile, unchanged.
struct FwdFusedParams {
  const void* q;
  const void* k_pe;
  const void* c_kv;
  const void* w_t;
  void* out;
  float* lse;
  int S, H, d_c, n_qblocks;
  float scale_log2;
  int causal;
};

// Latent rows [kt, kt + NROWS) of batch b -> sC (row pitch `pitch` elements): direct
// global->LDS loads, one wave instruction per row and 64-chunk segment (lane l lands
// 16*l bytes after the segment start), NROWS / NW rows per wave; rows past S are
// zero-filled by LDS stores. DCF: d_c at compile time (0: the run-time dc). Whole tiles
// take the loads with no per-row test.
template <typename T, int NROWS, int NW, int DCF>
__device__ __forceinline__ void load_latent_rows(const T* __restrict__ cg, T* sC, int pitch, int b, int S, int dc,
                                                 int kt, int wave, int l) {
  constexpr int E = Elems16<T>::n;
  static_assert(NROWS % NW == 0, "whole rows per wave");
  const int row_chunks = DCF > 0 ? DCF / E : dc / E;
  auto rows = [&](auto whole) {
#pragma unroll
    for (int i = 0; i < NROWS / NW; ++i) {
      const int row = wave + i * NW, key = kt + row;
      T* dst = sC + row * pitch;
      for (int seg = 0; seg < row_chunks; seg += 64) {
        const int c = seg + l;
        if (c < row_chunks) {
          if (decltype(whole)::value || key < S) g2lds16(cg + ((size_t)(b * S + key) * dc + (size_t)c * E), dst + seg * E);
          else *reinterpret_cast<chunk16*>(dst + c * E) = zero_chunk();
        }
      }
    }
  };
  if (kt + NROWS <= S) rows(std::true_type{});
  else rows(std::false_type{});
}

// DCF: d_c as a compile-time constant (0: the run-time P.d_c, up to DCMAX)
template <typename T, int DN, int DR, int DV, int BC, int WPH, int DCMAX, int DCF>
__global__ __launch_bounds__(64 * WPH) void attn_fwd_fused_kernel(FwdFusedParams P) {
  constexpr int DQK = DN + DR, DKVH = DN + DV, E = Elems16<T>::n, NT = 64 * WPH, NW = WPH;
  constexpr int PK = DN + 8, PP = DR + 8, PV = DV + 32 / (int)sizeof(T), PC = DCMAX + 8;
  constexpr int NCBLK = DKVH / 32, NKB = BC / 32;
  constexpr int NCB = NCBLK >= NW ? NCBLK / NW : 1;  // column blocks rebuilt per wave
  static_assert(NCBLK % NW == 0 || NCBLK < NW, "column blocks must split over the waves");
  __shared__ __attribute__((aligned(16))) T sK[BC * PK];
  __shared__ __attribute__((aligned(16))) T sP[BC * PP];
  __shared__ __attribute__((aligned(16))) T sV[BC * PV];
  __shared__ __attribute__((aligned(16))) T sC[BC * PC];

  const T* __restrict__ q = (const T*)P.q;
  const T* __restrict__ kpe = (const T*)P.k_pe;
  const T* __restrict__ cg = (const T*)P.c_kv;
  const T* __restrict__ wt = (const T*)P.w_t;
  const int S = P.S, H = P.H, dc = P.d_c;

  const int total = P.n_qblocks * H * gridDim.y;
  const int lin = xcd_remap(blockIdx.x + gridDim.x * blockIdx.y, total);
  const int qb = P.n_qblocks - 1 - lin % P.n_qblocks;
  const int bh = lin / P.n_qblocks;
  const int b = bh / H, h = bh % H;

  const int tid = threadIdx.x, wave = tid >> 6, l = tid & 63, n = l & 31, g = l >> 5;
  const int q0 = qb * 32 * WPH + wave * 32;
  const int my_q = q0 + n;
  const int wg_qend = min(S, (qb + 1) * 32 * WPH);
  const int kend = P.causal ? wg_qend : S;

  frag_t<T> qf[DQK / 16];
  {
    const bool ok = my_q < S;
    const T* qrow = q + ((size_t)(b * S + (ok ? my_q : 0)) * H + h) * DQK;
#pragma unroll
    for (int ks = 0; ks < DQK / 16; ++ks) {
      if (ok) qf[ks] = *reinterpret_cast<const frag_t<T>*>(qrow + ks * 16 + 8 * g);
      else
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[ks][e] = to_elem<T>(0.f);
    }
  }
  f32x16 oacc[DV / 32];
#pragma unroll
  for (int i = 0; i < DV / 32; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[i][r] = 0.f;
  float m = -INFINITY, lsum = 0.f;

  // k_pe tile -> sP (through registers; small)
  constexpr int PCH = BC * (DR / E);
  constexpr int PPT = (PCH + NT - 1) / NT;
  chunk16 pst[PPT];
  auto load_p = [&](int kt) {
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int c = tid + i * NT;
      pst[i] = zero_chunk();
      if (c < PCH) {
        const int row = c / (DR / E), j = c % (DR / E);
        if (kt + row < S) pst[i] = *reinterpret_cast<const chunk16*>(kpe + (size_t)(b * S + kt + row) * DR + j * E);
      }
    }
  };
  auto store_p = [&]() {
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int c = tid + i * NT;
      if (c < PCH) {
        const int row = c / (DR / E), j = c % (DR / E);
        *reinterpret_cast<chunk16*>(sP + row * PP + j * E) = pst[i];
      }
    }
  };

  load_latent_rows<T, BC, NW, DCF>(cg, sC, PC, b, S, dc, 0, wave, l);
  load_p(0);
  for (int kt = 0; kt < kend; kt += BC) {
    wait_vmem();                    // this wave's direct loads into sC have landed
    __syncthreads();                // all of sC present; previous tile's sK/sV/sP consumed
    store_p();
    // rebuild K_nope / V of this tile: KV^T[col][key] = sum_c W^T[col][c] * c[key][c]
    const int cb0 = wave * NCB;
    if (cb0 < NCBLK) {
      f32x16 acc[NCB][NKB];
#pragma unroll
      for (int i = 0; i < NCB; ++i)
#pragma unroll
        for (int j = 0; j < NKB; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
      // W^T in fragment order: the fragment of column block cb and contraction step ks is
      // 64 lanes x 8 contiguous elements (one coalesced 1 KB read in bf16)
      const int nks = dc / 16;
      const T* wrow[NCB];
#pragma unroll
      for (int i = 0; i < NCB; ++i) wrow[i] = wt + (size_t)(h * NCBLK + cb0 + i) * nks * 512 + l * 8;
      if constexpr (DCF > 0 && NCB == 1) {
        // d_c known at compile time: the W^T fragments stream from L2 through a ring of
        // WR registers, WR contraction steps ahead of their MFMAs (one load in flight per
        // step would leave every step waiting for L2)
        constexpr int NKS = DCF / 16, WR = 16;
        static_assert(NKS >= WR, "ring shorter than the contraction");
        // wave-uniform fragment base (scalar registers) + one per-lane offset
        const T* wsb = wt + (size_t)__builtin_amdgcn_readfirstlane(h * NCBLK + cb0) * NKS * 512;
        const int loff = l * 8;
        auto wfrag = [&](int ks) { return *reinterpret_cast<const frag_t<T>*>(wsb + ks * 512 + loff); };
        frag_t<T> ar[WR];
#pragma unroll
        for (int u = 0; u < WR; ++u) ar[u] = wfrag(u);
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          const frag_t<T> a = ar[ks % WR];
          if (ks + WR < NKS) ar[ks % WR] = wfrag(ks + WR);
          frag_t<T> bb[NKB];
#pragma unroll
          for (int j = 0; j < NKB; ++j) bb[j] = lds_frag<T>(sC + (j * 32 + n) * PC + ks * 16 + 8 * g);
#pragma unroll
          for (int j = 0; j < NKB; ++j) mma(acc[0][j], a, bb[j]);
        }
      } else {
        for (int ks = 0; ks < dc / 16; ++ks) {
          frag_t<T> a[NCB], bb[NKB];
#pragma unroll
          for (int i = 0; i < NCB; ++i) a[i] = *reinterpret_cast<const frag_t<T>*>(wrow[i] + ks * 512);
#pragma unroll
          for (int j = 0; j < NKB; ++j) bb[j] = lds_frag<T>(sC + (j * 32 + n) * PC + ks * 16 + 8 * g);
#pragma unroll
          for (int i = 0; i < NCB; ++i)
#pragma unroll
            for (int j = 0; j < NKB; ++j) mma(acc[i][j], a[i], bb[j]);
        }
      }
#pragma unroll
      for (int i = 0; i < NCB; ++i)
#pragma unroll
        for (int j = 0; j < NKB; ++j)
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            const int col = (cb0 + i) * 32 + rr * 8 + g * 4;
            const int key = j * 32 + n;
            typename FragOf<T>::half v;
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = to_elem<T>(acc[i][j][4 * rr + e]);
            T* dst = col < DN ? sK + key * PK + col : sV + key * PV + (col - DN);
            *reinterpret_cast<typename FragOf<T>::half*>(dst) = v;
          }
    }
    __syncthreads();  // sK / sV / sP complete; sC free
    if (kt + BC < kend) {
      load_latent_rows<T, BC, NW, DCF>(cg, sC, PC, b, S, dc, kt + BC, wave, l);
      load_p(kt + BC);
    }
    fwd_tile<T, DN, DR, DV, BC>(sK, PK, sP, PP, sV, PV, qf, oacc, m, lsum, kt, q0, my_q, S, P.scale_log2,
                                P.causal, true);
    __syncthreads();  // everyone done reading sK / sV / sP before the next rebuild
  }

  if (my_q >= S) return;
  const float ltot = wave_xor32_sum(lsum);
  const float inv = 1.f / ltot;
  T* orow = (T*)P.out + ((size_t)(b * S + my_q) * H + h) * DV;
#pragma unroll
  for (int db = 0; db < DV / 32; ++db)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      typename FragOf<T>::half v;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = to_elem<T>(oacc[db][4 * rr + e] * inv);
      *reinterpret_cast<typename FragOf<T>::half*>(orow + db * 32 + rr * 8 + g * 4) = v;
    }
  if (g == 0) P.lse[(size_t)(b * H + h) * S + my_q] = (m + fast_log2(ltot)) * 0.69314718055994530942f;
}

// W_kv_b^T in MFMA A-fragment order, one thread per output element: block (cb, ks) of 512
// elements holds, for lane l = 32 g + n, the 8 elements
// w_t[32 cb + r(n)][16 ks + 8 g + e] = w[16 ks + 8 g + e][32 cb + r(n)], with r(n) = n, or
// with PI the order pi (bits 2 and 3 of n swapped) that the backward's rebuilds use (K =
// d_c rows of w, a multiple of 16; N = H*(DN+DV) columns, a multiple of 32). A wave reads
// one fragment as 1 KB of contiguous memory.
template <typename T, bool PI>
__global__ __launch_bounds__(256) void frag_w_kernel(const T* __restrict__ w, T* __restrict__ wf, int K, int N) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long long)K * N) return;
  const int nks = K / 16;
  const long long blk = i / 512;
  const int within = (int)(i % 512), lane = within >> 3, e = within & 7;
  const int cb = (int)(blk / nks), ks = (int)(blk % nks);
  const int n = lane & 31, r = PI ? (n & ~12) | ((n & 4) << 1) | ((n & 8) >> 1) : n;
  const int col = cb * 32 + r, k = ks * 16 + 8 * (lane >> 5) + e;
  wf[i] = w[(size_t)k * N + col];
}

template <typename T, int DN, int DR, int DV> struct FwdTiles;
template <int DN, int DR, int DV> struct FwdTiles<bf16, DN, DR, DV> {
  static constexpr int BC = 64, WPH = 4, G = 1;
};
template <int DN, int DR, int DV> struct FwdTiles<float, DN, DR, DV> {
  static constexpr int BC = 32, WPH = 4, G = 1;
};

}  // namespace

// The bf16 forward picks its workgroup size by the grid it gives: 256 queries (fewer
// re-reads of the K/V tiles) while that still yields this many workgroups (two per CU),
// 128 below. Both sizes run the same per-wave computation in the same order, so results
// do not depend on the choice. (The same rule for the key-stationary backward measured
// slower with few heads: its longest workgroup, the first keys', sets the time whatever
// its width.)
constexpr int kFwdFillGroups = 512;
// Heads per workgroup of the bf16 ring forward (one shared k_pe tile per key tile).
constexpr int kFwdRingHeads = 1;

template <typename T, int DN, int DR, int DV>
hipError_t launch_attn_fwd(const AttnFwdArgs& a, hipStream_t st) {
  using Tl = FwdTiles<T, DN, DR, DV>;
  constexpr int BR = 32 * Tl::WPH;
  FwdParams P;
  P.q = a.q; P.k_pe = a.k_pe; P.kv = a.kv; P.out = a.out; P.lse = a.lse;
  P.S = a.S; P.H = a.H;
  P.n_qblocks = (a.S + BR - 1) / BR;
  P.n_hgroups = (a.H + Tl::G - 1) / Tl::G;
  P.scale_log2 = a.scale * 1.4426950408889634f;
  P.causal = a.causal;
  dim3 grid(P.n_qblocks * P.n_hgroups, a.B, 1);
  if constexpr (sizeof(T) == 2 && DN == 128 && DR == 64 && DV == 128 && Tl::G == 1) {
    // 8 waves: 256 queries of one head per workgroup, which halves the K/V tile
    // traffic of 4 waves (measured 8 % faster at S = 16384); 4 waves when 8 would leave
    // fewer than kFwdFillGroups workgroups (few heads or short sequences)
    auto ring = [&](auto rw) {
      constexpr int RW = decltype(rw)::value, RG = kFwdRingHeads, RBR = 32 * RW / RG;
      P.n_qblocks = (a.S + RBR - 1) / RBR;
      P.n_hgroups = (a.H + RG - 1) / RG;
      attn_fwd_ring_kernel<DN, DR, DV, Tl::BC, RW, RG><<<dim3(P.n_qblocks * P.n_hgroups, a.B, 1), 64 * RW, 0, st>>>(P);
    };
    if ((long long)((a.S + 255) / 256) * P.n_hgroups * a.B >= kFwdFillGroups) ring(std::integral_constant<int, 8>{});
    else ring(std::integral_constant<int, 4>{});
  } else {
    using Cfg = FwdCfg<T, DN, DR, DV, Tl::BC, Tl::WPH, Tl::G, false>;
    attn_fwd_kernel<T, DN, DR, DV, Tl::BC, Tl::WPH, Tl::G, false><<<grid, Cfg::NT, 0, st>>>(P);
  }
  return hipGetLastError();
}

template <typename T, int DN, int DR, int DV>
hipError_t launch_attn_fwd_fused(const AttnFwdArgs& a, void* w_t_ws, hipStream_t st) {
  using Tl = FwdTiles<T, DN, DR, DV>;
  // bf16: 8 waves, so 256 queries of the workgroup share each rebuilt K/V tile (the
  // rebuild costs d_c * d_kvh / Br times the attention flops; 4 waves: 13.3 ms at
  // S = 16384, 8 waves: 5.7 ms)
  constexpr int FW = sizeof(T) == 2 ? 8 : Tl::WPH;
  constexpr int BR = 32 * FW;
  const int N = a.H * (DN + DV);
  const long long nw = (long long)a.d_c * N;
  frag_w_kernel<T, false><<<(unsigned)((nw + 255) / 256), 256, 0, st>>>((const T*)a.w, (T*)w_t_ws, a.d_c, N);
  FwdFusedParams P;
  P.q = a.q; P.k_pe = a.k_pe; P.c_kv = a.c_kv; P.w_t = w_t_ws; P.out = a.out; P.lse = a.lse;
  P.S = a.S; P.H = a.H; P.d_c = a.d_c; P.n_qblocks = (a.S + BR - 1) / BR;
  P.scale_log2 = a.scale * 1.4426950408889634f;
  P.causal = a.causal;
  dim3 grid(P.n_qblocks * a.H, a.B, 1);
  if (a.d_c == kFusedMaxDc)
    attn_fwd_fused_kernel<T, DN, DR, DV, Tl::BC, FW, kFusedMaxDc, kFusedMaxDc><<<grid, 64 * FW, 0, st>>>(P);
  else
    attn_fwd_fused_kernel<T, DN, DR, DV, Tl::BC, FW, kFusedMaxDc, 0><<<grid, 64 * FW, 0, st>>>(P);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_frag_w_pi(const T* w, T* w_t, int K, int N, hipStream_t st) {
  const long long nw = (long long)K * N;
  frag_w_kernel<T, true><<<(unsigned)((nw + 255) / 256), 256, 0, st>>>(w, w_t, K, N);
  return hipGetLastError();
}
template hipError_t launch_frag_w_pi<bf16>(const bf16*, bf16*, int, int, hipStream_t);

#define LAGA_INST_FWD(T, DN, DR, DV)                                                      \
  template hipError_t launch_attn_fwd<T, DN, DR, DV>(const AttnFwdArgs&, hipStream_t);    \
  template hipError_t launch_attn_fwd_fused<T, DN, DR, DV>(const AttnFwdArgs&, void*, hipStream_t);
LAGA_INST_FWD(bf16, 128, 64, 128)
LAGA_INST_FWD(float, 128, 64, 128)
LAGA_INST_FWD(bf16, 32, 16, 32)
LAGA_INST_FWD(float, 32, 16, 32)
LAGA_INST_FWD(bf16, 64, 32, 64)
LAGA_INST_FWD(float, 64, 32, 64)

}  // namespace laga
