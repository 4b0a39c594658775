// dQ pass of the attention backward (gfx950); see attn_bwd.hip for the whole backward.
// Built with MFMA results kept in VGPRs (the dZ arithmetic on the dP accumulators of
// the recomputing kernel then needs no AGPR<->VGPR copies).
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


// dQ recomputed without any S x S buffer (bf16, 192/128-wide heads): the forward's
// structure with dP and dS added. A workgroup of 8 waves owns 256 queries of one head (a
// wave 32, lane <-> query); 64-key tiles of K = [K_nope || k_pe] and V stream through a
// two-stage LDS ring of direct global->LDS loads into XOR-swizzled tiles. Per 32-key
// block: S^T = K Q^T and dP^T = V dO^T (A = K / V rows from LDS, B = the wave's Q and dO
// in registers, fragments read three products ahead), P^T = exp2(S^T scale_log2 - lse2),
// dS^T = P^T (dP^T - delta) in the accumulators' lanes, then dQ^T += K^T dS^T with K^T
// from transposing LDS reads and dS^T straight from the accumulators. The arithmetic
// per element is the key-stationary pass's (S and dP on the same MFMA products, the
// same exp2 argument, dS rounded once to bf16) and dQ sums the keys in ascending
// 16-wide steps, as the pass over the stored dS^T does: dq is bitwise equal to it.
template <int DN, int DR, int DV, int NW>
__global__ __launch_bounds__(64 * NW, 1) void dq_rec_kernel(BwdParams P) {
  using T = bf16;
  constexpr int DQK = DN + DR, DKVH = DN + DV, BC = 64, BR = 32 * NW;
  constexpr int KCPR = DN / 8, PCPR = DR / 8, VCPR = DV / 8;
  constexpr int NKS = DQK / 16, NVS = DV / 16, NDB = DQK / 32, NDN = DN / 32;
  static_assert(KCPR == 16 && PCPR == 8 && VCPR == 16, "swizzles are defined for 128/64/128-wide rows");
  // two ring stages as distinct LDS objects (compile-time stage offsets in the reads)
  __shared__ __attribute__((aligned(16))) T sK0[BC * DN], sK1[BC * DN];
  __shared__ __attribute__((aligned(16))) T sP0[BC * DR], sP1[BC * DR];
  __shared__ __attribute__((aligned(16))) T sV0[BC * DV], sV1[BC * DV];

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

  const int tid = threadIdx.x, l = tid & 63, n = l & 31, g = l >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q0 = qblk * BR + wave * 32;
  const int my_q = q0 + n;
  const int kend = P.causal ? min(S, (qblk + 1) * BR) : S;

  frag_t<T> qf[NKS], of[NVS];
  float lse2 = 0.f, dlt = 0.f;
  {
    const bool ok = my_q < S;
    const size_t base = (size_t)(b * S + (ok ? my_q : 0)) * H + h;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      qf[ks] = *reinterpret_cast<const frag_t<T>*>(q + base * DQK + ks * 16 + 8 * g);
      if (!ok) qf[ks] = frag_t<T>{};
    }
#pragma unroll
    for (int ks = 0; ks < NVS; ++ks) {
      of[ks] = *reinterpret_cast<const frag_t<T>*>(dout + base * DV + ks * 16 + 8 * g);
      if (!ok) of[ks] = frag_t<T>{};
    }
    if (ok) {
      lse2 = P.lse2[(size_t)(b * H + h) * P.S_pad + my_q];
      dlt = P.delta[(size_t)(b * H + h) * P.S_pad + my_q];
    }
  }
  f32x16 dqa[NDB];
#pragma unroll
  for (int i = 0; i < NDB; ++i) dqa[i] = f32x16{};

  // key rows past S are clamped to S - 1 (valid memory) and masked below
  SwzRowFill<T, BC, KCPR, NW> kfill, vfill;
  SwzRowFill<T, BC, PCPR, NW> pfill;
  kfill.init(wave, l, H * DKVH);
  vfill.init(wave, l, H * DKVH);
  pfill.init(wave, l, DR);
  auto fill_rows = [&](T* dk, T* dp, T* dv, int kt, int rows) {
    const T* kvb = kv + ((size_t)(b * S + kt) * H + h) * DKVH;
    kfill.fill(dk, wave, l, kvb, H * DKVH, rows);
    vfill.fill(dv, wave, l, kvb + DN, H * DKVH, rows);
    pfill.fill(dp, wave, l, kpe + (size_t)(b * S + kt) * DR, DR, rows);
  };
  // one branch per tile: whole tiles take the copies with no per-instruction row test
  auto fill = [&](T* dk, T* dp, T* dv, int kt) {
    if (S - kt >= BC) fill_rows(dk, dp, dv, kt, BC);
    else fill_rows(dk, dp, dv, kt, S - kt);
  };

  constexpr int PF = 3;
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
    if (P.causal && kt > q0 + 31) return;  // wave-uniform: every key of the tile is masked
    const T* tk = ST == 0 ? sK0 : sK1;
    const T* tp = ST == 0 ? sP0 : sP1;
    const T* tv = ST == 0 ? sV0 : sV1;
    const bool need_mask = (P.causal && kt + BC - 1 > q0) || (kt + BC > S);
#pragma unroll
    for (int kb = 0; kb < BC / 32; ++kb) {
      // product i of S^T (even i < 16 and i >= 16: contraction step a_ks(i) of K) and of
      // dP^T (odd i < 16: step i / 2 of V), alternating accumulators
      auto a_is_s = [](int i) { return i >= 16 || (i & 1) == 0; };
      auto a_ks = [](int i) { return i >= 16 ? 8 + (i - 16) : i >> 1; };
      auto a_frag = [&](int i) {
        const int ks = a_ks(i), row = kb * 32 + n;
        if (!a_is_s(i)) return swz_frag<T, VCPR>(tv, row, 2 * ks + g);
        return ks < DN / 16 ? swz_frag<T, KCPR>(tk, row, 2 * ks + g)
                            : swz_frag<T, PCPR>(tp, row, 2 * (ks - DN / 16) + g);
      };
      constexpr int NA = NKS + NVS;  // 20 products
      f32x16 sa, dp;
      {
        frag_t<T> ab[PF + 1];
#pragma unroll
        for (int i = 0; i < PF; ++i) ab[i] = a_frag(i);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < NA; ++i) {
          if (i + PF < NA) ab[(i + PF) % (PF + 1)] = a_frag(i + PF);
          if (a_is_s(i))
            sa = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ab[i % (PF + 1)], qf[a_ks(i)], i == 0 ? f32x16{} : sa,
                                                         0, 0, 0);
          else
            dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ab[i % (PF + 1)], of[a_ks(i)], i == 1 ? f32x16{} : dp,
                                                         0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      if (need_mask) {
        asm volatile("");  // a kept branch: only tiles on the diagonal or at the end
        // live keys: accumulator row (r/4)*8 + r%4 of key block kb < klim - kt - 32 kb - 4 g
        const int lim = (P.causal ? min(S, my_q + 1) : S) - kt - 32 * kb - 4 * g;
#pragma unroll
        for (int r = 0; r < 16; ++r) sa[r] = (r >> 2) * 8 + (r & 3) < lim ? sa[r] : -INFINITY;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = fast_exp2(__builtin_fmaf(sa[r], P.scale_log2, -lse2));
        dp[r] = p * (dp[r] - dlt);
      }
      bf16x8 zf[2];
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) zf[kk] = acc_to_frag<T>(dp, kk);
      // dQ^T += K^T dS^T: product i = 16-key chunk kk = i / NDB, dQ block db = i % NDB
      auto k_tr = [&](int i) {
        const int kk = i / NDB, db = i % NDB, ra = kb * 32 + kk * 16 + 4 * g;
        return db < NDN ? swz_tr_frag<KCPR>(tk, ra, ra + 8, db * 32)
                        : swz_tr_frag<PCPR>(tp, ra, ra + 8, (db - NDN) * 32);
      };
      constexpr int NQ = 2 * NDB;  // 12 products
      {
        frag_t<T> kb_[PF + 1];
#pragma unroll
        for (int i = 0; i < PF; ++i) kb_[i] = k_tr(i);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
          if (i + PF < NQ) kb_[(i + PF) % (PF + 1)] = k_tr(i + PF);
          mma(dqa[i % NDB], kb_[i % (PF + 1)], zf[i / NDB]);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  };
  for (int it = 0; it < ntiles; it += 2) {
    step(std::integral_constant<int, 0>{}, it);
    if (it + 1 < ntiles) step(std::integral_constant<int, 1>{}, it + 1);
  }

  if (my_q >= S) return;
  T* dqr = (T*)P.dq + ((size_t)(b * S + my_q) * H + h) * DQK;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      bf16x4 v;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = to_elem<T>(dqa[db][4 * rr + e] * P.scale);
      *reinterpret_cast<bf16x4*>(dqr + db * 32 + rr * 8 + g * 4) = v;
    }
}

// dQ from the stored dS^T (bf16, 192/128-wide heads): the key-stationary pass leaves
// dS^T = P * (dP - delta) of every causal (query tile, key) pair in the workspace, so
// this pass is a streaming product dQ^T (192 x 32 per wave) += K^T dS^T over the
// tile's keys, with no recomputation of S or dP. A workgroup of WPH waves owns WPH
// consecutive 32-query tiles of one head; key blocks of 32 stream through an NS-stage
// LDS ring of direct global->LDS loads: the K = [K_nope || k_pe] rows of the block
// (shared, padded pitch 28 chunks) and each wave's own 32 x 32 dS^T block (64-byte
// rows). Both MFMA operands come from transposing reads:
//   A = K^T (lane: head dim, 8 keys), B = dS^T (lane: query, the same 8 keys).
// Every wave issues the same number of loads per stage (the K fill is rounded up to
// whole rounds of the workgroup, and key blocks past a wave's queries load a dummy
// block that is not read), so the ring waits can count loads exactly.
template <int DN, int DR, int DV, int WPH, int NS, int TPW>
__global__ __launch_bounds__(64 * WPH, 1) void dq_ds_kernel(BwdParams P) {
  using T = bf16;
  constexpr int DQK = DN + DR, DKVH = DN + DV, KB = 32, NW = WPH;
  constexpr int KCPR = DQK / 8, NCPR = DN / 8, KP = KCPR + 4;  // pitch % 8 == 4
  static_assert(KCPR % 4 == 0 && DQK % 32 == 0 && (NS == 3 || NS == 4), "192-wide K rows, 3 or 4 stages");
  static_assert(TPW == 1 || TPW == 2, "one or two query tiles per wave");
  constexpr int KCH = (KB * KP + 64 * NW - 1) / (64 * NW) * (64 * NW);  // K chunks, whole rounds
  constexpr int F = KCH / 64 / NW + 2 * TPW;                           // loads per wave per stage
  constexpr int DSE = NW * TPW * KB * 32;                              // dS^T elements per stage
  __shared__ __attribute__((aligned(16))) T sK0[KCH * 8], sK1[KCH * 8], sK2[KCH * 8], sK3[KCH * 8];
  __shared__ __attribute__((aligned(16))) T sD0[DSE], sD1[DSE], sD2[DSE], sD3[DSE];

  const T* __restrict__ kpe = (const T*)P.k_pe;
  const T* __restrict__ kv = (const T*)P.kv;
  const T* __restrict__ ds = (const T*)P.ds;
  const int S = P.S, H = P.H, TT = P.ds_T;

  const int total = P.n_blocks * H * gridDim.y;
  const int lin = xcd_remap(blockIdx.x + gridDim.x * blockIdx.y, total);
  const int qblk = P.n_blocks - 1 - lin % P.n_blocks;  // heavy first
  const int bh = lin / P.n_blocks;
  const int b = bh / H, h = bh % H;

  const int tid = threadIdx.x, wave = tid >> 6, l = tid & 63, n = l & 31, g = l >> 5;
  // this wave's query tiles t0 .. t0 + TPW - 1 (consecutive, so tile i sees 32 i more keys)
  const int t0 = (qblk * NW + wave) * TPW;
  int nk[TPW];
  const T* dtile[TPW];
#pragma unroll
  for (int i = 0; i < TPW; ++i) {
    const bool ok = t0 + i < TT;
    nk[i] = ok ? ds_tile_keys(TT, P.causal, t0 + i) : 0;  // keys stored for the tile
    dtile[i] = ds + (ok ? ds_tile_offset(TT, P.causal, bh, t0 + i) : 0);
  }
  const int kend = P.causal ? min(S, (qblk + 1) * NW * TPW * 32) : S;
  const int ntiles = (kend + KB - 1) / KB;

  f32x16 dqa[TPW][DQK / 32];
#pragma unroll
  for (int i = 0; i < TPW; ++i)
#pragma unroll
    for (int j = 0; j < DQK / 32; ++j) dqa[i][j] = f32x16{};

  auto fill = [&](T* dk, T* dd, int kt) {
    pad_fill_chunks<T, KB, KCPR, KP, NW, KCH>(dk, wave, l, [&](int r, int c) {
      const size_t row = (size_t)(b * S + min(kt + r, S - 1));
      return c < NCPR ? kv + (row * H + h) * DKVH + c * 8 : kpe + row * DR + (c - NCPR) * 8;
    });
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
      const T* src = kt < nk[i] ? dtile[i] + (size_t)kt * 32 : dtile[i];  // dummy block when not stored
      T* dst = dd + (wave * TPW + i) * KB * 32;
      g2lds16(src + l * 8, dst);
      g2lds16(src + 512 + l * 8, dst + 512);
    }
  };

  // Every step refills a stage, past the last block with in-bounds dummies (clamped K
  // rows, the tile's first dS block) that nobody reads, so NS - 2 stages of loads are
  // always in flight behind the awaited one and the waits need no branch.
  fill(sK0, sD0, 0);
  fill(sK1, sD1, KB);
  if constexpr (NS == 4) fill(sK2, sD2, 2 * KB);
  // one K fragment feeds the MFMAs of every tile of the wave that sees the key block
  auto product = [&](const T* tk, const T* td, auto first) {
    constexpr int I0 = decltype(first)::value;  // tiles before I0 do not see this block
#pragma unroll
    for (int kk = 0; kk < KB / 16; ++kk) {
      const int ra = kk * 16 + 4 * g;
      bf16x8 zf[TPW];
#pragma unroll
      for (int i = I0; i < TPW; ++i) zf[i] = pad_tr_frag<4>(td + i * KB * 32, ra, ra + 8, 0);
#pragma unroll
      for (int db = 0; db < DQK / 32; ++db) {
        const bf16x8 kf = pad_tr_frag<KP>(tk, ra, ra + 8, db * 32);
#pragma unroll
        for (int i = I0; i < TPW; ++i) mma(dqa[i][db], kf, zf[i]);
      }
    }
  };
  auto step = [&](auto stage, int it) {
    constexpr int ST = decltype(stage)::value;
    const int kt = it * KB;
    wait_vmem_le<(NS - 2) * F>();  // this wave's loads of block `it` have landed
    __syncthreads();  // ... and everyone's; the stage filled next (read last at it - 1) is free
    {
      constexpr int NX = (ST + NS - 1) % NS;
      T* nk_ = NX == 0 ? sK0 : NX == 1 ? sK1 : NX == 2 ? sK2 : sK3;
      T* nd_ = NX == 0 ? sD0 : NX == 1 ? sD1 : NX == 2 ? sD2 : sD3;
      fill(nk_, nd_, kt + (NS - 1) * KB);
    }
    const T* tk = ST == 0 ? sK0 : ST == 1 ? sK1 : ST == 2 ? sK2 : sK3;
    const T* td = (ST == 0 ? sD0 : ST == 1 ? sD1 : ST == 2 ? sD2 : sD3) + wave * TPW * KB * 32;
    // wave-uniform: key blocks past a tile's queries hold no dS for it; nk[i] grows with i
    if (kt < nk[0]) product(tk, td, std::integral_constant<int, 0>{});
    else if (TPW > 1 && kt < nk[TPW - 1]) product(tk, td, std::integral_constant<int, TPW - 1>{});
  };
  for (int it = 0; it < ntiles; it += NS) {
    step(std::integral_constant<int, 0>{}, it);
    if (it + 1 < ntiles) step(std::integral_constant<int, 1>{}, it + 1);
    if (it + 2 < ntiles) step(std::integral_constant<int, 2>{}, it + 2);
    if constexpr (NS == 4)
      if (it + 3 < ntiles) step(std::integral_constant<int, NS - 1>{}, it + 3);
  }

  wait_vmem();  // the surplus loads land before the workgroup's LDS is released
  // accumulator column n holds the query stored at position n of the dS^T rows
#pragma unroll
  for (int i = 0; i < TPW; ++i) {
    const int my_q = (t0 + i) * 32 + ds_query_of_position(n);
    if (t0 + i >= TT || my_q >= S) continue;
    T* dqr = (T*)P.dq + ((size_t)(b * S + my_q) * H + h) * DQK;
#pragma unroll
    for (int db = 0; db < DQK / 32; ++db)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        bf16x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = to_elem<T>(dqa[i][db][4 * rr + e] * P.scale);
        *reinterpret_cast<bf16x4*>(dqr + db * 32 + rr * 8 + g * 4) = v;
      }
  }
}

// dQ from the stored dS^T with K/V rebuilt on chip (kv_mode FUSED; bf16, 192/128-wide
// heads): as dq_ds_kernel, but no per-head K exists in HBM, so each step's K tile is built
// in LDS: the K_nope rows of its 64 keys from the latent (KV^T = W_h^T c^T over d_c in
// ascending 16-wide steps, the up-projection GEMM's operand roles and rounding, so the
// tile equals the materialised kv bit for bit, and dq equals dq_ds_kernel's), the k_pe
// rows loaded as they are. Wave w rebuilds the 32 x 32 block (key half w / 4, K_nope
// columns 32 (w % 4) ..): every wave does the same 32 MFMAs per step, beside its 24 of
// the dQ product. The rebuild repeats for every query block of 256 rows (the price of a
// query-stationary pass: d_c * d_nope / (256 * d_qk) of its product flops, 1.33x).
template <int DN, int DR, int DV>
__global__ __launch_bounds__(512, 1) void dq_ds_fused_kernel(BwdParams P) {
  using T = bf16;
  constexpr int DQK = DN + DR, DKVH = DN + DV, NW = 8, KB = 64;
  constexpr int KP = DQK / 8 + 4;  // K tile pitch in 16-byte chunks (% 8 == 4: transposing reads)
  static_assert(DN == 4 * 32 && DR == 64, "four 32-column K_nope blocks, 64-wide k_pe");
  __shared__ __attribute__((aligned(16))) T sK[KB * KP * 8];
  __shared__ __attribute__((aligned(16))) T sD[NW * 2 * 32 * 32];

  const T* __restrict__ kpe = (const T*)P.k_pe;
  const T* __restrict__ ds = (const T*)P.ds;
  const int S = P.S, H = P.H, TT = P.ds_T, dc = P.d_c;

  const int total = P.n_blocks * H * gridDim.y;
  const int lin = xcd_remap(blockIdx.x + gridDim.x * blockIdx.y, total);
  const int qblk = P.n_blocks - 1 - lin % P.n_blocks;  // heavy first
  const int bh = lin / P.n_blocks;
  const int b = bh / H, h = bh % H;

  const int tid = threadIdx.x, wave = tid >> 6, l = tid & 63, n = l & 31, g = l >> 5;
  const int t = qblk * NW + wave;  // this wave's query tile
  const bool wave_ok = t < TT;
  const int nk = wave_ok ? ds_tile_keys(TT, P.causal, t) : 0;
  const T* dtile = ds + (wave_ok ? ds_tile_offset(TT, P.causal, bh, t) : 0);
  const int kend = P.causal ? min(S, (qblk + 1) * NW * 32) : S;
  const int nsteps = (kend + KB - 1) / KB;

  // this wave's share of the rebuild: key half rk, K_nope column block rb; W^T rows in the
  // order pi (bits 2 and 3 swapped) so that lane (n, g) holds columns 16 hh + 8 g + e (the
  // fragment-ordered copy of W^T holds them so: fragment (block rb, step ks) at wt + ks * 512)
  const int rk = wave >> 2, rb = wave & 3;
  const T* wt = (const T*)P.w_t + ((size_t)h * (DKVH / 32) + rb) * (dc / 16) * 512 + l * 8;
  const T* cg = (const T*)P.c_kv + (size_t)b * S * dc + 8 * g;

  f32x16 dqa[DQK / 32];
#pragma unroll
  for (int i = 0; i < DQK / 32; ++i) dqa[i] = f32x16{};

  for (int st = 0; st < nsteps; ++st) {
    const int kt = st * KB;
    __syncthreads();  // the previous step's reads of sK / sD are done
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {  // this wave's dS^T blocks of the step (a dummy when not stored)
      const int kb = kt + 32 * sub;
      const T* src = kb < nk ? dtile + (size_t)kb * 32 : dtile;
      g2lds16(src + l * 8, sD + (wave * 2 + sub) * 1024);
      g2lds16(src + 512 + l * 8, sD + (wave * 2 + sub) * 1024 + 512);
    }
    {  // k_pe rows: wave w copies keys 8 w .. 8 w + 7 (rows past S clamped: their dS is zero)
      const int r = wave * 8 + (l >> 3);
      const int key = min(kt + r, S - 1);
      const chunk16 v = *reinterpret_cast<const chunk16*>(kpe + (size_t)(b * S + key) * DR + (l & 7) * 8);
      *reinterpret_cast<chunk16*>(sK + r * KP * 8 + DN + (l & 7) * 8) = v;
    }
    {  // K_nope block (rk, rb)
      const int key = min(kt + 32 * rk + n, S - 1);
      const T* cr = cg + (size_t)key * dc;
      f32x16 acc = f32x16{};
      for (int k0 = 0; k0 < dc / 16; k0 += 8) {  // d_c % 128 == 0: 16 loads in flight, then 8 MFMAs
        frag_t<T> wa[8], cb[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          wa[j] = *reinterpret_cast<const frag_t<T>*>(wt + (k0 + j) * 512);
          cb[j] = *reinterpret_cast<const frag_t<T>*>(cr + (k0 + j) * 16);
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) mma(acc, wa[j], cb[j]);
      }
      T* dst = sK + (32 * rk + n) * KP * 8 + rb * 32 + 8 * g;
      *reinterpret_cast<bf16x8*>(dst) = acc_to_frag<T>(acc, 0);
      *reinterpret_cast<bf16x8*>(dst + 16) = acc_to_frag<T>(acc, 1);
    }
    wait_vmem();
    __syncthreads();
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      if (kt + 32 * sub < nk) {  // wave-uniform: key blocks past the tile's queries hold no dS
        const T* tk = sK + 32 * sub * KP * 8;
        const T* td = sD + (wave * 2 + sub) * 1024;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          const int ra = kk * 16 + 4 * g;
          const bf16x8 zf = pad_tr_frag<4>(td, ra, ra + 8, 0);
#pragma unroll
          for (int db = 0; db < DQK / 32; ++db) mma(dqa[db], pad_tr_frag<KP>(tk, ra, ra + 8, db * 32), zf);
        }
      }
    }
  }

  const int my_q = t * 32 + ds_query_of_position(n);
  if (!wave_ok || my_q >= S) return;
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

// The same product with the K_nope rebuild organised around its operand traffic (d_c =
// 512): 4 waves (one per SIMD); wave w owns K_nope column block w and keeps its 32 rows of
// W_h^T (pi-ordered, 32 fragments) in registers for the whole kernel, and TPW
// consecutive 32-query tiles (the rebuilt K tile serves 32 * 4 * TPW queries, which sets
// the rebuild's share of the work: 1.33x the dQ products at TPW = 2). Per 64-key step the
// latent rows are copied once into LDS (direct loads, one 1 KB row per wave instruction,
// rows padded to 65 chunks: conflict-free row fragments) and each wave rebuilds its
// column block for both 32-key halves (two independent accumulator chains), so W_h^T is
// read once per workgroup and each latent row once per step. The copies of step s + 1
// (latent rows into the then free sC, dS^T blocks into the other of two sD stages, k_pe
// rows into registers) are issued right after the rebuild of step s, so that they land
// while the step's dQ products run. Operand roles, contraction order and rounding are
// those of dq_ds_fused_kernel: the K tile and dq are the same bit for bit.
template <int DN, int DR, int DV, int DC, int TPW>
__global__ __launch_bounds__(256, 1) void dq_ds_fused2_kernel(BwdParams P) {
  using T = bf16;
  constexpr int DQK = DN + DR, DKVH = DN + DV, NW = 4, KB = 64, NKS = DC / 16;
  constexpr int KP = DQK / 8 + 4;  // K tile pitch in 16-byte chunks (% 8 == 4: transposing reads)
  constexpr int CP = DC / 8 + 1;   // latent row pitch in chunks (odd: row fragments conflict-free)
  constexpr int DSW = TPW * 2 * 32 * 32;  // dS^T elements per wave and step
  static_assert(DN == NW * 32 && DR == 64 && DC == 64 * 8, "one 32-column K_nope block per wave; a latent row per copy");
  static_assert(TPW == 1 || TPW == 2, "one or two query tiles per wave");
  static_assert(KB * DR / 8 == 64 * NW * 2, "two k_pe chunks per thread and step");
  __shared__ __attribute__((aligned(16))) T sC[KB * CP * 8];
  __shared__ __attribute__((aligned(16))) T sK[KB * KP * 8];
  __shared__ __attribute__((aligned(16))) T sD0[NW * DSW], sD1[NW * DSW];

  const T* __restrict__ kpe = (const T*)P.k_pe;
  const T* __restrict__ ds = (const T*)P.ds;
  const int S = P.S, H = P.H, TT = P.ds_T;

  const int total = P.n_blocks * H * gridDim.y;
  const int lin = xcd_remap(blockIdx.x + gridDim.x * blockIdx.y, total);
  const int qblk = P.n_blocks - 1 - lin % P.n_blocks;  // heavy first
  const int bh = lin / P.n_blocks;
  const int b = bh / H, h = bh % H;

  const int tid = threadIdx.x, l = tid & 63, n = l & 31, g = l >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) & (NW - 1);
  const int t0 = (qblk * NW + wave) * TPW;  // this wave's query tiles t0 .. t0 + TPW - 1
  int nk[TPW];
  const T* dtile[TPW];
#pragma unroll
  for (int i = 0; i < TPW; ++i) {
    const bool ok = t0 + i < TT;
    nk[i] = ok ? ds_tile_keys(TT, P.causal, t0 + i) : 0;  // keys stored for the tile
    dtile[i] = ds + (ok ? ds_tile_offset(TT, P.causal, bh, t0 + i) : 0);
  }
  const int kend = P.causal ? min(S, (qblk + 1) * NW * TPW * 32) : S;
  const int nsteps = (kend + KB - 1) / KB;

  // W_h^T rows of this wave's column block in the order pi (bits 2 and 3 swapped), so
  // that lane (n, g) of the rebuild accumulator holds columns 16 hh + 8 g + e (the
  // fragment-ordered copy of W^T holds them so)
  frag_t<T> wf[NKS];
  {
    // W_h^T in fragment order: fragment (column block wave, step ks) at wt + ks * 512
    const T* wt = (const T*)P.w_t + ((size_t)h * (DKVH / 32) + wave) * NKS * 512 + l * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) wf[ks] = *reinterpret_cast<const frag_t<T>*>(wt + ks * 512);
  }
  const T* cg = (const T*)P.c_kv + (size_t)b * S * DC;

  f32x16 dqa[TPW][DQK / 32];
#pragma unroll
  for (int i = 0; i < TPW; ++i)
#pragma unroll
    for (int j = 0; j < DQK / 32; ++j) dqa[i][j] = f32x16{};

  // copies of step s: latent rows kt .. kt + 63 (rows past S clamped: their dS is zero),
  // wave w rows 16 w ..; the wave's dS^T blocks (a dummy block when not stored); k_pe rows
  // through registers (stored into the K tile after the next barrier)
  auto load_latent = [&](int kt) {
#pragma unroll
    for (int i = 0; i < KB / NW; ++i) {
      const int r = wave * (KB / NW) + i;
      g2lds16(cg + (size_t)min(kt + r, S - 1) * DC + l * 8, sC + r * CP * 8);
    }
  };
  auto load_ds = [&](T* sD, int kt) {
#pragma unroll
    for (int i = 0; i < TPW; ++i)
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
        const int kb = kt + 32 * sub;
        const T* src = kb < nk[i] ? dtile[i] + (size_t)kb * 32 : dtile[i];
        T* dst = sD + wave * DSW + (i * 2 + sub) * 1024;
        g2lds16(src + l * 8, dst);
        g2lds16(src + 512 + l * 8, dst + 512);
      }
  };
  chunk16 pe[2];
  auto load_pe = [&](int kt) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = tid + i * 64 * NW, r = c / (DR / 8), ch = c % (DR / 8);
      pe[i] = *reinterpret_cast<const chunk16*>(kpe + (size_t)(b * S + min(kt + r, S - 1)) * DR + ch * 8);
    }
  };
  auto store_pe = [&]() {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = tid + i * 64 * NW, r = c / (DR / 8), ch = c % (DR / 8);
      *reinterpret_cast<chunk16*>(sK + r * KP * 8 + DN + ch * 8) = pe[i];
    }
  };

  constexpr int PF = 3;
  load_latent(0);
  load_ds(sD0, 0);
  load_pe(0);
  auto step = [&](auto stage, int st) {
    constexpr int SD = decltype(stage)::value;
    T* sDc = SD == 0 ? sD0 : sD1;  // this step's dS^T stage
    T* sDn = SD == 0 ? sD1 : sD0;  // the next step's
    const int kt = st * KB;
    wait_vmem();      // this wave's copies of step st (latent rows, dS^T, k_pe) have landed
    __syncthreads();  // everyone's; the previous step's reads of sK and of sDn are done
    store_pe();
    {  // K_nope column block `wave` for keys kt .. kt + 63: two chains, one per 32-key half
      auto c_frag = [&](int i) {  // product i: contraction step i / 2 of key half i % 2
        return *reinterpret_cast<const frag_t<T>*>(sC + (32 * (i & 1) + n) * CP * 8 + (i >> 1) * 16 + 8 * g);
      };
      f32x16 acc[2] = {f32x16{}, f32x16{}};
      frag_t<T> cb[PF + 1];
#pragma unroll
      for (int i = 0; i < PF; ++i) cb[i] = c_frag(i);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < 2 * NKS; ++i) {
        if (i + PF < 2 * NKS) cb[(i + PF) % (PF + 1)] = c_frag(i + PF);
        mma(acc[i & 1], wf[i >> 1], cb[i % (PF + 1)]);
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
        T* dst = sK + (32 * kh + n) * KP * 8 + wave * 32 + 8 * g;
        *reinterpret_cast<bf16x8*>(dst) = acc_to_frag<T>(acc[kh], 0);
        *reinterpret_cast<bf16x8*>(dst + 16) = acc_to_frag<T>(acc[kh], 1);
      }
    }
    __syncthreads();  // the whole K tile is in LDS; every wave's reads of sC are done
    if (st + 1 < nsteps) {  // the next step's copies, behind this step's dQ products
      load_latent(kt + KB);
      load_ds(sDn, kt + KB);
      load_pe(kt + KB);
    }
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      const T* tk = sK + 32 * sub * KP * 8;
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const int ra = kk * 16 + 4 * g;
        bf16x8 zf[TPW];
#pragma unroll
        for (int i = 0; i < TPW; ++i) zf[i] = pad_tr_frag<4>(sDc + wave * DSW + (i * 2 + sub) * 1024, ra, ra + 8, 0);
#pragma unroll
        for (int db = 0; db < DQK / 32; ++db) {
          const bf16x8 kf = pad_tr_frag<KP>(tk, ra, ra + 8, db * 32);
          // wave-uniform: key blocks past a tile's queries hold no dS for it
#pragma unroll
          for (int i = 0; i < TPW; ++i)
            if (kt + 32 * sub < nk[i]) mma(dqa[i][db], kf, zf[i]);
        }
      }
    }
  };
  for (int st = 0; st < nsteps; st += 2) {
    step(std::integral_constant<int, 0>{}, st);
    if (st + 1 < nsteps) step(std::integral_constant<int, 1>{}, st + 1);
  }

#pragma unroll
  for (int i = 0; i < TPW; ++i) {
    const int my_q = (t0 + i) * 32 + ds_query_of_position(n);
    if (t0 + i >= TT || my_q >= S) continue;
    T* dqr = (T*)P.dq + ((size_t)(b * S + my_q) * H + h) * DQK;
#pragma unroll
    for (int db = 0; db < DQK / 32; ++db)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        bf16x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = to_elem<T>(dqa[i][db][4 * rr + e] * P.scale);
        *reinterpret_cast<bf16x4*>(dqr + db * 32 + rr * 8 + g * 4) = v;
      }
  }
}

}  // namespace

// dq_ds_kernel's shapes: 8 waves (two per SIMD, which hides the latency of the dS^T
// stream). With two 32-query tiles per wave a K fragment read from LDS feeds two MFMAs,
// halving the K traffic through LDS, over a three-stage ring (four do not fit in LDS at
// 46 KB a stage); it needs a grid of at least two workgroups per CU, below which one
// tile per wave over a four-stage ring (twice the workgroups) is faster. Measured (16
// heads, dQ stage alone): S=16384 0.98 ms (two tiles) against 1.04 ms (one); S=8192 0.357
// against 0.278 ms; S=2048 0.084 against 0.050 ms. Both shapes give the same bits. 4 waves
// with two tiles 1.37 ms, with one 1.63 ms at S=16384.
constexpr int kDqWaves = 8;
constexpr long long kDqWideMinGroups = 512;

// dq_rec_kernel's shape: 4 waves (one per SIMD, 128 queries per workgroup). Measured at
// S=16384, H=16: 2.16-2.38 ms; 8 waves need more than their 256 registers (98 spilled):
// 7.8 ms. Interleaving one key block's dS arithmetic with the other's MFMAs in a pinned
// order measured 2 % slower than the plain order.
#ifndef DQ_REC_WAVES
#define DQ_REC_WAVES 4
#endif

template <typename T, int DN, int DR, int DV>
hipError_t launch_bwd_dq(bwd::BwdParams P, int B, hipStream_t st) {
  using Tl = BwdTiles<T>;
  constexpr int BR = 32 * Tl::WPH_Q;
  P.n_blocks = (P.S + BR - 1) / BR;
  if constexpr (sizeof(T) == 2 && DN + DR == 192 && DV == 128) {
    if (P.ds) {
      if (P.w_t && P.d_c == kFusedMaxDc) {
        constexpr int TPW = 2;
        P.n_blocks = (P.ds_T + 4 * TPW - 1) / (4 * TPW);
        dq_ds_fused2_kernel<DN, DR, DV, kFusedMaxDc, TPW><<<dim3(P.n_blocks * P.H, B), 256, 0, st>>>(P);
      } else if (P.w_t) {
        constexpr int WPH = 8;
        P.n_blocks = (P.ds_T + WPH - 1) / WPH;
        dq_ds_fused_kernel<DN, DR, DV><<<dim3(P.n_blocks * P.H, B), 64 * WPH, 0, st>>>(P);
      } else {
        // kDqWaves waves x 1 or 2 query tiles of 32 per workgroup
        const int nb_wide = (P.ds_T + 2 * kDqWaves - 1) / (2 * kDqWaves);
        if ((long long)nb_wide * P.H * B >= kDqWideMinGroups) {
          P.n_blocks = nb_wide;
          dq_ds_kernel<DN, DR, DV, kDqWaves, 3, 2><<<dim3(P.n_blocks * P.H, B), 64 * kDqWaves, 0, st>>>(P);
        } else {
          P.n_blocks = (P.ds_T + kDqWaves - 1) / kDqWaves;
          dq_ds_kernel<DN, DR, DV, kDqWaves, 4, 1><<<dim3(P.n_blocks * P.H, B), 64 * kDqWaves, 0, st>>>(P);
        }
      }
      return hipGetLastError();
    }
  }
  if constexpr (sizeof(T) == 2 && DN == 128 && DR == 64 && DV == 128) {
    // no dS^T store: recompute S, P, dP and dS per key tile
    constexpr int RW = DQ_REC_WAVES;
    P.n_blocks = (P.S + 32 * RW - 1) / (32 * RW);
    dq_rec_kernel<DN, DR, DV, RW><<<dim3(P.n_blocks * P.H, B), 64 * RW, 0, st>>>(P);
    return hipGetLastError();
  }
  dq_kernel<T, DN, DR, DV, Tl::BC, Tl::WPH_Q><<<dim3(P.n_blocks * P.H, B), 64 * Tl::WPH_Q, 0, st>>>(P);
  return hipGetLastError();
}

#define LAGA_INST_DQ(T, DN, DR, DV) template hipError_t launch_bwd_dq<T, DN, DR, DV>(bwd::BwdParams, int, hipStream_t);
LAGA_INST_DQ(bf16, 128, 64, 128)
LAGA_INST_DQ(float, 128, 64, 128)
LAGA_INST_DQ(bf16, 32, 16, 32)
LAGA_INST_DQ(float, 32, 16, 32)
LAGA_INST_DQ(bf16, 64, 32, 64)
LAGA_INST_DQ(float, 64, 32, 64)

}  // namespace laga
