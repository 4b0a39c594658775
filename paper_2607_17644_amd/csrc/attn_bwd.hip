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
//   dkdv32_kernel  key-stationary dK/dV for bf16 with 192/128-wide heads: a wave owns
//                  32 keys of one head and sweeps the query tiles at or after them;
//                  lane <-> key layout (S = Q K^T with K in registers), so P and dZ
//                  feed dV^T += dO^T P and dK^T += Q^T dZ directly from the
//                  accumulators, with dO^T / Q^T read by transposing LDS reads;
//                  software-pipelined on the 32x32x16 MFMA (see there); unless dq is
//                  to be recomputed, it also stores dS^T for the dQ pass
//   dkpe_kernel    dk_pe = sum over heads (ascending) of the per-head k_pe parts
// in attn_bwd_kv.hip: dkdv_kernel, the same key-stationary pass for the other element
// types and head widths; and in attn_bwd_dq.hip: dq_kernel (query-stationary: a
// workgroup owns 32*WPH queries of one head and sweeps the key tiles up to the
// diagonal, recomputing S and dP - the price of not accumulating dQ with atomics), and
// for bf16 with 192/128-wide heads dq_ds_kernel (dQ as a product over the stored dS^T),
// dq_rec_kernel (dQ recomputed, no S x S buffer) and the fused-mode dQ kernels that
// rebuild K from the latent.
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

// Key-stationary dK/dV for bf16 with 192/128-wide heads: 32 keys per wave on the
// 32x32x16 MFMA, one wave per SIMD (4 waves, 128 keys per workgroup). The wave's K and V
// rows (A operands) and its dK^T / dV^T accumulators stay in registers for the whole
// sweep (about 450 registers with the pipeline below); a 32x32x16 fragment read from LDS
// feeds 32 Kflop, so per (query, key) pair the kernel reads half the LDS bytes of a
// 16-key layout. Per 32-query tile t:
//   A(t): S = Q K^T, dP = dO V^T        20 MFMAs on Q / dO row fragments
//   B(t): P = exp2(S c - lse2), dZ = P (dP - delta), the dS^T store    VALU
//   C(t): dV^T += dO^T P, dK^T += Q^T dZ  20 MFMAs on transposing reads of dO / Q
// In the first key block of each head (keys 0..127) the rope band of dK^T also takes dZ's
// low part (dZ as a bf16 pair hi + lo, 4 more MFMAs per tile): dk_pe sums that band over
// every head, and the first keys are the ones every query attends to, so there the bf16
// rounding of dZ, summed over all queries, is the largest error of the block's gradients;
// a key j's share of it scales with sum_i P_ij^2, which falls off quickly past the first
// keys. dK_nope, dV and dQ take the hi part only.
// With no second wave on its SIMD to hide latencies, the wave overlaps B(t-1) with A(t)
// (the softmax of one tile beside the MFMAs of the next; S and dP of consecutive tiles
// alternate between two accumulator sets), then runs C(t-1); the instruction order is
// fixed with sched_barrier, LDS reads issued three MFMAs ahead, each exponential one
// slot before the product that uses it. Query tiles (Q, dO, and each wave's copy of
// the tile's lse2 / delta rows) stream through a four-slot LDS ring of direct
// global->LDS loads into XOR-swizzled tiles, two tiles ahead. Every wave sweeps all of
// the workgroup's tiles (those before its own keys run fully masked and add exact
// zeros), so a tile's ring slot is the same in every wave: the loop is unrolled over
// the four slots and every LDS read is a per-lane base register plus an immediate
// offset, with no address arithmetic in the loop. The per-wave issue rate, not the LDS,
// is then its limit. It also stores dZ (bf16) as dS^T for the dQ pass.
// Low part of an accumulator half rounded to bf16: bf16(x - float(hi)) for the 8 values
// that acc_to_frag turned into `hi`, so that hi + lo carries about 16 significant bits
// (x - float(hi) is exact in fp32).
__device__ __forceinline__ bf16x8 acc_lo_frag(const f32x16& acc, int half, const bf16x8& hi) {
  typedef float f32x8v __attribute__((ext_vector_type(8)));
  f32x8v v;
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = acc[8 * half + e] - (float)hi[e];
  return __builtin_convertvector(v, bf16x8);
}

template <int DN, int DR, int DV, bool STORE_DS, bool FUSED>
__global__ __launch_bounds__(256, 1) void dkdv32_kernel(BwdParams P) {
  using T = bf16;
  constexpr int DQK = DN + DR, DKVH = DN + DV, NW = 4, BK = 32 * NW, BQ = 32, NS = 4;
  constexpr int QCPR = DQK / 8, OCPR = DV / 8;
  static_assert(QCPR == 24 && OCPR == 16, "swizzles are defined for 192/128-wide rows");
  constexpr int QCH = BQ * QCPR, OCH = BQ * OCPR;
  constexpr int KQ = QCH / 64 / NW, KO = OCH / 64 / NW;
  static_assert(KQ * 64 * NW == QCH && KO * 64 * NW == OCH && 5 * (KQ + KO) <= 32, "load split");
  constexpr int F = KQ + KO + 1;
  constexpr int QTB = QCH * 16, OTB = OCH * 16;  // tile bytes
  // dK^T blocks RB, RB + 1 are the rope band [DN, DN + DR): their product takes dZ as a bf16
  // pair hi + lo, because dk_pe sums that band over every head and every query
  constexpr int RB = DN / 32;
  static_assert(DR == 64 && RB + 2 == DQK / 32, "two 32-wide rope blocks at the end of dK^T");
  __shared__ __attribute__((aligned(16))) T sQ[NS][QCH * 8];
  __shared__ __attribute__((aligned(16))) T sO[NS][OCH * 8];
  __shared__ __attribute__((aligned(16))) float sL[NS][NW][256];

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

  const int tid = threadIdx.x, l = tid & 63, n = l & 31, g = l >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) & (NW - 1);
  const int k0 = kb * BK + wave * 32;
  const int my_k = k0 + n;
  const bool key_ok = my_k < S;
  const size_t krow = (size_t)(b * S + (key_ok ? my_k : 0));
  const int q_lo = P.causal ? my_k : 0;
  const unsigned q_span = key_ok ? (unsigned)(S - q_lo) : 0u;

  const int qt_begin = P.causal ? kb * BK : 0;
  const int ntiles = (S - qt_begin + BQ - 1) / BQ;

  const size_t hrow0 = (size_t)(b * S) * H + h;
  uint32_t qoff[KQ], ooff[KO], rows = 0;
#pragma unroll
  for (int k = 0; k < KQ; ++k) {
    const int p = (wave + k * NW) * 64 + l, r = p / QCPR, c = (p % QCPR) ^ swz<QCPR>(r);
    qoff[k] = 2u * (r * H * DQK + c * 8);
    rows |= (uint32_t)r << (5 * k);
  }
#pragma unroll
  for (int k = 0; k < KO; ++k) {
    const int p = (wave + k * NW) * 64 + l, r = p / OCPR, c = (p % OCPR) ^ swz<OCPR>(r);
    ooff[k] = 2u * (r * H * DV + c * 8);
    rows |= (uint32_t)r << (5 * (KQ + k));
  }
  const float* llane = ((l & 15) < 8 ? P.lse2 : P.delta) + (size_t)bh * P.S_pad + 4 * (l & 7);
  auto fill = [&](int st, int qt) {
    const T* qb = q + (hrow0 + (size_t)qt * H) * DQK;
    const T* ob = dout + (hrow0 + (size_t)qt * H) * DV;
    if (qt + BQ <= S) {
#pragma unroll
      for (int k = 0; k < KQ; ++k) g2lds16_so(qb, qoff[k], &sQ[st][(wave + k * NW) * 512]);
#pragma unroll
      for (int k = 0; k < KO; ++k) g2lds16_so(ob, ooff[k], &sO[st][(wave + k * NW) * 512]);
    } else {
      const int rmax = S - 1 - qt;
#pragma unroll
      for (int k = 0; k < KQ; ++k) {
        const int over = max((int)((rows >> (5 * k)) & 31u) - rmax, 0);
        g2lds16_so(qb, qoff[k] - 2u * over * H * DQK, &sQ[st][(wave + k * NW) * 512]);
      }
#pragma unroll
      for (int k = 0; k < KO; ++k) {
        const int over = max((int)((rows >> (5 * (KQ + k))) & 31u) - rmax, 0);
        g2lds16_so(ob, ooff[k] - 2u * over * H * DV, &sO[st][(wave + k * NW) * 512]);
      }
    }
    g2lds16(llane + qt, sL[st][wave]);
  };

  frag_t<T> kf[DQK / 16], vf[DV / 16];
  if constexpr (FUSED) {
    // The wave's K_nope / V rows rebuilt from the latent: KV^T (kv columns x 32 keys) =
    // W_h^T c^T, contracted over d_c in ascending 16-wide steps from zero with A = rows of
    // W^T and B = rows of c - the operand roles, order and bf16 rounding of the up-
    // projection GEMM, so every element equals the materialised kv bit for bit. The
    // accumulator lays lane (n, g) on rows 8 (r / 4) + 4 g + r % 4 of a 32-column block;
    // feeding W^T's rows in the order pi (bits 2 and 3 of the row swapped) puts columns
    // 16 h + 8 g + e (h = r / 8, e = r % 8) there instead, which is exactly the layout of
    // the two 16-wide B-operand fragments of that block: no data movement afterwards.
    static_assert(DN % 32 == 0 && DV % 32 == 0, "32-column blocks");
    const int dc = P.d_c;
    // W_h^T in fragment order with each block's rows in the order pi (written so by the
    // first stage): fragment (column block b, step ks) at wt + (b * dc / 16 + ks) * 512,
    // one coalesced 1 KB read per wave
    const T* wt = (const T*)P.w_t + (size_t)h * (DKVH / 32) * (dc / 16) * 512 + l * 8;
    const T* cr = (const T*)P.c_kv + krow * dc + 8 * g;
    constexpr int NB = DKVH / 32;
    f32x16 acc[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[b] = f32x16{};
    // groups of four 16-wide steps (d_c % 128 == 0): 36 loads in flight, then 32 MFMAs
    for (int k0 = 0; k0 < dc / 16; k0 += 4) {
      frag_t<T> cf[4], wf[4][NB];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        cf[j] = *reinterpret_cast<const frag_t<T>*>(cr + (k0 + j) * 16);
#pragma unroll
        for (int b = 0; b < NB; ++b)
          wf[j][b] = *reinterpret_cast<const frag_t<T>*>(wt + ((size_t)b * (dc / 16) + k0 + j) * 512);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int b = 0; b < NB; ++b) mma(acc[b], wf[j][b], cf[j]);
    }
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const frag_t<T> f = key_ok ? acc_to_frag<T>(acc[b], hh) : frag_t<T>{};
        if (b < DN / 32) kf[2 * b + hh] = f;
        else vf[2 * (b - DN / 32) + hh] = f;
      }
#pragma unroll
    for (int ks = DN / 16; ks < DQK / 16; ++ks) {
      kf[ks] = *reinterpret_cast<const frag_t<T>*>(kpe + krow * DR + (ks - DN / 16) * 16 + 8 * g);
      if (!key_ok) kf[ks] = frag_t<T>{};
    }
  } else {
    const T* kvr = kv + (krow * H + h) * DKVH;
#pragma unroll
    for (int ks = 0; ks < DQK / 16; ++ks) {
      const T* src = ks < DN / 16 ? kvr + ks * 16 + 8 * g : kpe + krow * DR + (ks - DN / 16) * 16 + 8 * g;
      kf[ks] = *reinterpret_cast<const frag_t<T>*>(src);
      if (!key_ok) kf[ks] = frag_t<T>{};
    }
#pragma unroll
    for (int ks = 0; ks < DV / 16; ++ks) {
      vf[ks] = *reinterpret_cast<const frag_t<T>*>(kvr + DN + ks * 16 + 8 * g);
      if (!key_ok) vf[ks] = frag_t<T>{};
    }
  }
  f32x16 dk[DQK / 32], dv[DV / 32];
#pragma unroll
  for (int i = 0; i < DQK / 32; ++i) dk[i] = f32x16{};
#pragma unroll
  for (int i = 0; i < DV / 32; ++i) dv[i] = f32x16{};

  // per-lane LDS addresses inside slot 0 of each ring (laundered through an empty asm so
  // that the compiler keeps one register per base and folds slot and step offsets into
  // the reads' immediate offsets); other slots and steps are immediates
  typedef __attribute__((address_space(3))) const char* lptr;
  typedef __attribute__((address_space(3))) const frag_t<T> lfrag;
  typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
  auto base = [](const void* arr, uint32_t off) {
    lptr p = (lptr)(const char*)arr + off;
    asm volatile("" : "+v"(p));
    return p;
  };
  lptr Qr[4], Qa[2], Qbo[2], Or[DV / 16], Oa[DV / 32], Obo[DV / 32];
  {
    const int s16 = l & 15, ra = 4 * g + (s16 >> 2), rb = ra + 8;
    const int lc = 2 * ((l >> 4) & 1) + ((s16 & 3) >> 1), e4 = 4 * (s16 & 1);
    const int sq = swz<QCPR>(n), so = swz<OCPR>(n);
#pragma unroll
    for (int j = 0; j < 4; ++j) Qr[j] = base(sQ, 2u * (n * DQK + ((2 * j + g) ^ sq) * 8));
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      Qa[j] = base(sQ, 2u * (ra * DQK + ((4 * j + lc) ^ swz<QCPR>(ra)) * 8 + e4));
      Qbo[j] = base(sQ, 2u * (rb * DQK + ((4 * j + lc) ^ swz<QCPR>(rb)) * 8 + e4));
    }
#pragma unroll
    for (int ks = 0; ks < DV / 16; ++ks) Or[ks] = base(sO, 2u * (n * DV + ((2 * ks + g) ^ so) * 8));
#pragma unroll
    for (int db = 0; db < DV / 32; ++db) {
      Oa[db] = base(sO, 2u * (ra * DV + ((4 * db + lc) ^ swz<OCPR>(ra)) * 8 + e4));
      Obo[db] = base(sO, 2u * (rb * DV + ((4 * db + lc) ^ swz<OCPR>(rb)) * 8 + e4));
    }
  }
  auto tr = [](lptr pa, lptr pb) {
    const bf16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)pa);
    const bf16x4 y = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)pb);
    return __builtin_shufflevector(x, y, 0, 1, 2, 3, 4, 5, 6, 7);
  };
  auto rowq = [&](int st, int ks) { return *(lfrag*)(Qr[ks & 3] + (st * QTB + (ks >> 2) * 128)); };
  auto rowo = [&](int st, int ks) { return *(lfrag*)(Or[ks] + st * OTB); };
  // C operand i of tile slot st: query half kk = i / 10; blocks 0..5 of dK^T, then 0..3 of dV^T
  auto c_read = [&](int st, int i) {
    const int kk = i / 10, m = i % 10;
    if (m < DQK / 32) {
      const int c = st * QTB + kk * 16 * DQK * 2 + (m >> 1) * 128;
      return tr(Qa[m & 1] + c, Qbo[m & 1] + c);
    }
    const int db = m - DQK / 32, c = st * OTB + kk * 16 * DV * 2;
    return tr(Oa[db] + c, Obo[db] + c);
  };
  auto step_a = [&](int st, f32x16& sa, f32x16& dp) {
    sa = f32x16{};
    dp = f32x16{};
#pragma unroll
    for (int ks = 0; ks < DQK / 16; ++ks) {
      mma(sa, rowq(st, ks), kf[ks]);
      if (ks < DV / 16) mma(dp, rowo(st, ks), vf[ks]);
    }
  };
  auto mask_b = [&](int j, f32x16& sa) {
    const int qt = qt_begin + j * BQ;
    if ((P.causal && qt < k0 + 31) || qt + BQ > S || k0 + 32 > S) {
      asm volatile("");
#pragma unroll
      for (int r = 0; r < 16; ++r)
        sa[r] = (unsigned)(qt + (r >> 2) * 8 + g * 4 + (r & 3) - q_lo) < q_span ? sa[r] : -INFINITY;
    }
  };
  auto step_b = [&](auto hc, int st, const f32x16& sa, const f32x16& dp, bf16x8 (&pf)[2], bf16x8 (&zf)[2],
                    bf16x8 (&zl)[2]) {
    constexpr bool HILO = decltype(hc)::value;
    const float* tl = sL[st][wave];
    f32x16 p, z;
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const f32x4 lq = *reinterpret_cast<const f32x4*>(tl + rr * 8 + g * 4);
      const f32x4 dq = *reinterpret_cast<const f32x4*>(tl + BQ + rr * 8 + g * 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        p[rr * 4 + e] = fast_exp2(__builtin_fmaf(sa[rr * 4 + e], P.scale_log2, -lq[e]));
        z[rr * 4 + e] = p[rr * 4 + e] * (dp[rr * 4 + e] - dq[e]);
      }
    }
#pragma unroll
    for (int kk = 0; kk < BQ / 16; ++kk) {
      pf[kk] = acc_to_frag<T>(p, kk);
      zf[kk] = acc_to_frag<T>(z, kk);
      if constexpr (HILO) zl[kk] = acc_lo_frag(z, kk, zf[kk]);
    }
  };
  T* const dsw = STORE_DS ? (T*)P.ds + ds_tile_offset(P.ds_T, P.causal, bh, 0) + (size_t)k0 * BQ : nullptr;
  auto store_ds = [&](int j, const bf16x8 (&zf)[2]) {
    if constexpr (!STORE_DS) return;
    const int t = (qt_begin + j * BQ) / BQ;
    if (my_k < ds_tile_keys(P.ds_T, P.causal, t)) {
      // accumulator element r of this lane is query 8 (r / 4) + 4 g + r % 4: position 16 g + r.
      // Non-temporal: the store is read back only by the dQ pass, long after this kernel.
      T* dsr = dsw + (P.causal ? (size_t)512 * t * (t + 1) : (size_t)1024 * P.ds_T * t) + (n * BQ + g * 16);
#pragma unroll
      for (int kk = 0; kk < BQ / 16; ++kk)
        __builtin_nontemporal_store(zf[kk], reinterpret_cast<bf16x8*>(dsr + kk * 8));
    }
  };
  // Every tile step refills a slot, past the end with another copy of the last tile (a
  // slot nobody reads any more), so one tile of copies is always in flight behind the
  // awaited one and the wait needs no branch.
  auto tile_q = [&](int j) { return qt_begin + min(j, ntiles - 1) * BQ; };
  auto sync = [&](int j) {
    wait_vmem_le<F>();
    lds_barrier();
    fill((j + 2) % NS, tile_q(j + 2));
  };

  // The sweep over the query tiles, compiled twice: with HILO the rope band of dK^T takes
  // dZ as a bf16 pair hi + lo (the first key block of each head, see above).
  auto sweep = [&](auto hc) {
  constexpr bool HILO = decltype(hc)::value;
  fill(0, qt_begin);
  fill(1, tile_q(1));
  f32x16 sa0, dp0, sa1, dp1;
  bf16x8 pf[2], zf[2], zl[2];
  sync(0);
  step_a(0, sa0, dp0);
  constexpr int PF = 3;
  // step of tile jj (slot K = jj % 4): B(jj - 1) beside A(jj), then C(jj - 1)
  auto step = [&](auto kc, int jj) {
    constexpr int K = decltype(kc)::value;
    constexpr int ST = K, SP = (K + NS - 1) % NS, ODD = K & 1;
    f32x16& sa_a = ODD ? sa1 : sa0;
    f32x16& dp_a = ODD ? dp1 : dp0;
    f32x16& sa_b = ODD ? sa0 : sa1;
    f32x16& dp_b = ODD ? dp0 : dp1;
    sync(jj);
    mask_b(jj - 1, sa_b);
    const float* tl = sL[SP][wave];
    f32x4 lq[4], dq[4];
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      lq[rr] = *reinterpret_cast<const f32x4*>(tl + rr * 8 + g * 4);
      dq[rr] = *reinterpret_cast<const f32x4*>(tl + BQ + rr * 8 + g * 4);
    }
    auto a_is_s = [](int i) { return i >= 16 || (i & 1) == 0; };
    auto a_ks = [](int i) { return i >= 16 ? 8 + (i - 16) : i >> 1; };
    auto a_read = [&](int i) { return a_is_s(i) ? rowq(ST, a_ks(i)) : rowo(ST, a_ks(i)); };
    frag_t<T> ab[PF + 1];
#pragma unroll
    for (int i = 0; i < PF; ++i) ab[i] = a_read(i);
    __builtin_amdgcn_sched_barrier(0);
    f32x16 p, z;
#pragma unroll
    for (int i = 0; i < 20; ++i) {
      if (i + PF < 20) ab[(i + PF) % (PF + 1)] = a_read(i + PF);
      if (a_is_s(i))
        sa_a = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ab[i % (PF + 1)], kf[a_ks(i)], i == 0 ? f32x16{} : sa_a,
                                                       0, 0, 0);
      else
        dp_a = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ab[i % (PF + 1)], vf[a_ks(i)], i == 1 ? f32x16{} : dp_a,
                                                       0, 0, 0);
      // softmax element i (exp issued one slot before its product)
      if (i < 16) p[i] = fast_exp2(__builtin_fmaf(sa_b[i], P.scale_log2, -lq[i >> 2][i & 3]));
      if (i >= 1 && i <= 16) z[i - 1] = p[i - 1] * (dp_b[i - 1] - dq[(i - 1) >> 2][(i - 1) & 3]);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int kk = 0; kk < BQ / 16; ++kk) {
      pf[kk] = acc_to_frag<T>(p, kk);
      zf[kk] = acc_to_frag<T>(z, kk);
      if constexpr (HILO) zl[kk] = acc_lo_frag(z, kk, zf[kk]);
    }
    bf16x8 cb[PF + 1], c_r0, c_r1;
#pragma unroll
    for (int i = 0; i < PF; ++i) cb[i] = c_read(SP, i);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < 20; ++i) {
      if (i + PF < 20) cb[(i + PF) % (PF + 1)] = c_read(SP, i + PF);
      const int kk = i / 10, m = i % 10;
      if (m < DQK / 32) mma(dk[m], cb[i % (PF + 1)], zf[kk]);
      else mma(dv[m - DQK / 32], cb[i % (PF + 1)], pf[kk]);
      // the rope band of dK (blocks RB, RB + 1) also takes dZ's low part, each one
      // product later so that no MFMA waits on the one just before it
      if constexpr (HILO) {
        if (m == RB) c_r0 = cb[i % (PF + 1)];
        if (m == RB + 1) {
          c_r1 = cb[i % (PF + 1)];
          mma(dk[RB], c_r0, zl[kk]);
        }
        if (m == RB + 2) mma(dk[RB + 1], c_r1, zl[kk]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    store_ds(jj - 1, zf);
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  {
    int j = 1;
    for (; j + 3 < ntiles; j += 4) {
      step(I1{}, j);
      step(I2{}, j + 1);
      step(I3{}, j + 2);
      step(I0{}, j + 3);
    }
    if (j < ntiles) step(I1{}, j++);
    if (j < ntiles) step(I2{}, j++);
    if (j < ntiles) step(I3{}, j++);
  }
  // the last tile's B and C (its slot and parity are not known at compile time)
  {
    const int jl = ntiles - 1, sl = jl % NS;
    if (jl & 1) {
      mask_b(jl, sa1);
      step_b(hc, sl, sa1, dp1, pf, zf, zl);
    } else {
      mask_b(jl, sa0);
      step_b(hc, sl, sa0, dp0, pf, zf, zl);
    }
#pragma unroll
    for (int i = 0; i < 20; ++i) {
      const int kk = i / 10, m = i % 10;
      const bf16x8 c = c_read(sl, i);
      if (m < DQK / 32) mma(dk[m], c, zf[kk]);
      else mma(dv[m - DQK / 32], c, pf[kk]);
      if (HILO && m >= RB && m < DQK / 32) mma(dk[m], c, zl[kk]);
    }
    store_ds(jl, zf);
  }
  };
  if (kb == 0) sweep(std::true_type{});
  else sweep(std::false_type{});
  wait_vmem();  // the surplus copies land before the workgroup's LDS is released

  if (!key_ok) return;
  const size_t row = krow * H + h;
  T* dkvr = (T*)P.dkv + row * DKVH;
  T* dkvl = (T*)P.dkv_lo + row * DKVH;
  float* dper = P.dkpe_h + row * DR;
  auto put = [&](int col, const f32x4& v) {
    bf16x4 hi, lo;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      hi[e] = to_elem<T>(v[e]);
      lo[e] = to_elem<T>(v[e] - to_f32(hi[e]));
    }
    *reinterpret_cast<bf16x4*>(dkvr + col) = hi;
    *reinterpret_cast<bf16x4*>(dkvl + col) = lo;
  };
#pragma unroll
  for (int db = 0; db < DQK / 32; ++db)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int d = db * 32 + rr * 8 + g * 4;
      f32x4 v;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = dk[db][4 * rr + e] * P.scale;
      if (d >= DN) *reinterpret_cast<f32x4*>(dper + (d - DN)) = v;
      else put(d, v);
    }
#pragma unroll
  for (int db = 0; db < DV / 32; ++db)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      f32x4 v;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = dv[db][4 * rr + e];
      put(DN + db * 32 + rr * 8 + g * 4, v);
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
  P.c_kv = a.c_kv; P.w_t = a.w_t; P.d_c = a.d_c;
  if (stage == 0) {
    const int BS = a.B * a.S;
    delta_kernel<T, DV><<<(BS + 3) / 4, 256, 0, st>>>((const T*)a.out, (const T*)a.dout, a.lse, a.delta, a.lse2,
                                                      a.S, a.S_pad, a.H, BS);
  } else if (stage == 1) {
    if constexpr (sizeof(T) == 2 && DN + DR == 192 && DV == 128) {
      P.n_blocks = (a.S + 127) / 128;
      const dim3 grid(P.n_blocks * a.H, a.B);
      if (a.w_t) {
        if (a.ds) dkdv32_kernel<DN, DR, DV, true, true><<<grid, 256, 0, st>>>(P);
        else dkdv32_kernel<DN, DR, DV, false, true><<<grid, 256, 0, st>>>(P);
      } else {
        if (a.ds) dkdv32_kernel<DN, DR, DV, true, false><<<grid, 256, 0, st>>>(P);
        else dkdv32_kernel<DN, DR, DV, false, false><<<grid, 256, 0, st>>>(P);
      }
    } else {
      return launch_dkdv_generic<T, DN, DR, DV>(P, a.B, st);
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
LAGA_INST_BWD(bf16, 64, 32, 64)
LAGA_INST_BWD(float, 64, 32, 64)

}  // namespace laga
