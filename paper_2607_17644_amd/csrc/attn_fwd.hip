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

    const bool active = head_ok && q0 < S && (!P.causal || kt <= q0 + 31);
    if (!active) continue;

    f32x16 sacc[BC / 32];
#pragma unroll
    for (int kb = 0; kb < BC / 32; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[kb][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < DQK / 16; ++ks) {
        const frag_t<T> a = ks < DN / 16
            ? lds_frag<T>(sKh + (kb * 32 + n) * C::PK + ks * 16 + 8 * g)
            : lds_frag<T>(sP + (kb * 32 + n) * C::PP + (ks - DN / 16) * 16 + 8 * g);
        mma(sacc[kb], a, qf[ks]);
      }
    }

    // scale (base 2) and mask; only tiles crossing the diagonal or the end need the mask
    const bool need_mask = (P.causal && kt + BC - 1 > q0) || (kt + BC > S);
    float mloc = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < BC / 32; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float s = sacc[kb][r] * P.scale_log2;
        if (need_mask) {
          const int key = kt + kb * 32 + (r >> 2) * 8 + g * 4 + (r & 3);
          if (key >= S || (P.causal && key > my_q)) s = -INFINITY;
        }
        sacc[kb][r] = s;
        mloc = fmaxf(mloc, s);
      }
    mloc = wave_xor32_max(mloc);
    const float m_new = fmaxf(m, mloc);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = fast_exp2(m - m_use);
    float ps = 0.f;
#pragma unroll
    for (int kb = 0; kb < BC / 32; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = fast_exp2(sacc[kb][r] - m_use);
        sacc[kb][r] = p;
        ps += p;
      }
    lsum = lsum * alpha + ps;
    m = m_new;
#pragma unroll
    for (int i = 0; i < DV / 32; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[i][r] *= alpha;

    frag_t<T> pf[BC / 16];
#pragma unroll
    for (int kk = 0; kk < BC / 16; ++kk) pf[kk] = acc_to_frag<T>(sacc[kk >> 1], kk & 1);
#pragma unroll
    for (int db = 0; db < DV / 32; ++db)
#pragma unroll
      for (int kk = 0; kk < BC / 16; ++kk) {
        const int ra = kk * 16 + 4 * g;
        const frag_t<T> a = TrRead<T>::get(sVh, C::PV, ra, ra + 8, db * 32);
        mma(oacc[db], a, pf[kk]);
      }
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

template <typename T, int DN, int DR, int DV> struct FwdTiles;
template <int DN, int DR, int DV> struct FwdTiles<bf16, DN, DR, DV> {
  static constexpr int BC = 64, WPH = 4, G = 1;
};
template <int DN, int DR, int DV> struct FwdTiles<float, DN, DR, DV> {
  static constexpr int BC = 32, WPH = 4, G = 1;
};

}  // namespace

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
  using Cfg = FwdCfg<T, DN, DR, DV, Tl::BC, Tl::WPH, Tl::G, false>;
  attn_fwd_kernel<T, DN, DR, DV, Tl::BC, Tl::WPH, Tl::G, false><<<grid, Cfg::NT, 0, st>>>(P);
  return hipGetLastError();
}

#define LAGA_INST_FWD(T, DN, DR, DV) template hipError_t launch_attn_fwd<T, DN, DR, DV>(const AttnFwdArgs&, hipStream_t);
LAGA_INST_FWD(bf16, 128, 64, 128)
LAGA_INST_FWD(float, 128, 64, 128)
LAGA_INST_FWD(bf16, 32, 16, 32)
LAGA_INST_FWD(float, 32, 16, 32)

}  // namespace laga
