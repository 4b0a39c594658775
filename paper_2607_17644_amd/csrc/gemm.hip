// MFMA GEMMs of the up-projection and its backward (gfx950).
//
//   reconstruct : kv[B*S, H*(d_nope+d_v)] = c_kv[B*S, d_c] @ W_kv_b     (Alg. 1 step 4)
//   dc          : dc_kv[B*S, d_c] = dKV[B*S, H*(d_nope+d_v)] @ W_kv_b^T   (fp32 out)
//   dW          : dW[d_c, H*(d_nope+d_v)] = c_kv^T @ dKV  (split over tokens,
//                 fixed-order reduction: deterministic)
//
// One kernel template covers all three: each operand is either "k-contiguous"
// (stored [rows][K]) or "k-strided" (stored [K][rows]); both are staged into
// LDS as stored and strided operands are read back with transposing LDS reads,
// so there is no transpose pass anywhere. The output tile is computed as
// C^T = B^T A^T block by block, which puts 4 consecutive output columns in each
// lane's accumulators for vectorised stores.
//
// The reconstruct (a 512-long contraction writing 256 bytes per output row and head)
// runs as a persistent variant of the large-tile kernel that spreads each tile's
// stores over the next tile's MFMAs (gemm_stream_kernel); dc and dW, whose dKV operand
// comes as a bf16 pair hi + lo, run the large tiles on eight waves (gemm_big8_kernel).
//
// Per output element the contraction runs over K in ascending 16-wide steps
// (one MFMA each) with fp32 accumulation; tile shapes and the dW token split do
// not depend on N, so a column of the output is bit-identical whatever N (the
// number of heads) is. (dc_kv's contraction runs over the heads and may be split
// into partials summed in a fixed order.)
// direct global->LDS copies issued as inline assembly (exact LDS-read waits; the
// ring orders the copies with explicit waits and barriers)
#define LAGA_LDS_DMA_ASM 1
#include "common.hpp"
#include "kernels.hpp"

namespace laga {

namespace {

constexpr int kThreads = 256;

template <typename T, bool KSTRIDED, int ROWS, int BK>
struct OperandTile {
  static constexpr int E = Elems16<T>::n;                      // elements per 16-byte chunk
  // k-contiguous rows: +8 elements keeps 16-byte fragment reads conflict-free and
  // fp32 rows 32-byte aligned; k-strided rows: +32 bytes for the transposing reads.
  static constexpr int PITCH = KSTRIDED ? ROWS + 32 / (int)sizeof(T) : BK + 8;
  static constexpr int LDS_ELEMS = KSTRIDED ? BK * PITCH : ROWS * PITCH;
  static constexpr int CHUNKS = ROWS * BK / E;
  static constexpr int PER_THREAD = CHUNKS / kThreads;
  static_assert(CHUNKS % kThreads == 0, "tile must split evenly over the workgroup");

  chunk16 reg[PER_THREAD];

  // Global -> registers. rows [r0, r_end) valid, k [k0, k_end) valid; zero fill outside.
  __device__ __forceinline__ void load(const T* __restrict__ g, int ld, int r0, int r_end, int k0, int k_end) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int c = tid + i * kThreads;
      int r, k;
      if (!KSTRIDED) { r = c / (BK / E); k = (c % (BK / E)) * E; }
      else { k = c / (ROWS / E); r = (c % (ROWS / E)) * E; }
      const int gr = r0 + r, gk = k0 + k;
      const bool ok = (gr < r_end) && (gk < k_end);
      const T* src = KSTRIDED ? g + (size_t)gk * ld + gr : g + (size_t)gr * ld + gk;
      reg[i] = ok ? *reinterpret_cast<const chunk16*>(src) : zero_chunk();
    }
  }
  __device__ __forceinline__ void store(T* s) const {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int c = tid + i * kThreads;
      int r, k;
      if (!KSTRIDED) { r = c / (BK / E); k = (c % (BK / E)) * E; }
      else { k = c / (ROWS / E); r = (c % (ROWS / E)) * E; }
      T* dst = KSTRIDED ? s + k * PITCH + r : s + r * PITCH + k;
      *reinterpret_cast<chunk16*>(dst) = reg[i];
    }
  }
  // Fragment for the 32-row block starting at rb, contraction step ks.
  static __device__ __forceinline__ frag_t<T> frag(const T* s, int rb, int ks) {
    const int l = threadIdx.x & 63, g = l >> 5;
    if (!KSTRIDED) return lds_frag<T>(s + (rb + (l & 31)) * PITCH + ks * 16 + 8 * g);
    const int ra = ks * 16 + 8 * g;
    return TrRead<T>::get(s, PITCH, ra, ra + 4, rb);
  }
};

template <typename TO>
__device__ __forceinline__ void store4(TO* p, float a, float b, float c, float d);
template <>
__device__ __forceinline__ void store4<float>(float* p, float a, float b, float c, float d) {
  f32x4 v = {a, b, c, d};
  *reinterpret_cast<f32x4*>(p) = v;
}
template <>
__device__ __forceinline__ void store4<bf16>(bf16* p, float a, float b, float c, float d) {
  bf16x4 v = {(bf16)a, (bf16)b, (bf16)c, (bf16)d};
  *reinterpret_cast<bf16x4*>(p) = v;
}

// C (+ blockIdx.z * split_stride) [M][N] = A[M][K-range] B[K-range][N]
// SPLIT = 1: A is the sum of two arrays A + A2 of the same layout; SPLIT = 2: B = B + B2.
// (A value held as a bf16 pair hi + lo keeps ~16 significant bits through a bf16 MFMA;
// per k-step the hi product is accumulated before the lo product.)
template <typename T, typename TO, bool A_KS, bool B_KS, int BM, int BN, int BK, int SPLIT>
__global__ __launch_bounds__(kThreads) void gemm_kernel(
    const T* __restrict__ A, const T* __restrict__ B, const T* __restrict__ X2, TO* __restrict__ C,
    int M, int N, int K, int lda, int ldb, int ldc, int k_chunk, long long split_stride) {
  using TA = OperandTile<T, A_KS, BM, BK>;
  using TB = OperandTile<T, B_KS, BN, BK>;
  constexpr int WM = BM / 64, WN = BN / 64;  // 32x32 blocks per wave along m and n
  constexpr int A2_ELEMS = SPLIT == 1 ? TA::LDS_ELEMS : 1;
  constexpr int B2_ELEMS = SPLIT == 2 ? TB::LDS_ELEMS : 1;
  __shared__ __attribute__((aligned(16))) T sA[TA::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) T sB[TB::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) T sA2[A2_ELEMS];
  __shared__ __attribute__((aligned(16))) T sB2[B2_ELEMS];

  const int n_tiles = (N + BN - 1) / BN;
  const int m_tiles = (M + BM - 1) / BM;
  const int lin = xcd_remap(blockIdx.x, n_tiles * m_tiles);
  const int tn = lin % n_tiles, tm = lin / n_tiles;
  const int m0 = tm * BM, n0 = tn * BN;
  const int kb = blockIdx.z * k_chunk;
  const int ke = min(K, kb + k_chunk);

  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63, g = l >> 5;
  const int wm = wave & 1, wn = wave >> 1;

  f32x16 acc[WN][WM];
#pragma unroll
  for (int j = 0; j < WN; ++j)
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[j][i][r] = 0.f;

  TA ta, ta2; TB tb, tb2;
  auto load = [&](int k0) {
    ta.load(A, lda, m0, M, k0, ke);
    tb.load(B, ldb, n0, N, k0, ke);
    if (SPLIT == 1) ta2.load(X2, lda, m0, M, k0, ke);
    if (SPLIT == 2) tb2.load(X2, ldb, n0, N, k0, ke);
  };
  auto store = [&]() {
    ta.store(sA); tb.store(sB);
    if (SPLIT == 1) ta2.store(sA2);
    if (SPLIT == 2) tb2.store(sB2);
  };
  load(kb);
  store();
  __syncthreads();
  for (int k0 = kb; k0 < ke; k0 += BK) {
    const bool more = k0 + BK < ke;
    if (more) load(k0 + BK);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      frag_t<T> fa[WM], fb[WN];
#pragma unroll
      for (int i = 0; i < WM; ++i) fa[i] = TA::frag(sA, (wm * WM + i) * 32, ks);
#pragma unroll
      for (int j = 0; j < WN; ++j) fb[j] = TB::frag(sB, (wn * WN + j) * 32, ks);
      if (SPLIT == 0) {
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
          for (int i = 0; i < WM; ++i) mma(acc[j][i], fb[j], fa[i]);
      } else if (SPLIT == 1) {
        frag_t<T> fa2[WM];
#pragma unroll
        for (int i = 0; i < WM; ++i) fa2[i] = TA::frag(sA2, (wm * WM + i) * 32, ks);
        // all hi products, then all lo ones (per accumulator the same order; see gemm_big_kernel)
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
          for (int i = 0; i < WM; ++i) mma(acc[j][i], fb[j], fa[i]);
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
          for (int i = 0; i < WM; ++i) mma(acc[j][i], fb[j], fa2[i]);
      } else {
        frag_t<T> fb2[WN];
#pragma unroll
        for (int j = 0; j < WN; ++j) fb2[j] = TB::frag(sB2, (wn * WN + j) * 32, ks);
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
          for (int i = 0; i < WM; ++i) mma(acc[j][i], fb[j], fa[i]);
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
          for (int i = 0; i < WM; ++i) mma(acc[j][i], fb2[j], fa[i]);
      }
    }
    __syncthreads();
    if (more) { store(); __syncthreads(); }
  }

  TO* Cz = C + blockIdx.z * split_stride;
#pragma unroll
  for (int j = 0; j < WN; ++j)
#pragma unroll
    for (int i = 0; i < WM; ++i) {
      const int m = m0 + (wm * WM + i) * 32 + (l & 31);
      if (m >= M) continue;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int n = n0 + (wn * WN + j) * 32 + rr * 8 + g * 4;
        if (n < N)
          store4<TO>(Cz + (size_t)m * ldc + n, acc[j][i][4 * rr], acc[j][i][4 * rr + 1],
                     acc[j][i][4 * rr + 2], acc[j][i][4 * rr + 3]);
      }
    }
}

// ------------------------------------------------------------------ large tiles (bf16)
// A workgroup of four waves computes a BM x BN output tile (BM * BN = 4 * 128 * 128),
// one wave per SIMD, each wave 128 x 128 (4 x 4 blocks of 32 x 32, 256 accumulator
// registers per lane): an LDS operand fragment then feeds four MFMAs, so LDS reads
// stay well under the LDS rate. Besides 256 x 256, 128 x 512 and 512 x 128 tiles cover
// a whole 512-wide side, so the other (large) operand is read from memory once (the
// backward's dc and dW take those shapes on gemm_big8_kernel below, two waves per SIMD).
// The contraction advances 32 at a time through an LDS ring of NSLOT stages filled by
// direct global->LDS copies issued NSLOT - 1 stages ahead (a stage of MFMAs is shorter
// than the latency of a load from memory); one barrier per stage, placed inside the
// second half of the stage's MFMAs, with the next stage's first operands read before
// the last MFMAs.
//
// Operand tiles are ROWS (the non-contraction index) x 32 contraction indices, stored
// unpadded as the copies fill them (a wave instruction fills 64 consecutive 16-byte
// chunks), with an XOR swizzle of the chunk index that keeps the operand reads
// conflict-free under the LDS bank model:
//   k-contiguous ([ROWS][32]: 4 chunks per row): chunk c of row r at c ^ ((r >> 2) & 3).
//     A row fragment read (32 rows, one chunk per half-wave) then covers 16 distinct
//     16-byte slots in each 16-lane pass.
//   k-strided ([32][ROWS]: ROWS / 8 chunks per k row, rows a multiple of 256 bytes):
//     chunk c of k row r at c ^ (4 (r & 3)). A transposing read covers 4 consecutive
//     k rows x 4 chunks per half-wave, which the XOR spreads over the four 64-byte
//     quarters of the banks.
constexpr int kGK = 32;  // contraction per stage

// This lane's share of the copies of one operand tile (ROWS / 16 instructions, wave w
// of NWV issues w, w + NWV, ...).
template <bool KS, int ROWS, int NWV = 4>
struct GFill {
  static constexpr int NI = ROWS / 16, PER = NI / NWV, CPR = ROWS / 8;
  static_assert(PER * NWV == NI, "whole copy instructions per wave");
  uint32_t off[PER];  // byte offsets from the stage origin of the operand
  // r0: first row (column for KS) of the tile; rlim: number of rows (columns) in the operand.
  __device__ __forceinline__ void init(int wave, int l, int ld, int r0, int rlim) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int p = (wave + NWV * i) * 64 + l;
      if (!KS) {
        const int row = p >> 2, c = (p & 3) ^ ((row >> 2) & 3);
        off[i] = 2u * (uint32_t)(min(r0 + row, rlim - 1) * ld + c * 8);  // rows past the end read the last
      } else {
        const int kr = p / CPR, c = (p % CPR) ^ (4 * (kr & 3));
        off[i] = 2u * (uint32_t)(kr * ld + min(r0 + c * 8, rlim - 8));  // columns past the end likewise
      }
    }
  }
  __device__ __forceinline__ void fill(const bf16* stage_origin, bf16* tile, int wave) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) g2lds16_so(stage_origin, off[i], tile + (wave + NWV * i) * 512);
  }
};

// Operand fragments of one wave's BW 32-row blocks (rows 32 BW wsel .. of the tile),
// contraction step ks (16 wide) of the stage.
template <bool KS, int ROWS, int BW = 4>
struct GRead {
  static_assert(BW == 2 || BW == 4, "two or four blocks per wave");
  int off[BW > 2 ? BW : 2];  // element offsets: k-contiguous uses [0..1] (per ks), k-strided one per block
  __device__ __forceinline__ void init(int l, int wsel) {
    const int g = l >> 5;
    if (!KS) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) off[ks] = (l & 31) * kGK + ((2 * ks + g) ^ ((l >> 2) & 3)) * 8;
    } else {
      // transposing read of k rows ra + s/4 (ra = 16 ks + 8 g; second half ra + 4) and
      // columns 32 b + 16 ((l >> 4) & 1) + 4 (s & 3) .. +3, s = l % 16, b = BW wsel + j;
      // logical chunk 4 b + lc of k row r sits at chunk 4 (b ^ (r & 3)) + lc, r & 3 = s / 4
      const int s = l & 15, j4 = s >> 2, lc = 2 * ((l >> 4) & 1) + ((s & 3) >> 1);
#pragma unroll
      for (int j = 0; j < BW; ++j)
        off[j] = j4 * ROWS + 8 * g * ROWS + (4 * ((BW * wsel + j) ^ j4) + lc) * 8 + 4 * (s & 1);
    }
  }
  __device__ __forceinline__ bf16x8 get(const bf16* tile, int wsel, int ks, int j) const {
    if (!KS) return *reinterpret_cast<const bf16x8*>(tile + (32 * BW * wsel + 32 * j) * kGK + off[ks]);
    typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
    const bf16* p = tile + off[j] + 16 * ks * ROWS;
    const bf16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)p);
    const bf16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p + 4 * ROWS));
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  }
};

// C (+ blockIdx.z * split_stride) [M][N] = A[M][k range] B[k range][N], bf16 operands,
// fp32 accumulation. SPLIT as in gemm_kernel (1: A + X2, 2: B + X2; hi before lo per
// k-step). The k range of a split is a multiple of 32; M, N multiples of 8.
template <int BM, int BN, bool A_KS, bool B_KS, int SPLIT, typename TO>
__global__ __launch_bounds__(256, 1) void gemm_big_kernel(
    const bf16* __restrict__ A, const bf16* __restrict__ B, const bf16* __restrict__ X2, TO* __restrict__ C,
    int M, int N, int K, int lda, int ldb, int ldc, int k_chunk, long long split_stride) {
  static_assert(BM * BN == 4 * 128 * 128 && BM % 128 == 0 && BN % 128 == 0, "four 128 x 128 waves");
  constexpr int WM = BM / 128;                     // waves along m
  constexpr int NT = SPLIT ? 3 : 2;                // operand tiles per stage: A, B (, X2)
  constexpr int NSLOT = SPLIT ? 3 : 4;             // ring depth (LDS: 144 or 128 KB)
  constexpr bool X_KS = SPLIT == 1 ? A_KS : B_KS;
  constexpr int XR = SPLIT == 1 ? BM : BN;         // rows of the X2 tile
  constexpr int TA = BM * kGK, TB = BN * kGK, TX = SPLIT ? XR * kGK : 0;
  constexpr int STAGE = TA + TB + TX;              // elements per stage
  __shared__ __attribute__((aligned(16))) bf16 sm[NSLOT * STAGE];

  const int n_tiles = (N + BN - 1) / BN, m_tiles = (M + BM - 1) / BM;
  const int lin = xcd_remap(blockIdx.x, n_tiles * m_tiles);
  const int tn = lin % n_tiles, tm = lin / n_tiles;
  const int m0 = tm * BM, n0 = tn * BN;
  const int kb = blockIdx.z * k_chunk;
  const int nst = (min(K, kb + k_chunk) - kb) / kGK;  // stages

  const int l = threadIdx.x & 63, g = l >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) & 3;
  const int wm = wave % WM, wn = wave / WM;

  GFill<A_KS, BM> fa;
  GFill<B_KS, BN> fb;
  GFill<X_KS, XR> fx;
  fa.init(wave, l, lda, m0, M);
  fb.init(wave, l, ldb, n0, N);
  if (SPLIT) fx.init(wave, l, SPLIT == 1 ? lda : ldb, SPLIT == 1 ? m0 : n0, SPLIT == 1 ? M : N);
  auto fill = [&](int slot, int k) {
    bf16* st = sm + slot * STAGE;
    fa.fill(A_KS ? A + (size_t)k * lda : A + k, st, wave);
    fb.fill(B_KS ? B + (size_t)k * ldb : B + k, st + TA, wave);
    if (SPLIT == 1) fx.fill(A_KS ? X2 + (size_t)k * lda : X2 + k, st + TA + TB, wave);
    if (SPLIT == 2) fx.fill(B_KS ? X2 + (size_t)k * ldb : X2 + k, st + TA + TB, wave);
  };
  constexpr int F = GFill<A_KS, BM>::PER + GFill<B_KS, BN>::PER + (SPLIT ? GFill<X_KS, XR>::PER : 0);
  // wait until the copies of a stage have landed while `ahead` later stages may still
  // be in flight (copies complete in issue order)
  auto wait_stage = [](int ahead) {
    if (ahead >= 3) wait_vmem_le<3 * F>();
    else if (ahead == 2) wait_vmem_le<2 * F>();
    else if (ahead == 1) wait_vmem_le<F>();
    else wait_vmem();
  };
  static_assert(NSLOT <= 4 && 3 * F < 64, "vmcnt range");

  GRead<A_KS, BM> ra;
  GRead<B_KS, BN> rb;
  GRead<X_KS, XR> rx;
  ra.init(l, wm);
  rb.init(l, wn);
  const int xsel = SPLIT == 1 ? wm : wn;
  if (SPLIT) rx.init(l, xsel);

  f32x16 acc[4][4];  // [n block][m block]: C^T blocks, lane <-> m, 4 consecutive n per lane
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[j][i] = f32x16{};

  bf16x8 fA[2][4], fB[2][4], fX[2][4];  // operands of contraction steps 0 and 1 of a stage
  auto read = [&](int slot, int ks) {
    const bf16* st = sm + slot * STAGE;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      fA[ks][j] = ra.get(st, wm, ks, j);
      fB[ks][j] = rb.get(st + TA, wn, ks, j);
      if (SPLIT) fX[ks][j] = rx.get(st + TA + TB, xsel, ks, j);
    }
  };
  // n blocks [j0, j1) of step ks. With a low-half operand every accumulator takes the hi
  // product before the lo one as before, but all hi products of the call are issued first:
  // an MFMA that accumulates onto the one just issued waits for its result, so back-to-back
  // hi, lo pairs on one accumulator would run the matrix unit at half rate.
  auto mmas = [&](int ks, int j0, int j1) {
#pragma unroll
    for (int j = j0; j < j1; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) mma(acc[j][i], fB[ks][j], fA[ks][i]);
    if (SPLIT)
#pragma unroll
      for (int j = j0; j < j1; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (SPLIT == 1) mma(acc[j][i], fB[ks][j], fX[ks][i]);
          if (SPLIT == 2) mma(acc[j][i], fX[ks][j], fA[ks][i]);
        }
  };

  const int npre = min(NSLOT, nst);
  for (int t = 0; t < npre; ++t) fill(t, kb + t * kGK);
  wait_stage(npre - 1);  // stage 0 has landed
  lds_barrier();
  read(0, 0);
  // (the last stage is peeled: every trip of the loop then ends with the next stage's
  // first operands in flight, and the compiler's LDS waits stay exact)
  // Instruction order within a stage (the scheduler would otherwise bunch the LDS
  // reads and the waits on them): step-1 reads interleaved with the step-0 MFMAs, in
  // four groups; then half of the step-1 MFMAs; barrier and copies; the next stage's
  // step-0 reads interleaved with the other half.
  constexpr int RPS = (A_KS ? 8 : 4) + (B_KS ? 8 : 4) + (SPLIT ? (X_KS ? 8 : 4) : 0);  // LDS reads per step
  constexpr int MPJ = SPLIT ? 8 : 4;  // MFMAs per n block and step
  constexpr int DS_READ = 0x100, MFMA = 0x008;
  for (int t = 0; t < nst - 1; ++t) {
    const int slot = t % NSLOT;
    read(slot, 1);
    mmas(0, 0, 4);
    mmas(1, 0, 2);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      __builtin_amdgcn_sched_group_barrier(DS_READ, RPS / 4, 0);
      __builtin_amdgcn_sched_group_barrier(MFMA, MPJ, 0);
    }
    __builtin_amdgcn_sched_group_barrier(MFMA, 2 * MPJ, 0);
    __builtin_amdgcn_sched_barrier(0);
    wait_stage(min(NSLOT - 2, nst - 2 - t));  // this wave's copies of stage t + 1 have landed
    lds_barrier();  // ... everyone's; and every read of stage t is done
    if (t + NSLOT < nst) fill(slot, kb + (t + NSLOT) * kGK);
    __builtin_amdgcn_sched_barrier(0);
    read((t + 1) % NSLOT, 0);
    mmas(1, 2, 4);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      __builtin_amdgcn_sched_group_barrier(DS_READ, RPS / 2, 0);
      __builtin_amdgcn_sched_group_barrier(MFMA, MPJ, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  read((nst - 1) % NSLOT, 1);
  mmas(0, 0, 4);
  mmas(1, 0, 4);

  TO* Cz = C + blockIdx.z * split_stride;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + 128 * wm + 32 * i + (l & 31);
      if (m >= M) continue;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int n = n0 + 128 * wn + 32 * j + rr * 8 + g * 4;
        if (n < N)
          store4<TO>(Cz + (size_t)m * ldc + n, acc[j][i][4 * rr], acc[j][i][4 * rr + 1], acc[j][i][4 * rr + 2],
                     acc[j][i][4 * rr + 3]);
      }
    }
}

// The same product on eight waves, two per SIMD (the backward's dc and dW, whose dKV
// operand is a bf16 pair hi + lo, and W_o's backward): each wave owns 64 x 128
// (BM <= BN) or 128 x 64 of the output, 8 accumulator blocks (128 registers), so two
// waves fit on a SIMD and one wave's copies, LDS reads and barrier waits overlap the
// other's MFMAs. Stages, copies, swizzles and the per-element accumulation order
// (ascending 16-wide steps, hi before lo per step) are gemm_big_kernel's, so results
// are bit-identical to it.
template <int BM, int BN, bool A_KS, bool B_KS, int SPLIT, typename TO>
__global__ __launch_bounds__(512, 1) void gemm_big8_kernel(
    const bf16* __restrict__ A, const bf16* __restrict__ B, const bf16* __restrict__ X2, TO* __restrict__ C,
    int M, int N, int K, int lda, int ldb, int ldc, int k_chunk, long long split_stride) {
  static_assert(BM * BN == 4 * 128 * 128, "the 4-wave tile shapes");
  constexpr int NWV = 8;
  constexpr int WGM = BM <= BN ? 2 : 4, WGN = NWV / WGM;  // waves along m, along n
  constexpr int WTM = BM / WGM, WTN = BN / WGN;           // one wave's output tile
  constexpr int NI = WTM / 32, NJ = WTN / 32;             // its 32 x 32 blocks
  static_assert(NI * NJ == 8 && (NI == 2 || NI == 4) && (NJ == 2 || NJ == 4), "8 blocks per wave");
  constexpr int NSLOT = SPLIT ? 3 : 4;                    // ring depth (144 or 128 KB)
  constexpr bool X_KS = SPLIT == 1 ? A_KS : B_KS;
  constexpr int XR = SPLIT == 1 ? BM : BN;
  constexpr int XB = SPLIT == 1 ? NI : NJ;                // X2 blocks per wave
  constexpr int TA = BM * kGK, TB = BN * kGK, TX = SPLIT ? XR * kGK : 0;
  constexpr int STAGE = TA + TB + TX;
  __shared__ __attribute__((aligned(16))) bf16 sm[NSLOT * STAGE];

  const int n_tiles = (N + BN - 1) / BN, m_tiles = (M + BM - 1) / BM;
  const int lin = xcd_remap(blockIdx.x, n_tiles * m_tiles);
  const int tn = lin % n_tiles, tm = lin / n_tiles;
  const int m0 = tm * BM, n0 = tn * BN;
  const int kb = blockIdx.z * k_chunk;
  const int nst = (min(K, kb + k_chunk) - kb) / kGK;

  const int l = threadIdx.x & 63, g = l >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) & (NWV - 1);
  const int wm = wave % WGM, wn = wave / WGM;

  GFill<A_KS, BM, NWV> fa;
  GFill<B_KS, BN, NWV> fb;
  GFill<X_KS, XR, NWV> fx;
  fa.init(wave, l, lda, m0, M);
  fb.init(wave, l, ldb, n0, N);
  if (SPLIT) fx.init(wave, l, SPLIT == 1 ? lda : ldb, SPLIT == 1 ? m0 : n0, SPLIT == 1 ? M : N);
  auto fill = [&](int slot, int k) {
    bf16* st = sm + slot * STAGE;
    fa.fill(A_KS ? A + (size_t)k * lda : A + k, st, wave);
    fb.fill(B_KS ? B + (size_t)k * ldb : B + k, st + TA, wave);
    if (SPLIT == 1) fx.fill(A_KS ? X2 + (size_t)k * lda : X2 + k, st + TA + TB, wave);
    if (SPLIT == 2) fx.fill(B_KS ? X2 + (size_t)k * ldb : X2 + k, st + TA + TB, wave);
  };
  constexpr int F = GFill<A_KS, BM, NWV>::PER + GFill<B_KS, BN, NWV>::PER + (SPLIT ? GFill<X_KS, XR, NWV>::PER : 0);
  auto wait_stage = [](int ahead) {
    if (ahead >= 3) wait_vmem_le<3 * F>();
    else if (ahead == 2) wait_vmem_le<2 * F>();
    else if (ahead == 1) wait_vmem_le<F>();
    else wait_vmem();
  };
  static_assert(3 * F < 64, "vmcnt range");

  GRead<A_KS, BM, NI> ra;
  GRead<B_KS, BN, NJ> rb;
  GRead<X_KS, XR, XB> rx;
  ra.init(l, wm);
  rb.init(l, wn);
  const int xsel = SPLIT == 1 ? wm : wn;
  if (SPLIT) rx.init(l, xsel);

  f32x16 acc[NJ][NI];  // [n block][m block]: C^T blocks, lane <-> m, 4 consecutive n per lane
#pragma unroll
  for (int j = 0; j < NJ; ++j)
#pragma unroll
    for (int i = 0; i < NI; ++i) acc[j][i] = f32x16{};

  bf16x8 fA[2][NI], fB[2][NJ], fX[2][XB];
  auto read = [&](int slot, int ks) {
    const bf16* st = sm + slot * STAGE;
#pragma unroll
    for (int i = 0; i < NI; ++i) fA[ks][i] = ra.get(st, wm, ks, i);
#pragma unroll
    for (int j = 0; j < NJ; ++j) fB[ks][j] = rb.get(st + TA, wn, ks, j);
    if (SPLIT)
#pragma unroll
      for (int x = 0; x < XB; ++x) fX[ks][x] = rx.get(st + TA + TB, xsel, ks, x);
  };
  // every hi product of the step, then every lo one (per accumulator: hi before lo)
  auto mmas = [&](int ks) {
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int i = 0; i < NI; ++i) mma(acc[j][i], fB[ks][j], fA[ks][i]);
    if (SPLIT)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int i = 0; i < NI; ++i) {
          if (SPLIT == 1) mma(acc[j][i], fB[ks][j], fX[ks][i]);
          if (SPLIT == 2) mma(acc[j][i], fX[ks][j], fA[ks][i]);
        }
  };

  const int npre = min(NSLOT, nst);
  for (int t = 0; t < npre; ++t) fill(t, kb + t * kGK);
  wait_stage(npre - 1);
  lds_barrier();
  read(0, 0);
  for (int t = 0; t < nst - 1; ++t) {
    const int slot = t % NSLOT;
    read(slot, 1);
    mmas(0);
    wait_stage(min(NSLOT - 2, nst - 2 - t));  // this wave's copies of stage t + 1 have landed
    lds_barrier();                            // ... everyone's; every read of stage t is done
    if (t + NSLOT < nst) fill(slot, kb + (t + NSLOT) * kGK);
    read((t + 1) % NSLOT, 0);
    mmas(1);
  }
  read((nst - 1) % NSLOT, 1);
  mmas(0);
  mmas(1);

  TO* Cz = C + blockIdx.z * split_stride;
#pragma unroll
  for (int j = 0; j < NJ; ++j)
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int m = m0 + WTM * wm + 32 * i + (l & 31);
      if (m >= M) continue;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int n = n0 + WTN * wn + 32 * j + rr * 8 + g * 4;
        if (n < N)
          store4<TO>(Cz + (size_t)m * ldc + n, acc[j][i][4 * rr], acc[j][i][4 * rr + 1], acc[j][i][4 * rr + 2],
                     acc[j][i][4 * rr + 3]);
      }
    }
}

// ------------------------------------------------------------------ streamed large tiles (bf16 out)
// The 256 x 256 tile (no split, bf16 output) for a short contraction such as the
// latent's 512, where the 256 x 256 x 2-byte results of a tile take as long to write as
// its MFMAs take to compute, and a workgroup per tile writes them all at once while
// every other CU does the same. Here a persistent workgroup takes tiles q = blockIdx.x,
// + gridDim.x, ... and one LDS ring runs through all of them (the next tile's first
// stages are copied while the current one finishes). Eight waves, two per SIMD, each
// own 128 x 64 of the tile (8 accumulator blocks). A finished tile's accumulators are
// rounded to bf16 and paired across the two half-waves (v_permlane32_swap: 8
// consecutive columns per lane) into 16 16-byte stores per wave, issued one per stage
// over the 16 stages of the next tile, so the writes run at an even rate behind the
// MFMAs. Per output element the products are accumulated in the same order as in
// gemm_big_kernel: the results are bitwise equal.
//
// Stores and copies share the in-order vmcnt counter: the stores issued in the last
// three stages are younger than the copies a stage waits for (those were issued three
// stages back) and older than none of them, so the ring's wait allows exactly that
// many more operations in flight.
constexpr int kStreamStoreStages = 16;  // stages over which a tile's stores are spread


template <int BM, int BN, bool A_KS, bool B_KS>
__global__ __launch_bounds__(512, 1) void gemm_stream_kernel(const bf16* __restrict__ A, const bf16* __restrict__ B,
                                                             bf16* __restrict__ C, int M, int N, int K, int lda,
                                                             int ldb, int ldc) {
  static_assert(BM == 256 && BN == 256, "eight 128 x 64 waves");
  constexpr int WM = 2;  // waves along m (128 rows each); four along n (64 columns each)
  constexpr int NSLOT = 4;
  constexpr int TA = BM * kGK, TB = BN * kGK, STAGE = TA + TB;
  __shared__ __attribute__((aligned(16))) bf16 sm[NSLOT * STAGE];
  typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;

  const int n_tiles = N / BN, n_items = n_tiles * (M / BM);
  const int G = gridDim.x, nst = K / kGK;                    // nst >= kStreamStoreStages
  const int mine = (n_items - 1 - (int)blockIdx.x) / G + 1;  // tiles of this workgroup
  const int total = mine * nst;                              // stages of this workgroup

  const int l = threadIdx.x & 63, g = l >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) & 7;
  const int wm = wave % WM, wn = wave / WM;

  GFill<A_KS, BM, 8> fa;
  GFill<B_KS, BN, 8> fb;
  fa.init(wave, l, lda, 0, BM);  // offsets within a tile; the tile origin goes into the base
  fb.init(wave, l, ldb, 0, BN);
  auto tile_at = [&](int it, int& m0, int& n0) {
    const int lin = xcd_remap((int)blockIdx.x + it * G, n_items);
    n0 = (lin % n_tiles) * BN;
    m0 = (lin / n_tiles) * BM;
  };
  int f_loc = 0, f_it = 0, f_m0, f_n0;  // the next stage to copy
  tile_at(0, f_m0, f_n0);
  auto fill_next = [&](int slot) {
    const int k = f_loc * kGK;
    bf16* st = sm + slot * STAGE;
    fa.fill(A_KS ? A + (size_t)k * lda + f_m0 : A + (size_t)f_m0 * lda + k, st, wave);
    fb.fill(B_KS ? B + (size_t)k * ldb + f_n0 : B + (size_t)f_n0 * ldb + k, st + TA, wave);
    if (++f_loc == nst) {
      f_loc = 0;
      if (++f_it < mine) {
        tile_at(f_it, f_m0, f_n0);
      } else {  // past the last stage: copy it again into slots nobody reads any more
        f_it = mine - 1;
        f_loc = nst - 1;
      }
    }
  };
  constexpr int F = GFill<A_KS, BM, 8>::PER + GFill<B_KS, BN, 8>::PER;  // copies per wave and stage
  constexpr int Y = 3;  // stores younger than the copies a stage waits for, in steady state
  static_assert(3 * F + Y + 2 < 64, "vmcnt range");

  GRead<A_KS, BM, 4> ra;
  GRead<B_KS, BN, 2> rb;
  ra.init(l, wm);
  rb.init(l, wn);

  f32x16 acc[2][4];
  bf16x8 fA[2][4], fB[2][2];
  u32x4 pay[8][2];  // the previous tile's results, block (j, i) = 4 j + i, as stored
  auto read = [&](int slot, int ks) {
    const bf16* st = sm + slot * STAGE;
#pragma unroll
    for (int i = 0; i < 4; ++i) fA[ks][i] = ra.get(st, wm, ks, i);
#pragma unroll
    for (int j = 0; j < 2; ++j) fB[ks][j] = rb.get(st + TA, wn, ks, j);
  };
  auto mmas = [&](int ks, int j0, int j1) {
#pragma unroll
    for (int j = j0; j < j1; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) mma(acc[j][i], fB[ks][j], fA[ks][i]);
  };
  // Results of block (j, i) as two 16-byte stores per lane: lane half g takes columns
  // 16 p + 8 g .. + 7 (p = 0, 1) of its row; within a lane the 16 accumulators are 4
  // runs (rr) of 4 consecutive columns at 8 rr + 4 g, so runs 2p and 2p + 1 are
  // exchanged with the other half-wave.
  auto pack = [&](int j, int i, u32x4 (&out)[2]) {
    uint32_t x[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
      const bf16x2 v = {(bf16)acc[j][i][2 * e], (bf16)acc[j][i][2 * e + 1]};
      x[e] = __builtin_bit_cast(uint32_t, v);
    }
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const auto r = __builtin_amdgcn_permlane32_swap(x[4 * p], x[4 * p + 2], false, false);
      const auto s = __builtin_amdgcn_permlane32_swap(x[4 * p + 1], x[4 * p + 3], false, false);
      out[p] = u32x4{r[0], s[0], r[1], s[1]};
    }
  };
  // half hh (columns 16 hh .. of the block) of block b: one 16-byte store per lane
  auto store = [&](const u32x4 (&v)[2], int m0, int n0, int b, int hh) {
    const int j = b >> 2, i = b & 3;
    bf16* row = C + (size_t)(m0 + 128 * wm + 32 * i + (l & 31)) * ldc + n0 + 64 * wn + 32 * j + 8 * g;
    *reinterpret_cast<u32x4*>(row + 16 * hh) = v[hh];
  };

  constexpr int RPS = (A_KS ? 8 : 4) + (B_KS ? 4 : 2);  // LDS reads per step
  constexpr int DS_READ = 0x100, MFMA = 0x008;
  // First half of stage t: step-1 reads interleaved with the step-0 MFMAs (which
  // restart every accumulator from zero in the first stage of a tile), then half of
  // the step-1 MFMAs.
  auto head = [&](int t, bool first) {
    read(t % NSLOT, 1);
    if (first) {
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          acc[j][i] = f32x16{};
          mma(acc[j][i], fB[0][j], fA[0][i]);
        }
    } else {
      mmas(0, 0, 2);
    }
    mmas(1, 0, 1);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      __builtin_amdgcn_sched_group_barrier(DS_READ, RPS / 4, 0);
      __builtin_amdgcn_sched_group_barrier(MFMA, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(MFMA, 4, 0);
    __builtin_amdgcn_sched_barrier(0);
  };
  // Second half of stage t: wait for stage t + 1, barrier, refill the slot of stage t,
  // read the step-0 operands of stage t + 1 with the other half of the step-1 MFMAs.
  // Every stage refills a slot (past the end with copies of the last stage), so two
  // stages of copies are always in flight behind the awaited one. With EXACT the wait
  // also leaves the Y stores of the last three stages in flight (they are younger than
  // the copies of stage t + 1, issued three stages back); otherwise it waits for them.
  // (s_waitcnt takes its count as an immediate: a count chosen at run time costs taken
  // branches every stage, which leave the matrix unit idle.)
  auto tail = [&](int t, auto exact) {
    if (decltype(exact)::value) wait_vmem_le<2 * F + Y>();
    else wait_vmem_le<2 * F>();
    lds_barrier();
    fill_next(t % NSLOT);
    __builtin_amdgcn_sched_barrier(0);
    read((t + 1) % NSLOT, 0);  // (after the last stage: a harmless read of a stale slot)
    mmas(1, 1, 2);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      __builtin_amdgcn_sched_group_barrier(DS_READ, RPS / 2, 0);
      __builtin_amdgcn_sched_group_barrier(MFMA, 2, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  };

  for (int t = 0; t < NSLOT; ++t) fill_next(t);  // (total >= kStreamStoreStages > NSLOT)
  wait_vmem_le<(NSLOT - 1) * F>();
  lds_barrier();
  read(0, 0);

  int c_m0 = 0, c_n0 = 0;  // the tile being accumulated
  int e_m0 = 0, e_n0 = 0;  // the tile whose results are being stored
  int t = 0;
  // the first kStreamStoreStages stages of tile it, storing the previous tile's results
  auto first_stages = [&](int it, auto exact) {
#pragma unroll
    for (int s = 0; s < kStreamStoreStages; ++s, ++t) {
      head(t, s == 0);
      if (it > 0) store(pay[s >> 1], e_m0, e_n0, s >> 1, s & 1);
      tail(t, exact);
    }
  };
  for (int it = 0; it < mine; ++it) {
    tile_at(it, c_m0, c_n0);
    // From the third tile on (and with exactly kStreamStoreStages stages per tile) every
    // stage has stores of its own and of the two stages before it in flight.
    if (it >= 2 && nst == kStreamStoreStages) first_stages(it, std::true_type{});
    else first_stages(it, std::false_type{});
    for (int s = kStreamStoreStages; s < nst; ++s, ++t) {
      head(t, false);
      tail(t, std::false_type{});
    }
#pragma unroll
    for (int b = 0; b < 8; ++b) pack(b >> 2, b & 3, pay[b]);
    e_m0 = c_m0;
    e_n0 = c_n0;
  }
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    store(pay[b], e_m0, e_n0, b, 0);
    store(pay[b], e_m0, e_n0, b, 1);
  }
  wait_vmem();  // the surplus copies land before the workgroup's LDS is released
}

// The streamed kernel applies to whole tiles and at least kStreamStoreStages stages per tile.
bool gemm_stream_ok(int M, int N, int K, size_t a_elems, size_t b_elems) {
  return M % 256 == 0 && N % 256 == 0 && K % kGK == 0 && K / kGK >= kStreamStoreStages && 2 * a_elems < (1ull << 32) &&
         2 * b_elems < (1ull << 32);
}

// The large-tile kernel applies to bf16 operands whose contraction range splits into
// multiples of 32, with M and N multiples of 8, and whose byte offsets within an
// operand fit the 32-bit offsets of the copies.
bool gemm_big_ok(int M, int N, int K, int k_chunk, size_t a_elems, size_t b_elems) {
  return K % kGK == 0 && k_chunk % kGK == 0 && M % 8 == 0 && N % 8 == 0 && M >= 8 && N >= 8 &&
         2 * a_elems < (1ull << 32) && 2 * b_elems < (1ull << 32);
}

// dst[i] = sum_{s < nsplit} src[s * stride + i], in ascending s (float4 granularity).
__global__ __launch_bounds__(256) void split_reduce_kernel(const float* __restrict__ src, float* __restrict__ dst,
                                                           long long n4, int nsplit, long long stride) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  f32x4 s = reinterpret_cast<const f32x4*>(src)[i];
  for (int k = 1; k < nsplit; ++k) {
    f32x4 v = reinterpret_cast<const f32x4*>(src + k * stride)[i];
    s += v;
  }
  reinterpret_cast<f32x4*>(dst)[i] = s;
}

template <typename T> struct GemmCfg;
template <> struct GemmCfg<bf16> { static constexpr int BM = 128, BN = 128, BK = 32; };
template <> struct GemmCfg<float> { static constexpr int BM = 64, BN = 64, BK = 16; };

inline int grid_tiles(int M, int N, int BM, int BN) { return ((M + BM - 1) / BM) * ((N + BN - 1) / BN); }
constexpr int kCUs = 256;  // compute units of the gfx950 part (one streamed workgroup each)

}  // namespace

template <typename T>
hipError_t launch_reconstruct(const T* c, const T* w, T* kv, int M, int N, int K, hipStream_t st) {
  using G = GemmCfg<T>;
  if constexpr (sizeof(T) == 2) {
    if (gemm_stream_ok(M, N, K, (size_t)M * K, (size_t)K * N)) {
      const int tiles = grid_tiles(M, N, 256, 256);
      gemm_stream_kernel<256, 256, false, true><<<tiles < kCUs ? tiles : kCUs, 512, 0, st>>>(
          c, w, kv, M, N, K, /*lda=*/K, /*ldb=*/N, /*ldc=*/N);
      return hipGetLastError();
    }
    if (gemm_big_ok(M, N, K, K, (size_t)M * K, (size_t)K * N)) {
      gemm_big_kernel<256, 256, false, true, 0, bf16><<<grid_tiles(M, N, 256, 256), 256, 0, st>>>(
          c, w, nullptr, kv, M, N, K, /*lda=*/K, /*ldb=*/N, /*ldc=*/N, /*k_chunk=*/K, 0);
      return hipGetLastError();
    }
  }
  dim3 grid(grid_tiles(M, N, G::BM, G::BN), 1, 1);
  gemm_kernel<T, T, false, true, G::BM, G::BN, G::BK, 0><<<grid, kThreads, 0, st>>>(
      c, w, nullptr, kv, M, N, K, /*lda=*/K, /*ldb=*/N, /*ldc=*/N, /*k_chunk=*/K, 0);
  return hipGetLastError();
}

namespace {
constexpr int kMinGemmBlocks = 512;  // workgroups wanted per GEMM launch (256 CUs)
// dc's output has d_c columns: a side of more than 256 takes 128 x 512 tiles (dKV read once)
inline int dc_bm(int d_c) { return d_c > 256 ? 128 : 256; }
}  // namespace

int dw_split_tokens(int tokens) {
  int s = 2048;
  while (s > 512 && (tokens + s - 1) / s < 4) s /= 2;
  return s;
}
size_t dw_split_count(int tokens) {
  const int s = dw_split_tokens(tokens);
  return (size_t)((tokens + s - 1) / s);
}
int dc_split_count(int tokens, int d_c, int K) {
  const bool big = gemm_big_ok(tokens, d_c, K, kGK, (size_t)tokens * K, (size_t)d_c * K);
  const int tiles = big ? grid_tiles(tokens, d_c, dc_bm(d_c), 65536 / dc_bm(d_c))
                        : grid_tiles(tokens, d_c, GemmCfg<bf16>::BM, GemmCfg<bf16>::BN);
  // at least 256 contraction indices (one 192/128-wide head) per split, and one split
  const int max_split = K >= 512 ? K / 256 : 1;
  // large tiles: one workgroup per CU (256) is enough; small tiles want two or more
  const int want = big ? 256 : kMinGemmBlocks;
  int n = (want + tiles - 1) / tiles;
  return n < 1 ? 1 : (n > max_split ? max_split : n);
}
size_t gemm_partial_elems(int tokens, int d_c, int K) {
  const size_t dw = dw_split_count(tokens) > 1 ? dw_split_count(tokens) * (size_t)d_c * K : 0;
  const int ndc = dc_split_count(tokens, d_c, K);
  const size_t dc = ndc > 1 ? (size_t)ndc * tokens * d_c : 0;
  return dw > dc ? dw : dc;
}

template <typename T>
hipError_t launch_dc(const T* dkv, const T* dkv_lo, const T* w, float* dc, float* partial, int M, int N, int K,
                     hipStream_t st) {
  // dc[M=tokens][N=d_c] = (dKV + dKV_lo)[M][K=H*dkvh] @ W^T ; W stored [N][K] (k-contiguous).
  // With a split contraction each split writes its partial and a fixed-order reduce sums them.
  using G = GemmCfg<T>;
  const int nsplit = sizeof(T) == 2 ? dc_split_count(M, N, K) : 1;
  const int k_chunk = (K / nsplit + G::BK - 1) / G::BK * G::BK;
  const int nz = (K + k_chunk - 1) / k_chunk;
  float* target = nz == 1 ? dc : partial;
  dim3 grid(grid_tiles(M, N, G::BM, G::BN), 1, nz);
  if constexpr (sizeof(T) == 2) {
    if (dkv_lo && gemm_big_ok(M, N, K, k_chunk, (size_t)M * K, (size_t)N * K)) {
      if (dc_bm(N) == 128)
        gemm_big8_kernel<128, 512, false, false, 1, float><<<dim3(grid_tiles(M, N, 128, 512), 1, nz), 512, 0, st>>>(
            dkv, w, dkv_lo, target, M, N, K, K, K, N, k_chunk, (long long)M * N);
      else
        gemm_big8_kernel<256, 256, false, false, 1, float><<<dim3(grid_tiles(M, N, 256, 256), 1, nz), 512, 0, st>>>(
            dkv, w, dkv_lo, target, M, N, K, K, K, N, k_chunk, (long long)M * N);
      grid.x = 0;  // done
    }
  }
  if (grid.x == 0) {
  } else if (dkv_lo)
    gemm_kernel<T, float, false, false, G::BM, G::BN, G::BK, 1><<<grid, kThreads, 0, st>>>(
        dkv, w, dkv_lo, target, M, N, K, K, K, N, k_chunk, (long long)M * N);
  else
    gemm_kernel<T, float, false, false, G::BM, G::BN, G::BK, 0><<<grid, kThreads, 0, st>>>(
        dkv, w, nullptr, target, M, N, K, K, K, N, k_chunk, (long long)M * N);
  if (nz > 1) {
    const long long n4 = (long long)M * N / 4;
    split_reduce_kernel<<<(unsigned)((n4 + 255) / 256), 256, 0, st>>>(partial, dc, n4, nz, (long long)M * N);
  }
  return hipGetLastError();
}

template <typename T>
hipError_t launch_dw(const T* c, const T* dkv, const T* dkv_lo, float* dw, float* partial, int M, int N, int K,
                     hipStream_t st) {
  // dW[M=d_c][N=H*dkvh] = c^T @ (dKV + dKV_lo); c stored [K=tokens][M] and dKV [K][N]: both k-strided.
  using G = GemmCfg<T>;
  const int split = dw_split_tokens(K);
  const int nsplit = (int)dw_split_count(K);
  float* target = nsplit == 1 ? dw : partial;
  dim3 grid(grid_tiles(M, N, G::BM, G::BN), 1, nsplit);
  if constexpr (sizeof(T) == 2) {
    if (dkv_lo && gemm_big_ok(M, N, K, split, (size_t)K * M, (size_t)K * N)) {
      if (M > 256)
        gemm_big8_kernel<512, 128, true, true, 2, float><<<dim3(grid_tiles(M, N, 512, 128), 1, nsplit), 512, 0, st>>>(
            c, dkv, dkv_lo, target, M, N, K, M, N, N, split, (long long)M * N);
      else
        gemm_big8_kernel<256, 256, true, true, 2, float><<<dim3(grid_tiles(M, N, 256, 256), 1, nsplit), 512, 0, st>>>(
            c, dkv, dkv_lo, target, M, N, K, M, N, N, split, (long long)M * N);
      grid.x = 0;  // done
    }
  }
  if (grid.x == 0) {
  } else if (dkv_lo)
    gemm_kernel<T, float, true, true, G::BM, G::BN, G::BK, 2><<<grid, kThreads, 0, st>>>(
        c, dkv, dkv_lo, target, M, N, K, M, N, N, split, (long long)M * N);
  else
    gemm_kernel<T, float, true, true, G::BM, G::BN, G::BK, 0><<<grid, kThreads, 0, st>>>(
        c, dkv, nullptr, target, M, N, K, M, N, N, split, (long long)M * N);
  if (nsplit > 1) {
    const long long n4 = (long long)M * N / 4;
    split_reduce_kernel<<<(unsigned)((n4 + 255) / 256), 256, 0, st>>>(partial, dw, n4, nsplit, (long long)M * N);
  }
  return hipGetLastError();
}

template <typename T>
hipError_t launch_gemm_nt(const T* a, const T* w, T* c, int M, int N, int K, hipStream_t st) {
  // c[M][N] = a[M][K] @ w^T, w stored [N][K] (both k-contiguous); element-dtype output
  using G = GemmCfg<T>;
  if constexpr (sizeof(T) == 2) {
    if (gemm_big_ok(M, N, K, K, (size_t)M * K, (size_t)N * K)) {
      gemm_big8_kernel<256, 256, false, false, 0, bf16><<<grid_tiles(M, N, 256, 256), 512, 0, st>>>(
          a, w, nullptr, c, M, N, K, K, K, N, K, 0);
      return hipGetLastError();
    }
  }
  gemm_kernel<T, T, false, false, G::BM, G::BN, G::BK, 0><<<dim3(grid_tiles(M, N, G::BM, G::BN), 1, 1), kThreads,
                                                              0, st>>>(a, w, nullptr, c, M, N, K, K, K, N, K, 0);
  return hipGetLastError();
}

int gemm_tn_splits(int M, int N, int K, int esize) {
  const bool big = esize == 2 && gemm_big_ok(M, N, K, kGK, (size_t)K * M, (size_t)K * N);
  const int tiles = big ? grid_tiles(M, N, 256, 256) : grid_tiles(M, N, GemmCfg<bf16>::BM, GemmCfg<bf16>::BN);
  const int want = big ? 256 : kMinGemmBlocks;
  int n = (want + tiles - 1) / tiles;
  const int max_split = (K + 511) / 512;
  return n < 1 ? 1 : (n > max_split ? max_split : n);
}

template <typename T>
hipError_t launch_gemm_tn(const T* a, const T* b, float* c, float* partial, int M, int N, int K, int nsplit,
                          hipStream_t st) {
  // c[M][N] = a^T @ b with a stored [K][M] and b [K][N] (both k-strided), fp32 output; the
  // contraction split into nsplit ranges of whole 32-index stages, summed in ascending order
  using G = GemmCfg<T>;
  const int split = ((K + nsplit - 1) / nsplit + 31) / 32 * 32;
  const int nz = (K + split - 1) / split;
  float* target = nz == 1 ? c : partial;
  bool done = false;
  if constexpr (sizeof(T) == 2) {
    if (gemm_big_ok(M, N, K, split, (size_t)K * M, (size_t)K * N)) {
      gemm_big8_kernel<256, 256, true, true, 0, float><<<dim3(grid_tiles(M, N, 256, 256), 1, nz), 512, 0, st>>>(
          a, b, nullptr, target, M, N, K, M, N, N, split, (long long)M * N);
      done = true;
    }
  }
  if (!done)
    gemm_kernel<T, float, true, true, G::BM, G::BN, G::BK, 0><<<dim3(grid_tiles(M, N, G::BM, G::BN), 1, nz),
                                                                kThreads, 0, st>>>(
        a, b, nullptr, target, M, N, K, M, N, N, split, (long long)M * N);
  if (nz > 1) {
    const long long n4 = (long long)M * N / 4;
    split_reduce_kernel<<<(unsigned)((n4 + 255) / 256), 256, 0, st>>>(partial, c, n4, nz, (long long)M * N);
  }
  return hipGetLastError();
}

template hipError_t launch_gemm_nt<bf16>(const bf16*, const bf16*, bf16*, int, int, int, hipStream_t);
template hipError_t launch_gemm_nt<float>(const float*, const float*, float*, int, int, int, hipStream_t);
template hipError_t launch_gemm_tn<bf16>(const bf16*, const bf16*, float*, float*, int, int, int, int, hipStream_t);
template hipError_t launch_gemm_tn<float>(const float*, const float*, float*, float*, int, int, int, int,
                                          hipStream_t);
template hipError_t launch_reconstruct<bf16>(const bf16*, const bf16*, bf16*, int, int, int, hipStream_t);
template hipError_t launch_reconstruct<float>(const float*, const float*, float*, int, int, int, hipStream_t);
template hipError_t launch_dc<bf16>(const bf16*, const bf16*, const bf16*, float*, float*, int, int, int, hipStream_t);
template hipError_t launch_dc<float>(const float*, const float*, const float*, float*, float*, int, int, int,
                                     hipStream_t);
template hipError_t launch_dw<bf16>(const bf16*, const bf16*, const bf16*, float*, float*, int, int, int, hipStream_t);
template hipError_t launch_dw<float>(const float*, const float*, const float*, float*, float*, int, int, int,
                                     hipStream_t);

}  // namespace laga
