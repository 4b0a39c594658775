// C ABI of the per-rank LAGA attention block: validation, workspace layout and
// dispatch to the gfx950 kernels. Declarations and conventions: include/laga.h.
#include <math.h>
#include <stdint.h>

#include <mutex>

#include "laga.h"
#include "kernels.hpp"
#include "bwd_common.hpp"

using namespace laga;

namespace {

constexpr int64_t kMaxElems = (int64_t)1 << 31;  // 32-bit element offsets inside kernels

struct Dims {
  int B, S, H, d_c, dn, dr, dv;
  int dqk() const { return dn + dr; }
  int dkvh() const { return dn + dv; }
};

bool is_v3(const laga_problem_t* p) { return p->d_nope == 128 && p->d_rope == 64 && p->d_v == 128; }
bool is_small(const laga_problem_t* p) { return p->d_nope == 32 && p->d_rope == 16 && p->d_v == 32; }
bool is_half(const laga_problem_t* p) { return p->d_nope == 64 && p->d_rope == 32 && p->d_v == 64; }

laga_status_t validate(const laga_problem_t* p, Dims* d) {
  if (!p) return LAGA_ERR_NULL;
  if (p->batch <= 0 || p->seq_len <= 0 || p->n_heads <= 0 || p->d_c <= 0 || p->d_nope <= 0 ||
      p->d_rope <= 0 || p->d_v <= 0)
    return LAGA_ERR_SHAPE;
  if (!isfinite(p->softmax_scale) || !(p->softmax_scale > 0.f)) return LAGA_ERR_SHAPE;
  if ((p->causal != 0 && p->causal != 1) || (p->deterministic != 0 && p->deterministic != 1) ||
      (p->dq_mode != LAGA_DQ_FROM_STORE && p->dq_mode != LAGA_DQ_RECOMPUTE))
    return LAGA_ERR_UNSUPPORTED;
  if (p->dtype != LAGA_DTYPE_BF16 && p->dtype != LAGA_DTYPE_FP32) return LAGA_ERR_UNSUPPORTED;
  if (p->kv_mode != LAGA_KV_MATERIALIZED && p->kv_mode != LAGA_KV_FUSED) return LAGA_ERR_UNSUPPORTED;
  if (!is_v3(p) && !is_small(p) && !is_half(p)) return LAGA_ERR_UNSUPPORTED;
  if (p->d_c % 32 != 0 || p->d_c > 1024) return LAGA_ERR_UNSUPPORTED;
  // each factor below 2^31 before any product is formed, so no product overflows int64
  if (p->batch >= kMaxElems || p->seq_len >= kMaxElems || p->n_heads >= kMaxElems) return LAGA_ERR_UNSUPPORTED;
  const int64_t tok = p->batch * p->seq_len;
  const int64_t wide = p->n_heads * (p->d_nope + (p->d_rope > p->d_v ? p->d_rope : p->d_v) +
                                     (p->d_nope > p->d_v ? p->d_nope : p->d_v));
  if (tok >= kMaxElems || wide >= kMaxElems || tok * wide >= kMaxElems || tok * p->d_c >= kMaxElems ||
      p->d_c * p->n_heads * (p->d_nope + p->d_v) * 16 >= kMaxElems)
    return LAGA_ERR_UNSUPPORTED;
  d->B = (int)p->batch; d->S = (int)p->seq_len; d->H = (int)p->n_heads; d->d_c = (int)p->d_c;
  d->dn = (int)p->d_nope; d->dr = (int)p->d_rope; d->dv = (int)p->d_v;
  return LAGA_OK;
}

bool misaligned(const void* ptr) { return ((uintptr_t)ptr & 15u) != 0; }

size_t elem_size(const laga_problem_t* p) { return p->dtype == LAGA_DTYPE_BF16 ? 2 : 4; }

size_t round_up(size_t x) { return (x + 255) & ~(size_t)255; }

// Backward workspace: [delta | lse2 | dKV | dKV low halves (bf16) | dK_pe per head | GEMM split partials |
// fused mode: W_kv_b^T (K/V rebuilt on chip) or the kv rebuild | dS^T store (bf16 with 192/128-wide heads)]
struct BwdWs {
  size_t delta, lse2, dkv, dkv_lo, dkpe_h, dw_part, kv, w_t, ds, total;
};
bool stores_ds(const laga_problem_t* p) {
  return p->dtype == LAGA_DTYPE_BF16 && is_v3(p) && p->dq_mode == LAGA_DQ_FROM_STORE;
}
// Fused mode without kv: the key-stationary and dQ kernels rebuild K/V tiles on chip from
// c_kv and W_kv_b^T (bf16 with 192/128-wide heads, dq from the store, d_c a multiple of
// 128 up to kFusedMaxDc); other problems rebuild kv once into the workspace and run the
// materialised kernels.
bool kv_on_chip(const laga_problem_t* p) {
  return p->kv_mode == LAGA_KV_FUSED && stores_ds(p) && p->d_c <= kFusedMaxDc && p->d_c % 128 == 0;
}
int s_pad(int S) { return (S + kRowPad - 1) / kRowPad * kRowPad; }
BwdWs bwd_layout(const laga_problem_t* p, const Dims& d) {
  BwdWs w{};
  const size_t tok = (size_t)d.B * d.S;
  size_t off = 0;
  w.delta = off; off += round_up(sizeof(float) * d.B * d.H * s_pad(d.S));
  w.lse2 = off; off += round_up(sizeof(float) * d.B * d.H * s_pad(d.S));
  w.dkv = off; off += round_up(elem_size(p) * tok * d.H * d.dkvh());
  w.dkv_lo = off; off += p->dtype == LAGA_DTYPE_BF16 ? round_up(elem_size(p) * tok * d.H * d.dkvh()) : 0;
  w.dkpe_h = off; off += round_up(sizeof(float) * tok * d.H * d.dr);
  const size_t np = gemm_partial_elems((int)tok, d.d_c, d.H * d.dkvh());
  w.dw_part = off; off += np > 0 ? round_up(sizeof(float) * np) : 0;
  const bool fused = p->kv_mode == LAGA_KV_FUSED;
  w.kv = off; off += fused && !kv_on_chip(p) ? round_up(elem_size(p) * tok * d.H * d.dkvh()) : 0;
  w.w_t = off; off += kv_on_chip(p) ? round_up(elem_size(p) * (size_t)d.d_c * d.H * d.dkvh()) : 0;
  w.ds = off;
  off += stores_ds(p) ? round_up(sizeof(uint16_t) * (size_t)d.B * d.H * bwd::ds_head_elems((d.S + 31) / 32, p->causal)) : 0;
  w.total = off;
  return w;
}

// Forward workspace: the fused mode keeps W_kv_b^T (H*(d_nope+d_v) x d_c) there.
size_t fwd_ws_bytes(const laga_problem_t* p, const Dims& d) {
  if (p->kv_mode != LAGA_KV_FUSED) return 0;
  return round_up(elem_size(p) * (size_t)d.d_c * d.H * d.dkvh());
}

laga_status_t from_hip(hipError_t e) { return e == hipSuccess ? LAGA_OK : LAGA_ERR_DEVICE; }

// Producers: d_gamma partial rows of the backward.
size_t prologue_ws_bytes(const Dims& d) {
  const long long tok = (long long)d.B * d.S;
  return round_up(sizeof(float) * (size_t)(prologue_bwd_rows(tok) + prologue_sum_groups(tok)) * d.d_c);
}

laga_status_t validate_prologue(const laga_problem_t* p, const laga_prologue_t* cfg, Dims* d) {
  if (!cfg) return LAGA_ERR_NULL;
  laga_status_t s = validate(p, d);
  if (s != LAGA_OK) return s;
  if (!isfinite(cfg->eps) || cfg->eps < 0.f || !isfinite(cfg->rope_base) || !(cfg->rope_base > 1.f) ||
      cfg->position_offset < 0 || cfg->position_offset > ((int64_t)1 << 53) - 1 - d->S)
    return LAGA_ERR_SHAPE;
  // the rotation kernels give each lane one 8-element chunk of a band: d_rope / 8 must divide 64
  if (d->dr % 8 != 0 || 64 % (d->dr / 8) != 0) return LAGA_ERR_UNSUPPORTED;
  return LAGA_OK;
}

PrologueArgs prologue_args(const laga_problem_t* p, const laga_prologue_t* cfg, const Dims& d) {
  PrologueArgs a{};
  a.B = d.B; a.S = d.S; a.H = d.H; a.d_c = d.d_c; a.d_nope = d.dn; a.d_rope = d.dr; a.d_qk = d.dqk();
  a.position_offset = cfg->position_offset;
  a.eps = cfg->eps;
  a.log2_base = log2((double)cfg->rope_base);
  (void)p;
  return a;
}

// Output projection (Alg. 1 step 7): sizes, validation, workspace.
struct OutDims {
  int T, F, D;
};
laga_status_t validate_out_proj(const laga_out_proj_t* p, OutDims* d) {
  if (!p) return LAGA_ERR_NULL;
  if (p->tokens <= 0 || p->n_heads <= 0 || p->d_v <= 0 || p->d_model <= 0) return LAGA_ERR_SHAPE;
  if (p->reserved != 0 || (p->dtype != LAGA_DTYPE_BF16 && p->dtype != LAGA_DTYPE_FP32)) return LAGA_ERR_UNSUPPORTED;
  // each factor below 2^31 before any product is formed, so no product overflows int64
  if (p->tokens >= kMaxElems || p->n_heads >= kMaxElems || p->d_v >= kMaxElems || p->d_model >= kMaxElems)
    return LAGA_ERR_UNSUPPORTED;
  const int64_t F = p->n_heads * p->d_v;
  if (F % 16 != 0 || p->d_model % 16 != 0) return LAGA_ERR_UNSUPPORTED;
  if (F >= kMaxElems || p->tokens * F >= kMaxElems || p->tokens * p->d_model >= kMaxElems ||
      F * p->d_model >= kMaxElems)
    return LAGA_ERR_UNSUPPORTED;
  d->T = (int)p->tokens; d->F = (int)F; d->D = (int)p->d_model;
  return LAGA_OK;
}
int out_proj_splits(const laga_out_proj_t* p, const OutDims& d) {
  return gemm_tn_splits(d.F, d.D, d.T, p->dtype == LAGA_DTYPE_BF16 ? 2 : 4);
}
size_t out_proj_ws_bytes(const laga_out_proj_t* p, const OutDims& d) {
  const int n = out_proj_splits(p, d);
  return n > 1 ? round_up(sizeof(float) * (size_t)n * d.F * d.D) : 0;
}

template <typename T>
laga_status_t reconstruct_t(const Dims& d, const void* c, const void* w, void* kv, hipStream_t st) {
  return from_hip(launch_reconstruct<T>((const T*)c, (const T*)w, (T*)kv, d.B * d.S, d.H * d.dkvh(), d.d_c, st));
}

}  // namespace

// Device memory of laga_attn_bwd_noalloc: the backward's workspace for callers that
// cannot allocate. Each GPU the library runs on holds its own copy until the process
// ends. Host code never uses this name as an address (on the host it is only a handle
// for hipGetSymbolAddress); kernels get the per-device address found below.
static __device__ __align__(256) unsigned char scratch[LAGA_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices];  // device address of `scratch` on each device, once known

// Address of `scratch` on the current device (looked up once per device, with that device
// current). The stream must belong to the current device.
laga_status_t scratch_address(hipStream_t st, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return LAGA_ERR_DEVICE;
  if (st) {
    hipDevice_t sd = -1;
    if (hipStreamGetDevice(st, &sd) != hipSuccess || sd != dev) return LAGA_ERR_DEVICE;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return LAGA_ERR_DEVICE;
    g_scratch_dev[dev] = ptr;
  }
  *out = g_scratch_dev[dev];
  return LAGA_OK;
}

}  // namespace

extern "C" {

int laga_abi_version(void) { return LAGA_ABI_VERSION; }

const char* laga_status_string(laga_status_t s) {
  switch (s) {
    case LAGA_OK: return "LAGA_OK: success";
    case LAGA_ERR_NULL: return "LAGA_ERR_NULL: a required pointer is NULL";
    case LAGA_ERR_SHAPE: return "LAGA_ERR_SHAPE: a dimension is not positive or the scale is not finite and positive";
    case LAGA_ERR_UNSUPPORTED: return "LAGA_ERR_UNSUPPORTED: head dims, d_c, dtype, mode or size not supported by this library";
    case LAGA_ERR_ALIGN: return "LAGA_ERR_ALIGN: a pointer is not 16-byte aligned";
    case LAGA_ERR_WORKSPACE: return "LAGA_ERR_WORKSPACE: workspace smaller than laga_workspace_bytes()";
    case LAGA_ERR_DEVICE: return "LAGA_ERR_DEVICE: the HIP runtime reported a launch error";
    case LAGA_ERR_SCRATCH:
      return "LAGA_ERR_SCRATCH: the problem needs more workspace than the no-alloc entry point's fixed "
             "device array holds (LAGA_NOALLOC_SCRATCH_BYTES)";
  }
  return "unknown laga_status_t";
}

size_t laga_workspace_bytes(const laga_problem_t* p, int op) {
  Dims d;
  if (validate(p, &d) != LAGA_OK) return 0;
  if (op == LAGA_OP_FWD) return fwd_ws_bytes(p, d);
  if (op == LAGA_OP_BWD) return bwd_layout(p, d).total;
  if (op == LAGA_OP_PROLOGUE_BWD) return prologue_ws_bytes(d);
  return 0;
}

laga_status_t laga_prologue_fwd(const laga_problem_t* p, const laga_prologue_t* cfg, const void* latent_raw,
                                const void* gamma, const void* kpe_raw, void* q, void* c_kv, void* k_pe,
                                float* rstd, void* stream) {
  Dims d;
  laga_status_t s = validate_prologue(p, cfg, &d);
  if (s != LAGA_OK) return s;
  if (!latent_raw || !kpe_raw || !c_kv || !k_pe || !rstd) return LAGA_ERR_NULL;
  if (misaligned(latent_raw) || misaligned(kpe_raw) || misaligned(c_kv) || misaligned(k_pe) ||
      misaligned(rstd) || (gamma && misaligned(gamma)) || (q && misaligned(q)))
    return LAGA_ERR_ALIGN;
  PrologueArgs a = prologue_args(p, cfg, d);
  a.latent_raw = latent_raw; a.gamma = gamma; a.kpe_raw = kpe_raw; a.q = q; a.c_kv = c_kv; a.k_pe = k_pe;
  a.rstd = rstd;
  hipStream_t st = (hipStream_t)stream;
  return from_hip(p->dtype == LAGA_DTYPE_BF16 ? launch_prologue_fwd<bf16>(a, st) : launch_prologue_fwd<float>(a, st));
}

laga_status_t laga_prologue_bwd(const laga_problem_t* p, const laga_prologue_t* cfg, const void* latent_raw,
                                const void* gamma, const float* rstd, const float* dc_kv, const float* dk_pe,
                                void* dq, float* d_latent_raw, float* d_kpe_raw, float* d_gamma, void* workspace,
                                size_t workspace_bytes, void* stream) {
  Dims d;
  laga_status_t s = validate_prologue(p, cfg, &d);
  if (s != LAGA_OK) return s;
  if (!latent_raw || !rstd || !dc_kv || !dk_pe || !d_latent_raw || !d_kpe_raw || (gamma && !d_gamma))
    return LAGA_ERR_NULL;
  if (misaligned(latent_raw) || misaligned(rstd) || misaligned(dc_kv) || misaligned(dk_pe) ||
      misaligned(d_latent_raw) || misaligned(d_kpe_raw) || (gamma && misaligned(gamma)) ||
      (gamma && misaligned(d_gamma)) || (dq && misaligned(dq)))
    return LAGA_ERR_ALIGN;
  if (gamma) {
    if (!workspace || workspace_bytes < prologue_ws_bytes(d)) return LAGA_ERR_WORKSPACE;
    if (misaligned(workspace)) return LAGA_ERR_ALIGN;
  }
  PrologueArgs a = prologue_args(p, cfg, d);
  a.latent_raw = latent_raw; a.gamma = gamma; a.rstd_in = rstd; a.dc_kv = dc_kv; a.dk_pe = dk_pe; a.q = dq;
  a.d_latent = d_latent_raw; a.d_kpe = d_kpe_raw;
  a.d_gamma = gamma ? d_gamma : nullptr;
  a.partial = gamma ? (float*)workspace : nullptr;
  hipStream_t st = (hipStream_t)stream;
  return from_hip(p->dtype == LAGA_DTYPE_BF16 ? launch_prologue_bwd<bf16>(a, st) : launch_prologue_bwd<float>(a, st));
}

size_t laga_out_proj_workspace_bytes(const laga_out_proj_t* p) {
  OutDims d;
  if (validate_out_proj(p, &d) != LAGA_OK) return 0;
  return out_proj_ws_bytes(p, d);
}

laga_status_t laga_out_proj_fwd(const laga_out_proj_t* p, const void* out, const void* w_o, void* y, void* stream) {
  OutDims d;
  laga_status_t s = validate_out_proj(p, &d);
  if (s != LAGA_OK) return s;
  if (!out || !w_o || !y) return LAGA_ERR_NULL;
  if (misaligned(out) || misaligned(w_o) || misaligned(y)) return LAGA_ERR_ALIGN;
  hipStream_t st = (hipStream_t)stream;
  // y[T][D] = out[T][F] @ w_o[F][D]: the up-projection's GEMM (w_o k-strided)
  return from_hip(p->dtype == LAGA_DTYPE_BF16
                      ? launch_reconstruct<bf16>((const bf16*)out, (const bf16*)w_o, (bf16*)y, d.T, d.D, d.F, st)
                      : launch_reconstruct<float>((const float*)out, (const float*)w_o, (float*)y, d.T, d.D, d.F, st));
}

laga_status_t laga_out_proj_bwd(const laga_out_proj_t* p, const void* out, const void* w_o, const void* dy,
                                void* d_out, float* dw_o, void* workspace, size_t workspace_bytes, void* stream) {
  OutDims d;
  laga_status_t s = validate_out_proj(p, &d);
  if (s != LAGA_OK) return s;
  if (!out || !w_o || !dy || !d_out || !dw_o) return LAGA_ERR_NULL;
  if (misaligned(out) || misaligned(w_o) || misaligned(dy) || misaligned(d_out) || misaligned(dw_o))
    return LAGA_ERR_ALIGN;
  const size_t need = out_proj_ws_bytes(p, d);
  if (need > 0 && (!workspace || workspace_bytes < need)) return LAGA_ERR_WORKSPACE;
  if (need > 0 && misaligned(workspace)) return LAGA_ERR_ALIGN;
  hipStream_t st = (hipStream_t)stream;
  const int ns = out_proj_splits(p, d);
  hipError_t e;
  if (p->dtype == LAGA_DTYPE_BF16) {
    // d_out[T][F] = dy[T][D] @ w_o^T (w_o stored [F][D]: k-contiguous); dw_o[F][D] = out^T @ dy
    e = launch_gemm_nt<bf16>((const bf16*)dy, (const bf16*)w_o, (bf16*)d_out, d.T, d.F, d.D, st);
    if (e == hipSuccess)
      e = launch_gemm_tn<bf16>((const bf16*)out, (const bf16*)dy, dw_o, (float*)workspace, d.F, d.D, d.T, ns, st);
  } else {
    e = launch_gemm_nt<float>((const float*)dy, (const float*)w_o, (float*)d_out, d.T, d.F, d.D, st);
    if (e == hipSuccess)
      e = launch_gemm_tn<float>((const float*)out, (const float*)dy, dw_o, (float*)workspace, d.F, d.D, d.T, ns, st);
  }
  return from_hip(e);
}

laga_status_t laga_reconstruct_kv(const laga_problem_t* p, const void* c_kv, const void* w_kv_b, void* kv,
                                  void* stream) {
  Dims d;
  laga_status_t s = validate(p, &d);
  if (s != LAGA_OK) return s;
  if (!c_kv || !w_kv_b || !kv) return LAGA_ERR_NULL;
  if (misaligned(c_kv) || misaligned(w_kv_b) || misaligned(kv)) return LAGA_ERR_ALIGN;
  hipStream_t st = (hipStream_t)stream;
  return p->dtype == LAGA_DTYPE_BF16 ? reconstruct_t<bf16>(d, c_kv, w_kv_b, kv, st)
                                     : reconstruct_t<float>(d, c_kv, w_kv_b, kv, st);
}

laga_status_t laga_attn_fwd(const laga_problem_t* p, const void* q, const void* c_kv, const void* k_pe,
                            const void* w_kv_b, const void* kv, void* out, float* lse, void* workspace,
                            size_t workspace_bytes, void* stream) {
  Dims d;
  laga_status_t s = validate(p, &d);
  if (s != LAGA_OK) return s;
  const bool fused = p->kv_mode == LAGA_KV_FUSED;
  if (!q || !c_kv || !k_pe || !w_kv_b || !out || !lse || (!fused && !kv)) return LAGA_ERR_NULL;
  if (misaligned(q) || misaligned(c_kv) || misaligned(k_pe) || misaligned(w_kv_b) || misaligned(out) ||
      misaligned(lse) || (!fused && misaligned(kv)))
    return LAGA_ERR_ALIGN;
  const size_t need = fwd_ws_bytes(p, d);
  if (need > 0 && (!workspace || workspace_bytes < need)) return LAGA_ERR_WORKSPACE;
  if (need > 0 && misaligned(workspace)) return LAGA_ERR_ALIGN;
  if (fused && d.d_c > kFusedMaxDc) return LAGA_ERR_UNSUPPORTED;
  AttnFwdArgs a{};
  a.q = q; a.k_pe = k_pe; a.kv = kv; a.c_kv = c_kv; a.w = w_kv_b; a.out = out; a.lse = lse;
  a.B = d.B; a.S = d.S; a.H = d.H; a.d_c = d.d_c; a.scale = p->softmax_scale; a.causal = p->causal;
  hipStream_t st = (hipStream_t)stream;
  const bool bf = p->dtype == LAGA_DTYPE_BF16;
  if (fused) {
    if (is_v3(p))
      return from_hip(bf ? launch_attn_fwd_fused<bf16, 128, 64, 128>(a, workspace, st)
                         : launch_attn_fwd_fused<float, 128, 64, 128>(a, workspace, st));
    if (is_half(p))
      return from_hip(bf ? launch_attn_fwd_fused<bf16, 64, 32, 64>(a, workspace, st)
                         : launch_attn_fwd_fused<float, 64, 32, 64>(a, workspace, st));
    return from_hip(bf ? launch_attn_fwd_fused<bf16, 32, 16, 32>(a, workspace, st)
                       : launch_attn_fwd_fused<float, 32, 16, 32>(a, workspace, st));
  }
  if (is_v3(p)) return from_hip(bf ? launch_attn_fwd<bf16, 128, 64, 128>(a, st) : launch_attn_fwd<float, 128, 64, 128>(a, st));
  if (is_half(p)) return from_hip(bf ? launch_attn_fwd<bf16, 64, 32, 64>(a, st) : launch_attn_fwd<float, 64, 32, 64>(a, st));
  return from_hip(bf ? launch_attn_fwd<bf16, 32, 16, 32>(a, st) : launch_attn_fwd<float, 32, 16, 32>(a, st));
}

laga_status_t laga_attn_bwd_stage(int stage, const laga_problem_t* p, const void* q, const void* c_kv,
                                  const void* k_pe, const void* w_kv_b, const void* kv, const void* out,
                                  const float* lse, const void* dout, void* dq, float* dc_kv, float* dk_pe,
                                  float* dw_kv_b, void* workspace, size_t workspace_bytes, void* stream) {
  Dims d;
  laga_status_t s = validate(p, &d);
  if (s != LAGA_OK) return s;
  if (stage < LAGA_BWD_PREPARE || stage > LAGA_BWD_FINISH) return LAGA_ERR_UNSUPPORTED;
  const bool fused = p->kv_mode == LAGA_KV_FUSED;
  if (!q || !c_kv || !k_pe || !w_kv_b || !out || !lse || !dout || !dq || !dc_kv || !dk_pe || !dw_kv_b ||
      (!fused && !kv))
    return LAGA_ERR_NULL;
  const void* ptrs[] = {q, c_kv, k_pe, w_kv_b, out, lse, dout, dq, dc_kv, dk_pe, dw_kv_b};
  for (const void* x : ptrs)
    if (misaligned(x)) return LAGA_ERR_ALIGN;
  if (kv && misaligned(kv)) return LAGA_ERR_ALIGN;
  const BwdWs ws = bwd_layout(p, d);
  if (!workspace || workspace_bytes < ws.total) return LAGA_ERR_WORKSPACE;
  if (misaligned(workspace)) return LAGA_ERR_ALIGN;
  char* wsb = (char*)workspace;
  hipStream_t st = (hipStream_t)stream;
  const bool bf = p->dtype == LAGA_DTYPE_BF16;
  const bool v3 = is_v3(p);

  const bool on_chip = fused && !kv && kv_on_chip(p);
  if (on_chip) {
    // the kernels rebuild K/V tiles from c_kv and W_kv_b^T, written in fragment order in the
    // first stage
    if (stage == LAGA_BWD_PREPARE) {
      hipError_t e = launch_frag_w_pi<bf16>((const bf16*)w_kv_b, (bf16*)(wsb + ws.w_t), d.d_c, d.H * d.dkvh(), st);
      if (e != hipSuccess) return LAGA_ERR_DEVICE;
    }
  } else if (fused && !kv) {
    // K/V are rebuilt (same GEMM as laga_reconstruct_kv) into the workspace in the first stage.
    void* kvw = wsb + ws.kv;
    if (stage == LAGA_BWD_PREPARE) {
      s = bf ? reconstruct_t<bf16>(d, c_kv, w_kv_b, kvw, st) : reconstruct_t<float>(d, c_kv, w_kv_b, kvw, st);
      if (s != LAGA_OK) return s;
    }
    kv = kvw;
  }
  AttnBwdArgs a{};
  a.c_kv = c_kv; a.d_c = d.d_c;
  a.w_t = on_chip ? wsb + ws.w_t : nullptr;
  a.q = q; a.k_pe = k_pe; a.kv = kv; a.out = out; a.dout = dout; a.lse = lse; a.dq = dq;
  a.delta = (float*)(wsb + ws.delta); a.dkv = wsb + ws.dkv; a.dkpe_h = (float*)(wsb + ws.dkpe_h);
  a.lse2 = (float*)(wsb + ws.lse2); a.S_pad = s_pad(d.S);
  a.dkv_lo = bf ? wsb + ws.dkv_lo : nullptr;
  a.dk_pe = dk_pe;
  a.ds = stores_ds(p) ? wsb + ws.ds : nullptr;
  a.B = d.B; a.S = d.S; a.H = d.H; a.scale = p->softmax_scale; a.causal = p->causal;
  hipError_t e;
  const int kstage = stage == LAGA_BWD_PREPARE ? 0 : stage == LAGA_BWD_DKDV ? 1 : stage == LAGA_BWD_DQ ? 2 : 3;
  if (v3) e = bf ? launch_attn_bwd<bf16, 128, 64, 128>(a, kstage, st) : launch_attn_bwd<float, 128, 64, 128>(a, kstage, st);
  else if (is_half(p))
    e = bf ? launch_attn_bwd<bf16, 64, 32, 64>(a, kstage, st) : launch_attn_bwd<float, 64, 32, 64>(a, kstage, st);
  else e = bf ? launch_attn_bwd<bf16, 32, 16, 32>(a, kstage, st) : launch_attn_bwd<float, 32, 16, 32>(a, kstage, st);
  if (e != hipSuccess || stage != LAGA_BWD_FINISH) return from_hip(e);

  const int tok = d.B * d.S, ncol = d.H * d.dkvh();
  float* part = (float*)(wsb + ws.dw_part);
  if (bf) {
    const bf16* hi = (const bf16*)a.dkv;
    const bf16* lo = (const bf16*)a.dkv_lo;
    e = launch_dc<bf16>(hi, lo, (const bf16*)w_kv_b, dc_kv, part, tok, d.d_c, ncol, st);
    if (e == hipSuccess) e = launch_dw<bf16>((const bf16*)c_kv, hi, lo, dw_kv_b, part, d.d_c, ncol, tok, st);
  } else {
    const float* g = (const float*)a.dkv;
    e = launch_dc<float>(g, nullptr, (const float*)w_kv_b, dc_kv, part, tok, d.d_c, ncol, st);
    if (e == hipSuccess) e = launch_dw<float>((const float*)c_kv, g, nullptr, dw_kv_b, part, d.d_c, ncol, tok, st);
  }
  return from_hip(e);
}

laga_status_t laga_attn_bwd(const laga_problem_t* p, const void* q, const void* c_kv, const void* k_pe,
                            const void* w_kv_b, const void* kv, const void* out, const float* lse,
                            const void* dout, void* dq, float* dc_kv, float* dk_pe, float* dw_kv_b,
                            void* workspace, size_t workspace_bytes, void* stream) {
  for (int stage = LAGA_BWD_PREPARE; stage <= LAGA_BWD_FINISH; ++stage) {
    laga_status_t s = laga_attn_bwd_stage(stage, p, q, c_kv, k_pe, w_kv_b, kv, out, lse, dout, dq, dc_kv, dk_pe,
                                          dw_kv_b, workspace, workspace_bytes, stream);
    if (s != LAGA_OK) return s;
  }
  return LAGA_OK;
}

laga_status_t laga_attn_bwd_noalloc(const laga_problem_t* p, const void* q, const void* c_kv, const void* k_pe,
                                    const void* w_kv_b, const void* kv, const void* out, const float* lse,
                                    const void* dout, void* dq, float* dc_kv, float* dk_pe, float* dw_kv_b,
                                    void* stream) {
  Dims d;
  laga_status_t s = validate(p, &d);
  if (s != LAGA_OK) return s;
  if (bwd_layout(p, d).total > (size_t)LAGA_NOALLOC_SCRATCH_BYTES) return LAGA_ERR_SCRATCH;
  void* ws = nullptr;
  s = scratch_address((hipStream_t)stream, &ws);
  if (s != LAGA_OK) return s;
  // nothing in the workspace needs to start at zero: every stage writes what a later one reads
  return laga_attn_bwd(p, q, c_kv, k_pe, w_kv_b, kv, out, lse, dout, dq, dc_kv, dk_pe, dw_kv_b, ws,
                       (size_t)LAGA_NOALLOC_SCRATCH_BYTES, stream);
}

}  // extern "C"
