/*
 * A plain C consumer of the library's C ABI (include/laga.h): no PyTorch, no C++.
 * It reads a problem's inputs from fp32 files, runs Alg. 1 steps 4-5 and their
 * backward through laga_reconstruct_kv, laga_attn_fwd and laga_attn_bwd on one HIP
 * stream with device buffers it allocates itself, and writes every output back as
 * fp32 files. The test that drives it compares those files with the CPU oracle.
 *
 * usage: laga_c_demo DIR B S H d_c d_nope d_rope d_v causal
 *   DIR holds c_kv.f32 k_pe.f32 q.f32 w_kv_b.f32 dout.f32 (row-major, the layouts of
 *   laga.h); the program writes kv.f32 out.f32 lse.f32 dq.f32 dc_kv.f32 dk_pe.f32
 *   dw_kv_b.f32 there. The problem runs in the fp32 element type. Exit code 0 on
 *   success, 1 on a library or runtime error (the message names the call).
 */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "laga.h"

static char g_dir[4096];

static int fail_hip(const char* what, hipError_t e) {
  fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
  return 1;
}

static int fail_laga(const char* what, laga_status_t s) {
  fprintf(stderr, "%s: %s\n", what, laga_status_string(s));
  return 1;
}

/* device buffer of n floats, filled from DIR/name if `load` */
static int dev_buffer(const char* name, size_t n, int load, float** dptr) {
  hipError_t e = hipMalloc((void**)dptr, n * sizeof(float) + 16);
  if (e != hipSuccess) return fail_hip("hipMalloc", e);
  if (!load) return 0;
  char path[4200];
  snprintf(path, sizeof path, "%s/%s.f32", g_dir, name);
  FILE* f = fopen(path, "rb");
  if (!f) { fprintf(stderr, "cannot open %s\n", path); return 1; }
  float* h = (float*)malloc(n * sizeof(float));
  size_t got = h ? fread(h, sizeof(float), n, f) : 0;
  fclose(f);
  if (got != n) { fprintf(stderr, "%s: expected %zu floats, read %zu\n", path, n, got); free(h); return 1; }
  e = hipMemcpy(*dptr, h, n * sizeof(float), hipMemcpyHostToDevice);
  free(h);
  return e == hipSuccess ? 0 : fail_hip("hipMemcpy to device", e);
}

static int save(const char* name, const float* d, size_t n) {
  float* h = (float*)malloc(n * sizeof(float));
  if (!h) return 1;
  hipError_t e = hipMemcpy(h, d, n * sizeof(float), hipMemcpyDeviceToHost);
  if (e != hipSuccess) { free(h); return fail_hip("hipMemcpy to host", e); }
  char path[4200];
  snprintf(path, sizeof path, "%s/%s.f32", g_dir, name);
  FILE* f = fopen(path, "wb");
  size_t put = f ? fwrite(h, sizeof(float), n, f) : 0;
  if (f) fclose(f);
  free(h);
  if (put != n) { fprintf(stderr, "cannot write %s\n", path); return 1; }
  return 0;
}

int main(int argc, char** argv) {
  if (argc != 10) {
    fprintf(stderr, "usage: %s DIR B S H d_c d_nope d_rope d_v causal\n", argv[0]);
    return 2;
  }
  snprintf(g_dir, sizeof g_dir, "%s", argv[1]);
  laga_problem_t p;
  memset(&p, 0, sizeof p);
  p.batch = atoll(argv[2]); p.seq_len = atoll(argv[3]); p.n_heads = atoll(argv[4]);
  p.d_c = atoll(argv[5]); p.d_nope = atoll(argv[6]); p.d_rope = atoll(argv[7]); p.d_v = atoll(argv[8]);
  p.causal = atoi(argv[9]);
  p.softmax_scale = 1.0f / sqrtf((float)(p.d_nope + p.d_rope));
  p.dtype = LAGA_DTYPE_FP32;
  p.kv_mode = LAGA_KV_MATERIALIZED;
  p.deterministic = 1;
  if (laga_abi_version() != LAGA_ABI_VERSION) {
    fprintf(stderr, "library ABI %d, header %d\n", laga_abi_version(), LAGA_ABI_VERSION);
    return 1;
  }

  const size_t B = p.batch, S = p.seq_len, H = p.n_heads, dqk = p.d_nope + p.d_rope, dkvh = p.d_nope + p.d_v;
  const size_t n_c = B * S * p.d_c, n_pe = B * S * p.d_rope, n_q = B * S * H * dqk, n_w = p.d_c * H * dkvh;
  const size_t n_kv = B * S * H * dkvh, n_out = B * S * H * p.d_v, n_lse = B * H * S;
  float *c, *pe, *q, *w, *dout, *kv, *out, *lse, *dq, *dc, *dpe, *dw;
  if (dev_buffer("c_kv", n_c, 1, &c) || dev_buffer("k_pe", n_pe, 1, &pe) || dev_buffer("q", n_q, 1, &q) ||
      dev_buffer("w_kv_b", n_w, 1, &w) || dev_buffer("dout", n_out, 1, &dout) || dev_buffer("kv", n_kv, 0, &kv) ||
      dev_buffer("out", n_out, 0, &out) || dev_buffer("lse", n_lse, 0, &lse) || dev_buffer("dq", n_q, 0, &dq) ||
      dev_buffer("dc_kv", n_c, 0, &dc) || dev_buffer("dk_pe", n_pe, 0, &dpe) || dev_buffer("dw_kv_b", n_w, 0, &dw))
    return 1;

  const size_t ws_f = laga_workspace_bytes(&p, LAGA_OP_FWD), ws_b = laga_workspace_bytes(&p, LAGA_OP_BWD);
  void* ws = NULL;
  const size_t ws_n = ws_f > ws_b ? ws_f : ws_b;
  hipError_t e = hipMalloc(&ws, ws_n > 0 ? ws_n : 16);
  if (e != hipSuccess) return fail_hip("hipMalloc workspace", e);
  hipStream_t st;
  e = hipStreamCreate(&st);
  if (e != hipSuccess) return fail_hip("hipStreamCreate", e);

  laga_status_t s = laga_reconstruct_kv(&p, c, w, kv, st);
  if (s != LAGA_OK) return fail_laga("laga_reconstruct_kv", s);
  s = laga_attn_fwd(&p, q, c, pe, w, kv, out, lse, ws, ws_n, st);
  if (s != LAGA_OK) return fail_laga("laga_attn_fwd", s);
  s = laga_attn_bwd(&p, q, c, pe, w, kv, out, lse, dout, dq, dc, dpe, dw, ws, ws_n, st);
  if (s != LAGA_OK) return fail_laga("laga_attn_bwd", s);
  e = hipStreamSynchronize(st);
  if (e != hipSuccess) return fail_hip("hipStreamSynchronize", e);

  if (save("kv", kv, n_kv) || save("out", out, n_out) || save("lse", lse, n_lse) || save("dq", dq, n_q) ||
      save("dc_kv", dc, n_c) || save("dk_pe", dpe, n_pe) || save("dw_kv_b", dw, n_w))
    return 1;
  float* bufs[] = {c, pe, q, w, dout, kv, out, lse, dq, dc, dpe, dw};
  for (size_t i = 0; i < sizeof bufs / sizeof bufs[0]; ++i) hipFree(bufs[i]);
  hipFree(ws);
  hipStreamDestroy(st);
  printf("laga_c_demo: B=%zu S=%zu H=%zu done\n", B, S, H);
  return 0;
}
