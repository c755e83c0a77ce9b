/* A forward of the attention share driven from C, with plain hipMalloc buffers and no
 * PyTorch: Q = 0 makes the softmax uniform over the visible keys, so O_i is the mean of
 * V_0..V_i and LSE_i = ln(i + 1) (one causal document of 300 tokens, 2 heads), computed
 * here in double precision.  Exit status 0 when both are within the parity tolerances. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <hip/hip_runtime_api.h>
#include "hydra_attn.h"

static uint16_t bf16(float x) { uint32_t u; memcpy(&u, &x, 4); u += 0x7fff + ((u >> 16) & 1); return (uint16_t)(u >> 16); }
static float f32(uint16_t b) { uint32_t u = (uint32_t)b << 16; float x; memcpy(&x, &u, 4); return x; }

int main(void) {
  const int H = 2, N = 300;
  int32_t cu[2] = {0, N};
  hydra_problem_t p;
  memset(&p, 0, sizeof p);
  p.n_heads = H; p.d_qk = 192; p.d_v = 128; p.cu_seqlens = cu; p.n_docs = 1;
  p.q.n_segs = 1; p.q.len[0] = N; p.kv.n_segs = 1; p.kv.len[0] = N;
  size_t nq = (size_t)N * H * 192, nv = (size_t)N * H * 128;
  uint16_t *hq = calloc(nq, 2), *hk = malloc(nq * 2), *hv = malloc(nv * 2);
  srand(1);
  for (size_t i = 0; i < nq; ++i) hk[i] = bf16((float)rand() / RAND_MAX - 0.5f);
  for (size_t i = 0; i < nv; ++i) hv[i] = bf16((float)rand() / RAND_MAX - 0.5f);
  void *q, *k, *v, *o, *lse, *ws;
  size_t wsb = hydra_workspace_size(&p);
  if (hipMalloc(&q, nq * 2) || hipMalloc(&k, nq * 2) || hipMalloc(&v, nv * 2) || hipMalloc(&o, nv * 4) ||
      hipMalloc(&lse, (size_t)N * H * 4) || hipMalloc(&ws, wsb)) { printf("alloc failed\n"); return 1; }
  hipMemcpy(q, hq, nq * 2, hipMemcpyHostToDevice);
  hipMemcpy(k, hk, nq * 2, hipMemcpyHostToDevice);
  hipMemcpy(v, hv, nv * 2, hipMemcpyHostToDevice);
  int rc = hydra_attn_fwd(&p, q, k, v, (float*)o, (float*)lse, NULL, ws, wsb, NULL);
  if (rc != HYDRA_OK) { printf("fwd %s\n", hydra_strerror(rc)); return 1; }
  if (hipDeviceSynchronize() != hipSuccess) { printf("sync failed\n"); return 1; }
  float *ho = malloc(nv * 4), *hl = malloc((size_t)N * H * 4);
  hipMemcpy(ho, o, nv * 4, hipMemcpyDeviceToHost);
  hipMemcpy(hl, lse, (size_t)N * H * 4, hipMemcpyDeviceToHost);
  /* Q = 0: uniform softmax over the visible keys, O_i = mean_{j<=i} V_j, LSE_i = ln(i+1) */
  double max_o = 0, max_l = 0;
  for (int h = 0; h < H; ++h)
    for (int d = 0; d < 128; ++d) {
      double run = 0;
      for (int i = 0; i < N; ++i) {
        run += f32(hv[((size_t)i * H + h) * 128 + d]);
        double e = fabs(ho[((size_t)i * H + h) * 128 + d] - run / (i + 1));
        if (e > max_o) max_o = e;
      }
    }
  for (int h = 0; h < H; ++h)
    for (int i = 0; i < N; ++i) {
      double e = fabs(hl[(size_t)h * N + i] - log((double)(i + 1)));
      if (e > max_l) max_l = e;
    }
  printf("max_o %.3e max_lse %.3e\n", max_o, max_l);
  return (max_o <= 1e-2 && max_l <= 1e-3) ? 0 : 2;
}
