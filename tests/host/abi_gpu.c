/* The C ABI driven from a C11 program on the GPU, with device memory from the HIP C
 * API and no Python: ppas_kv_append then ppas_attn_step on a small mixed step (a
 * prefill chunk and two decode rows over a scrambled block table).
 *
 * Closed form: every cached and new value row of KV head g is the same vector v_g,
 * so the softmax-weighted mean of the values is v_g for every row and query head of
 * group g, whatever Q and K hold. The kernels' rounding stays far below half a bf16
 * unit, so each output element must equal v_g's bf16 bits exactly. The page writes
 * are checked address by address against the page-scatter rule: the new positions'
 * slots hold a sentinel before the append, which the attention would otherwise read.
 * The step runs with the default plan and with small key splits (split rows, merged
 * by the second launch). */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "ppas.h"

#define HKV 2
#define HQ 16
#define D 128
#define P 16
#define NSEQ 3
#define STRIDE 19
#define NPAGES 30
#define SENTINEL 0xFFFFu

#define CHECK(c)                                                   \
  do {                                                             \
    if (!(c)) {                                                    \
      printf("FAIL %s:%d %s\n", __FILE__, __LINE__, #c);           \
      return 1;                                                    \
    }                                                              \
  } while (0)
#define HIP(c) CHECK((c) == hipSuccess)

static uint32_t lcg_state = 12345u;
/* k / 64 for k in [-64, 64]: exactly representable in bf16 */
static uint16_t rnd_bf16(void) {
  float f;
  uint32_t u;
  lcg_state = lcg_state * 1664525u + 1013904223u;
  f = (float)((int)((lcg_state >> 8) % 129u) - 64) / 64.f;
  memcpy(&u, &f, 4);
  return (uint16_t)(u >> 16);
}
static uint16_t bf16_of(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return (uint16_t)(u >> 16); /* exact for the values used here */
}
/* v_g[d] = (d mod 32 - 16) / 8 + g: multiples of 1/8, exact in bf16 */
static uint16_t v_of(int g, int d) { return bf16_of((float)(d % 32 - 16) / 8.f + (float)g); }

static size_t k_index(int page, int g, int slot, int d) {
  return ((((size_t)page * HKV + g) * (D / 8) + d / 8) * P + slot) * 8 + d % 8;
}
static size_t v_index(int page, int g, int slot, int d) { return (((size_t)page * HKV + g) * D + d) * P + slot; }

/* With opts == NULL: ppas_attn_step. Otherwise a step plan made with opts, launched
 * twice (the plan serves several calls) and destroyed. */
static int run_step(const ppas_shape* sh, const ppas_seq* seqs, int T, void* out, void* q, void* kp, void* vp,
                    const int32_t* bt_dev, const int32_t* bt_host, uint16_t* host_out, const ppas_plan_opts* opts) {
  size_t ws_bytes = ppas_attn_workspace_bytes(sh, seqs, NSEQ);
  void* ws = NULL;
  int t, h, d, rep;
  ppas_step_plan* plan = NULL;
  ppas_plan_info info;
  if (opts) {
    CHECK(ppas_step_plan_create(sh, seqs, NSEQ, bt_host, STRIDE, opts, &plan) == PPAS_OK && plan != NULL);
    CHECK(ppas_step_plan_info(plan, &info) == PPAS_OK);
    CHECK(info.n_merge > 0);   /* the forced splits give merged rows */
    ws_bytes = (size_t)info.workspace_bytes;
  }
  CHECK(ws_bytes >= 256);
  HIP(hipMalloc(&ws, ws_bytes));
  if (opts) {
    CHECK(ppas_attn_step_planned(plan, out, q, kp, vp, bt_dev, ws, ws_bytes - 1, NULL, NULL) == PPAS_ENOSPACE);
    HIP(hipMemset(out, 0, (size_t)T * HQ * D * 2));
    for (rep = 0; rep < 2; ++rep)
      CHECK(ppas_attn_step_planned(plan, out, q, kp, vp, bt_dev, ws, ws_bytes, NULL, NULL) == PPAS_OK);
    ppas_step_plan_destroy(plan);
  } else {
    CHECK(ppas_attn_step(sh, out, q, kp, vp, seqs, NSEQ, bt_dev, STRIDE, bt_host, ws, ws_bytes - 1, NULL) ==
          PPAS_ENOSPACE);
    HIP(hipMemset(out, 0, (size_t)T * HQ * D * 2));
    CHECK(ppas_attn_step(sh, out, q, kp, vp, seqs, NSEQ, bt_dev, STRIDE, bt_host, ws, ws_bytes, NULL) == PPAS_OK);
  }
  HIP(hipDeviceSynchronize());
  HIP(hipMemcpy(host_out, out, (size_t)T * HQ * D * 2, hipMemcpyDeviceToHost));
  HIP(hipFree(ws));
  for (t = 0; t < T; ++t)
    for (h = 0; h < HQ; ++h)
      for (d = 0; d < D; ++d) CHECK(host_out[((size_t)t * HQ + h) * D + d] == v_of(h / (HQ / HKV), d));
  return 0;
}

int main(void) {
  ppas_shape sh = {HQ, HKV, D, P, NPAGES, 0.08838834764831845f};
  /* (query_start, n_query, cached_len): a decode row, a 37-token chunk, a decode row */
  ppas_seq seqs[NSEQ] = {{0, 1, 40}, {1, 37, 5}, {38, 1, 300}};
  const int T = 39;
  int32_t bt[NSEQ][STRIDE];
  size_t kpool = (size_t)NPAGES * HKV * P * D, nrow = (size_t)T * HKV * D, nq = (size_t)T * HQ * D;
  uint16_t *hk = malloc(kpool * 2), *hv = malloc(kpool * 2), *hq = malloc(nq * 2);
  uint16_t *hkn = malloc(nrow * 2), *hvn = malloc(nrow * 2), *hout = malloc(nq * 2);
  void *kp, *vp, *q, *kn, *vn, *out;
  int32_t* bt_dev;
  int s, i, g, d, j = 0, page, slot, pos;
  size_t e;
  CHECK(hk && hv && hq && hkn && hvn && hout);

  /* scrambled block table: logical page j of the step goes to (7 j + 3) mod 30 */
  for (s = 0; s < NSEQ; ++s)
    for (i = 0; i < STRIDE; ++i)
      bt[s][i] = i * P < seqs[s].cached_len + seqs[s].n_query ? (7 * j++ + 3) % NPAGES : -1;

  for (e = 0; e < kpool; ++e) hk[e] = rnd_bf16();
  for (page = 0; page < NPAGES; ++page)
    for (g = 0; g < HKV; ++g)
      for (d = 0; d < D; ++d)
        for (slot = 0; slot < P; ++slot) hv[v_index(page, g, slot, d)] = v_of(g, d);
  for (s = 0; s < NSEQ; ++s)
    for (i = 0; i < seqs[s].n_query; ++i) {
      pos = seqs[s].cached_len + i;
      for (g = 0; g < HKV; ++g)
        for (d = 0; d < D; ++d) {
          hk[k_index(bt[s][pos / P], g, pos % P, d)] = SENTINEL;
          hv[v_index(bt[s][pos / P], g, pos % P, d)] = SENTINEL;
        }
    }
  for (e = 0; e < nq; ++e) hq[e] = rnd_bf16();
  for (e = 0; e < nrow; ++e) {
    hkn[e] = rnd_bf16();
    hvn[e] = v_of((int)(e / D % HKV), (int)(e % D));
  }

  HIP(hipMalloc(&kp, kpool * 2));
  HIP(hipMalloc(&vp, kpool * 2));
  HIP(hipMalloc(&q, nq * 2));
  HIP(hipMalloc(&kn, nrow * 2));
  HIP(hipMalloc(&vn, nrow * 2));
  HIP(hipMalloc(&out, nq * 2));
  HIP(hipMalloc((void**)&bt_dev, sizeof(bt)));
  HIP(hipMemcpy(kp, hk, kpool * 2, hipMemcpyHostToDevice));
  HIP(hipMemcpy(vp, hv, kpool * 2, hipMemcpyHostToDevice));
  HIP(hipMemcpy(q, hq, nq * 2, hipMemcpyHostToDevice));
  HIP(hipMemcpy(kn, hkn, nrow * 2, hipMemcpyHostToDevice));
  HIP(hipMemcpy(vn, hvn, nrow * 2, hipMemcpyHostToDevice));
  HIP(hipMemcpy(bt_dev, bt, sizeof(bt), hipMemcpyHostToDevice));

  /* refused on the host before any device work */
  CHECK(ppas_kv_append(&sh, kp, vp, NULL, vn, seqs, NSEQ, bt_dev, STRIDE, &bt[0][0], NULL) == PPAS_EINVAL);
  CHECK(ppas_rope_kv_append(&sh, 0.f, q, kp, vp, kn, vn, seqs, NSEQ, bt_dev, STRIDE, &bt[0][0], NULL) ==
        PPAS_EINVAL);

  CHECK(ppas_kv_append(&sh, kp, vp, kn, vn, seqs, NSEQ, bt_dev, STRIDE, &bt[0][0], NULL) == PPAS_OK);
  HIP(hipDeviceSynchronize());
  HIP(hipMemcpy(hk, kp, kpool * 2, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(hv, vp, kpool * 2, hipMemcpyDeviceToHost));
  for (s = 0; s < NSEQ; ++s)
    for (i = 0; i < seqs[s].n_query; ++i) {
      pos = seqs[s].cached_len + i;
      for (g = 0; g < HKV; ++g)
        for (d = 0; d < D; ++d) {
          e = ((size_t)(seqs[s].query_start + i) * HKV + g) * D + d;
          CHECK(hk[k_index(bt[s][pos / P], g, pos % P, d)] == hkn[e]);
          CHECK(hv[v_index(bt[s][pos / P], g, pos % P, d)] == hvn[e]);
        }
    }

  if (run_step(&sh, seqs, T, out, q, kp, vp, bt_dev, &bt[0][0], hout, NULL)) return 1;
  {
    ppas_plan_opts split = {64, 64, 0, 0};
    if (run_step(&sh, seqs, T, out, q, kp, vp, bt_dev, &bt[0][0], hout, &split)) return 1;
  }

  HIP(hipFree(kp));
  HIP(hipFree(vp));
  HIP(hipFree(q));
  HIP(hipFree(kn));
  HIP(hipFree(vn));
  HIP(hipFree(out));
  HIP(hipFree(bt_dev));
  free(hk);
  free(hv);
  free(hq);
  free(hkn);
  free(hvn);
  free(hout);
  printf("ok\n");
  return 0;
}
