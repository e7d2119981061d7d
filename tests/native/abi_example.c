/*
 * The C ABI used from plain C: device buffers from the HIP runtime, no
 * Python and no torch.  One tree-verification step on a small batch,
 * checked against closed forms:
 *   - with every key zero the softmax is uniform, so a node's output is the
 *     mean of the values it may see (cache rows below kv_len, its ancestors
 *     and itself; Sec. 2.2);
 *   - with every draft token equal to the target's prediction at its parent,
 *     the acceptance ends at the deepest node (lowest index among equals),
 *     root first (Sec. 2.4).
 * Exit status 0 on success.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "treeverify.h"

#define B 2
#define N 37
#define HQ 8
#define HKV 2
#define D 128
#define LMAX 300
#define V 1000
#define DMAX 40

static uint16_t to_bf16(float f) {  /* round to nearest even */
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFF + ((u >> 16) & 1);
  return (uint16_t)(u >> 16);
}
static float from_bf16(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}
static float frand(unsigned* s) {  /* uniform in [-1, 1) */
  *s = *s * 1664525u + 1013904223u;
  return (float)((*s >> 8) & 0xFFFF) / 32768.0f - 1.0f;
}
#define CHECK(x)                                                            \
  do {                                                                      \
    if ((x) != hipSuccess) {                                                \
      fprintf(stderr, "HIP error at line %d\n", __LINE__);                 \
      return 2;                                                             \
    }                                                                       \
  } while (0)

int main(void) {
  static uint16_t q[B * N * HQ * D], kc[B * LMAX * HKV * D], vc[B * LMAX * HKV * D];
  static uint16_t kt[B * N * HKV * D], vt[B * N * HKV * D], out[B * N * HQ * D];
  static int32_t parent[B * N], kvl[B] = {LMAX, 45}, draft[B * N];
  static float logits[B * N * V];
  unsigned seed = 12345u;
  for (size_t i = 0; i < sizeof(q) / 2; ++i) q[i] = to_bf16(frand(&seed));
  for (size_t i = 0; i < sizeof(vc) / 2; ++i) vc[i] = to_bf16(frand(&seed));
  for (size_t i = 0; i < sizeof(vt) / 2; ++i) vt[i] = to_bf16(frand(&seed));
  memset(kc, 0, sizeof(kc));
  memset(kt, 0, sizeof(kt));
  for (int b = 0; b < B; ++b)
    for (int i = 0; i < N; ++i) {
      seed = seed * 1664525u + 1013904223u;
      parent[b * N + i] = i == 0 ? -1 : (int)((seed >> 8) % (unsigned)i);
    }
  /* target prediction at node i is token (7 i + b) % V; every draft matches */
  for (int b = 0; b < B; ++b)
    for (int i = 0; i < N; ++i) {
      for (int v = 0; v < V; ++v) logits[(b * N + i) * V + v] = 0.f;
      logits[(b * N + i) * V + (7 * i + b) % V] = 1.f;
      draft[b * N + i] = i == 0 ? 0 : (7 * parent[b * N + i] + b) % V;
    }

  void *dq, *dkc, *dvc, *dkt, *dvt, *dout, *dpar, *dkvl, *dlog, *ddraft, *dlen, *dpath, *dws, *dws2;
  CHECK(hipMalloc(&dq, sizeof(q)));
  CHECK(hipMalloc(&dkc, sizeof(kc)));
  CHECK(hipMalloc(&dvc, sizeof(vc)));
  CHECK(hipMalloc(&dkt, sizeof(kt)));
  CHECK(hipMalloc(&dvt, sizeof(vt)));
  CHECK(hipMalloc(&dout, sizeof(out)));
  CHECK(hipMalloc(&dpar, sizeof(parent)));
  CHECK(hipMalloc(&dkvl, sizeof(kvl)));
  CHECK(hipMalloc(&dlog, sizeof(logits)));
  CHECK(hipMalloc(&ddraft, sizeof(draft)));
  CHECK(hipMalloc(&dlen, B * 4));
  CHECK(hipMalloc(&dpath, B * DMAX * 4));
  const size_t wsa = tv_tree_verify_attention_workspace(B, N, HQ, HKV, D, LMAX);
  const size_t wsb = tv_tree_accept_workspace(B, N, V);
  if (wsa == 0 || wsb == 0) {
    fprintf(stderr, "workspace query failed\n");
    return 1;
  }
  CHECK(hipMalloc(&dws, wsa));
  CHECK(hipMalloc(&dws2, wsb));
  CHECK(hipMemset(dws, 0, wsa));  /* workspaces are zero-filled once before first use */
  CHECK(hipMemset(dws2, 0, wsb));
  CHECK(hipMemcpy(dq, q, sizeof(q), hipMemcpyHostToDevice));
  CHECK(hipMemcpy(dkc, kc, sizeof(kc), hipMemcpyHostToDevice));
  CHECK(hipMemcpy(dvc, vc, sizeof(vc), hipMemcpyHostToDevice));
  CHECK(hipMemcpy(dkt, kt, sizeof(kt), hipMemcpyHostToDevice));
  CHECK(hipMemcpy(dvt, vt, sizeof(vt), hipMemcpyHostToDevice));
  CHECK(hipMemcpy(dpar, parent, sizeof(parent), hipMemcpyHostToDevice));
  CHECK(hipMemcpy(dkvl, kvl, sizeof(kvl), hipMemcpyHostToDevice));
  CHECK(hipMemcpy(dlog, logits, sizeof(logits), hipMemcpyHostToDevice));
  CHECK(hipMemcpy(ddraft, draft, sizeof(draft), hipMemcpyHostToDevice));

  int rc = tv_tree_verify_attention(dq, dkc, dvc, dkt, dvt, (const int32_t*)dpar,
                                    (const int32_t*)dkvl, dout, B, N, HQ, HKV, D, LMAX, 0.f, dws,
                                    wsa, NULL);
  if (rc != TV_OK) {
    fprintf(stderr, "attention: %s\n", tv_status_string(rc));
    return 1;
  }
  int32_t len[B], path[B * DMAX];
  rc = tv_tree_accept(dlog, TV_F32, (const int32_t*)ddraft, (const int32_t*)dpar, B, N, V, DMAX,
                      (int32_t*)dlen, (int32_t*)dpath, NULL, dws2, wsb, NULL);
  if (rc != TV_OK) {
    fprintf(stderr, "accept: %s\n", tv_status_string(rc));
    return 1;
  }
  CHECK(hipDeviceSynchronize());
  CHECK(hipMemcpy(out, dout, sizeof(out), hipMemcpyDeviceToHost));
  CHECK(hipMemcpy(len, dlen, sizeof(len), hipMemcpyDeviceToHost));
  CHECK(hipMemcpy(path, dpath, sizeof(path), hipMemcpyDeviceToHost));

  double worst = 0.0;
  int bad_path = 0;
  for (int b = 0; b < B; ++b) {
    int depth[N];
    depth[0] = 0;
    for (int i = 1; i < N; ++i) depth[i] = depth[parent[b * N + i]] + 1;
    for (int i = 0; i < N; ++i)
      for (int h = 0; h < HQ; ++h) {
        const int g = h / (HQ / HKV);
        for (int d = 0; d < D; ++d) {
          double sum = 0.0;
          int cnt = 0;
          for (int t = 0; t < kvl[b]; ++t, ++cnt)
            sum += from_bf16(vc[((b * LMAX + t) * HKV + g) * D + d]);
          for (int u = i; u != -1; u = parent[b * N + u], ++cnt)
            sum += from_bf16(vt[((b * N + u) * HKV + g) * D + d]);
          const double err =
              fabs(from_bf16(out[((b * N + i) * HQ + h) * D + d]) - sum / cnt);
          if (err > worst) worst = err;
        }
      }
    int best = 0;
    for (int i = 1; i < N; ++i)
      if (depth[i] > depth[best]) best = i;
    if (len[b] != depth[best] + 1) bad_path = 1;
    for (int k = depth[best], u = best; k >= 0; --k, u = parent[b * N + u])
      if (k < DMAX && path[b * DMAX + k] != u) bad_path = 1;
  }
  printf("abi_example: attention max abs err %.3e, accept_len {%d, %d}\n", worst, len[0], len[1]);
  if (worst > 1e-2 || bad_path) {
    fprintf(stderr, "abi_example: FAILED\n");
    return 1;
  }
  printf("abi_example: OK\n");
  return 0;
}
