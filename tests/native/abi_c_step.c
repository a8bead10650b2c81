/* One denoising step driven from plain C99 through the C ABI and the HIP
   runtime's C API (no Python, no torch), on inputs whose results have closed
   forms: hidden row r is one-hot at column r % 16 (value 1) and vocabulary
   row v of W_head is one-hot at column v % 16 (value 2), so the logits of
   position r are 2 for the k entries v = r % 16 (mod 16) and 0 elsewhere:
   candidate r % 16 (the lowest of the tied maxima), confidence
   1 / (k + (V - k) e^-2), entropy -sum q log q.  Every position is masked
   and no confidence exceeds 0.9, so each sequence falls back to its
   leftmost masked position (Algorithm 2). */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "fork_step.h"

#define B 2
#define L 8
#define D 16
#define V 40
#define BL 4

static uint16_t bf16(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  return (uint16_t)(u >> 16); /* exact for 0, 1 and 2 */
}

#define CHECK_HIP(x)                                                  \
  do {                                                                \
    if ((x) != hipSuccess) {                                          \
      fprintf(stderr, "HIP call failed at line %d\n", __LINE__);     \
      return 10;                                                      \
    }                                                                 \
  } while (0)

int main(void) {
  static uint16_t h[B * L * D], w[V * D];
  int32_t tokens[B * L], bstart[B], fallback[B];
  uint8_t mask[B * L];
  float conf[B * L], ent[B * L], logp[B * L];
  int r, v, b;
  for (r = 0; r < B * L; ++r) h[r * D + r % D] = bf16(1.0f);
  for (v = 0; v < V; ++v) w[v * D + v % D] = bf16(2.0f);
  for (r = 0; r < B * L; ++r) {
    tokens[r] = -1;
    mask[r] = 1;
  }
  for (b = 0; b < B; ++b) bstart[b] = 0;

  void *dh, *dw, *dt, *dm, *db, *dc, *de, *dl, *df;
  CHECK_HIP(hipMalloc(&dh, sizeof h));
  CHECK_HIP(hipMalloc(&dw, sizeof w));
  CHECK_HIP(hipMalloc(&dt, sizeof tokens));
  CHECK_HIP(hipMalloc(&dm, sizeof mask));
  CHECK_HIP(hipMalloc(&db, sizeof bstart));
  CHECK_HIP(hipMalloc(&dc, sizeof conf));
  CHECK_HIP(hipMalloc(&de, sizeof ent));
  CHECK_HIP(hipMalloc(&dl, sizeof logp));
  CHECK_HIP(hipMalloc(&df, sizeof fallback));
  CHECK_HIP(hipMemcpy(dh, h, sizeof h, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(dw, w, sizeof w, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(dt, tokens, sizeof tokens, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(dm, mask, sizeof mask, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(db, bstart, sizeof bstart, hipMemcpyHostToDevice));

  int rc = fork_step(dh, dw, (int32_t*)dt, (uint8_t*)dm, (int32_t*)db, BL, 0.9f, (float*)dc,
                     (float*)de, (float*)dl, (int32_t*)df, B, L, D, V, FORK_BF16, NULL);
  if (rc != FORK_OK) {
    fprintf(stderr, "fork_step: %d %s\n", rc, fork_last_error());
    return 1;
  }
  CHECK_HIP(hipDeviceSynchronize());
  CHECK_HIP(hipMemcpy(tokens, dt, sizeof tokens, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(mask, dm, sizeof mask, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(bstart, db, sizeof bstart, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(conf, dc, sizeof conf, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(ent, de, sizeof ent, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(logp, dl, sizeof logp, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(fallback, df, sizeof fallback, hipMemcpyDeviceToHost));

  int bad = 0;
  for (r = 0; r < B * L; ++r) {
    const int k = (V - r % D + D - 1) / D; /* entries v < V with v = r (mod 16) */
    const double s = k + (V - k) * exp(-2.0);
    const double q1 = 1.0 / s, q0 = exp(-2.0) / s;
    const double H = -(k * q1 * log(q1) + (V - k) * q0 * log(q0));
    if (fabs(conf[r] - q1) > 1e-5 || fabs(ent[r] - H) > 1e-4 || fabs(logp[r] - log(q1)) > 1e-4) {
      fprintf(stderr, "row %d: conf %g (%g) entropy %g (%g) logp %g (%g)\n", r, conf[r], q1,
              ent[r], H, logp[r], log(q1));
      ++bad;
    }
  }
  for (b = 0; b < B; ++b) {
    const int first = b * L; /* leftmost masked position of the block */
    if (fallback[b] != FORK_STEP_FALLBACK || bstart[b] != 0 || mask[first] != 0 ||
        tokens[first] != first % D) {
      fprintf(stderr, "sequence %d: fallback %d block_start %d token %d\n", b, fallback[b],
              bstart[b], tokens[first]);
      ++bad;
    }
    for (r = first + 1; r < first + L; ++r)
      if (mask[r] != 1 || tokens[r] != -1) ++bad;
  }
  hipFree(dh);
  hipFree(dw);
  hipFree(dt);
  hipFree(dm);
  hipFree(db);
  hipFree(dc);
  hipFree(de);
  hipFree(dl);
  hipFree(df);
  fork_release();
  if (bad) return 2;
  printf("c step ok\n");
  return 0;
}
