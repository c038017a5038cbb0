/* Drives the host-side paths of the C ABI that run without a GPU, for a build of
 * libripple whose host code is compiled with AddressSanitizer: argument checks,
 * snapshot validation, the threaded per-row sort of a large snapshot (weighted and
 * unweighted, directed and undirected), the error path taken when no device can
 * be selected, and ripple_destroy of every partly built context. Prints one line
 * per case; exits 0 when every call returned what it must. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "ripple.h"

static int failures = 0;

static void expect(const char *what, ripple_status got, ripple_status want) {
  printf("%-48s status %d (want %d)\n", what, (int)got, (int)want);
  if (got != want) ++failures;
}

static ripple_status load(int64_t n, int64_t m, const int32_t *src, const int32_t *dst, int undirected,
                          const float *weight, ripple_ctx **ctx) {
  ripple_graph_desc g;
  memset(&g, 0, sizeof(g));
  g.num_vertices = n;
  g.num_edges = m;
  g.src = src;
  g.dst = dst;
  g.undirected = undirected;
  g.slack = 0.25f;
  g.min_slack = 4;
  g.weight = weight;
  return ripple_load_graph(&g, ctx);
}

int main(void) {
  ripple_ctx *ctx = (ripple_ctx *)0x1;
  int32_t s2[2] = {0, 1}, d2[2] = {1, 2};
  expect("NULL out pointer", ripple_load_graph(NULL, NULL), RIPPLE_E_INVALID);
  expect("NULL descriptor", ripple_load_graph(NULL, &ctx), RIPPLE_E_INVALID);
  expect("no vertices", load(0, 0, NULL, NULL, 0, NULL, &ctx), RIPPLE_E_INVALID);
  expect("edges without arrays", load(4, 2, NULL, NULL, 0, NULL, &ctx), RIPPLE_E_INVALID);
  int32_t bad_d[2] = {1, 9};
  expect("id out of range", load(4, 2, s2, bad_d, 0, NULL, &ctx), RIPPLE_E_INVALID);
  int32_t loop_d[2] = {1, 1};
  expect("self-loop", load(4, 2, s2, loop_d, 0, NULL, &ctx), RIPPLE_E_INVALID);
  int32_t rep_s[2] = {0, 0}, rep_d[2] = {1, 1};
  expect("repeated arc", load(4, 2, rep_s, rep_d, 0, NULL, &ctx), RIPPLE_E_INVALID);
  int32_t und_s[2] = {0, 1}, und_d[2] = {1, 0};
  expect("undirected pair listed twice", load(4, 2, und_s, und_d, 1, NULL, &ctx), RIPPLE_E_INVALID);
  float nan_w[2] = {1.0f, 0.0f};
  nan_w[1] = nan_w[1] / nan_w[1];
  expect("weight not finite", load(4, 2, s2, d2, 0, nan_w, &ctx), RIPPLE_E_INVALID);
  if (ctx != NULL) ++failures;  /* every failed load leaves *out NULL */
  printf("last load error: %s\n", ripple_last_error(NULL));

  /* a snapshot of 200,000 vertices and 1.6M arcs passes validation and is sorted by
   * the host threads; with no GPU the device cannot be selected, so the context
   * ends in RIPPLE_E_DEVICE and is destroyed on the way out */
  const int64_t n = 200000, m = 1600000;
  int32_t *src = malloc(sizeof(int32_t) * m), *dst = malloc(sizeof(int32_t) * m);
  float *w = malloc(sizeof(float) * m);
  for (int64_t i = 0; i < m; ++i) {  /* distinct arcs: vertex u -> u+1 .. u+8 */
    src[i] = (int32_t)(i / 8);
    dst[i] = (int32_t)((i / 8 + 1 + i % 8) % n);
    w[i] = 0.5f + (float)(i % 7) / 8.0f;
  }
  const ripple_status st = load(n, m, src, dst, 0, NULL, &ctx);
  printf("%-48s status %d (%s)\n", "large directed snapshot, no device", (int)st, ripple_last_error(NULL));
  if (st != RIPPLE_E_DEVICE && st != RIPPLE_OK) ++failures;
  if (st == RIPPLE_OK) ripple_destroy(ctx);
  const ripple_status sw = load(n, m, src, dst, 0, w, &ctx);
  printf("%-48s status %d\n", "large weighted snapshot, no device", (int)sw);
  if (sw != RIPPLE_E_DEVICE && sw != RIPPLE_OK) ++failures;
  if (sw == RIPPLE_OK) ripple_destroy(ctx);
  /* undirected: keep u < v so that no edge is listed twice */
  int64_t mu = 0;
  for (int64_t i = 0; i < m; ++i)
    if (src[i] < dst[i]) {
      src[mu] = src[i];
      dst[mu] = dst[i];
      ++mu;
    }
  const ripple_status su = load(n, mu, src, dst, 1, NULL, &ctx);
  printf("%-48s status %d\n", "large undirected snapshot, no device", (int)su);
  if (su != RIPPLE_E_DEVICE && su != RIPPLE_OK) ++failures;
  if (su == RIPPLE_OK) ripple_destroy(ctx);
  free(src);
  free(dst);
  free(w);

  expect("apply on NULL context", ripple_apply_updates(NULL, NULL, 0, NULL, 0, NULL), RIPPLE_E_INVALID);
  expect("static read on NULL context", ripple_get_embeddings_static(NULL, 0, NULL, 0, NULL), RIPPLE_E_INVALID);
  int64_t bytes = 0;
  expect("device bytes of NULL context", ripple_device_bytes(NULL, &bytes), RIPPLE_E_INVALID);
  ripple_destroy(NULL);
  printf("%s\n", failures == 0 ? "asan host ok" : "asan host FAILED");
  return failures == 0 ? 0 : 1;
}
