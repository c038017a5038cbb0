/* A plain C99 client of the C ABI (include/ripple.h), used by the tests to show
 * that the library needs nothing but the header and the shared library.
 *
 *   ripple_client IN OUT
 *
 * IN (written by the test, little-endian): int64 n, m, L, agg, nbatches; int32
 * dims[L+1], relu[L]; int32 src[m], dst[m]; float x[n][d0]; per layer l = 1..L:
 * int64 has_self, then float w_self[d_l][d_{l-1}] if has_self, w_neigh
 * [d_l][d_{l-1}], bias[d_l]; per batch: int64 num_ops, num_feat_rows, then the
 * ops (16 bytes each) and float feat_rows[num_feat_rows][d0].
 *
 * OUT: per batch and layer l = 0..L, int64 |A^l| and its ids (int32); then
 * H^l of every vertex (float [n][d_l]) for l = 0..L; then the int32 statuses of
 * four calls that must fail (NULL context, an op naming a vertex out of range, a
 * feature row out of range, an unknown kind), the last of which must leave the
 * embeddings as they were.
 *
 * Exit status 0 when every call that must succeed did; the first failure is
 * printed with ripple_last_error. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "ripple.h"

static FILE *in_f, *out_f;

static void die(const char *what, ripple_ctx *ctx, ripple_status st) {
  fprintf(stderr, "ripple_client: %s failed (status %d): %s\n", what, (int)st, ripple_last_error(ctx));
  exit(1);
}

static void *take(size_t bytes) {
  void *p = malloc(bytes ? bytes : 1);
  if (p == NULL || (bytes && fread(p, 1, bytes, in_f) != bytes)) {
    fprintf(stderr, "ripple_client: short input\n");
    exit(2);
  }
  return p;
}

static int64_t take_i64(void) {
  int64_t v;
  if (fread(&v, sizeof v, 1, in_f) != 1) {
    fprintf(stderr, "ripple_client: short input\n");
    exit(2);
  }
  return v;
}

static void put(const void *p, size_t bytes) {
  if (bytes && fwrite(p, 1, bytes, out_f) != bytes) {
    fprintf(stderr, "ripple_client: write failed\n");
    exit(2);
  }
}

int main(int argc, char **argv) {
  if (argc != 3) {
    fprintf(stderr, "usage: ripple_client IN OUT\n");
    return 2;
  }
  in_f = fopen(argv[1], "rb");
  out_f = fopen(argv[2], "wb");
  if (in_f == NULL || out_f == NULL) {
    fprintf(stderr, "ripple_client: cannot open files\n");
    return 2;
  }
  const int64_t n = take_i64(), m = take_i64(), L = take_i64(), agg = take_i64(), nbatches = take_i64();
  if (n < 1 || m < 0 || L < 1 || L > RIPPLE_MAX_LAYERS) {
    fprintf(stderr, "ripple_client: bad header\n");
    return 2;
  }
  int32_t *dims = take(sizeof(int32_t) * (size_t)(L + 1));
  int32_t *relu = take(sizeof(int32_t) * (size_t)L);
  int32_t *src = take(sizeof(int32_t) * (size_t)m);
  int32_t *dst = take(sizeof(int32_t) * (size_t)m);
  float *x = take(sizeof(float) * (size_t)(n * dims[0]));
  const float *w_self[RIPPLE_MAX_LAYERS] = {0}, *w_neigh[RIPPLE_MAX_LAYERS] = {0}, *bias[RIPPLE_MAX_LAYERS] = {0};
  for (int64_t l = 1; l <= L; ++l) {
    const size_t w = sizeof(float) * (size_t)dims[l] * (size_t)dims[l - 1];
    if (take_i64()) w_self[l - 1] = take(w);
    w_neigh[l - 1] = take(w);
    bias[l - 1] = take(sizeof(float) * (size_t)dims[l]);
  }

  ripple_graph_desc g;
  memset(&g, 0, sizeof g);
  g.num_vertices = n;
  g.num_edges = m;
  g.src = src;
  g.dst = dst;
  g.slack = 0.25f;
  g.min_slack = 4;
  ripple_ctx *ctx = NULL;
  ripple_status st = ripple_load_graph(&g, &ctx);
  if (st != RIPPLE_OK) die("ripple_load_graph", NULL, st);

  ripple_model_desc md;
  memset(&md, 0, sizeof md);
  md.num_layers = (int32_t)L;
  md.agg = (int32_t)agg;
  md.dims = dims;
  md.w_self = w_self;
  md.w_neigh = w_neigh;
  md.bias = bias;
  md.relu = relu;
  md.gemm_prec = RIPPLE_GEMM_FP32;
  md.transform_first = -1;
  if ((st = ripple_init_embeddings(ctx, x, &md)) != RIPPLE_OK) die("ripple_init_embeddings", ctx, st);

  int32_t *ids = malloc(sizeof(int32_t) * (size_t)n);
  for (int64_t b = 0; b < nbatches; ++b) {
    const int64_t nops = take_i64(), nfeat = take_i64();
    ripple_op *ops = take(sizeof(ripple_op) * (size_t)nops);
    float *feat = take(sizeof(float) * (size_t)(nfeat * dims[0]));
    ripple_batch_stats stats;
    if ((st = ripple_apply_updates(ctx, ops, nops, nfeat ? feat : NULL, nfeat, &stats)) != RIPPLE_OK)
      die("ripple_apply_updates", ctx, st);
    if (stats.num_ops != nops) {
      fprintf(stderr, "ripple_client: stats.num_ops %lld != %lld\n", (long long)stats.num_ops, (long long)nops);
      return 1;
    }
    for (int32_t l = 0; l <= L; ++l) {
      int64_t count = -1;
      if ((st = ripple_get_affected(ctx, l, ids, n, &count)) != RIPPLE_OK) die("ripple_get_affected", ctx, st);
      put(&count, sizeof count);
      put(ids, sizeof(int32_t) * (size_t)count);
    }
    free(ops);
    free(feat);
  }
  size_t hmax = 0;
  for (int64_t l = 0; l <= L; ++l)
    if ((size_t)dims[l] > hmax) hmax = (size_t)dims[l];
  float *h = malloc(sizeof(float) * (size_t)n * hmax);
  float *h_after = malloc(sizeof(float) * (size_t)n * hmax);
  for (int32_t l = 0; l <= L; ++l) {
    if ((st = ripple_get_embeddings(ctx, l, NULL, n, h)) != RIPPLE_OK) die("ripple_get_embeddings", ctx, st);
    put(h, sizeof(float) * (size_t)n * (size_t)dims[l]);
  }

  /* calls that must fail, leaving the state as it was */
  int32_t bad[4];
  ripple_op op;
  bad[0] = (int32_t)ripple_apply_updates(NULL, NULL, 0, NULL, 0, NULL);
  op.kind = RIPPLE_OP_INSERT;
  op.u = 0;
  op.v = (int32_t)n; /* out of range */
  op.feat_row = -1;
  bad[1] = (int32_t)ripple_apply_updates(ctx, &op, 1, NULL, 0, NULL);
  op.kind = RIPPLE_OP_FEATURE;
  op.v = -1;
  op.feat_row = 3; /* no feature block */
  bad[2] = (int32_t)ripple_apply_updates(ctx, &op, 1, NULL, 0, NULL);
  op.kind = 9; /* unknown */
  bad[3] = (int32_t)ripple_apply_updates(ctx, &op, 1, NULL, 0, NULL);
  if ((st = ripple_get_embeddings(ctx, (int32_t)L, NULL, n, h_after)) != RIPPLE_OK)
    die("ripple_get_embeddings", ctx, st);
  if (memcmp(h, h_after, sizeof(float) * (size_t)n * (size_t)dims[L]) != 0) {
    /* h holds H^L from the loop above */
    fprintf(stderr, "ripple_client: a rejected batch changed H^L\n");
    return 1;
  }
  put(bad, sizeof bad);
  ripple_destroy(ctx);
  fclose(out_f);
  fclose(in_f);
  printf("ripple_client: ok\n");
  return 0;
}
