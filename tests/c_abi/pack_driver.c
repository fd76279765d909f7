/* Drives libflowpool through its C ABI alone (no Python, no torch): reads a
 * workload from a file, writes every sample into a pool, plans microbatches
 * with plan_microbatches, packs each with pack_microbatch (odd-numbered
 * microbatches with pack_microbatch_noalloc) and writes the
 * results to a file, which the test compares with the oracle.
 *
 * Input (little-endian; i32 unless noted):
 *   hidden, page_tokens, vocab, n_samples, capacity, n_mb, cost_k
 *   table: vocab * hidden u16
 *   per sample: n_text, n_img, text_ids[n_text], img_pos[n_img],
 *               img_ntok[n_img], image rows: sum(img_ntok) * hidden u16
 * Output:
 *   n_mb, assign[n_samples]
 *   per microbatch: n_tokens, max_seqlen, k, cu_seqlens[k + 1],
 *                   position_ids[n_tokens], rows: n_tokens * hidden u16
 * Exit status 0 on success; 1 with a message on stderr otherwise. */

#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "flowpool.h"

static void die(const char* what) {
  fprintf(stderr, "pack_driver: %s failed: %s\n", what, fp_last_error());
  exit(1);
}

static void hip_ok(hipError_t e, const char* what) {
  if (e != hipSuccess) {
    fprintf(stderr, "pack_driver: %s failed: %s\n", what, hipGetErrorString(e));
    exit(1);
  }
}

static void* xmalloc(size_t n) {
  void* p = malloc(n ? n : 1);
  if (!p) {
    fprintf(stderr, "pack_driver: out of host memory\n");
    exit(1);
  }
  return p;
}

static void rd(void* dst, size_t size, size_t count, FILE* f) {
  if (count && fread(dst, size, count, f) != count) {
    fprintf(stderr, "pack_driver: short input\n");
    exit(1);
  }
}

static void wr(const void* src, size_t size, size_t count, FILE* f) {
  if (count && fwrite(src, size, count, f) != count) {
    fprintf(stderr, "pack_driver: short write\n");
    exit(1);
  }
}

int main(int argc, char** argv) {
  if (argc != 3) {
    fprintf(stderr, "usage: pack_driver INPUT OUTPUT\n");
    return 1;
  }
  FILE* in = fopen(argv[1], "rb");
  if (!in) {
    fprintf(stderr, "pack_driver: cannot open %s\n", argv[1]);
    return 1;
  }
  int32_t hdr[7];
  rd(hdr, 4, 7, in);
  const int32_t hidden = hdr[0], page_tokens = hdr[1], vocab = hdr[2], n = hdr[3];
  const int32_t capacity = hdr[4], n_mb = hdr[5], cost_k = hdr[6];
  if (hidden <= 0 || page_tokens <= 0 || vocab <= 0 || n <= 0 || n_mb <= 0) {
    fprintf(stderr, "pack_driver: bad header\n");
    return 1;
  }
  const size_t row = 2 * (size_t)hidden;
  uint16_t* table = (uint16_t*)xmalloc(row * (size_t)vocab);
  rd(table, row, (size_t)vocab, in);

  int32_t* n_text = (int32_t*)xmalloc(4 * (size_t)n);
  int32_t* n_img = (int32_t*)xmalloc(4 * (size_t)n);
  int32_t** text = (int32_t**)xmalloc(sizeof(void*) * (size_t)n);
  int32_t** pos = (int32_t**)xmalloc(sizeof(void*) * (size_t)n);
  int32_t** ntok = (int32_t**)xmalloc(sizeof(void*) * (size_t)n);
  uint16_t** vis = (uint16_t**)xmalloc(sizeof(void*) * (size_t)n);
  int64_t* n_vis = (int64_t*)xmalloc(8 * (size_t)n);
  int64_t pages = 0;
  for (int32_t i = 0; i < n; ++i) {
    int32_t c[2];
    rd(c, 4, 2, in);
    n_text[i] = c[0];
    n_img[i] = c[1];
    text[i] = (int32_t*)xmalloc(4 * (size_t)c[0]);
    pos[i] = (int32_t*)xmalloc(4 * (size_t)c[1]);
    ntok[i] = (int32_t*)xmalloc(4 * (size_t)c[1]);
    rd(text[i], 4, (size_t)c[0], in);
    rd(pos[i], 4, (size_t)c[1], in);
    rd(ntok[i], 4, (size_t)c[1], in);
    n_vis[i] = 0;
    for (int32_t j = 0; j < c[1]; ++j) n_vis[i] += ntok[i][j];
    vis[i] = (uint16_t*)xmalloc(row * (size_t)n_vis[i]);
    rd(vis[i], row, (size_t)n_vis[i], in);
    pages += (n_vis[i] + page_tokens - 1) / page_tokens;
  }
  fclose(in);

  fp_pool_config cfg;
  fp_config_init(&cfg);
  cfg.hidden = hidden;
  cfg.page_tokens = page_tokens;
  cfg.hbm_pages = pages + 8;
  cfg.vocab = vocab;
  fp_pool* pool = NULL;
  if (pool_create(&cfg, &pool) != FP_OK) die("pool_create");

  void* d_table = NULL;
  hip_ok(hipMalloc(&d_table, row * (size_t)vocab), "hipMalloc(table)");
  hip_ok(hipMemcpy(d_table, table, row * (size_t)vocab, hipMemcpyHostToDevice), "hipMemcpy(table)");

  uint64_t* ids = (uint64_t*)xmalloc(8 * (size_t)n);
  for (int32_t i = 0; i < n; ++i) {
    void* d_vis = NULL;
    if (n_vis[i]) {
      hip_ok(hipMalloc(&d_vis, row * (size_t)n_vis[i]), "hipMalloc(image rows)");
      hip_ok(hipMemcpy(d_vis, vis[i], row * (size_t)n_vis[i], hipMemcpyHostToDevice), "hipMemcpy(image rows)");
    }
    if (pool_write_sample(pool, text[i], n_text[i], pos[i], ntok[i], n_img[i], d_vis, NULL, NULL, &ids[i]) != FP_OK)
      die("pool_write_sample");
    hip_ok(hipDeviceSynchronize(), "hipDeviceSynchronize");
    if (d_vis) hip_ok(hipFree(d_vis), "hipFree(image rows)");
  }

  int32_t* assign = (int32_t*)xmalloc(4 * (size_t)n);
  int32_t* mb_tokens = (int32_t*)xmalloc(4 * (size_t)n_mb);
  int32_t* mb_max = (int32_t*)xmalloc(4 * (size_t)n_mb);
  int64_t* mb_cost = (int64_t*)xmalloc(8 * (size_t)n_mb);
  if (plan_microbatches(pool, ids, n, capacity, n_mb, cost_k, FP_PLAN_LPT, assign, mb_tokens, mb_cost, mb_max, NULL,
                        NULL) != FP_OK)
    die("plan_microbatches");

  FILE* out = fopen(argv[2], "wb");
  if (!out) {
    fprintf(stderr, "pack_driver: cannot create %s\n", argv[2]);
    return 1;
  }
  wr(&n_mb, 4, 1, out);
  wr(assign, 4, (size_t)n, out);
  uint64_t* members = (uint64_t*)xmalloc(8 * (size_t)n);
  for (int32_t j = 0; j < n_mb; ++j) {
    int32_t k = 0;
    for (int32_t i = 0; i < n; ++i)
      if (assign[i] == j) members[k++] = ids[i];
    const int64_t cap = mb_tokens[j] > 0 ? mb_tokens[j] : 1;
    void *d_out = NULL, *d_cu = NULL, *d_pos = NULL;
    hip_ok(hipMalloc(&d_out, row * (size_t)cap), "hipMalloc(out)");
    hip_ok(hipMalloc(&d_cu, 4 * ((size_t)k + 1)), "hipMalloc(cu)");
    hip_ok(hipMalloc(&d_pos, 4 * (size_t)cap), "hipMalloc(pos)");
    int32_t n_tok = 0, mx = 0;
    /* odd microbatches through the entry point that allocates nothing */
    fp_status st = (j & 1) ? pack_microbatch_noalloc(pool, members, k, d_table, vocab, d_out, cap, (int32_t*)d_cu,
                                                     (int32_t*)d_pos, &n_tok, &mx, FP_TIER_MASK_ALL, NULL)
                           : pack_microbatch(pool, members, k, d_table, vocab, d_out, cap, (int32_t*)d_cu,
                                             (int32_t*)d_pos, &n_tok, &mx, FP_TIER_MASK_ALL, NULL);
    if (st != FP_OK) die((j & 1) ? "pack_microbatch_noalloc" : "pack_microbatch");
    hip_ok(hipDeviceSynchronize(), "hipDeviceSynchronize");
    int32_t* cu = (int32_t*)xmalloc(4 * ((size_t)k + 1));
    int32_t* p = (int32_t*)xmalloc(4 * (size_t)cap);
    uint16_t* rows = (uint16_t*)xmalloc(row * (size_t)cap);
    hip_ok(hipMemcpy(cu, d_cu, 4 * ((size_t)k + 1), hipMemcpyDeviceToHost), "hipMemcpy(cu)");
    hip_ok(hipMemcpy(p, d_pos, 4 * (size_t)n_tok, hipMemcpyDeviceToHost), "hipMemcpy(pos)");
    hip_ok(hipMemcpy(rows, d_out, row * (size_t)n_tok, hipMemcpyDeviceToHost), "hipMemcpy(rows)");
    const int32_t head[3] = {n_tok, mx, k};
    wr(head, 4, 3, out);
    wr(cu, 4, (size_t)k + 1, out);
    wr(p, 4, (size_t)n_tok, out);
    wr(rows, row, (size_t)n_tok, out);
    free(cu);
    free(p);
    free(rows);
    hip_ok(hipFree(d_out), "hipFree(out)");
    hip_ok(hipFree(d_cu), "hipFree(cu)");
    hip_ok(hipFree(d_pos), "hipFree(pos)");
  }
  fclose(out);
  for (int32_t i = 0; i < n; ++i)
    if (pool_free_sample(pool, ids[i]) != FP_OK) die("pool_free_sample");
  hip_ok(hipDeviceSynchronize(), "hipDeviceSynchronize");
  if (pool_destroy(pool) != FP_OK) die("pool_destroy");
  hip_ok(hipFree(d_table), "hipFree(table)");
  return 0;
}
