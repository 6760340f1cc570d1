/* oracle_sanitize_main.c -- drives every entry of the CPU oracle under the
 * address and undefined-behaviour sanitizers (built and run by
 * tests/test_oracle_sanitize.py on the host; test infrastructure only).
 *
 * argv: blob file, then the model fields n_layers hidden n_q_heads n_kv_heads
 * head_dim ffn n_codes vocab max_draft dtype topk draft_len, then a file with
 * the frame hidden vector (float32[hidden]) followed by the uniforms
 * (float32[n_codes][3]) and c0 as int32. Prints one line per call and exits 0
 * when every call returned its expected status. */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../oracle/rvqsd_oracle.h"

static void* slurp(const char* path, size_t* n) {
  FILE* f = fopen(path, "rb");
  if (!f) return NULL;
  fseek(f, 0, SEEK_END);
  long len = ftell(f);
  fseek(f, 0, SEEK_SET);
  void* buf = malloc((size_t)len);
  if (buf && fread(buf, 1, (size_t)len, f) != (size_t)len) { free(buf); buf = NULL; }
  fclose(f);
  *n = (size_t)len;
  return buf;
}

#define EXPECT(cond, what)                          \
  do {                                              \
    if (!(cond)) {                                  \
      fprintf(stderr, "FAILED: %s\n", what);        \
      return 1;                                     \
    }                                               \
    printf("ok %s\n", what);                        \
  } while (0)

int main(int argc, char** argv) {
  if (argc != 16) {
    fprintf(stderr, "usage: blob 12 model fields inputs\n");
    return 2;
  }
  size_t nb = 0, ni = 0;
  void* blob = slurp(argv[1], &nb);
  orc_cfg c;
  memset(&c, 0, sizeof(c));
  int32_t* fld[] = {&c.n_layers, &c.hidden, &c.n_q_heads, &c.n_kv_heads, &c.head_dim, &c.ffn,
                    &c.n_codes, &c.vocab, &c.max_draft, &c.dtype, &c.topk, &c.draft_len};
  for (int i = 0; i < 12; ++i) *fld[i] = atoi(argv[2 + i]);
  c.qk_norm = 1;
  c.rms_eps = 1e-6;
  c.rope_base = 1e6;
  c.temperature = 0.9;
  unsigned char* in = (unsigned char*)slurp(argv[14], &ni);
  EXPECT(blob && in && ni == (size_t)(c.hidden + 3 * c.n_codes + 1) * 4, "inputs read");
  const float* f = (const float*)in;
  const float* uni = f + c.hidden;
  int32_t c0;
  memcpy(&c0, uni + 3 * c.n_codes, 4);
  (void)argv[15];

  int32_t st = 0;
  EXPECT(orc_create(NULL, blob, nb, &st) == NULL && st == ORC_EINVAL, "null cfg rejected");
  EXPECT(orc_create(&c, blob, nb - 4, &st) == NULL && st == ORC_EBLOB, "short blob rejected");
  orc_cfg bad = c;
  bad.draft_len = bad.max_draft + 1;
  EXPECT(orc_create(&bad, blob, nb, &st) == NULL && st == ORC_EINVAL, "draft_len > max_draft rejected");

  const int H = c.hidden, V = c.vocab, n = c.n_codes;
  int32_t codes[16], ar[16];
  double* h = (double*)malloc(sizeof(double) * (n + 1) * H);
  double* lg = (double*)malloc(sizeof(double) * V);
  double* rows = (double*)malloc(sizeof(double) * 40 * H);
  for (int i = 0; i < 40 * H; ++i) rows[i] = (double)((i * 37) % 101) / 50.0 - 1.0;
  double* tl = (double*)malloc(sizeof(double) * 16 * 16 * V * 2);
  orc_round rr[16];
  for (int mode = 0; mode <= 2; ++mode) {
    c.draft_mode = mode;
    orc_model* m = orc_create(&c, blob, nb, &st);
    EXPECT(m && st == ORC_OK, "create");
    int32_t ic[16];
    for (int s = 0; s < n; ++s) ic[s] = (c0 + 5 * s) % V;
    EXPECT(orc_forward(m, f, ic, n + 1, h) == ORC_OK, "forward, every position");
    EXPECT(orc_forward(m, f, ic, n + 2, h) == ORC_EINVAL, "forward past the frame rejected");
    EXPECT(orc_forward_vectors(m, rows, 40, rows + 0) == ORC_OK, "forward over 40 vector positions (in place)");
    EXPECT(orc_forward_vectors(m, rows, ORC_MAX_VECTOR_POS + 1, rows) == ORC_EINVAL, "too many vector positions rejected");
    EXPECT(orc_logits(m, h + H, 1, 0, lg) == ORC_OK, "logits");
    EXPECT(orc_logits(m, h + H, n + 1, 0, lg) == ORC_EINVAL, "head past the last rejected");
    if (c.max_draft > 0) EXPECT(orc_logits(m, h + H, n, c.max_draft, lg) == ORC_OK, "logits with the last offset");
    int32_t idx[256];
    double pr[256];
    int k = orc_topk_softmax(lg, V, c.topk, 0.9, idx, pr);
    EXPECT(k > 0 && orc_sample(idx, pr, k, 0.999) >= 0, "top-k softmax and sample");
    int32_t tok = -1;
    EXPECT(orc_accept_or_resample(idx, pr, k, idx, pr, k, idx[0], 0.5, 0.5, &tok) >= 0, "accept or resample");
    EXPECT(orc_ar_frame(m, f, c0, uni, ar) == ORC_OK, "AR frame");
    EXPECT(orc_ar_frame(m, f, V, uni, ar) == ORC_EINVAL, "bad c0 rejected");
    orc_stats S;
    orc_trace T;
    T.rounds = rr;
    T.verify_logits = tl;
    T.draft_logits = tl + 16 * 16 * V;
    T.max_rounds = 16;
    T.n_rounds = 0;
    EXPECT(orc_spec_frame(m, f, c0, uni, codes, &S, &T, NULL, NULL) == ORC_OK, "speculative frame, traced");
    EXPECT(S.target_calls == 1 + S.rounds && T.n_rounds == S.target_calls, "round accounting");
    T.n_rounds = 0;
    T.max_rounds = 2;
    EXPECT(orc_spec_frame(m, f, c0, uni, codes, &S, &T, NULL, NULL) == ORC_OK, "trace shorter than the frame");
    EXPECT(orc_spec_frame(m, f, c0, uni, codes, NULL, NULL, NULL, NULL) == ORC_OK, "untraced frame");
    if (mode == 0 && c.draft_len >= 2 && c.topk >= 2) {
      /* the sparse tree of Fig. 2 (depth 3 is cut to the draft length) */
      orc_tree t;
      memset(&t, 0, sizeof(t));
      const int par[8] = {0, 0, 1, 1, 2, 3, 5, 5}, rk[8] = {0, 1, 0, 1, 0, 0, 0, 1};
      t.n_nodes = 8;
      for (int r = 1; r <= 8; ++r) { t.parent[r] = par[r - 1]; t.rank[r] = rk[r - 1]; }
      int32_t mask[81];
      EXPECT(orc_tree_mask(&t, mask) == ORC_OK && mask[8 * 9 + 5] == 1 && mask[8 * 9 + 3] == 0, "tree mask");
      orc_tree_round tr[16];
      double* tv = (double*)malloc(sizeof(double) * 16 * (ORC_MAX_TREE + 1) * V);
      orc_tree_trace TT = {tr, tv, tl, 16, 0};
      EXPECT(orc_tree_frame(m, &t, f, c0, uni, codes, &S, &TT, NULL, NULL) == ORC_OK, "tree frame, traced");
      EXPECT(orc_tree_frame(m, &t, f, c0, uni, codes, &S, NULL, NULL, NULL) == ORC_OK, "tree frame, untraced");
      t.parent[2] = 2;
      EXPECT(orc_tree_frame(m, &t, f, c0, uni, codes, &S, NULL, NULL, NULL) == ORC_EINVAL, "malformed tree rejected");
      free(tv);
    }
    orc_destroy(m);
  }
  float u2[45];
  orc_uniforms_from_seed(12345, 15, u2);
  EXPECT(u2[0] >= 0.f && u2[44] < 1.f, "uniforms from a seed");
  free(h); free(lg); free(rows); free(tl); free(blob); free(in);
  printf("ALL OK\n");
  return 0;
}
