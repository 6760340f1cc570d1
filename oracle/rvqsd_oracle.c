/* rvqsd_oracle.c -- CPU oracle (TEST INFRASTRUCTURE; see rvqsd_oracle.h).
 *
 * Plain loops in fp64. Every call recomputes the forward pass over the whole
 * prefix from scratch (no KV cache): causal attention makes the hidden state at
 * position s depend only on the inputs at positions <= s, so a cache is an
 * optimisation the oracle does not need.
 *
 * Readings of points the paper leaves open (the paper only fixes the layer
 * counts, the per-position tables/heads and the sampling rule):
 *   - block: pre-norm decoder layer with RMSNorm, per-head RMSNorm of q and k
 *     (flag qk_norm), rotate-half RoPE over the full head dimension, causal
 *     grouped-query attention scaled by 1/sqrt(d), SwiGLU MLP, no biases, a
 *     final RMSNorm before the heads;
 *   - prefix: position 0 is the frame hidden vector used as is, position 1
 *     consumes c_0 through E_0 (Fig. 1); RoPE positions restart at 0 per frame;
 *   - the offset b_j is added to the final-normed hidden state, i.e. to the
 *     vector LMH consumes (Sec. 2.2, "h_k + b_j");
 *   - drafts are sampled from the top-k, temperature-T softmax of the draft
 *     logits (a greedy mode takes the argmax);
 *   - top-k ties go to the lower token index; the inverse CDF walks the support
 *     in ascending token order; acceptance is the strict test u*q(d) < p(d);
 *     a residual with no mass falls back to p;
 *   - the uniforms of a frame are indexed by code position s and slot
 *     (draft, accept, sample), never by round.
 */
#include "rvqsd_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define MAX_POS 17   /* 1 frame-hidden position + up to 16 code positions */

/* Every weight is held as the exact value it stands for, in double: f32 and bf16
 * values widen exactly; an int8 matrix (W8A16, dtype 2) holds s[o] * q[o][i], the
 * product of its row's fp32 scale and int8 code, which a double represents exactly. */
struct orc_model {
  orc_cfg cfg;
  double* store;
  /* per layer */
  const double **attn_norm, **wq, **wk, **wv, **q_norm, **k_norm, **wo, **mlp_norm, **wgate, **wup, **wdown;
  const double* final_norm;
  const double** emb; /* [n_codes], E_i embeds c_i */
  const double** lmh; /* [n_codes + 1], LMH_s emits c_s (index 0 unused) */
  const double* offsets; /* [max_draft][H] */
};

int32_t orc_abi_version(void) { return 1; }

void orc_set_threads(int32_t n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

int32_t orc_get_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* ------------------------------------------------------------------ blob */

static uint32_t rd32(const unsigned char* p) {
  return (uint32_t)p[0] | ((uint32_t)p[1] << 8) | ((uint32_t)p[2] << 16) | ((uint32_t)p[3] << 24);
}

static float bf16_to_float(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

orc_model* orc_create(const orc_cfg* cfg, const void* blob, size_t blob_bytes, int32_t* status) {
  int32_t st = ORC_OK;
  orc_model* m = NULL;
  if (!cfg || !blob) { st = ORC_EINVAL; goto out; }
  {
    const orc_cfg* c = cfg;
    if (c->n_layers <= 0 || c->hidden <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0 ||
        (c->head_dim % 2) != 0 || c->ffn <= 0 || c->n_codes <= 0 || c->n_codes > MAX_POS - 1 || c->vocab <= 0 ||
        c->max_draft < 0 || c->topk <= 0 || c->draft_len < 0 || c->draft_len > c->max_draft ||
        (c->n_q_heads % c->n_kv_heads) != 0 || !(c->temperature > 0.0) || (c->dtype < 0 || c->dtype > 2) ||
        c->draft_mode < 0 || c->draft_mode > 2) {
      st = ORC_EINVAL;
      goto out;
    }
  }
  {
    const unsigned char* b = (const unsigned char*)blob;
    if (blob_bytes < 64 || memcmp(b, "RVQSDW1\0", 8) != 0 || rd32(b + 8) != 1) { st = ORC_EBLOB; goto out; }
    const uint32_t want[10] = {(uint32_t)cfg->dtype, (uint32_t)cfg->n_layers, (uint32_t)cfg->hidden,
                               (uint32_t)cfg->n_q_heads, (uint32_t)cfg->n_kv_heads, (uint32_t)cfg->head_dim,
                               (uint32_t)cfg->ffn, (uint32_t)cfg->n_codes, (uint32_t)cfg->vocab,
                               (uint32_t)cfg->max_draft};
    for (int i = 0; i < 10; ++i)
      if (rd32(b + 12 + 4 * i) != want[i]) { st = ORC_EBLOB; goto out; }
  }
  {
    const int L = cfg->n_layers, H = cfg->hidden, d = cfg->head_dim, F = cfg->ffn, V = cfg->vocab, n = cfg->n_codes;
    const size_t qd = (size_t)cfg->n_q_heads * d, kd = (size_t)cfg->n_kv_heads * d;
    /* bytes of a [rows][cols] matrix in the blob: f32, bf16, or int8 codes + fp32 row
     * scales padded to 16 bytes */
#define MAT_BYTES(rows, cols)                                                                  \
  (cfg->dtype == 0 ? (size_t)(rows) * (cols) * 4                                               \
                   : cfg->dtype == 1 ? (size_t)(rows) * (cols) * 2                             \
                                     : (((size_t)(rows) * (cols) + 4 * (size_t)(rows) + 15) / 16 * 16))
    size_t n_vec = 0, n_mat = 0, mat_bytes = 0;
    n_vec += (size_t)L * (H + d + d + H);
    n_mat += (size_t)L * (qd * H + 2 * kd * H + H * qd + 2 * (size_t)F * H + (size_t)H * F);
    mat_bytes += (size_t)L * (MAT_BYTES(qd, H) + 2 * MAT_BYTES(kd, H) + MAT_BYTES(H, qd) + 2 * MAT_BYTES(F, H) +
                              MAT_BYTES(H, F));
    n_vec += H;
    n_mat += (size_t)2 * n * V * H;
    mat_bytes += (size_t)2 * n * MAT_BYTES(V, H);
    n_vec += (size_t)cfg->max_draft * H;
    if (blob_bytes != 64 + n_vec * 4 + mat_bytes) { st = ORC_EBLOB; goto out; }

    m = (orc_model*)calloc(1, sizeof(orc_model));
    if (!m) { st = ORC_ENOMEM; goto out; }
    m->cfg = *cfg;
    m->store = (double*)malloc((n_vec + n_mat) * sizeof(double));
    const double*** lay[11] = {&m->attn_norm, &m->wq, &m->wk, &m->wv, &m->q_norm, &m->k_norm,
                               &m->wo, &m->mlp_norm, &m->wgate, &m->wup, &m->wdown};
    int fail = !m->store;
    for (int i = 0; i < 11; ++i) {
      *lay[i] = (const double**)calloc((size_t)L, sizeof(double*));
      fail |= !*lay[i];
    }
    m->emb = (const double**)calloc((size_t)n, sizeof(double*));
    m->lmh = (const double**)calloc((size_t)n + 1, sizeof(double*));
    if (fail || !m->emb || !m->lmh) { st = ORC_ENOMEM; goto out; }

    const unsigned char* src = (const unsigned char*)blob + 64;
    double* dst = m->store;
    /* one tensor of `rows` x `cols` elements; vectors are f32, matrices f32, bf16 or int8
     * codes with fp32 row scales (weight = scale * code) */
#define TAKE(ptr, rows, cols, is_mat)                                                           \
  do {                                                                                          \
    const size_t r_ = (rows), c_ = (cols), cnt_ = r_ * c_;                                      \
    (ptr) = dst;                                                                                \
    if ((is_mat) && cfg->dtype == 1) {                                                          \
      for (size_t i_ = 0; i_ < cnt_; ++i_)                                                      \
        dst[i_] = (double)bf16_to_float((uint16_t)(src[2 * i_] | (src[2 * i_ + 1] << 8)));      \
      src += 2 * cnt_;                                                                          \
    } else if ((is_mat) && cfg->dtype == 2) {                                                   \
      const unsigned char* sc_ = src + cnt_;                                                    \
      for (size_t o_ = 0; o_ < r_; ++o_) {                                                      \
        float s_;                                                                               \
        memcpy(&s_, sc_ + 4 * o_, 4);                                                           \
        for (size_t i_ = 0; i_ < c_; ++i_)                                                      \
          dst[o_ * c_ + i_] = (double)s_ * (double)(int8_t)src[o_ * c_ + i_];                   \
      }                                                                                         \
      src += MAT_BYTES(r_, c_);                                                                 \
    } else {                                                                                    \
      for (size_t i_ = 0; i_ < cnt_; ++i_) {                                                    \
        float f_;                                                                               \
        memcpy(&f_, src + 4 * i_, 4);                                                           \
        dst[i_] = (double)f_;                                                                   \
      }                                                                                         \
      src += 4 * cnt_;                                                                          \
    }                                                                                           \
    dst += cnt_;                                                                                \
  } while (0)
    for (int l = 0; l < L; ++l) {
      TAKE(m->attn_norm[l], 1, (size_t)H, 0);
      TAKE(m->wq[l], qd, (size_t)H, 1);
      TAKE(m->wk[l], kd, (size_t)H, 1);
      TAKE(m->wv[l], kd, (size_t)H, 1);
      TAKE(m->q_norm[l], 1, (size_t)d, 0);
      TAKE(m->k_norm[l], 1, (size_t)d, 0);
      TAKE(m->wo[l], (size_t)H, qd, 1);
      TAKE(m->mlp_norm[l], 1, (size_t)H, 0);
      TAKE(m->wgate[l], (size_t)F, (size_t)H, 1);
      TAKE(m->wup[l], (size_t)F, (size_t)H, 1);
      TAKE(m->wdown[l], (size_t)H, (size_t)F, 1);
    }
    TAKE(m->final_norm, 1, (size_t)H, 0);
    for (int i = 0; i < n; ++i) TAKE(m->emb[i], (size_t)V, (size_t)H, 1);
    for (int t = 1; t <= n; ++t) TAKE(m->lmh[t], (size_t)V, (size_t)H, 1);
    TAKE(m->offsets, (size_t)cfg->max_draft, (size_t)H, 0);
#undef TAKE
#undef MAT_BYTES
  }
out:
  if (st != ORC_OK && m) { orc_destroy(m); m = NULL; }
  if (status) *status = st;
  return m;
}

void orc_destroy(orc_model* m) {
  if (!m) return;
  free(m->store);
  free((void*)m->attn_norm); free((void*)m->wq); free((void*)m->wk); free((void*)m->wv);
  free((void*)m->q_norm); free((void*)m->k_norm); free((void*)m->wo); free((void*)m->mlp_norm);
  free((void*)m->wgate); free((void*)m->wup); free((void*)m->wdown);
  free((void*)m->emb); free((void*)m->lmh);
  free(m);
}

/* --------------------------------------------------------------- forward */

/* y = x / sqrt(mean(x^2) + eps) * g */
static void rmsnorm(const double* x, const double* g, int n, double eps, double* y) {
  double ss = 0.0;
  for (int i = 0; i < n; ++i) ss += x[i] * x[i];
  double r = 1.0 / sqrt(ss / n + eps);
  for (int i = 0; i < n; ++i) y[i] = x[i] * r * g[i];
}

/* Y[p][o] = sum_k W[o][k] * X[p][k] for p < np (W: [rows][cols]) */
static void matmul(const double* W, int rows, int cols, const double* X, int np, double* Y) {
#pragma omp parallel for schedule(static) if ((long)rows * cols * np >= 1L << 18)
  for (int o = 0; o < rows; ++o) {
    const double* w = W + (size_t)o * cols;
    for (int p = 0; p < np; ++p) {
      const double* x = X + (size_t)p * cols;
      double acc = 0.0;
      for (int k = 0; k < cols; ++k) acc += w[k] * x[k];
      Y[(size_t)p * rows + o] = acc;
    }
  }
}

/* rotate-half RoPE at position pos: pairs (i, i + d/2), angle pos * base^(-2i/d) */
static void rope(double* v, int d, int pos, double base) {
  int h = d / 2;
  for (int i = 0; i < h; ++i) {
    double theta = (double)pos * pow(base, -2.0 * i / d);
    double c = cos(theta), s = sin(theta);
    double a = v[i], b = v[i + h];
    v[i] = a * c - b * s;
    v[i + h] = b * c + a * s;
  }
}

static double silu(double z) { return z / (1.0 + exp(-z)); }

/* The decoder stack over input rows x[np][H] (overwritten): positions 0..np-1,
 * causal attention, final RMSNorm into hfin[np][H]. */
static int32_t forward_rows(orc_model* m, double* x, int32_t np, double* hfin) {
  const orc_cfg* c = &m->cfg;
  const int H = c->hidden, d = c->head_dim, nq = c->n_q_heads, nkv = c->n_kv_heads, F = c->ffn;
  const int qd = nq * d, kd = nkv * d, rep = nq / nkv;
  double* a = (double*)malloc(sizeof(double) * np * H);
  double* Q = (double*)malloc(sizeof(double) * np * qd);
  double* Kc = (double*)malloc(sizeof(double) * np * kd);
  double* Vc = (double*)malloc(sizeof(double) * np * kd);
  double* O = (double*)malloc(sizeof(double) * np * qd);
  double* Y = (double*)malloc(sizeof(double) * np * (H > F ? H : F));
  double* G = (double*)malloc(sizeof(double) * np * F);
  double* U = (double*)malloc(sizeof(double) * np * F);
  double* tmp = (double*)malloc(sizeof(double) * (d > np ? d : np));
  if (!a || !Q || !Kc || !Vc || !O || !Y || !G || !U || !tmp) {
    free(a); free(Q); free(Kc); free(Vc); free(O); free(Y); free(G); free(U); free(tmp);
    return ORC_ENOMEM;
  }

  const double scale = 1.0 / sqrt((double)d);
  for (int l = 0; l < c->n_layers; ++l) {
    for (int p = 0; p < np; ++p) rmsnorm(x + (size_t)p * H, m->attn_norm[l], H, c->rms_eps, a + (size_t)p * H);
    matmul(m->wq[l], qd, H, a, np, Q);
    matmul(m->wk[l], kd, H, a, np, Kc);
    matmul(m->wv[l], kd, H, a, np, Vc);
    for (int p = 0; p < np; ++p) {
      for (int h = 0; h < nq; ++h) {
        double* q = Q + (size_t)p * qd + (size_t)h * d;
        if (c->qk_norm) {
          rmsnorm(q, m->q_norm[l], d, c->rms_eps, tmp);
          memcpy(q, tmp, sizeof(double) * d);
        }
        rope(q, d, p, c->rope_base);
      }
      for (int g = 0; g < nkv; ++g) {
        double* k = Kc + (size_t)p * kd + (size_t)g * d;
        if (c->qk_norm) {
          rmsnorm(k, m->k_norm[l], d, c->rms_eps, tmp);
          memcpy(k, tmp, sizeof(double) * d);
        }
        rope(k, d, p, c->rope_base);
      }
    }
    /* causal grouped-query attention: q head h reads kv head h / rep */
    for (int p = 0; p < np; ++p) {
      for (int h = 0; h < nq; ++h) {
        const int g = h / rep;
        const double* q = Q + (size_t)p * qd + (size_t)h * d;
        double mx = -INFINITY;
        for (int t = 0; t <= p; ++t) {
          const double* k = Kc + (size_t)t * kd + (size_t)g * d;
          double sc = 0.0;
          for (int i = 0; i < d; ++i) sc += q[i] * k[i];
          tmp[t] = sc * scale;
          if (tmp[t] > mx) mx = tmp[t];
        }
        double z = 0.0;
        for (int t = 0; t <= p; ++t) {
          tmp[t] = exp(tmp[t] - mx);
          z += tmp[t];
        }
        double* o = O + (size_t)p * qd + (size_t)h * d;
        for (int i = 0; i < d; ++i) {
          double acc = 0.0;
          for (int t = 0; t <= p; ++t) acc += tmp[t] * Vc[(size_t)t * kd + (size_t)g * d + i];
          o[i] = acc / z;
        }
      }
    }
    matmul(m->wo[l], H, qd, O, np, Y);
    for (size_t i = 0; i < (size_t)np * H; ++i) x[i] += Y[i];
    for (int p = 0; p < np; ++p) rmsnorm(x + (size_t)p * H, m->mlp_norm[l], H, c->rms_eps, a + (size_t)p * H);
    matmul(m->wgate[l], F, H, a, np, G);
    matmul(m->wup[l], F, H, a, np, U);
    for (size_t i = 0; i < (size_t)np * F; ++i) G[i] = silu(G[i]) * U[i];
    matmul(m->wdown[l], H, F, G, np, Y);
    for (size_t i = 0; i < (size_t)np * H; ++i) x[i] += Y[i];
  }
  for (int p = 0; p < np; ++p) rmsnorm(x + (size_t)p * H, m->final_norm, H, c->rms_eps, hfin + (size_t)p * H);

  free(a); free(Q); free(Kc); free(Vc); free(O); free(Y); free(G); free(U); free(tmp);
  return ORC_OK;
}

int32_t orc_forward(orc_model* m, const float* frame_hidden, const int32_t* in_codes, int32_t n_pos, double* hfin) {
  if (!m || !frame_hidden || !hfin || n_pos < 1 || n_pos > m->cfg.n_codes + 1 || (n_pos > 1 && !in_codes))
    return ORC_EINVAL;
  const orc_cfg* c = &m->cfg;
  const int H = c->hidden, np = n_pos;
  for (int s = 1; s < np; ++s)
    if (in_codes[s - 1] < 0 || in_codes[s - 1] >= c->vocab) return ORC_EINVAL;
  double* x = (double*)malloc(sizeof(double) * np * H);
  if (!x) return ORC_ENOMEM;
  /* inputs: x_0 = frame hidden, x_s = E_{s-1}[code consumed at s] */
  for (int i = 0; i < H; ++i) x[i] = (double)frame_hidden[i];
  for (int s = 1; s < np; ++s) {
    const double* e = m->emb[s - 1] + (size_t)in_codes[s - 1] * H;
    for (int i = 0; i < H; ++i) x[(size_t)s * H + i] = e[i];
  }
  const int32_t st = forward_rows(m, x, np, hfin);
  free(x);
  return st;
}

int32_t orc_forward_vectors(orc_model* m, const double* rows, int32_t n_pos, double* hfin) {
  if (!m || !rows || !hfin || n_pos < 1 || n_pos > ORC_MAX_VECTOR_POS) return ORC_EINVAL;
  const size_t cnt = (size_t)n_pos * m->cfg.hidden;
  double* x = (double*)malloc(sizeof(double) * cnt);
  if (!x) return ORC_ENOMEM;
  memcpy(x, rows, sizeof(double) * cnt);
  const int32_t st = forward_rows(m, x, n_pos, hfin);
  free(x);
  return st;
}

int32_t orc_logits(orc_model* m, const double* h, int32_t head, int32_t offset, double* out) {
  if (!m || !h || !out || head < 1 || head > m->cfg.n_codes || offset < 0 || offset > m->cfg.max_draft)
    return ORC_EINVAL;
  const int H = m->cfg.hidden;
  double* v = (double*)malloc(sizeof(double) * H);
  if (!v) return ORC_ENOMEM;
  for (int i = 0; i < H; ++i) v[i] = h[i] + (offset > 0 ? m->offsets[(size_t)(offset - 1) * H + i] : 0.0);
  matmul(m->lmh[head], m->cfg.vocab, H, v, 1, out);
  free(v);
  return ORC_OK;
}

/* ------------------------------------------------------------- decisions */

typedef struct {
  double v;
  int32_t i;
} vi_t;

static int cmp_desc(const void* pa, const void* pb) {
  const vi_t* a = (const vi_t*)pa;
  const vi_t* b = (const vi_t*)pb;
  if (a->v > b->v) return -1;
  if (a->v < b->v) return 1;
  return a->i < b->i ? -1 : (a->i > b->i ? 1 : 0);
}

static int cmp_idx(const void* pa, const void* pb) {
  const vi_t* a = (const vi_t*)pa;
  const vi_t* b = (const vi_t*)pb;
  return a->i < b->i ? -1 : (a->i > b->i ? 1 : 0);
}

/* top-k selection + tempered softmax over the selected logits; also reports the
 * gap between the k-th and (k+1)-th largest logits (INFINITY if none). */
static int32_t topk_softmax_gap(const double* logits, int32_t V, int32_t topk, double T, int32_t* idx_out,
                                double* prob_out, double* gap) {
  vi_t* a = (vi_t*)malloc(sizeof(vi_t) * V);
  if (!a) return ORC_ENOMEM;
  for (int i = 0; i < V; ++i) {
    double v = logits[i];
    a[i].v = isnan(v) ? -INFINITY : v; /* non-finite logits count as -inf */
    a[i].i = i;
  }
  qsort(a, (size_t)V, sizeof(vi_t), cmp_desc);
  int n = topk < V ? topk : V;
  if (gap) *gap = (n < V) ? a[n - 1].v - a[n].v : INFINITY;
  double mu = a[0].v;
  if (!(mu > -INFINITY) || isinf(mu)) {
    free(a);
    return ORC_ENUMERIC;
  }
  qsort(a, (size_t)n, sizeof(vi_t), cmp_idx);
  double z = 0.0;
  for (int j = 0; j < n; ++j) {
    double w = exp((a[j].v - mu) / T);
    prob_out[j] = w;
    z += w;
  }
  for (int j = 0; j < n; ++j) {
    idx_out[j] = a[j].i;
    prob_out[j] = prob_out[j] / z;
  }
  free(a);
  return n;
}

int32_t orc_topk_softmax(const double* logits, int32_t vocab, int32_t topk, double temperature, int32_t* idx_out,
                         double* prob_out) {
  if (!logits || !idx_out || !prob_out || vocab <= 0 || topk <= 0 || !(temperature > 0.0)) return ORC_EINVAL;
  return topk_softmax_gap(logits, vocab, topk, temperature, idx_out, prob_out, NULL);
}

typedef struct {
  orc_probe_fn fn;
  void* ctx;
  double margin; /* running min |u - breakpoint| */
} dctx_t;

/* inverse CDF over the support in array (ascending token) order */
static int32_t sample_dist(const int32_t* idx, const double* w, int32_t n, double u, dctx_t* dc, int32_t uidx) {
  double z = 0.0;
  for (int j = 0; j < n; ++j) z += w[j];
  double thr = u * z;
  if (dc) {
    double* bp = (double*)malloc(sizeof(double) * (size_t)n);
    int nb = 0;
    double cum = 0.0;
    for (int j = 0; j < n; ++j) {
      cum += w[j];
      double b = cum / z;
      if (bp && b < 1.0) bp[nb++] = b;
      double dist = fabs(u - b);
      if (dist < dc->margin) dc->margin = dist;
    }
    if (dc->fn && bp) dc->fn(dc->ctx, uidx, bp, nb);
    free(bp);
  }
  double cum = 0.0;
  for (int j = 0; j < n; ++j) {
    cum += w[j];
    if (cum > thr) return idx[j];
  }
  for (int j = n - 1; j >= 0; --j)
    if (w[j] > 0.0) return idx[j];
  return idx[n - 1];
}

int32_t orc_sample(const int32_t* idx, const double* prob, int32_t n, double u) {
  if (!idx || !prob || n <= 0) return ORC_EINVAL;
  return sample_dist(idx, prob, n, u, NULL, -1);
}

static double prob_of(const int32_t* idx, const double* p, int32_t n, int32_t tok) {
  for (int j = 0; j < n; ++j)
    if (idx[j] == tok) return p[j];
  return 0.0;
}

static int32_t accept_or_resample(const int32_t* pidx, const double* pp, int32_t np, const int32_t* qidx,
                                  const double* qp, int32_t nq, int32_t d, double u_acc, double u_samp,
                                  int32_t* token, dctx_t* dc, int32_t s) {
  double qd = prob_of(qidx, qp, nq, d);
  double pd = prob_of(pidx, pp, np, d);
  if (dc) {
    double bp = qd > 0.0 ? pd / qd : 0.0;
    double dist = fabs(u_acc - bp);
    if (dist < dc->margin) dc->margin = dist;
    if (dc->fn) {
      int nb = (bp > 0.0 && bp < 1.0) ? 1 : 0;
      dc->fn(dc->ctx, (s - 1) * 3 + 1, &bp, nb);
    }
  }
  if (u_acc * qd < pd) return 1;
  /* residual max(0, p - q) on p's support; no mass -> p */
  double* r = (double*)malloc(sizeof(double) * (size_t)np);
  if (!r) return ORC_ENOMEM;
  double rs = 0.0;
  for (int j = 0; j < np; ++j) {
    double v = pp[j] - prob_of(qidx, qp, nq, pidx[j]);
    r[j] = v > 0.0 ? v : 0.0;
    rs += r[j];
  }
  if (!(rs > 0.0))
    for (int j = 0; j < np; ++j) r[j] = pp[j];
  *token = sample_dist(pidx, r, np, u_samp, dc, (s - 1) * 3 + 2);
  free(r);
  return 0;
}

int32_t orc_accept_or_resample(const int32_t* pidx, const double* pp, int32_t np, const int32_t* qidx,
                               const double* qp, int32_t nq, int32_t d, double u_acc, double u_samp,
                               int32_t* token) {
  if (!pidx || !pp || !qidx || !qp || !token || np <= 0 || nq <= 0) return ORC_EINVAL;
  return accept_or_resample(pidx, pp, np, qidx, qp, nq, d, u_acc, u_samp, token, NULL, 1);
}

/* ----------------------------------------------------------------- frames */

static double U(const float* uni, int s, int slot) { return (double)uni[(s - 1) * 3 + slot]; }

int32_t orc_ar_frame(orc_model* m, const float* frame_hidden, int32_t c0, const float* uniforms, int32_t* out_codes) {
  if (!m || !frame_hidden || !uniforms || !out_codes || c0 < 0 || c0 >= m->cfg.vocab) return ORC_EINVAL;
  const orc_cfg* c = &m->cfg;
  const int n = c->n_codes, H = c->hidden, V = c->vocab;
  int32_t codes[MAX_POS];
  double* hfin = (double*)malloc(sizeof(double) * (n + 1) * H);
  double* lg = (double*)malloc(sizeof(double) * V);
  int32_t* idx = (int32_t*)malloc(sizeof(int32_t) * V);
  double* pr = (double*)malloc(sizeof(double) * V);
  int32_t st = (hfin && lg && idx && pr) ? ORC_OK : ORC_ENOMEM;
  codes[0] = c0;
  /* c_s ~ topk-softmax(LMH_s(h_s) / T), h_s from the committed c_0..c_{s-1} */
  for (int s = 1; s <= n && st == ORC_OK; ++s) {
    st = orc_forward(m, frame_hidden, codes, s + 1, hfin);
    if (st != ORC_OK) break;
    st = orc_logits(m, hfin + (size_t)s * H, s, 0, lg);
    if (st != ORC_OK) break;
    int32_t k = topk_softmax_gap(lg, V, c->topk, c->temperature, idx, pr, NULL);
    if (k < 0) { st = k; break; }
    codes[s] = sample_dist(idx, pr, k, U(uniforms, s, 2), NULL, -1);
  }
  if (st == ORC_OK)
    for (int s = 1; s <= n; ++s) out_codes[s - 1] = codes[s];
  free(hfin); free(lg); free(idx); free(pr);
  return st;
}

/* one proposal distribution for a drafted position */
typedef struct {
  int32_t n;
  int32_t* idx;
  double* p;
} dist_t;

int32_t orc_spec_frame(orc_model* m, const float* frame_hidden, int32_t c0, const float* uniforms,
                       int32_t* out_codes, orc_stats* stats, orc_trace* trace, orc_probe_fn probe,
                       void* probe_ctx) {
  if (!m || !frame_hidden || !uniforms || !out_codes || c0 < 0 || c0 >= m->cfg.vocab) return ORC_EINVAL;
  const orc_cfg* c = &m->cfg;
  const int n = c->n_codes, H = c->hidden, V = c->vocab, K = c->draft_len;
  const int T_ROWS = 16;
  int32_t st = ORC_OK;
  int32_t codes[MAX_POS];   /* committed c_0..c_n */
  int32_t inputs[MAX_POS];  /* code consumed at position s is inputs[s-1] */
  int32_t drafts[MAX_POS];  /* d_s */
  orc_stats S = {0, 0, 0, 0, 0};
  dctx_t dc = {probe, probe_ctx, INFINITY};

  double* hfin = (double*)malloc(sizeof(double) * (n + 1) * H);
  double* hanc = (double*)malloc(sizeof(double) * H);
  double* lg = (double*)malloc(sizeof(double) * V);
  int32_t* pidx = (int32_t*)malloc(sizeof(int32_t) * V);
  double* pp = (double*)malloc(sizeof(double) * V);
  dist_t q[MAX_POS];
  for (int s = 0; s < MAX_POS; ++s) {
    q[s].n = 0;
    q[s].idx = (int32_t*)malloc(sizeof(int32_t) * V);
    q[s].p = (double*)malloc(sizeof(double) * V);
    if (!q[s].idx || !q[s].p) st = ORC_ENOMEM;
  }
  if (!hfin || !hanc || !lg || !pidx || !pp) st = ORC_ENOMEM;

  orc_round* rec = NULL;
  double gap = INFINITY, round_gap = INFINITY;
  codes[0] = c0;
  int m_anchor = 0;

  /* prefix pass: positions 0 (frame hidden) and 1 (E_0[c_0]) */
  if (st == ORC_OK) {
    inputs[0] = c0;
    st = orc_forward(m, frame_hidden, inputs, 2, hfin);
  }
  if (st == ORC_OK) {
    S.target_calls = 1;
    if (trace && trace->rounds && trace->n_rounds < trace->max_rounds) {
      rec = &trace->rounds[trace->n_rounds];
      memset(rec, 0, sizeof(*rec));
      rec->m = 0; rec->kp = 0; rec->n_rows = 2; rec->token = -1;
    }
    st = orc_logits(m, hfin + H, 1, 0, lg);
  }
  if (st == ORC_OK) {
    if (rec && trace->verify_logits)
      memcpy(trace->verify_logits + (size_t)trace->n_rounds * T_ROWS * V, lg, sizeof(double) * V);
    dc.margin = INFINITY;
    int32_t k = topk_softmax_gap(lg, V, c->topk, c->temperature, pidx, pp, &gap);
    if (k < 0) st = k;
    else {
      codes[1] = sample_dist(pidx, pp, k, U(uniforms, 1, 2), &dc, 2);
      m_anchor = 1;
      memcpy(hanc, hfin + H, sizeof(double) * H);
      if (rec) { rec->m_new = 1; rec->token = codes[1]; rec->margin = dc.margin; rec->topk_gap = gap; }
    }
    if (rec) trace->n_rounds++;
  }

  while (st == ORC_OK && m_anchor < n) {
    const int mm = m_anchor;
    const int kp = K < n - mm ? K : n - mm;
    const int R = (kp + 1) < (n - mm) ? (kp + 1) : (n - mm);
    dc.margin = INFINITY;
    round_gap = INFINITY;
    rec = NULL;
    if (trace && trace->rounds && trace->n_rounds < trace->max_rounds) {
      rec = &trace->rounds[trace->n_rounds];
      memset(rec, 0, sizeof(*rec));
      rec->m = mm; rec->kp = kp; rec->n_rows = R; rec->token = -1;
    }
    for (int s = 0; s <= mm; ++s) inputs[s] = codes[s];

    /* draft proposal for positions mm+1 .. mm+kp */
    for (int j = 1; j <= kp && st == ORC_OK; ++j) {
      const int t = mm + j;
      if (c->draft_mode == ORC_DRAFT_SELF) {
        /* the target's own distribution at t given c_0..c_mm and d_{mm+1..t-1} */
        for (int s = mm + 1; s < t; ++s) inputs[s] = drafts[s];
        st = orc_forward(m, frame_hidden, inputs, t + 1, hfin);
        if (st == ORC_OK) st = orc_logits(m, hfin + (size_t)t * H, t, 0, lg);
      } else {
        st = orc_logits(m, hanc, t, j, lg);
      }
      if (st != ORC_OK) break;
      if (rec && trace->draft_logits)
        memcpy(trace->draft_logits + ((size_t)trace->n_rounds * T_ROWS + (j - 1)) * V, lg, sizeof(double) * V);
      int32_t k = topk_softmax_gap(lg, V, c->topk, c->temperature, q[t].idx, q[t].p, &gap);
      if (k < 0) { st = k; break; }
      if (gap < round_gap) round_gap = gap;
      if (c->draft_mode == ORC_DRAFT_GREEDY) {
        /* argmax = highest probability, lower index on ties */
        int best = 0;
        for (int r = 1; r < k; ++r)
          if (q[t].p[r] > q[t].p[best]) best = r;
        drafts[t] = q[t].idx[best];
        q[t].idx[0] = drafts[t];
        q[t].p[0] = 1.0;
        q[t].n = 1;
      } else {
        q[t].n = k;
        drafts[t] = sample_dist(q[t].idx, q[t].p, k, U(uniforms, t, 0), &dc, (t - 1) * 3 + 0);
      }
      if (rec) rec->drafts[j - 1] = drafts[t];
    }
    if (st != ORC_OK) break;

    /* verification pass over positions mm+1 .. mm+R, inputs c_mm, d_{mm+1}, ... */
    for (int s = mm + 1; s < mm + R; ++s) inputs[s] = drafts[s];
    st = orc_forward(m, frame_hidden, inputs, mm + R + 1, hfin);
    if (st != ORC_OK) break;
    S.target_calls++;
    S.rounds++;
    S.drafted += kp;

    int m_new = -1, acc = 0;
    for (int j = 1; j <= kp && st == ORC_OK; ++j) {
      const int t = mm + j;
      st = orc_logits(m, hfin + (size_t)t * H, t, 0, lg);
      if (st != ORC_OK) break;
      if (rec && trace->verify_logits)
        memcpy(trace->verify_logits + ((size_t)trace->n_rounds * T_ROWS + (j - 1)) * V, lg, sizeof(double) * V);
      int32_t k = topk_softmax_gap(lg, V, c->topk, c->temperature, pidx, pp, &gap);
      if (k < 0) { st = k; break; }
      if (gap < round_gap) round_gap = gap;
      int32_t tok = -1;
      if (accept_or_resample(pidx, pp, k, q[t].idx, q[t].p, q[t].n, drafts[t], U(uniforms, t, 1),
                             U(uniforms, t, 2), &tok, &dc, t)) {
        codes[t] = drafts[t];
        acc++;
        S.accept_mask |= 1u << t;
      } else {
        codes[t] = tok;
        m_new = t;
        if (rec) rec->token = tok;
        break;
      }
    }
    if (st != ORC_OK) break;
    if (m_new < 0) {
      if (mm + kp < n) {
        /* every draft accepted: one more token from p at mm+kp+1 */
        const int t = mm + kp + 1;
        st = orc_logits(m, hfin + (size_t)t * H, t, 0, lg);
        if (st != ORC_OK) break;
        if (rec && trace->verify_logits)
          memcpy(trace->verify_logits + ((size_t)trace->n_rounds * T_ROWS + kp) * V, lg, sizeof(double) * V);
        int32_t k = topk_softmax_gap(lg, V, c->topk, c->temperature, pidx, pp, &gap);
        if (k < 0) { st = k; break; }
        if (gap < round_gap) round_gap = gap;
        codes[t] = sample_dist(pidx, pp, k, U(uniforms, t, 2), &dc, (t - 1) * 3 + 2);
        if (rec) rec->token = codes[t];
        m_new = t;
      } else {
        m_new = n;
      }
    }
    S.accepted += acc;
    if (m_new < n) memcpy(hanc, hfin + (size_t)m_new * H, sizeof(double) * H);
    if (rec) {
      rec->m_new = m_new;
      rec->accepted = acc;
      rec->margin = dc.margin;
      rec->topk_gap = round_gap;
      trace->n_rounds++;
    }
    m_anchor = m_new;
  }

  if (st == ORC_OK) {
    for (int s = 1; s <= n; ++s) out_codes[s - 1] = codes[s];
    if (stats) *stats = S;
  }
  for (int s = 0; s < MAX_POS; ++s) { free(q[s].idx); free(q[s].p); }
  free(hfin); free(hanc); free(lg); free(pidx); free(pp);
  return st;
}

/* ------------------------------------------------------ sparse-tree frames */

/* depth of every packed row; ORC_EINVAL unless parents precede their children, the
 * packing is breadth-first (depth never decreases) and siblings have distinct ranks */
static int32_t tree_depths(const orc_tree* t, int* depth) {
  if (!t || t->n_nodes < 0 || t->n_nodes > ORC_MAX_TREE) return ORC_EINVAL;
  depth[0] = 0;
  for (int r = 1; r <= t->n_nodes; ++r) {
    const int pr = t->parent[r];
    if (pr < 0 || pr >= r || t->rank[r] < 0) return ORC_EINVAL;
    depth[r] = depth[pr] + 1;
    if (depth[r] < depth[r - 1] || depth[r] > MAX_POS - 1) return ORC_EINVAL;
    for (int q = 1; q < r; ++q)
      if (t->parent[q] == pr && t->rank[q] == t->rank[r]) return ORC_EINVAL;
  }
  return ORC_OK;
}

int32_t orc_tree_mask(const orc_tree* t, int32_t* mask) {
  int depth[ORC_MAX_TREE + 1];
  if (!mask || tree_depths(t, depth) != ORC_OK) return ORC_EINVAL;
  const int n = t->n_nodes + 1;
  for (int i = 0; i < n; ++i) {
    for (int j = 0; j < n; ++j) mask[i * n + j] = 0;
    /* row i, then its parent, up to the root */
    for (int a = i;; a = t->parent[a]) {
      mask[i * n + a] = 1;
      if (a == 0) break;
    }
  }
  return ORC_OK;
}

int32_t orc_tree_hidden(orc_model* m, const orc_tree* t, const float* frame_hidden, const int32_t* committed,
                        int32_t m_anchor, const int32_t* tokens, int32_t n_rows, double* hrows) {
  int depth[ORC_MAX_TREE + 1];
  if (!m || !frame_hidden || !committed || !hrows || n_rows < 1 || tree_depths(t, depth) != ORC_OK ||
      n_rows > t->n_nodes + 1 || m_anchor < 0 || (n_rows > 1 && !tokens))
    return ORC_EINVAL;
  const int H = m->cfg.hidden;
  if (m_anchor + 1 + depth[n_rows - 1] > m->cfg.n_codes) return ORC_EINVAL;
  int done[ORC_MAX_TREE + 1] = {0};
  double* h = (double*)malloc(sizeof(double) * (MAX_POS + 1) * H);
  if (!h) return ORC_ENOMEM;
  int32_t st = ORC_OK;
  /* each row's hidden state is the causal forward over its own path: the committed
   * codes c_0..c_m, then the tokens of its ancestors and itself; one forward per
   * leaf of the rows serves every row on that leaf's path */
  for (int r = n_rows - 1; r >= 0 && st == ORC_OK; --r) {
    if (done[r]) continue;
    int path[MAX_POS];
    int np = 0;
    for (int a = r; a != 0; a = t->parent[a]) path[np++] = a;  /* r, parent, ..., depth-1 row */
    int32_t in[MAX_POS];
    for (int s = 0; s <= m_anchor; ++s) in[s] = committed[s];
    for (int d = 1; d <= np; ++d) in[m_anchor + d] = tokens[path[np - d]];
    st = orc_forward(m, frame_hidden, in, m_anchor + 2 + np, h);
    if (st != ORC_OK) break;
    memcpy(hrows, h + (size_t)(m_anchor + 1) * H, sizeof(double) * H);  /* the root row */
    done[0] = 1;
    for (int d = 1; d <= np; ++d) {
      const int row = path[np - d];
      memcpy(hrows + (size_t)row * H, h + (size_t)(m_anchor + 1 + d) * H, sizeof(double) * H);
      done[row] = 1;
    }
  }
  free(h);
  return st;
}

/* the n largest logits' indices in ranked order: larger value first, ties to the lower index */
static int32_t ranked_candidates(const double* logits, int32_t V, int32_t n, int32_t* out, double* gap, int32_t need) {
  vi_t* a = (vi_t*)malloc(sizeof(vi_t) * V);
  if (!a) return ORC_ENOMEM;
  for (int i = 0; i < V; ++i) {
    a[i].v = isnan(logits[i]) ? -INFINITY : logits[i];
    a[i].i = i;
  }
  qsort(a, (size_t)V, sizeof(vi_t), cmp_desc);
  for (int r = 0; r < n; ++r) out[r] = a[r].i;
  /* smallest gap between consecutive ranks among those that decide a candidate */
  double g = INFINITY;
  for (int r = 0; r < need && r + 1 < V; ++r)
    if (a[r].v - a[r + 1].v < g) g = a[r].v - a[r + 1].v;
  *gap = g;
  free(a);
  return n;
}

int32_t orc_tree_frame(orc_model* m, const orc_tree* t, const float* frame_hidden, int32_t c0, const float* uniforms,
                       int32_t* out_codes, orc_stats* stats, orc_tree_trace* trace, orc_probe_fn probe,
                       void* probe_ctx) {
  int depth[ORC_MAX_TREE + 1];
  if (!m || !frame_hidden || !uniforms || !out_codes || c0 < 0 || c0 >= m->cfg.vocab ||
      tree_depths(t, depth) != ORC_OK)
    return ORC_EINVAL;
  const orc_cfg* c = &m->cfg;
  const int n = c->n_codes, H = c->hidden, V = c->vocab, K = c->draft_len, N = t->n_nodes;
  const int nsup = c->topk < V ? c->topk : V;
  for (int r = 1; r <= N; ++r)
    if (t->rank[r] >= nsup) return ORC_EINVAL; /* every candidate must exist in the draft's support */
  int32_t st = ORC_OK;
  int32_t codes[MAX_POS];
  orc_stats S = {0, 0, 0, 0, 0};
  dctx_t dc = {probe, probe_ctx, INFINITY};
  double* hfin = (double*)malloc(sizeof(double) * (n + 1) * H);
  double* hanc = (double*)malloc(sizeof(double) * H);
  double* hrows = (double*)malloc(sizeof(double) * (N + 1) * H);
  double* lg = (double*)malloc(sizeof(double) * V);
  int32_t* pidx = (int32_t*)malloc(sizeof(int32_t) * V);
  double* pp = (double*)malloc(sizeof(double) * V);
  double* res = (double*)malloc(sizeof(double) * V);
  int32_t* cand = (int32_t*)malloc(sizeof(int32_t) * (MAX_POS) * nsup);
  if (!hfin || !hanc || !hrows || !lg || !pidx || !pp || !res || !cand) st = ORC_ENOMEM;
  double gap = INFINITY;
  codes[0] = c0;
  int m_anchor = 0;
  orc_tree_round* rec = NULL;
  const size_t TR = ORC_MAX_TREE + 1;

  /* prefix pass: positions 0 (frame hidden) and 1 (E_0[c_0]); c_1 from p_1 */
  if (st == ORC_OK) st = orc_forward(m, frame_hidden, codes, 2, hfin);
  if (st == ORC_OK) st = orc_logits(m, hfin + H, 1, 0, lg);
  if (st == ORC_OK) {
    S.target_calls = 1;
    if (trace && trace->rounds && trace->n_rounds < trace->max_rounds) {
      rec = &trace->rounds[trace->n_rounds];
      memset(rec, 0, sizeof(*rec));
      rec->n_rows = 2;
      rec->token = -1;
      rec->tokens[0] = c0;
      if (trace->verify_logits) memcpy(trace->verify_logits + (size_t)trace->n_rounds * TR * V, lg, sizeof(double) * V);
    }
    int32_t k = topk_softmax_gap(lg, V, c->topk, c->temperature, pidx, pp, &gap);
    if (k < 0) st = k;
    else {
      dc.margin = INFINITY;
      codes[1] = sample_dist(pidx, pp, k, U(uniforms, 1, 2), &dc, 2);
      m_anchor = 1;
      memcpy(hanc, hfin + H, sizeof(double) * H);
      if (rec) { rec->m_new = 1; rec->token = codes[1]; rec->margin = dc.margin; rec->topk_gap = gap; trace->n_rounds++; }
    }
  }

  while (st == ORC_OK && m_anchor < n) {
    const int mm = m_anchor;
    const int kp = K < n - mm ? K : n - mm;
    /* candidates: nodes down to depth K'; packed rows: those whose position m + 1 + depth is a
     * code position (a candidate for position n_codes is verified but consumed by no row) */
    int n_cand = 1;
    while (n_cand <= N && depth[n_cand] <= kp) ++n_cand;
    int n_rows = 1;
    while (n_rows < n_cand && mm + 1 + depth[n_rows] <= n) ++n_rows;
    dc.margin = INFINITY;
    double round_gap = INFINITY;
    rec = NULL;
    if (trace && trace->rounds && trace->n_rounds < trace->max_rounds) {
      rec = &trace->rounds[trace->n_rounds];
      memset(rec, 0, sizeof(*rec));
      rec->m = mm; rec->depth = kp; rec->n_rows = n_rows; rec->n_cand = n_cand; rec->token = -1;
    }
    /* draft candidates of every depth, from the anchor's hidden state plus b_d */
    int max_rank[MAX_POS];
    for (int d = 0; d < MAX_POS; ++d) max_rank[d] = -1;
    for (int r = 1; r < n_cand; ++r)
      if (t->rank[r] > max_rank[depth[r]]) max_rank[depth[r]] = t->rank[r];
    for (int d = 1; d <= kp && st == ORC_OK; ++d) {
      st = orc_logits(m, hanc, mm + d, d, lg);
      if (st != ORC_OK) break;
      if (rec && trace->draft_logits)
        memcpy(trace->draft_logits + ((size_t)trace->n_rounds * 16 + (d - 1)) * V, lg, sizeof(double) * V);
      double g;
      const int32_t k = ranked_candidates(lg, V, nsup, cand + (size_t)d * nsup, &g, max_rank[d] + 1);
      if (k < 0) { st = k; break; }
      if (max_rank[d] >= 0 && g < round_gap) round_gap = g;
    }
    if (st != ORC_OK) break;
    int32_t tokens[ORC_MAX_TREE + 1];
    tokens[0] = codes[mm];
    for (int r = 1; r < n_cand; ++r) tokens[r] = cand[(size_t)depth[r] * nsup + t->rank[r]];
    if (rec) memcpy(rec->tokens, tokens, sizeof(int32_t) * n_cand);
    /* verification: every packed row's hidden state under the ancestor mask */
    st = orc_tree_hidden(m, t, frame_hidden, codes, mm, tokens, n_rows, hrows);
    if (st != ORC_OK) break;
    S.target_calls++;
    S.rounds++;
    S.drafted += n_cand - 1;
    if (rec && trace->verify_logits)
      for (int r = 0; r < n_rows && st == ORC_OK; ++r) {
        st = orc_logits(m, hrows + (size_t)r * H, mm + 1 + depth[r], 0, lg);
        memcpy(trace->verify_logits + ((size_t)trace->n_rounds * TR + r) * V, lg, sizeof(double) * V);
      }
    if (st != ORC_OK) break;
    /* walk from the root: children tried in increasing rank under p of the current row */
    int cur = 0, s = mm + 1, acc = 0, m_new = -1;
    while (st == ORC_OK) {
      st = orc_logits(m, hrows + (size_t)cur * H, s, 0, lg);
      if (st != ORC_OK) break;
      const int32_t k = topk_softmax_gap(lg, V, c->topk, c->temperature, pidx, pp, &gap);
      if (k < 0) { st = k; break; }
      if (gap < round_gap) round_gap = gap;
      int kids[ORC_MAX_TREE];
      int nk = 0;
      for (int r = cur + 1; r < n_cand; ++r)
        if (t->parent[r] == cur) {
          int at = nk++;
          while (at > 0 && t->rank[kids[at - 1]] > t->rank[r]) { kids[at] = kids[at - 1]; --at; }
          kids[at] = r;
        }
      int taken = -1;
      if (nk > 0) {
        const double u = U(uniforms, s, 1);
        double bps[ORC_MAX_TREE];
        int nb = 0;
        double cum = 0.0;
        for (int i = 0; i < nk; ++i) {
          cum += prob_of(pidx, pp, k, tokens[kids[i]]);
          if (cum < 1.0) bps[nb++] = cum;
          if (fabs(u - cum) < dc.margin) dc.margin = fabs(u - cum);
          if (taken < 0 && u < cum) taken = kids[i];
        }
        if (dc.fn) dc.fn(dc.ctx, (s - 1) * 3 + 1, bps, nb);
      }
      if (taken >= 0) {
        codes[s] = tokens[taken];
        S.accept_mask |= 1u << s;
        if (rec) rec->path[acc] = taken;
        ++acc;
        cur = taken;
        ++s;
        if (s > n) { m_new = n; break; }
        continue;
      }
      /* no child accepted: the residual p without the children's tokens (p itself if empty) */
      double rs = 0.0;
      for (int j = 0; j < k; ++j) {
        int is_kid = 0;
        for (int i = 0; i < nk; ++i) is_kid |= tokens[kids[i]] == pidx[j];
        res[j] = is_kid ? 0.0 : pp[j];
        rs += res[j];
      }
      if (!(rs > 0.0))
        for (int j = 0; j < k; ++j) res[j] = pp[j];
      codes[s] = sample_dist(pidx, res, k, U(uniforms, s, 2), &dc, (s - 1) * 3 + 2);
      if (rec) rec->token = codes[s];
      m_new = s;
      break;
    }
    if (st != ORC_OK) break;
    S.accepted += acc;
    /* the next anchor's hidden state: the row that produced c_{m_new} */
    if (m_new < n) memcpy(hanc, hrows + (size_t)cur * H, sizeof(double) * H);
    if (rec) {
      rec->m_new = m_new;
      rec->accepted = acc;
      rec->margin = dc.margin;
      rec->topk_gap = round_gap;
      trace->n_rounds++;
    }
    m_anchor = m_new;
  }
  if (st == ORC_OK) {
    for (int s2 = 1; s2 <= n; ++s2) out_codes[s2 - 1] = codes[s2];
    if (stats) *stats = S;
  }
  free(hfin); free(hanc); free(hrows); free(lg); free(pidx); free(pp); free(res); free(cand);
  return st;
}

/* ------------------------------------------------------------- uniforms */

uint64_t orc_splitmix64_at(uint64_t seed, uint64_t n) {
  /* state after n+1 increments of the golden-ratio constant, then the output mix */
  uint64_t z = seed + (n + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

void orc_uniforms_from_seed(uint64_t seed, int32_t n_codes, float* out) {
  for (int i = 0; i < n_codes * 3; ++i)
    out[i] = (float)((double)(orc_splitmix64_at(seed, (uint64_t)i) >> 40) * (1.0 / 16777216.0));
}
