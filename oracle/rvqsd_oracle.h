/* rvqsd_oracle.h -- CPU oracle for RVQ-position-aware speculative decoding.
 *
 * TEST INFRASTRUCTURE. This library is the slow, plain reference that the GPU
 * library is checked against. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load it; the product path never does.
 * It shares no code with the GPU library.
 *
 * What it computes (paper: "RVQ Position Aware Speculative Decoding for On
 * Device Text to Speech"):
 *   - the inner MultiCodeDecoder of Fig. 1: position 0 holds the frame hidden
 *     vector, position s >= 1 consumes code c_{s-1} through its own table
 *     E_{s-1}, and the final hidden state at position s is projected by its own
 *     head LMH_s to emit c_s (Sec. 2.1, "multiheaded by construction");
 *   - plain autoregressive top-k sampling of c_1..c_n (the deployed baseline);
 *   - the speculative frame: drafts for positions k+j from LMH_{k+j}(h_k + b_j)
 *     with K shared offsets b_1..b_K (Sec. 2.2, Fig. 3), one verification pass
 *     over the committed token and the drafts, and the standard speculative
 *     acceptance rule with residual resampling (Sec. 2.2, citing Leviathan et
 *     al. and Chen et al.).
 * All arithmetic is fp64 over the exact weight values stored in the blob.
 */
#ifndef RVQSD_ORACLE_H
#define RVQSD_ORACLE_H
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ORC_OK 0
#define ORC_EINVAL (-1)
#define ORC_EBLOB (-2)
#define ORC_ENOMEM (-3)
#define ORC_ENUMERIC (-6)

/* draft_mode */
#define ORC_DRAFT_SAMPLED 0 /* d ~ q = topk-softmax(LMH_{m+j}(h_m + b_j) / T), with u_draft */
#define ORC_DRAFT_GREEDY 1  /* d = argmax of the draft logits, q = point mass on d */
#define ORC_DRAFT_SELF 2    /* q = the target's own p at m+j (sequential target passes): every draft accepted */

typedef struct {
  int32_t n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn;
  int32_t n_codes;   /* residual codes per frame (15 in the paper) */
  int32_t vocab;     /* codebook size per position */
  int32_t max_draft; /* number of offsets stored in the blob */
  int32_t dtype;     /* matrix storage in the blob: 0 = f32, 1 = bf16, 2 = int8 codes with fp32 row scales */
  int32_t qk_norm;   /* 1: per-head RMSNorm of q and k before RoPE */
  int32_t topk;
  int32_t draft_len; /* K; 0 = plain autoregressive */
  int32_t draft_mode;
  double rms_eps, rope_base, temperature;
} orc_cfg;

typedef struct orc_model orc_model;

typedef struct {
  int32_t target_calls; /* verification passes incl. the 2-token prefix pass */
  int32_t rounds;       /* speculative rounds after the prefix */
  int32_t drafted;      /* sum of K' over rounds */
  int32_t accepted;     /* accepted drafts */
  uint32_t accept_mask; /* bit s set when the draft at position s was accepted */
} orc_stats;

typedef struct {
  int32_t m, kp, n_rows, m_new;
  int32_t drafts[16];   /* d_{m+1} .. d_{m+kp} */
  int32_t accepted;     /* accepted drafts this round */
  int32_t token;        /* resampled / bonus / prefix token committed at m_new, -1 if none */
  double margin;        /* min |u - breakpoint| over the decisions of this round */
  double topk_gap;      /* min gap l_(topk) - l_(topk+1) over the top-k selections of this round */
} orc_round;

typedef struct {
  orc_round* rounds;      /* [max_rounds] */
  double* verify_logits;  /* nullable, [max_rounds][16][vocab]: row r = position m+1+r (prefix: row 0 = position 1) */
  double* draft_logits;   /* nullable, [max_rounds][16][vocab]: j-1 = LMH_{m+j}(h_m + b_j) of the round's anchor */
  int32_t max_rounds;
  int32_t n_rounds;
} orc_trace;

/* Called at each consumption of a pre-drawn uniform: index = (s-1)*3 + slot
 * (slot 0 draft, 1 accept, 2 sample) and the points in [0,1) at which the
 * decision taken with that uniform changes. */
typedef void (*orc_probe_fn)(void* ctx, int32_t uniform_index, const double* breakpoints, int32_t n);

int32_t orc_abi_version(void);
orc_model* orc_create(const orc_cfg* cfg, const void* blob, size_t blob_bytes, int32_t* status);
void orc_destroy(orc_model* m);
void orc_set_threads(int32_t n);
int32_t orc_get_threads(void);

/* Final-normed hidden states h_0..h_{n_pos-1}; in_codes[s-1] is the code
 * consumed at position s (s >= 1). hfin: [n_pos][H]. */
int32_t orc_forward(orc_model* m, const float* frame_hidden, const int32_t* in_codes, int32_t n_pos, double* hfin);

/* The same decoder stack over caller-given input rows (fp64 [n_pos][hidden]) at
 * positions 0..n_pos-1: the outer CodeDecoder of Fig. 1, whose input per frame
 * is a vector, not an embedded code. Final-normed hidden states into hfin. */
#define ORC_MAX_VECTOR_POS 4096
int32_t orc_forward_vectors(orc_model* m, const double* rows, int32_t n_pos, double* hfin);
/* LMH_head (1..n_codes) applied to h (+ b_offset if offset >= 1). out: [vocab]. */
int32_t orc_logits(orc_model* m, const double* h, int32_t head, int32_t offset, double* out);

/* Decision primitives (fp64). Support is returned in ascending token order. */
int32_t orc_topk_softmax(const double* logits, int32_t vocab, int32_t topk, double temperature,
                         int32_t* idx_out, double* prob_out);
int32_t orc_sample(const int32_t* idx, const double* prob, int32_t n, double u);
/* Returns 1 when draft d is accepted, else 0 and *token = residual sample. */
int32_t orc_accept_or_resample(const int32_t* pidx, const double* pp, int32_t np,
                               const int32_t* qidx, const double* qp, int32_t nq,
                               int32_t d, double u_acc, double u_samp, int32_t* token);

/* Plain autoregressive top-k sampling of c_1..c_n (uses u_samp only). uniforms: [n_codes][3]. */
int32_t orc_ar_frame(orc_model* m, const float* frame_hidden, int32_t c0, const float* uniforms, int32_t* out_codes);
/* Speculative frame. trace, probe nullable. */
int32_t orc_spec_frame(orc_model* m, const float* frame_hidden, int32_t c0, const float* uniforms,
                       int32_t* out_codes, orc_stats* stats, orc_trace* trace,
                       orc_probe_fn probe, void* probe_ctx);

/* ---- Sparse-tree verification (Sec. 2.2, "Tree attention increases acceptance rate",
 * Fig. 2) ----
 * A tree of N draft nodes is packed with the committed token's row (the root, row 0)
 * into one query of N + 1 rows, rows 1..N in breadth-first order (depth never
 * decreases). Row r >= 1 holds the token of rank rank[r] among the draft candidates of
 * its depth d: the top-ranked support of q_{m+d} = topk-softmax(LMH_{m+d}(h_m + b_d) / T),
 * shared by every node of that depth. Row r sits at position m + 1 + depth(r) and
 * attends to the committed prefix and to its ancestors (and itself) only.
 * Verification walks the tree from the root: at a node at position s, its children
 * (in increasing rank) are tried in turn under p_s = topk-softmax(LMH_s(h_node) / T),
 * child i accepted iff sum_{l < i} p(x_l) <= u_acc[s] < sum_{l <= i} p(x_l) (the
 * standard rule with a point-mass draft per candidate, each rejection leaving the
 * residual p without that candidate); when no child is accepted, c_s is drawn with
 * u_samp[s] from p with every child's token removed (p itself when nothing is left). */
#define ORC_MAX_TREE 80
typedef struct {
  int32_t n_nodes;                     /* N <= ORC_MAX_TREE */
  int32_t parent[ORC_MAX_TREE + 1];    /* parent row of row r (r >= 1), 0 = the root; parent[r] < r */
  int32_t rank[ORC_MAX_TREE + 1];      /* rank of row r's token among its depth's candidates */
} orc_tree;

typedef struct {
  int32_t m, depth, n_rows, m_new;     /* depth: deepest level drafted this round (K'); n_rows: packed
                                        * rows computed (a candidate at position n_codes + 1 has none) */
  int32_t n_cand;                      /* root + candidate nodes of the round (depth <= K') */
  int32_t accepted, token;             /* accepted nodes; committed residual / bonus / prefix token (-1 none) */
  int32_t tokens[ORC_MAX_TREE + 1];    /* token consumed by each packed row (row 0: c_m) */
  int32_t path[16];                    /* accepted rows, depth 1 .. accepted */
  double margin, topk_gap;
} orc_tree_round;

typedef struct {
  orc_tree_round* rounds;
  double* verify_logits;  /* nullable, [max_rounds][ORC_MAX_TREE + 1][vocab]: LMH_{pos(r)}(h_r) of packed row r */
  double* draft_logits;   /* nullable, [max_rounds][16][vocab]: d-1 = LMH_{m+d}(h_m + b_d) */
  int32_t max_rounds;
  int32_t n_rounds;
} orc_tree_trace;

/* Ancestor mask of the packed query: mask[i][j] = 1 iff row j is row i or an ancestor
 * of it. mask: [(N+1)*(N+1)]. Returns ORC_EINVAL for a tree that is not in packed form. */
int32_t orc_tree_mask(const orc_tree* t, int32_t* mask);
/* Final-normed hidden states of the packed rows for committed codes c_0..c_m
 * (committed[0..m]) and row tokens tokens[1..n_rows-1]: row r at position
 * m + 1 + depth(r) over its own path (the mask's definition). hrows: [n_rows][H]. */
int32_t orc_tree_hidden(orc_model* m, const orc_tree* t, const float* frame_hidden, const int32_t* committed,
                        int32_t m_anchor, const int32_t* tokens, int32_t n_rows, double* hrows);
/* Speculative frame with tree drafting (draft_len = the deepest level K). */
int32_t orc_tree_frame(orc_model* m, const orc_tree* t, const float* frame_hidden, int32_t c0, const float* uniforms,
                       int32_t* out_codes, orc_stats* stats, orc_tree_trace* trace, orc_probe_fn probe,
                       void* probe_ctx);

/* Uniforms from a 64-bit seed with SplitMix64 (Steele, Lea, Flood 2014): the
 * (n+1)-th output of the generator seeded with `seed` gives uniform n, as its
 * top 24 bits times 2^-24. out: [n_codes][3]. */
void orc_uniforms_from_seed(uint64_t seed, int32_t n_codes, float* out);
uint64_t orc_splitmix64_at(uint64_t seed, uint64_t n);

#ifdef __cplusplus
}
#endif
#endif
