/* rvqsd.h -- C ABI of the MI355X (gfx950) library for RVQ-position-aware
 * speculative decoding of the inner MultiCodeDecoder loop.
 *
 * Paper: "RVQ Position Aware Speculative Decoding for On Device Text to
 * Speech". Per 80 ms audio frame, an outer decoder emits the coarse code c_0
 * and an inner decoder emits the 15 residual codes c_1..c_15 one at a time
 * (Fig. 1). This library runs that inner loop speculatively: the model's own
 * per-position heads, fed the anchor hidden state plus a per-distance offset
 * b_j, draft the next K codes (Sec. 2.2, Fig. 3); one verification pass over
 * the committed code and the drafts decides them with the standard
 * speculative acceptance rule and residual resampling, which keeps the output
 * distribution equal to plain top-k sampling (Sec. 2.2, Sec. 3.2).
 *
 * Conventions
 *  - All functions return an rvqsd_status; negative values are errors and
 *    rvqsd_last_error() (thread-local) holds a message. No C++ exception
 *    crosses this boundary.
 *  - "host" pointers are ordinary CPU memory; "device" pointers are HIP
 *    device allocations on the device current when the model was created.
 *  - Codes and positions are int32; activations, logits and probabilities are
 *    fp32 on the device; sampling decisions are taken in fp64.
 *  - Uniform table layout: float[n_codes][3] in [0,1), row s-1 for code
 *    position s, columns (u_draft, u_accept, u_sample).
 */
#ifndef RVQSD_H
#define RVQSD_H
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RVQSD_ABI_VERSION 1

typedef int32_t rvqsd_status;
#define RVQSD_OK 0
#define RVQSD_EINVAL (-1)       /* bad configuration, shape, code value or null pointer */
#define RVQSD_EBLOB (-2)        /* weight blob size / magic / version / shape mismatch */
#define RVQSD_ENOMEM (-3)       /* device or pinned host allocation failed */
#define RVQSD_EHIP (-4)         /* HIP runtime error; message kept in rvqsd_last_error() */
#define RVQSD_EUNSUPPORTED (-5) /* configuration the kernels do not support (see rvqsd_create) */
#define RVQSD_ENUMERIC (-6)     /* every logit of a row was non-finite */
#define RVQSD_ETIMEOUT (-7)     /* a workgroup waited too long for another (kernel exited early) */

#define RVQSD_DTYPE_F32 0
#define RVQSD_DTYPE_BF16 1
/* W8A16 (Sec. 3.4): int8 codes per matrix row followed by the row's fp32 scale
 * (weight = scale * code), zero-padded to 16 bytes; decoded on MFMA with the
 * activations at fp32 accuracy (bf16 hi + lo); draft_len <= 7, single-frame
 * calls and the allocation-free decode only */
#define RVQSD_DTYPE_I8 2

/* Model configuration. The shape fields must equal the weight blob's header. */
typedef struct {
  int32_t abi_version; /* RVQSD_ABI_VERSION */
  int32_t n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn;
  int32_t n_codes;     /* residual codes per frame, 1..15 */
  int32_t vocab;       /* codebook size per position, 2..65536 */
  int32_t max_draft;   /* offsets stored in the blob */
  int32_t dtype;       /* RVQSD_DTYPE_*: storage of the matrices */
  int32_t qk_norm;     /* 1: per-head RMSNorm of q and k before RoPE */
  int32_t topk;        /* 1..256 */
  int32_t draft_len;   /* K, 0..min(max_draft, 14); 0 = plain autoregressive sampling */
  int32_t draft_greedy;/* 0: drafts sampled from the draft distribution; 1: its argmax */
  int32_t matrix_path; /* projections and LM heads of the single-frame kernel: 0 = matrix cores
                        * (MFMA, activations as bf16 hi + lo) for bf16 and int8 weights when a
                        * pass has at most 8 rows, else the VALU GEMV; 1 = the VALU GEMV (bf16
                        * or f32 weights; EUNSUPPORTED for int8). Same results within the
                        * logit tolerance; the choice is a measured one (bench.py --gemv). */
  int32_t reserved[2];
  double rms_eps, rope_base, temperature;
} rvqsd_cfg;

/* One weight blob (host memory): 64-byte header + tensors, layout documented
 * in paper_2609_37007_amd/synth.py. rvqsd_create copies it; the caller keeps
 * ownership and may free it on return. */
typedef struct {
  const void* data;
  uint64_t bytes;
} rvqsd_weights;

/* Per-frame statistics. */
typedef struct {
  int32_t target_calls; /* verification passes including the 2-row prefix pass */
  int32_t rounds;       /* speculative rounds after the prefix pass */
  int32_t drafted;      /* sum over rounds of the drafts verified */
  int32_t accepted;     /* accepted drafts */
  uint32_t accept_mask; /* bit s set when the draft at code position s was accepted */
  int32_t status;       /* device-side status of this frame (RVQSD_OK or an error) */
  uint64_t weight_bytes;/* algorithmic bytes the frame's passes must read (weights + gathered rows + KV) */
  uint64_t clk_start, clk_end; /* device constant clock (100 MHz) at kernel start / end: the frame's
                                * device time in microseconds is (clk_end - clk_start) / 100; every
                                * pass of the frame, the prefix pass included, is a verification pass,
                                * so this is also its verification time */
} rvqsd_stats;

/* Optional per-round trace (device buffers, caller-owned). Any pointer may be NULL.
 *  logits: float[max_rounds][rvqsd_trace_slots(model)][vocab]: slot r < 16 = verify
 *          logits of row r (position first_pos + r), slot 16 + r*K + (j-1) = draft
 *          logits LMH_{s+j}(h_s + b_j) of row r.
 *  rounds: int32[max_rounds][32]: m, K', first_pos, rows, m_new, accepted, token,
 *          pass index, drafts d_{m+1..m+K'} at [8..8+K'), then reserved.
 *  clock:  uint64[max_rounds][5*n_layers+5]: device clock (workgroup 0's view) at the end
 *          of each phase of a pass: per layer QKV, attention, O, gate/up, down at
 *          [5l..5l+4], then the LM heads [5L], sampling [5L+1] and the commit [5L+2],
 *          which ends the pass; the last two entries are unused.
 *  wg_clock: uint64[max_rounds][5*n_layers+5][workgroups]: the same for every workgroup.
 *  wg_ready: uint64[max_rounds][5*n_layers+5][workgroups]: device clock at which each
 *          workgroup held every input of the phase (after its last wait), 0 if it had none. */
typedef struct {
  float* logits;
  int32_t* rounds;
  uint64_t* clock;
  uint64_t* wg_clock;
  int32_t max_rounds;
  uint64_t* wg_ready;
} rvqsd_trace;

typedef struct rvqsd_model rvqsd_model;
typedef struct rvqsd_stream rvqsd_stream;

/* Static information about a created model. */
typedef struct {
  int32_t workgroups;       /* workgroups of the frame kernel (one per compute unit) */
  int32_t threads;          /* threads per workgroup */
  int32_t max_rows;         /* rows per pass the kernel is instantiated for */
  int32_t trace_slots;      /* logit slots per traced round */
  uint64_t lds_bytes;       /* dynamic LDS per workgroup */
  uint64_t layer_weight_bytes; /* bytes of the L decoder layers (matrices + gains) */
  uint64_t head_bytes;      /* bytes of one LM head (vocab x hidden) */
  uint64_t emb_row_bytes;   /* bytes of one embedding row */
  uint64_t device_weight_bytes; /* device memory holding the weights */
} rvqsd_info;

/* Create a model: validates cfg against the blob, copies the weights to the
 * current HIP device. The weights are those of the inner MultiCodeDecoder
 * (Fig. 1): its decoder layers, the per-position code tables E_0..E_{n-1} and
 * LM heads LMH_1..LMH_n (Sec. 2.1), the final norm and the draft offsets
 * b_1..b_max_draft (Sec. 2.2, Fig. 3). Errors: EINVAL (bad cfg / NULL), EBLOB, EUNSUPPORTED
 * (hidden, q/kv width and ffn must be multiples of 512 for bf16 and 256 for
 * f32, head_dim a multiple of 64, n_kv_heads <= 256 workgroups, ...), ENOMEM, EHIP. */
rvqsd_status rvqsd_create(const rvqsd_weights* w, const rvqsd_cfg* cfg, rvqsd_model** out);
void rvqsd_destroy(rvqsd_model* m);
rvqsd_status rvqsd_model_info(const rvqsd_model* m, rvqsd_info* out);

/* Create a decode stream on a caller-owned hipStream_t (borrowed, never
 * destroyed; NULL = the null stream): the state of one frame's speculative
 * rounds (Sec. 2.2), i.e. the KV cache of positions 0..15 and the exchange
 * buffers of the frame kernel. max_streams (1..16) is the number of
 * independent frame streams the batched calls below decode together; with 1
 * only the single-frame calls are available. Batched streams need bf16
 * weights, max_streams * max(draft_len + 1, 2) <= 80 rows, hidden a multiple
 * of 512 (at most 2048) and q width and ffn multiples of 256 (else EUNSUPPORTED).
 * A stream owns its device work buffers and pinned staging; use one host
 * thread per stream. */
rvqsd_status rvqsd_stream_create(rvqsd_model* m, void* hip_stream, int32_t max_streams, rvqsd_stream** out);
void rvqsd_stream_destroy(rvqsd_stream* s);

/* Create a decode stream that verifies a sparse draft tree instead of a chain
 * (Sec. 2.2, "Tree attention increases acceptance rate", Fig. 2). Each round
 * drafts, for every depth d <= min(draft_len, codes left), the candidates of
 * q_{m+d} = topk-softmax(LMH_{m+d}(h_m + b_d) / T) ranked by logit (ties to the
 * lower token); the tree's nodes take the candidates of their depth by rank,
 * shared by every parent. The committed token's row (the root) and the nodes
 * form one query, each row attending to the committed prefix and to its
 * ancestors only; the nodes' children are tried in increasing rank under the
 * target distribution of their parent's row (child i accepted iff
 * sum_{l<i} p(x_l) <= u_accept < sum_{l<=i} p(x_l)), and with none accepted the
 * code is drawn with u_sample from p without the children's tokens. The output
 * distribution stays that of plain top-k sampling.
 * Tree (host arrays, length n_nodes, rows 1..n_nodes of the packed query):
 * parents[i] = parent row of row i+1 (0 = the root, always an earlier row),
 * ranks[i] = candidate rank of row i+1's token (< min(topk, vocab)); rows are
 * packed breadth first (depth never decreases), siblings have distinct ranks,
 * depth <= draft_len. lanes (1..16) frames are decoded together by the batched
 * calls (lanes * (n_nodes + 1) <= 80 rows); the single-frame calls run one frame
 * through the same kernel. Batched traces use round records of 128 ints
 * ([0..7] as a chain round, [8] candidate rows, [16..) accepted rows,
 * [32..) candidate tokens) and logit slots r (verify row r) and
 * max(16, n_nodes + 1) + r*draft_len + j - 1 (draft row (r, j)). Needs bf16
 * weights and the batched stream's shape limits; EINVAL for a malformed tree,
 * EUNSUPPORTED when the rows or their LDS do not fit. */
rvqsd_status rvqsd_tree_stream_create(rvqsd_model* m, void* hip_stream, int32_t lanes, int32_t n_nodes,
                                      const int32_t* parents, const int32_t* ranks, rvqsd_stream** out);

/* Decode one frame (host pointers, synchronous): the inner loop of Fig. 1
 * run speculatively as in Sec. 2.2 and Fig. 3. Position 0 holds frame_hidden
 * (float[hidden], the outer decoder's state), position 1 consumes c0 (in
 * [0, vocab)) through E_0; each round drafts the next K' codes from the
 * anchor's heads LMH_{m+j}(h_m + b_j), verifies them in one pass and keeps
 * them by the acceptance rule with residual resampling (bonus code when all
 * are accepted). Uniforms expanded from rng_seed with SplitMix64 (see
 * rvqsd_uniforms_from_seed). Writes out_codes[n_codes] (codes c_1..c_n) and
 * *out_stats (nullable) only on success. */
rvqsd_status rvqsd_decode_frame(rvqsd_stream* s, const float* frame_hidden, int32_t c0, uint64_t rng_seed,
                                int32_t* out_codes, rvqsd_stats* out_stats);

/* Same with a caller-supplied uniform table (host float[n_codes][3], each in
 * [0, 1): the draft, accept and sample draws of Sec. 2.2 per code position;
 * EINVAL otherwise). */
rvqsd_status rvqsd_decode_frame_u(rvqsd_stream* s, const float* frame_hidden, int32_t c0, const float* uniforms,
                                  int32_t* out_codes, rvqsd_stats* out_stats);

/* rvqsd_decode_frame_u enqueued with device pointers only (the same frame
 * of Sec. 2.2); returns after the launch, the caller synchronises. d_c0:
 * int32[1]; d_uniforms: float[n_codes][3]; d_out_codes: int32[n_codes];
 * d_stats: rvqsd_stats[1] (written by the device; its status field reports
 * device-side errors). A c0 outside [0, vocab) or a uniform outside [0, 1)
 * (NaN included) is found on the device: the frame is not decoded, its status
 * is EINVAL and its codes -1, and the stream stays usable. Inputs must stay
 * valid until the stream reaches the frame. */
rvqsd_status rvqsd_decode_frame_async(rvqsd_stream* s, const float* d_frame_hidden, const int32_t* d_c0,
                                      const float* d_uniforms, int32_t* d_out_codes, rvqsd_stats* d_stats);

/* n frames of one stream in order, as n calls of rvqsd_decode_frame_async would
 * decode them (the same codes and counts; Sec. 2.2 per frame), with up to 1024
 * frames per launch of the persistent kernel, so the GPU does not idle between
 * frames. Device pointers: d_frame_hidden float[n][hidden],
 * d_c0 int32[n], d_uniforms float[n][n_codes][3], d_out_codes out
 * int32[n][n_codes], d_stats out rvqsd_stats[n]. While a trace is set
 * (rvqsd_set_trace), and on a tree stream, every frame gets a launch of its
 * own. EINVAL for a null
 * argument or n < 0; device-side errors as in rvqsd_decode_frame_async, per
 * frame. */
rvqsd_status rvqsd_decode_frames_async(rvqsd_stream* s, int32_t n, const float* d_frame_hidden, const int32_t* d_c0,
                                       const float* d_uniforms, int32_t* d_out_codes, rvqsd_stats* d_stats);

/* rvqsd_decode_frame_async for callers that cannot allocate memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation. It
 * needs no stream object: the frame's device buffers (exchange words, KV cache,
 * parameter block) live in a fixed 16 MiB array of this library on each GPU it
 * runs on, held until the process ends; the call allocates nothing (no
 * hipMalloc, hipFree or allocating library routine) and enqueues two kernels on
 * hip_stream (NULL = the null stream): one that clears that array's frame region
 * and writes the parameter block, then the frame kernel. Arguments and outputs
 * as rvqsd_decode_frame_async (device pointers; d_stats reports device-side
 * errors); the codes equal a fresh stream's. Every call on one GPU shares its
 * array: calls whose work overlaps on that GPU (other streams, other threads)
 * race and must be serialised by the caller. EUNSUPPORTED when the model's frame
 * buffers exceed the array (model info: the 1024-wide 2048-code model needs 5.6
 * MB at draft length 4, 12.8 MB at 14); EINVAL for a null argument or when the
 * current device is not the model's. */
rvqsd_status rvqsd_decode_frame_noalloc(const rvqsd_model* m, void* hip_stream, const float* d_frame_hidden,
                                        const int32_t* d_c0, const float* d_uniforms, int32_t* d_out_codes,
                                        rvqsd_stats* d_stats);

/* Decode n independent frames with max_streams of them in flight (the
 * multi-stream verification of a batch of utterances; each frame is the same
 * problem as rvqsd_decode_frame_u). Frame f runs in lane f % max_streams after
 * frame f - max_streams of that lane; every pass verifies the rows of all
 * lanes at once, so each projection streams its weights once for up to 80 rows
 * and the LM heads serve every lane whose rows need them (Sec. 2.2 applied per
 * lane). Host arrays: frame_hidden float[n][hidden], c0 int32[n], uniforms
 * float[n][n_codes][3]; outputs out_codes int32[n][n_codes], out_stats
 * rvqsd_stats[n] (nullable; weight_bytes = the bytes the frame's passes would
 * read alone). Synchronous. EINVAL for a bad c0, uniform or non-finite input
 * (nothing decoded); device errors: the first frame status that is not OK. */
rvqsd_status rvqsd_decode_frames_batched(rvqsd_stream* s, int32_t n, const float* frame_hidden, const int32_t* c0,
                                         const float* uniforms, int32_t* out_codes, rvqsd_stats* out_stats);

/* Same with device pointers only (same layouts, d_stats required); returns
 * after the launch. A frame whose c0 is out of range or any of whose
 * uniforms lies outside [0, 1) (NaN included) gets status EINVAL and codes -1; after a device-side error every frame not completed gets that
 * error in its status and codes -1. Inputs must stay valid until the stream
 * reaches the launch. */
rvqsd_status rvqsd_decode_frames_batched_async(rvqsd_stream* s, int32_t n, const float* d_frame_hidden,
                                               const int32_t* d_c0, const float* d_uniforms, int32_t* d_out_codes,
                                               rvqsd_stats* d_stats);

/* Install (logits or rounds non-NULL) or remove (both NULL) a per-frame trace of
 * the later batched calls of a stream created with max_streams >= 2: frame f <
 * max_frames of a call, pass (prefix = 0) < max_rounds of that frame. Device
 * buffers, caller-owned, layouts as the single-frame trace of rvqsd_set_trace
 * with a leading frame index: logits float[max_frames][max_rounds]
 * [rvqsd_info.trace_slots][vocab] (slot r < 16 = verify row r, 16 + r*K + j-1 =
 * draft row (r, j)); rounds int32[max_frames][max_rounds][32]. Only the slots a
 * pass uses are written. Synchronises the stream. EINVAL: max_rounds or
 * max_frames < 1 with a buffer; EUNSUPPORTED: a single-frame stream. */
rvqsd_status rvqsd_set_batch_trace(rvqsd_stream* s, float* logits, int32_t* rounds, int32_t max_rounds,
                                   int32_t max_frames);

/* Passes run by the last batched call of the stream and their algorithmic
 * bytes (layer weights and each LM head used, once per pass; gathered rows;
 * KV cache read). Synchronises the stream. */
rvqsd_status rvqsd_batch_totals(rvqsd_stream* s, uint64_t* passes, uint64_t* bytes);

/* ---- Outer CodeDecoder step and the full per-frame pipeline (Fig. 1) ----
 * The outer decoder emits c_0 once per frame from an input vector that adds the
 * frame's text-side vector t and the embeddings of the previous frame's 16
 * codes; its final-normed hidden state is the inner loop's frame_hidden.
 * outer_model: a model created with rvqsd_create from the outer decoder's blob
 * (same block layout; n_codes = 1: its E_0 table over the outer codebook and its
 * head; max_draft = draft_len = 0). code_tables: host, [n_tables][table_vocab]
 * [hidden] bf16, the embeddings of codes 1..n_tables (copied). c_0 is a top-k,
 * temperature-T draw over the first min(outer vocab, table_vocab) logits (the
 * codes the inner model can embed). max_frames (<= 4096) bounds the KV cache,
 * which grows by one position per frame until rvqsd_outer_reset. bf16 only,
 * hidden a multiple of 512 (<= 2048), q width and ffn multiples of 256. */
typedef struct rvqsd_outer rvqsd_outer;
rvqsd_status rvqsd_outer_create(rvqsd_model* outer_model, const void* code_tables, int32_t n_tables,
                                int32_t table_vocab, int32_t topk, double temperature, int32_t max_frames,
                                rvqsd_outer** out);
void rvqsd_outer_destroy(rvqsd_outer* o);
/* Next frame is position 0 again (no previous codes). Call when the stream is idle. */
rvqsd_status rvqsd_outer_reset(rvqsd_outer* o);

/* Enqueue n frames of the full pipeline on the inner stream s (device pointers,
 * returns after the launches): per frame one outer step (c_0 and the hidden
 * state) and one inner frame decode (c_1..c_15), chained on the device with no
 * host synchronisation. d_t float[n][hidden] (16-byte aligned, else EINVAL);
 * d_u_c0 float[n] (uniform of each c_0 draw); d_uniforms float[n][n_codes][3]
 * (inner uniforms); d_codes out int32[n][1 + n_codes] (c_0, c_1..c_n); d_stats
 * out rvqsd_stats[n] (inner loop; an outer-step error shows as c_0 = -1 and
 * status EINVAL); d_hidden out float[n][hidden] or NULL. The outer tables must
 * match the inner model (n_tables = n_codes, table_vocab = vocab); EUNSUPPORTED
 * beyond max_frames. */
rvqsd_status rvqsd_pipeline_frames_async(rvqsd_stream* s, rvqsd_outer* o, int32_t n, const float* d_t,
                                         const float* d_u_c0, const float* d_uniforms, int32_t* d_codes,
                                         rvqsd_stats* d_stats, float* d_hidden);

/* Return a stream to its initial state. Needed after a frame enqueued with
 * rvqsd_decode_frame_async reported a device-side error other than EINVAL in
 * its stats (later frames on the stream then fail with RVQSD_EHIP until the
 * reset); the synchronous calls reset by themselves. Synchronises the stream. */
rvqsd_status rvqsd_stream_reset(rvqsd_stream* s);

/* Install (trace != NULL) or remove (NULL) a per-round trace for later frames
 * of this stream (layouts at rvqsd_trace): the verify logits LMH_s(h_s) and the
 * draft logits LMH_{s+j}(h_s + b_j) of every row of every pass, and the round
 * records (anchor, drafts, accepted count, committed token) of the speculative
 * rounds of Sec. 2.2; the buffers stay the caller's. Synchronises the stream.
 * EINVAL for a NULL stream or max_rounds < 0. */
rvqsd_status rvqsd_set_trace(rvqsd_stream* s, const rvqsd_trace* trace);

/* The library's uniform generator (host only): uniform i = (n_codes*3 table
 * order) is the top 24 bits of the (i+1)-th SplitMix64 output (Steele, Lea,
 * Flood 2014) for the given seed, times 2^-24. out: float[n_codes][3]. */
rvqsd_status rvqsd_uniforms_from_seed(uint64_t seed, int32_t n_codes, float* out);

const char* rvqsd_status_str(rvqsd_status st);
const char* rvqsd_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
