// rvqsd_internal.h -- launch parameters shared by the host runtime and the frame kernel.
#pragma once
#include <stdint.h>

#include "../../include/rvqsd.h"

namespace rvqsd {

constexpr int kThreads = 512;          // threads per workgroup (8 wave64s)
constexpr int kWaves = kThreads / 64;
constexpr int kMaxCodes = 15;          // residual codes per frame (positions 1..15)
constexpr int kMaxPos = 16;            // positions 0..15
constexpr int kMaxRows = 16;           // rows of one pass (K+1 <= 15, prefix 2)
constexpr int kSlotDraft0 = kMaxRows;  // logit slot of the first draft row
constexpr int kMaxTopk = 256;
constexpr int kTraceRoundInts = 32;    // ints per traced round
constexpr int kTopkCand = 64;          // values the boundary bucket of the bucket top-k may hold
constexpr int kTopkBuckets = 1024;     // value buckets of the bucket top-k
// MFMA path (bf16 weights, <= 8 rows per pass): 512-wide k units per wave, i.e.
// the largest hidden, q width and FFN it takes are 512 times these.
constexpr int kUptH = 2, kUptQ = 4, kUptF = 6;

// Phase ids inside a pass (tag = epoch_base + pass * phases_per_pass + phase + 1).
constexpr int kPhQKV = 0, kPhAttn = 1, kPhO = 2, kPhGU = 3, kPhDown = 4;  // + 5 * layer
inline __host__ __device__ int phases_per_pass(int L) { return 5 * L + 4; }
inline __host__ __device__ int ph_heads(int L) { return 5 * L; }
inline __host__ __device__ int ph_sample(int L) { return 5 * L + 1; }

struct KParams {
  // model dimensions
  int32_t L, H, nq, nkv, d, F, n_codes, V, K, topk, greedy, qk_norm, max_draft;
  int32_t qdim, kvdim, nqkv;
  float rms_eps;
  double temperature, rope_base;
  int32_t nwg;          // workgroups in the launch
  int32_t stage_cols;   // floats per activation row that fit the LDS staging area
  // weights: one device buffer holding the blob payload (header stripped), byte offsets
  const uint8_t* wbase;
  uint64_t layer_stride;
  uint64_t o_attn_norm, o_wq, o_wk, o_wv, o_qn, o_kn, o_wo, o_mlp_norm, o_wg, o_wu, o_wd;  // inside a layer
  uint64_t o_final_norm, o_emb0, o_lmh1, o_offsets, table_stride;                      // global
  uint64_t emb_row_bytes;  // bytes read to gather one embedding row (int8: codes and the row scale)
  // activation exchange buffers: fp32 bit patterns whose lowest mantissa bit
  // carries the parity of the write epoch (every epoch rewrites every word)
  uint32_t* xb;    // [kMaxRows][H]      residual stream (parity 0 after O, 1 after down)
  uint32_t* qkvb;  // [kMaxRows][nqkv]   q | k | v
  uint32_t* attnb; // [kMaxRows][qdim]   attention output
  uint32_t* actb;  // [kMaxRows][F]      SiLU(gate) * up
  uint32_t* pass_count;  // passes run by this stream so far (0xffffffff: poisoned by an error)
  // tagged 64-bit words: high 32 bits = tag, low 32 bits = payload
  uint64_t* logb;  // [2][n_slots][V]    verify + draft logits (by pass parity)
  uint64_t* vres;  // [2][kMaxRows]      verify results (accept flag | token)
  uint64_t* drec;  // [2][n_slots][drec_words] draft records: token, then (idx, prob lo, prob hi) x support
  int32_t n_slots, drec_words;
  float* kvc;      // [nq][L][kMaxPos][2][d] KV cache of each attention workgroup (k after norm and RoPE, v)
  const float* rope;  // [kMaxPos][d/2][2] cos, sin of position * rope_base^(-2i/d) (held by the model)
  int32_t work_floats;  // floats of the LDS work area (the attention constants follow it)
  uint64_t* status; // device status word: (epoch_base << 32) | error code of that frame
  // trace (nullable)
  float* tr_logits;    // [tr_max_rounds][n_slots][V]
  int32_t* tr_rounds;  // [tr_max_rounds][kTraceRoundInts]
  uint64_t* tr_clock;  // [tr_max_rounds][phases_per_pass + 1]
  uint64_t* tr_wgclock;  // [tr_max_rounds][phases_per_pass + 1][nwg]
  uint64_t* tr_wgready;  // [tr_max_rounds][phases_per_pass + 1][nwg] input-complete time
  int32_t tr_max_rounds;
};

// Per-frame arguments, passed by value at each launch (device pointers).
struct FrameArgs {
  const float* frame_hidden;  // [H]
  const int32_t* c0;          // [1]
  const float* uniforms;      // [n_codes][3]
  int32_t* out_codes;         // [n_codes]
  rvqsd_stats* out_stats;     // [1]
  uint32_t epoch_base;        // tags of this frame are epoch_base + 1 ..
  // frames of one launch: frame f reads and writes each array above at f times its frame
  // stride and tags from epoch_base + f * epoch_step; fbar counts arrivals between frames
  // (cleared before a launch of more than one frame)
  int32_t n_frames;
  uint32_t epoch_step;
  uint32_t* fbar;
};

// Device buffers of one frame decode (the exchange words, the KV cache and the
// parameter block), laid out from one base address:
//   parity words (x, q/k/v, attention output, activation; initialised to parity 1) |
//   pass count | tagged words (logits, verdicts, draft records, status; cleared to
//   tag 0) | KV cache | parameter block. A decode stream owns one such region; the
//   allocation-free entry point places it in a fixed device array.
struct FrameLayout {
  size_t o_x, o_qkv, o_attn, o_act;  // parity words
  size_t par_begin, par_end;
  size_t o_pc;                       // pass count
  size_t o_log, o_vres, o_drec, o_status;  // tagged words
  size_t tag_begin, tag_end;
  size_t o_kvc, o_kp;
  size_t bytes;                      // total, 256-byte aligned
  int32_t n_slots, drec_words;
};

inline FrameLayout frame_layout(const KParams& k) {
  FrameLayout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += (bytes + 255) & ~(size_t)255;
    return at;
  };
  L.n_slots = kSlotDraft0 + kMaxRows * k.K;
  L.drec_words = 1 + 3 * kMaxTopk;
  const size_t H = (size_t)k.H, V = (size_t)k.V;
  L.par_begin = off;
  L.o_x = take(kMaxRows * H * 4);
  L.o_qkv = take((size_t)kMaxRows * k.nqkv * 4);
  L.o_attn = take((size_t)kMaxRows * k.qdim * 4);
  L.o_act = take((size_t)kMaxRows * k.F * 4);
  L.par_end = off;
  L.o_pc = take(4);
  L.tag_begin = off;
  L.o_log = take((size_t)2 * L.n_slots * V * 8);
  L.o_vres = take((size_t)2 * kMaxRows * 8);
  L.o_drec = take((size_t)2 * L.n_slots * L.drec_words * 8);
  L.o_status = take(8);
  L.tag_end = off;
  L.o_kvc = take((size_t)k.nq * k.L * kMaxPos * 2 * k.d * 4);
  L.o_kp = take(sizeof(KParams));
  L.bytes = off;
  return L;
}

// Point the buffer fields of k into the region at base (device address).
inline void frame_bind(KParams* k, uint8_t* base, const FrameLayout& L) {
  k->n_slots = L.n_slots;
  k->drec_words = L.drec_words;
  k->xb = (uint32_t*)(base + L.o_x);
  k->qkvb = (uint32_t*)(base + L.o_qkv);
  k->attnb = (uint32_t*)(base + L.o_attn);
  k->actb = (uint32_t*)(base + L.o_act);
  k->pass_count = (uint32_t*)(base + L.o_pc);
  k->logb = (uint64_t*)(base + L.o_log);
  k->vres = (uint64_t*)(base + L.o_vres);
  k->drec = (uint64_t*)(base + L.o_drec);
  k->status = (uint64_t*)(base + L.o_status);
  k->kvc = (float*)(base + L.o_kvc);
}

// Frame tags step per frame: enough for every pass and phase of one frame.
inline uint32_t frame_epoch_step(int L) {
  const int tags_per_frame = kMaxPos * phases_per_pass(L) + 2;
  return (uint32_t)((tags_per_frame + 4095) & ~4095);
}

// Record st and msg as the calling thread's last error (rvqsd_last_error); returns st.
int set_last_error(int st, const char* msg);

// Host entry into the kernel translation unit. gp: KParams in device memory.
int launch_frame(const KParams* gp, const FrameArgs& fa, int nwg, int dtype, int mr, bool mfma, void* stream,
                 size_t lds_bytes, char* err, size_t errlen);

// ---------------------------------------------------------------- batched path
// Independent frame streams ("lanes") verified together: lane i owns rows
// i * rpl .. i * rpl + rpl - 1 of every pass (rpl = max(K + 1, 2)), so a
// projection multiplies M = lanes * rpl rows at once on MFMA tiles.
constexpr int kMaxLanes = 16;
constexpr int kOutOSplit = 4, kOutDSplit = 3;  // k splits of the outer step's O and down projections
constexpr int kBatchMaxRows = 80;  // lanes * rpl: five 16-row MFMA tiles
constexpr int kBatchMTiles = kBatchMaxRows / 16;
constexpr int kBatchRedFloats = 16 * kBatchMTiles * 256;  // LDS partial tiles of one MFMA unit (k parts x n-tiles)
// lane state record (int32 words)
constexpr int kLnActive = 0, kLnFrame = 1, kLnPass = 2, kLnM = 3, kLnKp = 4, kLnFirst = 5, kLnRows = 6,
              kLnPrevAnchor = 7, kLnCalls = 8, kLnRounds = 9, kLnDrafted = 10, kLnAccepted = 11, kLnMask = 12,
              kLnStatus = 13, kLnBytesLo = 14, kLnBytesHi = 15, kLnClkLo = 16, kLnClkHi = 17,
              kLnCandN = 18,  // tree lanes: candidate rows of the pass (root + nodes down to depth K')
              kLnCodes = 32, kLnDrafts = 48, kLnInCode = 64,
              kLnCand = 80,   // tree lanes: token of every candidate row (row 0: the committed c_m)
              kLaneInts = kLnCand + kBatchMaxRows + 16;
// sparse-tree lanes: a tree of up to kBatchMaxRows - 1 draft nodes per lane
constexpr int kMaxTreeRows = kBatchMaxRows;
constexpr int kTreeRoundInts = 128;  // ints per traced round of a tree lane

struct BParams {
  const KParams* k;     // device copy of the stream's parameter block (dimensions, weights, rotary table)
  int32_t lanes, rpl, M, nwg;
  // sparse-tree verification (Sec. 2.2, Fig. 2): every lane's rows after its prefix pass are
  // the committed token's row (the root) and a draft tree packed breadth first; rpl = nodes + 1
  int32_t tree;         // 0: chain rows (the committed code and K drafts), 1: tree rows
  int32_t tree_nodes;
  int32_t kv_slots;     // KV slots per (lane, layer, kv head): committed positions, then the pass's rows
  int32_t slot_draft0;  // first draft slot of the trace layout (16 for chains, max(16, rpl) for trees)
  int32_t t_parent[kMaxTreeRows];   // row r >= 1: parent row
  int32_t t_rank[kMaxTreeRows];     // row r >= 1: rank of its token among its depth's candidates
  int32_t t_depth[kMaxTreeRows];    // row 0: 0
  uint64_t t_anc[kMaxTreeRows][2];  // ancestor-or-self bits of row r over rows 0..127
  int32_t t_need[kMaxCodes + 1];    // depth d: candidates to rank (largest rank at d plus one)
  int32_t ks_qkv, ks_o, ks_down;  // k splits of the projections whose partial sums the next phase adds
  int32_t hrows;        // LM-head input rows: M * (K + 1) (row i * (K + 1) + j: row i plus offset b_j)
  int32_t sup_words;    // 64-bit words of one support record: 1 + 2 * topk
  int32_t* lane;        // [lanes][kLaneInts]
  float* x;             // [M][H] residual stream
  uint32_t* a;          // [M][max(H, qdim, F)] split activations (8-element chunks: 4 words hi, 4 words lo)
  uint32_t* ah;         // [hrows][H] split LM-head inputs
  float* part;          // [max ks][M][max N] partial sums
  float* kv;            // [lanes][L][nkv][kv_slots][2][d] KV cache (k after norm and RoPE, v)
  float* logits;        // [hrows][V]
  int32_t* vres;        // [lanes][rpl] verdicts: token | accepted << 31 (chain); token | (child row + 1) << 24 (tree)
  uint64_t* drec;       // [2][lanes][rpl][K][sup_words] draft records: token, idx[topk], prob bits[topk]
                        // (tree lanes: count, then the ranked candidate tokens)
  uint32_t* bar;        // barrier words: [0] top counter, [64 (1 + x)] counter of XCD x, [64 * 9] generation
  int32_t* status;      // first device-side error of the launch (0 = none)
  unsigned long long* totals;  // [0] passes (rounds of the batch), [1] their algorithmic bytes
  // per-frame trace (nullable), frames f < tr_frames of a call, passes < tr_max_rounds of the frame:
  // logits in the single-stream slot layout, round records as the single-stream trace's
  float* tr_logits;     // [tr_frames][tr_max_rounds][n_slots][V]
  int32_t* tr_rounds;   // [tr_frames][tr_max_rounds][kTraceRoundInts] (tree lanes: kTreeRoundInts)
  int32_t tr_max_rounds, tr_frames, tr_slots;
};

// Per-call arguments (device pointers), passed by value.
struct BCall {
  const float* frame_hidden;  // [n][H]
  const int32_t* c0;          // [n]
  const float* uniforms;      // [n][n_codes][3]
  int32_t* out_codes;         // [n][n_codes]
  rvqsd_stats* out_stats;     // [n]
  int32_t n;
};

int launch_batch(const BParams* bp, const BCall& call, int nwg, void* stream, size_t lds_bytes, bool tree,
                 char* err, size_t errlen);

// ---------------------------------------------------------------- outer decoder step
// The outer CodeDecoder of the per-frame pipeline: one position per frame, a KV
// cache that grows across frames, c_0 sampled from its head.
constexpr int kAttnChunks = 16;       // key chunks per query head the split aims for (split-sequence attention)
constexpr int kAttnKVFloats = 32768;  // LDS floats for one chunk's keys and values (128 KB)
constexpr int kMaxOuterFrames = 4096; // KV capacity of the outer decoder at most
constexpr int kAttnMaxChunks = 64;    // chunks per head at most: 4096 positions in chunks of >= 64 (head_dim <= 256)
// Key positions per chunk when np positions are attended: about np / kAttnChunks,
// at most what kAttnKVFloats holds for keys and values of head dimension d.
constexpr int attn_chunk_len(int np, int d) {
  return (np + kAttnChunks - 1) / kAttnChunks < kAttnKVFloats / (2 * d) ? (np + kAttnChunks - 1) / kAttnChunks
                                                                       : kAttnKVFloats / (2 * d);
}

struct OParams {
  const KParams* k;      // the outer model's parameter block (dimensions, weights)
  int32_t nwg, M;        // M = 1 row
  int32_t ks_qkv, ks_o, ks_down;
  int32_t n_tables, table_vocab, max_frames, topk;
  double temperature;
  const uint16_t* tables;  // [n_tables][table_vocab][H] bf16: embeddings of codes 1..n_tables
  const float* rope;     // [max_frames][d/2][2] cos, sin of position * rope_base^(-2i/d)
  float* x;              // [H] residual stream
  uint32_t* a;           // [2][max(H, qdim, F)] split activations
  float* part;           // [max ks][max N] partial sums
  float* kv;             // [L][nkv][max_frames][2][d] KV cache (k after norm and RoPE, v)
  float* apart;          // [nq][kAttnMaxChunks][d + 2] per-chunk attention partials (max, sum, o)
  float* logits;         // [V]
  uint32_t* bar;         // grid barrier words
  int32_t* status;       // first device-side error of the step (0 = none)
  // tagged exchange words of the step without grid barriers (upper 32 bits: the tag of the write),
  // one set per layer
  uint64_t* tq;          // [L][nqkv] QKV outputs
  uint64_t* tch;         // [L][nq][kAttnMaxChunks][d + 2] attention chunk partials (max, sum, o)
  uint64_t* tat;         // [L][qdim] merged attention output
  uint64_t* top;         // [L][kOutOSplit][H] O partial sums
  uint64_t* tact;        // [L][F] SwiGLU activations
  uint64_t* tdp;         // [L][kOutDSplit][H] down partial sums
  uint64_t* tlog;        // [V] head logits
  int32_t xoff;          // float offset in dynamic LDS of the residual row every workgroup keeps
  int32_t ks_o2, ks_d2;  // k splits of its O and down projections (<= kOutOSplit, kOutDSplit)
};

// Per-step arguments (device pointers), passed by value.
struct OCall {
  const float* t;            // [H] this frame's text-side input vector
  const float* u_c0;         // [1] uniform of the c_0 draw
  const int32_t* prev_codes; // [1 + n_tables] codes of the previous frame (nullptr at position 0)
  int32_t* c0_out;           // [1] sampled c_0 (-1 after a device error)
  float* hidden_out;         // [H] final-normed hidden state (the inner loop's frame input)
  int32_t pos;               // position = frame index since the last reset
  uint32_t epoch;            // launch counter of this outer step object (tags its exchange words)
};

// flow_steps 0: the step with a grid barrier between phases; 1 .. kFlowSteps: the step without
// grid barriers, whose units hold up to flow_steps 64-wide k steps per wave of weights in registers
// (k ranges up to 512 kFlowSteps)
constexpr int kFlowSteps = 2;
int launch_outer(const OParams* op, const OCall& call, int nwg, void* stream, size_t lds_bytes, int flow_steps,
                 char* err, size_t errlen);
int frame_lds_head_floats(int mr, int cpw);
int frame_max_rows(int K);

}  // namespace rvqsd

// A created model (host object behind the opaque rvqsd_model handle).
struct rvqsd_model {
  rvqsd_cfg cfg;
  int device;
  int nwg;
  int mr;               // rows the frame kernel is instantiated for
  bool mfma;            // projections and heads on the matrix cores (else the VALU GEMV)
  int wbytes;           // bytes per matrix element
  size_t lds_bytes;
  int stage_cols;
  void* dweights;       // the blob payload, then the rotary table
  uint64_t dweight_bytes;
  size_t frame_bytes;   // device buffers of one frame decode (FrameLayout::bytes)
  rvqsd::KParams base;  // dimensions, weight offsets and the rotary table; buffers are set per decode region
};
