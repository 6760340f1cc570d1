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
  const float* rope;  // [kMaxPos][d/2][2] cos, sin of position * rope_base^(-2i/d)
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
};

// Host entry into the kernel translation unit. gp: KParams in device memory.
int launch_frame(const KParams* gp, const FrameArgs& fa, int nwg, int dtype, int mr, void* stream,
                 size_t lds_bytes, char* err, size_t errlen);
int frame_lds_head_floats(int mr, int cpw);
int frame_max_rows(int K);

}  // namespace rvqsd
