// rvqsd_api.cpp -- host runtime behind the C ABI declared in include/rvqsd.h.
//
// Owns the device copy of the weights (the blob payload, header stripped, so
// every tensor starts 16-byte aligned), the per-stream exchange buffers and
// the launch of the persistent frame kernel. No exception crosses the ABI.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>

#include "../../include/rvqsd.h"
#include "rvqsd_internal.h"

using namespace rvqsd;

namespace {

thread_local char g_err[512] = "";

int set_err(int st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

#define HIPCHK(expr)                                                                     \
  do {                                                                                   \
    hipError_t e_ = (expr);                                                              \
    if (e_ != hipSuccess) return set_err(RVQSD_EHIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

uint32_t rd32(const unsigned char* p) {
  return (uint32_t)p[0] | ((uint32_t)p[1] << 8) | ((uint32_t)p[2] << 16) | ((uint32_t)p[3] << 24);
}

uint64_t splitmix64_at(uint64_t seed, uint64_t n) {
  uint64_t z = seed + (n + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Allocation failures can be injected by tests: RVQSD_TEST_FAIL_ALLOC=n fails the n-th device
// allocation counted from the moment the variable took its current value.
int g_alloc_count = 0;
char g_alloc_env[32] = "";
hipError_t dev_alloc(void** p, size_t bytes) {
  const char* f = getenv("RVQSD_TEST_FAIL_ALLOC");
  if (f) {
    if (strncmp(f, g_alloc_env, sizeof(g_alloc_env) - 1) != 0) {
      snprintf(g_alloc_env, sizeof(g_alloc_env), "%s", f);
      g_alloc_count = 0;
    }
    if (atoi(f) == ++g_alloc_count) {
      *p = nullptr;
      return hipErrorOutOfMemory;
    }
  } else {
    g_alloc_env[0] = '\0';
  }
  return hipMalloc(p, bytes);
}

}  // namespace

int rvqsd::set_last_error(int st, const char* msg) { return set_err(st, "%s", msg); }

struct rvqsd_stream {
  rvqsd_model* m;
  hipStream_t stream;
  KParams kp;           // host copy of the parameter block
  KParams* dkp;         // device copy
  void* dbuf;           // all exchange buffers in one allocation
  size_t dbuf_bytes;
  uint64_t* status;
  // synchronous-path staging
  float* h_in;          // pinned: frame hidden [H], uniforms [n][3], c0 (as int bits)
  int32_t* h_out;       // pinned: codes [n], then stats
  float* d_in;
  int32_t* d_out;
  uint32_t epoch;       // tag base of the next frame
  uint32_t epoch_step;
  uint32_t* fbar;       // arrivals between the frames of one launch (in dbuf)
  size_t par_begin, par_end;  // byte range of dbuf holding the parity-word buffers (pass count follows)
  size_t tag_begin, tag_end;  // byte range of dbuf holding the tagged words
  // batched path (max_streams > 1)
  int lanes;            // frame streams decoded together
  int tree;             // 1: every lane verifies a sparse draft tree (the batched kernel's tree rows)
  void* bbuf;           // batched work buffers; the barrier, status and totals words come first
  size_t bsync_bytes;   // bytes of those words (cleared before every launch)
  BParams bp;           // host copy of the batched parameter block
  BParams* dbp;         // device copy
  size_t blds;          // dynamic LDS of the batched kernel
  void* bstage;         // device staging of the synchronous batched call
  size_t bstage_bytes;
};

struct rvqsd_outer {
  rvqsd_model* m;       // the outer decoder (blob with one code table and one head)
  void* buf;            // device buffers and parameter blocks
  OParams op;           // host copy
  OParams* dop;         // device copy
  KParams* dkp;         // device copy of the outer model's parameter block
  int32_t* last_codes;  // device [1 + n_tables]: codes of the last frame of the previous call
  float* f;             // device [H]: hidden state handed to the inner loop when the caller keeps none
  size_t sync_bytes;    // barrier and status words at the start of buf
  size_t lds;
  int pos;              // frames decoded since the last reset
  int n_tables;
  uint32_t epoch;       // launches so far (tags the exchange words of the step without grid barriers)
  int flow_steps;       // > 0: the step without grid barriers, its units' k steps per wave
};

namespace {

int validate_cfg(const rvqsd_cfg* c, int nwg) {
  if (c->abi_version != RVQSD_ABI_VERSION)
    return set_err(RVQSD_EINVAL, "abi_version %d, library is %d", c->abi_version, RVQSD_ABI_VERSION);
  if (c->n_layers <= 0 || c->hidden <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0 ||
      c->ffn <= 0 || c->n_codes < 1 || c->n_codes > kMaxCodes || c->vocab < 2 || c->max_draft < 0 ||
      c->topk < 1 || c->draft_len < 0 || c->draft_len > c->max_draft || !(c->temperature > 0.0) ||
      !(c->rms_eps > 0.0) || !(c->rope_base > 0.0) || (c->dtype < RVQSD_DTYPE_F32 || c->dtype > RVQSD_DTYPE_I8) ||
      (c->n_q_heads % c->n_kv_heads) != 0 || (c->qk_norm != 0 && c->qk_norm != 1) ||
      (c->draft_greedy != 0 && c->draft_greedy != 1) || (c->matrix_path != 0 && c->matrix_path != 1))
    return set_err(RVQSD_EINVAL, "invalid configuration field");
  if (c->dtype == RVQSD_DTYPE_I8 && c->matrix_path == 1)
    return set_err(RVQSD_EUNSUPPORTED, "int8 weights run on the matrix cores only (matrix_path 0)");
  const int epc = c->dtype == RVQSD_DTYPE_F32 ? 4 : 8;
  const int qd = c->n_q_heads * c->head_dim;
  const int quant = 64 * epc;
  if (c->hidden % quant || qd % quant || c->ffn % quant)
    return set_err(RVQSD_EUNSUPPORTED, "hidden, n_q_heads*head_dim and ffn must be multiples of %d", quant);
  if (c->hidden / epc > kThreads || qd / epc > kThreads || c->ffn / epc > kThreads)
    return set_err(RVQSD_EUNSUPPORTED, "a reduction dimension exceeds %d elements", kThreads * epc);
  // every workgroup must take part in every full-activation phase (parity exchange)
  if (c->hidden % nwg || (qd + 2 * c->n_kv_heads * c->head_dim) < nwg || c->ffn < nwg)
    return set_err(RVQSD_EUNSUPPORTED, "hidden must be a multiple of, and q/k/v width and ffn at least, %d", nwg);
  if (c->head_dim % 64 || c->head_dim > 256) return set_err(RVQSD_EUNSUPPORTED, "head_dim must be 64, 128, 192 or 256");
  if (c->topk > kMaxTopk) return set_err(RVQSD_EUNSUPPORTED, "topk > %d", kMaxTopk);
  if (c->vocab > 16384) return set_err(RVQSD_EUNSUPPORTED, "vocab > 16384");
  if (c->draft_len > 14) return set_err(RVQSD_EUNSUPPORTED, "draft_len > 14");
  if (c->n_q_heads > nwg) return set_err(RVQSD_EUNSUPPORTED, "more query heads than workgroups");
  if (kSlotDraft0 + (c->draft_len + 1) * c->draft_len > nwg)
    return set_err(RVQSD_EUNSUPPORTED, "not enough workgroups for the sampling slots");
  if ((c->hidden + nwg - 1) / nwg > 32) return set_err(RVQSD_EUNSUPPORTED, "hidden > 32 * workgroups");
  return RVQSD_OK;
}

// Work-area floats needed by every phase for a given staging width.
size_t work_floats(const rvqsd_cfg* c, int nwg, int mr, bool mfma, int stage_cols) {
  const int H = c->hidden, qd = c->n_q_heads * c->head_dim, kd = c->n_kv_heads * c->head_dim, F = c->ffn;
  const int V = c->vocab, d = c->head_dim, K = c->draft_len;
  const int cpw = (H + nwg - 1) / nwg;
  const int rpw_qkv = (qd + 2 * kd + nwg - 1) / nwg;
  const int fpw = (F + nwg - 1) / nwg;
  int nh_max = 2 * K + 1 < c->n_codes ? 2 * K + 1 : c->n_codes;
  if (nh_max < 1) nh_max = 1;
  const int wph_min = nwg / nh_max;
  const int rpw_heads = (V + wph_min - 1) / wph_min;
  auto tiles = [](int rows) { return (size_t)((rows + 15) / 16); };
  size_t w = 0;
  auto need = [&](size_t f) {
    if (f > w) w = f;
  };
  if (mfma) {
    // MFMA phases: split activations, chunk sums of squares, wave partial tiles, outputs
    // split rows carry 4 words of padding; wave partials: 1 tile (QKV, O, down),
    // 2 (gate/up), 5 (heads) at a time
    // (+ one row scale per output row for int8 weights)
    need((size_t)mr * (H + 4) + (size_t)mr * (H / 8) + kWaves * 256 + tiles(rpw_qkv) * 16 * (mr + 1) + (size_t)mr * H);
    need((size_t)mr * (H + 4) + (size_t)mr * (H / 8) + kWaves * 2 * 256 + tiles(2 * fpw) * 16 * (mr + 1));
    need((size_t)mr * (qd + 4) + kWaves * 256 + tiles(cpw) * 16 * (mr + 1));
    need((size_t)mr * (F + 4) + kWaves * 256 + tiles(cpw) * 16 * (mr + 1));
    need((size_t)mr * H + (size_t)mr * (H + 4) + kWaves * 5 * 256 + tiles(rpw_heads) * 16 * (mr + 1));
  } else {
    int rows_out = rpw_qkv;
    if (2 * fpw > rows_out) rows_out = 2 * fpw;
    if (rpw_heads > rows_out) rows_out = rpw_heads;
    need((size_t)mr * H + (size_t)rows_out * mr);
    need((size_t)mr * stage_cols + (size_t)cpw * mr);
  }
  need((size_t)3 * kMaxRows * d + (size_t)kMaxPos * (2 * d + 4) + (size_t)kMaxRows * kMaxPos);  // attention: q, k, v rows, the head's KV, softmax weights
  need((size_t)V + 2 * kMaxTopk + 2 + 2 * 3 * kMaxTopk + kMaxTopk + kTopkBuckets + 8);  // sampling
  return w;
}

// Largest k split of a projection (K columns, kw k parts per workgroup) that divides K into
// 64-wide steps and keeps the units (column groups x splits) within one per workgroup.
int pick_ks(int K, int kw, int colgroups, int nwg) {
  const int steps = K / (kw * 64);
  int best = 1;
  for (int ks = 1; ks <= steps && ks <= 32; ++ks)  // the partial-sum readers take at most 32 splits
    if (steps % ks == 0 && colgroups * ks <= nwg) best = ks;
  return best;
}

// Work buffers and parameter block of the batched kernel.
// Validate a packed draft tree (rows 1..n of the query; row 0 is the committed token's row)
// and fill the tree fields of b.
int tree_setup(BParams& b, const rvqsd_cfg& c, int n, const int32_t* parents, const int32_t* ranks) {
  if (n < 1 || n > kMaxTreeRows - 1 || !parents || !ranks)
    return set_err(RVQSD_EINVAL, "a tree needs 1..%d nodes and its parents and ranks", kMaxTreeRows - 1);
  const int nsup = c.topk < c.vocab ? c.topk : c.vocab;
  b.tree = 1;
  b.tree_nodes = n;
  b.t_depth[0] = 0;
  for (int r = 1; r <= n; ++r) {
    const int pr = parents[r - 1], rk = ranks[r - 1];
    if (pr < 0 || pr >= r) return set_err(RVQSD_EINVAL, "node %d: parent %d is not an earlier row", r, pr);
    if (rk < 0 || rk >= nsup) return set_err(RVQSD_EINVAL, "node %d: rank %d outside the top-%d candidates", r, rk, nsup);
    b.t_parent[r] = pr;
    b.t_rank[r] = rk;
    b.t_depth[r] = b.t_depth[pr] + 1;
    if (b.t_depth[r] < b.t_depth[r - 1])
      return set_err(RVQSD_EINVAL, "node %d: rows must be packed breadth first (depth never decreases)", r);
    if (b.t_depth[r] > c.draft_len)
      return set_err(RVQSD_EINVAL, "node %d at depth %d: deeper than draft_len %d", r, b.t_depth[r], c.draft_len);
    for (int q = 1; q < r; ++q)
      if (b.t_parent[q] == pr && b.t_rank[q] == rk) return set_err(RVQSD_EINVAL, "nodes %d and %d: same parent and rank", q, r);
    if (b.t_need[b.t_depth[r]] < rk + 1) b.t_need[b.t_depth[r]] = rk + 1;
  }
  for (int r = 0; r <= n; ++r) {
    b.t_anc[r][0] = b.t_anc[r][1] = 0;
    for (int a = r;; a = b.t_parent[a]) {
      b.t_anc[r][a >> 6] |= 1ull << (a & 63);
      if (a == 0) break;
    }
  }
  return RVQSD_OK;
}

int batch_setup(rvqsd_stream* s, int lanes, int tree_n = 0, const int32_t* parents = nullptr,
                const int32_t* ranks = nullptr) {
  const rvqsd_model* m = s->m;
  const KParams& k = s->kp;
  const rvqsd_cfg& c = m->cfg;
  BParams b;
  memset(&b, 0, sizeof(b));
  if (tree_n) {
    const int st = tree_setup(b, c, tree_n, parents, ranks);
    if (st) return st;
  }
  const int rpl = tree_n ? tree_n + 1 : (c.draft_len + 1 < 2 ? 2 : c.draft_len + 1);
  const int M = lanes * rpl;
  if (c.dtype != RVQSD_DTYPE_BF16) return set_err(RVQSD_EUNSUPPORTED, "batched streams need bf16 weights");
  if (M > kBatchMaxRows)
    return set_err(RVQSD_EUNSUPPORTED, "max_streams * max(draft_len + 1, 2) = %d rows > %d", M, kBatchMaxRows);
  if (k.H % 512 || k.qdim % 256 || k.F % 256 || k.H > 2048)
    return set_err(RVQSD_EUNSUPPORTED, "batched streams need hidden %% 512 == 0 (<= 2048), q width and ffn %% 256 == 0");
  if (m->nwg < 8) return set_err(RVQSD_EUNSUPPORTED, "batched streams need at least 8 workgroups");
  b.lanes = lanes;
  b.kv_slots = tree_n ? kMaxPos + rpl : kMaxPos;
  b.slot_draft0 = rpl > kSlotDraft0 ? rpl : kSlotDraft0;
  b.tr_slots = tree_n ? b.slot_draft0 + rpl * k.K : kSlotDraft0 + kMaxRows * k.K;
  b.rpl = rpl;
  b.M = M;
  b.nwg = m->nwg;
  // 64-column units with the k range of a unit split over 4 waves (and over units by ks)
  b.ks_qkv = pick_ks(k.H, 4, (k.nqkv + 63) / 64, m->nwg);
  b.ks_o = pick_ks(k.qdim, 4, (k.H + 63) / 64, m->nwg);
  b.ks_down = pick_ks(k.F, 4, (k.H + 63) / 64, m->nwg);
  b.hrows = M * (k.K + 1);
  b.sup_words = 1 + 2 * k.topk;
  const size_t kmax = (size_t)(k.H > k.qdim ? (k.H > k.F ? k.H : k.F) : (k.qdim > k.F ? k.qdim : k.F));
  size_t part = (size_t)b.ks_qkv * M * k.nqkv;
  if ((size_t)b.ks_o * M * k.H > part) part = (size_t)b.ks_o * M * k.H;
  if ((size_t)b.ks_down * M * k.H > part) part = (size_t)b.ks_down * M * k.H;
  const int kd = k.K > 0 ? k.K : 1;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += (bytes + 255) & ~(size_t)255;
    return at;
  };
  const size_t o_bar = take(10 * 64 * 4), o_status = take(4), o_tot = take(16);
  const size_t sync_bytes = off;
  const size_t o_lane = take((size_t)lanes * kLaneInts * 4), o_x = take((size_t)M * k.H * 4),
               o_a = take(2 * (size_t)M * kmax * 4), o_ah = take((size_t)b.hrows * k.H * 4),
               o_part = take(part * 4), o_kv = take((size_t)lanes * k.L * k.nkv * b.kv_slots * 2 * k.d * 4),
               o_log = take((size_t)b.hrows * k.V * 4), o_vres = take((size_t)lanes * rpl * 4),
               o_drec = take((size_t)2 * lanes * rpl * kd * b.sup_words * 8), o_bp = take(sizeof(BParams));
  hipError_t e = dev_alloc(&s->bbuf, off);
  if (e != hipSuccess) {
    s->bbuf = nullptr;
    return set_err(RVQSD_ENOMEM, "batched buffers (%zu bytes): %s", off, hipGetErrorString(e));
  }
  uint8_t* base = (uint8_t*)s->bbuf;
  b.k = s->dkp;
  b.bar = (uint32_t*)(base + o_bar);
  b.status = (int32_t*)(base + o_status);
  b.totals = (unsigned long long*)(base + o_tot);
  b.lane = (int32_t*)(base + o_lane);
  b.x = (float*)(base + o_x);
  b.a = (uint32_t*)(base + o_a);
  b.ah = (uint32_t*)(base + o_ah);
  b.part = (float*)(base + o_part);
  b.kv = (float*)(base + o_kv);
  b.logits = (float*)(base + o_log);
  b.vres = (int32_t*)(base + o_vres);
  b.drec = (uint64_t*)(base + o_drec);
  s->dbp = (BParams*)(base + o_bp);
  s->bp = b;
  s->bsync_bytes = sync_bytes;
  s->lanes = lanes;
  e = hipMemset(s->bbuf, 0, off);
  if (e == hipSuccess) e = hipMemcpy(s->dbp, &s->bp, sizeof(BParams), hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(s->bbuf);
    s->bbuf = nullptr;
    return set_err(RVQSD_EHIP, "batched buffers: %s", hipGetErrorString(e));
  }
  // LDS: projection tiles and the SiLU staging, attention rows, sampling arrays, one row
  size_t lds = ((size_t)kBatchRedFloats + (size_t)kBatchMaxRows * 16) * 4;
  const size_t attn = tree_n ? ((size_t)rpl * k.d + (size_t)b.kv_slots * 2 * k.d + (size_t)kWaves * b.kv_slots) * 4
                             : ((size_t)2 * kMaxRows * k.d + (size_t)kMaxPos * (2 * k.d + 4) + kMaxRows * kMaxPos) * 4;
  const size_t samp = ((size_t)k.V + 2 * kMaxTopk) * 4 + 8 + 3 * kMaxTopk * 8 + kMaxTopk * 4 + kTopkBuckets * 4;
  if (attn > lds) lds = attn;
  if (samp > lds) lds = samp;
  if ((size_t)k.H * 4 > lds) lds = (size_t)k.H * 4;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, m->device) == hipSuccess && lds + 64 + 16384 > (size_t)prop.sharedMemPerBlock) {
    (void)hipFree(s->bbuf);
    s->bbuf = nullptr;
    return set_err(RVQSD_EUNSUPPORTED, "the batched kernel needs %zu bytes of LDS (tree of %d rows), %zu available",
                   lds + 64, rpl, (size_t)prop.sharedMemPerBlock);
  }
  s->blds = lds + 64;
  s->tree = tree_n ? 1 : 0;
  return RVQSD_OK;
}

}  // namespace

extern "C" {

const char* rvqsd_last_error(void) { return g_err; }

const char* rvqsd_status_str(rvqsd_status st) {
  switch (st) {
    case RVQSD_OK: return "ok";
    case RVQSD_EINVAL: return "invalid argument";
    case RVQSD_EBLOB: return "bad weight blob";
    case RVQSD_ENOMEM: return "out of memory";
    case RVQSD_EHIP: return "HIP runtime error";
    case RVQSD_EUNSUPPORTED: return "unsupported configuration";
    case RVQSD_ENUMERIC: return "non-finite logits";
    case RVQSD_ETIMEOUT: return "workgroup wait timed out";
    default: return "unknown status";
  }
}

rvqsd_status rvqsd_uniforms_from_seed(uint64_t seed, int32_t n_codes, float* out) {
  if (!out || n_codes < 1 || n_codes > kMaxCodes) return set_err(RVQSD_EINVAL, "bad arguments");
  for (int i = 0; i < n_codes * 3; ++i)
    out[i] = (float)((double)(splitmix64_at(seed, (uint64_t)i) >> 40) * (1.0 / 16777216.0));
  return RVQSD_OK;
}

rvqsd_status rvqsd_create(const rvqsd_weights* w, const rvqsd_cfg* cfg, rvqsd_model** out) {
  if (!w || !cfg || !out || !w->data) return set_err(RVQSD_EINVAL, "null argument");
  *out = nullptr;
  int dev = 0;
  HIPCHK(hipGetDevice(&dev));
  hipDeviceProp_t prop;
  HIPCHK(hipGetDeviceProperties(&prop, dev));
  const int nwg = prop.multiProcessorCount;
  int st = validate_cfg(cfg, nwg);
  if (st) return st;
  if (!prop.cooperativeLaunch) return set_err(RVQSD_EUNSUPPORTED, "device lacks cooperative launch");

  // blob header
  const unsigned char* b = (const unsigned char*)w->data;
  if (w->bytes < 64 || memcmp(b, "RVQSDW1\0", 8) != 0 || rd32(b + 8) != 1)
    return set_err(RVQSD_EBLOB, "bad magic or version");
  const uint32_t want[10] = {(uint32_t)cfg->dtype, (uint32_t)cfg->n_layers, (uint32_t)cfg->hidden,
                             (uint32_t)cfg->n_q_heads, (uint32_t)cfg->n_kv_heads, (uint32_t)cfg->head_dim,
                             (uint32_t)cfg->ffn, (uint32_t)cfg->n_codes, (uint32_t)cfg->vocab,
                             (uint32_t)cfg->max_draft};
  for (int i = 0; i < 10; ++i)
    if (rd32(b + 12 + 4 * i) != want[i]) return set_err(RVQSD_EBLOB, "header field %d = %u, cfg has %u", i, rd32(b + 12 + 4 * i), want[i]);

  KParams k;
  memset(&k, 0, sizeof(k));
  k.L = cfg->n_layers;
  k.H = cfg->hidden;
  k.nq = cfg->n_q_heads;
  k.nkv = cfg->n_kv_heads;
  k.d = cfg->head_dim;
  k.F = cfg->ffn;
  k.n_codes = cfg->n_codes;
  k.V = cfg->vocab;
  k.K = cfg->draft_len;
  k.topk = cfg->topk;
  k.greedy = cfg->draft_greedy;
  k.qk_norm = cfg->qk_norm;
  k.max_draft = cfg->max_draft;
  k.qdim = k.nq * k.d;
  k.kvdim = k.nkv * k.d;
  k.nqkv = k.qdim + 2 * k.kvdim;
  k.rms_eps = (float)cfg->rms_eps;
  k.temperature = cfg->temperature;
  k.rope_base = cfg->rope_base;
  k.nwg = nwg;
  const uint64_t wb = cfg->dtype == RVQSD_DTYPE_F32 ? 4 : (cfg->dtype == RVQSD_DTYPE_BF16 ? 2 : 1);
  const uint64_t H = k.H, qd = k.qdim, kd = k.kvdim, F = k.F, d = k.d, V = k.V, n = k.n_codes;
  // bytes of a [rows][cols] matrix: int8 codes are followed by fp32 row scales, padded to 16 bytes
  auto mat = [&](uint64_t rows, uint64_t cols) -> uint64_t {
    return cfg->dtype == RVQSD_DTYPE_I8 ? (rows * cols + 4 * rows + 15) / 16 * 16 : rows * cols * wb;
  };
  uint64_t o = 0;
  k.o_attn_norm = o; o += H * 4;
  k.o_wq = o; o += mat(qd, H);
  k.o_wk = o; o += mat(kd, H);
  k.o_wv = o; o += mat(kd, H);
  k.o_qn = o; o += d * 4;
  k.o_kn = o; o += d * 4;
  k.o_wo = o; o += mat(H, qd);
  k.o_mlp_norm = o; o += H * 4;
  k.o_wg = o; o += mat(F, H);
  k.o_wu = o; o += mat(F, H);
  k.o_wd = o; o += mat(H, F);
  k.layer_stride = o;
  o = k.layer_stride * k.L;
  k.o_final_norm = o; o += H * 4;
  k.table_stride = mat(V, H);
  k.emb_row_bytes = cfg->dtype == RVQSD_DTYPE_I8 ? H + 4 : H * wb;
  k.o_emb0 = o; o += n * k.table_stride;
  k.o_lmh1 = o; o += n * k.table_stride;
  k.o_offsets = o; o += (uint64_t)cfg->max_draft * H * 4;
  if (w->bytes != 64 + o) return set_err(RVQSD_EBLOB, "blob has %llu bytes, expected %llu", (unsigned long long)w->bytes, (unsigned long long)(64 + o));

  rvqsd_model* m = new (std::nothrow) rvqsd_model;
  if (!m) return set_err(RVQSD_ENOMEM, "host allocation");
  memset(m, 0, sizeof(*m));
  m->cfg = *cfg;
  m->device = dev;
  m->nwg = nwg;
  m->mr = frame_max_rows(cfg->draft_len);
  m->mfma = cfg->dtype != RVQSD_DTYPE_F32 && m->mr <= 8 && cfg->matrix_path == 0;
  if (cfg->dtype == RVQSD_DTYPE_I8 && m->mr > 8) {
    delete m;
    return set_err(RVQSD_EUNSUPPORTED, "int8 weights run on the matrix-core path only: draft_len <= 7");
  }
  if (cfg->dtype == RVQSD_DTYPE_I8) {
    // every workgroup holds one row scale per thread for the head rows it multiplies
    int nh = 2 * cfg->draft_len + 1 < cfg->n_codes ? 2 * cfg->draft_len + 1 : cfg->n_codes;
    if (nh < 1) nh = 1;
    const int rpw = (cfg->vocab + nwg / nh - 1) / (nwg / nh);
    if (rpw > kThreads || (int)((k.nqkv + nwg - 1) / nwg) > kThreads || 2 * (int)((k.F + nwg - 1) / nwg) > kThreads) {
      delete m;
      return set_err(RVQSD_EUNSUPPORTED, "int8 weights: a workgroup's rows of one matrix exceed %d", kThreads);
    }
  }
  if (m->mfma &&
      (k.H > 512 * kUptH || k.qdim > 512 * kUptQ || k.F > 512 * kUptF)) {
    delete m;
    return set_err(RVQSD_EUNSUPPORTED, "bf16 matrix path takes hidden <= %d, n_q_heads*head_dim <= %d, ffn <= %d",
                   512 * kUptH, 512 * kUptQ, 512 * kUptF);
  }
  m->wbytes = (int)wb;
  m->dweight_bytes = o;
  // the rotary table follows the weights: [kMaxPos][d/2][2] cos, sin of position * base^(-2i/d)
  const uint64_t rope_off = (o + 255) & ~(uint64_t)255;
  const size_t rope_bytes = (size_t)kMaxPos * (k.d / 2) * 2 * sizeof(float);
  // LDS: stage the widest activation if it fits, else the down projection polls its chunks directly
  const int cpw = (k.H + nwg - 1) / nwg;
  const size_t head = (size_t)frame_lds_head_floats(m->mr, cpw);
  const size_t budget = (size_t)prop.sharedMemPerBlock - 6 * 1024;  // leave room for static shared state
  // projections stage their input rows in LDS, except a down projection whose
  // chunks have one thread each: it polls them directly
  const int epc = cfg->dtype == RVQSD_DTYPE_F32 ? 4 : 8;
  int stage = (int)(qd > H ? qd : H);
  if (2 * ((int)F / epc) <= kThreads && (int)F > stage) stage = (int)F;
  const size_t work = work_floats(cfg, nwg, m->mr, m->mfma, stage);
  size_t lds = (head + work) * 4;
  if (lds > budget) {
    delete m;
    return set_err(RVQSD_EUNSUPPORTED, "needs %zu bytes of LDS per workgroup, %zu available", lds, budget);
  }
  const size_t attn_const_floats = (size_t)k.L * 2 * k.d + (size_t)kMaxPos * k.d;  // q/k gains + rotary table
  lds += attn_const_floats * 4;
  if (lds > budget) {
    delete m;
    return set_err(RVQSD_EUNSUPPORTED, "needs %zu bytes of LDS per workgroup, %zu available", lds, budget);
  }
  k.work_floats = (int32_t)work;
  m->lds_bytes = lds;
  m->stage_cols = stage;
  k.stage_cols = stage;
  hipError_t e = dev_alloc(&m->dweights, rope_off + rope_bytes);
  if (e != hipSuccess) {
    delete m;
    return set_err(RVQSD_ENOMEM, "device weights (%llu bytes): %s", (unsigned long long)o, hipGetErrorString(e));
  }
  e = hipMemcpy(m->dweights, b + 64, o, hipMemcpyHostToDevice);
  if (e == hipSuccess) {
    // computed in double, stored as float
    const int half = k.d / 2;
    float* tab = (float*)malloc(rope_bytes);
    if (!tab) e = hipErrorOutOfMemory;
    for (int pos = 0; tab && pos < kMaxPos; ++pos)
      for (int i = 0; i < half; ++i) {
        const double th = (double)pos * pow(k.rope_base, -2.0 * (double)i / (double)k.d);
        tab[(pos * half + i) * 2 + 0] = (float)cos(th);
        tab[(pos * half + i) * 2 + 1] = (float)sin(th);
      }
    if (tab) e = hipMemcpy((uint8_t*)m->dweights + rope_off, tab, rope_bytes, hipMemcpyHostToDevice);
    free(tab);
  }
  if (e != hipSuccess) {
    (void)hipFree(m->dweights);
    delete m;
    return set_err(RVQSD_EHIP, "weight upload: %s", hipGetErrorString(e));
  }
  k.wbase = (const uint8_t*)m->dweights;
  k.rope = (const float*)((const uint8_t*)m->dweights + rope_off);
  const FrameLayout fl = frame_layout(k);
  m->frame_bytes = fl.bytes;
  m->base = k;
  *out = m;
  return RVQSD_OK;
}

void rvqsd_destroy(rvqsd_model* m) {
  if (!m) return;
  (void)hipFree(m->dweights);
  delete m;
}

rvqsd_status rvqsd_model_info(const rvqsd_model* m, rvqsd_info* out) {
  if (!m || !out) return set_err(RVQSD_EINVAL, "null argument");
  out->workgroups = m->nwg;
  out->threads = kThreads;
  out->max_rows = m->mr;
  out->trace_slots = kSlotDraft0 + kMaxRows * m->cfg.draft_len;
  out->lds_bytes = m->lds_bytes;
  out->layer_weight_bytes = m->base.layer_stride * (uint64_t)m->base.L;
  out->head_bytes = m->base.table_stride;
  out->emb_row_bytes = m->base.emb_row_bytes;
  out->device_weight_bytes = m->dweight_bytes;
  return RVQSD_OK;
}

static rvqsd_status stream_create(rvqsd_model* m, void* hip_stream, int32_t max_streams, int32_t tree_n,
                                  const int32_t* parents, const int32_t* ranks, rvqsd_stream** out);

rvqsd_status rvqsd_stream_create(rvqsd_model* m, void* hip_stream, int32_t max_streams, rvqsd_stream** out) {
  return stream_create(m, hip_stream, max_streams, 0, nullptr, nullptr, out);
}

rvqsd_status rvqsd_tree_stream_create(rvqsd_model* m, void* hip_stream, int32_t lanes, int32_t n_nodes,
                                      const int32_t* parents, const int32_t* ranks, rvqsd_stream** out) {
  if (n_nodes < 1) return set_err(RVQSD_EINVAL, "a tree needs at least one node");
  return stream_create(m, hip_stream, lanes, n_nodes, parents, ranks, out);
}

static rvqsd_status stream_create(rvqsd_model* m, void* hip_stream, int32_t max_streams, int32_t tree_n,
                                  const int32_t* parents, const int32_t* ranks, rvqsd_stream** out) {
  if (!m || !out) return set_err(RVQSD_EINVAL, "null argument");
  if (max_streams < 1 || max_streams > kMaxLanes) return set_err(RVQSD_EINVAL, "max_streams must be 1..%d", kMaxLanes);
  *out = nullptr;
  rvqsd_stream* s = new (std::nothrow) rvqsd_stream;
  if (!s) return set_err(RVQSD_ENOMEM, "host allocation");
  memset(s, 0, sizeof(*s));
  s->m = m;
  s->stream = (hipStream_t)hip_stream;
  KParams k = m->base;
  const size_t H = k.H;
  // the frame buffers, then this stream's staging of the synchronous calls
  const FrameLayout fl = frame_layout(k);
  size_t off = fl.bytes;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += (bytes + 255) & ~(size_t)255;
    return at;
  };
  const size_t o_in = take(((size_t)H + 3 * kMaxCodes + 4) * 4),
               o_out = take((kMaxCodes + 1) * 4 + sizeof(rvqsd_stats) + 64), o_fbar = take(4);
  s->dbuf_bytes = off;
  hipError_t e = dev_alloc(&s->dbuf, off);
  if (e != hipSuccess) {
    delete s;
    return set_err(RVQSD_ENOMEM, "stream buffers (%zu bytes): %s", off, hipGetErrorString(e));
  }
  s->fbar = (uint32_t*)((uint8_t*)s->dbuf + o_fbar);
  e = hipMemset(s->dbuf, 0, off);
  if (e == hipSuccess)
    e = hipMemsetD8((hipDeviceptr_t)((uint8_t*)s->dbuf + fl.par_begin), 0x01, fl.par_end - fl.par_begin);
  if (e == hipSuccess) e = hipHostMalloc((void**)&s->h_in, ((size_t)H + 3 * kMaxCodes + 4) * 4, hipHostMallocDefault);
  if (e == hipSuccess) e = hipHostMalloc((void**)&s->h_out, (kMaxCodes + 1) * 4 + sizeof(rvqsd_stats) + 64, hipHostMallocDefault);
  if (e != hipSuccess) {
    if (s->h_in) (void)hipHostFree(s->h_in);
    (void)hipFree(s->dbuf);
    delete s;
    return set_err(RVQSD_ENOMEM, "stream staging: %s", hipGetErrorString(e));
  }
  uint8_t* base = (uint8_t*)s->dbuf;
  frame_bind(&k, base, fl);
  s->par_begin = fl.par_begin;
  s->par_end = fl.par_end;
  s->tag_begin = fl.tag_begin;
  s->tag_end = fl.tag_end;
  s->status = k.status;
  s->d_in = (float*)(base + o_in);
  s->d_out = (int32_t*)(base + o_out);
  s->dkp = (KParams*)(base + fl.o_kp);
  s->kp = k;
  e = hipMemcpy(s->dkp, &s->kp, sizeof(KParams), hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipHostFree(s->h_in);
    (void)hipHostFree(s->h_out);
    (void)hipFree(s->dbuf);
    delete s;
    return set_err(RVQSD_EHIP, "parameter upload: %s", hipGetErrorString(e));
  }
  s->epoch_step = frame_epoch_step(k.L);
  s->epoch = s->epoch_step;
  s->lanes = 1;
  if (max_streams > 1 || tree_n > 0) {
    const int st = batch_setup(s, max_streams, tree_n, parents, ranks);
    if (st != RVQSD_OK) {
      (void)hipHostFree(s->h_in);
      (void)hipHostFree(s->h_out);
      (void)hipFree(s->dbuf);
      delete s;
      return st;
    }
  }
  *out = s;
  return RVQSD_OK;
}

void rvqsd_stream_destroy(rvqsd_stream* s) {
  if (!s) return;
  (void)hipStreamSynchronize(s->stream);
  (void)hipHostFree(s->h_in);
  (void)hipHostFree(s->h_out);
  (void)hipFree(s->dbuf);
  if (s->bbuf) (void)hipFree(s->bbuf);
  if (s->bstage) (void)hipFree(s->bstage);
  delete s;
}

rvqsd_status rvqsd_set_trace(rvqsd_stream* s, const rvqsd_trace* t) {
  if (!s) return set_err(RVQSD_EINVAL, "null stream");
  if (t && t->max_rounds < 0) return set_err(RVQSD_EINVAL, "max_rounds < 0");
  s->kp.tr_logits = t ? t->logits : nullptr;
  s->kp.tr_rounds = t ? t->rounds : nullptr;
  s->kp.tr_clock = t ? t->clock : nullptr;
  s->kp.tr_wgclock = t ? t->wg_clock : nullptr;
  s->kp.tr_wgready = t ? t->wg_ready : nullptr;
  s->kp.tr_max_rounds = t ? t->max_rounds : 0;
  HIPCHK(hipStreamSynchronize(s->stream));
  HIPCHK(hipMemcpy(s->dkp, &s->kp, sizeof(KParams), hipMemcpyHostToDevice));
  return RVQSD_OK;
}

static rvqsd_status launch_one(rvqsd_stream* s, const float* d_fh, const int32_t* d_c0, const float* d_u,
                               int32_t* d_codes, rvqsd_stats* d_stats) {
  // tags of stale words from earlier frames never equal a later frame's tags; on wrap, clear everything
  if ((uint64_t)s->epoch + 2ull * s->epoch_step >= 0xFFFFFFFFull) {
    // clears the tagged words only: the parity words and the pass count keep their state
    HIPCHK(hipMemsetAsync((uint8_t*)s->dbuf + s->tag_begin, 0, s->tag_end - s->tag_begin, s->stream));
    s->epoch = s->epoch_step;
  }
  FrameArgs fa;
  fa.frame_hidden = d_fh;
  fa.c0 = d_c0;
  fa.uniforms = d_u;
  fa.out_codes = d_codes;
  fa.out_stats = d_stats;
  fa.epoch_base = s->epoch;
  fa.n_frames = 1;
  fa.epoch_step = 0;
  fa.fbar = s->fbar;
  s->epoch += s->epoch_step;
  char err[256];
  int st = launch_frame(s->dkp, fa, s->m->nwg, s->m->cfg.dtype, s->m->mr, s->m->mfma, (void*)s->stream, s->m->lds_bytes, err,
                        sizeof(err));
  if (st) return set_err(st, "%s", err);
  return RVQSD_OK;
}

// frames of one launch at most (about 1.4 s of the 1024-wide model)
constexpr int kFramesPerLaunch = 1024;

rvqsd_status rvqsd_decode_frames_async(rvqsd_stream* s, int32_t n, const float* d_frame_hidden, const int32_t* d_c0,
                                       const float* d_uniforms, int32_t* d_out_codes, rvqsd_stats* d_stats) {
  if (!s || !d_frame_hidden || !d_c0 || !d_uniforms || !d_out_codes || !d_stats)
    return set_err(RVQSD_EINVAL, "null argument");
  if (n < 0) return set_err(RVQSD_EINVAL, "n = %d < 0", n);
  const size_t H = s->m->base.H, nc = s->m->base.n_codes;
  if (s->tree) {  // tree streams decode through the batched kernel, a frame per call
    for (int f = 0; f < n; ++f) {
      rvqsd_status st = rvqsd_decode_frame_async(s, d_frame_hidden + f * H, d_c0 + f, d_uniforms + f * nc * 3,
                                                 d_out_codes + f * nc, d_stats + f);
      if (st) return st;
    }
    return RVQSD_OK;
  }
  // a trace records the passes of one frame: traced frames get a launch each
  const KParams& kp = s->kp;
  const bool traced = kp.tr_logits || kp.tr_rounds || kp.tr_clock || kp.tr_wgclock || kp.tr_wgready;
  for (int f0 = 0; f0 < n;) {
    const int cnt = traced ? 1 : (n - f0 < kFramesPerLaunch ? n - f0 : kFramesPerLaunch);
    if (cnt == 1) {
      rvqsd_status st = launch_one(s, d_frame_hidden + f0 * H, d_c0 + f0, d_uniforms + f0 * nc * 3, d_out_codes + f0 * nc,
                                   d_stats + f0);
      if (st) return st;
      f0 += 1;
      continue;
    }
    // the tags of every frame of the launch must stay below the wrap
    if ((uint64_t)s->epoch + (uint64_t)(cnt + 1) * s->epoch_step >= 0xFFFFFFFFull) {
      HIPCHK(hipMemsetAsync((uint8_t*)s->dbuf + s->tag_begin, 0, s->tag_end - s->tag_begin, s->stream));
      s->epoch = s->epoch_step;
    }
    HIPCHK(hipMemsetAsync(s->fbar, 0, sizeof(uint32_t), s->stream));
    FrameArgs fa;
    fa.frame_hidden = d_frame_hidden + f0 * H;
    fa.c0 = d_c0 + f0;
    fa.uniforms = d_uniforms + f0 * nc * 3;
    fa.out_codes = d_out_codes + f0 * nc;
    fa.out_stats = d_stats + f0;
    fa.epoch_base = s->epoch;
    fa.n_frames = cnt;
    fa.epoch_step = s->epoch_step;
    fa.fbar = s->fbar;
    s->epoch += (uint32_t)cnt * s->epoch_step;
    char err[256];
    int st = launch_frame(s->dkp, fa, s->m->nwg, s->m->cfg.dtype, s->m->mr, s->m->mfma, (void*)s->stream, s->m->lds_bytes,
                          err, sizeof(err));
    if (st) return set_err(st, "%s", err);
    f0 += cnt;
  }
  return RVQSD_OK;
}

rvqsd_status rvqsd_stream_reset(rvqsd_stream* s) {
  if (!s) return set_err(RVQSD_EINVAL, "null stream");
  HIPCHK(hipStreamSynchronize(s->stream));
  // parity words back to parity 1, pass count and every tagged word back to 0
  uint8_t* base = (uint8_t*)s->dbuf;
  HIPCHK(hipMemsetD8((hipDeviceptr_t)(base + s->par_begin), 0x01, s->par_end - s->par_begin));
  HIPCHK(hipMemset(base + s->par_end, 0, s->tag_end - s->par_end));
  HIPCHK(hipDeviceSynchronize());
  s->epoch = s->epoch_step;
  return RVQSD_OK;
}

rvqsd_status rvqsd_decode_frame_async(rvqsd_stream* s, const float* d_frame_hidden, const int32_t* d_c0,
                                      const float* d_uniforms, int32_t* d_out_codes, rvqsd_stats* d_stats) {
  if (!s || !d_frame_hidden || !d_c0 || !d_uniforms || !d_out_codes || !d_stats)
    return set_err(RVQSD_EINVAL, "null argument");
  if (s->tree) return rvqsd_decode_frames_batched_async(s, 1, d_frame_hidden, d_c0, d_uniforms, d_out_codes, d_stats);
  return launch_one(s, d_frame_hidden, d_c0, d_uniforms, d_out_codes, d_stats);
}

rvqsd_status rvqsd_decode_frame_u(rvqsd_stream* s, const float* frame_hidden, int32_t c0, const float* uniforms,
                                  int32_t* out_codes, rvqsd_stats* out_stats) {
  if (!s || !frame_hidden || !uniforms || !out_codes) return set_err(RVQSD_EINVAL, "null argument");
  if (s->tree) return rvqsd_decode_frames_batched(s, 1, frame_hidden, &c0, uniforms, out_codes, out_stats);
  const rvqsd_cfg& c = s->m->cfg;
  if (c0 < 0 || c0 >= c.vocab) return set_err(RVQSD_EINVAL, "c0 = %d outside [0, %d)", c0, c.vocab);
  const int H = c.hidden, n = c.n_codes;
  for (int i = 0; i < 3 * n; ++i)
    if (!(uniforms[i] >= 0.f && uniforms[i] < 1.f)) return set_err(RVQSD_EINVAL, "uniform %d outside [0, 1)", i);
  for (int i = 0; i < H; ++i)
    if (!std::isfinite(frame_hidden[i])) return set_err(RVQSD_EINVAL, "frame_hidden[%d] is not finite", i);
  // pinned staging: hidden [H] | uniforms [3n] | c0
  memcpy(s->h_in, frame_hidden, (size_t)H * 4);
  memcpy(s->h_in + H, uniforms, (size_t)3 * n * 4);
  memcpy(s->h_in + H + 3 * kMaxCodes, &c0, 4);
  const size_t in_bytes = ((size_t)H + 3 * kMaxCodes + 1) * 4;
  HIPCHK(hipMemcpyAsync(s->d_in, s->h_in, in_bytes, hipMemcpyHostToDevice, s->stream));
  int32_t* d_codes = s->d_out;
  rvqsd_stats* d_stats = (rvqsd_stats*)(s->d_out + kMaxCodes + 1);
  int st = launch_one(s, s->d_in, (const int32_t*)(s->d_in + H + 3 * kMaxCodes), s->d_in + H, d_codes, d_stats);
  if (st) return st;
  const size_t out_bytes = (kMaxCodes + 1) * 4 + sizeof(rvqsd_stats);
  HIPCHK(hipMemcpyAsync(s->h_out, s->d_out, out_bytes, hipMemcpyDeviceToHost, s->stream));
  HIPCHK(hipStreamSynchronize(s->stream));
  rvqsd_stats hs;
  memcpy(&hs, s->h_out + kMaxCodes + 1, sizeof(hs));
  if (hs.status != RVQSD_OK) {
    const int dst = hs.status;
    (void)rvqsd_stream_reset(s);
    return set_err(dst, "device reported %s", rvqsd_status_str(dst));
  }
  memcpy(out_codes, s->h_out, (size_t)n * 4);
  if (out_stats) *out_stats = hs;
  return RVQSD_OK;
}

rvqsd_status rvqsd_decode_frames_batched_async(rvqsd_stream* s, int32_t n, const float* d_frame_hidden,
                                               const int32_t* d_c0, const float* d_uniforms, int32_t* d_out_codes,
                                               rvqsd_stats* d_stats) {
  if (!s) return set_err(RVQSD_EINVAL, "null stream");
  if (n < 0) return set_err(RVQSD_EINVAL, "n = %d < 0", n);
  if (!s->bbuf) return set_err(RVQSD_EUNSUPPORTED, "the stream was created with max_streams = 1");
  if (n == 0) return RVQSD_OK;
  if (!d_frame_hidden || !d_c0 || !d_uniforms || !d_out_codes || !d_stats) return set_err(RVQSD_EINVAL, "null argument");
  HIPCHK(hipMemsetAsync(s->bbuf, 0, s->bsync_bytes, s->stream));
  BCall call;
  call.frame_hidden = d_frame_hidden;
  call.c0 = d_c0;
  call.uniforms = d_uniforms;
  call.out_codes = d_out_codes;
  call.out_stats = d_stats;
  call.n = n;
  char err[256];
  const int st = launch_batch(s->dbp, call, s->m->nwg, (void*)s->stream, s->blds, s->tree != 0, err, sizeof(err));
  if (st) return set_err(st, "%s", err);
  return RVQSD_OK;
}

rvqsd_status rvqsd_decode_frames_batched(rvqsd_stream* s, int32_t n, const float* frame_hidden, const int32_t* c0,
                                         const float* uniforms, int32_t* out_codes, rvqsd_stats* out_stats) {
  if (!s) return set_err(RVQSD_EINVAL, "null stream");
  if (n < 0) return set_err(RVQSD_EINVAL, "n = %d < 0", n);
  if (!s->bbuf) return set_err(RVQSD_EUNSUPPORTED, "the stream was created with max_streams = 1");
  if (n == 0) return RVQSD_OK;
  if (!frame_hidden || !c0 || !uniforms || !out_codes) return set_err(RVQSD_EINVAL, "null argument");
  const rvqsd_cfg& c = s->m->cfg;
  const int H = c.hidden, nc = c.n_codes;
  for (int f = 0; f < n; ++f)
    if (c0[f] < 0 || c0[f] >= c.vocab) return set_err(RVQSD_EINVAL, "c0[%d] = %d outside [0, %d)", f, c0[f], c.vocab);
  for (size_t i = 0; i < (size_t)n * 3 * nc; ++i)
    if (!(uniforms[i] >= 0.f && uniforms[i] < 1.f)) return set_err(RVQSD_EINVAL, "uniform %zu outside [0, 1)", i);
  for (size_t i = 0; i < (size_t)n * H; ++i)
    if (!std::isfinite(frame_hidden[i])) return set_err(RVQSD_EINVAL, "frame_hidden[%zu] is not finite", i);
  // device staging: hidden [n][H] | uniforms [n][3 nc] | c0 [n] | codes [n][nc] | stats [n]
  const size_t b_h = (size_t)n * H * 4, b_u = (size_t)n * 3 * nc * 4, b_c = (size_t)n * 4, b_o = (size_t)n * nc * 4;
  const size_t o_u = (b_h + 255) & ~(size_t)255, o_c = o_u + ((b_u + 255) & ~(size_t)255),
               o_o = o_c + ((b_c + 255) & ~(size_t)255), o_s = o_o + ((b_o + 255) & ~(size_t)255),
               need = o_s + (size_t)n * sizeof(rvqsd_stats);
  if (need > s->bstage_bytes) {
    if (s->bstage) (void)hipFree(s->bstage);
    s->bstage = nullptr;
    s->bstage_bytes = 0;
    hipError_t e = dev_alloc(&s->bstage, need);
    if (e != hipSuccess) {
      s->bstage = nullptr;
      return set_err(RVQSD_ENOMEM, "batched staging (%zu bytes): %s", need, hipGetErrorString(e));
    }
    s->bstage_bytes = need;
  }
  uint8_t* d = (uint8_t*)s->bstage;
  HIPCHK(hipMemcpyAsync(d, frame_hidden, b_h, hipMemcpyHostToDevice, s->stream));
  HIPCHK(hipMemcpyAsync(d + o_u, uniforms, b_u, hipMemcpyHostToDevice, s->stream));
  HIPCHK(hipMemcpyAsync(d + o_c, c0, b_c, hipMemcpyHostToDevice, s->stream));
  int st = rvqsd_decode_frames_batched_async(s, n, (const float*)d, (const int32_t*)(d + o_c), (const float*)(d + o_u),
                                             (int32_t*)(d + o_o), (rvqsd_stats*)(d + o_s));
  if (st) return st;
  HIPCHK(hipMemcpyAsync(out_codes, d + o_o, b_o, hipMemcpyDeviceToHost, s->stream));
  rvqsd_stats* hs = out_stats;
  rvqsd_stats* tmp = nullptr;
  if (!hs) {
    tmp = (rvqsd_stats*)malloc((size_t)n * sizeof(rvqsd_stats));
    if (!tmp) return set_err(RVQSD_ENOMEM, "host allocation");
    hs = tmp;
  }
  hipError_t e = hipMemcpyAsync(hs, d + o_s, (size_t)n * sizeof(rvqsd_stats), hipMemcpyDeviceToHost, s->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
  int dev = RVQSD_OK;
  for (int f = 0; e == hipSuccess && f < n && dev == RVQSD_OK; ++f) dev = hs[f].status;
  free(tmp);
  if (e != hipSuccess) return set_err(RVQSD_EHIP, "batched decode: %s", hipGetErrorString(e));
  if (dev != RVQSD_OK) return set_err(dev, "device reported %s", rvqsd_status_str(dev));
  return RVQSD_OK;
}

rvqsd_status rvqsd_set_batch_trace(rvqsd_stream* s, float* logits, int32_t* rounds, int32_t max_rounds,
                                   int32_t max_frames) {
  if (!s) return set_err(RVQSD_EINVAL, "null stream");
  if (!s->bbuf) return set_err(RVQSD_EUNSUPPORTED, "the stream was created with max_streams = 1");
  const bool on = logits || rounds;
  if (on && (max_rounds < 1 || max_frames < 1)) return set_err(RVQSD_EINVAL, "max_rounds and max_frames must be >= 1");
  s->bp.tr_logits = on ? logits : nullptr;
  s->bp.tr_rounds = on ? rounds : nullptr;
  s->bp.tr_max_rounds = on ? max_rounds : 0;
  s->bp.tr_frames = on ? max_frames : 0;
  HIPCHK(hipStreamSynchronize(s->stream));
  HIPCHK(hipMemcpy(s->dbp, &s->bp, sizeof(BParams), hipMemcpyHostToDevice));
  return RVQSD_OK;
}

rvqsd_status rvqsd_batch_totals(rvqsd_stream* s, uint64_t* passes, uint64_t* bytes) {
  if (!s || !passes || !bytes) return set_err(RVQSD_EINVAL, "null argument");
  if (!s->bbuf) return set_err(RVQSD_EUNSUPPORTED, "the stream was created with max_streams = 1");
  unsigned long long t[2];
  HIPCHK(hipStreamSynchronize(s->stream));
  HIPCHK(hipMemcpy(t, s->bp.totals, sizeof(t), hipMemcpyDeviceToHost));
  *passes = t[0];
  *bytes = t[1];
  return RVQSD_OK;
}

rvqsd_status rvqsd_outer_create(rvqsd_model* m, const void* code_tables, int32_t n_tables, int32_t table_vocab,
                                int32_t topk, double temperature, int32_t max_frames, rvqsd_outer** out) {
  if (!m || !out || (n_tables > 0 && !code_tables)) return set_err(RVQSD_EINVAL, "null argument");
  *out = nullptr;
  const KParams& k = m->base;
  if (n_tables < 0 || n_tables > kMaxCodes || table_vocab < 1 || topk < 1 || topk > kMaxTopk ||
      !(temperature > 0.0) || max_frames < 1 || max_frames > kMaxOuterFrames)
    return set_err(RVQSD_EINVAL, "invalid outer-step argument");
  if (m->cfg.dtype != RVQSD_DTYPE_BF16) return set_err(RVQSD_EUNSUPPORTED, "the outer step needs bf16 weights");
  if (k.H % 512 || k.qdim % 256 || k.F % 256 || k.H > 2048 || m->nwg < 8)
    return set_err(RVQSD_EUNSUPPORTED, "the outer step needs hidden %% 512 == 0 (<= 2048), q width and ffn %% 256 == 0");
  rvqsd_outer* o = new (std::nothrow) rvqsd_outer;
  if (!o) return set_err(RVQSD_ENOMEM, "host allocation");
  memset(o, 0, sizeof(*o));
  o->m = m;
  o->n_tables = n_tables;
  OParams b;
  memset(&b, 0, sizeof(b));
  b.nwg = m->nwg;
  b.M = 1;
  b.ks_qkv = pick_ks(k.H, 4, (k.nqkv + 63) / 64, m->nwg);
  b.ks_o = pick_ks(k.qdim, 4, (k.H + 63) / 64, m->nwg);
  b.ks_down = pick_ks(k.F, 4, (k.H + 63) / 64, m->nwg);
  b.n_tables = n_tables;
  b.table_vocab = table_vocab;
  b.max_frames = max_frames;
  b.topk = topk;
  b.temperature = temperature;
  const size_t kmax = (size_t)(k.H > k.qdim ? (k.H > k.F ? k.H : k.F) : (k.qdim > k.F ? k.qdim : k.F));
  // the step without grid barriers: units of 16 rows over the whole k range or the fewest k splits
  // (each a multiple of 512: eight waves of 64-wide steps) whose range fits a unit's registers; fewer
  // splits mean fewer partial sums for every workgroup to read
  auto split512 = [](int K, int most) {
    for (int ks = 1; ks <= most; ++ks)
      if (K % (ks * 512) == 0 && K / ks <= kFlowSteps * 512) return ks;
    return 0;
  };
  b.ks_o2 = split512(k.qdim, kOutOSplit);
  b.ks_d2 = split512(k.F, kOutDSplit);
  // its poll staging (the partial sums, a k range) stays below the split input row in LDS, and a
  // unit's weights fit in registers (at most kFlowSteps 64-wide k steps per wave)
  const int stage = kBatchRedFloats + kBatchMaxRows * 16;
  int flow_steps = 0;
  if (k.H % 512 == 0 && b.ks_o2 > 0 && b.ks_d2 > 0 && k.nqkv % 16 == 0 && kOutOSplit * k.H <= stage &&
      k.qdim / b.ks_o2 <= stage && k.F / b.ks_d2 <= stage) {
    int kr = k.H;
    if (k.qdim / b.ks_o2 > kr) kr = k.qdim / b.ks_o2;
    if (k.F / b.ks_d2 > kr) kr = k.F / b.ks_d2;
    if (kr <= kFlowSteps * 512) flow_steps = kr / 512;
  }
  const bool flow = flow_steps > 0;
  size_t part = (size_t)b.ks_qkv * k.nqkv;
  if ((size_t)b.ks_o * k.H > part) part = (size_t)b.ks_o * k.H;
  if ((size_t)b.ks_down * k.H > part) part = (size_t)b.ks_down * k.H;
  const size_t tab_bytes = (size_t)n_tables * table_vocab * k.H * 2;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += (bytes + 255) & ~(size_t)255;
    return at;
  };
  const size_t o_bar = take(10 * 64 * 4), o_status = take(4);
  const size_t sync_bytes = off;
  const size_t o_tab = take(tab_bytes), o_rope = take((size_t)max_frames * k.d * 4), o_x = take((size_t)k.H * 4),
               o_a = take(2 * kmax * 4), o_part = take(part * 4),
               o_kv = take((size_t)k.L * k.nkv * max_frames * 2 * k.d * 4),
               o_apart = take((size_t)k.nq * kAttnMaxChunks * (k.d + 2) * 4), o_log = take((size_t)k.V * 4),
               o_last = take((size_t)(1 + kMaxCodes) * 4), o_f = take((size_t)k.H * 4), o_op = take(sizeof(OParams)),
               o_kp = take(sizeof(KParams));
  size_t o_tq = 0, o_tch = 0, o_tat = 0, o_top = 0, o_tact = 0, o_tdp = 0, o_tlog = 0;
  if (flow) {
    // tagged exchange words, one set per layer
    o_tq = take((size_t)k.L * k.nqkv * 8);
    o_tch = take((size_t)k.L * k.nq * kAttnMaxChunks * (k.d + 2) * 8);
    o_tat = take((size_t)k.L * k.qdim * 8);
    o_top = take((size_t)k.L * kOutOSplit * k.H * 8);
    o_tact = take((size_t)k.L * k.F * 8);
    o_tdp = take((size_t)k.L * kOutDSplit * k.H * 8);
    o_tlog = take((size_t)k.V * 8);
  }
  hipError_t e = dev_alloc(&o->buf, off);
  if (e != hipSuccess) {
    delete o;
    return set_err(RVQSD_ENOMEM, "outer-step buffers (%zu bytes): %s", off, hipGetErrorString(e));
  }
  uint8_t* base = (uint8_t*)o->buf;
  b.k = (const KParams*)(base + o_kp);
  b.bar = (uint32_t*)(base + o_bar);
  b.status = (int32_t*)(base + o_status);
  b.tables = (const uint16_t*)(base + o_tab);
  b.rope = (const float*)(base + o_rope);
  b.x = (float*)(base + o_x);
  b.a = (uint32_t*)(base + o_a);
  b.part = (float*)(base + o_part);
  b.kv = (float*)(base + o_kv);
  b.apart = (float*)(base + o_apart);
  b.logits = (float*)(base + o_log);
  if (flow) {
    b.tq = (uint64_t*)(base + o_tq);
    b.tch = (uint64_t*)(base + o_tch);
    b.tat = (uint64_t*)(base + o_tat);
    b.top = (uint64_t*)(base + o_top);
    b.tact = (uint64_t*)(base + o_tact);
    b.tdp = (uint64_t*)(base + o_tdp);
    b.tlog = (uint64_t*)(base + o_tlog);
  }
  o->last_codes = (int32_t*)(base + o_last);
  o->f = (float*)(base + o_f);
  o->dop = (OParams*)(base + o_op);
  o->dkp = (KParams*)(base + o_kp);
  size_t lds = ((size_t)kBatchRedFloats + (size_t)kBatchMaxRows * 16) * 4;
  const size_t samp = ((size_t)k.V + 2 * kMaxTopk) * 4 + 8 + kMaxTopk * 8 + kTopkBuckets * 4;
  // attention: q, k, v, scores, group sums, then the chunk's keys and values (16-byte aligned)
  const size_t chunk = (size_t)attn_chunk_len(max_frames, k.d), G = (size_t)(kThreads / k.d);
  const size_t attn = (((3 * (size_t)k.d + chunk + G * k.d + G + 3) & ~(size_t)3) + chunk * 2 * k.d) * 4;
  // merge: the chunk partials of one head, the chunk weights and the merged output
  const size_t merge = ((size_t)kAttnMaxChunks * (k.d + 2) + kAttnMaxChunks + k.d) * 4;
  if (samp > lds) lds = samp;
  if (attn > lds) lds = attn;
  if (merge > lds) lds = merge;
  if ((size_t)k.H * 4 > lds) lds = (size_t)k.H * 4;
  if (flow) {
    // the step without barriers also keeps its split input row after the unit area and the
    // residual row after everything else
    size_t need = ((size_t)kBatchRedFloats + (size_t)kBatchMaxRows * 16 + kmax) * 4;
    if ((size_t)kOutOSplit * k.H * 4 > need) need = (size_t)kOutOSplit * k.H * 4;
    if (lds > need) need = lds;
    need = (need + 15) / 16 * 16;
    b.xoff = (int32_t)(need / 4);
    lds = need + (size_t)k.H * 4;
  }
  o->flow_steps = flow_steps;
  o->op = b;
  o->sync_bytes = sync_bytes;
  e = hipMemset(o->buf, 0, off);
  if (e == hipSuccess && tab_bytes) e = hipMemcpy((void*)b.tables, code_tables, tab_bytes, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(o->dop, &o->op, sizeof(OParams), hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(o->dkp, &m->base, sizeof(KParams), hipMemcpyHostToDevice);
  if (e == hipSuccess) {
    // rotary table of every frame position, computed in double
    const int half = k.d / 2;
    float* tab = (float*)malloc((size_t)max_frames * half * 2 * sizeof(float));
    if (!tab) e = hipErrorOutOfMemory;
    for (int pos = 0; tab && pos < max_frames; ++pos)
      for (int i = 0; i < half; ++i) {
        const double th = (double)pos * pow(k.rope_base, -2.0 * (double)i / (double)k.d);
        tab[(pos * half + i) * 2 + 0] = (float)cos(th);
        tab[(pos * half + i) * 2 + 1] = (float)sin(th);
      }
    if (tab) e = hipMemcpy((void*)b.rope, tab, (size_t)max_frames * half * 2 * sizeof(float), hipMemcpyHostToDevice);
    free(tab);
  }
  if (e != hipSuccess) {
    (void)hipFree(o->buf);
    delete o;
    return set_err(RVQSD_EHIP, "outer-step set-up: %s", hipGetErrorString(e));
  }
  o->lds = lds + 64;
  *out = o;
  return RVQSD_OK;
}

void rvqsd_outer_destroy(rvqsd_outer* o) {
  if (!o) return;
  (void)hipDeviceSynchronize();
  (void)hipFree(o->buf);
  delete o;
}

rvqsd_status rvqsd_outer_reset(rvqsd_outer* o) {
  if (!o) return set_err(RVQSD_EINVAL, "null argument");
  o->pos = 0;
  return RVQSD_OK;
}

rvqsd_status rvqsd_pipeline_frames_async(rvqsd_stream* s, rvqsd_outer* o, int32_t n, const float* d_t,
                                         const float* d_u_c0, const float* d_uniforms, int32_t* d_codes,
                                         rvqsd_stats* d_stats, float* d_hidden) {
  if (!s || !o) return set_err(RVQSD_EINVAL, "null argument");
  if (n < 0) return set_err(RVQSD_EINVAL, "n = %d < 0", n);
  if (n == 0) return RVQSD_OK;
  if (!d_t || !d_u_c0 || !d_uniforms || !d_codes || !d_stats) return set_err(RVQSD_EINVAL, "null argument");
  if ((uintptr_t)d_t % 16) return set_err(RVQSD_EINVAL, "d_t must be 16-byte aligned");
  const rvqsd_cfg& ic = s->m->cfg;
  const KParams& ok = o->m->base;
  if (ic.hidden != ok.H) return set_err(RVQSD_EINVAL, "inner hidden %d != outer hidden %d", ic.hidden, ok.H);
  if (o->n_tables != ic.n_codes || o->op.table_vocab != ic.vocab)
    return set_err(RVQSD_EINVAL, "outer code tables (%d x %d) do not match the inner model (%d codes of %d)",
                   o->n_tables, o->op.table_vocab, ic.n_codes, ic.vocab);
  if (o->pos + n > o->op.max_frames)
    return set_err(RVQSD_EUNSUPPORTED, "%d frames after %d exceed the outer KV capacity %d", n, o->pos,
                   o->op.max_frames);
  const int nc = ic.n_codes, H = ok.H;
  float* fbuf = d_hidden;
  for (int i = 0; i < n; ++i) {
    HIPCHK(hipMemsetAsync(o->buf, 0, o->sync_bytes, s->stream));
    OCall c;
    c.t = d_t + (size_t)i * H;
    c.u_c0 = d_u_c0 + i;
    c.prev_codes = o->pos == 0 ? nullptr : (i > 0 ? d_codes + (size_t)(i - 1) * (1 + nc) : o->last_codes);
    c.c0_out = d_codes + (size_t)i * (1 + nc);
    c.hidden_out = fbuf ? fbuf + (size_t)i * H : o->f;
    c.pos = o->pos;
    if (++o->epoch == 0) o->epoch = 1;  // the exchange words start at 0: launch number 0 is never used
    c.epoch = o->epoch;
    char err[256];
    int st = launch_outer(o->dop, c, o->m->nwg, (void*)s->stream, o->lds, o->flow_steps, err, sizeof(err));
    if (st) return set_err(st, "%s", err);
    st = launch_one(s, c.hidden_out, c.c0_out, d_uniforms + (size_t)i * nc * 3, c.c0_out + 1, d_stats + i);
    if (st) return st;
    o->pos += 1;
  }
  HIPCHK(hipMemcpyAsync(o->last_codes, d_codes + (size_t)(n - 1) * (1 + nc), (size_t)(1 + nc) * 4,
                        hipMemcpyDeviceToDevice, s->stream));
  return RVQSD_OK;
}

rvqsd_status rvqsd_decode_frame(rvqsd_stream* s, const float* frame_hidden, int32_t c0, uint64_t rng_seed,
                                int32_t* out_codes, rvqsd_stats* out_stats) {
  if (!s) return set_err(RVQSD_EINVAL, "null stream");
  float u[kMaxCodes * 3];
  rvqsd_status st = rvqsd_uniforms_from_seed(rng_seed, s->m->cfg.n_codes, u);
  if (st) return st;
  return rvqsd_decode_frame_u(s, frame_hidden, c0, u, out_codes, out_stats);
}

}  // extern "C"
