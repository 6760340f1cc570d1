// rvqsd_frame.hip -- persistent frame kernel (gfx950) for RVQ-position-aware speculative decoding.
//
// One cooperative launch decodes one frame: the 2-row prefix pass, then
// speculative rounds until the 15 residual codes are committed (paper Fig. 1
// inner loop, Sec. 2.2 drafting and verification). Every pass runs, for each
// decoder layer, five phases (QKV, attention, O, gate/up, down), then the
// per-position LM heads and the fused top-k / softmax / accept / resample /
// draft phase. The accept chain of a round is folded into the start of the
// next pass: every workgroup reads the per-position verdicts and derives the
// new anchor itself, so no phase is spent on it.
//
// Workgroups exchange activations through 64-bit words whose high half is a
// tag (frame epoch + pass + phase) and whose low half is the fp32 payload.
// Producers write them and consumers poll them with relaxed device-scope
// atomic accesses: no cache-wide fences, no grid barrier. Every wait is
// bounded; a timed-out or failed workgroup records an error in the device
// status word, and every other wait gives up as soon as it sees it, so the
// grid always drains.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rvqsd_device.h"
#include "rvqsd_internal.h"

namespace rvqsd {

template <typename WT>
struct WTraits;
template <>
struct WTraits<float> {
  static constexpr int EPC = 4;  // elements per 16-byte chunk
  __device__ static __forceinline__ void widen(const W16& c, float* w) {
    w[0] = __uint_as_float(c.x);
    w[1] = __uint_as_float(c.y);
    w[2] = __uint_as_float(c.z);
    w[3] = __uint_as_float(c.w);
  }
  __device__ static __forceinline__ float one(const float* p, size_t i) { return G(p)[i]; }
};
template <>
struct WTraits<bf16_t> {
  static constexpr int EPC = 8;
  __device__ static __forceinline__ void widen(const W16& c, float* w) {
    w[0] = __uint_as_float(c.x << 16);
    w[1] = __uint_as_float(c.x & 0xffff0000u);
    w[2] = __uint_as_float(c.y << 16);
    w[3] = __uint_as_float(c.y & 0xffff0000u);
    w[4] = __uint_as_float(c.z << 16);
    w[5] = __uint_as_float(c.z & 0xffff0000u);
    w[6] = __uint_as_float(c.w << 16);
    w[7] = __uint_as_float(c.w & 0xffff0000u);
  }
  __device__ static __forceinline__ float one(const bf16_t* p, size_t i) { return __uint_as_float((uint32_t)G(p)[i] << 16); }
};

// ---------------------------------------------------------- shared state

struct Shared {
  FrameArgs fa;
  int abort;
  int pass, m, kp, first_pos, rows;
  int prev_anchor_row;  // row, in the previous pass, of the current anchor m
  int codes[kMaxPos + 1];
  int drafts[kMaxPos + 1];
  int in_code[kMaxPos + 1];  // code consumed at position s (s >= 1)
  float rstd[kMaxRows];
  // statistics (kept by every workgroup, written by workgroup 0)
  int st_calls, st_rounds, st_drafted, st_accepted;
  unsigned st_mask;
  unsigned long long st_bytes;
  // sampling scratch
  TopkShared tk;
  int n_sup, n_q;
  int tok, acc;
  float uni[kMaxCodes * 3];  // this frame's uniforms (draft, accept, sample) per position 1..15
  // vectors of the LM head this workgroup multiplies (heads phase)
  int hv_n, hv_row[kMaxRows], hv_off[kMaxRows], hv_slot[kMaxRows];
};

struct Ctx {
  const KParams* p;
  Shared* sh;
  float* dyn;       // dynamic LDS
  float* xown;      // [kMaxRows][cpw] residual columns owned by this workgroup
  float* red;       // [kWaves][RPT * MR] reduction scratch
  float* work;      // union area
  float* attn_const;  // [L][2][d] q/k norm gains, then [kMaxPos][d/2][2] rotary table (attention workgroups)
  int cpw;          // residual columns per workgroup
  uint32_t tag_base;
  uint32_t pass0;   // passes this stream ran before this frame
  uint64_t* rdy;    // trace: this workgroup's input-complete stamp of the current phase (nullable)
};

// Parity of the per-layer buffers (q/k/v, attention output, activation): one write per
// layer per pass, so it alternates with every write. It counts from the start of the frame:
// a frame begins with every such word at parity 1 (set when the stream is created, and again
// by the frame kernel at the end of every complete frame), and its first write has parity 0.
// The parity thus depends only on the pass and the layer within the frame, and so does the
// lowest mantissa bit of every exchanged value: a frame's codes do not depend on what the
// stream decoded before it.
__device__ __forceinline__ uint32_t par_layer(const Ctx& c, int pass, int l) {
  return (uint32_t)(((uint64_t)pass * (uint64_t)c.p->L + (uint64_t)l) & 1u);
}
constexpr uint32_t kParO = 0, kParDown = 1;  // residual stream: written after O, then after down

__device__ __forceinline__ uint32_t tag_of(const Ctx& c, int pass, int phase) {
  return c.tag_base + (uint32_t)(pass * phases_per_pass(c.p->L) + phase + 1);
}

__device__ __forceinline__ bool status_set(const KParams* p, uint32_t epoch) {
  uint64_t s = __hip_atomic_load(G(p->status), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return (uint32_t)(s >> 32) == epoch && (int32_t)(uint32_t)s != 0;
}
__device__ __forceinline__ void status_raise(const KParams* p, uint32_t epoch, int code) {
  __hip_atomic_store(G(p->status), ((uint64_t)epoch << 32) | (uint32_t)code, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Poll n tagged words; addr(i) gives word i, sink(i, payload) receives it.
// Per-thread words: i = tid, tid + kThreads, ... Returns false if this thread gave up.
template <typename Addr, typename Sink>
__device__ __forceinline__ bool poll_words(const Ctx& c, int n, uint32_t tag, Addr addr, Sink sink) {
  for (int base = 0; base < n; base += 4 * kThreads) {
    int idx[4];
    bool got[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      idx[k] = base + k * kThreads + tid();
      got[k] = idx[k] >= n;
    }
    uint64_t t0 = 0;
    int spins = 0;
    while (true) {
      uint64_t v[4];
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (!got[k]) v[k] = xload(addr(idx[k]));
      bool all = true;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (!got[k]) {
          if ((uint32_t)(v[k] >> 32) == tag) {
            got[k] = true;
            sink(idx[k], (uint32_t)v[k]);
          } else {
            all = false;
          }
        }
      }
      if (all) break;
      if ((++spins & 31) == 0) {
        uint64_t now = dclock();
        if (t0 == 0) {
          t0 = now;
        } else if (now - t0 > kTimeoutTicks) {
          status_raise(c.p, c.tag_base, RVQSD_ETIMEOUT);
          return false;
        }
        if (status_set(c.p, c.tag_base)) return false;
      }
    }
  }
  return true;
}

template <typename Sink>
__device__ __forceinline__ bool poll_range(const Ctx& c, const uint64_t* src, int n, uint32_t tag, Sink sink) {
  return poll_words(c, n, tag, [=](int i) { return src + i; }, sink);
}

// Poll n4 groups of four parity words; addr(i) gives group i (16-byte aligned),
// sink(i, w) receives the group's words once all four carry parity `par`.
template <typename Addr, typename Sink>
__device__ __forceinline__ bool poll_quads(const Ctx& c, int n4, uint32_t par, Addr addr, Sink sink) {
  constexpr int B = 4;
  for (int base = 0; base < n4; base += B * kThreads) {
    int idx[B];
    bool got[B];
#pragma unroll
    for (int k = 0; k < B; ++k) {
      idx[k] = base + k * kThreads + tid();
      got[k] = idx[k] >= n4;
    }
    uint64_t t0 = 0;
    int spins = 0;
    while (true) {
      W16 v[B];
#pragma unroll
      for (int k = 0; k < B; ++k) {
        v[k] = (W16)(0u);
        if (!got[k]) v[k] = pload4(addr(idx[k]));
      }
#pragma unroll
      for (int k = 0; k < B; ++k) vm_wait(v[k]);
      bool all = true;
#pragma unroll
      for (int k = 0; k < B; ++k) {
        if (!got[k]) {
          if ((v[k][0] & 1u) == par && (v[k][1] & 1u) == par && (v[k][2] & 1u) == par && (v[k][3] & 1u) == par) {
            got[k] = true;
            sink(idx[k], v[k]);
          } else {
            all = false;
          }
        }
      }
      if (all) break;
      if ((++spins & 31) == 0) {
        const uint64_t now = dclock();
        if (t0 == 0) {
          t0 = now;
        } else if (now - t0 > kTimeoutTicks) {
          status_raise(c.p, c.tag_base, RVQSD_ETIMEOUT);
          return false;
        }
        if (status_set(c.p, c.tag_base)) return false;
      }
    }
  }
  return true;
}

// Barrier of the workgroup that also agrees on abort.
__device__ __forceinline__ bool wg_sync_ok(const Ctx& c, bool ok) {
  if (!ok) c.sh->abort = 1;
  __syncthreads();
  if (c.rdy && tid() == 0) *G(c.rdy) = __builtin_amdgcn_s_memrealtime();
  return c.sh->abort == 0;
}

// --------------------------------------------------------------- weights

template <typename WT>
__device__ __forceinline__ const WT* wptr(const KParams* p, uint64_t off) {
  return reinterpret_cast<const WT*>(p->wbase + off);
}
__device__ __forceinline__ const float* fptr(const KParams* p, uint64_t off) {
  return reinterpret_cast<const float*>(p->wbase + off);
}
__device__ __forceinline__ uint64_t layer_off(const KParams* p, int l, uint64_t o) {
  return (uint64_t)l * p->layer_stride + o;
}

// ------------------------------------------------------------------ GEMV
// Computes out[r][m] = sum_k W[row r][k] * X[m][k] for the workgroup's nrows
// rows (r < nrows) and MR activation rows. Thread (rg, kc): kc = 16-byte chunk
// of the reduction dimension, rg = row group; rows r = rg + i * n_rg.
// The weight chunks of the first batch are loaded before the activations are
// awaited, so the weight stream overlaps the wait.

template <typename WT, int MR, int RPT, bool PIPE = false>
struct Gemv {
  static constexpr int EPC = WTraits<WT>::EPC;
  static constexpr int NVR = (RPT + 1) * MR;  // reduced values per wave: rows x MR, then MR sums of squares
  int nkc, n_rg, rg, kc, nrows;
  bool active;
  W16 wreg[RPT];
  W16 wnext[PIPE ? RPT : 1];
  float gain[EPC];  // this thread's chunk of an RMSNorm gain (prefetched with the weights)

  __device__ __forceinline__ void setup(int K, int nrows_) {
    nkc = K / EPC;
    n_rg = kThreads / nkc;
    rg = tid() / nkc;
    kc = tid() % nkc;
    active = rg < n_rg;
    nrows = nrows_;
  }
  template <typename RowPtr>
  __device__ __forceinline__ void load_into(W16 (&dst)[RPT], int batch, RowPtr rowptr) {
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const int r = rg + (batch * RPT + i) * n_rg;
      if (active && r < nrows) {
        const WT* w = rowptr(r) + (size_t)kc * EPC;
        dst[i] = *G(reinterpret_cast<const W16*>(w));
      } else {
        dst[i] = (W16)(0u);
      }
    }
  }
  template <typename RowPtr>
  __device__ __forceinline__ void load(int batch, RowPtr rowptr) {
    load_into(wreg, batch, rowptr);
  }
  __device__ __forceinline__ void load_gain(const float* gsrc) {
#pragma unroll
    for (int e = 0; e < EPC; ++e)
      gain[e] = active ? G(gsrc)[kc * EPC + e] : 1.f;
  }
  // out[r * MR + m] = sum_k W[r][k] * xg[m][k] (LDS), times rstd_m when sq != nullptr,
  // where sq[m] is this thread's sum of squares of the raw activation chunk and
  // rstd_m = 1 / sqrt(sum_k x[m][k]^2 / K + eps). Each value is summed over the
  // wave with DPP (total in lane 63), then over the waves of its row group in LDS.
  template <typename RowPtr>
  __device__ __forceinline__ void run(const Ctx& c, const float (&xg)[MR][EPC], RowPtr rowptr, float* out,
                                      const float* sq = nullptr) {
    const int lane = tid() & 63, wave = tid() >> 6;
    const int rows_per_thread = (nrows + n_rg - 1) / n_rg;
    const int nbatch = (rows_per_thread + RPT - 1) / RPT;
    const int wpg = nkc / 64;  // waves per row group
    const float inv_k = 1.f / (float)(nkc * EPC);
    if (sq) {
#pragma unroll
      for (int m = 0; m < MR; ++m) {
        const float v = wave_sum63((rg == 0 && active) ? sq[m] : 0.f);
        if (lane == 63) c.red[wave * NVR + RPT * MR + m] = v;
      }
    }
    for (int b = 0; b < nbatch; ++b) {
      if constexpr (PIPE) {
        if (b + 1 < nbatch) load_into(wnext, b + 1, rowptr);
      } else {
        if (b > 0) load(b, rowptr);
      }
      const int nb = min(RPT, rows_per_thread - b * RPT);  // uniform across the workgroup
#pragma unroll
      for (int i = 0; i < RPT; ++i) {
        if (i < nb) {
          float w[EPC];
          WTraits<WT>::widen(wreg[i], w);
#pragma unroll
          for (int m = 0; m < MR; ++m) {
            float a = 0.f;
#pragma unroll
            for (int e = 0; e < EPC; ++e) a = fmaf(w[e], xg[m][e], a);
            a = wave_sum63(a);
            if (lane == 63) c.red[wave * NVR + i * MR + m] = a;
          }
        }
      }
      lds_barrier();
      const int total = n_rg * nb * MR;
      for (int t = tid(); t < total; t += kThreads) {
        const int g = t / (nb * MR), im = t % (nb * MR), i = im / MR, m = im % MR;
        const int r = g + (b * RPT + i) * n_rg;
        if (r < nrows) {
          float sum = 0.f;
          for (int w = g * wpg; w < (g + 1) * wpg; ++w) sum += c.red[w * NVR + im];
          if (sq) {
            float ss = 0.f;
            for (int w = 0; w < wpg; ++w) ss += c.red[w * NVR + RPT * MR + m];
            sum *= __builtin_amdgcn_rsqf(ss * inv_k + (float)c.p->rms_eps);
          }
          out[r * MR + m] = sum;
        }
      }
      lds_barrier();
      if constexpr (PIPE) {
#pragma unroll
        for (int i = 0; i < RPT; ++i) wreg[i] = wnext[i];
      }
    }
  }
};

// ---------------------------------------------------------- MFMA GEMV (bf16)
// For bf16 weights and up to 8 activation rows the projections run on
// v_mfma_f32_16x16x32_bf16. Lane layout of that instruction (checked on gfx950):
// lane l holds A[l%16][8*(l/16) + j], B[8*(l/16) + j][l%16] and returns
// D[4*(l/16) + v][l%16]. A = 16 weight rows, B = activations (column m = row m
// of the pass). The order of the 32 products inside one instruction is free, so
// lane group q = l/16 takes the 16 consecutive k's 64u + 16q .. 64u + 16q + 15 of
// a 64-wide unit u in two instructions: each lane loads 32 contiguous bytes of
// its weight row and the four groups read the row's full 128-byte line.
// The fp32 activations enter as a bf16 pair hi + lo (|x - hi - lo| <= 2^-16 |x|),
// so each unit is four instructions and the product keeps fp32-level accuracy.
// Units (16-row tile t, unit u) are g = t * U + u with U = K / 64 a multiple of
// 8; wave w takes g = w, w + 8, ..., so each wave holds one accumulator per tile
// and the 8 wave partials are added once in LDS.


template <typename WT>
struct IsBf16 {
  static constexpr bool value = false;
};
template <>
struct IsBf16<bf16_t> {
  static constexpr bool value = true;
};
// int8 weight codes with fp32 per-row scales (W8A16): MFMA path only
template <typename WT>
struct IsI8 {
  static constexpr bool value = false;
};
template <>
struct IsI8<int8_t> {
  static constexpr bool value = true;
};

// Scale of row `row` of the [rows][cols] matrix at byte offset off: its fp32 row scale for
// int8 codes (stored after the codes), 1 otherwise.
template <typename WE>
__device__ __forceinline__ float row_scale(const KParams* p, uint64_t off, int rows, int cols, int row) {
  if constexpr (IsI8<WE>::value)
    return G(reinterpret_cast<const float*>(p->wbase + off + (uint64_t)rows * cols))[row];
  else
    return 1.f;
}

// 16 int8 codes (one 16-byte load) -> the same values as two groups of 8 bf16 (exact:
// every integer in [-128, 127] is a bf16)
__device__ __forceinline__ uint32_t i8pair_bf16(uint32_t w, int sh) {
  const float f0 = (float)(int8_t)(uint8_t)(w >> sh), f1 = (float)(int8_t)(uint8_t)(w >> (sh + 8));
  return (__float_as_uint(f0) >> 16) | (__float_as_uint(f1) & 0xffff0000u);
}
__device__ __forceinline__ void widen_i8x16(const W16& v, W16& lo, W16& hi) {
  lo[0] = i8pair_bf16(v[0], 0);
  lo[1] = i8pair_bf16(v[0], 16);
  lo[2] = i8pair_bf16(v[1], 0);
  lo[3] = i8pair_bf16(v[1], 16);
  hi[0] = i8pair_bf16(v[2], 0);
  hi[1] = i8pair_bf16(v[2], 16);
  hi[2] = i8pair_bf16(v[3], 0);
  hi[3] = i8pair_bf16(v[3], 16);
}

// Split activations in LDS: row m, 8-element chunk q -> 8 words at m * (K + 4) + q * 8:
// 4 words of hi, then 4 words of lo. The 4 words of padding per row put the 16
// rows that one MFMA operand read touches on different LDS banks.
__device__ __forceinline__ int split_stride(int K) { return K + 4; }
__device__ __forceinline__ void put_split(uint32_t* xsp, int stride, int m, int q, const float (&x)[8]) {
  W16 hi, lo;
  split8(x, hi, lo);
  *reinterpret_cast<W16*>(xsp + (size_t)m * stride + q * 8) = hi;
  *reinterpret_cast<W16*>(xsp + (size_t)m * stride + q * 8 + 4) = lo;
}

// Poll rows 0..R-1 of a parity activation buffer [kMaxRows][K] chunk by chunk
// (8 floats = two 16-byte halves) and store them split into xsp. With GAIN the
// stored value is gain[k] * x (gain global, [K]) and sqc ([R][K/8]) receives
// each chunk's sum of squares of the raw x for the row's RMSNorm.
// Chunk i of the pass is handled by thread i % kThreads; up to CB chunks per
// thread are in flight at once.
template <int CB, bool GAIN>
__device__ __forceinline__ bool stage_split(const Ctx& c, const uint32_t* src, int K, int R, uint32_t par,
                                            const float* gain, uint32_t* xsp, float* sqc) {
  const int nch = K >> 3, total = R * nch;
  for (int base = 0; base < total; base += CB * kThreads) {
    uint32_t pending = 0;  // bit 4b + w: word w of chunk b still missing
#pragma unroll
    for (int b = 0; b < CB; ++b)
      if (base + b * kThreads + tid() < total) pending |= 0xfu << (4 * b);
    float gv[GAIN ? CB : 1][8];
    if constexpr (GAIN) {
#pragma unroll
      for (int b = 0; b < CB; ++b) {
        const int idx = base + b * kThreads + tid();
        const int kq = idx < total ? (idx % nch) * 8 : 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) gv[b][e] = G(gain)[kq + e];
      }
    }
    uint64_t v[CB][4];
    uint64_t t0 = 0;
    int spins = 0;
    while (pending) {
      // 16-byte loads: half hh of a chunk (words 4 hh .. 4 hh + 3) is reloaded while any of its words is missing
      W16 v4[CB][2];
#pragma unroll
      for (int b = 0; b < CB; ++b) {
        const int idx = base + b * kThreads + tid();
        const int m = idx / nch, q = idx - m * nch;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          v4[b][hh] = (W16)(0u);
          if (pending & (3u << (4 * b + 2 * hh))) v4[b][hh] = pload4(src + (size_t)m * K + q * 8 + 4 * hh);
        }
      }
#pragma unroll
      for (int b = 0; b < CB; ++b)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) vm_wait(v4[b][hh]);
#pragma unroll
      for (int b = 0; b < CB; ++b)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
          if (pending & (3u << (4 * b + 2 * hh))) {
            v[b][2 * hh] = (uint64_t)v4[b][hh][0] | ((uint64_t)v4[b][hh][1] << 32);
            v[b][2 * hh + 1] = (uint64_t)v4[b][hh][2] | ((uint64_t)v4[b][hh][3] << 32);
          }
#pragma unroll
      for (int b = 0; b < CB; ++b)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
          if (pending & (3u << (4 * b + 2 * hh))) {
            const W16 w4 = v4[b][hh];
            if ((w4[0] & 1u) == par && (w4[1] & 1u) == par && (w4[2] & 1u) == par && (w4[3] & 1u) == par)
              pending &= ~(3u << (4 * b + 2 * hh));
          }
      if (!pending) break;
      if ((++spins & 31) == 0) {
        const uint64_t now = dclock();
        if (t0 == 0) {
          t0 = now;
        } else if (now - t0 > kTimeoutTicks) {
          status_raise(c.p, c.tag_base, RVQSD_ETIMEOUT);
          return wg_sync_ok(c, false);
        }
        if (status_set(c.p, c.tag_base)) return wg_sync_ok(c, false);
      }
    }
#pragma unroll
    for (int b = 0; b < CB; ++b) {
      const int idx = base + b * kThreads + tid();
      if (idx < total) {
        float x[8], s2 = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          x[2 * w] = __uint_as_float((uint32_t)v[b][w]);
          x[2 * w + 1] = __uint_as_float((uint32_t)(v[b][w] >> 32));
        }
        const int m = idx / nch;
        if constexpr (GAIN) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            s2 = fmaf(x[e], x[e], s2);
            x[e] *= gv[b][e];
          }
        }
        put_split(xsp, split_stride(K), m, idx - m * nch, x);
      }
      if constexpr (GAIN) {
        // the 64 chunks of a wave belong to one row (K is a multiple of 512): one sum per wave,
        // sqc[idx / 64] (row m owns sqc[m * K / 512 ..])
        const int i0 = base + b * kThreads + (tid() & ~63);
        if (i0 < total) {
          float s2 = 0.f;
          if (idx < total) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
              const float a0 = __uint_as_float((uint32_t)v[b][w]), a1 = __uint_as_float((uint32_t)(v[b][w] >> 32));
              s2 = fmaf(a0, a0, fmaf(a1, a1, s2));
            }
          }
          s2 = wave_sum63(s2);
          if ((tid() & 63) == 63) sqc[i0 >> 6] = s2;
        }
      }
    }
  }
  return wg_sync_ok(c, true);
}
// 1 / sqrt(mean of squares + eps) of staged row m from the per-wave sums of stage_split / gather_split_rows
// (RMSNorm scales here and below use the hardware reciprocal square root, within 1 ulp)
__device__ __forceinline__ float rstd_of(const Ctx& c, const float* sqc, int K, int m) {
  const int G = K >> 9;
  float s = 0.f;
  for (int k = 0; k < G; ++k) s += sqc[m * G + k];
  return __builtin_amdgcn_rsqf(s / (float)K + (float)c.p->rms_eps);
}

// rstd[m] from the per-wave sums of stage_split / gather_split_rows, m < R.
__device__ __forceinline__ void rstd_from_chunks_w(const Ctx& c, const float* sqc, int K, int R) {
  if (tid() < R) c.sh->rstd[tid()] = rstd_of(c, sqc, K, tid());
  __syncthreads();
}
// rstd[m] = 1 / sqrt(sum of the row's chunk sums / K + eps), m < R (one wave per row).
__device__ __forceinline__ void rstd_from_chunks(const Ctx& c, const float* sqc, int K, int R) {
  const int lane = tid() & 63, wave = tid() >> 6, nch = K >> 3;
  for (int m = wave; m < R; m += kWaves) {
    float s = 0.f;
    for (int q = lane; q < nch; q += 64) s += sqc[m * nch + q];
    s = wave_sum63(s);
    if (lane == 63) c.sh->rstd[m] = __builtin_amdgcn_rsqf(s / (float)K + (float)c.p->rms_eps);
  }
  __syncthreads();
}

// out[r * MR + m] = sum_k W[row r][k] * X[m][k] for the workgroup's nrows rows,
// W bf16 row-major with row pointer rowptr(r), X split in LDS (xsp, rows < R).
// Wave w owns the 64-wide units u = w, w + 8, ... (upt = K / 512 of them) of
// every 16-row tile, so one read of a unit's B operand serves all tiles. Up to
// NT tiles are held at a time (tile groups), UPT >= upt. Each wave writes its
// partial tiles to red[kWaves][NT][256]; reduce() adds the 8 partials.
template <int MR, int NT, int UPT, typename WE = bf16_t>
struct MTile {
  int U, upt, ntiles, nrows, wave, lane;
  W16 a[NT][UPT][2];

  __device__ __forceinline__ void setup(int K, int nrows_) {
    U = K >> 6;
    upt = U >> 3;
    nrows = nrows_;
    ntiles = (nrows + 15) >> 4;
    wave = __builtin_amdgcn_readfirstlane(tid() >> 6);
    lane = tid() & 63;
  }
  // weights of tiles tb .. tb + NT - 1
  template <typename RowPtr>
  __device__ __forceinline__ void load(int tb, RowPtr rowptr) {
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
      const int row = ((tb + tt) << 4) + (lane & 15);
#pragma unroll
      for (int j = 0; j < UPT; ++j) {
        W16 v0 = (W16)(0u), v1 = (W16)(0u);
        if (tb + tt < ntiles && j < upt && row < nrows) {
          const WE* w = rowptr(row) + (wave + 8 * j) * 64 + 16 * (lane >> 4);
          v0 = *G(reinterpret_cast<const W16*>(w));  // int8: all 16 codes
          if constexpr (!IsI8<WE>::value) v1 = *G(reinterpret_cast<const W16*>(w + 8));
        }
        a[tt][j][0] = v0;
        a[tt][j][1] = v1;
      }
    }
  }
  // B operand of unit j for this lane (zero for activation rows >= R)
  __device__ __forceinline__ void load_b(const uint32_t* xrow, bool live, int j, W16 (&bv)[4]) const {
    if (live) {
      const uint32_t* bp = xrow + (size_t)(wave + 8 * j) * 64;
      bv[0] = *reinterpret_cast<const W16*>(bp);
      bv[1] = *reinterpret_cast<const W16*>(bp + 4);
      bv[2] = *reinterpret_cast<const W16*>(bp + 8);
      bv[3] = *reinterpret_cast<const W16*>(bp + 12);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) bv[q] = (W16)(0u);
    }
  }
  // tiles tb .. tb + NT - 1 (weights already loaded when preloaded); the hi and
  // lo products accumulate separately
  template <typename RowPtr>
  __device__ __forceinline__ void mma(int tb, bool preloaded, RowPtr rowptr, const uint32_t* xsp, int R, float* red) {
    const int m = lane & 15, q = lane >> 4;
    const bool live = m < R;
    if (!preloaded) load(tb, rowptr);
    const uint32_t* xrow = xsp + (size_t)m * split_stride(U * 64) + 16 * q;
    f32x4 acc[NT][2];
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) acc[tt][0] = acc[tt][1] = (f32x4){0.f, 0.f, 0.f, 0.f};
    W16 b[UPT][4];
    load_b(xrow, live, 0, b[0]);
#pragma unroll
    for (int j = 0; j < UPT; ++j) {
      if (j < upt) {
        if (j + 1 < UPT && j + 1 < upt) load_b(xrow, live, j + 1, b[j + 1]);
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) {
          if (tb + tt < ntiles) {
            W16 w0 = a[tt][j][0], w1 = a[tt][j][1];
            if constexpr (IsI8<WE>::value) widen_i8x16(a[tt][j][0], w0, w1);
            const bf16x8 a0 = __builtin_bit_cast(bf16x8, w0), a1 = __builtin_bit_cast(bf16x8, w1);
            acc[tt][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, __builtin_bit_cast(bf16x8, b[j][0]), acc[tt][0], 0, 0, 0);
            acc[tt][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, __builtin_bit_cast(bf16x8, b[j][1]), acc[tt][1], 0, 0, 0);
            acc[tt][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, __builtin_bit_cast(bf16x8, b[j][2]), acc[tt][0], 0, 0, 0);
            acc[tt][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, __builtin_bit_cast(bf16x8, b[j][3]), acc[tt][1], 0, 0, 0);
          }
        }
      }
    }
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
      if (tb + tt < ntiles) {
        const f32x4 s4 = acc[tt][0] + acc[tt][1];
        float* dst = red + ((size_t)(wave * NT + tt) << 8);
#pragma unroll
        for (int v = 0; v < 4; ++v) dst[((4 * q + v) << 4) + m] = s4[v];
      }
    }
  }
  // out[r * MR + mm] for rows r of tiles tb .. tb + NT - 1 (r < nrows), mm < MR: the
  // sum of the 8 wave partials, times rstd[mm] when given
  __device__ __forceinline__ void reduce(const float* red, float* out, const float* rstd, int tb) const {
    const int r0 = tb << 4, r1 = min((tb + NT) << 4, nrows);
    for (int o = tid(); o < (r1 - r0) * MR; o += kThreads) {
      const int r = r0 + o / MR, mm = o % MR, t = (r >> 4) - tb, i = r & 15;
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) s += red[((w * NT + t) << 8) + (i << 4) + mm];
      out[r * MR + mm] = rstd ? s * rstd[mm] : s;
    }
  }
  // one tile group (ntiles <= NT, weights preloaded), wave partials in red after the barrier;
  // psum(red, r, m) then gives the product of row r and activation row m
  __device__ __forceinline__ void run1(const uint32_t* xsp, int R, float* red) {
    mma(0, true, [](int) -> const WE* { return nullptr; }, xsp, R, red);
    lds_barrier();
  }
  __device__ __forceinline__ float psum(const float* red, int r, int m) const {
    const int t = r >> 4, i = r & 15;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) s += red[((w * NT + t) << 8) + (i << 4) + m];
    return s;
  }
  // whole product for nrows rows: tile groups of NT, weights of the first group preloaded
  template <typename RowPtr>
  __device__ __forceinline__ void run(RowPtr rowptr, const uint32_t* xsp, int R, float* red, float* out,
                                      const float* rstd) {
    for (int tb = 0; tb < ntiles; tb += NT) {
      mma(tb, tb == 0, rowptr, xsp, R, red);
      lds_barrier();
      reduce(red, out, rstd, tb);
      lds_barrier();
    }
  }
};

// This thread's chunk of the staged activations xs[MR][ld] (k = kc*EPC ..),
// times g[e] when g != nullptr; sq[m] = sum of squares of the raw chunk.
// Threads outside the row groups get zeros.
template <int MR, int EPC>
__device__ __forceinline__ void chunk_from_lds(const float* xs, int ld, int kc, bool active, const float* g,
                                               float (&xg)[MR][EPC], float (&sq)[MR]) {
#pragma unroll
  for (int m = 0; m < MR; ++m) {
    float s2 = 0.f;
#pragma unroll
    for (int e = 0; e < EPC; ++e) {
      const float x = active ? xs[m * ld + kc * EPC + e] : 0.f;
      s2 = fmaf(x, x, s2);
      xg[m][e] = g ? x * g[e] : x;
    }
    sq[m] = s2;
  }
}

// Stage R rows of a parity activation buffer [kMaxRows][ncols] into LDS
// xs[MR][ncols] (rows >= R zero-filled).
template <int MR>
__device__ __forceinline__ bool stage_par(const Ctx& c, const uint32_t* src, int ncols, int R, uint32_t par, float* xs) {
  for (int i = tid(); i < (MR - R) * ncols; i += kThreads) xs[R * ncols + i] = 0.f;
  const bool ok = poll_quads(
      c, R * ncols / 4, par, [=](int i) { return src + 4 * i; },
      [=](int i, W16 w) {
#pragma unroll
        for (int e = 0; e < 4; ++e) xs[4 * i + e] = __uint_as_float(w[e]);
      });
  return wg_sync_ok(c, ok);
}

// rstd[m] = 1 / sqrt(mean(xs[m]^2) + eps) for m < R, 0 above.
template <int MR>
__device__ __forceinline__ void row_rstd(const Ctx& c, const float* xs, int ncols, int R) {
  const int lane = tid() & 63, wave = tid() >> 6;
  for (int m = wave; m < MR; m += kWaves) {
    float s = 0.f;
    if (m < R)
      for (int k = lane; k < ncols; k += 64) s += xs[m * ncols + k] * xs[m * ncols + k];
    s = wave_sum63(s);
    if (lane == 63) c.sh->rstd[m] = m < R ? __builtin_amdgcn_rsqf(s / (float)ncols + (float)c.p->rms_eps) : 0.f;
  }
  __syncthreads();
}

// ------------------------------------------------------------- pass phases

// Layer-0 input rows: position 0 = frame hidden vector, position s >= 1 = E_{s-1}[code consumed at s].
template <typename WT, int MR>
__device__ __forceinline__ void gather_rows(const Ctx& c, float* xs) {
  const KParams* p = c.p;
  const Shared* sh = c.sh;
  const int H = p->H, R = sh->rows;
  for (int i = tid(); i < MR * H; i += kThreads) {
    int r = i / H, k = i % H;
    float v = 0.f;
    if (r < R) {
      int s = sh->first_pos + r;
      if (s == 0) {
        v = G(sh->fa.frame_hidden)[k];
      } else {
        const WT* tab = wptr<WT>(p, p->o_emb0 + (uint64_t)(s - 1) * p->table_stride);
        v = WTraits<WT>::one(tab, (size_t)sh->in_code[s] * H + k);
      }
    }
    xs[i] = v;
  }
  __syncthreads();
}

// Layer-0 input rows of the bf16 path, gathered straight into the split layout
// (as stage_split does for the exchanged rows): chunk (m, q) = 8 values of row m,
// one 16-byte embedding load; this workgroup's residual columns go to xown, the
// gain-scaled values to xsp, and one sum of squares per wave (64 chunks of one
// row, hidden a multiple of 512) to sqc. Rows R.. of xown are zero.
template <typename WE, int MR>
__device__ __forceinline__ void gather_split_rows(const Ctx& c, uint32_t* xsp, const float* gain, float* sqc) {
  const KParams* p = c.p;
  const Shared* sh = c.sh;
  const int H = p->H, R = sh->rows, nch = H >> 3, total = R * nch;
  const int o0 = blockIdx.x * c.cpw;
  for (int i = tid(); i < kMaxRows * c.cpw; i += kThreads)
    if (i / c.cpw >= R || o0 + i % c.cpw >= H) c.xown[i] = 0.f;
  for (int base = 0; base < total; base += kThreads) {
    const int idx = base + tid();
    float s2 = 0.f;
    if (idx < total) {
      const int m = idx / nch, q = idx - m * nch, s = sh->first_pos + m;
      float x[8];
      if (s == 0) {
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = G(sh->fa.frame_hidden)[8 * q + e];
      } else if constexpr (IsI8<WE>::value) {
        // int8 row: 8 codes times the row's scale
        const uint64_t toff = p->o_emb0 + (uint64_t)(s - 1) * p->table_stride;
        const int code = sh->in_code[s];
        const uint64_t w = *G(reinterpret_cast<const uint64_t*>(p->wbase + toff + (size_t)code * H + 8 * q));
        const float sc = row_scale<WE>(p, toff, p->V, H, code);
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = (float)(int8_t)(uint8_t)(w >> (8 * e)) * sc;
      } else {
        const bf16_t* tab = wptr<bf16_t>(p, p->o_emb0 + (uint64_t)(s - 1) * p->table_stride);
        const W16 w = *G(reinterpret_cast<const W16*>(tab + (size_t)sh->in_code[s] * H + 8 * q));
        WTraits<bf16_t>::widen(w, x);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int j = 8 * q + e - o0;
        if (j >= 0 && j < c.cpw) c.xown[m * c.cpw + j] = x[e];
        s2 = fmaf(x[e], x[e], s2);
        x[e] *= G(gain)[8 * q + e];
      }
      put_split(xsp, split_stride(H), m, q, x);
    }
    const int i0 = base + (tid() & ~63);
    if (i0 < total) {
      s2 = wave_sum63(s2);
      if ((tid() & 63) == 63) sqc[i0 >> 6] = s2;
    }
  }
  __syncthreads();
}

template <typename WT, int MR, int RPT>
__device__ __forceinline__ bool phase_qkv(const Ctx& c, int l) {
  const KParams* p = c.p;
  const Shared* sh = c.sh;
  const int H = p->H, R = sh->rows, N = p->nqkv;
  const int rpw = (N + p->nwg - 1) / p->nwg, row0 = blockIdx.x * rpw;
  const int nrows = max(0, min(rpw, N - row0));
  const WT* wq = wptr<WT>(p, layer_off(p, l, p->o_wq));
  const WT* wk = wptr<WT>(p, layer_off(p, l, p->o_wk));
  const WT* wv = wptr<WT>(p, layer_off(p, l, p->o_wv));
  const int qd = p->qdim, kd = p->kvdim;
  auto rowptr = [&](int r) -> const WT* {
    int o = row0 + r;
    if (o < qd) return wq + (size_t)o * H;
    if (o < qd + kd) return wk + (size_t)(o - qd) * H;
    return wv + (size_t)(o - qd - kd) * H;
  };
  Gemv<WT, MR, RPT> g;
  g.setup(H, nrows);
  g.load(0, rowptr);
  g.load_gain(fptr(p, layer_off(p, l, p->o_attn_norm)));
  float* xs = c.work;
  float* out = c.work + MR * H;
  if (l == 0) {
    gather_rows<WT, MR>(c, xs);
    // keep this workgroup's residual columns
    const int o0 = blockIdx.x * c.cpw;
    for (int i = tid(); i < kMaxRows * c.cpw; i += kThreads) {
      int m = i / c.cpw, j = i % c.cpw;
      c.xown[i] = (m < MR && o0 + j < H) ? xs[m * H + o0 + j] : 0.f;
    }
  } else {
    if (nrows == 0) return true;
    if (!stage_par<MR>(c, p->xb, H, R, kParDown, xs)) return false;
  }
  if (nrows > 0) {
    float xg[MR][Gemv<WT, MR, RPT>::EPC], sq[MR];
    chunk_from_lds<MR, Gemv<WT, MR, RPT>::EPC>(xs, H, g.kc, g.active, g.gain, xg, sq);
    g.run(c, xg, rowptr, out, sq);
    const uint32_t par = par_layer(c, sh->pass, l);
    for (int i = tid(); i < MR * nrows; i += kThreads) {
      const int m = i / nrows, r = i % nrows;
      pstore(p->qkvb + (size_t)m * N + row0 + r, m < R ? out[r * MR + m] : 0.f, par);
    }
  }
  // the next phase reuses the work area: no wave may still be reading it
  lds_barrier();
  return true;
}

// Attention for query head h = blockIdx.x (h < nq): per-head RMSNorm of q and k,
// rotate-half RoPE, causal softmax over positions 0..s of each row, output to
// attnb. The KV cache of the head lives in device memory ([L][kMaxPos][2][d],
// k after norm and RoPE, v raw); the positions committed by earlier passes are
// prefetched into LDS while the workgroup waits for this pass's q, k and v.
// In LDS each position's k and v are padded to 2d + 4 floats so that the 16
// positions read by one wave fall on different banks.
// phase_attn for a head dimension D known at compile time (the 1024-wide model's 128): every
// per-lane loop has a fixed trip count (no per-element lane masks), the weighted value sum reads
// 16 bytes per lane (lane = position group gi, dimensions 4 li .. 4 li + 3; the groups are added
// across the wave in a fixed order), and the output goes out as one 16-byte parity store per lane.
template <int MR, int D>
__device__ __forceinline__ bool phase_attn_d(const Ctx& c, int l) {
  const KParams* p = c.p;
  const Shared* sh = c.sh;
  const int h = blockIdx.x;
  constexpr int half = D / 2;
  const int R = sh->rows, N = p->nqkv, fp = sh->first_pos;
  const int g = h / (p->nq / p->nkv);
  const int qoff = h * D, koff = p->qdim + g * D;
  constexpr int ps = 2 * D + 4;    // LDS floats per position
  float* qs = c.work;              // [kMaxRows][D], then ks, vs
  float* ks = qs + kMaxRows * D;
  float* vs = ks + kMaxRows * D;
  float* kv = vs + kMaxRows * D;   // [kMaxPos][ps]: k, v of every position
  float* pw_lds = kv + kMaxPos * ps;  // [kMaxRows][kMaxPos] softmax weights of each row
  uint64_t* gkv = reinterpret_cast<uint64_t*>(p->kvc + ((size_t)h * p->L + l) * kMaxPos * 2 * D);
  const int lane = tid() & 63, wave = tid() >> 6;
  // past positions 0 .. fp-1: issue the loads now, store them to LDS after the wait
  constexpr int KVW = (kMaxPos * D + kThreads - 1) / kThreads;  // 64-bit words per thread
  const int past_words = fp * D;
  uint64_t pw[KVW];
#pragma unroll
  for (int i = 0; i < KVW; ++i) {
    const int wi = tid() + i * kThreads;
    pw[i] = wi < past_words ? xload(gkv + wi) : 0ull;
  }
  const uint32_t par = par_layer(c, sh->pass, l);
  constexpr int d4 = D / 4;
  const int rd4 = R * d4, kvdim = p->kvdim;
  const uint32_t* qkvb = p->qkvb;
  bool ok = poll_quads(
      c, 3 * rd4, par,
      [=](int i) {
        const int part = i / rd4, rem = i - part * rd4, r = rem / d4, k = 4 * (rem - r * d4);
        const int off = part == 0 ? qoff : koff + (part - 1) * kvdim;
        return qkvb + (size_t)r * N + off + k;
      },
      [=](int i, W16 w) {
        const int part = i / rd4, rem = i - part * rd4;
        *reinterpret_cast<W16*>(qs + part * kMaxRows * D + 4 * rem) = w;
      });
#pragma unroll
  for (int i = 0; i < KVW; ++i) {
    const int wi = tid() + i * kThreads;
    if (wi < past_words) {
      const int pos = wi / D, w = wi - pos * D;
      reinterpret_cast<uint64_t*>(kv + (size_t)pos * ps)[w] = pw[i];
    }
  }
  if (!wg_sync_ok(c, ok)) return false;
  // per-head RMSNorm + RoPE of q (vectors 0..R-1) and k (R..2R-1), one half-wave per vector;
  // lane i of the half holds dimensions i + 32 j (j < D / 64) and their partners i + 32 j + D/2
  const float* qn = c.attn_const + (size_t)l * 2 * D;
  const float* kn = qn + D;
  const float* rope = c.attn_const + (size_t)p->L * 2 * D;
  constexpr int J = D / 64;
  const int hl = lane & 31;
  for (int v = 2 * wave + (lane >> 5); v < 2 * R; v += 2 * kWaves) {
    const bool isq = v < R;
    const int r = isq ? v : v - R;
    const float* x = isq ? qs + r * D : ks + r * D;
    const float* gn = isq ? qn : kn;
    const int pos = fp + r;
    float a[J], b[J], ga[J], gb[J], cs[J], sn[J];
    float s2 = 0.f;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int i = hl + 32 * j;
      a[j] = x[i];
      b[j] = x[i + half];
      ga[j] = gn[i];
      gb[j] = gn[i + half];
      cs[j] = rope[(pos * half + i) * 2];
      sn[j] = rope[(pos * half + i) * 2 + 1];
      s2 = fmaf(a[j], a[j], fmaf(b[j], b[j], s2));
    }
    float* dst = isq ? qs + r * D : kv + (size_t)pos * ps;
    // 1 / sqrt(mean of squares + eps) through the hardware reciprocal square root (1 ulp)
    const float rs = p->qk_norm ? __builtin_amdgcn_rsqf(half_sum(s2) * (1.f / (float)D) + (float)p->rms_eps) : 1.f;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int i = hl + 32 * j;
      float u = a[j], w = b[j];
      if (p->qk_norm) {
        u = u * rs * ga[j];
        w = w * rs * gb[j];
      }
      dst[i] = u * cs[j] - w * sn[j];
      dst[i + half] = w * cs[j] + u * sn[j];
    }
    if (!isq) {
#pragma unroll
      for (int j = 0; j < D / 32; ++j) kv[(size_t)pos * ps + D + hl + 32 * j] = vs[r * D + hl + 32 * j];
    }
  }
  __syncthreads();
  // device copy of the new k, v for later passes: the stores go out while the scores are computed
  for (int wi = tid(); wi < R * D; wi += kThreads) {
    const int pos = fp + wi / D, w = wi % D;
    __hip_atomic_store(G(gkv + (size_t)pos * D + w), reinterpret_cast<const uint64_t*>(kv + (size_t)pos * ps)[w],
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  // one wave per row. Scores: lane = (position t = lane / 4, quarter qj of the dimensions)
  const float scale = 1.f / sqrtf((float)D);
  const int npos = fp + R;  // positions holding this pass's keys and values
  constexpr int DQ = D / 4;
  constexpr int LPD = D / 4;                     // lanes per position group
  constexpr int NG = LPD >= 64 ? 1 : 64 / LPD;   // position groups
  constexpr int PPG = kMaxPos / NG;              // positions per group
  const int t = lane >> 2, qj = lane & 3;
  const int gi = lane / LPD, li = lane - gi * LPD;
  for (int r = wave; r < MR; r += kWaves) {
    if (r < R) {
      const int last = fp + r;
      float part = 0.f;
      if (t <= last) {
        const f32x4* qv = reinterpret_cast<const f32x4*>(qs + r * D + qj * DQ);
        const f32x4* kk = reinterpret_cast<const f32x4*>(kv + (size_t)t * ps + qj * DQ);
        float p0 = 0.f, p1 = 0.f;
#pragma unroll
        for (int e = 0; e < DQ / 4; ++e) {
          const f32x4 qa = qv[e], ka = kk[e];
          p0 = fmaf(qa.x, ka.x, p0);
          p1 = fmaf(qa.y, ka.y, p1);
          p0 = fmaf(qa.z, ka.z, p0);
          p1 = fmaf(qa.w, ka.w, p1);
        }
        part = p0 + p1;
      }
      part += dpp<0xB1>(part);
      part += dpp<0x4E>(part);
      const float sc = t <= last ? part * scale : -INFINITY;
      const float rm = row16_max(sc);
      const float mx = fmaxf(fmaxf(lane_val(rm, 15), lane_val(rm, 31)), fmaxf(lane_val(rm, 47), lane_val(rm, 63)));
      const float e = t <= last ? expf(sc - mx) : 0.f;
      const float rsum = row16_sum(qj == 0 ? e : 0.f);
      const float z = (lane_val(rsum, 15) + lane_val(rsum, 31)) + (lane_val(rsum, 47) + lane_val(rsum, 63));
      const float pr = e * __builtin_amdgcn_rcpf(z);
      // the row's weights go through LDS (written and read back by this wave only, in order);
      // positions at or past npos read the finite row npos - 1 (weight 0) instead of unset rows
      float* pwr = pw_lds + r * kMaxPos;
      if (qj == 0) pwr[t] = pr;
      f32x4 o = {0.f, 0.f, 0.f, 0.f};
      if (gi < NG) {
        f32x4 wq[PPG / 4];
#pragma unroll
        for (int q4 = 0; q4 < PPG / 4; ++q4) wq[q4] = reinterpret_cast<const f32x4*>(pwr + gi * PPG)[q4];
        f32x4 vv[PPG];
#pragma unroll
        for (int k = 0; k < PPG; ++k)
          vv[k] = *reinterpret_cast<const f32x4*>(kv + (size_t)min(gi * PPG + k, npos - 1) * ps + D + 4 * li);
#pragma unroll
        for (int k = 0; k < PPG; ++k) {
          const float w = wq[k >> 2][k & 3];
          o.x = fmaf(w, vv[k].x, o.x);
          o.y = fmaf(w, vv[k].y, o.y);
          o.z = fmaf(w, vv[k].z, o.z);
          o.w = fmaf(w, vv[k].w, o.w);
        }
      }
#pragma unroll
      for (int xo = LPD; xo < 64 && NG > 1; xo <<= 1) {
        o.x += __shfl_xor(o.x, xo, 64);
        o.y += __shfl_xor(o.y, xo, 64);
        o.z += __shfl_xor(o.z, xo, 64);
        o.w += __shfl_xor(o.w, xo, 64);
      }
      if (gi == 0) pstore4(p->attnb + (size_t)r * p->qdim + qoff + 4 * li, o.x, o.y, o.z, o.w, par);
    } else {
#pragma unroll
      for (int j = 0; j < (D + 63) / 64; ++j)
        if (lane + 64 * j < D) pstore(p->attnb + (size_t)r * p->qdim + qoff + lane + 64 * j, 0.f, par);
    }
  }
  // the next phase reuses the work area: no wave may still be reading it
  lds_barrier();
  return true;
}

template <int MR>
__device__ __forceinline__ bool phase_attn(const Ctx& c, int l) {
  const KParams* p = c.p;
  const Shared* sh = c.sh;
  const int h = blockIdx.x;
  if (h >= p->nq) return true;
  if (p->d == 128) return phase_attn_d<MR, 128>(c, l);
  const int d = p->d, R = sh->rows, N = p->nqkv, fp = sh->first_pos, half = d / 2;
  const int g = h / (p->nq / p->nkv);
  const int qoff = h * d, koff = p->qdim + g * d;
  const int ps = 2 * d + 4;        // LDS floats per position
  float* qs = c.work;              // [kMaxRows][d], then ks, vs
  float* ks = qs + kMaxRows * d;
  float* vs = ks + kMaxRows * d;
  float* kv = vs + kMaxRows * d;   // [kMaxPos][ps]: k, v of every position
  float* pw_lds = kv + kMaxPos * ps;  // [kMaxRows][kMaxPos] softmax weights of each row
  uint64_t* gkv = reinterpret_cast<uint64_t*>(p->kvc + ((size_t)h * p->L + l) * kMaxPos * 2 * d);
  const int lane = tid() & 63, wave = tid() >> 6;
  // past positions 0 .. fp-1: issue the loads now, store them to LDS after the wait
  constexpr int KVW = 8;  // 64-bit words per thread: up to 16 positions x 2 x 128 floats
  const int past_words = fp * d;  // fp * 2d floats = fp * d words
  uint64_t pw[KVW];
#pragma unroll
  for (int i = 0; i < KVW; ++i) {
    const int wi = tid() + i * kThreads;
    pw[i] = wi < past_words ? xload(gkv + wi) : 0ull;
  }
  const uint32_t par = par_layer(c, sh->pass, l);
  // q of head h, k and v of kv head g, for every row of the pass (groups of four words);
  // qs, ks, vs are consecutive [kMaxRows][d] blocks and v of kv head g follows k at +kvdim
  const int rd4 = R * d / 4, d4 = d / 4, kvdim = p->kvdim;
  const uint32_t* qkvb = p->qkvb;
  bool ok = poll_quads(
      c, 3 * rd4, par,
      [=](int i) {
        const int part = i / rd4, rem = i - part * rd4, r = rem / d4, k = 4 * (rem - r * d4);
        const int off = part == 0 ? qoff : koff + (part - 1) * kvdim;
        return qkvb + (size_t)r * N + off + k;
      },
      [=](int i, W16 w) {
        const int part = i / rd4, rem = i - part * rd4;
#pragma unroll
        for (int e = 0; e < 4; ++e) qs[part * kMaxRows * d + 4 * rem + e] = __uint_as_float(w[e]);
      });
#pragma unroll
  for (int i = 0; i < KVW; ++i) {
    const int wi = tid() + i * kThreads;
    if (wi < past_words) {
      const int pos = wi / d, w = wi - pos * d;
      reinterpret_cast<uint64_t*>(kv + (size_t)pos * ps)[w] = pw[i];
    }
  }
  if (!wg_sync_ok(c, ok)) return false;
  // per-head RMSNorm + RoPE of q (vectors 0..R-1) and k (R..2R-1), one half-wave
  // per vector; lane i of the half holds dimensions i + 32 j and their rotation
  // partners i + 32 j + d/2.
  const float* qn = c.attn_const + (size_t)l * 2 * d;
  const float* kn = qn + d;
  const float* rope = c.attn_const + (size_t)p->L * 2 * d;
  const int hl = lane & 31;
  for (int v = 2 * wave + (lane >> 5); v < 2 * R; v += 2 * kWaves) {
    const bool isq = v < R;
    const int r = isq ? v : v - R;
    const float* x = isq ? qs + r * d : ks + r * d;
    const float* gn = isq ? qn : kn;
    const int pos = fp + r;
    float a[4], b[4];
    float s2 = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = hl + 32 * j;
      a[j] = i < half ? x[i] : 0.f;
      b[j] = i < half ? x[i + half] : 0.f;
      s2 = fmaf(a[j], a[j], fmaf(b[j], b[j], s2));
    }
    float* dst = isq ? qs + r * d : kv + (size_t)pos * ps;
    const float rs = p->qk_norm ? __builtin_amdgcn_rsqf(half_sum(s2) / (float)d + (float)p->rms_eps) : 1.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = hl + 32 * j;
      if (i < half) {
        float u = a[j], w = b[j];
        if (p->qk_norm) {
          u = u * rs * gn[i];
          w = w * rs * gn[i + half];
        }
        const float cs = rope[(pos * half + i) * 2], sn = rope[(pos * half + i) * 2 + 1];
        dst[i] = u * cs - w * sn;
        dst[i + half] = w * cs + u * sn;
      }
    }
    if (!isq) {
      // v of this row next to its k
      for (int i = hl; i < d; i += 32) kv[(size_t)pos * ps + d + i] = vs[r * d + i];
    }
  }
  __syncthreads();
  // device copy of the new k, v for later passes: the stores go out while the scores are computed
  for (int wi = tid(); wi < R * d; wi += kThreads) {
    const int pos = fp + wi / d, w = wi % d;
    __hip_atomic_store(G(gkv + (size_t)pos * d + w), reinterpret_cast<const uint64_t*>(kv + (size_t)pos * ps)[w],
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  // one wave per row: lane = (position t = lane / 4, quarter j = lane % 4 of the dimensions)
  const float scale = 1.f / sqrtf((float)d);
  const int npos = fp + R;  // positions holding this pass's keys and values
  const int t = lane >> 2, qj = lane & 3, dq = d / 4;
  for (int r = wave; r < MR; r += kWaves) {
    if (r < R) {
      const int last = fp + r;  // causal: positions 0 .. last
      float part = 0.f;
      if (t <= last) {
        const float4* qv = reinterpret_cast<const float4*>(qs + r * d + qj * dq);
        const float4* kk = reinterpret_cast<const float4*>(kv + (size_t)t * ps + qj * dq);
        float p0 = 0.f, p1 = 0.f;
#pragma unroll 4
        for (int e = 0; e < dq / 4; ++e) {
          const float4 qa = qv[e], ka = kk[e];
          p0 = fmaf(qa.x, ka.x, p0);
          p1 = fmaf(qa.y, ka.y, p1);
          p0 = fmaf(qa.z, ka.z, p0);
          p1 = fmaf(qa.w, ka.w, p1);
        }
        part = p0 + p1;
      }
      part += dpp<0xB1>(part);  // quad sums: xor 1, xor 2
      part += dpp<0x4E>(part);
      const float sc = t <= last ? part * scale : -INFINITY;
      const float rm = row16_max(sc);
      const float mx = fmaxf(fmaxf(lane_val(rm, 15), lane_val(rm, 31)), fmaxf(lane_val(rm, 47), lane_val(rm, 63)));
      const float e = t <= last ? expf(sc - mx) : 0.f;
      const float rsum = row16_sum(qj == 0 ? e : 0.f);
      const float z = (lane_val(rsum, 15) + lane_val(rsum, 31)) + (lane_val(rsum, 47) + lane_val(rsum, 63));
      const float pr = e * __builtin_amdgcn_rcpf(z);
      // the row's weights go through LDS (written and read back by this wave only, in order)
      // and come back to every lane as four 16-byte broadcasts
      float* pwr = pw_lds + r * kMaxPos;
      if (qj == 0) pwr[t] = pr;
      f32x4 pq[kMaxPos / 4];
#pragma unroll
      for (int q4 = 0; q4 < kMaxPos / 4; ++q4) pq[q4] = reinterpret_cast<const f32x4*>(pwr)[q4];
      // o[r][i] = sum_t pr_t v[t][i] for i = lane + 64 j (head_dim <= 256). Positions after this
      // row's own carry weight 0; those at or past npos read the finite row npos - 1 instead
      // of their unset LDS rows, so all the value loads are issued before the products.
      float vv[kMaxPos][4];
#pragma unroll
      for (int tt = 0; tt < kMaxPos; ++tt)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          vv[tt][j] = lane + 64 * j < d ? kv[(size_t)min(tt, npos - 1) * ps + d + lane + 64 * j] : 0.f;
      float o[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int tt = 0; tt < kMaxPos; ++tt)
#pragma unroll
        for (int j = 0; j < 4; ++j) o[j] = fmaf(pq[tt >> 2][tt & 3], vv[tt][j], o[j]);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (lane + 64 * j < d) pstore(p->attnb + (size_t)r * p->qdim + qoff + lane + 64 * j, o[j], par);
    } else {
      for (int i = lane; i < d; i += 64) pstore(p->attnb + (size_t)r * p->qdim + qoff + i, 0.f, par);
    }
  }
  // the next phase reuses the work area: no wave may still be reading it
  lds_barrier();
  return true;
}

// O projection (layer l) or down projection: x_own += W * act; publish x_own.
template <typename WT, int MR, int RPT>
__device__ __forceinline__ bool phase_proj(const Ctx& c, int l, bool is_down) {
  const KParams* p = c.p;
  const Shared* sh = c.sh;
  const int H = p->H, R = sh->rows;
  const int K = is_down ? p->F : p->qdim;
  const int row0 = blockIdx.x * c.cpw;
  const int nrows = max(0, min(c.cpw, H - row0));
  const WT* W = wptr<WT>(p, layer_off(p, l, is_down ? p->o_wd : p->o_wo));
  auto rowptr = [&](int r) -> const WT* { return W + (size_t)(row0 + r) * K; };
  if (nrows == 0) return true;
  Gemv<WT, MR, RPT> g;
  g.setup(K, nrows);
  g.load(0, rowptr);
  const uint32_t* src = is_down ? p->actb : p->attnb;
  const uint32_t par = par_layer(c, sh->pass, l);
  constexpr int EPC = Gemv<WT, MR, RPT>::EPC;
  float xg[MR][EPC];
  float* out = c.work + (size_t)MR * p->stage_cols;
  if (K <= p->stage_cols) {
    float* xs = c.work;
    if (!stage_par<MR>(c, src, K, R, par, xs)) return false;
    float sq[MR];
    chunk_from_lds<MR, EPC>(xs, K, g.kc, g.active, (const float*)nullptr, xg, sq);
  } else {
    // one thread per chunk (n_rg == 1): poll this thread's chunk of every row directly,
    // all MR * EPC/2 pairs in flight at once
    bool ok = true;
#pragma unroll
    for (int m = 0; m < MR; ++m)
#pragma unroll
      for (int e = 0; e < EPC; ++e) xg[m][e] = 0.f;
    if (g.active) {
      constexpr int NP = MR * (EPC / 2);
      bool got[NP];
#pragma unroll
      for (int q = 0; q < NP; ++q) got[q] = (q / (EPC / 2)) >= R;
      uint64_t t0 = 0;
      int spins = 0;
      while (true) {
        uint64_t v[NP];
#pragma unroll
        for (int q = 0; q < NP; ++q)
          if (!got[q]) v[q] = pload2(src + (size_t)(q / (EPC / 2)) * K + (size_t)g.kc * EPC + 2 * (q % (EPC / 2)));
        bool all = true;
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          if (!got[q]) {
            const uint32_t lo = (uint32_t)v[q], hi = (uint32_t)(v[q] >> 32);
            if ((lo & 1u) == par && (hi & 1u) == par) {
              got[q] = true;
              xg[q / (EPC / 2)][2 * (q % (EPC / 2))] = __uint_as_float(lo);
              xg[q / (EPC / 2)][2 * (q % (EPC / 2)) + 1] = __uint_as_float(hi);
            } else {
              all = false;
            }
          }
        }
        if (all) break;
        if ((++spins & 31) == 0) {
          const uint64_t now = dclock();
          if (t0 == 0) t0 = now;
          else if (now - t0 > kTimeoutTicks) { status_raise(p, c.tag_base, RVQSD_ETIMEOUT); ok = false; break; }
          if (status_set(p, c.tag_base)) { ok = false; break; }
        }
      }
    }
    if (!wg_sync_ok(c, ok)) return false;
  }
  if (nrows > 0) {
    g.run(c, xg, rowptr, out);
    const uint32_t xpar = is_down ? kParDown : kParO;
    for (int i = tid(); i < MR * nrows; i += kThreads) {
      const int m = i / nrows, r = i % nrows;
      float v = 0.f;
      if (m < R) {
        v = c.xown[m * c.cpw + r] + out[r * MR + m];
        c.xown[m * c.cpw + r] = v;
      }
      pstore(p->xb + (size_t)m * H + row0 + r, v, xpar);
    }
  }
  __syncthreads();
  return true;
}

template <typename WT, int MR, int RPT>
__device__ __forceinline__ bool phase_gu(const Ctx& c, int l) {
  const KParams* p = c.p;
  const Shared* sh = c.sh;
  const int H = p->H, R = sh->rows, F = p->F;
  const int fpw = (F + p->nwg - 1) / p->nwg, f0 = blockIdx.x * fpw;
  const int nf = max(0, min(fpw, F - f0));
  const WT* wg = wptr<WT>(p, layer_off(p, l, p->o_wg));
  const WT* wu = wptr<WT>(p, layer_off(p, l, p->o_wu));
  auto rowptr = [&](int r) -> const WT* { return ((r & 1) ? wu : wg) + (size_t)(f0 + (r >> 1)) * H; };
  Gemv<WT, MR, RPT> g;
  g.setup(H, 2 * nf);
  g.load(0, rowptr);
  g.load_gain(fptr(p, layer_off(p, l, p->o_mlp_norm)));
  if (nf == 0) return true;
  float* xs = c.work;
  float* out = c.work + MR * H;
  if (!stage_par<MR>(c, p->xb, H, R, kParO, xs)) return false;
  {
    float xg[MR][Gemv<WT, MR, RPT>::EPC], sq[MR];
    chunk_from_lds<MR, Gemv<WT, MR, RPT>::EPC>(xs, H, g.kc, g.active, g.gain, xg, sq);
    g.run(c, xg, rowptr, out, sq);
    const uint32_t par = par_layer(c, sh->pass, l);
    for (int i = tid(); i < MR * nf; i += kThreads) {
      const int m = i / nf, j = i % nf;
      float a = 0.f;
      if (m < R) {
        const float gt = out[(2 * j) * MR + m], up = out[(2 * j + 1) * MR + m];
        a = gt / (1.f + expf(-gt)) * up;
      }
      pstore(p->actb + (size_t)m * F + f0 + j, a, par);
    }
  }
  lds_barrier();  // the work area is reused by the next phase
  return true;
}

// ------------------------------------------------ MFMA phases (bf16, <= 8 rows)
// Same partition of weight rows over workgroups as the phases above; the
// weights of the first round are loaded before the wait for the activations.

template <typename WE, int MR>
__device__ __forceinline__ bool phase_qkv_m(const Ctx& c, int l) {
  const KParams* p = c.p;
  const Shared* sh = c.sh;
  const int H = p->H, R = sh->rows, N = p->nqkv;
  const int rpw = (N + p->nwg - 1) / p->nwg, row0 = blockIdx.x * rpw;
  const int nrows = max(0, min(rpw, N - row0));
  const uint64_t oq = layer_off(p, l, p->o_wq), ok = layer_off(p, l, p->o_wk), ov = layer_off(p, l, p->o_wv);
  const WE* wq = wptr<WE>(p, oq);
  const WE* wk = wptr<WE>(p, ok);
  const WE* wv = wptr<WE>(p, ov);
  const int qd = p->qdim, kd = p->kvdim;
  auto rowptr = [&](int r) -> const WE* {
    const int o = row0 + r;
    if (o < qd) return wq + (size_t)o * H;
    if (o < qd + kd) return wk + (size_t)(o - qd) * H;
    return wv + (size_t)(o - qd - kd) * H;
  };
  MTile<MR, 1, kUptH, WE> mt;
  mt.setup(H, nrows);
  mt.load(0, rowptr);
  const float* gain = fptr(p, layer_off(p, l, p->o_attn_norm));
  uint32_t* xsp = reinterpret_cast<uint32_t*>(c.work);  // [MR][H + 4] split
  float* sqc = c.work + MR * (H + 4);                   // [MR][H/8]
  float* red = sqc + MR * (H >> 3);                     // [kWaves][1][256]
  float* out = red + kWaves * 256;                      // [nrows][MR]
  float* rsc = out + (size_t)((nrows + 15) & ~15) * MR;  // [nrows] row scales (int8 weights)
  // int8: the row scales are loaded into registers with the weights and reach LDS only
  // after the input wait (a store now would wait for every load in flight)
  float sc_reg = 0.f;
  if constexpr (IsI8<WE>::value) {
    if (tid() < nrows) {
      const int o = row0 + tid();
      sc_reg = o < qd ? row_scale<WE>(p, oq, qd, H, o)
                      : (o < qd + kd ? row_scale<WE>(p, ok, kd, H, o - qd) : row_scale<WE>(p, ov, kd, H, o - qd - kd));
    }
  }
  auto scale = [&](int r) -> float {
    if constexpr (IsI8<WE>::value) return rsc[r];
    else return 1.f;
  };
  if (l == 0) {
    gather_split_rows<WE, MR>(c, xsp, gain, sqc);
  } else {
    if (nrows == 0) return true;
    if (!stage_split<2, true>(c, p->xb, H, R, kParDown, gain, xsp, sqc)) return false;
  }
  if constexpr (IsI8<WE>::value)
    if (tid() < nrows) rsc[tid()] = sc_reg;  // read after the tile barrier below
  if (nrows > 0 && mt.ntiles <= 1) {
    mt.run1(xsp, R, red);
    const uint32_t par = par_layer(c, sh->pass, l);
    for (int i = tid(); i < MR * nrows; i += kThreads) {
      const int r = i / MR, m = i - r * MR;
      pstore(p->qkvb + (size_t)m * N + row0 + r, m < R ? mt.psum(red, r, m) * scale(r) * rstd_of(c, sqc, H, m) : 0.f,
             par);
    }
  } else if (nrows > 0) {
    rstd_from_chunks_w(c, sqc, H, R);
    mt.run(rowptr, xsp, R, red, out, sh->rstd);
    const uint32_t par = par_layer(c, sh->pass, l);
    for (int i = tid(); i < MR * nrows; i += kThreads) {
      const int m = i / nrows, r = i % nrows;
      pstore(p->qkvb + (size_t)m * N + row0 + r, m < R ? out[r * MR + m] * scale(r) : 0.f, par);
    }
  }
  lds_barrier();  // the work area is reused by the next phase
  return true;
}

// O projection (layer l) or down projection: x_own += W * act; publish x_own.
template <typename WE, int MR, int CB, int UPT>
__device__ __forceinline__ bool phase_proj_m(const Ctx& c, int l, bool is_down) {
  const KParams* p = c.p;
  const Shared* sh = c.sh;
  const int H = p->H, R = sh->rows;
  const int K = is_down ? p->F : p->qdim;
  const int row0 = blockIdx.x * c.cpw;
  const int nrows = max(0, min(c.cpw, H - row0));
  if (nrows == 0) return true;
  const uint64_t ow = layer_off(p, l, is_down ? p->o_wd : p->o_wo);
  const WE* W = wptr<WE>(p, ow);
  auto rowptr = [&](int r) -> const WE* { return W + (size_t)(row0 + r) * K; };
  MTile<MR, 1, UPT, WE> mt;
  mt.setup(K, nrows);
  mt.load(0, rowptr);
  uint32_t* xsp = reinterpret_cast<uint32_t*>(c.work);  // [MR][K + 4] split
  float* red = c.work + MR * (K + 4);                   // [kWaves][1][256]
  float* out = red + kWaves * 256;                      // [nrows][MR]
  float* rsc = out + (size_t)((nrows + 15) & ~15) * MR;  // [nrows] row scales (int8 weights)
  float sc_reg = 0.f;
  if constexpr (IsI8<WE>::value)
    if (tid() < nrows) sc_reg = row_scale<WE>(p, ow, H, K, row0 + tid());
  auto scale = [&](int r) -> float {
    if constexpr (IsI8<WE>::value) return rsc[r];
    else return 1.f;
  };
  const uint32_t* src = is_down ? p->actb : p->attnb;
  const uint32_t par = par_layer(c, sh->pass, l);
  if (!stage_split<CB, false>(c, src, K, R, par, nullptr, xsp, nullptr)) return false;
  if constexpr (IsI8<WE>::value)
    if (tid() < nrows) rsc[tid()] = sc_reg;
  const uint32_t xpar = is_down ? kParDown : kParO;
  if (mt.ntiles <= 1) {
    mt.run1(xsp, R, red);
    for (int i = tid(); i < MR * nrows; i += kThreads) {
      const int r = i / MR, m = i - r * MR;
      float v = 0.f;
      if (m < R) {
        v = c.xown[m * c.cpw + r] + mt.psum(red, r, m) * scale(r);
        c.xown[m * c.cpw + r] = v;
      }
      pstore(p->xb + (size_t)m * H + row0 + r, v, xpar);
    }
  } else {
    mt.run(rowptr, xsp, R, red, out, nullptr);
    for (int i = tid(); i < MR * nrows; i += kThreads) {
      const int m = i / nrows, r = i % nrows;
      float v = 0.f;
      if (m < R) {
        v = c.xown[m * c.cpw + r] + out[r * MR + m] * scale(r);
        c.xown[m * c.cpw + r] = v;
      }
      pstore(p->xb + (size_t)m * H + row0 + r, v, xpar);
    }
  }
  lds_barrier();  // the work area is reused by the next phase
  return true;
}

// gate and up rows interleaved (2j = gate row f0 + j, 2j + 1 = up row); act = SiLU(gate) * up.
template <typename WE, int MR>
__device__ __forceinline__ bool phase_gu_m(const Ctx& c, int l) {
  const KParams* p = c.p;
  const Shared* sh = c.sh;
  const int H = p->H, R = sh->rows, F = p->F;
  const int fpw = (F + p->nwg - 1) / p->nwg, f0 = blockIdx.x * fpw;
  const int nf = max(0, min(fpw, F - f0));
  if (nf == 0) return true;
  const uint64_t og = layer_off(p, l, p->o_wg), ou = layer_off(p, l, p->o_wu);
  const WE* wg = wptr<WE>(p, og);
  const WE* wu = wptr<WE>(p, ou);
  auto rowptr = [&](int r) -> const WE* { return ((r & 1) ? wu : wg) + (size_t)(f0 + (r >> 1)) * H; };
  MTile<MR, 2, kUptH, WE> mt;
  mt.setup(H, 2 * nf);
  mt.load(0, rowptr);
  uint32_t* xsp = reinterpret_cast<uint32_t*>(c.work);  // [MR][H + 4] split
  float* sqc = c.work + MR * (H + 4);                   // [MR][H/8]
  float* red = sqc + MR * (H >> 3);                     // [kWaves][2][256]
  float* out = red + kWaves * 2 * 256;                  // [2 nf][MR]
  float* rsc = out + (size_t)((2 * nf + 15) & ~15) * MR;  // [2 nf] row scales (int8 weights)
  float sc_reg = 0.f;
  if constexpr (IsI8<WE>::value)
    if (tid() < 2 * nf) sc_reg = row_scale<WE>(p, (tid() & 1) ? ou : og, F, H, f0 + (tid() >> 1));
  auto scale = [&](int r) -> float {
    if constexpr (IsI8<WE>::value) return rsc[r];
    else return 1.f;
  };
  const float* gain = fptr(p, layer_off(p, l, p->o_mlp_norm));
  if (!stage_split<2, true>(c, p->xb, H, R, kParO, gain, xsp, sqc)) return false;
  if constexpr (IsI8<WE>::value)
    if (tid() < 2 * nf) rsc[tid()] = sc_reg;
  const uint32_t par = par_layer(c, sh->pass, l);
  if (mt.ntiles <= 2) {
    mt.run1(xsp, R, red);
    for (int i = tid(); i < MR * nf; i += kThreads) {
      const int j = i / MR, m = i - j * MR;
      float a = 0.f;
      if (m < R) {
        const float rs = rstd_of(c, sqc, H, m);
        const float gt = mt.psum(red, 2 * j, m) * scale(2 * j) * rs, up = mt.psum(red, 2 * j + 1, m) * scale(2 * j + 1) * rs;
        a = gt / (1.f + expf(-gt)) * up;
      }
      pstore(p->actb + (size_t)m * F + f0 + j, a, par);
    }
  } else {
    rstd_from_chunks_w(c, sqc, H, R);
    mt.run(rowptr, xsp, R, red, out, sh->rstd);
    for (int i = tid(); i < MR * nf; i += kThreads) {
      const int m = i / nf, j = i % nf;
      float a = 0.f;
      if (m < R) {
        const float gt = out[(2 * j) * MR + m] * scale(2 * j), up = out[(2 * j + 1) * MR + m] * scale(2 * j + 1);
        a = gt / (1.f + expf(-gt)) * up;
      }
      pstore(p->actb + (size_t)m * F + f0 + j, a, par);
    }
  }
  lds_barrier();  // the work area is reused by the next phase
  return true;
}

// Pass geometry helpers ---------------------------------------------------
// verify rows: prefix -> row 1 only; later passes -> every row.
__device__ __forceinline__ bool is_verify_row(const Shared* sh, int r) { return sh->pass == 0 ? r == 1 : true; }
// rows whose position can become the next anchor (and therefore need drafts)
__device__ __forceinline__ int drafts_of_row(const KParams* p, const Shared* sh, int r) {
  const int s = sh->first_pos + r;
  if (s < 1 || s > p->n_codes - 1) return 0;
  if (sh->pass == 0 && r != 1) return 0;
  return min(p->K, p->n_codes - s);
}
__device__ __forceinline__ int draft_slot(const KParams* p, int r, int j) { return kSlotDraft0 + r * p->K + (j - 1); }

template <typename WT, int MR, int RPT>
__device__ __forceinline__ bool phase_heads(const Ctx& c) {
  const KParams* p = c.p;
  Shared* sh = c.sh;
  const int H = p->H, R = sh->rows, V = p->V, L = p->L;
  // heads touched by this pass
  int t_lo = 1 << 20, t_hi = -1;
  for (int r = 0; r < R; ++r) {
    const int s = sh->first_pos + r;
    if (is_verify_row(sh, r) && s >= 1) { t_lo = min(t_lo, s); t_hi = max(t_hi, s); }
    const int nd = drafts_of_row(p, sh, r);
    if (nd > 0) { t_lo = min(t_lo, s + 1); t_hi = max(t_hi, s + nd); }
  }
  const int nh = t_hi - t_lo + 1;
  const int wph = p->nwg / nh;
  const int hi = blockIdx.x / wph;
  const int t = t_lo + hi;
  const int rpw = (V + wph - 1) / wph, v0 = (blockIdx.x % wph) * rpw;
  const int nrows = hi < nh ? max(0, min(rpw, V - v0)) : 0;
  if (nrows == 0) return true;
  // this head's vectors: (row, offset j); j = 0 is the verify row at position t
  if (tid() == 0) {
    int nv = 0;
    for (int r = 0; r < R && nv < MR; ++r) {
      const int s = sh->first_pos + r;
      if (s == t && is_verify_row(sh, r)) {
        sh->hv_row[nv] = r; sh->hv_off[nv] = 0; sh->hv_slot[nv] = r; ++nv;
      }
      const int nd = drafts_of_row(p, sh, r);
      const int j = t - s;
      if (j >= 1 && j <= nd && nv < MR) {
        sh->hv_row[nv] = r; sh->hv_off[nv] = j; sh->hv_slot[nv] = draft_slot(p, r, j); ++nv;
      }
    }
    sh->hv_n = nv;
  }
  const WT* W = wptr<WT>(p, p->o_lmh1 + (uint64_t)(t - 1) * p->table_stride);
  auto rowptr = [&](int r) -> const WT* { return W + (size_t)(v0 + r) * H; };
  constexpr int RH = RPT;
  Gemv<WT, MR, RH, true> g;
  g.setup(H, nrows);
  g.load(0, rowptr);
  float* xs = c.work;
  float* out = c.work + MR * H;
  if (!stage_par<MR>(c, p->xb, H, R, kParDown, xs)) return false;
  row_rstd<MR>(c, xs, H, R);
  constexpr int EPC = Gemv<WT, MR, RH, true>::EPC;
  float xg[MR][EPC];
  const float* gn = fptr(p, p->o_final_norm);
  const float* ofs = fptr(p, p->o_offsets);
  const int nv = sh->hv_n;
#pragma unroll
  for (int v = 0; v < MR; ++v) {
    const bool use = g.active && v < nv;
    const int vr = use ? sh->hv_row[v] : 0, vo = use ? sh->hv_off[v] : 0;
    const float rs = use ? sh->rstd[vr] : 0.f;
#pragma unroll
    for (int e = 0; e < EPC; ++e) {
      float val = 0.f;
      if (use) {
        const int k = g.kc * EPC + e;
        val = xs[vr * H + k] * rs * G(gn)[k];
        if (vo > 0) val += G(ofs)[(size_t)(vo - 1) * H + k];
      }
      xg[v][e] = val;
    }
  }
  g.run(c, xg, rowptr, out);
  const uint32_t tag = tag_of(c, sh->pass, ph_heads(L));
  for (int i = tid(); i < nv * nrows; i += kThreads) {
    const int v = i / nrows, r = i % nrows;
    xstoref(p->logb + ((size_t)(sh->pass & 1) * p->n_slots + sh->hv_slot[v]) * V + v0 + r, tag, out[r * MR + v]);
  }
  lds_barrier();  // the work area is reused by the next phase
  return true;
}

// LM heads on MFMA: same head/row assignment as phase_heads. The vectors of a
// head (verify rows and h_s + b_j draft rows, final-normed) form the B columns;
// the head's rows are processed in groups of 4 tiles.
template <typename WE, int MR>
__device__ __forceinline__ bool phase_heads_m(const Ctx& c) {
  const KParams* p = c.p;
  Shared* sh = c.sh;
  const int H = p->H, R = sh->rows, V = p->V, L = p->L;
  int t_lo = 1 << 20, t_hi = -1;
  for (int r = 0; r < R; ++r) {
    const int s = sh->first_pos + r;
    if (is_verify_row(sh, r) && s >= 1) { t_lo = min(t_lo, s); t_hi = max(t_hi, s); }
    const int nd = drafts_of_row(p, sh, r);
    if (nd > 0) { t_lo = min(t_lo, s + 1); t_hi = max(t_hi, s + nd); }
  }
  const int nh = t_hi - t_lo + 1;
  const int wph = p->nwg / nh;
  const int hi = blockIdx.x / wph;
  const int t = t_lo + hi;
  const int rpw = (V + wph - 1) / wph, v0 = (blockIdx.x % wph) * rpw;
  const int nrows = hi < nh ? max(0, min(rpw, V - v0)) : 0;
  if (nrows == 0) return true;
  const uint64_t oh = p->o_lmh1 + (uint64_t)(t - 1) * p->table_stride;
  const WE* W = wptr<WE>(p, oh);
  auto rowptr = [&](int r) -> const WE* { return W + (size_t)(v0 + r) * H; };
  constexpr int TG = 5;  // tiles per group
  MTile<MR, TG, kUptH, WE> mt;
  mt.setup(H, nrows);
  mt.load(0, rowptr);
  if (tid() == 0) {
    int nv = 0;
    for (int r = 0; r < R && nv < MR; ++r) {
      const int s = sh->first_pos + r;
      if (s == t && is_verify_row(sh, r)) {
        sh->hv_row[nv] = r; sh->hv_off[nv] = 0; sh->hv_slot[nv] = r; ++nv;
      }
      const int nd = drafts_of_row(p, sh, r);
      const int j = t - s;
      if (j >= 1 && j <= nd && nv < MR) {
        sh->hv_row[nv] = r; sh->hv_off[nv] = j; sh->hv_slot[nv] = draft_slot(p, r, j); ++nv;
      }
    }
    sh->hv_n = nv;
  }
  __syncthreads();
  const int nv = sh->hv_n, nch = H >> 3;
  // this thread's vector chunks: final-norm gain and offset values, fetched before the wait
  constexpr int VC = (MR * 128 + kThreads - 1) / kThreads;  // chunks per thread at hidden <= 1024
  const float* gn = fptr(p, p->o_final_norm);
  const float* ofs = fptr(p, p->o_offsets);
  float* xs = c.work;                                         // [MR][H] fp32
  uint32_t* vsp = reinterpret_cast<uint32_t*>(xs + MR * H);   // [MR][H + 4] split vectors
  float* red = xs + MR * H + MR * (H + 4);                    // [kWaves][TG][256]
  float* out = red + kWaves * TG * 256;                       // [nrows][MR]
  float* rsc = out + (size_t)((nrows + 15) & ~15) * MR;       // [nrows] row scales (int8 weights)
  float sc_reg = 0.f;
  if constexpr (IsI8<WE>::value)
    if (tid() < nrows) sc_reg = row_scale<WE>(p, oh, V, H, v0 + tid());
  for (int base = 0; base < nv * nch; base += VC * kThreads) {
    float gq[VC][8], oq[VC][8];
#pragma unroll
    for (int b = 0; b < VC; ++b) {
      const int idx = base + b * kThreads + tid();
      const int v = idx / nch, q = idx - v * nch;
      const int vo = idx < nv * nch ? sh->hv_off[v] : 0;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        gq[b][e] = idx < nv * nch ? G(gn)[q * 8 + e] : 0.f;
        oq[b][e] = vo > 0 ? G(ofs)[(size_t)(vo - 1) * H + q * 8 + e] : 0.f;
      }
    }
    if (base == 0) {
      if (!stage_par<MR>(c, p->xb, H, R, kParDown, xs)) return false;
      row_rstd<MR>(c, xs, H, R);
    }
#pragma unroll
    for (int b = 0; b < VC; ++b) {
      const int idx = base + b * kThreads + tid();
      if (idx < nv * nch) {
        const int v = idx / nch, q = idx - v * nch, vr = sh->hv_row[v];
        const float rs = sh->rstd[vr];
        float x[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = xs[vr * H + q * 8 + e] * rs * gq[b][e] + oq[b][e];
        put_split(vsp, split_stride(H), v, q, x);
      }
    }
  }
  if constexpr (IsI8<WE>::value)
    if (tid() < nrows) rsc[tid()] = sc_reg;
  __syncthreads();
  mt.run(rowptr, vsp, nv, red, out, nullptr);
  const uint32_t tag = tag_of(c, sh->pass, ph_heads(L));
  for (int i = tid(); i < nv * nrows; i += kThreads) {
    const int v = i / nrows, r = i % nrows;
    float lgt = out[r * MR + v];
    if constexpr (IsI8<WE>::value) lgt *= rsc[r];
    xstoref(p->logb + ((size_t)(sh->pass & 1) * p->n_slots + sh->hv_slot[v]) * V + v0 + r, tag, lgt);
  }
  lds_barrier();  // the work area is reused by the next phase
  return true;
}

__device__ __forceinline__ double ufetch(const Shared* sh, int s, int slot) {
  return (double)sh->uni[(s - 1) * 3 + slot];
}

// Role of this workgroup's slot in the sampling phase: row >= 0 if active;
// j = 0 for a verify row, else draft offset j of that row.
__device__ __forceinline__ void slot_role(const KParams* p, const Shared* sh, int slot, int* row, int* j) {
  *row = -1;
  *j = 0;
  const int R = sh->rows;
  if (slot < kSlotDraft0) {
    if (slot < R && is_verify_row(sh, slot)) *row = slot;
  } else if (p->K > 0) {
    const int q = slot - kSlotDraft0;
    const int r = q / p->K, jj = q % p->K + 1;
    if (r < R && jj <= drafts_of_row(p, sh, r)) {
      *row = r;
      *j = jj;
    }
  }
}

__device__ __forceinline__ int support_size(const KParams* p) { return p->topk < p->V ? p->topk : p->V; }

template <int MR>
__device__ __forceinline__ bool phase_sample(const Ctx& c) {
  const KParams* p = c.p;
  Shared* sh = c.sh;
  const int V = p->V, slot = blockIdx.x, par = sh->pass & 1;
  int row, j;
  slot_role(p, sh, slot, &row, &j);
  if (row < 0) return true;
  const uint32_t tag = tag_of(c, sh->pass, ph_heads(p->L));
  const uint32_t otag = tag_of(c, sh->pass, ph_sample(p->L));
  float* lg = c.work;                                          // [V]
  int* sidx = reinterpret_cast<int*>(lg + V);                  // [kMaxTopk]
  float* slog = reinterpret_cast<float*>(sidx + kMaxTopk);     // [kMaxTopk]
  // fp64 arrays from the next 8-byte boundary (the work area is 8-byte aligned); an index,
  // not an integer cast of the pointer, so that the compiler keeps them in the LDS address space
  double* prob = reinterpret_cast<double*>(lg + ((V + 2 * kMaxTopk + 1) & ~1));  // [kMaxTopk]
  double* qprob = prob + kMaxTopk;                             // [kMaxTopk]
  double* res = qprob + kMaxTopk;                              // [kMaxTopk]
  int* qidx = reinterpret_cast<int*>(res + kMaxTopk);          // [kMaxTopk]
  const uint64_t* src = p->logb + ((size_t)par * p->n_slots + slot) * V;
  // a verify row with a draft: q of that draft was published by the previous pass, so it
  // is fetched first, while this pass's logits are still on their way
  const int t_pos = sh->first_pos + row + j;
  const int jv_pos = t_pos - sh->m;
  const bool has_draft = j == 0 && sh->pass > 0 && jv_pos <= sh->kp;
  const int nq = p->greedy ? 1 : support_size(p);
  bool ok = true;
  if (has_draft) {
    const int prev_slot = draft_slot(p, sh->prev_anchor_row, jv_pos);
    const uint64_t* rec = p->drec + ((size_t)(par ^ 1) * p->n_slots + prev_slot) * p->drec_words;
    const uint32_t ptag = tag_of(c, sh->pass - 1, ph_sample(p->L));
    ok = poll_range(c, rec + 1, 3 * nq, ptag, [&](int i, uint32_t v) {
      const int e = i / 3, f = i % 3;
      if (f == 0) qidx[e] = (int)v;
      else reinterpret_cast<uint32_t*>(qprob + e)[f - 1] = v;
    });
  }
  if (ok) ok = poll_range(c, src, V, tag, [&](int i, uint32_t v) { lg[i] = __uint_as_float(v); });
  if (!wg_sync_ok(c, ok)) return false;
  if (p->tr_logits && sh->pass < p->tr_max_rounds)
    for (int i = tid(); i < V; i += kThreads)
      G(p->tr_logits)[((size_t)sh->pass * p->n_slots + slot) * V + i] = lg[i];
  unsigned* hist = reinterpret_cast<unsigned*>(qidx + kMaxTopk);  // [kTopkBuckets]
  int n = topk_buckets(&c.sh->tk, lg, V, p->topk, sidx, slog, hist);
  if (n < 0) n = topk_select(&c.sh->tk, lg, V, p->topk, sidx, slog);
  if (tid() < 64) {
    bool fin = false;
    for (int i = tid(); i < n; i += 64) fin |= (slog[i] > -INFINITY && slog[i] < INFINITY);
    if (!__any(fin) && tid() == 0) status_raise(p, c.tag_base, RVQSD_ENUMERIC);
  }
  softmax_support(slog, n, p->temperature, prob);
  __syncthreads();
  const int t = sh->first_pos + row + j;  // code position decided by this slot
  if (j > 0) {
    // draft for position t from the hidden state of `row` plus offset b_j
    uint64_t* rec = p->drec + ((size_t)par * p->n_slots + slot) * p->drec_words;
    if (tid() < 64) {
      int pos;
      if (p->greedy) {
        double best = -1.0;
        int bi = n;
        for (int i = tid(); i < n; i += 64)
          if (prob[i] > best) { best = prob[i]; bi = i; }
        for (int o = 32; o > 0; o >>= 1) {
          double ob = __shfl_xor(best, o, 64);
          int oi = __shfl_xor(bi, o, 64);
          if (ob > best || (ob == best && oi < bi)) { best = ob; bi = oi; }
        }
        pos = bi;
      } else {
        pos = inverse_cdf(prob, n, ufetch(sh, t, 0));
      }
      if (tid() == 0) sh->tok = sidx[pos];
    }
    __syncthreads();
    const int nq = p->greedy ? 1 : n;
    const int tok = sh->tok;
    for (int i = tid(); i < nq; i += kThreads) {
      const int idx = p->greedy ? tok : sidx[i];
      const double pr = p->greedy ? 1.0 : prob[i];
      const uint64_t bits = (uint64_t)__double_as_longlong(pr);
      xstore(rec + 1 + 3 * i + 0, otag, (uint32_t)idx);
      xstore(rec + 1 + 3 * i + 1, otag, (uint32_t)bits);
      xstore(rec + 1 + 3 * i + 2, otag, (uint32_t)(bits >> 32));
    }
    if (tid() == 0) xstore(rec, otag, (uint32_t)tok);
    return true;
  }
  // verify row at position t
  if (has_draft) {
    // accept test of d_t against q_t, drafted last pass from the anchor's row
    if (tid() < 64) {
      const int d = sh->drafts[t];
      double pd = 0.0, qd = 0.0;
      for (int i = tid(); i < n; i += 64)
        if (sidx[i] == d) pd = prob[i];
      for (int i = tid(); i < nq; i += 64)
        if (qidx[i] == d) qd = qprob[i];
      pd = wave_sumd_dpp(pd);
      qd = wave_sumd_dpp(qd);
      const bool accept = ufetch(sh, t, 1) * qd < pd;
      int tok = d;
      if (!accept) {
        // residual max(0, p - q) on p's support; q looked up by binary search (ascending tokens)
        double rs = 0.0;
        for (int i = tid(); i < n; i += 64) {
          const int x = sidx[i];
          int lo = 0, hi2 = nq;
          while (lo < hi2) {
            const int mid = (lo + hi2) >> 1;
            if (qidx[mid] < x) lo = mid + 1;
            else hi2 = mid;
          }
          const double qx = (lo < nq && qidx[lo] == x) ? qprob[lo] : 0.0;
          const double v = prob[i] - qx;
          res[i] = v > 0.0 ? v : 0.0;
          rs += res[i];
        }
        rs = wave_sumd_dpp(rs);
        if (!(rs > 0.0))
          for (int i = tid(); i < n; i += 64) res[i] = prob[i];
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        const int pos = inverse_cdf(res, n, ufetch(sh, t, 2));
        tok = sidx[pos];
      }
      if (tid() == 0) xstore(p->vres + (size_t)par * kMaxRows + row, otag, (uint32_t)tok | (accept ? 0x80000000u : 0u));
    }
  } else {
    // the prefix token c_1, or the extra token after every draft was accepted
    if (tid() < 64) {
      const int pos = inverse_cdf(prob, n, ufetch(sh, t, 2));
      if (tid() == 0) xstore(p->vres + (size_t)par * kMaxRows + row, otag, (uint32_t)sidx[pos]);
    }
  }
  return true;
}

// Read every verdict and every candidate draft token of the pass just sampled
// (one word per thread), commit codes, pick the next anchor and its drafts.
// Returns false on abort. Leaves sh->m == n_codes when the frame is complete.
__device__ __forceinline__ bool commit_and_advance(const Ctx& c) {
  const KParams* p = c.p;
  Shared* sh = c.sh;
  const int n = p->n_codes, par = sh->pass & 1, R = sh->rows, K = p->K;
  const uint32_t tag = tag_of(c, sh->pass, ph_sample(p->L));
  __shared__ uint32_t vr[kMaxRows];
  __shared__ int dtok[kMaxRows][kMaxCodes + 1];
  __shared__ short wlist[kMaxRows * (kMaxCodes + 1)];  // r * 16 + j, j = 0 for the verdict of row r
  __shared__ int nlist;
  if (tid() == 0) {
    int k = 0;
    for (int r = 0; r < R; ++r) {
      if (is_verify_row(sh, r)) wlist[k++] = (short)(r * 16);
      const int nd = drafts_of_row(p, sh, r);
      for (int jj = 1; jj <= nd; ++jj) wlist[k++] = (short)(r * 16 + jj);
    }
    nlist = k;
  }
  __syncthreads();
  bool ok = poll_words(
      c, nlist, tag,
      [=](int i) -> const uint64_t* {
        const int e = wlist[i], r = e >> 4, jj = e & 15;
        if (jj == 0) return p->vres + (size_t)par * kMaxRows + r;
        return p->drec + ((size_t)par * p->n_slots + draft_slot(p, r, jj)) * p->drec_words;
      },
      [&](int i, uint32_t v) {
        const int e = wlist[i], r = e >> 4, jj = e & 15;
        if (jj == 0) vr[r] = v;
        else dtok[r][jj] = (int)v;
      });
  if (!wg_sync_ok(c, ok)) return false;
  if (tid() == 0) {
    const int m = sh->m, kp = sh->kp;
    int m_new = -1, acc = 0, tok = -1;
    if (sh->pass == 0) {
      sh->codes[1] = (int)(vr[1] & 0x7fffffffu);
      m_new = 1;
      tok = sh->codes[1];
    } else {
      for (int j = 1; j <= kp; ++j) {
        const uint32_t v = vr[j - 1];
        if (v & 0x80000000u) {
          sh->codes[m + j] = sh->drafts[m + j];
          ++acc;
          sh->st_mask |= 1u << (m + j);
        } else {
          sh->codes[m + j] = (int)(v & 0x7fffffffu);
          m_new = m + j;
          tok = sh->codes[m_new];
          break;
        }
      }
      if (m_new < 0) {
        if (R > kp) {
          sh->codes[m + kp + 1] = (int)(vr[kp] & 0x7fffffffu);
          m_new = m + kp + 1;
          tok = sh->codes[m_new];
        } else {
          m_new = n;
        }
      }
      sh->st_rounds += 1;
      sh->st_drafted += kp;
      sh->st_accepted += acc;
    }
    sh->st_calls += 1;
    if (blockIdx.x == 0 && p->tr_rounds && sh->pass < p->tr_max_rounds) {
      int32_t* tr = p->tr_rounds + (size_t)sh->pass * kTraceRoundInts;
      tr[0] = m; tr[1] = kp; tr[2] = sh->first_pos; tr[3] = R; tr[4] = m_new; tr[5] = acc; tr[6] = tok;
      tr[7] = sh->pass;
      for (int j = 1; j <= kp; ++j) tr[7 + j] = sh->drafts[m + j];
    }
    if (m_new < n) {
      const int arow = m_new - sh->first_pos;
      const int nd = min(K, n - m_new);
      for (int jj = 1; jj <= nd; ++jj) sh->drafts[m_new + jj] = dtok[arow][jj];
      sh->prev_anchor_row = arow;
      sh->kp = nd;
      sh->rows = min(nd + 1, n - m_new);
      sh->first_pos = m_new + 1;
      sh->in_code[m_new + 1] = sh->codes[m_new];
      for (int r = 1; r < sh->rows; ++r) sh->in_code[m_new + 1 + r] = sh->drafts[m_new + r];
    }
    sh->m = m_new;
    sh->pass += 1;
  }
  __syncthreads();
  return true;
}

// algorithmic bytes one pass must read: layer weights, the heads it touches,
// the gathered embedding rows and the KV cache it attends over
__device__ __forceinline__ unsigned long long pass_bytes(const Ctx& c) {
  const KParams* p = c.p;
  const Shared* sh = c.sh;
  int t_lo = 1 << 20, t_hi = -1;
  for (int r = 0; r < sh->rows; ++r) {
    const int s = sh->first_pos + r;
    if (is_verify_row(sh, r) && s >= 1) { t_lo = min(t_lo, s); t_hi = max(t_hi, s); }
    const int nd = drafts_of_row(p, sh, r);
    if (nd > 0) { t_lo = min(t_lo, s + 1); t_hi = max(t_hi, s + nd); }
  }
  unsigned long long b = (unsigned long long)p->L * p->layer_stride;
  b += (unsigned long long)(t_hi - t_lo + 1) * p->table_stride;
  for (int r = 0; r < sh->rows; ++r) b += (sh->first_pos + r == 0) ? 4ull * p->H : (unsigned long long)p->emb_row_bytes;
  b += (unsigned long long)p->L * (sh->first_pos + sh->rows) * p->nkv * p->d * 2 * 4;
  return b;
}

// One frame: the passes until its 15 codes are committed, then its statistics (workgroup 0)
template <typename WT, int MR, bool MF>
__device__ __forceinline__ void decode_frame(Ctx& c, const FrameArgs& fa) {
  const KParams* p = c.p;
  Shared& shs = *c.sh;
  // every uniform in [0, 1) (NaN fails), or the frame is not decoded and reports EINVAL;
  // every workgroup reads the same table, so all of them agree
  int u_bad = 0;
  if (tid() < 3 * p->n_codes) {
    const float u = G(fa.uniforms)[tid()];
    shs.uni[tid()] = u;
    u_bad = !(u >= 0.f && u < 1.f);
  }
  const bool u_ok = __syncthreads_or(u_bad) == 0;
  c.tag_base = fa.epoch_base;
  c.pass0 = __hip_atomic_load(G(p->pass_count), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  c.rdy = nullptr;
  const uint64_t t_start = dclock();
  const int c0 = fa.c0[0];
  const bool poisoned = c.pass0 == 0xffffffffu;
  const bool c0_ok = c0 >= 0 && c0 < p->V && u_ok && !poisoned;
  if (tid() == 0) {
    shs.fa = fa;
    shs.abort = c0_ok ? 0 : 1;
    shs.pass = 0;
    shs.m = 0;
    shs.kp = 0;
    shs.first_pos = 0;
    shs.rows = 2;
    shs.prev_anchor_row = 0;
    shs.codes[0] = c0;
    shs.in_code[1] = c0;
    shs.st_calls = shs.st_rounds = shs.st_drafted = shs.st_accepted = 0;
    shs.st_mask = 0;
    shs.st_bytes = 0;
  }
  __syncthreads();
  bool ok = c0_ok;
  const int L = p->L;
  while (ok) {
    if (blockIdx.x == 0 && tid() == 0) shs.st_bytes += pass_bytes(c);
    const int nph = phases_per_pass(L) + 1;
    const bool clk_on = blockIdx.x == 0 && p->tr_clock && shs.pass < p->tr_max_rounds;
    uint64_t* clk_row = clk_on ? p->tr_clock + (size_t)shs.pass * nph : nullptr;
    const bool wclk_on = p->tr_wgclock && shs.pass < p->tr_max_rounds;
    uint64_t* wclk = wclk_on ? p->tr_wgclock + (size_t)shs.pass * nph * p->nwg + blockIdx.x : nullptr;
    uint64_t* wrdy = (p->tr_wgready && shs.pass < p->tr_max_rounds)
                         ? p->tr_wgready + (size_t)shs.pass * nph * p->nwg + blockIdx.x
                         : nullptr;
#define RVQSD_READY(ph) c.rdy = wrdy ? wrdy + (size_t)(ph) * p->nwg : nullptr
#define RVQSD_STAMP(ph)                                                   \
  do {                                                                    \
    if (tid() == 0) {                                               \
      if (clk_on) clk_row[(ph)] = dclock();                               \
      if (wclk_on) wclk[(size_t)(ph) * p->nwg] = dclock();                \
    }                                                                     \
  } while (0)
    for (int l = 0; l < L && ok; ++l) {
      RVQSD_READY(5 * l + 0);
      if constexpr (MF) ok = phase_qkv_m<WT, MR>(c, l);
      else ok = phase_qkv<WT, MR, 4>(c, l);
      RVQSD_STAMP(5 * l + 0);
      RVQSD_READY(5 * l + 1);
      if (ok) ok = phase_attn<MR>(c, l);
      RVQSD_STAMP(5 * l + 1);
      RVQSD_READY(5 * l + 2);
      if constexpr (MF) {
        if (ok) ok = phase_proj_m<WT, MR, (MR + 1) / 2, kUptQ>(c, l, false);
      } else {
        if (ok) ok = phase_proj<WT, MR, 4>(c, l, false);
      }
      RVQSD_STAMP(5 * l + 2);
      RVQSD_READY(5 * l + 3);
      if constexpr (MF) {
        if (ok) ok = phase_gu_m<WT, MR>(c, l);
      } else {
        if (ok) ok = phase_gu<WT, MR, (MR <= 8 ? 8 : 4)>(c, l);
      }
      RVQSD_STAMP(5 * l + 3);
      RVQSD_READY(5 * l + 4);
      if constexpr (MF) {
        if (ok) ok = phase_proj_m<WT, MR, (3 * MR + 3) / 4, kUptF>(c, l, true);
      } else {
        if (ok) ok = phase_proj<WT, MR, 4>(c, l, true);
      }
      RVQSD_STAMP(5 * l + 4);
    }
    RVQSD_READY(ph_heads(L));
    if constexpr (MF) {
      if (ok) ok = phase_heads_m<WT, MR>(c);
    } else {
      if (ok) ok = phase_heads<WT, MR, (MR <= 5 ? 8 : 4)>(c);
    }
    RVQSD_STAMP(ph_heads(L));
    RVQSD_READY(ph_sample(L));
    if (ok) ok = phase_sample<MR>(c);
    RVQSD_STAMP(ph_sample(L));
    c.rdy = nullptr;
    ok = wg_sync_ok(c, ok);
    RVQSD_READY(ph_sample(L) + 1);
    if (ok) ok = commit_and_advance(c);
    RVQSD_STAMP(ph_sample(L) + 1);
    if (!ok || shs.m >= p->n_codes) break;
  }
#undef RVQSD_STAMP
#undef RVQSD_READY
  if (ok) {
    // back to parity 1 for the next frame. Every workgroup is past its last read of these words:
    // ending the frame took the last pass's verdicts, hence its logits, hence the residual after
    // the last down projection from every workgroup, each of which had read them all before.
    uint64_t* w2 = reinterpret_cast<uint64_t*>(p->qkvb);
    const int n2 = (int)((reinterpret_cast<const uint32_t*>(p->pass_count) - p->qkvb) / 2);
    for (int i = blockIdx.x * kThreads + tid(); i < n2; i += p->nwg * kThreads)
      __hip_atomic_store(G(w2 + i), 0x0101010101010101ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  if (blockIdx.x == 0 && tid() == 0) {
    rvqsd_stats* st = fa.out_stats;
    st->target_calls = shs.st_calls;
    st->rounds = shs.st_rounds;
    st->drafted = shs.st_drafted;
    st->accepted = shs.st_accepted;
    st->accept_mask = shs.st_mask;
    const uint64_t sw = __hip_atomic_load(G(p->status), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    int32_t status = ((uint32_t)(sw >> 32) == fa.epoch_base) ? (int32_t)(uint32_t)sw : 0;
    if (!c0_ok) status = poisoned ? RVQSD_EHIP : RVQSD_EINVAL;
    if (status == 0 && !ok) status = RVQSD_ETIMEOUT;
    // the parity state of the exchange buffers is only consistent after a complete frame
    if (!poisoned)
      __hip_atomic_store(G(p->pass_count), (ok && c0_ok) ? c.pass0 + (uint32_t)shs.pass : (c0_ok ? 0xffffffffu : c.pass0),
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    st->status = status;
    st->weight_bytes = shs.st_bytes;
    st->clk_start = t_start;
    st->clk_end = dclock();
    for (int s2 = 1; s2 <= p->n_codes; ++s2) fa.out_codes[s2 - 1] = ok ? shs.codes[s2] : -1;
  }
}

// Between two frames of one launch: every workgroup has ended the earlier frame (its parity
// resets and workgroup 0's statistics and pass count are done) before any starts the next.
// bar counts arrivals from 0 (cleared before the launch); the wait is bounded like every other.
__device__ __forceinline__ void frame_gap_sync(uint32_t* bar, uint32_t target) {
  __syncthreads();
  if (tid() == 0) {
    __hip_atomic_fetch_add(G(bar), 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    const uint64_t t0 = dclock();
    while (__hip_atomic_load(G(bar), __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < target)
      if (dclock() - t0 > kTimeoutTicks) break;  // the next frame then fails on its own waits
  }
  __syncthreads();
}

// MF: projections and LM heads on the matrix cores (bf16 or int8 weights, at most 8 rows), else
// on the VALU GEMV. fa.n_frames frames, frame f's arguments at stride f from fa's and its tags
// from fa.epoch_base + f * fa.epoch_step.
template <typename WT, int MR, bool MF>
__global__ void __launch_bounds__(kThreads, 1) frame_kernel(const KParams* __restrict__ gp, FrameArgs fa) {
  constexpr int RPT = MR <= 8 ? 8 : 4;
  __shared__ Shared shs;
  extern __shared__ __align__(16) float dyn[];
  const KParams* p = gp;
  Ctx c;
  c.p = p;
  c.sh = &shs;
  c.cpw = (p->H + p->nwg - 1) / p->nwg;
  c.dyn = dyn;
  c.xown = dyn;
  c.red = dyn + kMaxRows * c.cpw;
  c.work = c.red + kWaves * (RPT + 1) * MR;
  c.attn_const = c.work + p->work_floats;
  if ((int)blockIdx.x < p->nq) {
    const int d = p->d;
    for (int i = tid(); i < p->L * 2 * d; i += kThreads) {
      const int l = i / (2 * d), j = i % (2 * d);
      c.attn_const[i] = G(fptr(p, layer_off(p, l, j < d ? p->o_qn : p->o_kn)))[j % d];
    }
    for (int i = tid(); i < kMaxPos * d; i += kThreads) c.attn_const[p->L * 2 * d + i] = G(p->rope)[i];
  }
  for (int f = 0; f < fa.n_frames; ++f) {
    if (f > 0) frame_gap_sync(fa.fbar, (uint32_t)f * (uint32_t)p->nwg);
    FrameArgs fr = fa;
    fr.frame_hidden = fa.frame_hidden + (size_t)f * p->H;
    fr.c0 = fa.c0 + f;
    fr.uniforms = fa.uniforms + (size_t)f * 3 * p->n_codes;
    fr.out_codes = fa.out_codes + (size_t)f * p->n_codes;
    fr.out_stats = fa.out_stats + f;
    fr.epoch_base = fa.epoch_base + (uint32_t)f * fa.epoch_step;
    fr.n_frames = 1;
    decode_frame<WT, MR, MF>(c, fr);
  }
}

// ------------------------------------------------------------------- host

int frame_max_rows(int K) {
  const int need = K + 1 < 2 ? 2 : K + 1;
  if (need <= 2) return 2;
  if (need <= 4) return 4;
  if (need <= 5) return 5;
  if (need <= 8) return 8;
  return 16;
}

// floats of the per-workgroup regions in front of the work area
int frame_lds_head_floats(int mr, int cpw) {
  const int rpt = mr <= 8 ? 8 : 4;
  return kMaxRows * cpw + kWaves * (rpt + 1) * mr;
}

template <typename WT, int MR, bool MF>
static int launch_t(const KParams* gp, const FrameArgs& fa, int nwg, void* stream, size_t lds, char* err, size_t errlen) {
  const void* fn = reinterpret_cast<const void*>(&frame_kernel<WT, MR, MF>);
  static size_t attr_bytes = 0;  // per instantiation
  if (lds > attr_bytes) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) {
      snprintf(err, errlen, "hipFuncSetAttribute(%zu bytes LDS): %s", lds, hipGetErrorString(e));
      return RVQSD_EHIP;
    }
    attr_bytes = lds;
  }
  const KParams* gpp = gp;
  FrameArgs fac = fa;
  void* args[] = {&gpp, &fac};
  hipError_t e = hipLaunchCooperativeKernel(fn, dim3(nwg), dim3(kThreads), args, (unsigned)lds,
                                            reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) {
    snprintf(err, errlen, "hipLaunchCooperativeKernel: %s", hipGetErrorString(e));
    return RVQSD_EHIP;
  }
  return RVQSD_OK;
}

int launch_frame(const KParams* gp, const FrameArgs& fa, int nwg, int dtype, int mr, bool mfma, void* stream,
                 size_t lds_bytes, char* err, size_t errlen) {
#define RVQSD_CASE(T, M, F) \
  if (mr == M) return launch_t<T, M, F>(gp, fa, nwg, stream, lds_bytes, err, errlen);
  if (dtype == RVQSD_DTYPE_F32) {
    RVQSD_CASE(float, 2, false) RVQSD_CASE(float, 4, false) RVQSD_CASE(float, 5, false) RVQSD_CASE(float, 8, false)
    RVQSD_CASE(float, 16, false)
  } else if (dtype == RVQSD_DTYPE_I8) {
    if (mfma) { RVQSD_CASE(int8_t, 2, true) RVQSD_CASE(int8_t, 4, true) RVQSD_CASE(int8_t, 5, true) RVQSD_CASE(int8_t, 8, true) }
  } else if (mfma) {
    RVQSD_CASE(bf16_t, 2, true) RVQSD_CASE(bf16_t, 4, true) RVQSD_CASE(bf16_t, 5, true) RVQSD_CASE(bf16_t, 8, true)
  } else {
    RVQSD_CASE(bf16_t, 2, false) RVQSD_CASE(bf16_t, 4, false) RVQSD_CASE(bf16_t, 5, false) RVQSD_CASE(bf16_t, 8, false)
    RVQSD_CASE(bf16_t, 16, false)
  }
#undef RVQSD_CASE
  snprintf(err, errlen, "no kernel for %d rows", mr);
  return RVQSD_EUNSUPPORTED;
}

}  // namespace rvqsd
