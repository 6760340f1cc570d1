// rvqsd_batch.hip -- batched verification kernel (gfx950): several independent
// frame streams ("lanes") decoded together, every pass verifying all their
// rows at once.
//
// The speculative round of each lane is the one of the single-stream kernel
// (paper Sec. 2.2: offset drafts from the anchor's hidden state, one K+1-row
// verification pass with a KV cache, top-k rejection sampling with residual
// resampling). What changes is the shape: lane i owns rows i * rpl .. i * rpl +
// rpl - 1 of a pass, so every projection multiplies M = lanes * rpl <= 80
// activation rows by the weights it streams once, on MFMA tiles (five 16-row
// tiles), and the LM heads group the rows of all lanes that need the same
// per-position head.
//
// One cooperative launch runs every frame of the call. Lane i decodes frames
// i, i + lanes, i + 2 lanes, ...; when its frame completes it writes the codes
// and starts the next one in the same round, so lanes stay busy until their
// frames run out. Each round is a fixed chain of phases separated by a grid
// barrier:
//   commit + row setup (lane workgroups) | per layer: QKV, attention, O,
//   residual + norm, gate/up (SiLU * up fused), down, residual + norm |
//   LM heads | top-k / softmax / draft / accept-or-resample.
// Data crossing workgroups is written with device-coherent (sc1) stores; the
// barrier waits for this workgroup's stores to complete before it arrives,
// and after it one wave per workgroup runs an agent-scope acquire (cache
// invalidate), so the next phase reads with plain, cached loads. Every wait is bounded: a workgroup that times
// out records RVQSD_ETIMEOUT in the status word and every other one leaves at
// its next barrier.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "rvqsd_device.h"
#include "rvqsd_internal.h"

namespace rvqsd {

namespace {

// ------------------------------------------------------------ memory helpers

__device__ __forceinline__ uint32_t cld32(const void* p) {
  return __hip_atomic_load(G(reinterpret_cast<const uint32_t*>(p)), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void cst32(void* p, uint32_t v) {
  __hip_atomic_store(G(reinterpret_cast<uint32_t*>(p)), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void cst64(void* p, uint64_t v) {
  __hip_atomic_store(G(reinterpret_cast<uint64_t*>(p)), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// plain (cached) reads of data published before the last barrier
__device__ __forceinline__ float ldf(const float* p) { return *G(p); }
// Sum of KS <= kMaxSplit partial sums at p, p + stride, ... in split order; the loads are
// issued together (a loop with a run-time bound would wait for each before the next).
constexpr int kMaxSplit = 32;
template <bool COH = false>
__device__ __forceinline__ float sum_parts(const float* p, size_t stride, int KS) {
  float v[kMaxSplit];
#pragma unroll
  for (int k = 0; k < kMaxSplit; ++k)
    v[k] = k < KS ? (COH ? __uint_as_float(cld32(p + k * stride)) : ldf(p + k * stride)) : 0.f;
  float s = v[0];
#pragma unroll
  for (int k = 1; k < kMaxSplit; ++k) s += v[k];
  return s;
}
__device__ __forceinline__ void cstf(float* p, float v) { cst32(p, __float_as_uint(v)); }

// 8 activations -> one split chunk (4 words bf16 hi, 4 words bf16 lo) at dst
__device__ __forceinline__ void store_split(uint32_t* dst, const float (&x)[8]) {
  W16 hi, lo;
  split8(x, hi, lo);
  cst64(dst + 0, (uint64_t)hi[0] | ((uint64_t)hi[1] << 32));
  cst64(dst + 2, (uint64_t)hi[2] | ((uint64_t)hi[3] << 32));
  cst64(dst + 4, (uint64_t)lo[0] | ((uint64_t)lo[1] << 32));
  cst64(dst + 6, (uint64_t)lo[2] | ((uint64_t)lo[3] << 32));
}
__device__ __forceinline__ float cldf(const float* p) { return __uint_as_float(cld32(p)); }
__device__ __forceinline__ uint64_t cld64(const void* p) {
  return __hip_atomic_load(G(reinterpret_cast<const uint64_t*>(p)), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// dst[e] = src(e) for e < n, e = row * ncols + col -> src + row * row_stride + col; each thread
// issues 8 loads before it stores (a plain copy loop would wait for every load in turn)
template <bool COH>
__device__ __forceinline__ void lds_fill(float* dst, const float* src, int n, int ncols, size_t row_stride) {
  for (int base = 0; base < n; base += 8 * kThreads) {
    float v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int e = base + k * kThreads + tid();
      const float* a = src + (size_t)(e / ncols) * row_stride + (e % ncols);
      v[k] = e < n ? (COH ? cldf(a) : ldf(a)) : 0.f;
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int e = base + k * kThreads + tid();
      if (e < n) dst[e] = v[k];
    }
  }
}

__device__ __forceinline__ const bf16_t* bw(const KParams* p, uint64_t off) {
  return reinterpret_cast<const bf16_t*>(p->wbase + off);
}
__device__ __forceinline__ const float* bfw(const KParams* p, uint64_t off) {
  return reinterpret_cast<const float*>(p->wbase + off);
}
__device__ __forceinline__ uint64_t boff(const KParams* p, int l, uint64_t o) { return (uint64_t)l * p->layer_stride + o; }

template <typename BP>
__device__ __forceinline__ void raise_status(const BP* bp, int code) {
  int expected = 0;
  __hip_atomic_compare_exchange_strong(G(bp->status), &expected, code, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------------------------ shared state

struct BShared {
  TopkShared tk;
  int ln[kMaxLanes][kLaneInts];  // every lane's state, read at the start of the round
  int abort;
  int hl_n, hl_t;                // LM-head row list of the current unit
  int hl_row[kBatchMaxRows];
  float red[kWaves];
  int vr[kBatchMaxRows];         // commit: verdicts of the lane's rows
  int dt[kMaxRows][kMaxCodes];   // commit: draft tokens of every row of the lane (chain lanes)
  int tok;
  // tree lanes
  int kid[kMaxTreeRows];         // sampling: children of the row, in increasing rank
  int nkid;
  int c_mnew, c_arow, c_acc, c_m;  // commit: new anchor position and row, accepted nodes, old anchor
  int c_path[kMaxCodes + 1];     // commit: accepted rows, depth 1 .. c_acc
};

// ------------------------------------------------------------ grid barrier
// Arrival counts per XCD group (workgroup w is counted in group w % 8), the
// last arrival of a group bumps the top counter, the last group publishes the
// generation. Before arriving, every wave waits for its own stores.
template <typename BP, bool ACQ = true>
__device__ bool grid_sync(const BP* bp, uint32_t& gen, BShared* sh) {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  ++gen;
  if (tid() == 0) {
    const int nwg = bp->nwg, x = (int)blockIdx.x & 7;
    const uint32_t nx = (uint32_t)((nwg - x + 7) / 8);
    uint32_t* bar = bp->bar;
    const uint32_t prev = __hip_atomic_fetch_add(G(bar + 64 * (1 + x)), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (prev + 1 == gen * nx) {
      const uint32_t p2 = __hip_atomic_fetch_add(G(bar), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (p2 + 1 == gen * 8u) cst32(bar + 64 * 9, gen);
    }
    int ab = 0, spins = 0;
    uint64_t t0 = 0;
    while (cld32(bar + 64 * 9) < gen) {
      __builtin_amdgcn_s_sleep(1);
      if ((++spins & 31) == 0) {
        if (cld32(bp->status) != 0) {
          ab = 1;
          break;
        }
        const uint64_t now = dclock();
        if (t0 == 0) {
          t0 = now;
        } else if (now - t0 > kTimeoutTicks) {
          raise_status(bp, RVQSD_ETIMEOUT);
          ab = 1;
          break;
        }
      }
    }
    if (!ab && cld32(bp->status) != 0) ab = 1;
    sh->abort = ab;
  }
  // drop this CU's and this XCD's cached copies of lines written by others (not needed by
  // a kernel that reads every cross-workgroup value with device-coherent loads)
  if (ACQ && tid() < 64) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  __syncthreads();
  return sh->abort == 0;
}

// ------------------------------------------------------------ block helpers

__device__ __forceinline__ float block_sum(BShared* sh, float v) {
  v = wave_sum(v);
  const int lane = tid() & 63, wave = tid() >> 6;
  if (lane == 0) sh->red[wave] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) t += sh->red[w];
  __syncthreads();
  return t;
}

constexpr int kRowChunks = 4;  // 8-element chunks per lane of a row held in registers (hidden <= 2048)

// ------------------------------------------------------------ pass geometry

// A lane's pass has tree rows when the stream verifies trees and the prefix pass is done;
// the prefix pass (rows at positions 0 and 1) and chain lanes put row r at position first + r.
template <bool TR>
__device__ __forceinline__ bool tree_rows(const BParams* bp, const int* st) { return TR && st[kLnPass] > 0; }
template <bool TR>
__device__ __forceinline__ int row_pos(const BParams* bp, const int* st, int r) {
  return st[kLnFirst] + (tree_rows<TR>(bp, st) ? bp->t_depth[r] : r);
}
// whether row a is row r or one of its ancestors (the rows row r attends to)
template <bool TR>
__device__ __forceinline__ bool row_sees(const BParams* bp, const int* st, int r, int a) {
  if (!tree_rows<TR>(bp, st)) return a <= r;
  return (bp->t_anc[r][a >> 6] >> (a & 63)) & 1ull;
}
template <bool TR>
__device__ __forceinline__ bool row_is_verify(const BParams* bp, const int* st, int r) {
  return r < st[kLnRows] && row_pos<TR>(bp, st, r) >= 1 && (st[kLnPass] == 0 ? r == 1 : true);
}
template <bool TR>
__device__ __forceinline__ int row_drafts(const BParams* bp, const KParams* p, const int* st, int r) {
  const int s = row_pos<TR>(bp, st, r);
  if (r >= st[kLnRows] || s < 1 || s > p->n_codes - 1) return 0;
  if (st[kLnPass] == 0 && r != 1) return 0;
  return min(p->K, p->n_codes - s);
}
// LM-head input row of (lane row i, offset j) and whether it is used this pass
template <bool TR>
__device__ __forceinline__ bool head_slot_used(const BParams* bp, const KParams* p, const int* st, int r, int j) {
  if (!st[kLnActive]) return false;
  return j == 0 ? row_is_verify<TR>(bp, st, r) : j <= row_drafts<TR>(bp, p, st, r);
}

// ------------------------------------------------------------ MFMA tile unit
// Output features n0 .. n0 + 16 NTU - 1 (weight rows wrow(nt, m) of n-tile nt,
// nullptr when outside the matrix) over k in [k0, k0 + klen), for the
// activation rows rowof(i), i < 16 * mtiles (-1: padding). Wave w takes n-tile
// w % NTU and the k part w / NTU; the KW = 8 / NTU parts are added in LDS in a
// fixed order. On return red[(nt * kBatchMTiles + mt) * 256 + 4 * lane + v]
// holds D[feature 16 nt + 4 (lane / 16) + v][row 16 mt + lane % 16].
// MFMA roles as in the frame kernel: A = 16 weight rows, B = 16 activation
// rows; lane group q = lane / 16 covers the 16 consecutive k of a 64-wide step
// in two instructions, and the activation chunk of 8 enters as bf16 hi + lo.
// With STG (device-coherent operands, several n-tile groups) the activation
// words of each step are copied once per workgroup into LDS (at red, before
// the partial tiles are written there) and every wave reads its fragments from
// LDS: the waves of different n-tile groups share one copy instead of each
// reading it from the memory side. The k ranges of the waves, and so the
// summation order, are the same with and without STG.
// With ALDS, A is a split row block in LDS that the caller filled.
template <int NTU, int NTW, bool COH = false, bool STG = false, bool ALDS = false, typename WRow, typename RowOf>
__device__ __forceinline__ void gemm_unit(WRow wrow, int k0, int klen, const uint32_t* A, int lda, int mtiles,
                                          RowOf rowof, float* red) {
  constexpr int NG = NTU / NTW, KW = kWaves / NG;
  const int wave = __builtin_amdgcn_readfirstlane(tid() >> 6), lane = tid() & 63;
  const int ng = wave % NG, kw = wave / NG;
  const int kper = klen / KW;
  const int kb = k0 + kw * kper;
  const int q = lane >> 4, ml = lane & 15;
  const bf16_t* wp[NTW];
#pragma unroll
  for (int t = 0; t < NTW; ++t) {
    const bf16_t* wr = wrow(ng * NTW + t, ml);
    wp[t] = wr ? wr + kb + 16 * q : nullptr;
  }
  int arow[kBatchMTiles];
#pragma unroll
  for (int mt = 0; mt < kBatchMTiles; ++mt) arow[mt] = mt < mtiles ? rowof(16 * mt + ml) : -1;
  f32x4 acc[NTW][kBatchMTiles];
#pragma unroll
  for (int t = 0; t < NTW; ++t)
#pragma unroll
    for (int mt = 0; mt < kBatchMTiles; ++mt) acc[t][mt] = (f32x4){0.f, 0.f, 0.f, 0.f};
  const int nsteps = kper >> 6;
  if constexpr (STG) {
    static_assert(COH && NG > 1, "staging serves coherent operands shared by n-tile groups");
    // step u stages, for every k part kw, words kb(kw) + 64 u .. + 63 of each of the
    // 16 mtiles rows: stg[row][kw * 64 + j], row stride KW * 64 + 4 words
    constexpr int SW = KW * 64 + 4, NV = 16 * KW;  // row stride; 16-byte vectors per row
    constexpr int SPT = (kBatchMTiles * 16 * NV + kThreads - 1) / kThreads;
    static_assert(kBatchMTiles * 16 * SW <= kBatchRedFloats + kBatchMaxRows * 16, "staged rows fit the unit's LDS area");
    uint32_t* stg = reinterpret_cast<uint32_t*>(red);
    const int nvec = 16 * mtiles * NV;
    const __amdgpu_buffer_rsrc_t ars = coh_rsrc(A);
    for (int u = 0; u < nsteps; ++u) {
      W16 a0[NTW], a1[NTW];
#pragma unroll
      for (int t = 0; t < NTW; ++t) {
        a0[t] = a1[t] = (W16)(0u);
        if (wp[t]) {
          a0[t] = *G(reinterpret_cast<const W16*>(wp[t] + 64 * u));
          a1[t] = *G(reinterpret_cast<const W16*>(wp[t] + 64 * u + 8));
        }
      }
      W16 sv[SPT];
#pragma unroll
      for (int i = 0; i < SPT; ++i) {
        const int e = tid() + i * kThreads;
        sv[i] = (W16)(0u);
        if (e < nvec) {
          const int row = e / NV, rem = e - row * NV, pk = rem >> 4, j4 = rem & 15;
          const int ar = rowof(row);
          if (ar >= 0) sv[i] = bload4(ars, (uint32_t)((size_t)ar * lda + (k0 + pk * kper + 64 * u + 4 * j4)) * 4u);
        }
      }
      if (u > 0) __syncthreads();  // every wave is done with the previous step's copy
#pragma unroll
      for (int i = 0; i < SPT; ++i) {
        const int e = tid() + i * kThreads;
        if (e < nvec) {
          const int row = e / NV, rem = e - row * NV;
          *reinterpret_cast<W16*>(stg + row * SW + 4 * rem) = sv[i];
        }
      }
      __syncthreads();
#pragma unroll
      for (int t = 0; t < NTW; ++t) {
        const bf16x8 x0 = __builtin_bit_cast(bf16x8, a0[t]), x1 = __builtin_bit_cast(bf16x8, a1[t]);
#pragma unroll
        for (int mt = 0; mt < kBatchMTiles; ++mt) {
          if (mt < mtiles) {
            const uint32_t* sp = stg + (16 * mt + ml) * SW + kw * 64 + 16 * q;
            const W16 bh0 = *reinterpret_cast<const W16*>(sp), bl0 = *reinterpret_cast<const W16*>(sp + 4);
            const W16 bh1 = *reinterpret_cast<const W16*>(sp + 8), bl1 = *reinterpret_cast<const W16*>(sp + 12);
            acc[t][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x0, __builtin_bit_cast(bf16x8, bh0), acc[t][mt], 0, 0, 0);
            acc[t][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x0, __builtin_bit_cast(bf16x8, bl0), acc[t][mt], 0, 0, 0);
            acc[t][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x1, __builtin_bit_cast(bf16x8, bh1), acc[t][mt], 0, 0, 0);
            acc[t][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x1, __builtin_bit_cast(bf16x8, bl1), acc[t][mt], 0, 0, 0);
          }
        }
      }
    }
    __syncthreads();  // the staged copy is read before red receives the partial tiles
  } else
  for (int u = 0; u < nsteps; ++u) {
    W16 a0[NTW], a1[NTW];
#pragma unroll
    for (int t = 0; t < NTW; ++t) {
      a0[t] = a1[t] = (W16)(0u);
      if (wp[t]) {
        a0[t] = *G(reinterpret_cast<const W16*>(wp[t] + 64 * u));
        a1[t] = *G(reinterpret_cast<const W16*>(wp[t] + 64 * u + 8));
      }
    }
    const int chunk = (kb + 64 * u + 16 * q) >> 3;
    W16 bh0[kBatchMTiles], bl0[kBatchMTiles], bh1[kBatchMTiles], bl1[kBatchMTiles];
#pragma unroll
    for (int mt = 0; mt < kBatchMTiles; ++mt) {
      bh0[mt] = bl0[mt] = bh1[mt] = bl1[mt] = (W16)(0u);
      if (mt < mtiles && arow[mt] >= 0) {
        const uint32_t* ap = A + (size_t)arow[mt] * lda + (size_t)chunk * 8;
        if constexpr (ALDS) {
          bh0[mt] = *reinterpret_cast<const W16*>(ap);
          bl0[mt] = *reinterpret_cast<const W16*>(ap + 4);
          bh1[mt] = *reinterpret_cast<const W16*>(ap + 8);
          bl1[mt] = *reinterpret_cast<const W16*>(ap + 12);
        } else if constexpr (COH) {
          bh0[mt] = pload4(ap);
          bl0[mt] = pload4(ap + 4);
          bh1[mt] = pload4(ap + 8);
          bl1[mt] = pload4(ap + 12);
        } else {
          bh0[mt] = *G(reinterpret_cast<const W16*>(ap));
          bl0[mt] = *G(reinterpret_cast<const W16*>(ap + 4));
          bh1[mt] = *G(reinterpret_cast<const W16*>(ap + 8));
          bl1[mt] = *G(reinterpret_cast<const W16*>(ap + 12));
        }
      }
    }
    if constexpr (COH && !ALDS) {
      // the device-coherent loads are issued from inline assembly: wait for them explicitly
#pragma unroll
      for (int mt = 0; mt < kBatchMTiles; ++mt) {
        vm_wait(bh0[mt]);
        vm_wait(bl0[mt]);
        vm_wait(bh1[mt]);
        vm_wait(bl1[mt]);
      }
    }
#pragma unroll
    for (int t = 0; t < NTW; ++t) {
      const bf16x8 x0 = __builtin_bit_cast(bf16x8, a0[t]), x1 = __builtin_bit_cast(bf16x8, a1[t]);
#pragma unroll
      for (int mt = 0; mt < kBatchMTiles; ++mt) {
        if (mt < mtiles) {
          acc[t][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x0, __builtin_bit_cast(bf16x8, bh0[mt]), acc[t][mt], 0, 0, 0);
          acc[t][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x0, __builtin_bit_cast(bf16x8, bl0[mt]), acc[t][mt], 0, 0, 0);
          acc[t][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x1, __builtin_bit_cast(bf16x8, bh1[mt]), acc[t][mt], 0, 0, 0);
          acc[t][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x1, __builtin_bit_cast(bf16x8, bl1[mt]), acc[t][mt], 0, 0, 0);
        }
      }
    }
  }
#pragma unroll
  for (int t = 0; t < NTW; ++t)
#pragma unroll
    for (int mt = 0; mt < kBatchMTiles; ++mt)
      if (mt < mtiles)
        *reinterpret_cast<f32x4*>(red + ((size_t)((kw * NTU + ng * NTW + t) * kBatchMTiles + mt) << 8) + 4 * lane) =
            acc[t][mt];
  __syncthreads();
  if (KW > 1) {
    for (int e = tid(); e < NTU * mtiles * 256; e += kThreads) {
      const int t = e / (mtiles * 256), rem = e - t * (mtiles * 256), mt = rem >> 8, x = rem & 255;
      float sum = red[((size_t)(t * kBatchMTiles + mt) << 8) + x];
#pragma unroll
      for (int k = 1; k < KW; ++k) sum += red[((size_t)((k * NTU + t) * kBatchMTiles + mt) << 8) + x];
      red[((size_t)(t * kBatchMTiles + mt) << 8) + x] = sum;
    }
    __syncthreads();
  }
}
// LDS floats of one unit's k-part tiles
template <int NTU, int NTW>
constexpr int gemm_red_floats() {
  return kWaves / (NTU / NTW) * NTU * kBatchMTiles * 256;
}
constexpr int kProjNTW = 2, kGuNTW = 2;  // n-tiles per wave (activation fragments reused NTW times)
// LM-head units: 16 kHeadNTU columns, so that the 15 heads of the 1024-wide model take one unit per workgroup
constexpr int kHeadNTU = 8;
static_assert(gemm_red_floats<4, kProjNTW>() <= kBatchRedFloats && gemm_red_floats<2, kGuNTW>() <= kBatchRedFloats &&
                  gemm_red_floats<kHeadNTU, kProjNTW>() <= kBatchRedFloats,
              "LDS reduction area");

// ------------------------------------------------------------ projections

// Y partial sums: part[ks][i][n] = sum over k in split ks of A[i][k] W[n][k], for every row i < M.
// Inlined into the kernels: as out-of-line calls these two spill to scratch (the call ABI) and
// their phases run 4-6 us slower.
template <int NTU, typename BP, bool COH = false, bool STG = false>
__device__ __forceinline__ void proj_partial(const BP* bp, const bf16_t* W, int N, int K, int KS, const uint32_t* A, float* red) {
  const int M = bp->M, mtiles = (M + 15) >> 4;
  const int cg = (N + 16 * NTU - 1) / (16 * NTU), units = cg * KS, klen = K / KS;
  float* part = bp->part;
  for (int u = blockIdx.x; u < units; u += bp->nwg) {
    const int g = u % cg, ks = u / cg, n0 = g * 16 * NTU;
    auto wrow = [&](int nt, int m) -> const bf16_t* {
      const int f = n0 + 16 * nt + m;
      return f < N ? W + (size_t)f * K : nullptr;
    };
    auto rowof = [&](int i) { return i < M ? i : -1; };
    // staging pays from two row tiles on; with one the waves read their fragments directly
    if (STG && mtiles >= 2) gemm_unit<NTU, kProjNTW, COH, STG>(wrow, ks * klen, klen, A, K, mtiles, rowof, red);
    else gemm_unit<NTU, kProjNTW, COH, false>(wrow, ks * klen, klen, A, K, mtiles, rowof, red);
    for (int e = tid(); e < NTU * mtiles * 64; e += kThreads) {
      const int nt = e / (mtiles * 64), rem = e - nt * (mtiles * 64), mt = rem >> 6, ln = rem & 63;
      const int row = 16 * mt + (ln & 15), f = n0 + 16 * nt + 4 * (ln >> 4);
      if (row < M && f < N) {
        const float* s = red + ((size_t)(nt * kBatchMTiles + mt) << 8) + 4 * ln;
        float* dst = part + ((size_t)ks * M + row) * N + f;
        cst64(dst, (uint64_t)__float_as_uint(s[0]) | ((uint64_t)__float_as_uint(s[1]) << 32));
        cst64(dst + 2, (uint64_t)__float_as_uint(s[2]) | ((uint64_t)__float_as_uint(s[3]) << 32));
      }
    }
    __syncthreads();
  }
}

// gate/up: n-tile 0 = gate rows f0 .. f0 + 15, n-tile 1 = the same up rows, full k;
// act = SiLU(gate) * up goes straight to the split input of the down projection.
template <typename BP, bool COH = false>
__device__ __forceinline__ void phase_gu(const BP* bp, int l, const uint32_t* A, uint32_t* Aout, float* red) {
  const KParams* p = bp->k;
  const int M = bp->M, mtiles = (M + 15) >> 4, H = p->H, F = p->F;
  const bf16_t* wg = bw(p, boff(p, l, p->o_wg));
  const bf16_t* wu = bw(p, boff(p, l, p->o_wu));
  float* act = red + gemm_red_floats<2, kGuNTW>();  // [80][16]
  for (int u = blockIdx.x; u < F / 16; u += bp->nwg) {
    const int f0 = u * 16;
    gemm_unit<2, kGuNTW, COH>([&](int nt, int m) -> const bf16_t* { return (nt ? wu : wg) + (size_t)(f0 + m) * H; }, 0, H, A, H,
                 mtiles, [&](int i) { return i < M ? i : -1; }, red);
    for (int e = tid(); e < mtiles * 256; e += kThreads) {
      const int mt = e >> 8, x = e & 255, ln = x >> 2, v = x & 3;
      const float gt = red[((size_t)(0 * kBatchMTiles + mt) << 8) + x];
      const float up = red[((size_t)(1 * kBatchMTiles + mt) << 8) + x];
      act[(16 * mt + (ln & 15)) * 16 + 4 * (ln >> 4) + v] = gt / (1.f + expf(-gt)) * up;
    }
    __syncthreads();
    for (int c = tid(); c < 2 * M; c += kThreads) {
      const int row = c >> 1, h8 = c & 1;
      float x8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x8[e] = act[row * 16 + 8 * h8 + e];
      store_split(Aout + (size_t)row * F + f0 + 8 * h8, x8);
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------ attention
// Unit (lane, q head h): q, k, v of the lane's rows from the QKV partial sums,
// per-head RMSNorm and rotate-half RoPE, KV append (first q head of each kv
// group), causal softmax attention over positions 0 .. s, output split into the
// O projection's input.
// Attention of lanes whose rows form a draft tree (Sec. 2.2, Fig. 2): row r sits at
// position first + depth(r), its K/V at slot first + r, and it attends to the committed
// positions 0 .. first - 1 and to the slots of its ancestors and itself (the prefix
// pass: rows at positions 0 and 1, causal). One workgroup per (lane, query head); one
// wave per row for scores, softmax and output, the scores staged in LDS.
__device__ void phase_attn_tree(const BParams* bp, BShared* sh, int l, uint32_t* Aout, float* lds) {
  const KParams* p = bp->k;
  const int d = p->d, nq = p->nq, grp = nq / p->nkv, N = p->nqkv, KS = bp->ks_qkv, M = bp->M, half = d / 2;
  const int qdim = p->qdim, kvdim = p->kvdim, lane = tid() & 63, wave = tid() >> 6, slots = bp->kv_slots;
  const float scale = 1.f / sqrtf((float)d);
  float* qs = lds;                          // [rpl][d]: q rows, then each row's output
  float* kvs = qs + (size_t)bp->rpl * d;    // [slots][2][d]
  float* wsc = kvs + (size_t)slots * 2 * d; // [kWaves][slots] scores, then softmax weights
  const float* qn = bfw(p, boff(p, l, p->o_qn));
  const float* kn = bfw(p, boff(p, l, p->o_kn));
  for (int u = blockIdx.x; u < bp->lanes * nq; u += bp->nwg) {
    const int ln = u / nq, h = u - ln * nq, g = h / grp;
    const int* st = sh->ln[ln];
    if (!st[kLnActive]) continue;
    const int fp = st[kLnFirst], R = st[kLnRows], row0 = ln * bp->rpl;
    float* kvc = bp->kv + (((size_t)ln * p->L + l) * p->nkv + g) * slots * 2 * d;
    const int tot = R * 3 * d;
    for (int base = 0; base < tot; base += 4 * kThreads) {
      const float* src[4];
      float acc[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int e = base + k * kThreads + tid();
        const int r = e / (3 * d), w = e - r * 3 * d, part = w / d, i = w - part * d;
        const int col = part == 0 ? h * d + i : qdim + (part - 1) * kvdim + g * d + i;
        src[k] = e < tot ? bp->part + (size_t)(row0 + r) * N + col : nullptr;
        acc[k] = 0.f;
      }
      for (int ks0 = 0; ks0 < KS; ks0 += 4) {
        float t[4][4];
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            t[k][j] = (src[k] && ks0 + j < KS) ? cldf(src[k] + (size_t)(ks0 + j) * M * N) : 0.f;
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (ks0 + j < KS) acc[k] += t[k][j];
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int e = base + k * kThreads + tid();
        if (e < tot) {
          const int r = e / (3 * d), w = e - r * 3 * d, part = w / d, i = w - part * d;
          if (part == 0) qs[r * d + i] = acc[k];
          else kvs[(size_t)(fp + r) * 2 * d + (part - 1) * d + i] = acc[k];
        }
      }
    }
    lds_fill<true>(kvs, kvc, fp * 2 * d, 2 * d, (size_t)2 * d);
    __syncthreads();
    // q rows (v < R) and k rows (v >= R): norm + RoPE at the row's position, one wave per vector
    for (int v = wave; v < 2 * R; v += kWaves) {
      const bool isq = v < R;
      const int r = isq ? v : v - R, pos = row_pos<true>(bp, st, r);
      float* x = isq ? qs + r * d : kvs + (size_t)(fp + r) * 2 * d;
      const float* gn = isq ? qn : kn;
      float ss = 0.f;
      for (int i = lane; i < d; i += 64) ss = fmaf(x[i], x[i], ss);
      ss = wave_sum(ss);
      const float rs = p->qk_norm ? 1.f / sqrtf(ss / (float)d + p->rms_eps) : 1.f;
      for (int i = lane; i < half; i += 64) {
        float a = x[i], b = x[i + half];
        if (p->qk_norm) {
          a = a * rs * G(gn)[i];
          b = b * rs * G(gn)[i + half];
        }
        const float cs = G(p->rope)[(pos * half + i) * 2], sn = G(p->rope)[(pos * half + i) * 2 + 1];
        x[i] = a * cs - b * sn;
        x[i + half] = b * cs + a * sn;
      }
    }
    __syncthreads();
    if (h % grp == 0)
      for (int e = tid(); e < R * 2 * d; e += kThreads) cstf(kvc + (size_t)fp * 2 * d + e, kvs[(size_t)fp * 2 * d + e]);
    float* w = wsc + (size_t)wave * slots;
    for (int r = wave; r < R; r += kWaves) {
      const int nkeys = fp + R;
      float mx = -INFINITY;
      for (int t = 0; t < nkeys; ++t) {
        float sc = -INFINITY;
        if (t < fp || row_sees<true>(bp, st, r, t - fp)) {  // wave-uniform
          float a = 0.f;
          for (int i = lane; i < d; i += 64) a = fmaf(qs[r * d + i], kvs[(size_t)t * 2 * d + i], a);
          sc = wave_sum(a) * scale;
        }
        if (lane == 0) w[t] = sc;
        mx = fmaxf(mx, sc);
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      float z = 0.f;
      for (int t = lane; t < nkeys; t += 64) {
        const float e = expf(w[t] - mx);
        w[t] = e;
        z += e;
      }
      z = wave_sum(z);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      const float iz = 1.f / z;
      for (int i = lane; i < d; i += 64) {
        float o = 0.f;
        for (int t = 0; t < nkeys; ++t) o = fmaf(w[t], kvs[(size_t)t * 2 * d + d + i], o);
        qs[r * d + i] = o * iz;
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    for (int c = tid(); c < R * (d / 8); c += kThreads) {
      const int r = c / (d / 8), q8 = c - r * (d / 8);
      float x8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x8[e] = qs[r * d + 8 * q8 + e];
      store_split(Aout + (size_t)(row0 + r) * qdim + h * d + 8 * q8, x8);
    }
    __syncthreads();
  }
}

// phase_attn for a head dimension D known at compile time: K/V rows padded to 2D + 4 floats in
// LDS (no bank conflicts between positions), norm + RoPE one half-wave per vector with DPP
// sums, scores one wave per row with the 16 positions spread over the lanes (4 lanes each),
// softmax with DPP, and the weighted value sum over position groups of 16-byte reads added in a
// fixed order across the wave.
template <int D>
__device__ __forceinline__ void phase_attn_d(const BParams* bp, BShared* sh, int l, uint32_t* Aout, float* lds) {
  const KParams* p = bp->k;
  const int nq = p->nq, grp = nq / p->nkv, N = p->nqkv, KS = bp->ks_qkv, M = bp->M;
  constexpr int half = D / 2, PS = 2 * D + 4;
  const int qdim = p->qdim, kvdim = p->kvdim, lane = tid() & 63, wave = tid() >> 6;
  const float scale = 1.f / sqrtf((float)D);
  float* qs = lds;                          // [kMaxRows][D]
  float* kvs = qs + kMaxRows * D;           // [kMaxPos][PS]: k, then v
  float* os = kvs + kMaxPos * PS;           // [kMaxRows][D]
  float* pwl = os + kMaxRows * D;           // [kMaxRows][kMaxPos] softmax weights
  const float* qn = bfw(p, boff(p, l, p->o_qn));
  const float* kn = bfw(p, boff(p, l, p->o_kn));
  for (int u = blockIdx.x; u < bp->lanes * nq; u += bp->nwg) {
    const int ln = u / nq, h = u - ln * nq, g = h / grp;
    const int* st = sh->ln[ln];
    if (!st[kLnActive]) continue;
    const int fp = st[kLnFirst], R = st[kLnRows], row0 = ln * bp->rpl;
    float* kvc = bp->kv + (((size_t)ln * p->L + l) * p->nkv + g) * bp->kv_slots * 2 * D;
    // q, k, v of the lane's rows: the partial sums of 4 elements x 4 splits are in flight at once
    const int tot = R * 3 * D;
    for (int base = 0; base < tot; base += 4 * kThreads) {
      const float* src[4];
      float acc[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int e = base + k * kThreads + tid();
        const int r = e / (3 * D), w = e - r * 3 * D, part = w / D, i = w - part * D;
        const int col = part == 0 ? h * D + i : qdim + (part - 1) * kvdim + g * D + i;
        src[k] = e < tot ? bp->part + (size_t)(row0 + r) * N + col : nullptr;
        acc[k] = 0.f;
      }
      for (int ks0 = 0; ks0 < KS; ks0 += 4) {
        float t[4][4];
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            t[k][j] = (src[k] && ks0 + j < KS) ? cldf(src[k] + (size_t)(ks0 + j) * M * N) : 0.f;
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (ks0 + j < KS) acc[k] += t[k][j];
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int e = base + k * kThreads + tid();
        if (e < tot) {
          const int r = e / (3 * D), w = e - r * 3 * D, part = w / D, i = w - part * D;
          if (part == 0) qs[r * D + i] = acc[k];
          else kvs[(size_t)(fp + r) * PS + (part - 1) * D + i] = acc[k];
        }
      }
    }
    // committed positions 0 .. fp-1 from the lane's cache, eight loads in flight per thread
    for (int b0 = 0; b0 < fp * 2 * D; b0 += 8 * kThreads) {
      float v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int e = b0 + k * kThreads + tid();
        v[k] = e < fp * 2 * D ? cldf(kvc + e) : 0.f;
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int e = b0 + k * kThreads + tid();
        if (e < fp * 2 * D) kvs[(size_t)(e / (2 * D)) * PS + e % (2 * D)] = v[k];
      }
    }
    __syncthreads();
    // per-head RMSNorm + RoPE of q (vectors 0..R-1) and k (R..2R-1), one half-wave per vector;
    // lane i of the half holds dimensions i + 32 j (j < D / 64) and their partners i + 32 j + D/2
    constexpr int J = D / 64;
    const int hl = lane & 31;
    for (int v = 2 * wave + (lane >> 5); v < 2 * R; v += 2 * kWaves) {
      const bool isq = v < R;
      const int r = isq ? v : v - R, pos = fp + r;
      float* x = isq ? qs + r * D : kvs + (size_t)pos * PS;
      const float* gn = isq ? qn : kn;
      float a[J], b[J], ga[J], gb[J], cs[J], sn[J];
      float s2 = 0.f;
#pragma unroll
      for (int j = 0; j < J; ++j) {
        const int i = hl + 32 * j;
        a[j] = x[i];
        b[j] = x[i + half];
        ga[j] = G(gn)[i];
        gb[j] = G(gn)[i + half];
        cs[j] = G(p->rope)[(pos * half + i) * 2];
        sn[j] = G(p->rope)[(pos * half + i) * 2 + 1];
        s2 = fmaf(a[j], a[j], fmaf(b[j], b[j], s2));
      }
      const float rs = p->qk_norm ? __builtin_amdgcn_rsqf(half_sum(s2) * (1.f / (float)D) + (float)p->rms_eps) : 1.f;
#pragma unroll
      for (int j = 0; j < J; ++j) {
        const int i = hl + 32 * j;
        float ua = a[j], ub = b[j];
        if (p->qk_norm) {
          ua = ua * rs * ga[j];
          ub = ub * rs * gb[j];
        }
        x[i] = ua * cs[j] - ub * sn[j];
        x[i + half] = ub * cs[j] + ua * sn[j];
      }
    }
    __syncthreads();
    if (h % grp == 0)
      for (int e = tid(); e < R * 2 * D; e += kThreads)
        cstf(kvc + (size_t)fp * 2 * D + e, kvs[(size_t)(fp + e / (2 * D)) * PS + e % (2 * D)]);
    // one wave per row. Scores: lane = (position t = lane / 4, quarter qj of the dimensions);
    // values: lane = (position group gi, dimensions 4 li .. 4 li + 3)
    const int npos = fp + R;
    constexpr int DQ = D / 4, LPD = D / 4;
    constexpr int NG = LPD >= 64 ? 1 : 64 / LPD;
    constexpr int PPG = kMaxPos / NG;
    const int t = lane >> 2, qj = lane & 3;
    const int gi = lane / LPD, li = lane - gi * LPD;
    for (int r = wave; r < R; r += kWaves) {
      const int last = fp + r;  // causal: positions 0 .. last
      float part = 0.f;
      if (t <= last) {
        const f32x4* qv = reinterpret_cast<const f32x4*>(qs + r * D + qj * DQ);
        const f32x4* kk = reinterpret_cast<const f32x4*>(kvs + (size_t)t * PS + qj * DQ);
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
      part += dpp<0xB1>(part);  // quad sums: xor 1, xor 2
      part += dpp<0x4E>(part);
      const float sc = t <= last ? part * scale : -INFINITY;
      const float rm = row16_max(sc);
      const float mx = fmaxf(fmaxf(lane_val(rm, 15), lane_val(rm, 31)), fmaxf(lane_val(rm, 47), lane_val(rm, 63)));
      const float ex = t <= last ? expf(sc - mx) : 0.f;
      const float rsum = row16_sum(qj == 0 ? ex : 0.f);
      const float z = (lane_val(rsum, 15) + lane_val(rsum, 31)) + (lane_val(rsum, 47) + lane_val(rsum, 63));
      const float pr = ex / z;
      // the row's weights go through LDS (written and read back by this wave only, in order);
      // positions at or past npos read the finite row npos - 1 (weight 0) instead of unset rows
      float* pwr = pwl + r * kMaxPos;
      if (qj == 0) pwr[t] = pr;
      f32x4 o = {0.f, 0.f, 0.f, 0.f};
      if (gi < NG) {
        f32x4 wq[PPG / 4];
#pragma unroll
        for (int q4 = 0; q4 < PPG / 4; ++q4) wq[q4] = reinterpret_cast<const f32x4*>(pwr + gi * PPG)[q4];
        f32x4 vv[PPG];
#pragma unroll
        for (int k = 0; k < PPG; ++k)
          vv[k] = *reinterpret_cast<const f32x4*>(kvs + (size_t)min(gi * PPG + k, npos - 1) * PS + D + 4 * li);
#pragma unroll
        for (int k = 0; k < PPG; ++k) {
          const float w = wq[k >> 2][k & 3];
          o.x = fmaf(w, vv[k].x, o.x);
          o.y = fmaf(w, vv[k].y, o.y);
          o.z = fmaf(w, vv[k].z, o.z);
          o.w = fmaf(w, vv[k].w, o.w);
        }
      }
      // groups added in a fixed order: (g0 + g1) + (g2 + g3)
#pragma unroll
      for (int xo = LPD; xo < 64 && NG > 1; xo <<= 1) {
        o.x += __shfl_xor(o.x, xo, 64);
        o.y += __shfl_xor(o.y, xo, 64);
        o.z += __shfl_xor(o.z, xo, 64);
        o.w += __shfl_xor(o.w, xo, 64);
      }
      if (gi == 0) *reinterpret_cast<f32x4*>(os + r * D + 4 * li) = o;
    }
    __syncthreads();
    for (int c = tid(); c < R * (D / 8); c += kThreads) {
      const int r = c / (D / 8), q8 = c - r * (D / 8);
      float x8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x8[e] = os[r * D + 8 * q8 + e];
      store_split(Aout + (size_t)(row0 + r) * qdim + h * D + 8 * q8, x8);
    }
    __syncthreads();
  }
}

__device__ __forceinline__ void phase_attn(const BParams* bp, BShared* sh, int l, uint32_t* Aout, float* lds) {
  if (bp->k->d == 128) return phase_attn_d<128>(bp, sh, l, Aout, lds);
  if (bp->k->d == 64) return phase_attn_d<64>(bp, sh, l, Aout, lds);
  const KParams* p = bp->k;
  const int d = p->d, nq = p->nq, grp = nq / p->nkv, N = p->nqkv, KS = bp->ks_qkv, M = bp->M, half = d / 2;
  const int qdim = p->qdim, kvdim = p->kvdim, lane = tid() & 63, wave = tid() >> 6;
  const float scale = 1.f / sqrtf((float)d);
  float* qs = lds;                       // [kMaxRows][d]
  float* kvs = qs + kMaxRows * d;        // [kMaxPos][2][d]
  float* os = kvs + kMaxPos * 2 * d;     // [kMaxRows][d]
  const float* qn = bfw(p, boff(p, l, p->o_qn));
  const float* kn = bfw(p, boff(p, l, p->o_kn));
  for (int u = blockIdx.x; u < bp->lanes * nq; u += bp->nwg) {
    const int ln = u / nq, h = u - ln * nq, g = h / grp;
    const int* st = sh->ln[ln];
    if (!st[kLnActive]) continue;
    const int fp = st[kLnFirst], R = st[kLnRows], row0 = ln * bp->rpl;
    float* kvc = bp->kv + (((size_t)ln * p->L + l) * p->nkv + g) * bp->kv_slots * 2 * d;
    // q, k, v of the lane's rows: the partial sums of 4 elements x 4 splits are in flight at once
    const int tot = R * 3 * d;
    for (int base = 0; base < tot; base += 4 * kThreads) {
      const float* src[4];
      float acc[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int e = base + k * kThreads + tid();
        const int r = e / (3 * d), w = e - r * 3 * d, part = w / d, i = w - part * d;
        const int col = part == 0 ? h * d + i : qdim + (part - 1) * kvdim + g * d + i;
        src[k] = e < tot ? bp->part + (size_t)(row0 + r) * N + col : nullptr;
        acc[k] = 0.f;
      }
      for (int ks0 = 0; ks0 < KS; ks0 += 4) {
        float t[4][4];
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            t[k][j] = (src[k] && ks0 + j < KS) ? cldf(src[k] + (size_t)(ks0 + j) * M * N) : 0.f;
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (ks0 + j < KS) acc[k] += t[k][j];
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int e = base + k * kThreads + tid();
        if (e < tot) {
          const int r = e / (3 * d), w = e - r * 3 * d, part = w / d, i = w - part * d;
          if (part == 0) qs[r * d + i] = acc[k];
          else kvs[(size_t)(fp + r) * 2 * d + (part - 1) * d + i] = acc[k];
        }
      }
    }
    lds_fill<true>(kvs, kvc, fp * 2 * d, 2 * d, (size_t)2 * d);
    __syncthreads();
    // q rows (v < R) and k rows (v >= R): norm + RoPE, one wave per vector
    for (int v = wave; v < 2 * R; v += kWaves) {
      const bool isq = v < R;
      const int r = isq ? v : v - R, pos = fp + r;
      float* x = isq ? qs + r * d : kvs + (size_t)pos * 2 * d;
      const float* gn = isq ? qn : kn;
      float ss = 0.f;
      for (int i = lane; i < d; i += 64) ss = fmaf(x[i], x[i], ss);
      ss = wave_sum(ss);
      const float rs = p->qk_norm ? 1.f / sqrtf(ss / (float)d + p->rms_eps) : 1.f;
      for (int i = lane; i < half; i += 64) {
        float a = x[i], b = x[i + half];
        if (p->qk_norm) {
          a = a * rs * G(gn)[i];
          b = b * rs * G(gn)[i + half];
        }
        const float cs = G(p->rope)[(pos * half + i) * 2], sn = G(p->rope)[(pos * half + i) * 2 + 1];
        x[i] = a * cs - b * sn;
        x[i + half] = b * cs + a * sn;
      }
    }
    __syncthreads();
    if (h % grp == 0)
      for (int e = tid(); e < R * 2 * d; e += kThreads) cstf(kvc + (size_t)fp * 2 * d + e, kvs[(size_t)fp * 2 * d + e]);
    for (int r = wave; r < R; r += kWaves) {
      const int s = fp + r;
      float sc[kMaxPos];
      float mx = -INFINITY;
#pragma unroll
      for (int t = 0; t < kMaxPos; ++t) {
        sc[t] = -INFINITY;
        if (t <= s) {
          float a = 0.f;
          for (int i = lane; i < d; i += 64) a = fmaf(qs[r * d + i], kvs[(size_t)t * 2 * d + i], a);
          sc[t] = wave_sum(a) * scale;
          mx = fmaxf(mx, sc[t]);
        }
      }
      float z = 0.f;
#pragma unroll
      for (int t = 0; t < kMaxPos; ++t) {
        sc[t] = t <= s ? expf(sc[t] - mx) : 0.f;
        z += sc[t];
      }
      const float iz = 1.f / z;
      for (int i = lane; i < d; i += 64) {
        float o = 0.f;
#pragma unroll
        for (int t = 0; t < kMaxPos; ++t)
          if (t <= s) o = fmaf(sc[t], kvs[(size_t)t * 2 * d + d + i], o);
        os[r * d + i] = o * iz;
      }
    }
    __syncthreads();
    for (int c = tid(); c < R * (d / 8); c += kThreads) {
      const int r = c / (d / 8), q8 = c - r * (d / 8);
      float x8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x8[e] = os[r * d + 8 * q8 + e];
      store_split(Aout + (size_t)(row0 + r) * qdim + h * d + 8 * q8, x8);
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------ residual + norm
// Row i: x += sum of the KS partial sums of the projection just run, then the
// next input: RMSNorm(x) * gain split into Aout (mode 0), or the final norm
// h and the LM-head inputs h + b_j of the row's used slots (mode 1).
template <bool TR>
__device__ __forceinline__ void phase_resid(const BParams* bp, BShared* sh, int KS, const float* gain, uint32_t* Aout, int mode,
                            float* xs) {
  const KParams* p = bp->k;
  const int H = p->H, M = bp->M, K = p->K;
  for (int i = blockIdx.x; i < M; i += bp->nwg) {
    const int ln = i / bp->rpl, r = i - ln * bp->rpl;
    const int* st = sh->ln[ln];
    if (!st[kLnActive] || r >= st[kLnRows]) continue;
    float* x = bp->x + (size_t)i * H;
    float ss = 0.f;
    for (int e = tid(); e < H; e += kThreads) {
      const float v = cldf(x + e) + sum_parts<true>(bp->part + (size_t)i * H + e, (size_t)M * H, KS);
      cstf(x + e, v);
      xs[e] = v;
      ss = fmaf(v, v, ss);
    }
    ss = block_sum(sh, ss);
    const float rs = 1.f / sqrtf(ss / (float)H + p->rms_eps);
    for (int c = tid(); c < H / 8; c += kThreads) {
      float h8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) h8[e] = xs[8 * c + e] * rs * G(gain)[8 * c + e];
      if (mode == 0) {
        store_split(Aout + (size_t)i * H + 8 * c, h8);
      } else {
        const float* ofs = bfw(p, p->o_offsets);
        for (int j = 0; j <= K; ++j) {
          if (!head_slot_used<TR>(bp, p, st, r, j)) continue;
          float y8[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) y8[e] = j == 0 ? h8[e] : h8[e] + G(ofs)[(size_t)(j - 1) * H + 8 * c + e];
          store_split(bp->ah + ((size_t)i * (K + 1) + j) * H + 8 * c, y8);
        }
      }
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------ LM heads
// Unit (head t, 64 vocabulary columns): every used slot (lane row, offset j)
// whose position plus offset is t, i.e. the verify rows at position t and the
// draft rows of distance j from it.
template <bool TR>
__device__ __forceinline__ void phase_heads(const BParams* bp, BShared* sh, float* red) {
  const KParams* p = bp->k;
  const int H = p->H, V = p->V, K = p->K, n = p->n_codes, rpl = bp->rpl;
  constexpr int NTU = TR ? 4 : kHeadNTU;  // the tree instantiation spills with the wider unit
  const int cg = (V + 16 * NTU - 1) / (16 * NTU), ncand = bp->lanes * rpl * (K + 1);
  if (tid() == 0) sh->hl_t = -1;
  __syncthreads();
  for (int u = blockIdx.x; u < n * cg; u += bp->nwg) {
    const int t = 1 + u / cg, gi = u % cg;
    if (sh->hl_t != t) {
      // row list of head t in candidate order
      int cnt = 0;
      for (int base = 0; base < ncand; base += kThreads) {
        const int c = base + tid();
        bool use = false;
        if (c < ncand) {
          const int ln = c / (rpl * (K + 1)), rem = c - ln * rpl * (K + 1), r = rem / (K + 1), j = rem - r * (K + 1);
          const int* st = sh->ln[ln];
          use = head_slot_used<TR>(bp, p, st, r, j) && row_pos<TR>(bp, st, r) + j == t;
        }
        int tot;
        const int pos = block_excl_scan(&sh->tk, use ? 1 : 0, &tot);
        if (use && cnt + pos < kBatchMaxRows) sh->hl_row[cnt + pos] = c;
        cnt += tot;
        __syncthreads();
      }
      if (tid() == 0) {
        sh->hl_n = min(cnt, kBatchMaxRows);
        sh->hl_t = t;
        if (cnt > kBatchMaxRows) raise_status(bp, RVQSD_EUNSUPPORTED);
      }
      __syncthreads();
    }
    const int nr = sh->hl_n;
    if (nr == 0) continue;
    const int n0 = gi * 16 * NTU;
    const bf16_t* W = bw(p, p->o_lmh1 + (uint64_t)(t - 1) * p->table_stride);
    gemm_unit<NTU, kProjNTW, true, true>(
        [&](int nt, int m) -> const bf16_t* {
          const int f = n0 + 16 * nt + m;
          return f < V ? W + (size_t)f * H : nullptr;
        },
        0, H, bp->ah, H, (nr + 15) >> 4, [&](int i) { return i < nr ? sh->hl_row[i] : -1; }, red);
    for (int e = tid(); e < NTU * ((nr + 15) >> 4) * 256; e += kThreads) {
      const int mtiles = (nr + 15) >> 4;
      const int nt = e / (mtiles * 256), rem = e - nt * (mtiles * 256), mt = rem >> 8, x = rem & 255;
      const int ln = x >> 2, v = x & 3;
      const int i = 16 * mt + (ln & 15), f = n0 + 16 * nt + 4 * (ln >> 4) + v;
      if (i < nr && f < V) cstf(bp->logits + (size_t)sh->hl_row[i] * V + f, red[((size_t)(nt * kBatchMTiles + mt) << 8) + x]);
    }
    __syncthreads();
  }
}

// Algorithmic bytes of one batched pass: the layer weights and every LM head
// some lane uses (each read once), the gathered embedding rows and the KV
// cache every lane attends over.
// Called by the 64 threads of one wave: thread i counts stream lane i, and the
// wave adds the counts and merges the used heads (integer sums: the order does
// not matter). The result is valid in every thread.
template <bool TR>
__device__ unsigned long long pass_bytes_batch(const BParams* bp, const BShared* sh) {
  const KParams* p = bp->k;
  const int lane = tid() & 63;
  const int H = p->H;
  const unsigned long long kv_pos = (unsigned long long)p->L * p->nkv * p->d * 2 * 4;  // KV bytes per position
  unsigned used = 0;  // bit t: head t used
  unsigned long long b = 0;
  if (lane < bp->lanes) {
    const int* st = sh->ln[lane];
    if (st[kLnActive]) {
      const int first = st[kLnFirst], rows = st[kLnRows];
      for (int r = 0; r < rows; ++r) {
        const int s = row_pos<TR>(bp, st, r);
        if (row_is_verify<TR>(bp, st, r)) used |= 1u << s;
        const int nd = row_drafts<TR>(bp, p, st, r);
        for (int j = 1; j <= nd; ++j) used |= 1u << (s + j);
        b += (s == 0) ? 4ull * H : 2ull * H;
      }
      b += kv_pos * (unsigned long long)(first + rows);
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    used |= (unsigned)__shfl_xor((int)used, o);
    b += (unsigned long long)__shfl_xor((long long)b, o);
  }
  return b + (unsigned long long)p->L * p->layer_stride + (unsigned long long)__popc(used) * p->table_stride;
}

// ------------------------------------------------------------ sampling
// Slot (lane row r, offset j): top-k of its logits, tempered softmax in fp64,
// then: j >= 1 -> draft d_{s+j} (inverse CDF at u_draft, or argmax) and its
// proposal q, recorded for the next pass; j = 0 with a draft -> accept d iff
// u_acc q(d) < p(d), else resample from max(0, p - q) at u_samp; j = 0
// without a draft (prefix token, or the extra token after every draft was
// accepted) -> sample p at u_samp. Verdict: token | accepted << 31.
template <bool TR>
__device__ __forceinline__ void phase_sample(const BParams* bp, BShared* sh, const BCall& call, float* lds) {
  const KParams* p = bp->k;
  const int V = p->V, K = p->K, rpl = bp->rpl, n = p->n_codes, SW = bp->sup_words;
  float* lg = lds;                                            // [V]
  int* sidx = reinterpret_cast<int*>(lg + V);                 // [kMaxTopk]
  float* slog = reinterpret_cast<float*>(sidx + kMaxTopk);    // [kMaxTopk]
  // fp64 arrays from the next 8-byte boundary (lg is 8-byte aligned); an index, not an
  // integer cast of the pointer, so that the compiler keeps them in the LDS address space
  double* prob = reinterpret_cast<double*>(lg + ((V + 2 * kMaxTopk + 1) & ~1));  // [kMaxTopk]
  double* qprob = prob + kMaxTopk;
  double* res = qprob + kMaxTopk;
  int* qidx = reinterpret_cast<int*>(res + kMaxTopk);         // [kMaxTopk]
  unsigned* hist = reinterpret_cast<unsigned*>(qidx + kMaxTopk);  // [kTopkBuckets]
  const int nslots = bp->lanes * rpl * (K + 1);
  for (int u = blockIdx.x; u < nslots; u += bp->nwg) {
    const int ln = u / (rpl * (K + 1)), rem = u - ln * rpl * (K + 1), r = rem / (K + 1), j = rem - r * (K + 1);
    const int* st = sh->ln[ln];
    if (!head_slot_used<TR>(bp, p, st, r, j)) continue;
    const int pass = st[kLnPass], s = row_pos<TR>(bp, st, r), t = s + j;
    const float* U = call.uniforms + (size_t)st[kLnFrame] * n * 3;
    const bool tree_pass = tree_rows<TR>(bp, st);
    const bool has_draft = !TR && j == 0 && pass > 0 && r + 1 <= st[kLnKp];
    int nq = 0, dtok = -1;
    if (has_draft) {
      // q of d_t: drafted last pass from the anchor's row, offset r + 1; the whole support
      // area (topk entries, of which the first nq are this record's) is read together with
      // the header and the logits instead of after the header
      const uint64_t* rec = bp->drec + ((((size_t)((pass - 1) & 1) * bp->lanes + ln) * rpl + st[kLnPrevAnchor]) * K + r) * SW;
      const uint64_t w0 = cld64(rec);
      for (int i = tid(); i < p->topk; i += kThreads) {
        qidx[i] = (int)(uint32_t)cld64(rec + 1 + i);
        qprob[i] = __longlong_as_double((long long)cld64(rec + 1 + p->topk + i));
      }
      dtok = (int)(uint32_t)w0;
      nq = (int)(w0 >> 32);
    }
    const float* src = bp->logits + (size_t)u * V;
    lds_fill<true>(lg, src, V, V, 0);
    __syncthreads();
    if (bp->tr_logits && st[kLnFrame] < bp->tr_frames && pass < bp->tr_max_rounds) {
      // the slot layout of the single-stream trace: verify row r, then draft (r, j)
      const int slot = j == 0 ? r : bp->slot_draft0 + r * K + (j - 1);
      float* dst = bp->tr_logits + (((size_t)st[kLnFrame] * bp->tr_max_rounds + pass) * bp->tr_slots + slot) * V;
      for (int i = tid(); i < V; i += kThreads) dst[i] = lg[i];
    }
    int ns = topk_buckets(&sh->tk, lg, V, p->topk, sidx, slog, hist);
    if (ns < 0) ns = topk_select(&sh->tk, lg, V, p->topk, sidx, slog);
    if (tid() < 64) {
      bool fin = false;
      for (int i = tid(); i < ns; i += 64) fin |= (slog[i] > -INFINITY && slog[i] < INFINITY);
      if (!__any(fin) && tid() == 0) raise_status(bp, RVQSD_ENUMERIC);
    }
    if (TR && j > 0) {
      // tree lanes: the ranked candidates of depth j for the rows of a round anchored at
      // this row: rank = larger logit first, ties to the lower token (within the top-k
      // support, which holds every rank below top-k)
      const int need = min(bp->t_need[j], ns);
      uint64_t* rec = bp->drec + ((((size_t)(pass & 1) * bp->lanes + ln) * rpl + r) * K + (j - 1)) * SW;
      for (int i = tid(); i < ns; i += kThreads) {
        const float v = slog[i];
        const int x = sidx[i];
        int rank = 0;
        for (int k = 0; k < ns; ++k) rank += (slog[k] > v || (slog[k] == v && sidx[k] < x)) ? 1 : 0;
        if (rank < need) cst64(rec + 1 + rank, (uint64_t)(uint32_t)x);
      }
      if (tid() == 0) cst64(rec, (uint64_t)(uint32_t)need);
      __syncthreads();
      continue;
    }
    softmax_support(slog, ns, p->temperature, prob);
    __syncthreads();
    if (tree_pass) {
      // verify row of a tree: its children (rows of the next depth under it, the candidates
      // for position s) are tried in increasing rank; child i is accepted iff
      // sum_{l<i} p(x_l) <= u_acc < sum_{l<=i} p(x_l); with none accepted, c_s is drawn with
      // u_samp from p without the children's tokens (p itself when nothing is left)
      if (tid() == 0) {
        int nk = 0;
        const int ncand = st[kLnCandN];
        for (int c = r + 1; c < ncand; ++c)
          if (bp->t_parent[c] == r) {
            int at = nk++;
            while (at > 0 && bp->t_rank[sh->kid[at - 1]] > bp->t_rank[c]) { sh->kid[at] = sh->kid[at - 1]; --at; }
            sh->kid[at] = c;
          }
        sh->nkid = nk;
      }
      __syncthreads();
      if (tid() < 64) {
        const int nk = sh->nkid;
        const double ua = (double)U[(s - 1) * 3 + 1];
        double cum = 0.0;
        int taken = -1;
        for (int c = 0; c < nk; ++c) {
          const int x = st[kLnCand + sh->kid[c]];
          double pc = 0.0;
          for (int i = tid(); i < ns; i += 64)
            if (sidx[i] == x) pc = prob[i];
          cum += wave_sumd_dpp(pc);
          if (taken < 0 && ua < cum) taken = sh->kid[c];
        }
        int tok = 0;
        if (taken < 0) {
          double rs = 0.0;
          for (int i = tid(); i < ns; i += 64) {
            bool kid = false;
            for (int c = 0; c < nk; ++c) kid |= sidx[i] == st[kLnCand + sh->kid[c]];
            res[i] = kid ? 0.0 : prob[i];
            rs += res[i];
          }
          rs = wave_sumd_dpp(rs);
          if (!(rs > 0.0))
            for (int i = tid(); i < ns; i += 64) res[i] = prob[i];
          __builtin_amdgcn_wave_barrier();
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
          tok = sidx[inverse_cdf(res, ns, (double)U[(s - 1) * 3 + 2])];
        }
        if (tid() == 0) cst32(bp->vres + ln * rpl + r, (uint32_t)tok | ((uint32_t)(taken + 1) << 24));
      }
      __syncthreads();
      continue;
    }
    if (j > 0) {
      if (tid() < 64) {
        int pos;
        if (p->greedy) {
          double best = -1.0;
          int bi = ns;
          for (int i = tid(); i < ns; i += 64)
            if (prob[i] > best) { best = prob[i]; bi = i; }
          for (int o = 32; o > 0; o >>= 1) {
            const double ob = __shfl_xor(best, o, 64);
            const int oi = __shfl_xor(bi, o, 64);
            if (ob > best || (ob == best && oi < bi)) { best = ob; bi = oi; }
          }
          pos = bi;
        } else {
          pos = inverse_cdf(prob, ns, (double)U[(t - 1) * 3 + 0]);
        }
        if (tid() == 0) sh->tok = sidx[pos];
      }
      __syncthreads();
      const int tok = sh->tok, nrec = p->greedy ? 1 : ns;
      uint64_t* rec = bp->drec + ((((size_t)(pass & 1) * bp->lanes + ln) * rpl + r) * K + (j - 1)) * SW;
      for (int i = tid(); i < nrec; i += kThreads) {
        cst64(rec + 1 + i, (uint64_t)(uint32_t)(p->greedy ? tok : sidx[i]));
        cst64(rec + 1 + p->topk + i, (uint64_t)__double_as_longlong(p->greedy ? 1.0 : prob[i]));
      }
      if (tid() == 0) cst64(rec, (uint64_t)(uint32_t)tok | ((uint64_t)(uint32_t)nrec << 32));
    } else if (tid() < 64) {
      int tok;
      bool accept = false;
      if (has_draft) {
        double pd = 0.0, qd = 0.0;
        for (int i = tid(); i < ns; i += 64)
          if (sidx[i] == dtok) pd = prob[i];
        for (int i = tid(); i < nq; i += 64)
          if (qidx[i] == dtok) qd = qprob[i];
        pd = wave_sumd_dpp(pd);
        qd = wave_sumd_dpp(qd);
        accept = (double)U[(t - 1) * 3 + 1] * qd < pd;
        tok = dtok;
        if (!accept) {
          double rs = 0.0;
          for (int i = tid(); i < ns; i += 64) {
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
            for (int i = tid(); i < ns; i += 64) res[i] = prob[i];
          __builtin_amdgcn_wave_barrier();
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
          tok = sidx[inverse_cdf(res, ns, (double)U[(t - 1) * 3 + 2])];
        }
      } else {
        tok = sidx[inverse_cdf(prob, ns, (double)U[(t - 1) * 3 + 2])];
      }
      if (tid() == 0) cst32(bp->vres + ln * rpl + r, (uint32_t)tok | (accept ? 0x80000000u : 0u));
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------ commit + row setup
// Lane workgroup: commit the verdicts of the pass just sampled, pick the next
// anchor and its drafts (or finish the frame and start the lane's next one),
// then gather and normalise the new rows (layer 0 input). first: no pass yet.
// c0 in [0, V) and every uniform of the frame in [0, 1) (NaN fails): a frame that fails
// is not decoded; it reports EINVAL
__device__ __forceinline__ bool frame_inputs_ok(const BCall& call, int f, int V, int n) {
  const int c0 = call.c0[f];
  if (c0 < 0 || c0 >= V) return false;
  const float* U = call.uniforms + (size_t)f * n * 3;
  bool ok = true;
  for (int i = 0; i < 3 * n; ++i) {
    const float u = U[i];
    ok &= u >= 0.f && u < 1.f;
  }
  return ok;
}

template <bool TR>
__device__ __forceinline__ void lane_commit(const BParams* bp, BShared* sh, const BCall& call, bool first, float* xs,
                            uint32_t* A0) {
  const KParams* p = bp->k;
  const int lane_id = blockIdx.x, rpl = bp->rpl, K = p->K, n = p->n_codes, H = p->H;
  int* st = sh->ln[lane_id];
  int* gst = bp->lane + (size_t)lane_id * kLaneInts;
  // st already holds this lane's state: every workgroup loads all lane states at the start of a
  // pass, and only this workgroup writes them
  const int f_next = (first ? lane_id - bp->lanes : st[kLnFrame]) + bp->lanes;
  if (first) {
    for (int i = tid(); i < kLaneInts; i += kThreads) st[i] = 0;
    if (tid() == 0) st[kLnFrame] = lane_id - bp->lanes;
  }
  // inputs of the lane's next frame (c0 and its uniforms), checked by many threads now
  // rather than by one when the frame starts
  int c0_next = -1, bad_next = 0;
  if (f_next < call.n && tid() <= 3 * n) {
    if (tid() == 0) {
      c0_next = call.c0[f_next];
      bad_next = c0_next < 0 || c0_next >= p->V;
    } else {
      const float u = call.uniforms[(size_t)f_next * n * 3 + tid() - 1];
      bad_next = !(u >= 0.f && u < 1.f);
    }
  }
  const bool next_ok = !__syncthreads_or(bad_next);
  const bool was_active = !first && st[kLnActive];
  const bool tree_pass = was_active && tree_rows<TR>(bp, st);
  if (was_active) {
    const int R = st[kLnRows];
    for (int i = tid(); i < R; i += kThreads) sh->vr[i] = (int)cld32(bp->vres + lane_id * rpl + i);
    const int par = st[kLnPass] & 1;
    if (!TR)
      for (int i = tid(); i < R * K; i += kThreads) {
        const int r = i / K, jj = i - r * K;
        sh->dt[r][jj] = jj < row_drafts<TR>(bp, p, st, r)
                            ? (int)(uint32_t)cld64(bp->drec + ((((size_t)par * bp->lanes + lane_id) * rpl + r) * K + jj) * bp->sup_words)
                            : -1;
      }
  }
  __syncthreads();
  // tree lanes: commit the pass (the prefix token, or a walk of the verdicts from the root),
  // count it and trace it, before the candidates of the next round replace this round's
  if (tid() == 0) {
    sh->c_mnew = -1;
    if (was_active && TR) {
      const int m = st[kLnM], fp = st[kLnFirst], R = st[kLnRows];
      int* codes = st + kLnCodes;
      int cur = 1, acc = 0, m_new = 1, tok = -1;
      if (st[kLnPass] == 0) {
        codes[1] = sh->vr[1] & 0x7fffffff;
        tok = codes[1];
      } else {
        int pos = m + 1;
        cur = 0;
        while (true) {
          const int v = sh->vr[cur];
          const int child = (int)((uint32_t)v >> 24) - 1;
          if (child >= 0) {
            codes[pos] = st[kLnCand + child];
            st[kLnMask] |= 1 << pos;
            sh->c_path[acc++] = child;
            cur = child;
            if (++pos > n) { m_new = n; break; }
            continue;
          }
          codes[pos] = v & 0xffffff;
          tok = codes[pos];
          m_new = pos;
          break;
        }
        st[kLnRounds] += 1;
        st[kLnDrafted] += st[kLnCandN] - 1;
        st[kLnAccepted] += acc;
      }
      st[kLnCalls] += 1;
      if (st[kLnCalls] > n + 1) raise_status(bp, RVQSD_ETIMEOUT);
      if (bp->tr_rounds && st[kLnFrame] < bp->tr_frames && st[kLnPass] < bp->tr_max_rounds) {
        int32_t* tr = bp->tr_rounds + ((size_t)st[kLnFrame] * bp->tr_max_rounds + st[kLnPass]) * kTreeRoundInts;
        tr[0] = m; tr[1] = st[kLnKp]; tr[2] = fp; tr[3] = R; tr[4] = m_new; tr[5] = acc; tr[6] = tok;
        tr[7] = st[kLnPass];
        tr[8] = st[kLnPass] == 0 ? 2 : st[kLnCandN];
        for (int j = 0; j < acc; ++j) tr[16 + j] = sh->c_path[j];
        for (int r = 0; st[kLnPass] > 0 && r < st[kLnCandN]; ++r) tr[32 + r] = st[kLnCand + r];
      }
      sh->c_mnew = m_new;
      sh->c_arow = cur;
      sh->c_acc = acc;
      sh->c_m = m;
    }
  }
  __syncthreads();
  if (was_active && TR) {
    const int m = sh->c_m, acc = tree_pass ? sh->c_acc : 0, m_new = sh->c_mnew, arow = sh->c_arow;
    const int d = p->d, slots = bp->kv_slots;
    // KV of the accepted path: row path[j-1] (slot m+1+row) becomes position m+1+j, every
    // layer and kv head; destinations never overlap a later source (path[j-1] >= j)
    for (int j = 1; j <= acc; ++j) {
      const int src = m + 1 + sh->c_path[j - 1], dst = m + 1 + j;
      if (src == dst) continue;
      const int per = p->L * p->nkv * 2 * d;
      for (int e = tid(); e < per; e += kThreads) {
        const int lg = e / (2 * d), w = e - lg * 2 * d;
        float* base = bp->kv + ((size_t)lane_id * p->L * p->nkv + lg) * slots * 2 * d;
        cstf(base + (size_t)dst * 2 * d + w, cldf(base + (size_t)src * 2 * d + w));
      }
      __syncthreads();
    }
    // the next round's candidates: depth d's rank-r token from the new anchor row's drafts
    if (m_new < n) {
      const int kn = min(K, n - m_new), par = st[kLnPass] & 1;
      for (int r = 1 + tid(); r <= bp->tree_nodes; r += kThreads)
        if (bp->t_depth[r] <= kn)
          st[kLnCand + r] = (int)(uint32_t)cld64(bp->drec + ((((size_t)par * bp->lanes + lane_id) * rpl + arow) * K +
                                                         (bp->t_depth[r] - 1)) * bp->sup_words + 1 + bp->t_rank[r]);
    }
  }
  __syncthreads();
  if (tid() == 0) {
    bool start = first || !st[kLnActive];
    bool done = false;  // the lane's frame is complete
    if (!first && st[kLnActive] && TR) {
      // tree lanes: the pass was committed above; set up the next round
      const int m_new = sh->c_mnew;
      int* codes = st + kLnCodes;
      if (m_new < n) {
        const int kn = min(K, n - m_new);
        int ncand = 1;
        while (ncand <= bp->tree_nodes && bp->t_depth[ncand] <= kn) ++ncand;
        int R = 1;
        while (R < ncand && m_new + 1 + bp->t_depth[R] <= n) ++R;
        st[kLnCand + 0] = codes[m_new];
        st[kLnCandN] = ncand;
        st[kLnPrevAnchor] = sh->c_arow;
        st[kLnKp] = kn;
        st[kLnRows] = R;
        st[kLnFirst] = m_new + 1;
        st[kLnM] = m_new;
        st[kLnPass] += 1;
      } else {
        done = true;
      }
    }
    if (!first && st[kLnActive] && !TR) {
      const int m = st[kLnM], kp = st[kLnKp], R = st[kLnRows], fp = st[kLnFirst];
      int* codes = st + kLnCodes;
      int m_new = -1, acc = 0, tok = -1;
      if (st[kLnPass] == 0) {
        codes[1] = sh->vr[1] & 0x7fffffff;
        m_new = 1;
        tok = codes[1];
      } else {
        for (int j = 1; j <= kp; ++j) {
          const int v = sh->vr[j - 1];
          if (v & 0x80000000) {
            codes[m + j] = st[kLnDrafts + m + j];
            ++acc;
            st[kLnMask] |= 1 << (m + j);
          } else {
            codes[m + j] = v & 0x7fffffff;
            m_new = m + j;
            tok = codes[m_new];
            break;
          }
        }
        if (m_new < 0) {
          if (R > kp) {
            codes[m + kp + 1] = sh->vr[kp] & 0x7fffffff;
            m_new = m + kp + 1;
            tok = codes[m_new];
          } else {
            m_new = n;
          }
        }
        st[kLnRounds] += 1;
        st[kLnDrafted] += kp;
        st[kLnAccepted] += acc;
      }
      if (bp->tr_rounds && st[kLnFrame] < bp->tr_frames && st[kLnPass] < bp->tr_max_rounds) {
        int32_t* tr = bp->tr_rounds + ((size_t)st[kLnFrame] * bp->tr_max_rounds + st[kLnPass]) * kTraceRoundInts;
        tr[0] = m; tr[1] = kp; tr[2] = fp; tr[3] = R; tr[4] = m_new; tr[5] = acc; tr[6] = tok; tr[7] = st[kLnPass];
        for (int j = 1; j <= kp; ++j) tr[7 + j] = st[kLnDrafts + m + j];
      }
      st[kLnCalls] += 1;
      // every pass commits at least one code: a frame still open after n + 1 passes is a fault
      if (st[kLnCalls] > n + 1) raise_status(bp, RVQSD_ETIMEOUT);
      if (m_new < n) {
        const int arow = m_new - fp;
        const int nd = min(K, n - m_new);
        for (int jj = 1; jj <= nd; ++jj) st[kLnDrafts + m_new + jj] = sh->dt[arow][jj - 1];
        st[kLnPrevAnchor] = arow;
        st[kLnKp] = nd;
        st[kLnRows] = min(nd + 1, n - m_new);
        st[kLnFirst] = m_new + 1;
        st[kLnInCode + m_new + 1] = codes[m_new];
        for (int r = 1; r < st[kLnRows]; ++r) st[kLnInCode + m_new + 1 + r] = st[kLnDrafts + m_new + r];
        st[kLnM] = m_new;
        st[kLnPass] += 1;
      } else {
        done = true;
      }
    }
    if (done) {
      // frame complete
      const int f = st[kLnFrame];
      int* codes = st + kLnCodes;
      for (int s = 1; s <= n; ++s) call.out_codes[(size_t)f * n + s - 1] = codes[s];
      rvqsd_stats o;
      o.target_calls = st[kLnCalls];
      o.rounds = st[kLnRounds];
      o.drafted = st[kLnDrafted];
      o.accepted = st[kLnAccepted];
      o.accept_mask = (uint32_t)st[kLnMask];
      o.status = RVQSD_OK;
      o.weight_bytes = (uint64_t)(uint32_t)st[kLnBytesLo] | ((uint64_t)(uint32_t)st[kLnBytesHi] << 32);
      o.clk_start = (uint64_t)(uint32_t)st[kLnClkLo] | ((uint64_t)(uint32_t)st[kLnClkHi] << 32);
      o.clk_end = dclock();
      call.out_stats[f] = o;
      start = true;
    }
    if (start) {
      // the lane's next frame with a valid c0
      int f = st[kLnFrame] + bp->lanes;
      bool f_ok = next_ok;  // f == f_next
      while (f < call.n && !f_ok) {
        rvqsd_stats o = {};
        o.status = RVQSD_EINVAL;
        call.out_stats[f] = o;
        for (int s = 0; s < n; ++s) call.out_codes[(size_t)f * n + s] = -1;
        f += bp->lanes;
        f_ok = f < call.n && frame_inputs_ok(call, f, p->V, n);
        if (f < call.n) c0_next = call.c0[f];
      }
      for (int i = 0; i < kLaneInts; ++i) st[i] = 0;
      st[kLnFrame] = f;
      if (f < call.n) {
        const uint64_t now = dclock();
        st[kLnActive] = 1;
        st[kLnRows] = 2;
        st[kLnCodes] = c0_next;
        st[kLnInCode + 1] = c0_next;
        st[kLnClkLo] = (int)(uint32_t)now;
        st[kLnClkHi] = (int)(uint32_t)(now >> 32);
      }
    }
    if (st[kLnActive]) {
      // algorithmic bytes of this pass if the frame were decoded alone: layer weights,
      // the heads it touches, the gathered rows and the KV cache it attends over
      int t_lo = 1 << 20, t_hi = -1;
      for (int r = 0; r < st[kLnRows]; ++r) {
        const int s = row_pos<TR>(bp, st, r);
        if (row_is_verify<TR>(bp, st, r)) { t_lo = min(t_lo, s); t_hi = max(t_hi, s); }
        const int nd = row_drafts<TR>(bp, p, st, r);
        if (nd > 0) { t_lo = min(t_lo, s + 1); t_hi = max(t_hi, s + nd); }
      }
      unsigned long long b = (unsigned long long)p->L * p->layer_stride;
      if (t_hi >= t_lo) b += (unsigned long long)(t_hi - t_lo + 1) * p->table_stride;
      for (int r = 0; r < st[kLnRows]; ++r) b += (row_pos<TR>(bp, st, r) == 0) ? 4ull * H : 2ull * H;
      b += (unsigned long long)p->L * (st[kLnFirst] + st[kLnRows]) * p->nkv * p->d * 2 * 4;
      b += (uint64_t)(uint32_t)st[kLnBytesLo] | ((uint64_t)(uint32_t)st[kLnBytesHi] << 32);
      st[kLnBytesLo] = (int)(uint32_t)b;
      st[kLnBytesHi] = (int)(uint32_t)(b >> 32);
    }
  }
  __syncthreads();
  for (int i = tid(); i < kLaneInts; i += kThreads) cst32(gst + i, (uint32_t)st[i]);
  // layer-0 input of the lane's rows: one wave per row, lane l holds 8-element chunks l, l + 64, ..
  if (!st[kLnActive]) return;
  const float* g0 = bfw(p, p->o_attn_norm);
  const int lane = tid() & 63, wave = tid() >> 6, nch = H / 8;
  const bool tree_next = tree_rows<TR>(bp, st);
  for (int r = wave; r < st[kLnRows]; r += kWaves) {
    const int s = row_pos<TR>(bp, st, r), i = lane_id * rpl + r;
    const int code = tree_next ? st[kLnCand + r] : st[kLnInCode + s];
    float xv[kRowChunks][8];
    float ss = 0.f;
#pragma unroll
    for (int q = 0; q < kRowChunks; ++q) {
      const int c = lane + 64 * q;
      if (c < nch) {
        if (s == 0) {
          const float* fr = call.frame_hidden + (size_t)st[kLnFrame] * H + 8 * c;
#pragma unroll
          for (int e = 0; e < 8; ++e) xv[q][e] = G(fr)[e];
        } else {
          const bf16_t* tab = bw(p, p->o_emb0 + (uint64_t)(s - 1) * p->table_stride);
          const W16 w = *G(reinterpret_cast<const W16*>(tab + (size_t)code * H + 8 * c));
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            xv[q][2 * e] = __uint_as_float(w[e] << 16);
            xv[q][2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
          }
        }
        float* xd = bp->x + (size_t)i * H + 8 * c;
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          cst64(xd + e, (uint64_t)__float_as_uint(xv[q][e]) | ((uint64_t)__float_as_uint(xv[q][e + 1]) << 32));
          ss = fmaf(xv[q][e], xv[q][e], fmaf(xv[q][e + 1], xv[q][e + 1], ss));
        }
      }
    }
    ss = wave_sum(ss);
    const float rs = 1.f / sqrtf(ss / (float)H + p->rms_eps);
#pragma unroll
    for (int q = 0; q < kRowChunks; ++q) {
      const int c = lane + 64 * q;
      if (c < nch) {
        float h8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) h8[e] = xv[q][e] * rs * G(g0)[8 * c + e];
        store_split(A0 + (size_t)i * H + 8 * c, h8);
      }
    }
  }
}

// A lane's frames that did not complete when the launch ended early
__device__ void lane_abort(const BParams* bp, BShared* sh, const BCall& call) {
  if (tid() != 0) return;
  const int code = (int)cld32(bp->status);
  const int n = bp->k->n_codes;
  const int* st = sh->ln[blockIdx.x];
  int f = st[kLnActive] ? st[kLnFrame] : st[kLnFrame] + bp->lanes;
  if (f < 0) f = blockIdx.x;
  for (; f < call.n; f += bp->lanes) {
    rvqsd_stats o = {};
    o.status = code ? code : RVQSD_ETIMEOUT;
    call.out_stats[f] = o;
    for (int s = 0; s < n; ++s) call.out_codes[(size_t)f * n + s] = -1;
  }
}

template <bool TR>
__global__ void __launch_bounds__(kThreads, 1) batch_kernel(const BParams* __restrict__ bpp, BCall call) {
  __shared__ BShared shs;
  extern __shared__ __align__(16) float dyn[];
  const BParams* bp = bpp;
  const KParams* p = bp->k;
  BShared* sh = &shs;
  uint32_t gen = 0;
  const int L = p->L, H = p->H;
  uint32_t* A0 = bp->a;
  uint32_t* A1 = bp->a + (size_t)bp->M * max(max(H, p->qdim), p->F);
  const bool lane_wg = (int)blockIdx.x < bp->lanes;
  bool first = true, ok = true;
  // passes and their algorithmic bytes, counted by the last workgroup while the first
  // residual phase keeps it idle (it owns no row when nwg > M)
  const bool counter_wg = (int)blockIdx.x == bp->nwg - 1;
  unsigned long long n_pass = 0, n_bytes = 0;
  while (ok) {
    if (lane_wg) lane_commit<TR>(bp, sh, call, first, dyn, A0);
    first = false;
    if (!(ok = grid_sync<BParams, false>(bp, gen, sh))) break;
    for (int i = tid(); i < bp->lanes * kLaneInts; i += kThreads)
      sh->ln[i / kLaneInts][i % kLaneInts] = (int)cld32(bp->lane + i);
    __syncthreads();
    int any = 0;
    for (int i = 0; i < bp->lanes; ++i) any |= sh->ln[i][kLnActive];
    if (!any) break;
    for (int l = 0; l < L && ok; ++l) {
      proj_partial<4, BParams, true, true>(bp, bw(p, boff(p, l, p->o_wq)), p->nqkv, H, bp->ks_qkv, A0, dyn);
      ok = grid_sync<BParams, false>(bp, gen, sh);
      if (ok) {
        if (TR) phase_attn_tree(bp, sh, l, A1, dyn);
        else phase_attn(bp, sh, l, A1, dyn);
      }
      ok = ok && grid_sync<BParams, false>(bp, gen, sh);
      if (ok) proj_partial<4, BParams, true, true>(bp, bw(p, boff(p, l, p->o_wo)), H, p->qdim, bp->ks_o, A1, dyn);
      ok = ok && grid_sync<BParams, false>(bp, gen, sh);
      if (ok) phase_resid<TR>(bp, sh, bp->ks_o, bfw(p, boff(p, l, p->o_mlp_norm)), A0, 0, dyn);
      if (ok && l == 0 && counter_wg && tid() < 64) {
        const unsigned long long pb = pass_bytes_batch<TR>(bp, sh);
        if (tid() == 0) {
          n_pass += 1;
          n_bytes += pb;
        }
      }
      ok = ok && grid_sync<BParams, false>(bp, gen, sh);
      if (ok) phase_gu<BParams, true>(bp, l, A0, A1, dyn);
      ok = ok && grid_sync<BParams, false>(bp, gen, sh);
      if (ok) proj_partial<4, BParams, true, true>(bp, bw(p, boff(p, l, p->o_wd)), H, p->F, bp->ks_down, A1, dyn);
      ok = ok && grid_sync<BParams, false>(bp, gen, sh);
      if (ok) {
        if (l + 1 < L) phase_resid<TR>(bp, sh, bp->ks_down, bfw(p, boff(p, l + 1, p->o_attn_norm)), A0, 0, dyn);
        else phase_resid<TR>(bp, sh, bp->ks_down, bfw(p, p->o_final_norm), nullptr, 1, dyn);
      }
      ok = ok && grid_sync<BParams, false>(bp, gen, sh);
    }
    if (!ok) break;
    phase_heads<TR>(bp, sh, dyn);
    if (!(ok = grid_sync<BParams, false>(bp, gen, sh))) break;
    phase_sample<TR>(bp, sh, call, dyn);
    if (!(ok = grid_sync<BParams, false>(bp, gen, sh))) break;
  }
  if (!ok && lane_wg) lane_abort(bp, sh, call);
  if (counter_wg && tid() == 0) {
    bp->totals[0] = n_pass;
    bp->totals[1] = n_bytes;
  }
}

// ------------------------------------------------------------ outer decoder step
// One position of the outer CodeDecoder (Fig. 1): input row x = t + E_0[c_0] +
// sum_j E_j[c_j] of the previous frame, the decoder stack with the KV cache of
// all earlier frames, the head's logits over the codes the inner tables can
// embed, and a top-k, temperature-T draw of c_0. Same phase chain as the batched
// kernel with M = 1; attention is split over key chunks (16 per query head) whose
// partial softmax sums are merged by a second phase.

// row set-up (workgroup 0): x and the split, normalised layer-0 input
__device__ void outer_input(const OParams* op, BShared* sh, const OCall& call, uint32_t* A0, float* xs) {
  const KParams* p = op->k;
  const int H = p->H;
  float ss = 0.f;
  // the previous frame's codes (one thread each) must be in range (a failed frame leaves -1):
  // else no input
  __shared__ int pcodes[kMaxCodes + 1];
  __shared__ int pbad;
  const int nt = op->n_tables;
  if (tid() == 0) pbad = 0;
  __syncthreads();
  if (call.prev_codes && tid() <= nt) {
    const int c = G(call.prev_codes)[tid()];
    pcodes[tid()] = c;
    if (!(c >= 0 && c < (tid() == 0 ? min(p->V, op->table_vocab) : op->table_vocab))) pbad = 1;
  }
  __syncthreads();
  const bool codes_ok = call.prev_codes != nullptr && pbad == 0;
  if (call.prev_codes && !codes_ok && tid() == 0) raise_status(op, RVQSD_EINVAL);
  for (int e = tid(); e < H; e += kThreads) {
    float v = G(call.t)[e];
    if (codes_ok) {
      // every table row of this element is loaded before the sum (in table order) is taken
      const bf16_t* e0 = bw(p, p->o_emb0);
      uint32_t tv[kMaxCodes + 1];
      tv[0] = G(e0)[(size_t)pcodes[0] * H + e];
#pragma unroll
      for (int j = 1; j <= kMaxCodes; ++j)
        tv[j] = j <= nt ? G(op->tables)[((size_t)(j - 1) * op->table_vocab + pcodes[j]) * H + e] : 0u;
      v += __uint_as_float(tv[0] << 16);
#pragma unroll
      for (int j = 1; j <= kMaxCodes; ++j)
        if (j <= nt) v += __uint_as_float(tv[j] << 16);
    }
    cstf(op->x + e, v);
    xs[e] = v;
    ss = fmaf(v, v, ss);
  }
  ss = block_sum(sh, ss);
  const float rs = 1.f / sqrtf(ss / (float)H + p->rms_eps);
  const float* g0 = bfw(p, p->o_attn_norm);
  for (int c = tid(); c < H / 8; c += kThreads) {
    float h8[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) h8[e] = xs[8 * c + e] * rs * G(g0)[8 * c + e];
    store_split(A0 + 8 * c, h8);
  }
}

// dst[e] = src[e] for n4 16-byte groups (both 16-byte aligned); each thread has 16 loads in flight
__device__ __forceinline__ void lds_fill4(float* dst, const float* src, int n4) {
  for (int base = 0; base < n4; base += 16 * kThreads) {
    f32x4 v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int e = base + k * kThreads + tid();
      v[k] = e < n4 ? G(reinterpret_cast<const f32x4*>(src))[e] : (f32x4){0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int e = base + k * kThreads + tid();
      if (e < n4) reinterpret_cast<f32x4*>(dst)[e] = v[k];
    }
  }
}

// Chunk attention: unit (query head h, key chunk c) over the positions of that chunk.
// The chunk's keys and values come into LDS in one batch of loads; each position's
// softmax weight exp(s_t - max) is taken once, and the weighted sum of the values is
// split over nog = kThreads / d groups of positions that are added in group order.
__device__ void outer_attn(const OParams* op, BShared* sh, int l, int pos, float* lds) {
  const KParams* p = op->k;
  const int d = p->d, nq = p->nq, grp = nq / p->nkv, N = p->nqkv, KS = op->ks_qkv, half = d / 2;
  const int lane = tid() & 63, wave = tid() >> 6;
  const int np = pos + 1, ch = attn_chunk_len(np, d), nch = (np + ch - 1) / ch;
  const int nog = kThreads / d;
  float* qv = lds;                // [d]
  float* kn = qv + d;             // [d] this position's k
  float* vn = kn + d;             // [d] this position's v
  float* sc = vn + d;             // [ch] scores, then softmax weights
  float* og = sc + ch;            // [nog][d] group sums of the weighted values
  float* zg = og + nog * d;       // [nog] group sums of the weights
  float* kvs = lds + ((3 * d + ch + nog * d + nog + 3) & ~3);  // [ch][2d] the chunk's keys and values
  const float* qn = bfw(p, boff(p, l, p->o_qn));
  const float* kng = bfw(p, boff(p, l, p->o_kn));
  const float scale = 1.f / sqrtf((float)d);
  for (int u = blockIdx.x; u < nq * nch; u += op->nwg) {
    const int h = u / nch, c = u - h * nch, g = h / grp;
    const int t0 = c * ch, t1 = min(np, t0 + ch), n = t1 - t0;
    float* kvc = op->kv + (((size_t)l * p->nkv + g) * op->max_frames) * 2 * d;
    lds_fill4(kvs, kvc + (size_t)t0 * 2 * d, n * d / 2);
    for (int e = tid(); e < 3 * d; e += kThreads) {
      const int part = e / d, i = e - part * d;
      const int col = part == 0 ? h * d + i : p->qdim + (part - 1) * p->kvdim + g * d + i;
      const float v = sum_parts<true>(op->part + col, (size_t)N, KS);
      (part == 0 ? qv : part == 1 ? kn : vn)[i] = v;
    }
    __syncthreads();
    // per-head RMSNorm + RoPE of q (wave 0) and k (wave 1) at this position
    if (wave < 2) {
      float* x = wave == 0 ? qv : kn;
      const float* gn = wave == 0 ? qn : kng;
      float s2 = 0.f;
      for (int i = lane; i < d; i += 64) s2 = fmaf(x[i], x[i], s2);
      s2 = wave_sum(s2);
      const float rs = p->qk_norm ? 1.f / sqrtf(s2 / (float)d + p->rms_eps) : 1.f;
      for (int i = lane; i < half; i += 64) {
        float a = x[i], b = x[i + half];
        if (p->qk_norm) {
          a = a * rs * G(gn)[i];
          b = b * rs * G(gn)[i + half];
        }
        const float cs = G(op->rope)[((size_t)pos * half + i) * 2], sn = G(op->rope)[((size_t)pos * half + i) * 2 + 1];
        x[i] = a * cs - b * sn;
        x[i + half] = b * cs + a * sn;
      }
    }
    __syncthreads();
    if (h % grp == 0 && c == 0)
      for (int e = tid(); e < 2 * d; e += kThreads) cstf(kvc + (size_t)pos * 2 * d + e, e < d ? kn[e] : vn[e - d]);
    // this frame's position is not in the cache yet (it is written in this phase): its own k and v
    if (t1 - 1 == pos)
      for (int i = tid(); i < 2 * d; i += kThreads) kvs[(pos - t0) * 2 * d + i] = i < d ? kn[i] : vn[i - d];
    __syncthreads();
    // scores, one wave per position
    for (int t = wave; t < n; t += kWaves) {
      float a = 0.f;
      for (int i = lane; i < d; i += 64) a = fmaf(qv[i], kvs[t * 2 * d + i], a);
      a = wave_sum(a) * scale;
      if (lane == 0) sc[t] = a;
    }
    __syncthreads();
    float mx = -INFINITY;
    for (int t = 0; t < n; ++t) mx = fmaxf(mx, sc[t]);
    __syncthreads();  // every thread has its maximum before the scores become weights
    for (int t = tid(); t < n; t += kThreads) sc[t] = expf(sc[t] - mx);
    __syncthreads();
    if (tid() < nog * d) {
      const int gi = tid() / d, i = tid() - gi * d;
      float o = 0.f, z = 0.f;
      for (int t = gi; t < n; t += nog) {
        const float w = sc[t];
        o = fmaf(w, kvs[t * 2 * d + d + i], o);
        z += w;
      }
      og[gi * d + i] = o;
      if (i == 0) zg[gi] = z;
    }
    __syncthreads();
    float* dst = op->apart + ((size_t)h * kAttnMaxChunks + c) * (d + 2);
    for (int i = tid(); i < d; i += kThreads) {
      float o = og[i];
      for (int gi = 1; gi < nog; ++gi) o += og[gi * d + i];
      cstf(dst + 2 + i, o);
      if (i == 0) {
        float z = zg[0];
        for (int gi = 1; gi < nog; ++gi) z += zg[gi];
        cstf(dst, mx);
        cstf(dst + 1, z);
      }
    }
    __syncthreads();
  }
}

// merge the chunk partials of query head h (workgroup h) into the O projection's input
__device__ void outer_attn_merge(const OParams* op, int pos, uint32_t* Aout, float* lds) {
  const KParams* p = op->k;
  const int d = p->d, np = pos + 1, ch = attn_chunk_len(np, d), nch = (np + ch - 1) / ch;
  float* w = lds + nch * (d + 2);  // [nch] chunk weights exp(m_c - max)
  float* xo = w + nch;             // [d] the merged output
  for (int h = blockIdx.x; h < p->nq; h += op->nwg) {
    // the head's chunk partials (max, sum, o[d]) into LDS, all loads in flight together
    lds_fill<true>(lds, op->apart + (size_t)h * kAttnMaxChunks * (d + 2), nch * (d + 2), nch * (d + 2), 0);
    __syncthreads();
    float mx = -INFINITY;
    for (int c = 0; c < nch; ++c) mx = fmaxf(mx, lds[c * (d + 2)]);
    for (int c = tid(); c < nch; c += kThreads) w[c] = expf(lds[c * (d + 2)] - mx);
    __syncthreads();
    float z = 0.f;
    for (int c = 0; c < nch; ++c) z += lds[c * (d + 2) + 1] * w[c];
    const float iz = 1.f / z;
    for (int i = tid(); i < d; i += kThreads) {
      float o = 0.f;
      for (int c = 0; c < nch; ++c) o += lds[c * (d + 2) + 2 + i] * w[c];
      xo[i] = o * iz;
    }
    __syncthreads();
    for (int q8 = tid(); q8 < d / 8; q8 += kThreads) {
      float x8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x8[e] = xo[8 * q8 + e];
      store_split(Aout + h * d + 8 * q8, x8);
    }
    __syncthreads();
  }
}

// residual + norm of the single row (workgroup 0); final: hidden out and the head input
__device__ void outer_resid(const OParams* op, BShared* sh, int KS, const float* gain, uint32_t* Aout,
                            float* hidden_out, float* xs) {
  if (blockIdx.x != 0) return;
  const KParams* p = op->k;
  const int H = p->H;
  float ss = 0.f;
  for (int e = tid(); e < H; e += kThreads) {
    const float v = cldf(op->x + e) + sum_parts<true>(op->part + e, (size_t)H, KS);
    cstf(op->x + e, v);
    xs[e] = v;
    ss = fmaf(v, v, ss);
  }
  ss = block_sum(sh, ss);
  const float rs = 1.f / sqrtf(ss / (float)H + p->rms_eps);
  for (int c = tid(); c < H / 8; c += kThreads) {
    float h8[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) h8[e] = xs[8 * c + e] * rs * G(gain)[8 * c + e];
    store_split(Aout + 8 * c, h8);
    if (hidden_out)
#pragma unroll
      for (int e = 0; e < 8; ++e) hidden_out[8 * c + e] = h8[e];
  }
}

// c_0: top-k over the logits of the codes the inner tables embed, fp64 softmax, inverse CDF
__device__ void outer_sample(const OParams* op, BShared* sh, const OCall& call, float* lds) {
  if (blockIdx.x != 0) return;
  const KParams* p = op->k;
  const int V = min(p->V, op->table_vocab);
  float* lg = lds;
  int* sidx = reinterpret_cast<int*>(lg + V);
  float* slog = reinterpret_cast<float*>(sidx + kMaxTopk);
  double* prob = reinterpret_cast<double*>(lg + ((V + 2 * kMaxTopk + 1) & ~1));  // 8-byte aligned, as above
  unsigned* hist = reinterpret_cast<unsigned*>(prob + kMaxTopk);
  lds_fill<true>(lg, op->logits, V, V, 0);
  __syncthreads();
  int ns = topk_buckets(&sh->tk, lg, V, op->topk, sidx, slog, hist);
  if (ns < 0) ns = topk_select(&sh->tk, lg, V, op->topk, sidx, slog);
  softmax_support(slog, ns, op->temperature, prob);
  __syncthreads();
  if (tid() < 64) {
    bool fin = false;
    for (int i = tid(); i < ns; i += 64) fin |= (slog[i] > -INFINITY && slog[i] < INFINITY);
    const bool any_fin = __any(fin);
    const int pos = inverse_cdf(prob, ns, (double)G(call.u_c0)[0]);
    if (tid() == 0) {
      if (!any_fin) raise_status(op, RVQSD_ENUMERIC);
      call.c0_out[0] = any_fin ? sidx[pos] : -1;
    }
  }
}

__global__ void __launch_bounds__(kThreads, 1) outer_kernel(const OParams* __restrict__ opp, OCall call) {
  __shared__ BShared shs;
  extern __shared__ __align__(16) float dyn[];
  const OParams* op = opp;
  const KParams* p = op->k;
  BShared* sh = &shs;
  uint32_t gen = 0;
  const int L = p->L, H = p->H;
  uint32_t* A0 = op->a;
  uint32_t* A1 = op->a + max(max(H, p->qdim), p->F);
  if (blockIdx.x == 0) outer_input(op, sh, call, A0, dyn);
  bool ok = grid_sync<OParams, false>(op, gen, sh);
  for (int l = 0; l < L && ok; ++l) {
    proj_partial<4, OParams, true>(op, bw(p, boff(p, l, p->o_wq)), p->nqkv, H, op->ks_qkv, A0, dyn);
    ok = grid_sync<OParams, false>(op, gen, sh);
    if (ok) outer_attn(op, sh, l, call.pos, dyn);
    ok = ok && grid_sync<OParams, false>(op, gen, sh);
    if (ok) outer_attn_merge(op, call.pos, A1, dyn);
    ok = ok && grid_sync<OParams, false>(op, gen, sh);
    if (ok) proj_partial<4, OParams, true>(op, bw(p, boff(p, l, p->o_wo)), H, p->qdim, op->ks_o, A1, dyn);
    ok = ok && grid_sync<OParams, false>(op, gen, sh);
    if (ok) outer_resid(op, sh, op->ks_o, bfw(p, boff(p, l, p->o_mlp_norm)), A0, nullptr, dyn);
    ok = ok && grid_sync<OParams, false>(op, gen, sh);
    if (ok) phase_gu<OParams, true>(op, l, A0, A1, dyn);
    ok = ok && grid_sync<OParams, false>(op, gen, sh);
    if (ok) proj_partial<4, OParams, true>(op, bw(p, boff(p, l, p->o_wd)), H, p->F, op->ks_down, A1, dyn);
    ok = ok && grid_sync<OParams, false>(op, gen, sh);
    if (ok) {
      if (l + 1 < L) outer_resid(op, sh, op->ks_down, bfw(p, boff(p, l + 1, p->o_attn_norm)), A0, nullptr, dyn);
      else outer_resid(op, sh, op->ks_down, bfw(p, p->o_final_norm), A0, call.hidden_out, dyn);
    }
    ok = ok && grid_sync<OParams, false>(op, gen, sh);
  }
  if (ok) {
    // head: 64-column units over the full hidden width, one row
    const bf16_t* W = bw(p, p->o_lmh1);
    const int V = p->V;
    for (int u = blockIdx.x; u < (V + 63) / 64; u += op->nwg) {
      const int n0 = u * 64;
      gemm_unit<4, kProjNTW, true>(
          [&](int nt, int m) -> const bf16_t* {
            const int f = n0 + 16 * nt + m;
            return f < V ? W + (size_t)f * H : nullptr;
          },
          0, H, A0, H, 1, [&](int i) { return i < 1 ? 0 : -1; }, dyn);
      for (int e = tid(); e < 4 * 64; e += kThreads) {
        const int nt = e >> 6, ln = e & 63;
        if ((ln & 15) == 0) {
          const float* sv = dyn + ((size_t)(nt * kBatchMTiles) << 8) + 4 * ln;
          for (int v = 0; v < 4; ++v) {
            const int f = n0 + 16 * nt + 4 * (ln >> 4) + v;
            if (f < V) cstf(op->logits + f, sv[v]);
          }
        }
      }
      __syncthreads();
    }
    ok = grid_sync<OParams, false>(op, gen, sh);
  }
  if (ok) outer_sample(op, sh, call, dyn);
  if (!ok && blockIdx.x == 0 && tid() == 0) call.c0_out[0] = -1;
}

// ------------------------------------------------------------ outer step without grid barriers
// The same step as outer_kernel, with every value one workgroup hands to another carried by a
// 64-bit word whose upper half is the launch number of the write: a reader polls the words
// until they carry this launch's number, so no grid barrier separates the phases. Every layer
// and kind of value has words of its own, so no word is written twice in one launch and a
// reader that falls behind still finds its value; the next launch on the stream starts after
// this one has ended, and a launch that failed leaves only words of older launches. With one
// row, every workgroup keeps the whole residual row in LDS and adds the O and down partial sums
// to it itself, in split order, so all copies are equal.

__device__ __forceinline__ void tstore(uint64_t* p, uint32_t tag, float v) {
  cst64(p, ((uint64_t)tag << 32) | __float_as_uint(v));
}

// n tagged words: sink(i, payload) once word addr(i) carries tag. Thread t takes words t, t + 512,
// ...; up to eight loads in flight each. False for every thread when a wait ran out (2 s) or
// another workgroup raised the status.
template <typename Addr, typename Sink>
__device__ bool opoll(const OParams* op, int n, uint32_t tag, Addr addr, Sink sink) {
  constexpr int B = 8;
  int bad = 0;
  for (int base = 0; base < n && !bad; base += B * kThreads) {
    uint32_t pend = 0;
#pragma unroll
    for (int b = 0; b < B; ++b)
      if (base + b * kThreads + tid() < n) pend |= 1u << b;
    uint64_t t0 = 0;
    int spins = 0;
    while (pend) {
      uint64_t v[B];
#pragma unroll
      for (int b = 0; b < B; ++b) v[b] = (pend >> b) & 1u ? cld64(addr(base + b * kThreads + tid())) : 0ull;
#pragma unroll
      for (int b = 0; b < B; ++b)
        if (((pend >> b) & 1u) && (uint32_t)(v[b] >> 32) == tag) {
          sink(base + b * kThreads + tid(), (uint32_t)v[b]);
          pend &= ~(1u << b);
        }
      if (!pend) break;
      if ((++spins & 31) == 0) {
        const uint64_t now = dclock();
        if (t0 == 0) {
          t0 = now;
        } else if (now - t0 > kTimeoutTicks) {
          raise_status(op, RVQSD_ETIMEOUT);
          bad = 1;
          break;
        }
        if (cld32(op->status) != 0) {
          bad = 1;
          break;
        }
      }
    }
  }
  return !__syncthreads_or(bad);
}

// Thread c < H / 8 holds gain elements 8c .. 8c + 7 (H <= 8 kThreads), loaded ahead of the
// row they scale
struct Gain8 {
  f32x4 g0, g1;
};
__device__ __forceinline__ Gain8 gain_fetch(const float* gain, int H) {
  Gain8 g = {(f32x4){0.f, 0.f, 0.f, 0.f}, (f32x4){0.f, 0.f, 0.f, 0.f}};
  if (tid() < H / 8) {
    g.g0 = G(reinterpret_cast<const f32x4*>(gain))[2 * tid()];
    g.g1 = G(reinterpret_cast<const f32x4*>(gain))[2 * tid() + 1];
  }
  return g;
}

// x (LDS, [H]) normalised with the gain, split into the LDS row a; hidden_out (workgroup 0)
// receives the normalised values. ss_own: this thread's sum of squares over its elements
// e = tid(), tid() + kThreads, ... when the caller has it (fold_parts)
__device__ void norm_split(const OParams* op, BShared* sh, const float* x, const Gain8& gn, uint32_t* a,
                           float* hidden_out, const float* ss_own = nullptr) {
  const KParams* p = op->k;
  const int H = p->H;
  float ss = 0.f;
  if (ss_own) ss = *ss_own;
  else
    for (int e = tid(); e < H; e += kThreads) ss = fmaf(x[e], x[e], ss);
  ss = block_sum(sh, ss);  // its barrier also orders the caller's writes of x before the reads below
  const float rs = 1.f / sqrtf(ss / (float)H + p->rms_eps);
  const int c = tid();
  if (c < H / 8) {
    float h8[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      h8[e] = x[8 * c + e] * rs * gn.g0[e];
      h8[4 + e] = x[8 * c + 4 + e] * rs * gn.g1[e];
    }
    W16 hi, lo;
    split8(h8, hi, lo);
    *reinterpret_cast<W16*>(a + 8 * c) = hi;
    *reinterpret_cast<W16*>(a + 8 * c + 4) = lo;
    if (hidden_out && blockIdx.x == 0)
#pragma unroll
      for (int e = 0; e < 8; ++e) hidden_out[8 * c + e] = h8[e];
  }
  __syncthreads();
}

// x += the ns partial sums P[k][H] (tagged), in split order. With ss, the thread's sum of
// squares of the new x for norm_split, which must follow (its barrier ends this phase)
__device__ bool fold_parts(const OParams* op, const uint64_t* P, int ns, uint32_t tag, float* x, float* tmp,
                           float* ss = nullptr) {
  const int H = op->k->H;
  const bool ok = opoll(op, ns * H, tag, [=](int i) { return P + i; }, [&](int i, uint32_t v) { tmp[i] = __uint_as_float(v); });
  if (!ok) return false;
  float sq = 0.f;
  for (int e = tid(); e < H; e += kThreads) {
    float s2 = tmp[e];
    for (int k = 1; k < ns; ++k) s2 += tmp[(size_t)k * H + e];
    const float v = x[e] + s2;
    x[e] = v;
    sq = fmaf(v, v, sq);
  }
  if (ss) *ss = sq;
  else __syncthreads();
  return true;
}

// n tagged words from T into the split LDS row a at words k0 .. k0 + n - 1 (n a multiple of 8)
__device__ bool fill_split(const OParams* op, const uint64_t* T, int k0, int n, uint32_t tag, uint32_t* a, float* tmp) {
  const bool ok = opoll(op, n, tag, [=](int i) { return T + k0 + i; }, [&](int i, uint32_t v) { tmp[i] = __uint_as_float(v); });
  if (!ok) return false;
  for (int c = tid(); c < n / 8; c += kThreads) {
    float x8[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) x8[e] = tmp[8 * c + e];
    W16 hi, lo;
    split8(x8, hi, lo);
    *reinterpret_cast<W16*>(a + k0 + 8 * c) = hi;
    *reinterpret_cast<W16*>(a + k0 + 8 * c + 4) = lo;
  }
  __syncthreads();
  return true;
}

// A unit whose weight fragments are loaded into registers before its input row is ready, so the
// load overlaps the wait: NT n-tiles of 16 rows, k in [k0, k0 + klen) split over the eight waves
// in 64-wide steps (at most NS per wave).
template <int NT, int NS>
struct WPre {
  W16 a0[NT][NS], a1[NT][NS];
};
template <int NT, int NS, typename WRow>
__device__ __forceinline__ void wfetch(WPre<NT, NS>& w, WRow wrow, int k0, int klen) {
  const int wave = __builtin_amdgcn_readfirstlane(tid() >> 6), lane = tid() & 63;
  const int q = lane >> 4, ml = lane & 15;
  const int kper = klen / kWaves, kb = k0 + wave * kper, nsteps = kper >> 6;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const bf16_t* wr = wrow(t, ml);
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      w.a0[t][s] = w.a1[t][s] = (W16)(0u);
      if (wr && s < nsteps) {
        w.a0[t][s] = *G(reinterpret_cast<const W16*>(wr + kb + 16 * q + 64 * s));
        w.a1[t][s] = *G(reinterpret_cast<const W16*>(wr + kb + 16 * q + 64 * s + 8));
      }
    }
  }
}
// the unit's NT x 16 outputs for the one row held split in LDS (a, words k0 .. k0 + klen - 1):
// out(f, s) with s[t] the output of n-tile t, row f; the wave partials are added in wave order
template <int NT, int NS, typename Out>
__device__ __forceinline__ void wdot(const WPre<NT, NS>& w, int k0, int klen, const uint32_t* a, float* red, Out out) {
  const int wave = __builtin_amdgcn_readfirstlane(tid() >> 6), lane = tid() & 63;
  const int q = lane >> 4, ml = lane & 15;
  const int kper = klen / kWaves, kb = k0 + wave * kper, nsteps = kper >> 6;
  f32x4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    if (s < nsteps) {
      W16 bh0 = (W16)(0u), bl0 = bh0, bh1 = bh0, bl1 = bh0;
      if (ml == 0) {  // activation column 0 is the row; the other 15 stay zero
        const uint32_t* ap = a + kb + 64 * s + 16 * q;
        bh0 = *reinterpret_cast<const W16*>(ap);
        bl0 = *reinterpret_cast<const W16*>(ap + 4);
        bh1 = *reinterpret_cast<const W16*>(ap + 8);
        bl1 = *reinterpret_cast<const W16*>(ap + 12);
      }
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const bf16x8 x0 = __builtin_bit_cast(bf16x8, w.a0[t][s]), x1 = __builtin_bit_cast(bf16x8, w.a1[t][s]);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x0, __builtin_bit_cast(bf16x8, bh0), acc[t], 0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x0, __builtin_bit_cast(bf16x8, bl0), acc[t], 0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x1, __builtin_bit_cast(bf16x8, bh1), acc[t], 0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x1, __builtin_bit_cast(bf16x8, bl1), acc[t], 0, 0, 0);
      }
    }
  }
  // output row 4 q + v of n-tile t sits in lane 16 q, element v
  if (ml == 0)
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) red[(wave * NT + t) * 16 + 4 * q + v] = acc[t][v];
  __syncthreads();
  if (tid() < 16) {
    float sum[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      sum[t] = red[t * 16 + tid()];
      for (int wv = 1; wv < kWaves; ++wv) sum[t] += red[(wv * NT + t) * 16 + tid()];
    }
    out(tid(), sum);
  }
  __syncthreads();
}

template <int NS>
__global__ void __launch_bounds__(kThreads, 1) outer_flow_kernel(const OParams* __restrict__ opp, OCall call) {
  __shared__ BShared shs;
  extern __shared__ __align__(16) float dyn[];
  const OParams* op = opp;
  const KParams* p = op->k;
  BShared* sh = &shs;
  const int L = p->L, H = p->H, d = p->d, N = p->nqkv, qd = p->qdim, F = p->F, nq = p->nq;
  float* red = dyn;                                                      // unit partial tiles
  uint32_t* arow = reinterpret_cast<uint32_t*>(dyn + kBatchRedFloats + kBatchMaxRows * 16);  // split input row
  float* xr = dyn + op->xoff;                                            // the residual row [H]
  float* tmp = dyn;  // poll staging (before a unit runs, or in phases without units)
  const int pos = call.pos, np = pos + 1, ch = attn_chunk_len(np, d), nch = (np + ch - 1) / ch;
  bool ok = true;
  // x_0 = t + E_0[c_0] + sum_j E_j[c_j] of the previous frame, built by every workgroup
  {
    __shared__ int pcodes[kMaxCodes + 1];
    __shared__ int pbad;
    const int nt = op->n_tables;
    if (tid() == 0) pbad = 0;
    __syncthreads();
    if (call.prev_codes && tid() <= nt) {
      const int c = G(call.prev_codes)[tid()];
      pcodes[tid()] = c;
      if (!(c >= 0 && c < (tid() == 0 ? min(p->V, op->table_vocab) : op->table_vocab))) pbad = 1;
    }
    __syncthreads();
    const bool codes_ok = call.prev_codes != nullptr && pbad == 0;
    if (call.prev_codes && !codes_ok && tid() == 0 && blockIdx.x == 0) raise_status(op, RVQSD_EINVAL);
    // thread c takes elements 8c .. 8c + 7: every table row's 16 bytes are requested together,
    // then added in table order
    for (int c8 = tid(); c8 < H / 8; c8 += kThreads) {
      const f32x4 ta = G(reinterpret_cast<const f32x4*>(call.t))[2 * c8];
      const f32x4 tb = G(reinterpret_cast<const f32x4*>(call.t))[2 * c8 + 1];
      float v[8] = {ta[0], ta[1], ta[2], ta[3], tb[0], tb[1], tb[2], tb[3]};
      if (codes_ok) {
        const bf16_t* e0 = bw(p, p->o_emb0);
        W16 tv[kMaxCodes + 1];
        tv[0] = *G(reinterpret_cast<const W16*>(e0 + (size_t)pcodes[0] * H + 8 * c8));
#pragma unroll
        for (int j = 1; j <= kMaxCodes; ++j)
          tv[j] = j <= nt ? *G(reinterpret_cast<const W16*>(op->tables + ((size_t)(j - 1) * op->table_vocab + pcodes[j]) * H +
                                                            8 * c8))
                          : (W16)(0u);
#pragma unroll
        for (int j = 0; j <= kMaxCodes; ++j)
          if (j <= nt)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const uint32_t w = tv[j][e >> 1];
              v[e] += __uint_as_float((e & 1) ? (w & 0xFFFF0000u) : (w << 16));
            }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) xr[8 * c8 + e] = v[e];
    }
    __syncthreads();
  }
  const int grp = nq / p->nkv, half = d / 2;
  const int nwg = op->nwg, me = blockIdx.x;
  const int nuq = (N + 15) / 16, cg = H / 16, nuo = cg * op->ks_o2, nud = cg * op->ks_d2;
  const int klo = qd / op->ks_o2, kld = F / op->ks_d2;
  WPre<1, NS> w1;  // QKV, O and down units
  WPre<2, NS> w2;  // gate/up units
  for (int l = 0; l < L && ok; ++l) {
    const size_t b = (size_t)l;  // this layer's exchange words
    // ---- QKV: the residual row after layer l - 1, normalised; 16 output columns per unit
    const bf16_t* Wq = bw(p, boff(p, l, p->o_wq));  // q, k, v rows are consecutive in the blob
    auto qrows = [=](int u) {
      return [=](int, int m) -> const bf16_t* { return u * 16 + m < N ? Wq + (size_t)(u * 16 + m) * H : nullptr; };
    };
    if (me < nuq) wfetch(w1, qrows(me), 0, H);
    const Gain8 gan = gain_fetch(bfw(p, boff(p, l, p->o_attn_norm)), H);
    float ss = 0.f;
    if (l > 0) ok = fold_parts(op, op->tdp + (b - 1) * kOutDSplit * H, op->ks_d2, call.epoch, xr, tmp, &ss);
    if (!ok) break;
    norm_split(op, sh, xr, gan, arow, nullptr, l > 0 ? &ss : nullptr);
    {
      const uint32_t tg = call.epoch;
      for (int u = me; u < nuq; u += nwg) {
        if (u != me) wfetch(w1, qrows(u), 0, H);
        wdot(w1, 0, H, arow, red, [&](int f, const float* v) { if (u * 16 + f < N) tstore(op->tq + b * N + u * 16 + f, tg, v[0]); });
      }
    }
    // the first O unit's weights, loaded during attention
    const bf16_t* Wo = bw(p, boff(p, l, p->o_wo));
    auto orows = [=](int u) {
      const int g = u % cg;
      return [=](int, int m) -> const bf16_t* { return Wo + (size_t)(g * 16 + m) * qd; };
    };
    if (me < nuo) wfetch(w1, orows(me), (me / cg) * klo, klo);
    // ---- attention over the key chunks: unit (query head h, chunk c)
    for (int u = blockIdx.x; u < nq * nch && ok; u += op->nwg) {
      const int h = u / nch, c = u - h * nch, g = h / grp;
      const int t0 = c * ch, t1 = min(np, t0 + ch), n = t1 - t0;
      const int nog = kThreads / d;
      float* qv = dyn;  // [d], then k, v of this position
      float* kn = qv + d;
      float* vn = kn + d;
      float* sc = vn + d;                 // [ch]
      float* og = sc + ch;                // [nog][d]
      float* zg = og + nog * d;           // [nog]
      float* kvs = dyn + ((3 * d + ch + nog * d + nog + 3) & ~3);  // [ch][2d]
      float* kvc = op->kv + (((size_t)l * p->nkv + g) * op->max_frames) * 2 * d;
      const int lane = tid() & 63, wave = tid() >> 6;
      // waves 0 and 1 normalise and rotate q and k: their gains and this position's rotary
      // factors are loaded before the wait (head_dim <= 256: at most two elements per lane)
      float gl[2] = {1.f, 1.f}, gh[2] = {1.f, 1.f}, rc[2] = {0.f, 0.f}, rsn[2] = {0.f, 0.f};
      if (wave < 2) {
        const float* gn = bfw(p, boff(p, l, wave == 0 ? p->o_qn : p->o_kn));
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int i = lane + 64 * j;
          if (i < half) {
            if (p->qk_norm) {
              gl[j] = G(gn)[i];
              gh[j] = G(gn)[i + half];
            }
            rc[j] = G(op->rope)[((size_t)pos * half + i) * 2];
            rsn[j] = G(op->rope)[((size_t)pos * half + i) * 2 + 1];
          }
        }
      }
      lds_fill4(kvs, kvc + (size_t)t0 * 2 * d, n * d / 2);
      ok = opoll(op, 3 * d, call.epoch,
                 [=](int e) {
                   const int part = e / d, i = e - part * d;
                   const int col = part == 0 ? h * d + i : qd + (part - 1) * p->kvdim + g * d + i;
                   return op->tq + b * N + col;
                 },
                 [&](int e, uint32_t v) { dyn[e] = __uint_as_float(v); });
      if (!ok) break;
      if (wave < 2) {
        float* x = wave == 0 ? qv : kn;
        float s2 = 0.f;
        for (int i = lane; i < d; i += 64) s2 = fmaf(x[i], x[i], s2);
        s2 = wave_sum(s2);
        const float rs = p->qk_norm ? 1.f / sqrtf(s2 / (float)d + p->rms_eps) : 1.f;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int i = lane + 64 * j;
          if (i < half) {
            float a = x[i], bb = x[i + half];
            if (p->qk_norm) {
              a = a * rs * gl[j];
              bb = bb * rs * gh[j];
            }
            x[i] = a * rc[j] - bb * rsn[j];
            x[i + half] = bb * rc[j] + a * rsn[j];
          }
        }
      }
      __syncthreads();
      if (h % grp == 0 && c == 0)
        for (int e = tid(); e < 2 * d; e += kThreads) cstf(kvc + (size_t)pos * 2 * d + e, e < d ? kn[e] : vn[e - d]);
      if (t1 - 1 == pos)
        for (int i = tid(); i < 2 * d; i += kThreads) kvs[(pos - t0) * 2 * d + i] = i < d ? kn[i] : vn[i - d];
      __syncthreads();
      // scores: eight lanes per position, each over d / 32 of the float4s of q and k; the
      // position rotates the segment order so that the groups of a wave read different banks
      const float scale = 1.f / sqrtf((float)d);
      const int nseg = d / 32, gsub = tid() & 7;
      for (int t = tid() >> 3; t < n; t += kThreads / 8) {
        const float* kr = kvs + (size_t)t * 2 * d;
        int sg = t % nseg;
        float a = 0.f;
        for (int s2 = 0; s2 < nseg; ++s2) {
          const int v4 = 4 * (gsub + 8 * sg);
          const f32x4 kk = *reinterpret_cast<const f32x4*>(kr + v4), qq = *reinterpret_cast<const f32x4*>(qv + v4);
          a = fmaf(qq[0], kk[0], a);
          a = fmaf(qq[1], kk[1], a);
          a = fmaf(qq[2], kk[2], a);
          a = fmaf(qq[3], kk[3], a);
          if (++sg == nseg) sg = 0;
        }
        a += __shfl_xor(a, 1, 64);
        a += __shfl_xor(a, 2, 64);
        a += __shfl_xor(a, 4, 64);
        if (gsub == 0) sc[t] = a * scale;
      }
      __syncthreads();
      // every wave takes the maximum itself
      float mx = -INFINITY;
      for (int t = lane; t < n; t += 64) mx = fmaxf(mx, sc[t]);
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
      __syncthreads();
      for (int t = tid(); t < n; t += kThreads) sc[t] = expf(sc[t] - mx);
      __syncthreads();
      if (tid() < nog * d) {
        const int gi = tid() / d, i = tid() - gi * d;
        float o = 0.f, z = 0.f;
        for (int t = gi; t < n; t += nog) {
          const float w = sc[t];
          o = fmaf(w, kvs[t * 2 * d + d + i], o);
          z += w;
        }
        og[gi * d + i] = o;
        if (i == 0) zg[gi] = z;
      }
      __syncthreads();
      uint64_t* dst = op->tch + ((b * nq + h) * kAttnMaxChunks + c) * (d + 2);
      const uint32_t tg = call.epoch;
      for (int i = tid(); i < d; i += kThreads) {
        float o = og[i];
        for (int gi = 1; gi < nog; ++gi) o += og[gi * d + i];
        tstore(dst + 2 + i, tg, o);
        if (i == 0) {
          float z = zg[0];
          for (int gi = 1; gi < nog; ++gi) z += zg[gi];
          tstore(dst, tg, mx);
          tstore(dst + 1, tg, z);
        }
      }
      __syncthreads();
    }
    if (!ok) break;
    // ---- merge the chunk partials of head h (workgroup h)
    for (int h = blockIdx.x; h < nq && ok; h += op->nwg) {
      const uint64_t* src = op->tch + (b * nq + h) * kAttnMaxChunks * (d + 2);
      ok = opoll(op, nch * (d + 2), call.epoch, [=](int i) { return src + i; },
                 [&](int i, uint32_t v) { dyn[i] = __uint_as_float(v); });
      if (!ok) break;
      float* w = dyn + nch * (d + 2);
      const int lane = tid() & 63;
      float mx = -INFINITY;  // every wave takes the maximum and the normaliser itself
      for (int c = lane; c < nch; c += 64) mx = fmaxf(mx, dyn[c * (d + 2)]);
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
      for (int c = tid(); c < nch; c += kThreads) w[c] = expf(dyn[c * (d + 2)] - mx);
      __syncthreads();
      float z = 0.f;
      for (int c = lane; c < nch; c += 64) z += dyn[c * (d + 2) + 1] * w[c];
      z = wave_sum(z);
      const float iz = 1.f / z;
      const uint32_t tg = call.epoch;
      for (int i = tid(); i < d; i += kThreads) {
        float o = 0.f;
        for (int c = 0; c < nch; ++c) o += dyn[c * (d + 2) + 2 + i] * w[c];
        tstore(op->tat + b * qd + h * d + i, tg, o * iz);
      }
      __syncthreads();
    }
    if (!ok) break;
    // ---- O: unit (16 columns, k split ks): partial sums
    {
      const uint32_t tg = call.epoch;
      for (int u = me; u < nuo && ok; u += nwg) {
        const int g = u % cg, ks = u / cg;
        if (u != me) wfetch(w1, orows(u), ks * klo, klo);
        ok = fill_split(op, op->tat + b * qd, ks * klo, klo, call.epoch, arow, tmp);
        if (!ok) break;
        wdot(w1, ks * klo, klo, arow, red, [&](int f, const float* v) { tstore(op->top + (b * kOutOSplit + ks) * H + g * 16 + f, tg, v[0]); });
      }
    }
    if (!ok) break;
    // ---- gate/up: x += O partial sums; 16 features per unit (n-tile 0 gate, 1 up)
    const bf16_t* wg = bw(p, boff(p, l, p->o_wg));
    const bf16_t* wu = bw(p, boff(p, l, p->o_wu));
    auto gurows = [=](int u) {
      return [=](int nt, int m) -> const bf16_t* { return (nt ? wu : wg) + (size_t)(u * 16 + m) * H; };
    };
    if (me < F / 16) wfetch(w2, gurows(me), 0, H);
    const Gain8 gmn = gain_fetch(bfw(p, boff(p, l, p->o_mlp_norm)), H);
    ok = fold_parts(op, op->top + b * kOutOSplit * H, op->ks_o2, call.epoch, xr, tmp, me < F / 16 ? &ss : nullptr);
    if (!ok) break;
    if (me < F / 16) {
      norm_split(op, sh, xr, gmn, arow, nullptr, &ss);
      const uint32_t tg = call.epoch;
      for (int u = me; u < F / 16; u += nwg) {
        if (u != me) wfetch(w2, gurows(u), 0, H);
        wdot(w2, 0, H, arow, red, [&](int f, const float* v) {
          tstore(op->tact + b * F + u * 16 + f, tg, v[0] / (1.f + expf(-v[0])) * v[1]);
        });
      }
    }
    // ---- down: unit (16 columns, k split ks): partial sums
    {
      const bf16_t* Wd = bw(p, boff(p, l, p->o_wd));
      auto drows = [=](int u) {
        const int g = u % cg;
        return [=](int, int m) -> const bf16_t* { return Wd + (size_t)(g * 16 + m) * F; };
      };
      const uint32_t tg = call.epoch;
      for (int u = me; u < nud && ok; u += nwg) {
        const int g = u % cg, ks = u / cg;
        wfetch(w1, drows(u), ks * kld, kld);
        ok = fill_split(op, op->tact + b * F, ks * kld, kld, call.epoch, arow, tmp);
        if (!ok) break;
        wdot(w1, ks * kld, kld, arow, red, [&](int f, const float* v) { tstore(op->tdp + (b * kOutDSplit + ks) * H + g * 16 + f, tg, v[0]); });
      }
    }
  }
  // ---- head: x += the last down partial sums, final norm (hidden_out), logits
  const int Vh = p->V;
  const int nuh = (Vh + 15) / 16;
  if (ok && (me < nuh || me == 0)) {
    const bf16_t* Wh = bw(p, p->o_lmh1);
    auto hrows = [=](int u) {
      return [=](int, int m) -> const bf16_t* { return u * 16 + m < Vh ? Wh + (size_t)(u * 16 + m) * H : nullptr; };
    };
    if (me < nuh) wfetch(w1, hrows(me), 0, H);
    const Gain8 gfn = gain_fetch(bfw(p, p->o_final_norm), H);
    float ss = 0.f;
    ok = fold_parts(op, op->tdp + (size_t)(L - 1) * kOutDSplit * H, op->ks_d2, call.epoch, xr, tmp, &ss);
    if (ok) {
      norm_split(op, sh, xr, gfn, arow, call.hidden_out, &ss);
      const uint32_t tg = call.epoch;
      for (int u = me; u < nuh; u += nwg) {
        if (u != me) wfetch(w1, hrows(u), 0, H);
        wdot(w1, 0, H, arow, red, [&](int f, const float* v) { if (u * 16 + f < Vh) tstore(op->tlog + u * 16 + f, tg, v[0]); });
      }
    }
  }
  // ---- c_0: top-k over the logits of the codes the inner tables embed (workgroup 0)
  if (ok && blockIdx.x == 0) {
    const int V = min(Vh, op->table_vocab);
    float* lg = dyn;
    ok = opoll(op, V, call.epoch, [=](int i) { return op->tlog + i; }, [&](int i, uint32_t v) { lg[i] = __uint_as_float(v); });
    if (ok) {
      int* sidx = reinterpret_cast<int*>(lg + V);
      float* slog = reinterpret_cast<float*>(sidx + kMaxTopk);
      double* prob = reinterpret_cast<double*>(lg + ((V + 2 * kMaxTopk + 1) & ~1));
      unsigned* hist = reinterpret_cast<unsigned*>(prob + kMaxTopk);
      int ns = topk_buckets(&sh->tk, lg, V, op->topk, sidx, slog, hist);
      if (ns < 0) ns = topk_select(&sh->tk, lg, V, op->topk, sidx, slog);
      softmax_support(slog, ns, op->temperature, prob);
      __syncthreads();
      if (tid() < 64) {
        bool fin = false;
        for (int i = tid(); i < ns; i += 64) fin |= (slog[i] > -INFINITY && slog[i] < INFINITY);
        const bool any_fin = __any(fin);
        const int cp = inverse_cdf(prob, ns, (double)G(call.u_c0)[0]);
        if (tid() == 0) {
          if (!any_fin) raise_status(op, RVQSD_ENUMERIC);
          call.c0_out[0] = any_fin ? sidx[cp] : -1;
        }
      }
    }
  }
  if (!ok && blockIdx.x == 0 && tid() == 0) call.c0_out[0] = -1;
}

}  // namespace

// ------------------------------------------------------------------- host

// The tree and chain forms are separate instantiations: the chain kernel carries no tree code.
int launch_batch(const BParams* bp, const BCall& call, int nwg, void* stream, size_t lds_bytes, bool tree,
                 char* err, size_t errlen) {
  const void* fn = tree ? reinterpret_cast<const void*>(&batch_kernel<true>)
                        : reinterpret_cast<const void*>(&batch_kernel<false>);
  static size_t attr_bytes[2] = {0, 0};
  if (lds_bytes > attr_bytes[tree]) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
    if (e != hipSuccess) {
      snprintf(err, errlen, "hipFuncSetAttribute(%zu bytes LDS): %s", lds_bytes, hipGetErrorString(e));
      return RVQSD_EHIP;
    }
    attr_bytes[tree] = lds_bytes;
  }
  const BParams* bpp = bp;
  BCall c = call;
  void* args[] = {&bpp, &c};
  hipError_t e = hipLaunchCooperativeKernel(fn, dim3(nwg), dim3(kThreads), args, (unsigned)lds_bytes,
                                            reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) {
    snprintf(err, errlen, "hipLaunchCooperativeKernel: %s", hipGetErrorString(e));
    return RVQSD_EHIP;
  }
  return RVQSD_OK;
}

}  // namespace rvqsd

namespace rvqsd {

int launch_outer(const OParams* op, const OCall& call, int nwg, void* stream, size_t lds_bytes, int flow_steps, char* err,
                 size_t errlen) {
  // flow_steps 0: the step with grid barriers; else the one without, whose units hold their
  // weights in registers, flow_steps (<= kFlowSteps) 64-wide k steps per wave
  if (flow_steps < 0 || flow_steps > kFlowSteps) {
    snprintf(err, errlen, "outer step: %d k steps per wave (at most %d)", flow_steps, kFlowSteps);
    return RVQSD_EINVAL;
  }
  const bool flow = flow_steps > 0;
  const void* fn = flow ? reinterpret_cast<const void*>(&outer_flow_kernel<kFlowSteps>)
                        : reinterpret_cast<const void*>(&outer_kernel);
  const int slot = flow ? 1 : 0;
  static size_t attr_bytes[2] = {0, 0};
  if (lds_bytes > attr_bytes[slot]) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
    if (e != hipSuccess) {
      snprintf(err, errlen, "hipFuncSetAttribute(%zu bytes LDS): %s", lds_bytes, hipGetErrorString(e));
      return RVQSD_EHIP;
    }
    attr_bytes[slot] = lds_bytes;
  }
  const OParams* opa = op;
  OCall c = call;
  void* args[] = {&opa, &c};
  hipError_t e = hipLaunchCooperativeKernel(fn, dim3(nwg), dim3(kThreads), args, (unsigned)lds_bytes,
                                            reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) {
    snprintf(err, errlen, "hipLaunchCooperativeKernel: %s", hipGetErrorString(e));
    return RVQSD_EHIP;
  }
  return RVQSD_OK;
}

}  // namespace rvqsd
