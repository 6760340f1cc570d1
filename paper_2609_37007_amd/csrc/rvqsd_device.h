// rvqsd_device.h -- device helpers shared by the frame kernel and the batched kernel:
// global-address casts, tagged exchange words, wave reductions and scans on DPP,
// and the top-k / softmax / inverse-CDF steps of the sampling phase.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rvqsd_internal.h"

namespace rvqsd {

typedef uint16_t bf16_t;

constexpr uint64_t kTimeoutTicks = 200ull * 1000 * 1000;  // 2 s of the 100 MHz device clock

// The thread index behind an empty asm: values derived from it cannot be
// hoisted out of the pass loop, which keeps them from living across phases.
__device__ __forceinline__ int tid() {
  int t = (int)threadIdx.x;
  asm volatile("" : "+v"(t));
  return t;
}
// ------------------------------------------------------------------ helpers

// Pointers taken from the parameter block are generic; every device-memory
// access goes through these casts so that it compiles to a global (not flat)
// instruction.
#define RVQSD_GLOBAL __attribute__((address_space(1)))
template <typename T>
__device__ __forceinline__ RVQSD_GLOBAL T* G(T* q) {
  return (RVQSD_GLOBAL T*)q;
}
template <typename T>
__device__ __forceinline__ const RVQSD_GLOBAL T* G(const T* q) {
  return (const RVQSD_GLOBAL T*)q;
}

__device__ __forceinline__ uint64_t xload(const uint64_t* p) {
  return __hip_atomic_load(G(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void xstore(uint64_t* p, uint32_t tag, uint32_t payload) {
  __hip_atomic_store(G(p), ((uint64_t)tag << 32) | payload, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void xstoref(uint64_t* p, uint32_t tag, float v) { xstore(p, tag, __float_as_uint(v)); }
// activation word: fp32 with the lowest mantissa bit replaced by the epoch parity
__device__ __forceinline__ void pstore(uint32_t* p, float v, uint32_t par) {
  __hip_atomic_store(G(p), (__float_as_uint(v) & ~1u) | par, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t pload2(const uint32_t* p) {
  return __hip_atomic_load(G(reinterpret_cast<const uint64_t*>(p)), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Workgroup barrier for LDS traffic only: global loads stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}
__device__ __forceinline__ uint64_t dclock() { return __builtin_amdgcn_s_memrealtime(); }

// Sum over the 16 lanes of a DPP row (every lane of the row gets the sum):
// xor 1, xor 2 inside quads, then half-row mirror and row mirror.
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp<0x141>(v);  // row_half_mirror
  v += dpp<0x140>(v);  // row_mirror
  return v;
}
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_rows(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROWS, 0xF, false));
}
// Sum over the 64 lanes; the total is valid in lane 63 only.
__device__ __forceinline__ float wave_sum63(float v) {
  v = row16_sum(v);
  v += dpp_rows<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
  v += dpp_rows<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
  return v;
}
__device__ __forceinline__ float lane63(float v) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63)); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ double wave_sumd(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ double wave_maxd(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
  return v;
}
// Inclusive prefix sum over the 64 lanes with DPP: shifts 1, 2, 4, 8 inside each row
// of 16 lanes, then the last lane of row 0 (2) is added to rows 1, 3 (2, 3).
template <int CTRL, int ROWS>
__device__ __forceinline__ int dppi(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, ROWS, 0xF, false);
}
__device__ __forceinline__ int wave_scan_incl_dpp(int v) {
  v += dppi<0x111, 0xF>(v);  // row_shr:1
  v += dppi<0x112, 0xF>(v);  // row_shr:2
  v += dppi<0x114, 0xF>(v);  // row_shr:4
  v += dppi<0x118, 0xF>(v);  // row_shr:8
  v += dppi<0x142, 0xA>(v);  // row_bcast:15
  v += dppi<0x143, 0xC>(v);  // row_bcast:31
  return v;
}
template <int CTRL, int ROWS>
__device__ __forceinline__ double dppd(double v) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)u, CTRL, ROWS, 0xF, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(u >> 32), CTRL, ROWS, 0xF, false);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
__device__ __forceinline__ double wave_scan_incl_dppd(double v) {
  v += dppd<0x111, 0xF>(v);
  v += dppd<0x112, 0xF>(v);
  v += dppd<0x114, 0xF>(v);
  v += dppd<0x118, 0xF>(v);
  v += dppd<0x142, 0xA>(v);
  v += dppd<0x143, 0xC>(v);
  return v;
}
__device__ __forceinline__ double lane_vald(double v, int l) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
// sum / max over the 64 lanes (every lane gets the result): rows of 16 with DPP, then the 4 row totals
__device__ __forceinline__ double wave_sumd_dpp(double v) {
  v += dppd<0xB1, 0xF>(v);   // quad_perm [1,0,3,2]
  v += dppd<0x4E, 0xF>(v);   // quad_perm [2,3,0,1]
  v += dppd<0x141, 0xF>(v);  // row_half_mirror
  v += dppd<0x140, 0xF>(v);  // row_mirror
  return (lane_vald(v, 15) + lane_vald(v, 31)) + (lane_vald(v, 47) + lane_vald(v, 63));
}
__device__ __forceinline__ double wave_maxd_dpp(double v) {
  v = fmax(v, dppd<0xB1, 0xF>(v));
  v = fmax(v, dppd<0x4E, 0xF>(v));
  v = fmax(v, dppd<0x141, 0xF>(v));
  v = fmax(v, dppd<0x140, 0xF>(v));
  return fmax(fmax(lane_vald(v, 15), lane_vald(v, 31)), fmax(lane_vald(v, 47), lane_vald(v, 63)));
}

// inclusive prefix sum over the 64 lanes
__device__ __forceinline__ int wave_scan_incl(int v) {
  const int lane = tid() & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int t = __shfl_up(v, o, 64);
    if (lane >= o) v += t;
  }
  return v;
}
__device__ __forceinline__ double wave_scan_incld(double v) {
  const int lane = tid() & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    double t = __shfl_up(v, o, 64);
    if (lane >= o) v += t;
  }
  return v;
}

// 16 bytes of weights (a builtin vector type, so address-space qualified loads copy it)
typedef uint32_t W16 __attribute__((ext_vector_type(4)));

// Four parity words through one device-coherent 16-byte vector store (p 16-byte aligned): each
// word's lowest mantissa bit carries the parity; a reader checks every word on its own.
__device__ __forceinline__ void pstore4(uint32_t* p, float a, float b, float c, float d, uint32_t par) {
  W16 w;
  w[0] = (__float_as_uint(a) & ~1u) | par;
  w[1] = (__float_as_uint(b) & ~1u) | par;
  w[2] = (__float_as_uint(c) & ~1u) | par;
  w[3] = (__float_as_uint(d) & ~1u) | par;
  asm volatile("global_store_dwordx4 %0, %1, off sc1" ::"v"(p), "v"(w) : "memory");
}
// Four activation words through one device-coherent 16-byte load. The load is
// issued here and completes at vm_wait, which names the result as an operand so
// that no use of it is scheduled before the wait; several loads issued back to
// back are in flight together. Each 32-bit word is written atomically by its
// producer, so every word's parity bit is checked on its own.
__device__ __forceinline__ W16 pload4(const uint32_t* p) {
  W16 r;
  asm volatile("global_load_dwordx4 %0, %1, off sc1" : "=v"(r) : "v"(p) : "memory");
  return r;
}
__device__ __forceinline__ void vm_wait(W16& r) { asm volatile("s_waitcnt vmcnt(0)" : "+v"(r)::"memory"); }
// The same device-coherent 16-byte load as a raw buffer load with cache policy
// sc1 (resource of the given base, 32-bit data format, no stride or range limit).
// The compiler tracks it like any load and waits for it where the result is used,
// so it needs no vm_wait and is safe where register pressure makes the compiler
// copy registers between an inline-assembly load and its wait. Not for polling:
// a loop that re-reads one address must also clobber memory between the reads.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t coh_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, 0x7fffffff, 0x00020000);
}
__device__ __forceinline__ W16 bload4(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 16);
}

// Sum over the 32 lanes of each half of the wave (every lane gets its half's sum).
__device__ __forceinline__ float half_sum(float v) {
  v = row16_sum(v);
  v += dpp_rows<0x142, 0xA>(v);  // rows 1 and 3 += last lane of rows 0 and 2
  const float a = lane63(v) , b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 31));
  return (tid() & 32) ? a : b;
}
// max over the 16 lanes of each DPP row, in every lane of the row
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp<0xB1>(v));
  v = fmaxf(v, dpp<0x4E>(v));
  v = fmaxf(v, dpp<0x141>(v));
  v = fmaxf(v, dpp<0x140>(v));
  return v;
}
__device__ __forceinline__ float lane_val(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

// MFMA operand and accumulator types (v_mfma_f32_16x16x32_bf16)
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// fp32 -> bf16 bits, round to nearest even
__device__ __forceinline__ uint32_t bf16_bits_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}
// 8 floats -> hi (8 bf16) and lo (8 bf16, the rounded remainder)
__device__ __forceinline__ void split8(const float (&x)[8], W16& hi, W16& lo) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t a = bf16_bits_rne(x[2 * j]), b = bf16_bits_rne(x[2 * j + 1]);
    const uint32_t ra = bf16_bits_rne(x[2 * j] - __uint_as_float(a << 16));
    const uint32_t rb = bf16_bits_rne(x[2 * j + 1] - __uint_as_float(b << 16));
    hi[j] = a | (b << 16);
    lo[j] = ra | (rb << 16);
  }
}

// LDS scratch of the workgroup-wide top-k selection
struct TopkShared {
  unsigned hist[256];
  int iscan[kWaves];
  int sel_digit, sel_kk;
  float wmx[kWaves], wmn[kWaves];
  int wbad[kWaves];
  int sel_b, c_above, c_b, n_cand;
  int cand_idx[kTopkCand];
  float cand_val[kTopkCand];
};

// --------------------------------------------------------------- sampling
// order-preserving key of a float; NaN lowest
__device__ __forceinline__ uint32_t fkey(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// exclusive prefix over the workgroup in thread order; returns total via *total
__device__ __forceinline__ int block_excl_scan(TopkShared* sh, int v, int* total) {
  const int lane = tid() & 63, wave = tid() >> 6;
  int inc = wave_scan_incl_dpp(v);
  if (lane == 63) sh->iscan[wave] = inc;
  lds_barrier();
  int off = 0, tot = 0;
  for (int w = 0; w < kWaves; ++w) {
    if (w < wave) off += sh->iscan[w];
    tot += sh->iscan[w];
  }
  lds_barrier();
  *total = tot;
  return off + inc - v;
}

// Top-k of lg[V] (ties -> lower index), support in ascending token order:
// sidx[n], slog[n]. Returns n (<= topk).
__device__ __forceinline__ int topk_select(TopkShared* sh, const float* lg, int V, int topk, int* sidx, float* slog) {
  const int ept = (V + kThreads - 1) / kThreads;
  const int i0 = tid() * ept;
  const int kk0 = min(topk, V);
  uint32_t prefix = 0, pmask = 0;
  int kk = kk0;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = tid(); i < 256; i += kThreads) sh->hist[i] = 0;
    __syncthreads();
    for (int e = 0; e < ept; ++e) {
      int i = i0 + e;
      if (i < V) {
        uint32_t k = fkey(lg[i]);
        if ((k & pmask) == prefix) atomicAdd(&sh->hist[(k >> shift) & 255u], 1u);
      }
    }
    __syncthreads();
    if (tid() < 64) {
      const int lane = tid();
      int b[4], loc = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) { b[q] = (int)sh->hist[4 * lane + q]; loc += b[q]; }
      // number of elements in bins of higher lanes
      int incl_from_top = loc;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        int t = __shfl_down(incl_from_top, o, 64);
        if (lane + o < 64) incl_from_top += t;
      }
      int above = incl_from_top - loc;
#pragma unroll
      for (int q = 3; q >= 0; --q) {
        if (above < kk && kk <= above + b[q]) {
          sh->sel_digit = 4 * lane + q;
          sh->sel_kk = kk - above;
        }
        above += b[q];
      }
    }
    __syncthreads();
    prefix |= (uint32_t)sh->sel_digit << shift;
    pmask |= 255u << shift;
    kk = sh->sel_kk;
    __syncthreads();
  }
  // prefix = key of the kk0-th largest; take every key above it and the kk lowest-index equal keys
  int n_eq = 0;
  for (int e = 0; e < ept; ++e) {
    int i = i0 + e;
    if (i < V && fkey(lg[i]) == prefix) ++n_eq;
  }
  int tot;
  int eq_before = block_excl_scan(sh, n_eq, &tot);
  int n_sel = 0;
  unsigned selmask = 0;
  for (int e = 0; e < ept; ++e) {
    int i = i0 + e;
    if (i >= V) break;
    uint32_t k = fkey(lg[i]);
    bool s = k > prefix;
    if (k == prefix) {
      s = eq_before < kk;
      ++eq_before;
    }
    if (s) { selmask |= 1u << e; ++n_sel; }
  }
  int pos = block_excl_scan(sh, n_sel, &tot);
  for (int e = 0; e < ept; ++e) {
    if (selmask & (1u << e)) {
      sidx[pos] = i0 + e;
      slog[pos] = lg[i0 + e];
      ++pos;
    }
  }
  __syncthreads();
  return tot;
}

__device__ __forceinline__ float row16_min(float v) {
  v = fminf(v, dpp<0xB1>(v));
  v = fminf(v, dpp<0x4E>(v));
  v = fminf(v, dpp<0x141>(v));
  v = fminf(v, dpp<0x140>(v));
  return v;
}

// Top-k of lg[V] (ties -> lower index) through value buckets, support in ascending
// token order: sidx[n], slog[n]. The values are binned by b(v) = floor((max - v) *
// B / (max - min)), which never increases with v, so every value in a bucket
// below the one holding the k-th largest is strictly larger than every value in
// or above it; only that boundary bucket is ranked element by element (value,
// then index; +0 and -0 tie as in a plain comparison). Returns -1 (and leaves the
// outputs alone) when the row needs the general path: a value that is not
// finite, all values equal, or more than kTopkCand values in the boundary bucket.
static __device__ int topk_buckets(TopkShared* sh, const float* lg, int V, int topk, int* sidx, float* slog,
                            unsigned* hist) {
  const int ept = (V + kThreads - 1) / kThreads;
  const int i0 = tid() * ept;
  const int kk0 = min(topk, V);
  const int lane = tid() & 63, wave = tid() >> 6;
  for (int i = tid(); i < kTopkBuckets; i += kThreads) hist[i] = 0u;
  float mx = -INFINITY, mn = INFINITY;
  bool bad = false;
  for (int e = 0; e < ept; ++e) {
    const int i = i0 + e;
    if (i < V) {
      const float v = lg[i];
      bad |= !(fabsf(v) <= 3.402823466e38f);
      mx = fmaxf(mx, v);
      mn = fminf(mn, v);
    }
  }
  mx = row16_max(mx);
  mn = row16_min(mn);
  mx = fmaxf(fmaxf(lane_val(mx, 15), lane_val(mx, 31)), fmaxf(lane_val(mx, 47), lane_val(mx, 63)));
  mn = fminf(fminf(lane_val(mn, 15), lane_val(mn, 31)), fminf(lane_val(mn, 47), lane_val(mn, 63)));
  const bool wbad = __any(bad);
  if (lane == 0) {
    sh->wmx[wave] = mx;
    sh->wmn[wave] = mn;
    sh->wbad[wave] = wbad ? 1 : 0;
  }
  lds_barrier();
  int anybad = 0;
  for (int w = 0; w < kWaves; ++w) {
    mx = fmaxf(mx, sh->wmx[w]);
    mn = fminf(mn, sh->wmn[w]);
    anybad |= sh->wbad[w];
  }
  if (anybad || !(mx > mn)) return -1;
  const float scale = (float)kTopkBuckets / (mx - mn);
  auto bucket = [&](float v) -> int {
    const int b = (int)((mx - v) * scale);
    return b < kTopkBuckets - 1 ? b : kTopkBuckets - 1;
  };
  for (int e = 0; e < ept; ++e) {
    const int i = i0 + e;
    if (i < V) atomicAdd(&hist[bucket(lg[i])], 1u);
  }
  lds_barrier();
  if (wave == 0) {
    constexpr int BPL = kTopkBuckets / 64;  // buckets per lane
    int loc = 0;
#pragma unroll
    for (int q = 0; q < BPL; ++q) loc += (int)hist[BPL * lane + q];
    const int incl = wave_scan_incl_dpp(loc);
    const unsigned long long hit = __ballot(incl >= kk0);
    const int L = __ffsll((long long)hit) - 1;  // the total is V >= kk0, so some lane hits
    if (lane == L) {
      int cum = incl - loc;
      for (int q = 0; q < BPL; ++q) {
        const int h = (int)hist[BPL * lane + q];
        if (cum + h >= kk0) {
          sh->sel_b = BPL * lane + q;
          sh->c_above = cum;
          sh->c_b = h;
          break;
        }
        cum += h;
      }
      sh->n_cand = 0;
    }
  }
  lds_barrier();
  const int B = sh->sel_b, c_above = sh->c_above, c_b = sh->c_b;
  if (c_b > kTopkCand) return -1;
  for (int e = 0; e < ept; ++e) {
    const int i = i0 + e;
    if (i < V && bucket(lg[i]) == B) {
      const int k = atomicAdd(&sh->n_cand, 1);
      sh->cand_idx[k] = i;
      sh->cand_val[k] = lg[i];
    }
  }
  lds_barrier();
  const int need = kk0 - c_above;
  int n_sel = 0;
  unsigned selmask = 0;
  for (int e = 0; e < ept; ++e) {
    const int i = i0 + e;
    if (i >= V) break;
    const float v = lg[i];
    const int b = bucket(v);
    bool sel = b < B;
    if (b == B) {
      int rank = 0;
      for (int j = 0; j < c_b; ++j) {
        const float vj = sh->cand_val[j];
        rank += (vj > v || (vj == v && sh->cand_idx[j] < i)) ? 1 : 0;
      }
      sel = rank < need;
    }
    if (sel) {
      selmask |= 1u << e;
      ++n_sel;
    }
  }
  int tot;
  int pos = block_excl_scan(sh, n_sel, &tot);
  for (int e = 0; e < ept; ++e) {
    if (selmask & (1u << e)) {
      sidx[pos] = i0 + e;
      slog[pos] = lg[i0 + e];
      ++pos;
    }
  }
  lds_barrier();
  return tot;
}

// wave 0: probabilities of the top-k support, p = exp((l - max)/T) / Z in fp64
__device__ __forceinline__ void softmax_support(const float* slog, int n, double T, double* prob) {
  if (tid() >= 64) return;
  const int lane = tid();
  double mx = -INFINITY;
  for (int i = lane; i < n; i += 64) mx = fmax(mx, (double)slog[i]);
  mx = wave_maxd_dpp(mx);
  double z = 0.0;
  for (int i = lane; i < n; i += 64) {
    double w = exp(((double)slog[i] - mx) / T);
    prob[i] = w;
    z += w;
  }
  z = wave_sumd_dpp(z);
  for (int i = lane; i < n; i += 64) prob[i] = prob[i] / z;
}

// wave 0: inverse CDF of weights w[0..n) (ascending token order) at u; returns position
__device__ __forceinline__ int inverse_cdf(const double* w, int n, double u) {
  const int lane = tid();
  const int per = (n + 63) / 64;
  const int b = lane * per;
  double loc = 0.0;
  for (int q = 0; q < per; ++q)
    if (b + q < n) loc += w[b + q];
  double incl = wave_scan_incl_dppd(loc);
  double z = lane_vald(incl, 63);
  double thr = u * z;
  double cum = incl - loc;
  int found = -1;
  for (int q = 0; q < per; ++q) {
    if (b + q < n) {
      cum += w[b + q];
      if (found < 0 && cum > thr) found = b + q;
    }
  }
  unsigned long long bal = __ballot(found >= 0);
  if (bal) {
    int src = __ffsll((long long)bal) - 1;
    return __shfl(found, src, 64);
  }
  int last = -1;
  for (int q = 0; q < per; ++q)
    if (b + q < n && w[b + q] > 0.0) last = b + q;
  for (int o = 32; o > 0; o >>= 1) last = max(last, __shfl_xor(last, o, 64));
  return last < 0 ? n - 1 : last;
}

}  // namespace rvqsd
