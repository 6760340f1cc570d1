// rvqsd_noalloc.hip -- the frame decode for callers that cannot allocate memory.
//
// rvqsd_decode_frame_noalloc runs the same persistent frame kernel as
// rvqsd_decode_frame_async, but the frame's device buffers (exchange words, KV
// cache, parameter block; the layout of FrameLayout) live in `scratch`, a
// fixed array of this library on every GPU it runs on, instead of a stream's
// allocation. Each call first clears that region on the caller's stream with a
// small kernel (no memset node, so the two launches can be captured into a
// graph) and writes the parameter block, so every call starts from the state of
// a fresh stream and gives the codes a fresh stream gives.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstring>
#include <mutex>

#include "../../include/rvqsd.h"
#include "rvqsd_device.h"
#include "rvqsd_internal.h"

namespace rvqsd {

// One frame decode's buffers for models up to this size (FrameLayout::bytes):
// the 1024-wide, 2048-code model needs 5.6 MB at draft length 4 and 12.8 MB at 14.
constexpr size_t kNoAllocScratchBytes = 16u << 20;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

// Parity words to parity 1 (every byte 0x01), the pass count and the tagged
// words to 0, then the parameter block; one grid-stride pass.
__global__ void __launch_bounds__(256) noalloc_setup(uint8_t* base, size_t par_begin, size_t par_end,
                                                     size_t tag_end, KParams k, size_t o_kp) {
  const size_t n4 = tag_end / 4;
  uint32_t* w = reinterpret_cast<uint32_t*>(base);
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (size_t)gridDim.x * blockDim.x) {
    const size_t b = i * 4;
    w[i] = (b >= par_begin && b < par_end) ? 0x01010101u : 0u;
  }
  if (blockIdx.x == 0) {
    const uint32_t* src = reinterpret_cast<const uint32_t*>(&k);
    uint32_t* dst = reinterpret_cast<uint32_t*>(base + o_kp);
    for (int i = threadIdx.x; i < (int)(sizeof(KParams) / 4); i += blockDim.x) dst[i] = src[i];
  }
}

static_assert(sizeof(KParams) % 4 == 0, "parameter block is copied in 4-byte words");

namespace {

std::mutex g_mu;
uint8_t* g_ptr[kMaxDevices];  // device address of `scratch` on each device, looked up once

int scratch_of(int dev, uint8_t** out, char* err, size_t errlen) {
  if (dev < 0 || dev >= kMaxDevices) {
    snprintf(err, errlen, "device %d outside 0..%d", dev, kMaxDevices - 1);
    return RVQSD_EUNSUPPORTED;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    // the caller made `dev` current: the symbol's address on that device
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      snprintf(err, errlen, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
      return RVQSD_EHIP;
    }
    g_ptr[dev] = (uint8_t*)p;
  }
  *out = g_ptr[dev];
  return RVQSD_OK;
}

}  // namespace

}  // namespace rvqsd

namespace rvqsd {
int noalloc_launch(const rvqsd_model* m, void* hip_stream, const float* d_frame_hidden, const int32_t* d_c0,
                   const float* d_uniforms, int32_t* d_out_codes, rvqsd_stats* d_stats, char* err, size_t errlen);
}

using namespace rvqsd;

extern "C" rvqsd_status rvqsd_decode_frame_noalloc(const rvqsd_model* m, void* hip_stream, const float* d_frame_hidden,
                                                   const int32_t* d_c0, const float* d_uniforms, int32_t* d_out_codes,
                                                   rvqsd_stats* d_stats) {
  char err[256];
  const size_t errlen = sizeof(err);
  int st = noalloc_launch(m, hip_stream, d_frame_hidden, d_c0, d_uniforms, d_out_codes, d_stats, err, errlen);
  return st == RVQSD_OK ? RVQSD_OK : set_last_error(st, err);
}

namespace rvqsd {

int noalloc_launch(const rvqsd_model* m, void* hip_stream, const float* d_frame_hidden, const int32_t* d_c0,
                   const float* d_uniforms, int32_t* d_out_codes, rvqsd_stats* d_stats, char* err, size_t errlen) {
  if (!m || !d_frame_hidden || !d_c0 || !d_uniforms || !d_out_codes || !d_stats) {
    snprintf(err, errlen, "null argument");
    return RVQSD_EINVAL;
  }
  if (m->frame_bytes > kNoAllocScratchBytes) {
    snprintf(err, errlen, "the model needs %zu bytes of frame buffers; the allocation-free decode holds at most %zu",
             m->frame_bytes, kNoAllocScratchBytes);
    return RVQSD_EUNSUPPORTED;
  }
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    snprintf(err, errlen, "hipGetDevice: %s", hipGetErrorString(e));
    return RVQSD_EHIP;
  }
  if (dev != m->device) {
    snprintf(err, errlen, "current device %d, the model lives on device %d", dev, m->device);
    return RVQSD_EINVAL;
  }
  uint8_t* base = nullptr;
  const int st = scratch_of(dev, &base, err, errlen);
  if (st) return st;
  const FrameLayout fl = frame_layout(m->base);
  KParams k = m->base;
  frame_bind(&k, base, fl);
  hipStream_t hs = reinterpret_cast<hipStream_t>(hip_stream);
  const int blocks = (int)((fl.tag_end / 4 + 255) / 256 < 1024 ? (fl.tag_end / 4 + 255) / 256 : 1024);
  hipLaunchKernelGGL(noalloc_setup, dim3(blocks), dim3(256), 0, hs, base, fl.par_begin, fl.par_end, fl.tag_end, k,
                     fl.o_kp);
  e = hipGetLastError();
  if (e != hipSuccess) {
    snprintf(err, errlen, "set-up launch: %s", hipGetErrorString(e));
    return RVQSD_EHIP;
  }
  FrameArgs fa;
  fa.frame_hidden = d_frame_hidden;
  fa.c0 = d_c0;
  fa.uniforms = d_uniforms;
  fa.out_codes = d_out_codes;
  fa.out_stats = d_stats;
  fa.epoch_base = frame_epoch_step(k.L);  // every call starts from cleared tags
  fa.n_frames = 1;
  fa.epoch_step = 0;
  fa.fbar = nullptr;
  return launch_frame(reinterpret_cast<const KParams*>(base + fl.o_kp), fa, m->nwg, m->cfg.dtype, m->mr, m->mfma, hip_stream,
                      m->lds_bytes, err, errlen);
}

}  // namespace rvqsd
