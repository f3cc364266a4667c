// comba_chunk_fwd_noalloc: the chunk-wise forward on a static device scratch
// array, for callers that cannot allocate device memory (code under HIP graph
// capture, tight serving loops, harnesses that forbid hipMalloc).
//
// The forward's workspace (chunk tables, the per-chunk gates G and the int16
// UT-transform inverse M and score matrix A with their row scales) lives in
// `scratch`, a file-scope device array of kScratchBytes that every device the
// library runs on holds until the process ends.  In host code the name
// `scratch` is only a host-side stand-in: its device address is taken once per
// device with hipGetSymbolAddress, with that device current, and only that
// address is ever passed to kernels.  Nothing in the scratch has to start at
// zero: every byte a call reads was written earlier in the same call.  Calls
// that overlap in time on one device share the array and race; order them on
// one stream (or synchronise them).
#include <hip/hip_runtime.h>

#include <mutex>

#include "comba.h"
#include "comba_launch.h"

namespace {

constexpr size_t kScratchBytes = size_t(80) << 20;  // 80 MiB
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's scratch (nullptr on failure).
void* device_scratch() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

size_t comba_noalloc_scratch_bytes(void) { return kScratchBytes; }

comba_status comba_chunk_fwd_noalloc(const comba_shape* shape, const void* q, const void* k,
                                     const void* v, const float* g, const void* beta,
                                     const void* beta_tilde, const float* d, const float* h0,
                                     float* o, float* ht, void* stream) {
  if (!shape) return COMBA_ERR_NULL;
  // the plain scan's workspace must fit; the segmented scan runs only when its
  // buffers fit too (comba_chunk_fwd falls back to the plain scan otherwise)
  const size_t need = comba::fwd_workspace_bytes_plain(shape);
  if (need == 0) return COMBA_ERR_SHAPE;  // the shape itself is invalid
  if (need > kScratchBytes) return COMBA_ERR_SCRATCH;
  void* ws = device_scratch();
  if (!ws) return COMBA_ERR_HIP;
  return comba_chunk_fwd(shape, q, k, v, g, beta, beta_tilde, d, h0, o, ht, ws, kScratchBytes,
                         stream);
}

}  // extern "C"
