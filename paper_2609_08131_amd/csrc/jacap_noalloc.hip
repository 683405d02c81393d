// jacap_evict_noalloc: jacap_evict without a caller workspace, for callers that
// cannot allocate device memory (code under HIP graph capture, tight serving
// loops, harnesses that forbid hipMalloc). Its workspace is `scratch`, a
// file-scope device array of kScratchBytes that each GPU the library runs on
// holds until the process ends. The host never uses the array's name as an
// address: on the first call on a device (that device current) the array's
// device address is looked up with hipGetSymbolAddress and kept per device;
// kernels receive that pointer. No memory is allocated by the call.
//
// Every call on a GPU shares that GPU's scratch array, and it keeps the last
// call's contents: calls that overlap on one GPU (on different streams, or
// from several host threads) race on it. Everything a call reads from the
// scratch is written earlier in the same call (the status word and unit flags
// are cleared by its first kernel).
#include <mutex>

#include "jacap_internal.hpp"

namespace jacap {
namespace {

// Largest workspace the entry point serves (see jacap_workspace_size): one
// Llama-3-8B layer of 8 KV heads x 8192 tokens needs about 20 MiB, 32 layers
// of one 1024-token sequence about 50 MiB.
constexpr size_t kScratchBytes = size_t(64) << 20;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) char scratch[kScratchBytes];

std::mutex g_mu;
void* g_scratch[kMaxDevices];  // per device: the device address of `scratch`

// The device address of the current device's scratch array (looked up once
// per device).
jacap_status device_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return JACAP_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return JACAP_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return JACAP_ERR_HIP;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return JACAP_OK;
}

// The sticky status word of the call, copied out for the caller.
__global__ void copy_status_kernel(const uint32_t* __restrict__ src, uint32_t* __restrict__ dst) {
  if (threadIdx.x == 0) dst[0] = src[0];
}

}  // namespace
}  // namespace jacap

extern "C" {

jacap_status jacap_evict_noalloc(const jacap_config* cfg, const jacap_batch* batch,
                                 const void* q_win, const void* k, const void* v, float* scores,
                                 int32_t* idx, void* k_out, void* v_out, uint32_t* status,
                                 void* stream) {
  size_t need = 0;
  jacap_status s = jacap_workspace_size(cfg, batch, &need);
  if (s != JACAP_OK) return s;
  if (need > jacap::kScratchBytes) return JACAP_ERR_WORKSPACE;
  if (status && (reinterpret_cast<uintptr_t>(status) & 3u)) return JACAP_ERR_INVALID_ARG;
  s = jacap::check_evict_ptrs(cfg, batch, q_win, k, v, scores, idx, k_out, v_out);
  if (s != JACAP_OK) return s;
  void* ws = nullptr;
  s = jacap::device_scratch(&ws);
  if (s != JACAP_OK) return s;
  jacap::Launch L;
  s = jacap::prepare_launch(cfg, batch, ws, jacap::kScratchBytes, stream, &L);
  if (s != JACAP_OK) return s;
  L.timed = false;  // no events: recording one would allocate
  s = jacap::evict_prepared(L, q_win, k, v, scores, idx, k_out, v_out);
  if (s != JACAP_OK) return s;
  if (status) {
    jacap::copy_status_kernel<<<1, 64, 0, L.stream>>>(
        jacap::ws_ptr<uint32_t>(L.wsp, L.ws.status), status);
    if (hipGetLastError() != hipSuccess) return JACAP_ERR_HIP;
  }
  return JACAP_OK;
}

}  // extern "C"
