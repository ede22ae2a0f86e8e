// vt_layer_decode_noalloc: batch-1 decode of a shard with the workspace in
// a scratch array that the library holds itself, for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops,
// harnesses that forbid allocation).
//
// The array is a file-scope __device__ array: each GPU the library runs on
// holds its own copy, at its own address, until the process ends. In host
// code the array's name is only a stand-in, not a device address, so the
// host takes each device's address once with hipGetSymbolAddress and uses
// that pointer wherever the array's memory is meant (kernel arguments).
// Every call on a GPU shares that GPU's array and finds the previous call's
// contents in it: the synchronisation words the decode kernel needs at zero
// are cleared by a small fill kernel ahead of every call's decode launch.
// Calls that may overlap on one GPU (other streams, other threads) race on
// the array.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "internal.hpp"

namespace vt {
namespace {

constexpr size_t kScratchBytes = VT_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes % 256 == 0, "whole 256-byte blocks");

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
std::vector<void*> g_ptr;  // per device: the address of that device's scratch

// Device address of the current device's scratch array (taken once per device).
vt_status scratch_ptr(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(VT_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  std::lock_guard<std::mutex> lk(g_mu);
  if (static_cast<int>(g_ptr.size()) <= dev) g_ptr.resize(dev + 1, nullptr);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return fail(VT_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return VT_OK;
}

__global__ void copy_word(const uint32_t* src, uint32_t* dst) {
  if (threadIdx.x == 0) *dst = *src;
}

}  // namespace
}  // namespace vt

using namespace vt;

extern "C" vt_status vt_layer_decode_noalloc(const vt_shard_spec* spec, const vt_layer_weights* w,
                                             vt_kv_view* kv, const vt_layer_io* io, int32_t pos,
                                             uint32_t phases, uint32_t* wait_error, void* stream) {
  clear_error();
  if (!spec) return fail(VT_ERR_ARG, "null spec");
  if (reinterpret_cast<uintptr_t>(wait_error) % 4)
    return fail(VT_ERR_ALIGN, "wait_error is not 4-byte aligned");
  // the workspace this call needs: the attention records grow with the context
  const int32_t ctx = (phases & VT_ATTN) ? (kv ? std::max(pos + 1, 1) : 1) : 1;
  const size_t need = decode_workspace_bytes(*spec, ctx);
  if (need > kScratchBytes)
    return fail(VT_ERR_UNSUPPORTED,
                "this shape and context need %zu bytes of workspace; the allocation-free entry "
                "point holds %zu (use vt_layer_decode with a workspace)",
                need, kScratchBytes);
  void* ws = nullptr;
  vt_status st = scratch_ptr(&ws);
  if (st != VT_OK) return st;
  // the synchronisation words the decode kernel needs at zero are cleared
  // on the stream once the arguments have passed validation
  st = layer_decode_ws(spec, w, kv, io, pos, phases, ws, kScratchBytes, stream, true);
  if (st != VT_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipSuccess;
  if (wait_error) {
    hipLaunchKernelGGL(copy_word, dim3(1), dim3(64), 0, s,
                       reinterpret_cast<const uint32_t*>(static_cast<char*>(ws) + VT_WS_ERROR_WORD),
                       wait_error);
    e = hipGetLastError();
    if (e != hipSuccess) return fail(VT_ERR_HIP, "error word copy launch: %s", hipGetErrorString(e));
  }
  return VT_OK;
}
