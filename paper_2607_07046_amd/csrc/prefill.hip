// Prefill chunk of one device's shard (MFMA path). Placeholder until the
// GEMM and causal-attention kernels land.
#include <hip/hip_runtime.h>

#include "device.hpp"
#include "internal.hpp"

namespace vt {
size_t prefill_workspace_bytes(const vt_shard_spec&, int32_t, int32_t) { return 0; }
}  // namespace vt

extern "C" vt_status vt_layer_prefill_chunk(const vt_shard_spec* spec, const vt_layer_weights* w,
                                            vt_kv_view* kv, const vt_layer_io* io, int32_t n_tok,
                                            int32_t pos0, uint32_t phases, void* ws, size_t ws_bytes,
                                            void* stream) {
  (void)spec; (void)w; (void)kv; (void)io; (void)n_tok; (void)pos0; (void)phases; (void)ws;
  (void)ws_bytes; (void)stream;
  vt::clear_error();
  return vt::fail(VT_ERR_UNSUPPORTED, "prefill not built yet");
}
