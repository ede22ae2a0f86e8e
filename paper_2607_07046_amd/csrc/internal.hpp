// Host-side internals shared by the library's translation units.
#pragma once

#include <cstdarg>
#include <cstdint>

#include "voltron.h"

struct vt_shard_spec {
  vt_layer_dims dims;
  vt_shard_info info;
};

namespace vt {

// Record a formatted detail for vt_last_error() and return ``s``.
vt_status fail(vt_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

// Every buffer a kernel addresses through a buffer resource stays below 2 GiB.
constexpr int64_t kMaxBufferBytes = int64_t(1) << 31;

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Checks shared by the decode and prefill entry points.
vt_status check_layer_dims(const vt_layer_dims& d);
vt_status check_weights(const vt_shard_spec& s, const vt_layer_weights* w, bool attn, bool ffn);
vt_status check_kv(const vt_shard_spec& s, const vt_kv_view* kv, int32_t pos, int32_t n_tok);

}  // namespace vt

namespace vt {
size_t decode_workspace_bytes(const vt_shard_spec& s, int32_t max_ctx);
size_t prefill_workspace_bytes(const vt_shard_spec& s, int32_t max_tokens, int32_t max_ctx);
// Leading workspace bytes that hold the decode kernel's synchronisation words
// (zero between calls; no other entry point writes them).
size_t workspace_sync_bytes(const vt_shard_spec& s);
// vt_layer_decode; with ``clear_sync`` the workspace's synchronisation words
// are zeroed (by a kernel on ``stream``) once the arguments have passed
// validation, before the decode launch.
vt_status layer_decode_ws(const vt_shard_spec* spec, const vt_layer_weights* w, vt_kv_view* kv,
                          const vt_layer_io* io, int32_t pos, uint32_t phases, void* ws,
                          size_t ws_bytes, void* stream, bool clear_sync);
}  // namespace vt
