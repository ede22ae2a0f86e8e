"""ctypes binding of libvoltron.so (the C ABI declared in include/voltron.h).

Argument marshalling only: every step of the decoder-layer shard runs in the
library's HIP kernels. Functions keep the C names; a non-OK status raises
``VoltronError`` carrying the status and ``vt_last_error()``. Device buffers
are passed as integer addresses (e.g. ``tensor.data_ptr()``), streams as
``hipStream_t`` handles (e.g. ``torch.cuda.current_stream().cuda_stream``).
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libvoltron.so")

VT_OK = 0
VT_ERR_ARG = -1
VT_ERR_ALIGN = -2
VT_ERR_KV_FULL = -3
VT_ERR_POS = -4
VT_ERR_HIP = -5
VT_ERR_UNSUPPORTED = -6
VT_ERR_WORKSPACE = -7

VT_ATTN = 1
VT_FFN = 2
VT_STAGED = 0x100
VT_COOPERATIVE = 0x200

VT_PREC_FP16, VT_PREC_INT8, VT_PREC_INT4, VT_PREC_PRUNED = 0, 1, 2, 3
VT_W_INT8, VT_W_INT4 = 1, 2
VT_WS_ERROR_WORD = 8192  # byte offset of the workspace's barrier error word
VT_NOALLOC_SCRATCH_BYTES = 4 << 20  # the scratch array of vt_layer_decode_noalloc

# every symbol include/voltron.h declares
EXPORTS = ("vt_shard_spec_create", "vt_shard_spec_query", "vt_shard_spec_destroy",
           "vt_kv_append", "vt_workspace_size", "vt_layer_decode", "vt_layer_prefill_chunk",
           "vt_qplan", "vt_partial_encode", "vt_partial_decode_add",
           "vt_status_string", "vt_last_error", "vt_quantize_rows", "vt_layer_decode_q",
           "vt_shard_pack", "vt_kv_copy_heads", "vt_moe_workspace_size", "vt_moe_ffn_decode",
           "vt_stack_decode", "vt_layer_decode_noalloc", "vt_layer_decode_emit")


class VoltronError(RuntimeError):
    def __init__(self, status, detail):
        super().__init__(f"{status_string(status)} ({status}): {detail}")
        self.status = status
        self.detail = detail


class vt_layer_dims(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("ffn", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_base", ctypes.c_float), ("window", ctypes.c_int32)]


class vt_shard_info(ctypes.Structure):
    _fields_ = [("q_head_begin", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("kv_head_begin", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("col_begin", ctypes.c_int32), ("n_cols", ctypes.c_int32)]


class vt_layer_weights(ctypes.Structure):
    _fields_ = [("g_attn", ctypes.c_void_p),
                ("wq", ctypes.c_void_p), ("ld_q", ctypes.c_int64),
                ("wk", ctypes.c_void_p), ("ld_k", ctypes.c_int64),
                ("wv", ctypes.c_void_p), ("ld_v", ctypes.c_int64),
                ("wo", ctypes.c_void_p), ("ld_o", ctypes.c_int64),
                ("g_ffn", ctypes.c_void_p),
                ("wg", ctypes.c_void_p), ("ld_g", ctypes.c_int64),
                ("wu", ctypes.c_void_p), ("ld_u", ctypes.c_int64),
                ("wd", ctypes.c_void_p), ("ld_d", ctypes.c_int64)]


class vt_qmat(ctypes.Structure):
    _fields_ = [("codes", ctypes.c_void_p), ("ld_codes", ctypes.c_int64),
                ("scales", ctypes.c_void_p), ("ld_scales", ctypes.c_int64)]


class vt_layer_qweights(ctypes.Structure):
    _fields_ = [("prec", ctypes.c_int32), ("g_attn", ctypes.c_void_p),
                ("wq", vt_qmat), ("wk", vt_qmat), ("wv", vt_qmat), ("wo", vt_qmat),
                ("g_ffn", ctypes.c_void_p),
                ("wg", vt_qmat), ("wu", vt_qmat), ("wd", vt_qmat)]


class vt_moe_weights(ctypes.Structure):
    _fields_ = [("g_ffn", ctypes.c_void_p),
                ("wr", ctypes.c_void_p), ("ld_r", ctypes.c_int64),
                ("wg", ctypes.c_void_p), ("ld_g", ctypes.c_int64),
                ("wu", ctypes.c_void_p), ("ld_u", ctypes.c_int64),
                ("wd", ctypes.c_void_p), ("ld_d", ctypes.c_int64)]


class vt_kv_view(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("capacity", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("len", ctypes.c_int32)]


class vt_emit(ctypes.Structure):
    _fields_ = [("prec_attn", ctypes.c_void_p), ("off_attn", ctypes.c_void_p),
                ("msg_attn", ctypes.c_void_p), ("msg_attn_bytes", ctypes.c_size_t),
                ("prec_ffn", ctypes.c_void_p), ("off_ffn", ctypes.c_void_p),
                ("msg_ffn", ctypes.c_void_p), ("msg_ffn_bytes", ctypes.c_size_t)]


class vt_stack_weights(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("w", vt_layer_weights)]


class vt_kv_stack(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("n_layers", ctypes.c_int32),
                ("capacity", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("len", ctypes.c_int32)]


class vt_layer_io(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("peer_attn", ctypes.c_void_p),
                ("peer_ffn", ctypes.c_void_p), ("attn_partial", ctypes.c_void_p),
                ("h", ctypes.c_void_p), ("ffn_partial", ctypes.c_void_p),
                ("y", ctypes.c_void_p)]


_lib = None


def load_library(path=None):
    """Load the HIP library; raises if it has not been built."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it with paper_2607_07046_amd.build.build()")
    lib = ctypes.CDLL(p)
    P, I32, U32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32, ctypes.c_size_t
    lib.vt_shard_spec_create.argtypes = [ctypes.POINTER(vt_layer_dims), I32,
                                         ctypes.POINTER(ctypes.c_double),
                                         ctypes.POINTER(ctypes.c_double), I32,
                                         ctypes.POINTER(P)]
    lib.vt_shard_spec_query.argtypes = [P, ctypes.POINTER(vt_layer_dims),
                                        ctypes.POINTER(vt_shard_info)]
    lib.vt_shard_spec_destroy.argtypes = [P]
    lib.vt_shard_spec_destroy.restype = None
    lib.vt_kv_append.argtypes = [ctypes.POINTER(vt_kv_view), P, P, I32, I32, P]
    lib.vt_workspace_size.argtypes = [P, I32, I32, ctypes.POINTER(SZ)]
    lib.vt_layer_decode.argtypes = [P, ctypes.POINTER(vt_layer_weights),
                                    ctypes.POINTER(vt_kv_view), ctypes.POINTER(vt_layer_io),
                                    I32, U32, P, SZ, P]
    lib.vt_layer_prefill_chunk.argtypes = [P, ctypes.POINTER(vt_layer_weights),
                                           ctypes.POINTER(vt_kv_view),
                                           ctypes.POINTER(vt_layer_io), I32, I32, U32, P, SZ, P]
    I64 = ctypes.c_int64
    lib.vt_qplan.argtypes = [P, I32, I64, P, P, ctypes.POINTER(I64)]
    lib.vt_partial_encode.argtypes = [P, I32, P, P, P, SZ, P]
    lib.vt_partial_decode_add.argtypes = [P, SZ, I32, P, P, P, P, P]
    lib.vt_quantize_rows.argtypes = [P, I64, I32, I32, I32, P, I64, P, I64, P]
    lib.vt_layer_decode_q.argtypes = [P, ctypes.POINTER(vt_layer_qweights),
                                      ctypes.POINTER(vt_kv_view), ctypes.POINTER(vt_layer_io),
                                      I32, U32, P, SZ, P]
    lib.vt_shard_pack.argtypes = [P, ctypes.POINTER(vt_layer_weights),
                                  ctypes.POINTER(vt_layer_weights), P]
    lib.vt_kv_copy_heads.argtypes = [ctypes.POINTER(vt_kv_view), I32, ctypes.POINTER(vt_kv_view),
                                     I32, I32, I32, P]
    lib.vt_stack_decode.argtypes = [P, ctypes.POINTER(vt_stack_weights),
                                    ctypes.POINTER(vt_kv_stack), ctypes.POINTER(vt_layer_io), I32,
                                    P, SZ, P]
    lib.vt_layer_decode_noalloc.argtypes = [P, ctypes.POINTER(vt_layer_weights),
                                            ctypes.POINTER(vt_kv_view),
                                            ctypes.POINTER(vt_layer_io), I32, U32, P, P]
    lib.vt_layer_decode_emit.argtypes = [P, ctypes.POINTER(vt_layer_weights),
                                         ctypes.POINTER(vt_kv_view), ctypes.POINTER(vt_layer_io),
                                         I32, U32, ctypes.POINTER(vt_emit), P, SZ, P]
    lib.vt_moe_workspace_size.argtypes = [P, I32, I32, ctypes.POINTER(SZ)]
    lib.vt_moe_ffn_decode.argtypes = [P, ctypes.POINTER(vt_moe_weights), I32, I32,
                                      ctypes.POINTER(vt_layer_io), P, P, P, SZ, P]
    for name in ("vt_shard_spec_create", "vt_shard_spec_query", "vt_kv_append",
                 "vt_workspace_size", "vt_layer_decode", "vt_layer_prefill_chunk",
                 "vt_qplan", "vt_partial_encode", "vt_partial_decode_add",
                 "vt_quantize_rows", "vt_layer_decode_q", "vt_shard_pack", "vt_kv_copy_heads",
                 "vt_moe_workspace_size", "vt_moe_ffn_decode", "vt_stack_decode",
                 "vt_layer_decode_noalloc", "vt_layer_decode_emit"):
        getattr(lib, name).restype = ctypes.c_int
    lib.vt_status_string.argtypes = [ctypes.c_int]
    lib.vt_status_string.restype = ctypes.c_char_p
    lib.vt_last_error.argtypes = []
    lib.vt_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def status_string(status):
    return load_library().vt_status_string(status).decode()


def vt_last_error():
    return load_library().vt_last_error().decode()


def _check(status):
    if status != VT_OK:
        raise VoltronError(status, vt_last_error())


class ShardSpec:
    """Owns a vt_shard_spec handle."""

    def __init__(self, handle):
        self.handle = handle

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.vt_shard_spec_destroy(self.handle)
            self.handle = None


def vt_shard_spec_create(dims: vt_layer_dims, head_frac, col_frac, device) -> ShardSpec:
    n = len(head_frac)
    if len(col_frac) != n:
        raise ValueError("head and column fractions must have the same length")
    hf = (ctypes.c_double * max(n, 1))(*head_frac)
    cf = (ctypes.c_double * max(n, 1))(*col_frac)
    out = ctypes.c_void_p()
    _check(load_library().vt_shard_spec_create(ctypes.byref(dims), n, hf, cf, device,
                                               ctypes.byref(out)))
    return ShardSpec(out.value)


def vt_shard_spec_query(spec: ShardSpec):
    d, i = vt_layer_dims(), vt_shard_info()
    _check(load_library().vt_shard_spec_query(spec.handle, ctypes.byref(d), ctypes.byref(i)))
    return d, i


def vt_workspace_size(spec: ShardSpec, max_tokens: int, max_ctx: int) -> int:
    n = ctypes.c_size_t()
    _check(load_library().vt_workspace_size(spec.handle, max_tokens, max_ctx, ctypes.byref(n)))
    return n.value


def vt_kv_append(kv: vt_kv_view, k, v, n_tok, pos, stream=None):
    _check(load_library().vt_kv_append(ctypes.byref(kv), k, v, n_tok, pos, stream))


def vt_layer_decode(spec: ShardSpec, w: vt_layer_weights, kv, io: vt_layer_io, pos, phases,
                    ws, ws_bytes, stream=None):
    _check(load_library().vt_layer_decode(spec.handle, ctypes.byref(w),
                                          ctypes.byref(kv) if kv is not None else None,
                                          ctypes.byref(io), pos, phases, ws, ws_bytes, stream))


def vt_layer_decode_noalloc(spec: ShardSpec, w: vt_layer_weights, kv, io: vt_layer_io, pos,
                            phases, wait_error=None, stream=None):
    _check(load_library().vt_layer_decode_noalloc(spec.handle, ctypes.byref(w),
                                                  ctypes.byref(kv) if kv is not None else None,
                                                  ctypes.byref(io), pos, phases, wait_error,
                                                  stream))


def vt_layer_decode_emit(spec: ShardSpec, w: vt_layer_weights, kv, io: vt_layer_io, pos, phases,
                         emit: vt_emit, ws, ws_bytes, stream=None):
    _check(load_library().vt_layer_decode_emit(spec.handle, ctypes.byref(w),
                                               ctypes.byref(kv) if kv is not None else None,
                                               ctypes.byref(io), pos, phases, ctypes.byref(emit), ws,
                                               ws_bytes, stream))


def vt_stack_decode(spec: ShardSpec, w: vt_stack_weights, kv: vt_kv_stack, io: vt_layer_io, pos,
                    ws, ws_bytes, stream=None):
    _check(load_library().vt_stack_decode(spec.handle, ctypes.byref(w), ctypes.byref(kv),
                                          ctypes.byref(io), pos, ws, ws_bytes, stream))


def vt_layer_prefill_chunk(spec: ShardSpec, w: vt_layer_weights, kv, io: vt_layer_io, n_tok,
                           pos0, phases, ws, ws_bytes, stream=None):
    _check(load_library().vt_layer_prefill_chunk(spec.handle, ctypes.byref(w),
                                                 ctypes.byref(kv) if kv is not None else None,
                                                 ctypes.byref(io), n_tok, pos0, phases, ws,
                                                 ws_bytes, stream))


def vt_qplan(importance, budget_bytes):
    """Host plan: returns (prec uint8 [nb], offsets int32 [nb], total bytes)."""
    import numpy as np
    imp = np.ascontiguousarray(np.asarray(importance, dtype=np.float32))
    nb = imp.shape[0]
    prec = np.zeros(nb, dtype=np.uint8)
    offs = np.zeros(nb, dtype=np.int32)
    total = ctypes.c_int64(0)
    _check(load_library().vt_qplan(imp.ctypes.data, nb, int(budget_bytes), prec.ctypes.data,
                                   offs.ctypes.data, ctypes.byref(total)))
    return prec, offs, total.value


def vt_partial_encode(p, n, prec, offsets, msg, msg_bytes, stream=None):
    _check(load_library().vt_partial_encode(p, n, prec, offsets, msg, msg_bytes, stream))


def vt_partial_decode_add(msg, msg_bytes, n, prec, offsets, base, out, stream=None):
    _check(load_library().vt_partial_decode_add(msg, msg_bytes, n, prec, offsets, base, out,
                                                stream))


def vt_quantize_rows(w, ld, rows, cols, prec, codes, ld_codes, scales, ld_scales, stream=None):
    _check(load_library().vt_quantize_rows(w, ld, rows, cols, prec, codes, ld_codes, scales,
                                           ld_scales, stream))


def vt_layer_decode_q(spec: ShardSpec, w: vt_layer_qweights, kv, io: vt_layer_io, pos, phases,
                      ws, ws_bytes, stream=None):
    _check(load_library().vt_layer_decode_q(spec.handle, ctypes.byref(w),
                                            ctypes.byref(kv) if kv is not None else None,
                                            ctypes.byref(io), pos, phases, ws, ws_bytes, stream))


def vt_shard_pack(spec: ShardSpec, full: vt_layer_weights, out: vt_layer_weights, stream=None):
    _check(load_library().vt_shard_pack(spec.handle, ctypes.byref(full), ctypes.byref(out), stream))


def vt_kv_copy_heads(src: vt_kv_view, src_head0, dst: vt_kv_view, dst_head0, n_heads, n_pos,
                     stream=None):
    _check(load_library().vt_kv_copy_heads(ctypes.byref(src), src_head0, ctypes.byref(dst),
                                           dst_head0, n_heads, n_pos, stream))


def vt_moe_workspace_size(spec: ShardSpec, n_experts, top_k) -> int:
    n = ctypes.c_size_t(0)
    _check(load_library().vt_moe_workspace_size(spec.handle, n_experts, top_k, ctypes.byref(n)))
    return n.value


def vt_moe_ffn_decode(spec: ShardSpec, w: vt_moe_weights, n_experts, top_k, io: vt_layer_io,
                      sel_out, prob_out, ws, ws_bytes, stream=None):
    _check(load_library().vt_moe_ffn_decode(spec.handle, ctypes.byref(w), n_experts, top_k,
                                            ctypes.byref(io), sel_out, prob_out, ws, ws_bytes,
                                            stream))
