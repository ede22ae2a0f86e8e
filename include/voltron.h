/*
 * voltron.h - C ABI of one device's share of an unevenly tensor-parallel
 * decoder layer (Voltron, arXiv 2607.07046), on one AMD Instinct MI355X.
 *
 * What a shard is (paper Sec. 3.2.1, Fig. Motivation1(b)): under tensor
 * parallelism the main device broadcasts a layer's input activation, every
 * device computes its shard of the layer, and the results are aggregated on
 * the main device, once per layer. Sec. 4.2.1 assigns shards to devices
 * greedily by their performance, so shards are uneven. Here a shard is a
 * contiguous range of KV groups (a KV head plus the query heads sharing it,
 * Sec. 2.1 GQA) and a contiguous range of FFN columns. Its outputs are the
 * two partial sums (after the output linear O and after the FFN down
 * projection) that the aggregation would add up; the cross-device
 * reduction itself is not part of this library.
 *
 * Layer (Sec. 2.1, Fig. Background1(a)) with the readings the paper leaves
 * open: pre-norm RMSNorm; Q/K/V projections; rotary position embedding on
 * adjacent pairs (2i, 2i+1) by angle pos * rope_base^(-2i/head_dim); the new
 * token's K and V appended to the KV cache (Sec. 2.1, LLM Inference);
 * scaled dot-product attention with scale 1/sqrt(head_dim) over positions
 * 0..pos, query head j using KV head j / (n_heads / n_kv_heads); output
 * linear O; residual; RMSNorm; SwiGLU FFN down(silu(gate) * up); residual.
 * No biases.
 *
 * Conventions for every entry point:
 *  - Numbers are fp16 (IEEE binary16) in device memory unless stated;
 *    arithmetic accumulates in fp32.
 *  - Matrices are row-major, canonical out x in; "ld" is the row stride in
 *    elements. Every device pointer must be 16-byte aligned and every ld a
 *    multiple of 8, else VT_ERR_ALIGN.
 *  - The library never allocates device memory and never synchronises. All
 *    buffers are owned by the caller. Work is enqueued on ``stream`` (a
 *    hipStream_t; NULL is the default stream).
 *  - Arguments are validated before anything is enqueued; on error nothing
 *    is enqueued, no output and no ``kv->len`` changes, and
 *    vt_last_error() (thread-local) describes the problem. Faults inside a
 *    kernel surface at the caller's next synchronisation.
 */
#ifndef VOLTRON_H
#define VOLTRON_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum vt_status {
  VT_OK = 0,
  VT_ERR_ARG = -1,          /* null pointer, bad dimension, fraction or flag */
  VT_ERR_ALIGN = -2,        /* pointer not 16-byte aligned, or ld not a multiple of 8 */
  VT_ERR_KV_FULL = -3,      /* the append would pass the cache capacity */
  VT_ERR_POS = -4,          /* pos differs from kv->len */
  VT_ERR_HIP = -5,          /* a HIP runtime call failed */
  VT_ERR_UNSUPPORTED = -6,  /* shape outside what the kernels handle */
  VT_ERR_WORKSPACE = -7     /* workspace missing or smaller than vt_workspace_size */
} vt_status;

/* Shape of the whole (unsharded) layer. head_dim must be 64 or 128;
 * hidden a multiple of 8; n_heads a multiple of n_kv_heads. ``window`` > 0
 * makes the layer's attention a sliding window (a token at position p
 * attends to positions p - window + 1 .. p only, the local layers of the
 * gemma models of the paper's Table 3); 0 is full causal attention. */
typedef struct vt_layer_dims {
  int32_t hidden;
  int32_t n_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t ffn;
  float rms_eps;
  float rope_base;
  int32_t window;
} vt_layer_dims;

/* One device's shard: query heads [q_head_begin, +n_q_heads), KV heads
 * [kv_head_begin, +n_kv_heads) (n_q_heads = n_kv_heads * group) and FFN
 * columns [col_begin, +n_cols) of the layer. */
typedef struct vt_shard_info {
  int32_t q_head_begin;
  int32_t n_q_heads;
  int32_t kv_head_begin;
  int32_t n_kv_heads;
  int32_t col_begin;
  int32_t n_cols;
} vt_shard_info;

typedef struct vt_shard_spec vt_shard_spec; /* opaque, host-only, immutable */

/* Partition a layer over ``n_devices`` devices and describe ``device``'s
 * share (paper Sec. 4.2.1: greedy, performance-proportional shards).
 * head_frac[i] / col_frac[i] are device i's fractions of the KV groups and
 * of the FFN columns: finite, >= 0, each array summing to 1 within 1e-9.
 * Rounding: largest remainder. Device i gets floor(frac[i] * units) units
 * (product in IEEE double), then the units still unassigned go one each to
 * the devices with the largest fractional parts, the lower index first on
 * ties; devices take contiguous ranges in index order. A device may get no
 * heads or no columns; its partial sums are then zero.
 * On success *out receives a spec to free with vt_shard_spec_destroy. */
vt_status vt_shard_spec_create(const vt_layer_dims* dims, int32_t n_devices,
                               const double* head_frac, const double* col_frac,
                               int32_t device, vt_shard_spec** out);

/* Copy the spec's layer shape and shard ranges out (either may be NULL). */
vt_status vt_shard_spec_query(const vt_shard_spec* spec, vt_layer_dims* dims_out,
                              vt_shard_info* info_out);

void vt_shard_spec_destroy(vt_shard_spec* spec);

/* The shard's weights, caller-owned device fp16, rows as described (shard
 * rows / shard columns of the canonical layer tensors; the columns of wo
 * and wd are the shard's query-head features and FFN columns). Each ld is
 * the row stride in elements (>= row length, multiple of 8).
 *   g_attn [hidden]                 RMSNorm gain before attention
 *   wq [n_q_heads*head_dim][hidden]  wk, wv [n_kv_heads*head_dim][hidden]
 *   wo [hidden][n_q_heads*head_dim]
 *   g_ffn [hidden]                  RMSNorm gain before the FFN
 *   wg, wu [n_cols][hidden]         gate and up projections
 *   wd [hidden][n_cols]             down projection
 * Pointers of a part the shard does not have (no heads / no columns) may be
 * NULL. */
typedef struct vt_layer_weights {
  const void* g_attn;
  const void* wq; int64_t ld_q;
  const void* wk; int64_t ld_k;
  const void* wv; int64_t ld_v;
  const void* wo; int64_t ld_o;
  const void* g_ffn;
  const void* wg; int64_t ld_g;
  const void* wu; int64_t ld_u;
  const void* wd; int64_t ld_d;
} vt_layer_weights;

/* KV cache of the shard's KV heads for one layer: k and v are
 * [n_kv_heads][capacity][head_dim] fp16, caller-owned. ``len`` is the number
 * of positions filled (0..len-1); successful appends advance it on the host
 * when the work is enqueued. Keys are stored after rotation. */
typedef struct vt_kv_view {
  void* k;
  void* v;
  int32_t capacity;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t len;
} vt_kv_view;

/* Activations of T tokens (T = 1 for decode), each [T][hidden] fp16:
 *   x            in   layer input (the broadcast activation)
 *   peer_attn    in   nullable; sum of the other devices' attention partials
 *   peer_ffn     in   nullable; sum of the other devices' FFN partials
 *   attn_partial out  Wo[:, shard heads] * attention output   (VT_ATTN)
 *   h            out  x + attn_partial + peer_attn            (VT_ATTN)
 *                in   FFN input when VT_FFN runs without VT_ATTN
 *   ffn_partial  out  Wd[:, shard columns] * silu(gate) * up  (VT_FFN)
 *   y            out  nullable; h + ffn_partial + peer_ffn     (VT_FFN)
 * NULL peers count as zero. When both phases run, the FFN reads h as
 * written (rounded to fp16). */
typedef struct vt_layer_io {
  const void* x;
  const void* peer_attn;
  const void* peer_ffn;
  void* attn_partial;
  void* h;
  void* ffn_partial;
  void* y;
} vt_layer_io;

/* Phase mask bits for vt_layer_decode / vt_layer_prefill_chunk. */
#define VT_ATTN 1u          /* RMSNorm, QKV, RoPE, KV append, attention, O, h */
#define VT_FFN 2u           /* RMSNorm, gate/up, SiLU-gate, down, y */
#define VT_STAGED 0x100u    /* decode only: one kernel launch per stage instead
                               of the single persistent kernel (same results
                               up to fp32 rounding order, which is fixed) */
#define VT_COOPERATIVE 0x200u /* decode only, not with VT_STAGED: launch the
                               persistent kernel through the cooperative
                               launch, which guarantees that every workgroup
                               is resident at once or fails the call
                               (VT_ERR_HIP) before anything runs, instead of
                               the bounded wait's asynchronous error word;
                               costs launch time (same results bit for bit) */

/* Append n_tok tokens' keys and values at positions pos..pos+n_tok-1 of
 * every KV head (paper Sec. 2.1, LLM Inference: the K and V of new tokens
 * are accumulated into the KV cache). k, v: [n_tok][n_kv_heads][head_dim]
 * fp16 device. A pure copy: the stored bytes equal the input bytes and no
 * other byte of the cache changes. Requires pos == kv->len (VT_ERR_POS) and
 * pos + n_tok <= capacity (VT_ERR_KV_FULL); then kv->len = pos + n_tok. */
vt_status vt_kv_append(vt_kv_view* kv, const void* k, const void* v, int32_t n_tok,
                       int32_t pos, void* stream);

/* Bytes of device workspace that vt_layer_decode / vt_layer_prefill_chunk
 * need for this shard with up to ``max_tokens`` tokens per chunk (1 for
 * decode only) and ``max_ctx`` cached-plus-new positions. The workspace must
 * be zero-filled once before its first use; the library leaves its
 * synchronisation words zero after every call. One workspace must not be
 * used by two calls that may run at the same time.
 *
 * A persistent decode (or MoE) launch needs every one of its workgroups
 * (one per CU) resident at once; its grid barriers wait a bounded time (about
 * a second) and, should that ever expire (other work holding CUs), set the
 * 32-bit error word at byte offset VT_WS_ERROR_WORD of the workspace to
 * nonzero instead of hanging; the call's outputs are then undefined. The
 * library never clears that word: a caller that checks it reads it after
 * synchronising and zeroes it itself. A prefill chunk's GEMMs wait only for
 * workgroups that are already running, under the same bound and report. */
#define VT_WS_ERROR_WORD 8192
vt_status vt_workspace_size(const vt_shard_spec* spec, int32_t max_tokens,
                            int32_t max_ctx, size_t* bytes);

/* Batch-1 decode of one token at position ``pos`` through the shard
 * (paper Sec. 2.1 LLM Inference, Sec. 3.2.1 TP shard). ``phases`` is
 * VT_ATTN, VT_FFN or both, optionally with VT_STAGED or VT_COOPERATIVE. With VT_ATTN the
 * token's rotated key and its value are appended at slot ``pos`` of every
 * shard KV head (pos must equal kv->len and be < capacity; kv->len becomes
 * pos + 1) and attention covers positions 0..pos. ``kv`` and ``pos`` are
 * ignored without VT_ATTN. Outputs per vt_layer_io. */
vt_status vt_layer_decode(const vt_shard_spec* spec, const vt_layer_weights* w,
                          vt_kv_view* kv, const vt_layer_io* io, int32_t pos,
                          uint32_t phases, void* ws, size_t ws_bytes, void* stream);

/* ---- Decode without a caller workspace ----
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * step as vt_layer_decode, its workspace taken from a scratch array of
 * VT_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on
 * (until the process ends). Nothing is allocated and nothing synchronises.
 * Every call on a GPU shares that GPU's array: the call clears what must
 * start at zero (a small kernel on ``stream`` ahead of the decode), and
 * calls that may overlap on one GPU (other streams or threads) race.
 * VT_ERR_UNSUPPORTED when the shape and context need a larger workspace
 * than the array (vt_workspace_size of the spec with max_ctx = pos + 1).
 * ``wait_error`` (nullable, device, 4-byte aligned): receives the barrier
 * error word of this call (nonzero if a bounded grid wait expired and the
 * outputs are undefined), written on ``stream`` after the decode. Other
 * arguments, outputs and errors as vt_layer_decode. */
#define VT_NOALLOC_SCRATCH_BYTES (4u << 20)
vt_status vt_layer_decode_noalloc(const vt_shard_spec* spec, const vt_layer_weights* w,
                                  vt_kv_view* kv, const vt_layer_io* io, int32_t pos,
                                  uint32_t phases, uint32_t* wait_error, void* stream);

/* ---- A stack of layers decoded in one launch (paper Sec. 2.1: an LLM
 * stacks identically structured decoders; Sec. 3.2.1: the tensor-parallel
 * split repeats at every layer) ----
 * n_layers consecutive layers of one shard shape decode one token at
 * position ``pos``: layer 0's input is io->x and layer l's input is layer
 * l-1's output y (the single-device chain; the aggregation between layers
 * is what the peers stand for, NULL counting as zero). The results equal
 * n_layers calls of vt_layer_decode with VT_ATTN | VT_FFN, each fed the
 * previous call's y, bit for bit; one persistent launch runs them all, so
 * layer l+1's first weights stream while layer l ends. */
typedef struct vt_stack_weights {
  int32_t n_layers;      /* 1..4096 */
  vt_layer_weights w;    /* each pointer addresses n_layers consecutive copies of its
                            tensor: layer l's matrix starts l * rows * ld elements past
                            layer 0's (rows as in vt_layer_weights), its gains l * hidden
                            elements past; fp16 weights only */
} vt_stack_weights;

/* KV caches of a stack: k and v are [n_layers][n_kv_heads][capacity][head_dim]
 * fp16, caller-owned; ``len`` positions are filled in every layer. */
typedef struct vt_kv_stack {
  void* k;
  void* v;
  int32_t n_layers;
  int32_t capacity;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t len;
} vt_kv_stack;

/* One token through the stack. io->x: [hidden] in; io->attn_partial, h,
 * ffn_partial, y: [n_layers][hidden] out, all required (row l is layer l's
 * vector, as vt_layer_io describes it); io->peer_attn / peer_ffn: NULL or
 * [n_layers][hidden]. Every layer appends its token's key and value at slot
 * ``pos`` (pos must equal kv->len and be < capacity; kv->len becomes pos + 1).
 * Workspace as for vt_layer_decode (vt_workspace_size of the spec). Errors
 * as vt_layer_decode, plus VT_ERR_ARG when the weights' and the KV stack's
 * layer counts differ. */
vt_status vt_stack_decode(const vt_shard_spec* spec, const vt_stack_weights* w, vt_kv_stack* kv,
                          const vt_layer_io* io, int32_t pos, void* ws, size_t ws_bytes,
                          void* stream);

/* Prefill of a chunk of n_tok tokens at positions pos0..pos0+n_tok-1 (paper
 * Sec. 2.1: prompt tokens are processed in parallel). All n_tok keys and
 * values are appended (pos0 must equal kv->len); token t attends to
 * positions 0..pos0+t (the last dims.window of them in a sliding-window
 * layer). Activations in io are [n_tok][hidden]. The
 * projections run as fp16 matrix-core (MFMA) GEMMs with fp32 accumulation;
 * their activation operands are rounded to fp16 first. */
vt_status vt_layer_prefill_chunk(const vt_shard_spec* spec, const vt_layer_weights* w,
                                 vt_kv_view* kv, const vt_layer_io* io, int32_t n_tok,
                                 int32_t pos0, uint32_t phases, void* ws, size_t ws_bytes,
                                 void* stream);

/* ---- Block-quantised weight shards (paper Sec. 2.2 precision
 * heterogeneity, Sec. 4.2.2 importance-aware mixed precision, Sec. 4.3.1
 * precision scaling) ----
 * A layer's weights may be held at INT8 or INT4 instead of FP16; which
 * precision a layer gets is the caller's choice (the paper picks it per
 * layer by importance under a memory budget). The paper's own block
 * formats are not defined in it; this library's format is:
 *  - each row is cut into blocks of 32 consecutive input columns (the last
 *    block may be partial; its missing columns count as zero);
 *  - a block has one fp16 scale s = fp16(absmax / Q) (fp32 division, round
 *    to nearest even; Q = 127 for INT8, 7 for INT4) and codes
 *    c = clamp(rint(w / s), -Q, Q) (fp32 division, ties to even); s = 0
 *    (an all-zero block, or absmax / Q below the fp16 range) gives c = 0;
 *    the weight it stands for is c * s;
 *  - row r's codes start at codes + r * ld_codes (bytes): INT8 one
 *    two's-complement byte per column; INT4 offset-binary nibbles c + 8, 8
 *    columns per 4 bytes, column 8g + i (i < 4) in the low nibble of byte
 *    4g + i and column 8g + 4 + i in its high nibble. The codes of a row's
 *    last block past its columns are 0. ld_codes is a multiple of 16 and at
 *    least 32 (INT8) or 16 (INT4) bytes per block;
 *  - row r's scales (fp16, one per block in column order) start at
 *    scales + r * ld_scales (elements); ld_scales >= the block count; the
 *    scales pointer needs 2-byte alignment only. */
enum { VT_W_INT8 = 1, VT_W_INT4 = 2 };

typedef struct vt_qmat {
  const void* codes;
  int64_t ld_codes;  /* bytes */
  const void* scales;
  int64_t ld_scales; /* fp16 elements */
} vt_qmat;

/* A shard's weights in the block format, all seven matrices at one
 * precision ``prec`` (VT_W_INT8 or VT_W_INT4). Shapes and slicing as in
 * vt_layer_weights (wd's row length is the shard's column count; no
 * further padding is needed: its last block is padded by the format). The
 * RMSNorm gains stay fp16. */
typedef struct vt_layer_qweights {
  int32_t prec;
  const void* g_attn;
  vt_qmat wq, wk, wv, wo;
  const void* g_ffn;
  vt_qmat wg, wu, wd;
} vt_layer_qweights;

/* Quantise the fp16 matrix w (rows x cols, row stride ld elements) into
 * ``prec`` blocks: writes the code bytes of each row's blocks and their
 * scales; bytes past them (up to ld_codes / ld_scales) are left as they
 * are. codes holds rows * ld_codes bytes and scales rows * ld_scales fp16
 * elements (device). */
vt_status vt_quantize_rows(const void* w, int64_t ld, int32_t rows, int32_t cols, int32_t prec,
                           void* codes, int64_t ld_codes, void* scales, int64_t ld_scales,
                           void* stream);

/* vt_layer_decode over block-quantised weights: the same step, every
 * projection computed as sum over blocks of s * sum(c * x) with the fp16
 * input x and fp32 accumulation. Same arguments, errors and outputs; in
 * addition VT_ERR_UNSUPPORTED if a matrix row has more than 16384 columns. */
vt_status vt_layer_decode_q(const vt_shard_spec* spec, const vt_layer_qweights* w,
                            vt_kv_view* kv, const vt_layer_io* io, int32_t pos,
                            uint32_t phases, void* ws, size_t ws_bytes, void* stream);

/* ---- Elastic re-partition and shard-wise pruning (paper Sec. 4.3.1) ----
 * When devices come and go or run short of memory, the partition changes:
 * shards move between devices or are pruned (dropped whole, the kept
 * shards' partial sums then add up to the layer without the dropped heads
 * and columns). Shards are allocated separately, so a device packs its new
 * shard into new buffers on a second stream while it keeps decoding with
 * the old ones, and takes over the KV heads of the groups it now owns. A
 * pruned shard is simply not run; nothing here is needed for it. */

/* Gather ``spec``'s shard out of the whole layer's weights ``full`` (device,
 * canonical out x in: wq [n_heads*head_dim][hidden], wk and wv
 * [n_kv_heads*head_dim][hidden], wo [hidden][n_heads*head_dim], wg and wu
 * [ffn][hidden], wd [hidden][ffn], gains [hidden]; every ld a multiple of 8)
 * into the shard's buffers ``out`` (device, shaped as vt_layer_decode takes
 * them; out->ld_d >= n_cols rounded up to 8: the columns from n_cols to
 * that multiple of 8 are written as zero). Bit-exact copies enqueued on
 * ``stream``; both structs are read on the host only. */
vt_status vt_shard_pack(const vt_shard_spec* spec, const vt_layer_weights* full,
                        const vt_layer_weights* out, void* stream);

/* Copy positions 0..n_pos-1 of KV heads [src_head0, src_head0 + n_heads) of
 * ``src`` into heads [dst_head0, ...) of ``dst`` (keys and values; caches of
 * equal head_dim, any capacities >= n_pos), on ``stream``. Other slots and
 * dst->len are left as they are (the caller sets len once every head is
 * in place). */
vt_status vt_kv_copy_heads(const vt_kv_view* src, int32_t src_head0, const vt_kv_view* dst,
                           int32_t dst_head0, int32_t n_heads, int32_t n_pos, void* stream);

/* ---- Mixture-of-experts FFN (paper Sec. 2.1 FFN variants; Table 3's
 * MoE model) ----
 * The FFN sub-layer of an MoE layer, batch-1 decode, on one device's share:
 * w = RMSNorm(h) * g_ffn; router logits r = Wr w over the n_experts
 * experts; the top_k experts with the largest logits (ties: the lower
 * index) are selected; output = sum over them of p_e * Wd_e (silu(Wg_e w)
 * * (Wu_e w)), p = softmax(r) over all n_experts (not renormalised over
 * the selection). Tensor parallelism shards every expert by its FFN columns
 * as for the dense FFN, and every device routes for itself (the router is
 * small), so the devices' partial sums add up to the unsharded output. The
 * routed experts only: a shared expert is a dense FFN (vt_layer_decode
 * with VT_FFN). */

/* An MoE shard's weights (device, fp16, ld in elements, multiples of 8):
 * wr [n_experts][ld_r >= hidden] router rows; wg, wu
 * [n_experts][n_cols][ld >= hidden]: expert e's gate / up rows of the
 * shard's columns (spec's col_begin.. of the expert's FFN); wd
 * [n_experts][hidden][ld_d >= n_cols]: expert e's down rows over those
 * columns. Each matrix must span less than 2 GiB. With n_cols = 0 the
 * expert matrices may be NULL (the partial sum is then zero). */
typedef struct vt_moe_weights {
  const void* g_ffn;  /* [hidden] */
  const void* wr;
  int64_t ld_r;
  const void* wg;
  int64_t ld_g;
  const void* wu;
  int64_t ld_u;
  const void* wd;
  int64_t ld_d;
} vt_moe_weights;

/* Workspace bytes of vt_moe_ffn_decode (zero-filled once before its first
 * use; the synchronisation words are left zero after every call; not shared
 * by calls that may run at the same time; the barrier error word at
 * VT_WS_ERROR_WORD as for decode). 1 <= n_experts <= 256,
 * 1 <= top_k <= min(n_experts, 8), spec's n_cols < 32768. */
vt_status vt_moe_workspace_size(const vt_shard_spec* spec, int32_t n_experts, int32_t top_k,
                                size_t* bytes);

/* One token through the MoE FFN shard. ``spec``: the layer's shard spec
 * with dims.ffn one expert's FFN width (its n_cols / col_begin are the
 * shard's columns of every expert; the attention fields are not used).
 * Reads io->h and io->peer_ffn (optional); writes io->ffn_partial and, if
 * not NULL, io->y = h + ffn_partial + peer_ffn (fp32 sum, rounded once).
 * sel_out / prob_out (device, optional): the selected experts in
 * descending logit order and their probabilities [top_k]. hidden must be a
 * multiple of 8 up to 16384. */
vt_status vt_moe_ffn_decode(const vt_shard_spec* spec, const vt_moe_weights* w, int32_t n_experts,
                            int32_t top_k, const vt_layer_io* io, int32_t* sel_out, float* prob_out,
                            void* ws, size_t ws_bytes, void* stream);

/* ---- Communication scaling of the partial sums (paper Sec. 4.3.2) ----
 * To cut the bytes a device sends for the aggregation, its partial sums go
 * out in blocks of 32 activations, each at one precision; precisions are
 * lowered in ascending order of importance (Sec. 4.3.2 with the
 * importance-ordered lowering of Sec. 4.2.2) until the message fits a byte
 * budget, and pruned blocks are not sent at all.
 * Block wire format, blocks in index order, block b at offsets[b]:
 *   VT_PREC_FP16   64 bytes: the 32 fp16 values
 *   VT_PREC_INT8   36 bytes: fp32 scale s, 32 int8 codes; value = code * s
 *   VT_PREC_INT4   20 bytes: fp32 scale s, 16 bytes of 4-bit two's-complement
 *                  codes, element 2k in the low nibble of byte k
 *   VT_PREC_PRUNED  0 bytes: value 0
 * Quantisation of a block (symmetric absmax, fp32): s = absmax / Q with
 * Q = 127 (INT8) or 7 (INT4); code = clamp(rint(x / s), -Q, Q), rint
 * rounding half to even; an all-zero block has s = 0 and codes 0. */
enum { VT_PREC_FP16 = 0, VT_PREC_INT8 = 1, VT_PREC_INT4 = 2, VT_PREC_PRUNED = 3 };

/* Host-only plan for n_blocks blocks (1..2^24) with importance scores
 * importance[b] (finite; higher = more important; the caller sums, per
 * block, the importance of the weight shards that produce its activations).
 * All blocks start at FP16; in ascending importance (ties: lower index
 * first) blocks go FP16 -> INT8 one at a time until the message is at most
 * budget_bytes; if it is still larger, INT8 -> INT4 in the same order, then
 * INT4 -> pruned. Writes prec[n_blocks] (VT_PREC_*), offsets[n_blocks]
 * (bytes) and *total_bytes. All pointers are host memory. */
vt_status vt_qplan(const float* importance, int32_t n_blocks, int64_t budget_bytes,
                   uint8_t* prec, int32_t* offsets, int64_t* total_bytes);

/* Encode the fp16 partial sums p[n] (n a positive multiple of 32) into the
 * message msg[msg_bytes] (device) under a plan held in device memory
 * (prec[n/32], offsets[n/32], as vt_qplan wrote them). msg must be non-NULL
 * (16 bytes suffice for an all-pruned plan); nothing is written outside
 * [msg, msg + msg_bytes) whatever the plan holds. Bytes of msg not covered
 * by a block are left as they are. */
vt_status vt_partial_encode(const void* p, int32_t n, const uint8_t* prec, const int32_t* offsets,
                            void* msg, size_t msg_bytes, void* stream);

/* Receiver side: out[i] = fp16(base[i] + value[i]) for i < n, value as in the
 * wire format (code * s in fp32, then an fp32 add; base NULL reads as 0).
 * Reads outside [msg, msg + msg_bytes) return zero. out may equal base. */
vt_status vt_partial_decode_add(const void* msg, size_t msg_bytes, int32_t n, const uint8_t* prec,
                                const int32_t* offsets, const void* base, void* out, void* stream);

/* The same quantised messages emitted by the decode step itself: the O and
 * down projections' epilogues give each workgroup whole blocks of 32 output
 * rows, so a block's partial sums leave in the message as soon as they are
 * formed, with no further launch. For each partial (attention: io->
 * attn_partial; FFN: io->ffn_partial), a plan in device memory (prec and
 * offsets of hidden / 32 blocks, as vt_qplan writes them) and a message
 * buffer of msg_bytes (device); the bytes written equal what
 * vt_partial_encode writes for that partial vector, and nothing is written
 * outside [msg, msg + msg_bytes). A NULL message is not emitted. */
typedef struct vt_emit {
  const uint8_t* prec_attn;
  const int32_t* off_attn;
  void* msg_attn;
  size_t msg_attn_bytes;
  const uint8_t* prec_ffn;
  const int32_t* off_ffn;
  void* msg_ffn;
  size_t msg_ffn_bytes;
} vt_emit;

/* vt_layer_decode (fp16 weights, persistent launch) that also emits the
 * quantised partial sums per ``emit``. Outputs as vt_layer_decode, equal to
 * it up to the fp32 summation order of each row. VT_ERR_UNSUPPORTED with
 * VT_STAGED or when hidden is not a multiple of 32; VT_ERR_ARG when a
 * message is given without a plan or for a phase that does not run. */
vt_status vt_layer_decode_emit(const vt_shard_spec* spec, const vt_layer_weights* w,
                               vt_kv_view* kv, const vt_layer_io* io, int32_t pos,
                               uint32_t phases, const vt_emit* emit, void* ws, size_t ws_bytes,
                               void* stream);

/* Static text of a status code. */
const char* vt_status_string(vt_status s);

/* Detail of the last error on the calling thread ("" if none). */
const char* vt_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* VOLTRON_H */
