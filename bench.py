"""Decode-layer-shard throughput on one MI355X.

A step is one batch-1 decode token through the whole hot path (RMSNorm,
QKV, RoPE, KV append, attention, O, residual, RMSNorm, gate/up, SiLU-gate,
down, residual). The headline workload is the largest single-GPU one: the
13B-shaped 40-layer stack, 40% shard (16 of 40 heads, 5530 of 13824 FFN
columns), consecutive tokens from position 2048, each token through all 40
layers in one vt_stack_decode launch (layer l's y is layer l+1's x), every
layer appending to its own KV cache. Its 10.8 GB of weights per token
stream from HBM (far past the 256 MB Infinity Cache). Inputs are resident
in HBM before timing starts.

Prints one JSON line. ``value`` is tokens/s; the HBM figure is algorithmic
bytes per token / time per token; ``roofline`` reports the stack launch (one
per token) against the 8 TB/s HBM peak. Sections: ``decode_7b`` and
``decode_70b_gqa`` time single-layer shards (the 7B-shaped 30% shard at
position 1024 and the 70B-shaped GQA 25% shard at position 4096) with
rotated weight/KV copies (>= 768 MB) and the y -> x chain, each with its own
roofline block; ``per_layer_launches`` the same stack with one launch per
layer; ``prefill`` the 256-token prefill chunk (MFMA utilisation); ``comm``
the partial-sum transmission kernels; ``quant`` the 7B decode over INT8 and
INT4 block-quantised weights; ``repack`` the shard re-pack of an elastic
re-partition; ``moe`` the MoE FFN shard. ``cpu_baseline`` is the fp64
oracle timed on the host cores on a bounded sample of the headline workload
(a reference, not the target).
"""
import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode-layer-shard tokens/s and achieved HBM GB/s (% of peak), 1 MI355X"
HBM_PEAK_GBPS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0  # dense fp16 matrix-core peak
MALL_DEFEAT_BYTES = 768 * 2 ** 20


def algorithmic_bytes(dims, info, pos):
    """Bytes the decode step must move: every shard weight once, the cached
    K/V of the attended positions (0..pos-1, or a sliding window's) read
    plus the new K/V written, the gains, x in, and the four fp16 output
    vectors."""
    H, d = dims.hidden, dims.head_dim
    nq, nkv, F = info.n_q_heads, info.n_kv_heads, info.n_cols
    weights = 2 * ((nq + 2 * nkv) * d * H + H * nq * d + 3 * F * H)
    span = min(pos + 1, dims.window) if dims.window > 0 else pos + 1  # positions attended
    kv = 4 * nkv * d * span
    vectors = 2 * H * (2 + 1 + 4)  # gains, x, attn_partial/h/ffn_partial/y
    return weights + kv + vectors


DECODE_SOURCES = ("decode.hip", "gemv.hpp", "device.hpp")
MOE_SOURCES = ("moe.hip", "gemv.hpp", "device.hpp")
PROFILES = {"13b_stack": "decode_kernel_13b_stack40.md", "7b": "decode_kernel_7b_shard30.md",
            "70b_gqa": "decode_kernel_70b_gqa_shard25.md"}


def kernel_source_hash(files=DECODE_SOURCES):
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2607_07046_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary of
    the workload, or None if there is none or the kernel sources changed
    since the counters were taken."""
    import re
    try:
        with open(os.path.join(ROOT, "profiles", PROFILES[workload])) as f:
            txt = f.read()
    except (OSError, KeyError):
        return None
    m_hash = re.search(r"first 16 hex\): `([0-9a-f]{16})`", txt)
    m_traffic = re.search(r"\*\*([0-9,]+) B\*\*", txt)
    if not m_hash or not m_traffic or m_hash.group(1) != kernel_source_hash():
        return None
    return int(m_traffic.group(1).replace(",", ""))


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=60, help="timed tokens of the headline")
    ap.add_argument("--warmup", type=int, default=6)
    ap.add_argument("--config", default="13b_stack",
                    help="headline workload (synth.configs): a stack, or a single-layer decode "
                         "workload timed as the decode sections are")
    ap.add_argument("--decode-steps", type=int, default=2000,
                    help="timed steps of each single-layer decode section (0: skip)")
    ap.add_argument("--per-layer-tokens", type=int, default=8,
                    help="tokens of the stack run with one launch per layer (0: skip)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="host time budget of the oracle baseline (0: skip)")
    ap.add_argument("--prefill-steps", type=int, default=200,
                    help="timed prefill chunks of the prefill section (0: skip)")
    ap.add_argument("--prefill-tokens", type=int, default=0,
                    help="tokens per prefill chunk (default: the workload's 256)")
    ap.add_argument("--comm-steps", type=int, default=400,
                    help="timed calls of each partial-sum transmission kernel (0: skip)")
    ap.add_argument("--quant-steps", type=int, default=1000,
                    help="timed decode steps over INT8 and INT4 weight shards (0: skip)")
    ap.add_argument("--moe-steps", type=int, default=1000,
                    help="MoE FFN shard decode steps (0: skip)")
    ap.add_argument("--repack-reps", type=int, default=20,
                    help="timed shard packs of the re-partition section (0: skip)")
    ap.add_argument("--fraction-sweep", action="store_true",
                    help="also time the decode step of 7B- and 70B-shaped shards from 10%% to 100%% "
                         "of the layer and fit time = fixed + bytes / bandwidth (about a minute)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="instead of the bench: copy MIB MiB device-to-device 10 times "
                         "(the known-size kernel that scales the HBM byte counters), then "
                         "sum and fill the same bytes 10 times each (cross-checks)")
    return ap.parse_args()


def copy_calibration(mib):
    import torch
    n = mib * 2 ** 20 // 2
    src = torch.ones(n, dtype=torch.float16, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(10):
        dst.copy_(src)
    torch.cuda.synchronize()
    # cross-checks of the scale on kernels that only read or only write the
    # same size: a sum over src, a fill of dst
    for _ in range(10):
        src.sum(dtype=torch.float32)
    for _ in range(10):
        dst.fill_(0.5)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read_per_launch": n * 2,
                      "bytes_written_per_launch": n * 2, "launches": 10,
                      "cross_checks": "10 sums reading the same bytes, 10 fills writing them"}))


def lib_dims(wd):
    from paper_2607_07046_amd import voltron as vt
    return vt.vt_layer_dims(hidden=wd.hidden, n_heads=wd.n_heads, n_kv_heads=wd.n_kv_heads,
                            head_dim=wd.head_dim, ffn=wd.ffn, rms_eps=wd.rms_eps,
                            rope_base=wd.rope_base, window=wd.window)


def device_normal(seed):
    """Seeded fp16 N(mean, sigma) tensors drawn on the device (for weights
    too large to draw on the host quickly)."""
    import torch
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)

    def normal(shape, sigma, mean=0.0):
        t = torch.empty(shape, dtype=torch.float32, device="cuda")
        t.normal_(mean, sigma, generator=gen)
        return t.half()
    return normal


def roofline(step_bytes, ms, kernel, workload, launches_per_step=1):
    gbps = step_bytes / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "kernel": kernel, "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS,
            "unit": "GB/s", "frac": round(gbps / HBM_PEAK_GBPS, 4),
            "traffic": measured_traffic(workload),
            "traffic_unit": "B per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-scaled)",
            "launches_per_step": launches_per_step}


def windows(steps, nwin=20):
    nwin = max(1, min(nwin, steps))
    return [steps // nwin + (1 if w < steps % nwin else 0) for w in range(nwin)]


def stack_headline(wl, steps, warmup, per_layer_tokens):
    """The 40-layer stack, one vt_stack_decode launch per token, consecutive
    positions from the cached context. Weights drawn on the device with the
    workload's distributions (weights N(0, sigma), gains 1 + N(0, 0.1),
    cached K/V and token inputs N(0, 1)); the stack's parity against the
    oracle is the tests' (teacher-forced on every layer, and bit for bit
    against one launch per layer)."""
    import torch

    from paper_2607_07046_amd import pack
    from paper_2607_07046_amd import voltron as vt

    t0 = time.time()
    spec = vt.vt_shard_spec_create(lib_dims(wl.dims), wl.fracs, wl.fracs, wl.device)
    dims, info = vt.vt_shard_spec_query(spec)
    H, d, nkv, nq, F, L = (dims.hidden, dims.head_dim, info.n_kv_heads, info.n_q_heads,
                           info.n_cols, wl.n_layers)
    ntok = warmup + steps + per_layer_tokens
    cap = wl.ctx + ntok
    normal = device_normal(7046 * 1000 + wl.seed_id)
    fill = lambda name, shape: (normal(shape, 0.1, 1.0) if name.startswith("g_")
                                else normal(shape, wl.weight_sigma))
    st = pack.alloc_stack(dims, info, L, fill=fill)
    kc = torch.zeros((L, nkv, cap, d), dtype=torch.float16, device="cuda")
    vc = torch.zeros_like(kc)
    kc[:, :, :wl.ctx] = normal((L, nkv, wl.ctx, d), 1.0)
    vc[:, :, :wl.ctx] = normal((L, nkv, wl.ctx, d), 1.0)
    kv = vt.vt_kv_stack(k=kc.data_ptr(), v=vc.data_ptr(), n_layers=L, capacity=cap,
                        n_kv_heads=nkv, head_dim=d, len=wl.ctx)
    xs = normal((ntok, H), 1.0)
    ws_bytes = vt.vt_workspace_size(spec, 1, cap)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
    outs = {k: torch.empty((L, H), dtype=torch.float16, device="cuda")
            for k in ("p_attn", "h", "p_ffn", "y")}
    io = vt.vt_layer_io(x=None, peer_attn=None, peer_ffn=None,
                        attn_partial=outs["p_attn"].data_ptr(), h=outs["h"].data_ptr(),
                        ffn_partial=outs["p_ffn"].data_ptr(), y=outs["y"].data_ptr())
    torch.cuda.synchronize()
    setup_s = time.time() - t0
    stream = torch.cuda.current_stream().cuda_stream

    def token(i):
        io.x = xs[i].data_ptr()
        vt.vt_stack_decode(spec, st.struct, kv, io, wl.ctx + i, ws.data_ptr(), ws_bytes, stream)

    for i in range(warmup):
        token(i)
    torch.cuda.synchronize()
    wins = windows(steps)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(len(wins) + 1)]
    i = warmup
    evs[0].record()
    for w, n in enumerate(wins):
        for _ in range(n):
            token(i)
            i += 1
        evs[w + 1].record()
    torch.cuda.synchronize()
    ms = evs[0].elapsed_time(evs[-1])
    ms_step = ms / steps
    win_ms = np.array([evs[w].elapsed_time(evs[w + 1]) / wins[w] for w in range(len(wins))])
    err = int(ws[vt.VT_WS_ERROR_WORD:vt.VT_WS_ERROR_WORD + 4].view(torch.int32).item())
    if err:
        raise SystemExit("stack: a grid barrier's bounded wait expired (error word set)")
    if not torch.isfinite(outs["y"].float()).all():
        raise SystemExit("stack: non-finite output")
    if kv.len != wl.ctx + warmup + steps:
        raise SystemExit("stack: the KV length did not advance once per token")
    tok_bytes = [algorithmic_bytes(dims, info, wl.ctx + t) * L for t in range(warmup, warmup + steps)]
    mean_bytes = sum(tok_bytes) / steps
    res = {"ms_per_step": ms_step, "win_ms": win_ms, "bytes": mean_bytes, "setup_s": setup_s,
           "dims": dims, "info": info,
           "positions": f"{wl.ctx + warmup}..{wl.ctx + warmup + steps - 1} timed "
                        f"({warmup} warm-up tokens before)"}

    if per_layer_tokens > 0:
        # the same layers, one vt_layer_decode launch per layer, continuing the positions
        kvs = [vt.vt_kv_view(k=kc[l].data_ptr(), v=vc[l].data_ptr(), capacity=cap,
                             n_kv_heads=nkv, head_dim=d, len=kv.len) for l in range(L)]
        lw = [st.layer(l) for l in range(L)]
        lio = [vt.vt_layer_io(x=None, peer_attn=None, peer_ffn=None,
                              attn_partial=outs["p_attn"][l].data_ptr(),
                              h=outs["h"][l].data_ptr(), ffn_partial=outs["p_ffn"][l].data_ptr(),
                              y=outs["y"][l].data_ptr()) for l in range(L)]
        both = vt.VT_ATTN | vt.VT_FFN
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        p0 = kv.len
        a.record()
        for t in range(per_layer_tokens):
            for l in range(L):
                lio[l].x = xs[p0 - wl.ctx + t].data_ptr() if l == 0 else outs["y"][l - 1].data_ptr()
                vt.vt_layer_decode(spec, lw[l], kvs[l], lio[l], p0 + t, both, ws.data_ptr(),
                                   ws_bytes, stream)
        b.record()
        torch.cuda.synchronize()
        pl_ms = a.elapsed_time(b) / per_layer_tokens
        pl_bytes = sum(algorithmic_bytes(dims, info, p0 + t) * L
                       for t in range(per_layer_tokens)) / per_layer_tokens
        res["per_layer"] = {
            "ms_per_token": round(pl_ms, 4), "tokens_s": round(1e3 / pl_ms, 1),
            "us_per_layer": round(pl_ms * 1e3 / L, 2),
            "hbm_GBps": round(pl_bytes / (pl_ms * 1e-3) / 1e9, 1),
            "hbm_frac": round(pl_bytes / (pl_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
            "positions": f"{p0}..{p0 + per_layer_tokens - 1}",
            "launch": f"{L} vt_layer_decode launches per token, eager"}
    del st, kc, vc
    torch.cuda.empty_cache()
    return res


def chain_section(wl, steps, warmup, emit=False):
    """A single-layer decode workload: step i decodes weight/KV copy i mod R
    (R copies, >= 768 MB in all, so the Infinity Cache cannot serve the
    weights) at the workload's position and feeds its y to step i+1 as x.
    Steps are captured in HIP graphs keyed by (first step mod the rotation
    length, count), so every window continues the rotation and the chain
    where the previous one stopped; a window holds up to about 128 steps (a
    whole number of rotations), so graph launches do not add to the step.
    ``emit``: each step also emits both partial sums quantised
    (vt_layer_decode_emit) under plans that halve the fp16 message."""
    import torch

    from paper_2607_07046_amd import pack
    from paper_2607_07046_amd import voltron as vt
    from synth.gen import LayerInputs

    spec = vt.vt_shard_spec_create(lib_dims(wl.dims), wl.fracs, wl.fracs, wl.device)
    dims, info = vt.vt_shard_spec_query(spec)
    pos = wl.ctx
    step_bytes = algorithmic_bytes(dims, info, pos)
    copies = max(2, math.ceil(MALL_DEFEAT_BYTES / step_bytes))
    H, d, nkv, cap = dims.hidden, dims.head_dim, info.n_kv_heads, pos + 1
    li = LayerInputs(wl)
    w0 = pack.pack_shard(li, dims, info)
    k, v = li.kv_context_heads(info.kv_head_begin, info.kv_head_begin + nkv)
    layers = []
    for c in range(copies):
        t = {n: x.clone() for n, x in w0.tensors.items()} if c else w0.tensors
        kc = torch.zeros((nkv, cap, d), dtype=torch.float16, device="cuda")
        vc = torch.zeros_like(kc)
        kc[:, :pos] = torch.from_numpy(k).cuda()
        vc[:, :pos] = torch.from_numpy(v).cuda()
        kvv = vt.vt_kv_view(k=kc.data_ptr(), v=vc.data_ptr(), capacity=cap, n_kv_heads=nkv,
                            head_dim=d, len=pos)
        layers.append((t, pack.struct_of(t, dims, info, w0.struct.ld_d), kc, vc, kvv))
    ws_bytes = vt.vt_workspace_size(spec, 1, cap)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
    x0 = torch.from_numpy(li.x(0)).cuda()
    bufs = [x0.clone(), torch.empty_like(x0)]
    p_attn, h, p_ffn = (torch.empty(H, dtype=torch.float16, device="cuda") for _ in range(3))
    both = vt.VT_ATTN | vt.VT_FFN
    em = None
    if emit:
        nb = H // 32
        rng = np.random.default_rng(11)
        eplan = {}
        for name in ("attn", "ffn"):
            prec, offs, total = vt.vt_qplan(rng.random(nb).astype(np.float32), nb * 64 // 2)
            eplan[name] = (torch.from_numpy(prec).cuda(), torch.from_numpy(offs).cuda(),
                          torch.zeros(max(16, total), dtype=torch.uint8, device="cuda"), total)
        em = vt.vt_emit(prec_attn=eplan["attn"][0].data_ptr(), off_attn=eplan["attn"][1].data_ptr(),
                        msg_attn=eplan["attn"][2].data_ptr(), msg_attn_bytes=eplan["attn"][3],
                        prec_ffn=eplan["ffn"][0].data_ptr(), off_ffn=eplan["ffn"][1].data_ptr(),
                        msg_ffn=eplan["ffn"][2].data_ptr(), msg_ffn_bytes=eplan["ffn"][3])

    def enqueue(i, stream):
        _, stw, _, _, kvv = layers[i % copies]
        kvv.len = pos  # every step re-decodes position `pos` of its copy
        io = vt.vt_layer_io(x=bufs[i % 2].data_ptr(), peer_attn=None, peer_ffn=None,
                            attn_partial=p_attn.data_ptr(), h=h.data_ptr(),
                            ffn_partial=p_ffn.data_ptr(), y=bufs[(i + 1) % 2].data_ptr())
        if em is not None:
            vt.vt_layer_decode_emit(spec, stw, kvv, io, pos, both, em, ws.data_ptr(), ws_bytes,
                                    stream)
        else:
            vt.vt_layer_decode(spec, stw, kvv, io, pos, both, ws.data_ptr(), ws_bytes, stream)

    group = copies * (2 if copies % 2 else 1)  # the copy and buffer pattern repeats after this
    unit = group * max(1, 128 // group)       # steps per window (whole rotations)
    graphs = {}

    def graph(start, n):
        key = (start % group, n)
        if key not in graphs:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                s = torch.cuda.current_stream().cuda_stream
                for j in range(n):
                    enqueue(start + j, s)
            graphs[key] = g
        return graphs[key]

    def plan(start, n):
        """(start, count) windows of at most ``unit`` steps covering n steps, each
        ending on a multiple of ``unit`` where it can."""
        out = []
        while n > 0:
            c = min(n, unit - start % unit)
            out.append((start, c))
            start, n = start + c, n - c
        return out

    warm = plan(0, warmup)
    timed = plan(warmup, steps)
    for s0, n in warm + timed:  # capture everything before any timing
        graph(s0, n)
    for s0, n in warm:
        graph(s0, n).replay()
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(len(timed) + 1)]
    evs[0].record()
    for wi, (s0, n) in enumerate(timed):
        graph(s0, n).replay()
        evs[wi + 1].record()
    torch.cuda.synchronize()
    ms = evs[0].elapsed_time(evs[-1])
    ms_step = ms / steps
    win = np.array([evs[i].elapsed_time(evs[i + 1]) / timed[i][1] for i in range(len(timed))])
    if int(ws[vt.VT_WS_ERROR_WORD:vt.VT_WS_ERROR_WORD + 4].view(torch.int32).item()):
        raise SystemExit(f"{wl.key}: a grid barrier's bounded wait expired (error word set)")
    last = bufs[(warmup + steps) % 2]  # the y of the last timed step
    if not torch.isfinite(last.float()).all():
        raise SystemExit(f"{wl.key}: non-finite output after the timed steps")
    gbps = step_bytes / (ms_step * 1e-3) / 1e9
    out = {
        "workload": wl.key,
        "shape": f"hidden {H}, {wl.dims.n_heads}x{d} heads, {wl.dims.n_kv_heads} KV heads, "
                 f"FFN {wl.dims.ffn}; device {wl.device} of {list(wl.fracs)}: "
                 f"{info.n_q_heads} q / {info.n_kv_heads} kv heads, {info.n_cols} FFN cols",
        "pos": pos, "steps": steps, "warmup": warmup, "weight_copies": copies,
        "ms_per_step": round(ms_step, 6),
        "ms_per_step_windows": {"windows": len(timed),
                                "p10": round(float(np.percentile(win, 10)), 6),
                                "median": round(float(np.median(win)), 6),
                                "p90": round(float(np.percentile(win, 90)), 6)},
        "tokens_s": round(1e3 / ms_step, 1),
        "algorithmic_bytes_per_step": step_bytes,
        "hbm_GBps": round(gbps, 1),
        "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4),
        "roofline": roofline(step_bytes, ms_step, "decode_kernel<0, 4, 0, false, false>", wl.key),
        "launch": "persistent + hipgraph (windows keyed by rotation phase)",
    }
    if emit:
        out["emit"] = {name: {"message_bytes": eplan[name][3], "fp16_bytes": 2 * H}
                       for name in ("attn", "ffn")}
        out["roofline"] = None  # the roofline block belongs to the plain step
    res = (out, spec, dims, info, enqueue, copies, w0)
    return res


def main():
    args = parse()
    if args.copy_calibration:
        return copy_calibration(args.copy_calibration)
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only: the cross-device "
                                   "reduction is replaced by returning the shard's partial "
                                   "sums, so --gpus must be 1"}))
        sys.exit(2)
    import torch

    from synth import get

    wl = get(args.config)
    if wl.chunk:
        raise SystemExit("bench.py times decode workloads; the prefill chunk is reported "
                         "by its own section")
    torch.cuda.init()
    out = {"metric": METRIC}
    if wl.n_layers > 1:
        r = stack_headline(wl, args.steps, args.warmup, args.per_layer_tokens)
        dims, info = r["dims"], r["info"]
        ms_step = r["ms_per_step"]
        out.update({
            "value": round(1e3 / ms_step, 2), "unit": "tokens/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 6),
            "ms_per_step_windows": {"windows": len(r["win_ms"]),
                                    "p10": round(float(np.percentile(r["win_ms"], 10)), 6),
                                    "median": round(float(np.median(r["win_ms"])), 6),
                                    "p90": round(float(np.percentile(r["win_ms"], 90)), 6)},
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f16",
            "data": "synthetic",
            "config": {
                "workload": wl.key,
                "layer": f"{wl.n_layers} layers, hidden {dims.hidden}, {wl.dims.n_heads}x"
                         f"{dims.head_dim} heads, {wl.dims.n_kv_heads} KV heads, FFN {wl.dims.ffn}",
                "shard": f"device {wl.device} of fractions {list(wl.fracs)}: {info.n_q_heads} q "
                         f"heads, {info.n_kv_heads} kv heads, {info.n_cols} FFN cols",
                "positions": r["positions"],
                "launch": "one vt_stack_decode launch per token (all 40 layers), eager",
            },
            "hbm_GBps": round(r["bytes"] / (ms_step * 1e-3) / 1e9, 1),
            "hbm_frac_of_peak": round(r["bytes"] / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
            "algorithmic_bytes_per_step": int(r["bytes"]),
            "roofline": roofline(r["bytes"], ms_step, "decode_kernel<0, 4, 0, true, false> (40 layers per launch)",
                                 wl.key),
            "setup_s": round(r["setup_s"], 1),
        })
        if "per_layer" in r:
            out["per_layer_launches"] = r["per_layer"]
        sections = ("7b", "70b_gqa")
    else:
        sec, *_ = chain_section(wl, args.steps, args.warmup)
        out.update({
            "value": sec["tokens_s"], "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": sec["ms_per_step"],
            "ms_per_step_windows": sec["ms_per_step_windows"], "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "f16", "data": "synthetic",
            "config": {"workload": wl.key, "shard": sec["shape"], "pos": sec["pos"],
                       "weight_copies": sec["weight_copies"], "launch": sec["launch"]},
            "hbm_GBps": sec["hbm_GBps"], "hbm_frac_of_peak": sec["hbm_frac"],
            "algorithmic_bytes_per_step": sec["algorithmic_bytes_per_step"],
            "roofline": sec["roofline"]})
        sections = tuple(k for k in ("7b", "70b_gqa") if k != wl.key)
    c2 = None
    if args.decode_steps > 0:
        for key in sections:
            sec, spec2, dims2, info2, enq, copies, w0 = chain_section(
                get(key), args.decode_steps, max(1, args.decode_steps // 10))
            out["decode_" + key] = sec
            if key == "7b":
                c2 = (spec2, dims2, info2, enq, copies, w0)
            else:
                del enq, w0
            torch.cuda.empty_cache()
        if args.comm_steps > 0:
            # the 7B step emitting both partial sums quantised from its epilogues
            sec, *_ = chain_section(get("7b"), args.decode_steps, max(1, args.decode_steps // 10),
                                    emit=True)
            out["decode_7b_emit"] = {k: sec[k] for k in ("ms_per_step", "tokens_s", "emit", "launch")}
            out["decode_7b_emit"]["us_over_plain_step"] = round(
                (sec["ms_per_step"] - out["decode_7b"]["ms_per_step"]) * 1e3, 2)
    if args.prefill_steps > 0:
        out["prefill"] = prefill_section(args.prefill_steps, max(1, args.prefill_steps // 10),
                                         tokens=args.prefill_tokens)
    if args.comm_steps > 0:
        out["comm"] = comm_section(args.comm_steps)
    if c2 is not None and args.repack_reps > 0:
        spec2, dims2, info2, enq, copies, w0 = c2
        out["repack"] = repack_section(spec2, dims2, info2, get("7b"), args.repack_reps, enq, copies)
    if c2 is not None and args.quant_steps > 0:
        spec2, dims2, info2, enq, copies, w0 = c2
        out["quant"] = quant_section(spec2, dims2, info2, get("7b"), args.quant_steps,
                                     max(1, args.quant_steps // 10), w0)
    c2 = None
    torch.cuda.empty_cache()
    if args.moe_steps > 0:
        out["moe"] = moe_section(args.moe_steps, max(1, args.moe_steps // 10))
    if args.fraction_sweep:
        out["fraction_sweep"] = fraction_sweep_section()
    if args.cpu_seconds > 0:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def repack_section(spec, dims, info, wl, reps, enqueue, copies):
    """Elastic re-partition: vt_shard_pack of the decode_7b section's shard
    (7B-shaped layer, 30% shard) out of the whole layer's device weights (its
    bytes read and written), alone and
    while decode steps run on the default stream; the decode step time with
    and without a pack running beside it on a second stream (both at the
    default priority)."""
    import torch

    from paper_2607_07046_amd import pack
    from paper_2607_07046_amd import voltron as vt
    from synth.gen import LayerInputs

    full = pack.upload_full(LayerInputs(wl), dims)
    out = pack.alloc_shard(dims, info)
    shard_bytes = sum(t.numel() * 2 for t in out.tensors.values())
    side = torch.cuda.Stream()
    main = torch.cuda.current_stream()
    torch.cuda.synchronize()

    def packs(n):
        for _ in range(n):
            vt.vt_shard_pack(spec, full.struct, out.struct, side.cuda_stream)

    def decodes(n):
        for i in range(n):
            enqueue(i, main.cuda_stream)

    packs(2)
    decodes(2 * copies)
    torch.cuda.synchronize()
    ev = lambda: torch.cuda.Event(enable_timing=True)
    # pack alone
    a, b = ev(), ev()
    a.record(side)
    packs(reps)
    b.record(side)
    torch.cuda.synchronize()
    pack_us = a.elapsed_time(b) * 1e3 / reps
    # decode alone, eager launches (as in the concurrent case)
    nd = max(copies * 4, 40)
    a, b = ev(), ev()
    a.record(main)
    decodes(nd)
    b.record(main)
    torch.cuda.synchronize()
    dec_us = a.elapsed_time(b) * 1e3 / nd
    # both: the packs on the second stream, decodes on the default one
    a, b, c, e = ev(), ev(), ev(), ev()
    a.record(side)
    c.record(main)
    packs(reps)
    decodes(nd)
    b.record(side)
    e.record(main)
    torch.cuda.synchronize()
    pack_cc = a.elapsed_time(b) * 1e3 / reps
    dec_cc = c.elapsed_time(e) * 1e3 / nd
    moved = 2 * shard_bytes
    return {"shard_bytes": shard_bytes, "pack_us": round(pack_us, 2),
            "pack_GBps": round(moved / (pack_us * 1e-6) / 1e9, 1),
            "pack_hbm_frac": round(moved / (pack_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
            "decode_us_alone": round(dec_us, 2), "decode_us_with_pack": round(dec_cc, 2),
            "pack_us_with_decode": round(pack_cc, 2), "packs": reps, "decode_steps": nd,
            "note": "eager launches; bytes = the shard's weights read from the whole layer and "
                    "written to its own buffers"}


def quant_bytes(dims, info, pos, prec):
    """Bytes a decode step over block-quantised weights moves: each matrix's
    codes (32 or 16 bytes per block of 32 columns) and fp16 scales, the K/V
    read and written, the gains, x and the four fp16 outputs."""
    H, d = dims.hidden, dims.head_dim
    qd, kd, F = info.n_q_heads * d, info.n_kv_heads * d, info.n_cols
    per_block = (32 if prec == 1 else 16) + 2
    nb = lambda k: (k + 31) // 32
    weights = per_block * (qd * nb(H) + 2 * kd * nb(H) + H * nb(qd) + 2 * F * nb(H) + H * nb(F))
    span = min(pos + 1, dims.window) if dims.window > 0 else pos + 1
    return weights + 4 * kd * span + 2 * H * (2 + 1 + 4)


def quant_section(spec, dims, info, wl, steps, warmup, fp16_weights, eager=False):
    """Decode over the same shard with INT8 and INT4 block-quantised weights
    (vt_layer_decode_q). The codes are made once by vt_quantize_rows from
    the first fp16 copy and cloned into enough distinct copies (>= 768 MB)
    to keep the Infinity Cache from serving them; steps chain y -> x."""
    import torch

    from paper_2607_07046_amd import pack
    from paper_2607_07046_amd import voltron as vt
    from synth.gen import LayerInputs

    pos, H, d, nkv = wl.ctx, dims.hidden, dims.head_dim, info.n_kv_heads
    cap = pos + 1
    li = LayerInputs(wl)
    k, v = li.kv_context_heads(info.kv_head_begin, info.kv_head_begin + nkv)
    ws_bytes = vt.vt_workspace_size(spec, 1, cap)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
    x0 = torch.from_numpy(li.x(0)).cuda()
    res = {}
    for name, prec in (("int8", vt.VT_W_INT8), ("int4", vt.VT_W_INT4)):
        step_bytes = quant_bytes(dims, info, pos, prec)
        copies = max(1, math.ceil(MALL_DEFEAT_BYTES / step_bytes))
        q0 = pack.quantize_shard(fp16_weights, dims, info, prec)
        layers = []
        for c in range(copies):
            qc = pack.clone_qshard(q0) if c else q0
            st = qc.struct
            kc = torch.zeros((nkv, cap, d), dtype=torch.float16, device="cuda")
            vc = torch.zeros_like(kc)
            kc[:, :pos] = torch.from_numpy(k).cuda()
            vc[:, :pos] = torch.from_numpy(v).cuda()
            kv = vt.vt_kv_view(k=kc.data_ptr(), v=vc.data_ptr(), capacity=cap, n_kv_heads=nkv,
                               head_dim=d, len=pos)
            layers.append((qc, st, kc, vc, kv))
        bufs = [x0.clone(), torch.empty_like(x0)]
        p_attn, h, p_ffn = (torch.empty(H, dtype=torch.float16, device="cuda") for _ in range(3))

        def enqueue(i, stream):
            _, st, _, _, kv = layers[i % copies]
            kv.len = pos
            io = vt.vt_layer_io(x=bufs[i % 2].data_ptr(), peer_attn=None, peer_ffn=None,
                                attn_partial=p_attn.data_ptr(), h=h.data_ptr(),
                                ffn_partial=p_ffn.data_ptr(), y=bufs[(i + 1) % 2].data_ptr())
            vt.vt_layer_decode_q(spec, st, kv, io, pos, vt.VT_ATTN | vt.VT_FFN, ws.data_ptr(),
                                 ws_bytes, stream)

        group = copies * (2 if copies % 2 else 1)
        per_graph = group * max(1, 64 // group)
        g = None
        if not eager:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for i in range(per_graph):
                    enqueue(i, torch.cuda.current_stream().cuda_stream)

        def run(n):
            if g is None:
                for i in range(n):
                    enqueue(i, torch.cuda.current_stream().cuda_stream)
                return n
            reps = max(1, n // per_graph)
            for _ in range(reps):
                g.replay()
            return reps * per_graph

        run(warmup)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        n = run(steps)
        e1.record()
        torch.cuda.synchronize()
        ms_step = e0.elapsed_time(e1) / n
        if not torch.isfinite(bufs[0].float()).all():
            raise SystemExit(f"non-finite output of the {name} decode steps")
        gbps = step_bytes / (ms_step * 1e-3) / 1e9
        res[name] = {"ms_per_step": round(ms_step, 6), "tokens_s": round(1e3 / ms_step, 1),
                     "bytes_per_step": step_bytes, "hbm_GBps": round(gbps, 1),
                     "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4), "weight_copies": copies,
                     "steps": n}
        del layers, q0
    res["note"] = ("same shard and position as the decode_7b section (7B-shaped layer, 30% shard, "
                   "pos 1024); bytes = codes + fp16 block scales + K/V + vectors; the format is the "
                   "library's own 32-column block format")
    return res


def moe_bytes(wl, n_cols):
    """Algorithmic HBM bytes of one token through an MoE FFN shard: the
    router, the selected experts' gate/up rows and down columns of the
    shard, the gain, h in, the partial and y out."""
    H, E, k = wl.hidden, wl.n_experts, wl.top_k
    return 2 * (E * H + k * 3 * n_cols * H + 4 * H)


def _shard_step_us(H, nh, nkv, d, F, frac, pos, sigma):
    """Time of one fused decode step of device 0's share (fraction ``frac``
    of heads and FFN columns; the whole layer at 1.0) of a Llama-shaped
    layer at position ``pos``: weights drawn on the device (seeded), enough
    copies for 768 MB rotated, HIP-graph replays. Returns (info, bytes, us)."""
    import torch

    from paper_2607_07046_amd import pack
    from paper_2607_07046_amd import voltron as vt

    dims = vt.vt_layer_dims(hidden=H, n_heads=nh, n_kv_heads=nkv, head_dim=d, ffn=F, rms_eps=1e-5,
                            rope_base=10000.0, window=0)
    fr = [1.0] if frac >= 1.0 else [frac, 1.0 - frac]
    spec = vt.vt_shard_spec_create(dims, fr, fr, 0)
    dims, info = vt.vt_shard_spec_query(spec)
    nq, nk, nc = info.n_q_heads, info.n_kv_heads, info.n_cols
    step = algorithmic_bytes(dims, info, pos)
    copies = max(2, math.ceil(MALL_DEFEAT_BYTES / step))
    gen = torch.Generator(device="cuda")
    gen.manual_seed(7046)

    def normal(shape, sd, mean=0.0):
        t = torch.empty(shape, dtype=torch.float32, device="cuda")
        t.normal_(mean, sd, generator=gen)
        return t.half()

    ld_d = max(8, pack.round_up(nc, 8))
    cap = pos + 1
    layers = []
    for _ in range(copies):
        t = {"g_attn": normal((H,), 0.1, 1.0), "g_ffn": normal((H,), 0.1, 1.0),
             "wq": normal((nq * d, H), sigma), "wk": normal((nk * d, H), sigma),
             "wv": normal((nk * d, H), sigma), "wo": normal((H, nq * d), sigma),
             "wg": normal((nc, H), sigma), "wu": normal((nc, H), sigma)}
        wdn = torch.zeros((H, ld_d), dtype=torch.float16, device="cuda")
        wdn[:, :nc] = normal((H, nc), sigma)
        t["wd"] = wdn
        kc, vc = normal((nk, cap, d), 1.0), normal((nk, cap, d), 1.0)
        kv = vt.vt_kv_view(k=kc.data_ptr(), v=vc.data_ptr(), capacity=cap, n_kv_heads=nk,
                           head_dim=d, len=pos)
        layers.append((t, pack.struct_of(t, dims, info, ld_d), kc, vc, kv))
    ws_bytes = vt.vt_workspace_size(spec, 1, cap)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
    bufs = [normal((H,), 1.0), torch.empty(H, dtype=torch.float16, device="cuda")]
    pa, h, pf = (torch.empty(H, dtype=torch.float16, device="cuda") for _ in range(3))

    def enqueue(i, stream):
        _, st, _, _, kv = layers[i % copies]
        kv.len = pos
        io = vt.vt_layer_io(x=bufs[i % 2].data_ptr(), peer_attn=None, peer_ffn=None,
                            attn_partial=pa.data_ptr(), h=h.data_ptr(), ffn_partial=pf.data_ptr(),
                            y=bufs[(i + 1) % 2].data_ptr())
        vt.vt_layer_decode(spec, st, kv, io, pos, vt.VT_ATTN | vt.VT_FFN, ws.data_ptr(), ws_bytes,
                           stream)

    n = copies * 2 * max(1, 64 // (copies * 2))
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        s = torch.cuda.current_stream().cuda_stream
        for i in range(n):
            enqueue(i, s)
    for _ in range(3):
        graph.replay()
    torch.cuda.synchronize()
    reps = max(3, 400 // n)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(reps):
        graph.replay()
    end.record()
    torch.cuda.synchronize()
    us = start.elapsed_time(end) * 1e3 / (reps * n)
    if not torch.isfinite(bufs[0].float()).all():
        raise SystemExit("fraction sweep: non-finite output")
    del layers, graph
    torch.cuda.empty_cache()
    return info, step, us


def fraction_sweep_section():
    """The fused decode step of the 7B-shaped layer (position 1024) and the
    70B-shaped GQA layer (position 4096) at shard fractions from 10% to the
    whole layer, and a least-squares line time = fixed + bytes / bandwidth
    per layer shape: the bandwidth is what the weight streaming reaches, the
    fixed part is the step's dependency chain (barriers, staging,
    attention), which does not grow with the shard."""
    out = {}
    for name, shape, fracs in (("7b", (4096, 32, 32, 128, 11008, 1024, 0.02), (0.1, 0.2, 0.3, 0.5, 0.75, 1.0)),
                               ("70b_gqa", (8192, 64, 8, 128, 28672, 4096, 0.015), (0.125, 0.25, 0.5, 1.0))):
        H, nh, nkv, d, F, pos, sigma = shape
        rows = []
        for f in fracs:
            info, step, us = _shard_step_us(H, nh, nkv, d, F, f, pos, sigma)
            rows.append({"fraction": f, "q_heads": info.n_q_heads, "kv_heads": info.n_kv_heads,
                         "cols": info.n_cols, "bytes": int(step), "us_per_step": round(us, 2),
                         "GBps": round(step / us / 1e3, 1),
                         "hbm_frac": round(step / us / 1e3 / HBM_PEAK_GBPS, 4)})
        xb = np.array([r["bytes"] for r in rows], np.float64)
        yt = np.array([r["us_per_step"] for r in rows], np.float64)
        slope, icept = np.polyfit(xb, yt, 1)
        out[name] = {"rows": rows, "fit_fixed_us": round(float(icept), 2),
                     "fit_stream_GBps": round(float(1e-3 / slope), 1),
                     "fit_stream_frac": round(float(1e-3 / slope) / HBM_PEAK_GBPS, 4)}
    return out


def moe_section(steps, warmup, eager=False):
    """Batch-1 decode through the MoE FFN shard (device 0 of the MoE
    workload) with vt_moe_ffn_decode: 16 distinct tokens (each selects its
    own experts) over enough weight copies (>= 768 MB) to keep the Infinity
    Cache from serving them."""
    import torch

    from paper_2607_07046_amd import pack
    from paper_2607_07046_amd import voltron as vt
    from synth.configs import MOE_WORKLOADS
    from synth.gen import MoEInputs

    wl = MOE_WORKLOADS["moe"]
    mi = MoEInputs(wl)
    dims = vt.vt_layer_dims(hidden=wl.hidden, n_heads=1, n_kv_heads=1, head_dim=64,
                            ffn=wl.expert_ffn, rms_eps=wl.rms_eps, rope_base=1e4, window=0)
    spec = vt.vt_shard_spec_create(dims, wl.fracs, wl.fracs, wl.device)
    _, info = vt.vt_shard_spec_query(spec)
    nc = info.n_cols
    shard_bytes = 2 * wl.n_experts * 3 * nc * wl.hidden
    copies = max(1, math.ceil(MALL_DEFEAT_BYTES / shard_bytes))
    w0 = pack.pack_moe_shard(mi, info.col_begin, nc)
    shards = [w0]
    for _ in range(1, copies):
        t = {k: v.clone() for k, v in w0.tensors.items()}
        p = lambda x: x.data_ptr()
        shards.append(pack.MoEShardDev(t, vt.vt_moe_weights(
            g_ffn=p(t["g_ffn"]), wr=p(t["wr"]), ld_r=w0.struct.ld_r, wg=p(t["wg"]),
            ld_g=w0.struct.ld_g, wu=p(t["wu"]), ld_u=w0.struct.ld_u, wd=p(t["wd"]),
            ld_d=w0.struct.ld_d)))
    ntok = 16
    hs = torch.from_numpy(np.stack([mi.h(t) for t in range(ntok)])).cuda()
    H, k = wl.hidden, wl.top_k
    p_ffn, y = (torch.empty(H, dtype=torch.float16, device="cuda") for _ in range(2))
    sel = torch.empty(k, dtype=torch.int32, device="cuda")
    ws_bytes = vt.vt_moe_workspace_size(spec, wl.n_experts, k)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")

    def enqueue(i, stream):
        io = vt.vt_layer_io(x=None, peer_attn=None, peer_ffn=None, attn_partial=None,
                            h=hs[i % ntok].data_ptr(), ffn_partial=p_ffn.data_ptr(),
                            y=y.data_ptr())
        vt.vt_moe_ffn_decode(spec, shards[i % copies].struct, wl.n_experts, k, io,
                             sel.data_ptr(), None, ws.data_ptr(), ws_bytes, stream)

    per_graph = ntok * copies
    g = None
    if not eager:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(per_graph):
                enqueue(i, torch.cuda.current_stream().cuda_stream)

    def run(n):
        if g is None:
            for i in range(n):
                enqueue(i, torch.cuda.current_stream().cuda_stream)
            return n
        reps = max(1, n // per_graph)
        for _ in range(reps):
            g.replay()
        return reps * per_graph

    run(warmup)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    n = run(steps)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / n
    if not torch.isfinite(p_ffn.float()).all():
        raise SystemExit("non-finite output of the MoE decode steps")
    if ws[8192:8196].view(torch.int32).item() != 0:
        raise SystemExit("a grid barrier's bounded wait expired during the MoE steps")
    b = moe_bytes(wl, nc)
    gbps = b / (ms * 1e-3) / 1e9
    return {"workload": wl.title, "us_per_token": round(ms * 1e3, 3),
            "tokens_s": round(1e3 / ms, 1), "bytes_per_token": b, "hbm_GBps": round(gbps, 1),
            "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4), "weight_copies": copies, "steps": n,
            "launch": "one persistent kernel: router | route + gate/up | down"}


def comm_section(steps):
    """Transmission scaling of partial sums (vt_partial_encode /
    vt_partial_decode_add) for one decode partial (hidden 4096) and one
    256-token prefill partial, under a plan that halves the message
    (importance drawn per block, budget = half the FP16 size). 50 calls are
    captured per HIP graph; about ``steps`` calls are timed."""
    import numpy as np
    import torch

    from paper_2607_07046_amd import voltron as vt
    from synth.gen import vector

    res = {}
    for name, n in (("decode_partial_4096", 4096), ("prefill_partial_256x4096", 256 * 4096)):
        nb = n // 32
        rng = np.random.default_rng(11)
        prec, offs, total = vt.vt_qplan(rng.random(nb).astype(np.float32), nb * 64 // 2)
        p = torch.from_numpy(vector(21, n, 2.0)).cuda()
        base = torch.from_numpy(vector(22, n, 2.0)).cuda()
        out = torch.empty_like(base)
        prd, ofd = torch.from_numpy(prec).cuda(), torch.from_numpy(offs).cuda()
        msg = torch.zeros(max(16, total), dtype=torch.uint8, device="cuda")
        calls = {
            "encode": lambda s: vt.vt_partial_encode(p.data_ptr(), n, prd.data_ptr(), ofd.data_ptr(),
                                                     msg.data_ptr(), total, s),
            "decode_add": lambda s: vt.vt_partial_decode_add(msg.data_ptr(), total, n,
                                                             prd.data_ptr(), ofd.data_ptr(),
                                                             base.data_ptr(), out.data_ptr(), s),
        }
        bytes_moved = {"encode": 2 * n + total + 5 * nb, "decode_add": total + 4 * n + 5 * nb}
        entry = {"n": n, "message_bytes": total, "fp16_bytes": 2 * n,
                 "levels": {k: int((prec == v).sum()) for k, v in
                            (("fp16", 0), ("int8", 1), ("int4", 2), ("pruned", 3))}}
        per_graph = 50  # calls captured per graph, so host launch cost does not dominate
        reps = max(1, steps // per_graph)
        for cname, fn in calls.items():
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for _ in range(per_graph):
                    fn(torch.cuda.current_stream().cuda_stream)
            g.replay()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                g.replay()
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / (reps * per_graph)
            entry[cname] = {"us_per_call": round(us, 3),
                            "GBps": round(bytes_moved[cname] / (us * 1e-6) / 1e9, 1),
                            "hbm_frac": round(bytes_moved[cname] / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)}
        res[name] = entry
    res["note"] = ("bytes = fp16 input + message + plan for encode; message + plan + fp16 base "
                   "and output for decode_add; the 4096-value case is launch-bound")
    return res


def prefill_flops(dims, info, T, pos0):
    """Algorithmic flops of one prefill chunk: the five projection GEMMs and
    causal attention (Q K^T and P V over keys 0..pos0+t for token t)."""
    H, d = dims.hidden, dims.head_dim
    nq, nkv, F = info.n_q_heads, info.n_kv_heads, info.n_cols
    gemm = 2 * T * H * ((nq + 2 * nkv) * d + nq * d + 3 * F)
    keys = T * pos0 + T * (T + 1) // 2
    return gemm, 4 * d * nq * keys


def prefill_bytes(dims, info, T, pos0):
    """Bytes a prefill chunk must move: the shard weights once, the cached
    K/V read and the chunk's K/V written, gains, X in and four [T][H]
    outputs."""
    H, d = dims.hidden, dims.head_dim
    nq, nkv, F = info.n_q_heads, info.n_kv_heads, info.n_cols
    weights = 2 * ((nq + 2 * nkv) * d * H + H * nq * d + 3 * F * H)
    kv = 4 * nkv * d * (pos0 + T)
    return weights + kv + 2 * H * 2 + 2 * T * H * 5


def prefill_section(steps, warmup, eager=False, tokens=0):
    """Prefill chunk of 256 tokens (or ``tokens``) at positions 768.. through
    the 50% shard of the 7B-shaped layer (rotated weight/KV copies, >= 768
    MB), timed over ``steps`` chunks captured in HIP graphs."""
    import torch

    from paper_2607_07046_amd import pack
    from paper_2607_07046_amd import voltron as vt
    from synth import get
    from synth.gen import LayerInputs

    wl = get("7b_prefill")
    dev = torch.device("cuda:0")
    dims = vt.vt_layer_dims(hidden=wl.dims.hidden, n_heads=wl.dims.n_heads,
                            n_kv_heads=wl.dims.n_kv_heads, head_dim=wl.dims.head_dim,
                            ffn=wl.dims.ffn, rms_eps=wl.dims.rms_eps,
                            rope_base=wl.dims.rope_base, window=wl.dims.window)
    spec = vt.vt_shard_spec_create(dims, wl.fracs, wl.fracs, wl.device)
    dims, info = vt.vt_shard_spec_query(spec)
    T, pos0 = (tokens or wl.chunk), wl.ctx
    H, d, nkv, cap = dims.hidden, dims.head_dim, info.n_kv_heads, pos0 + T
    gemm_flops, attn_flops = prefill_flops(dims, info, T, pos0)
    nbytes = prefill_bytes(dims, info, T, pos0)
    copies = max(1, math.ceil(MALL_DEFEAT_BYTES / nbytes))
    layers = []
    for c in range(copies):
        li = LayerInputs(wl, layer=c)
        w = pack.pack_shard(li, dims, info, dev)
        kc = torch.zeros((nkv, cap, d), dtype=torch.float16, device=dev)
        vc = torch.zeros_like(kc)
        k, v = li.kv_context_heads(info.kv_head_begin, info.kv_head_begin + nkv)
        kc[:, :pos0] = torch.from_numpy(k).to(dev)
        vc[:, :pos0] = torch.from_numpy(v).to(dev)
        kv = vt.vt_kv_view(k=kc.data_ptr(), v=vc.data_ptr(), capacity=cap, n_kv_heads=nkv,
                           head_dim=d, len=pos0)
        layers.append((w, kc, vc, kv))
    X = torch.from_numpy(LayerInputs(wl).x_chunk(T)).to(dev)
    outs = [torch.empty((T, H), dtype=torch.float16, device=dev) for _ in range(4)]
    ws_bytes = vt.vt_workspace_size(spec, T, cap)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device=dev)
    io = vt.vt_layer_io(x=X.data_ptr(), peer_attn=None, peer_ffn=None,
                        attn_partial=outs[0].data_ptr(), h=outs[1].data_ptr(),
                        ffn_partial=outs[2].data_ptr(), y=outs[3].data_ptr())

    def enqueue(i, stream):
        w, _, _, kv = layers[i % copies]
        kv.len = pos0  # every chunk re-runs positions pos0.. of its copy
        vt.vt_layer_prefill_chunk(spec, w.struct, kv, io, T, pos0, vt.VT_ATTN | vt.VT_FFN,
                                  ws.data_ptr(), ws_bytes, stream)

    per_graph = copies * 4
    reps = max(1, steps // per_graph)
    if eager:
        def run_reps(k):
            for _ in range(k):
                for i in range(per_graph):
                    enqueue(i, torch.cuda.current_stream().cuda_stream)
    else:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            s = torch.cuda.current_stream().cuda_stream
            for i in range(per_graph):
                enqueue(i, s)

        def run_reps(k):
            for _ in range(k):
                g.replay()
    run_reps(max(1, warmup // per_graph))
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    run_reps(reps)
    end.record()
    torch.cuda.synchronize()
    n = reps * per_graph
    ms = start.elapsed_time(end) / n
    if not torch.isfinite(outs[3].float()).all():
        raise SystemExit("non-finite prefill output")
    flops = gemm_flops + attn_flops
    vendor = vendor_gemm_reference(T, [((info.n_q_heads + 2 * nkv) * d, H), (H, info.n_q_heads * d),
                                       (2 * info.n_cols, H), (H, info.n_cols)], steps)
    return {
        "workload": wl.key,
        "shape": f"{T} tokens at positions {pos0}..{pos0 + T - 1}, {info.n_q_heads} q / "
                 f"{nkv} kv heads, {info.n_cols} FFN cols, hidden {H}",
        "chunks": n,
        "weight_copies": copies,
        "ms_per_chunk": round(ms, 6),
        "tokens_s": round(T / (ms * 1e-3), 1),
        "gflop_per_chunk": round(flops / 1e9, 3),
        "gemm_gflop": round(gemm_flops / 1e9, 3),
        "attention_gflop": round(attn_flops / 1e9, 3),
        "tflops": round(flops / (ms * 1e-3) / 1e12, 2),
        "mfma_peak_tflops": MFMA_F16_PEAK_TFLOPS,
        "mfma_frac": round(flops / (ms * 1e-3) / 1e12 / MFMA_F16_PEAK_TFLOPS, 4),
        "algorithmic_bytes": nbytes,
        "hbm_GBps": round(nbytes / (ms * 1e-3) / 1e9, 1),
        "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
        "bound_us": round(max(flops / (MFMA_F16_PEAK_TFLOPS * 1e12),
                              nbytes / (HBM_PEAK_GBPS * 1e9)) * 1e6, 2),
        "launch": "6 kernels per chunk, " + ("eager" if eager else "hipgraph"),
        "vendor_gemm": vendor,
    }


def vendor_gemm_reference(M, shapes, steps):
    """For scale only: the vendor fp16 GEMM (torch.matmul, i.e. hipBLASLt)
    on the chunk's four projection shapes (M tokens x N outputs x K, weights
    [N][K] row-major as the shard stores them), plain products without the
    epilogues, rotated weight copies past the memory-side cache."""
    import torch

    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev).manual_seed(7)
    wbytes = sum(2 * n * k for n, k in shapes)
    copies = max(1, math.ceil(MALL_DEFEAT_BYTES / wbytes))
    names = ("qkv", "o", "gate_up", "down")
    acts = [torch.randn((M, k), generator=gen, device=dev, dtype=torch.float16) for _, k in shapes]
    ws = [[torch.randn((n, k), generator=gen, device=dev, dtype=torch.float16) * 0.02
           for n, k in shapes] for _ in range(copies)]
    outs = [torch.empty((M, n), device=dev, dtype=torch.float16) for n, _ in shapes]
    reps = max(copies, steps // 4)
    per = {}
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for j, name in enumerate(names):
        for i in range(copies):
            torch.matmul(acts[j], ws[i][j].t(), out=outs[j])
        torch.cuda.synchronize()
        ev[0].record()
        for i in range(reps):
            torch.matmul(acts[j], ws[i % copies][j].t(), out=outs[j])
        ev[1].record()
        torch.cuda.synchronize()
        per[name] = round(ev[0].elapsed_time(ev[1]) * 1e3 / reps, 2)
    del ws
    return {"what": "torch.matmul (hipBLASLt) fp16, the four GEMM shapes, no epilogues",
            "us_per_gemm": per, "us_total": round(sum(per.values()), 2)}


def cpu_baseline(wl, budget_s):
    """The fp64 oracle, as it stands, on the host cores: decode steps of the
    workload's shard (for a stack: layers 0 and 1 in turn) at its first
    decode position, inputs drawn per token, until the budget is spent;
    scaled to the headline's unit (a stack token is n_layers layer steps)."""
    import oracle
    from synth.gen import LayerInputs
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = 1
    d = wl.dims
    dd = d.head_dim
    r = oracle.shard_ranges(d.n_heads, d.n_kv_heads, d.ffn, wl.fracs, wl.fracs, wl.device)
    layers = []
    for layer in range(min(2, wl.n_layers)):
        li = LayerInputs(wl, layer=layer)
        w = oracle.ShardWeights(
            g_attn=li.g_attn(), wq=li.rows("wq", r.q_head_begin * dd,
                                           (r.q_head_begin + r.n_q_heads) * dd),
            wk=li.rows("wk", r.kv_head_begin * dd, (r.kv_head_begin + r.n_kv_heads) * dd),
            wv=li.rows("wv", r.kv_head_begin * dd, (r.kv_head_begin + r.n_kv_heads) * dd),
            wo=li.cols("wo", r.q_head_begin * dd, (r.q_head_begin + r.n_q_heads) * dd),
            g_ffn=li.g_ffn(), wg=li.rows("wg", r.col_begin, r.col_begin + r.n_cols),
            wu=li.rows("wu", r.col_begin, r.col_begin + r.n_cols),
            wd=li.cols("wd", r.col_begin, r.col_begin + r.n_cols))
        kc, vc = li.kv_context_heads(r.kv_head_begin, r.kv_head_begin + r.n_kv_heads)
        layers.append((li, w, kc, vc))
    n = 0
    t0 = time.perf_counter()
    while True:
        li, w, kc, vc = layers[n % len(layers)]
        oracle.decode(w, r.n_q_heads, r.n_kv_heads, dd, d.rms_eps, d.rope_base, li.x(n), kc, vc,
                      wl.ctx, window=d.window)
        n += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    per_step = el / n
    per_token = per_step * wl.n_layers
    what = (f"{n} fp64 oracle layer decodes (layers 0 and 1 in turn) of the {wl.key} shard at "
            f"position {wl.ctx}, inputs drawn per token, {el:.1f} s; a token is "
            f"{wl.n_layers} layer decodes" if wl.n_layers > 1 else
            f"{n} fp64 oracle decode steps of the {wl.key} shard at position {wl.ctx}, inputs "
            f"drawn per token; {el:.1f} s")
    return {"value": round(1.0 / per_token, 4), "unit": "tokens/s", "cores": threads,
            "kind": "oracle", "sample": what, "host_cpus": len(os.sched_getaffinity(0))}


if __name__ == "__main__":
    main()
