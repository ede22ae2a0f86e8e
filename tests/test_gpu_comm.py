"""GPU parity of the partial-sum transmission scaling (paper Sec. 4.3.2):
vt_partial_encode bit-exact against the oracle's message on seeded and
edge-case fp16 vectors for every precision mix, vt_partial_decode_add
bit-exact against the fp32-step definition, and a real decode step's
attention partial sent at INT8/INT4 and received within the quantisation
bound of the fp64 oracle's partial.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import comm as C
from paper_2607_07046_amd import voltron as vt
from synth.gen import LayerInputs, vector
from tests.common import oracle_decode, oracle_ranges, tiny_workload
from tests.gpu_common import GpuShard

pytestmark = pytest.mark.gpu


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.cuda() if dtype is None else t.to(dtype).cuda()


def run_encode(p16, prec, offs, total, fill=0xA5):
    n = p16.shape[0]
    pd = dev(p16.view(np.int16)).view(torch.float16)
    prd, ofd = dev(prec.astype(np.uint8)), dev(offs.astype(np.int32))
    cap = max(16, total + 16)
    msg = torch.full((cap,), fill, dtype=torch.uint8, device="cuda")
    vt.vt_partial_encode(pd.data_ptr(), n, prd.data_ptr(), ofd.data_ptr(), msg.data_ptr(), total)
    torch.cuda.synchronize()
    return msg.cpu().numpy(), prd, ofd, msg


def edge_vector(n):
    v = vector(7, n, 3.0).astype(np.float32)
    v[0:32] = 0.0                                            # zero block
    v[32:64] = np.float16(65504.0) * np.sign(np.arange(32) - 15.5)   # fp16 extremes
    v[64:96] = [127.0] + [2.5, 3.5, -2.5, -3.5, 0.5, 1.5, -0.5] * 4 + [0.0] * 3   # ties
    v[96:128] = np.float16(6e-8) * np.arange(32)             # subnormals
    return v.astype(np.float16)


PLANS = ["fp16", "int8", "int4", "mixed", "pruned"]


def plan_for(kind, nb, rng):
    if kind == "mixed":
        imp = rng.integers(0, 5, nb).astype(np.float32)
        return C.plan(imp, int(nb * 64 * 0.45))
    level = {"fp16": C.FP16, "int8": C.INT8, "int4": C.INT4, "pruned": C.PRUNED}[kind]
    prec = np.full(nb, level)
    size = np.array([C.BLOCK_BYTES[level]] * nb)
    return prec, np.concatenate([[0], np.cumsum(size)[:-1]]), int(size.sum())


@pytest.mark.parametrize("kind", PLANS)
@pytest.mark.parametrize("which", ["seeded", "edges"])
def test_encode_bit_exact(kind, which):
    n = 4096
    p16 = vector(1, n, 2.0) if which == "seeded" else edge_vector(n)
    prec, offs, total = plan_for(kind, n // 32, np.random.default_rng(5))
    got, *_ = run_encode(p16, prec, offs, total)
    want = C.encode(p16, prec, offs, total)
    assert np.array_equal(got[:total], want), np.flatnonzero(got[:total] != want)[:10]
    assert np.all(got[total:] == 0xA5)   # nothing past the message


@pytest.mark.parametrize("kind", PLANS)
def test_decode_add_bit_exact(kind):
    n = 2048
    p16 = vector(2, n, 1.5)
    base = vector(3, n, 4.0)
    prec, offs, total = plan_for(kind, n // 32, np.random.default_rng(6))
    msg_host = C.encode(p16, prec, offs, total)
    msg = dev(np.concatenate([msg_host, np.zeros(16, np.uint8)]))
    prd, ofd = dev(prec.astype(np.uint8)), dev(offs.astype(np.int32))
    bd = dev(base.view(np.int16)).view(torch.float16)
    out = torch.empty(n, dtype=torch.float16, device="cuda")
    vt.vt_partial_decode_add(msg.data_ptr(), total, n, prd.data_ptr(), ofd.data_ptr(),
                             bd.data_ptr(), out.data_ptr())
    torch.cuda.synchronize()
    # the definition's fp32 steps: value = code * s (fp32), then fp32 add, then fp16
    val = C.decode(msg_host, prec, offs, n).astype(np.float32)
    want = (base.astype(np.float32) + val).astype(np.float16)
    assert np.array_equal(out.cpu().numpy().view(np.int16), want.view(np.int16))


def test_message_bounded_by_its_size():
    # offsets pointing past the stated message size write nothing there
    n = 256
    p16 = vector(4, n)
    prec = np.full(n // 32, C.INT8)
    offs = np.arange(n // 32) * 36 + 1000
    got, *_ = run_encode(p16, prec, offs, 64, fill=0x5A)
    assert np.all(got == 0x5A)


def test_decode_step_partial_sent_quantized():
    wl = tiny_workload(401, 1024, 8, 8, 64, 1500, (0.5, 0.5), 0, 64, sigma=0.03)
    li = LayerInputs(wl)
    gs = GpuShard(wl, li=li)
    x = li.x(5)
    got = gs.decode(x, wl.ctx)
    kc, vc = gs.context()
    ref = oracle_decode(wl, li, oracle_ranges(wl), x, kc, vc, wl.ctx)
    n, nb = wl.dims.hidden, wl.dims.hidden // 32
    rng = np.random.default_rng(9)
    for budget in (nb * 36, nb * 20 + 200, nb * 28):
        prec, offs, total = vt.vt_qplan(rng.random(nb).astype(np.float32), budget)
        assert total <= budget
        p16 = got["p_attn"].astype(np.float16)
        _, prd, ofd, msg = run_encode(p16, prec, offs, total)
        out = torch.empty(n, dtype=torch.float16, device="cuda")
        vt.vt_partial_decode_add(msg.data_ptr(), total, n, prd.data_ptr(), ofd.data_ptr(), None,
                                 out.data_ptr())
        torch.cuda.synchronize()
        recv = out.float().cpu().numpy().astype(np.float64)
        p = ref["p_attn"]
        rms = np.sqrt(np.mean(p * p))
        for b in range(nb):
            sl = slice(32 * b, 32 * b + 32)
            level = int(prec[b])
            if level == C.PRUNED:
                assert not recv[sl].any()
                continue
            half_step = 0.0 if level == C.FP16 else np.max(np.abs(p[sl])) / C.QMAX[level] / 2
            bound = 1.05 * half_step + 2e-2 * np.maximum(np.abs(p[sl]), rms)
            assert np.all(np.abs(recv[sl] - p[sl]) <= bound), (budget, b, level)


def emit_case(wl, plans, staged=False, msg_bytes=None, li=None):
    """vt_layer_decode_emit with per-partial plans {'attn': (prec, offs, total), 'ffn': ...}:
    returns the outputs, the two messages (host bytes, filled with 0xA5 past what
    was written) and the device plan tensors."""
    li = li or LayerInputs(wl)
    gs = GpuShard(wl, li=li)
    x = li.x(2)
    H = gs.dims.hidden
    xt = torch.from_numpy(x).cuda()
    out = {k: torch.full((H,), float("nan"), dtype=torch.float16, device="cuda")
           for k in ("p_attn", "h", "p_ffn", "y")}
    dv = {}
    for name in ("attn", "ffn"):
        prec, offs, total = plans[name]
        cap = max(16, total + 64)
        dv[name] = (dev(prec.astype(np.uint8)), dev(offs.astype(np.int32)),
                    torch.full((cap,), 0xA5, dtype=torch.uint8, device="cuda"), total)
    em = vt.vt_emit(prec_attn=dv["attn"][0].data_ptr(), off_attn=dv["attn"][1].data_ptr(),
                    msg_attn=dv["attn"][2].data_ptr(),
                    msg_attn_bytes=dv["attn"][3] if msg_bytes is None else msg_bytes,
                    prec_ffn=dv["ffn"][0].data_ptr(), off_ffn=dv["ffn"][1].data_ptr(),
                    msg_ffn=dv["ffn"][2].data_ptr(),
                    msg_ffn_bytes=dv["ffn"][3] if msg_bytes is None else msg_bytes)
    io = vt.vt_layer_io(x=xt.data_ptr(), peer_attn=None, peer_ffn=None,
                        attn_partial=out["p_attn"].data_ptr(), h=out["h"].data_ptr(),
                        ffn_partial=out["p_ffn"].data_ptr(), y=out["y"].data_ptr())
    vt.vt_layer_decode_emit(gs.spec, gs.w.struct, gs.kv, io, wl.ctx,
                            vt.VT_ATTN | vt.VT_FFN | (vt.VT_STAGED if staged else 0), em,
                            gs.ws.data_ptr(), gs.ws_bytes, None)
    torch.cuda.synchronize()
    got = {k: v.float().cpu().numpy().astype(np.float64) for k, v in out.items()}
    msgs = {k: dv[k][2].cpu().numpy() for k in dv}
    assert not np.any(gs.sync_words()), "synchronisation words not cleared"
    return gs, x, got, msgs, dv


def plans_for(nb, rng, kind):
    if kind == "mixed":
        return {n: vt.vt_qplan(rng.random(nb).astype(np.float32), int(nb * 64 * f))
                for n, f in (("attn", 0.45), ("ffn", 0.3))}
    p = plan_for(kind, nb, rng)
    return {"attn": p, "ffn": p}


@pytest.mark.parametrize("kind", ["mixed", "fp16", "int8", "int4", "pruned"])
@pytest.mark.parametrize("key", ["tiny", "7b", "70b_gqa"])
def test_decode_emits_quantized_partials(key, kind):
    """The O and down epilogues emit exactly the message vt_partial_encode
    makes of the same call's partial sums; the decode outputs still match
    the oracle; a received partial is within the quantisation bound of the
    oracle's."""
    from synth import get
    from tests.common import assert_close, ffn_at_h16, oracle_shard_weights
    wl = get(key)
    li = LayerInputs(wl)
    nb = wl.dims.hidden // 32
    plans = plans_for(nb, np.random.default_rng(21), kind)
    gs, x, got, msgs, dv = emit_case(wl, plans, li=li)
    for name, part in (("attn", "p_attn"), ("ffn", "p_ffn")):
        prec, offs, total = plans[name]
        ref_msg, *_ = run_encode(got[part].astype(np.float16), prec, offs, total)
        assert np.array_equal(msgs[name][:total], ref_msg[:total]), name
        assert np.all(msgs[name][total:] == 0xA5), name      # nothing past the message
    kc, vc = gs.context()
    r = oracle_ranges(wl)
    ref = oracle_decode(wl, li, r, x, kc, vc, wl.ctx)
    for k in ("p_attn", "h", "p_ffn", "y"):
        assert_close(got[k], ref[k], f"{key} {kind} {k}")
    # the attention partial as the aggregating device receives it
    prec, offs, total = plans["attn"]
    n = wl.dims.hidden
    outr = torch.empty(n, dtype=torch.float16, device="cuda")
    vt.vt_partial_decode_add(dv["attn"][2].data_ptr(), total, n, dv["attn"][0].data_ptr(),
                             dv["attn"][1].data_ptr(), None, outr.data_ptr())
    torch.cuda.synchronize()
    recv = outr.float().cpu().numpy().astype(np.float64)
    p = ref["p_attn"]
    rms = np.sqrt(np.mean(p * p))
    for b in range(nb):
        sl = slice(32 * b, 32 * b + 32)
        level = int(prec[b])
        if level == C.PRUNED:
            assert not recv[sl].any()
            continue
        half_step = 0.0 if level == C.FP16 else np.max(np.abs(p[sl])) / C.QMAX[level] / 2
        bound = 1.05 * half_step + 2e-2 * np.maximum(np.abs(p[sl]), 0.2 * rms)
        assert np.all(np.abs(recv[sl] - p[sl]) <= bound), (key, kind, b, level)


def test_emit_message_bounded_by_its_size():
    """A message buffer shorter than the plan: bytes past msg_bytes stay as
    they were (the epilogue's stores are range-checked)."""
    wl = tiny_workload(402, 512, 8, 8, 64, 1000, (0.5, 0.5), 1, 32, sigma=0.03)
    nb = 512 // 32
    plans = plans_for(nb, np.random.default_rng(3), "int8")
    total = plans["attn"][2]
    gs, x, got, msgs, dv = emit_case(wl, plans, msg_bytes=total // 2)
    for name, part in (("attn", "p_attn"), ("ffn", "p_ffn")):
        prec, offs, tot = plans[name]
        ref_msg, *_ = run_encode(got[part].astype(np.float16), prec, offs, tot)
        half = total // 2
        # blocks that fit entirely below msg_bytes are written; nothing at or past it
        assert np.all(msgs[name][half:] == 0xA5), name
        whole = [b for b in range(nb) if offs[b] + 36 <= half]
        for b in whole:
            assert np.array_equal(msgs[name][offs[b]:offs[b] + 36], ref_msg[offs[b]:offs[b] + 36])


def test_emit_rejects_staged_and_planless_messages():
    wl = tiny_workload(403, 512, 8, 8, 64, 1000, (0.5, 0.5), 0, 16, sigma=0.03)
    nb = 512 // 32
    plans = plans_for(nb, np.random.default_rng(4), "fp16")
    with pytest.raises(vt.VoltronError) as e:
        emit_case(wl, plans, staged=True)
    assert e.value.status == vt.VT_ERR_UNSUPPORTED


def test_emit_rejects_hidden_not_a_multiple_of_32():
    """The message's 32-value blocks map whole onto the O and down rows of a
    workgroup only when the hidden size is a multiple of 32; otherwise the
    call is refused before anything runs."""
    wl = tiny_workload(404, 1032, 4, 2, 128, 900, (0.5, 0.5), 0, 16, sigma=0.03)
    nb = (1032 + 31) // 32
    plans = plans_for(nb, np.random.default_rng(5), "fp16")
    with pytest.raises(vt.VoltronError) as e:
        emit_case(wl, plans)
    assert e.value.status == vt.VT_ERR_UNSUPPORTED
