"""GPU parity of batch-1 decode (vt_layer_decode, vt_kv_append) against the
fp64 oracle, through the C ABI.

Bar: every fp16 output vector within max relative error 2e-2 (element-wise,
denominator floored at 0.2 of the reference vector's RMS) and normwise
relative error 1.5e-3 (derivation in tests/common.py), the FFN outputs
against the oracle's FFN at fp16(h); KV indexing
bit-exact (the appended slot holds the new key/value, every other cache
byte keeps its sentinel or context value, ``len`` advances by one).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_07046_amd import voltron as vt
from synth import get
from synth.gen import LayerInputs
from tests.common import (NORM_TOL, REL_TOL, _record, assert_close, ffn_at_h16, full_weights,
                          max_rel_err, norm_rel_err, oracle_ranges, oracle_shard_weights,
                          tiny_workload)
from tests.gpu_common import SENTINEL, GpuShard

pytestmark = pytest.mark.gpu

BOTH = vt.VT_ATTN | vt.VT_FFN
MODES = {"fused": 0, "staged": vt.VT_STAGED}

_cache = {}


def oracle_case(wl, device=None, li=None):
    """Oracle inputs/outputs of the workload's shard at its decode position."""
    key = (repr(wl), device)  # the whole workload: shapes, partition, context
    if key not in _cache:
        li = li or LayerInputs(wl)
        r = oracle_ranges(wl, device)
        w = oracle_shard_weights(li, r)
        kc, vc = li.kv_context_heads(r.kv_head_begin, r.kv_head_begin + r.n_kv_heads)
        d = wl.dims
        x = li.x(0)
        ref = oracle.decode(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base,
                            x, kc, vc, wl.ctx)
        ref = ffn_at_h16(w, d.rms_eps, ref)
        _cache[key] = (li, r, x, ref)
    return _cache[key]


def check_outputs(got, ref, keys=("p_attn", "h", "p_ffn", "y")):
    errs = {k: (max_rel_err(got[k], ref[k]), norm_rel_err(got[k], ref[k])) for k in keys}
    for k, (e, n) in errs.items():
        _record(k, e, n)
    bad = {k: e for k, e in errs.items() if not (e[0] <= REL_TOL and e[1] <= NORM_TOL)}
    assert not bad, f"(element-wise, normwise) relative errors {errs}"
    return errs


def check_kv(gs, ref, pos, k_before, v_before):
    kc, vc = gs.cache()
    assert gs.kv.len == pos + 1
    # every slot except pos is byte-identical to before
    mask = np.ones(kc.shape[1], bool)
    mask[pos] = False
    assert np.array_equal(kc[:, mask], k_before[:, mask])
    assert np.array_equal(vc[:, mask], v_before[:, mask])
    k_new = kc[:, pos].view(np.float16).astype(np.float64)
    v_new = vc[:, pos].view(np.float16).astype(np.float64)
    for g in range(k_new.shape[0]):
        assert_close(k_new[g], ref["k_new"][g], f"appended key of KV head {g}")
        assert_close(v_new[g], ref["v_new"][g], f"appended value of KV head {g}")


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("key", ["tiny", "7b", "70b_gqa"])
def test_decode_matches_oracle(key, mode):
    wl = get(key)
    li, r, x, ref = oracle_case(wl)
    gs = GpuShard(wl, li=li)
    assert (gs.info.n_q_heads, gs.info.n_kv_heads, gs.info.n_cols) == \
           (r.n_q_heads, r.n_kv_heads, r.n_cols)
    k0, v0 = gs.cache()
    got = gs.decode(x, wl.ctx, BOTH | MODES[mode])
    errs = check_outputs(got, ref)
    print(key, mode, errs)
    check_kv(gs, ref, wl.ctx, k0, v0)
    assert not np.any(gs.sync_words()), "synchronisation words not cleared"


def test_fused_staged_cooperative_and_repeat_are_bitwise_equal():
    wl = get("7b")
    li, r, x, ref = oracle_case(wl)
    outs = []
    for flags in (0, vt.VT_STAGED, 0, vt.VT_COOPERATIVE):
        gs = GpuShard(wl, li=li)
        outs.append((gs.decode(x, wl.ctx, BOTH | flags), gs.cache()))
    for o, c in outs[1:]:
        for k in ("p_attn", "h", "p_ffn", "y"):
            assert np.array_equal(o[k], outs[0][0][k]), k
        assert np.array_equal(c[0], outs[0][1][0]) and np.array_equal(c[1], outs[0][1][1])


@pytest.mark.parametrize("key", ["tiny", "7b"])
def test_all_shards_sum_to_unsharded_layer(key):
    """Sec. 3.2.1: the aggregated partials of every shard are the layer."""
    wl = get(key)
    d = wl.dims
    li = LayerInputs(wl)
    x = li.x(0)
    kc, vc = li.kv_context_heads(0, d.n_kv_heads)
    fw = full_weights(li)
    full = oracle.decode(fw, d.n_heads, d.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, x, kc,
                         vc, wl.ctx)
    shards = [GpuShard(wl, device=s, li=li) for s in range(len(wl.fracs))]
    parts = [gs.decode(x, wl.ctx, vt.VT_ATTN) for gs in shards]
    sum_attn = np.sum([p["p_attn"] for p in parts], axis=0)
    assert_close(sum_attn, full["p_attn"], "sum of attention partials")
    # aggregation on the main device (host stand-in), then the FFN shards
    h = (x.astype(np.float64) + sum_attn).astype(np.float16)
    ffn = [gs.decode(None, phases=vt.VT_FFN, h_in=h) for gs in shards]
    sum_ffn = np.sum([f["p_ffn"] for f in ffn], axis=0)
    full = ffn_at_h16(fw, d.rms_eps, full)
    assert_close(sum_ffn, full["p_ffn"], "sum of FFN partials")
    # peer semantics: shard 0 given the others' partials produces the full h and y
    peer_a = np.sum([p["p_attn"] for p in parts[1:]], axis=0).astype(np.float16)
    peer_f = np.sum([f["p_ffn"] for f in ffn[1:]], axis=0).astype(np.float16)
    gs0 = GpuShard(wl, device=0, li=li)
    got = gs0.decode(x, wl.ctx, BOTH, peer_attn=peer_a, peer_ffn=peer_f)
    assert_close(got["h"], full["h"], "h with peer partials")
    assert_close(got["y"], full["y"], "y with peer partials")


def test_consecutive_tokens_match_oracle_chain():
    wl = get("tiny")
    d = wl.dims
    li = LayerInputs(wl)
    r = oracle_ranges(wl)
    w = oracle_shard_weights(li, r)
    kc, vc = li.kv_context_heads(r.kv_head_begin, r.kv_head_begin + r.n_kv_heads)
    kc, vc = kc.astype(np.float64), vc.astype(np.float64)
    gs = GpuShard(wl, li=li, capacity=wl.ctx + 16)
    for t in range(12):
        pos = wl.ctx + t
        x = li.x(t)
        ref = oracle.decode(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base,
                            x, kc, vc, pos)
        ref = ffn_at_h16(w, d.rms_eps, ref)
        got = gs.decode(x, pos, BOTH | (vt.VT_STAGED if t % 2 else 0))
        check_outputs(got, ref)
        kc = np.concatenate([kc, ref["k_new"][:, None]], axis=1)
        vc = np.concatenate([vc, ref["v_new"][:, None]], axis=1)
    assert gs.kv.len == wl.ctx + 12


@pytest.mark.parametrize("mode", MODES)
def test_empty_cache_and_last_slot(mode):
    """pos = 0 (nothing cached) and an append into the last free slot."""
    wl = tiny_workload(201, 256, 4, 2, 64, 300, (0.5, 0.5), 1, 0, sigma=0.05)
    li, r, x, ref = oracle_case(wl)
    gs = GpuShard(wl, li=li, capacity=1)
    k0, v0 = gs.cache()
    got = gs.decode(x, 0, BOTH | MODES[mode])
    check_outputs(got, ref)
    check_kv(gs, ref, 0, k0, v0)
    with pytest.raises(vt.VoltronError) as e:
        gs.decode(x, 1, BOTH)
    assert e.value.status == vt.VT_ERR_KV_FULL


@pytest.mark.parametrize("mode", MODES)
def test_ragged_shapes_and_gqa_groups(mode):
    """Odd column counts (ragged last piece), head_dim 64 with GQA group 4,
    several attention chunks with a ragged last chunk."""
    wl = tiny_workload(202, 1024, 16, 4, 64, 3000, (0.37, 0.33, 0.30), 2, 150, sigma=0.03)
    li, r, x, ref = oracle_case(wl)
    gs = GpuShard(wl, li=li)
    assert gs.info.n_cols % 8 != 0
    k0, v0 = gs.cache()
    got = gs.decode(x, wl.ctx, BOTH | MODES[mode])
    check_outputs(got, ref)
    check_kv(gs, ref, wl.ctx, k0, v0)


# Seeded shapes with hidden sizes that are multiples of 8 but not of 16, 32
# or 64 (the last weight piece of every K = hidden row is ragged), hidden
# unequal to heads x head_dim, odd FFN shares, both head sizes, GQA groups
# and contexts over several attention chunks; drawn once from a fixed seed.
def _ragged_hidden_cases():
    rng = np.random.default_rng(20261203)
    out = []
    for i in range(4):
        d = (64, 128)[i % 2]
        nkv = int(rng.choice([1, 2, 4]))
        nh = max(2, nkv * int(rng.choice([1, 2, 4])))
        H = int(rng.choice([520, 776, 1032, 1288]))
        F = int(rng.integers(300, 1500))
        fr = (0.5, 0.5) if nh % 2 == 0 and nkv % 2 == 0 else (1.0,)
        dev = int(rng.integers(0, len(fr)))
        ctx = int(rng.integers(0, 300))
        out.append((600 + i, H, nh, nkv, d, F, fr, dev, ctx))
    return out


RAGGED_H = _ragged_hidden_cases()
RAGGED_IDS = [f"H{c[1]}-h{c[2]}-kv{c[3]}-d{c[4]}-F{c[5]}" for c in RAGGED_H]


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("case", RAGGED_H, ids=RAGGED_IDS)
def test_ragged_hidden_sizes(case, mode):
    wl = tiny_workload(*case, sigma=0.03)
    li, r, x, ref = oracle_case(wl)
    gs = GpuShard(wl, li=li)
    k0, v0 = gs.cache()
    pa, pf = li.peer("attn"), li.peer("ffn")
    d = wl.dims
    w = oracle_shard_weights(li, r)
    kc, vc = li.kv_context_heads(r.kv_head_begin, r.kv_head_begin + r.n_kv_heads)
    ref = oracle.decode(w, r.n_q_heads, r.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, x, kc,
                        vc, wl.ctx, pa, pf)
    ref = ffn_at_h16(w, d.rms_eps, ref, pf)
    got = gs.decode(x, wl.ctx, BOTH | MODES[mode], peer_attn=pa, peer_ffn=pf)
    check_outputs(got, ref)
    check_kv(gs, ref, wl.ctx, k0, v0)
    assert not np.any(gs.sync_words()), "synchronisation words not cleared"


GROUPS = {
    # seed, hidden, heads, kv, d, ffn, fracs, device, ctx: query heads per KV
    # head that are not powers of two
    "g3": (610, 1536, 12, 4, 128, 1000, (0.5, 0.5), 1, 333),
    "g7": (611, 1792, 28, 4, 64, 1200, (0.5, 0.5), 0, 515),
}


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("key", GROUPS)
def test_gqa_groups_not_powers_of_two(key, mode):
    wl = tiny_workload(*GROUPS[key], sigma=0.03)
    li, r, x, ref = oracle_case(wl)
    assert r.n_q_heads == r.n_kv_heads * (wl.dims.n_heads // wl.dims.n_kv_heads)
    gs = GpuShard(wl, li=li)
    k0, v0 = gs.cache()
    got = gs.decode(x, wl.ctx, BOTH | MODES[mode])
    check_outputs(got, ref)
    check_kv(gs, ref, wl.ctx, k0, v0)


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("ctx", [16000, 32767])
def test_long_contexts(ctx, mode):
    """Decode at 16000 and 32767 cached positions on a GQA shard (8 query
    heads over 2 KV heads, head size 128): many attention chunks, the merge
    of their partial records in several batches."""
    wl = tiny_workload(620 if ctx == 16000 else 621, 1024, 16, 4, 128, 2000, (0.5, 0.5), 0, ctx,
                       sigma=0.03)
    li, r, x, ref = oracle_case(wl)
    gs = GpuShard(wl, li=li)
    k0, v0 = gs.cache()
    got = gs.decode(x, wl.ctx, BOTH | MODES[mode])
    check_outputs(got, ref)
    check_kv(gs, ref, wl.ctx, k0, v0)
    assert not np.any(gs.sync_words()), "synchronisation words not cleared"


@pytest.mark.parametrize("mode", MODES)
def test_million_position_context(mode):
    """Decode after 1,000,000 cached positions (8 query heads over one KV
    head of 128; 256 MB each of cached keys and values): about 3900
    attention chunks per query head, whose partial records the merge reads
    in many batches."""
    wl = tiny_workload(622, 1024, 16, 2, 128, 2000, (0.5, 0.5), 0, 1_000_000, sigma=0.03)
    li, r, x, ref = oracle_case(wl)
    assert r.n_q_heads == 8 and r.n_kv_heads == 1
    gs = GpuShard(wl, li=li)
    k0, v0 = gs.cache()
    got = gs.decode(x, wl.ctx, BOTH | MODES[mode])
    check_outputs(got, ref)
    check_kv(gs, ref, wl.ctx, k0, v0)
    assert not np.any(gs.sync_words()), "synchronisation words not cleared"


@pytest.mark.parametrize("mode", MODES)
def test_long_context_head_dim_64(mode):
    """Decode after 100,000 cached positions with head size 64 (8 threads per
    position, 64 positions per pass, chunks of up to 512 positions), device
    1 of two: 8 query heads over 2 KV heads."""
    wl = tiny_workload(623, 1024, 16, 4, 64, 2000, (0.5, 0.5), 1, 100_000, sigma=0.03)
    li, r, x, ref = oracle_case(wl)
    assert r.n_q_heads == 8 and r.n_kv_heads == 2
    gs = GpuShard(wl, li=li)
    k0, v0 = gs.cache()
    got = gs.decode(x, wl.ctx, BOTH | MODES[mode])
    check_outputs(got, ref)
    check_kv(gs, ref, wl.ctx, k0, v0)
    assert not np.any(gs.sync_words()), "synchronisation words not cleared"


def test_empty_shard_outputs_zero_partials():
    """A device that gets no heads and no columns (e.g. one whose share was
    pruned away) contributes zero partials; h and y pass x and peers through."""
    wl = tiny_workload(203, 512, 8, 8, 64, 1376, (1.0, 0.0), 1, 16, sigma=0.02)
    li = LayerInputs(wl)
    gs = GpuShard(wl, li=li)
    assert gs.info.n_q_heads == 0 and gs.info.n_cols == 0
    x = li.x(0)
    pa, pf = li.peer("attn"), li.peer("ffn")
    got = gs.decode(x, wl.ctx, BOTH, peer_attn=pa, peer_ffn=pf)
    assert np.all(got["p_attn"] == 0) and np.all(got["p_ffn"] == 0)
    h = (x.astype(np.float64) + pa.astype(np.float64)).astype(np.float16).astype(np.float64)
    assert max_rel_err(got["h"], h) <= 1e-3
    assert max_rel_err(got["y"], h + pf.astype(np.float64)) <= 1e-2


def test_attn_only_then_ffn_only_equals_both():
    wl = get("tiny")
    li, r, x, ref = oracle_case(wl)
    a = GpuShard(wl, li=li)
    ga = a.decode(x, wl.ctx, vt.VT_ATTN)
    gf = a.decode(None, phases=vt.VT_FFN, h_in=ga["h"].astype(np.float16))
    b = GpuShard(wl, li=li)
    gb = b.decode(x, wl.ctx, BOTH)
    for k in ("p_attn", "h"):
        assert np.array_equal(ga[k], gb[k]), k
    for k in ("p_ffn", "y"):
        assert np.array_equal(gf[k], gb[k]), k


def test_kv_append_is_a_bit_exact_copy():
    wl = tiny_workload(204, 512, 8, 4, 128, 64, (0.5, 0.5), 0, 0)
    gs = GpuShard(wl, capacity=40, fill_ctx=False)
    rng = np.random.default_rng(5)
    nkv, d = gs.info.n_kv_heads, gs.dims.head_dim
    written = np.full((nkv, 40, d), SENTINEL, np.int16), np.full((nkv, 40, d), SENTINEL, np.int16)
    pos = 0
    for n in (7, 1, 0, 13, 19):
        bits_k = rng.integers(-2 ** 15, 2 ** 15, size=(n, nkv, d), dtype=np.int16)
        bits_v = rng.integers(-2 ** 15, 2 ** 15, size=(n, nkv, d), dtype=np.int16)
        gs.append(bits_k.view(np.float16), bits_v.view(np.float16))
        written[0][:, pos:pos + n] = np.transpose(bits_k, (1, 0, 2))
        written[1][:, pos:pos + n] = np.transpose(bits_v, (1, 0, 2))
        pos += n
        assert gs.kv.len == pos
        kc, vc = gs.cache()
        assert np.array_equal(kc, written[0]) and np.array_equal(vc, written[1])
    with pytest.raises(vt.VoltronError):
        gs.append(np.zeros((1, nkv, d), np.float16), np.zeros((1, nkv, d), np.float16))
