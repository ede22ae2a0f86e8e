"""GPU checks of elastic re-partition and shard-wise pruning (paper Sec.
4.3.1) through the C ABI:

* vt_shard_pack gathers every shard of several partitions out of the whole
  layer's device weights bit for bit (host slicing of the same seeded
  tensors is the reference; Wd's padding columns are zero);
* vt_kv_copy_heads moves KV heads bit for bit and touches nothing else;
* a layer decoded 50/50 is re-partitioned 25/75 mid-stream: the new shards
  are packed and their KV heads taken over on a second stream while the old
  shards decode, and the next token's partials over the new shards add up
  to the oracle's layer for that token;
* the kept shards of a pruned 4-way partition add up to the oracle's pruned
  layer (the dropped heads' and columns' contributions removed).
"""
import numpy as np
import pytest
import torch

import oracle
from oracle.prune import pruned_weights
from paper_2607_07046_amd import pack
from paper_2607_07046_amd import voltron as vt
from synth import get
from synth.gen import LayerInputs
from tests.common import assert_close, ffn_at_h16, full_weights, tiny_workload
from tests.gpu_common import SENTINEL, GpuShard, h16, lib_dims

pytestmark = pytest.mark.gpu

BOTH = vt.VT_ATTN | vt.VT_FFN


def spec_for(wl, fracs, dev):
    spec = vt.vt_shard_spec_create(lib_dims(wl.dims), fracs, fracs, dev)
    dims, info = vt.vt_shard_spec_query(spec)
    return spec, dims, info


CASES = {
    "tiny_2": lambda: (get("tiny"), (0.5, 0.5)),
    "ragged_3_gqa": lambda: (tiny_workload(421, 512, 8, 4, 64, 1000, (0.33, 0.34, 0.33), 0, 16),
                             (0.33, 0.34, 0.33)),
    "7b_3": lambda: (get("7b"), (0.5, 0.3, 0.2)),
    "ragged_h1032_gqa3": lambda: (tiny_workload(422, 1032, 12, 4, 128, 900, (0.5, 0.5), 1, 16),
                                  (0.5, 0.5)),
}


@pytest.mark.parametrize("case", CASES)
def test_shard_pack_bit_exact(case):
    wl, fracs = CASES[case]()
    li = LayerInputs(wl)
    full = None
    for dev in range(len(fracs)):
        spec, dims, info = spec_for(wl, fracs, dev)
        if full is None:
            full = pack.upload_full(li, dims)
        out = pack.alloc_shard(dims, info)
        for t in out.tensors.values():
            t.view(torch.int16).fill_(0x7C01)          # a NaN pattern: every byte must be written
        vt.vt_shard_pack(spec, full.struct, out.struct)
        torch.cuda.synchronize()
        ref = pack.pack_shard(li, dims, info)          # host slices of the same tensors
        for name, t in ref.tensors.items():
            got = out.tensors[name].view(torch.int16).cpu().numpy()
            want = t.view(torch.int16).cpu().numpy()
            assert got.shape == want.shape, (case, dev, name)
            assert np.array_equal(got, want), (case, dev, name)


def test_kv_copy_heads_bit_exact():
    rng = np.random.default_rng(5)
    d, cap_s, cap_d = 64, 40, 33
    src_k = torch.from_numpy(rng.integers(-30000, 30000, (5, cap_s, d)).astype(np.int16)).cuda()
    src_v = torch.from_numpy(rng.integers(-30000, 30000, (5, cap_s, d)).astype(np.int16)).cuda()
    dst_k = torch.full((4, cap_d, d), SENTINEL, dtype=torch.int16, device="cuda")
    dst_v = dst_k.clone()
    src = vt.vt_kv_view(k=src_k.data_ptr(), v=src_v.data_ptr(), capacity=cap_s, n_kv_heads=5,
                        head_dim=d, len=cap_s)
    dst = vt.vt_kv_view(k=dst_k.data_ptr(), v=dst_v.data_ptr(), capacity=cap_d, n_kv_heads=4,
                        head_dim=d, len=0)
    vt.vt_kv_copy_heads(src, 2, dst, 1, 3, 31)
    torch.cuda.synchronize()
    for s_, d_ in ((src_k, dst_k), (src_v, dst_v)):
        a, b = s_.cpu().numpy(), d_.cpu().numpy()
        assert np.array_equal(b[1:4, :31], a[2:5, :31])
        assert np.all(b[0] == SENTINEL) and np.all(b[1:4, 31:] == SENTINEL)
    assert dst.len == 0
    with pytest.raises(vt.VoltronError):
        vt.vt_kv_copy_heads(src, 3, dst, 0, 3, 10)      # past the source's heads
    with pytest.raises(vt.VoltronError):
        vt.vt_kv_copy_heads(src, 0, dst, 0, 1, 34)      # past the destination's capacity


def shards_step(shards, x, pos):
    """One token through every shard: attention partials summed on the
    host (the aggregation), then the FFN shards on that h."""
    parts = [gs.decode(x, pos, vt.VT_ATTN, want_y=False) for gs in shards]
    sum_attn = np.sum([p["p_attn"] for p in parts], axis=0)
    h = (x.astype(np.float64) + sum_attn).astype(np.float16)
    ffn = [gs.decode(None, phases=vt.VT_FFN, h_in=h) for gs in shards]
    return sum_attn, h, np.sum([f["p_ffn"] for f in ffn], axis=0)


def test_repartition_keeps_decoding():
    wl = get("tiny")
    d = wl.dims
    li = LayerInputs(wl)
    old_fr, new_fr = (0.5, 0.5), (0.25, 0.75)
    cap = wl.ctx + 4
    old = [GpuShard(wl, device=s, li=li, capacity=cap, fracs=old_fr) for s in range(2)]
    x0, x1 = li.x(0), li.x(1)
    kc, vc = li.kv_context_heads(0, d.n_kv_heads)
    W = full_weights(li)
    ref0 = oracle.decode(W, d.n_heads, d.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, x0,
                         kc, vc, wl.ctx)

    # the new partition's shards: weights packed and KV heads taken over on a
    # second stream while the old shards decode token 0 on the default one
    dims = lib_dims(d)
    full = pack.upload_full(li, dims)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    new = [GpuShard(wl, device=s, li=li, capacity=cap, fracs=new_fr, fill_ctx=False)
           for s in range(2)]
    with torch.cuda.stream(side):
        for gs in new:
            gs.w = pack.alloc_shard(gs.dims, gs.info)
            vt.vt_shard_pack(gs.spec, full.struct, gs.w.struct, side.cuda_stream)
    a0, h0, f0 = shards_step(old, x0, wl.ctx)
    assert_close(a0, ref0["p_attn"], "token 0 attention (old partition)")
    side.synchronize()
    # KV heads of every new shard from the old shard holding them (the old
    # shards have appended token 0 at slot ctx)
    n_pos = wl.ctx + 1
    for gs in new:
        g0, g1 = gs.info.kv_head_begin, gs.info.kv_head_begin + gs.info.n_kv_heads
        for og in old:
            o0, o1 = og.info.kv_head_begin, og.info.kv_head_begin + og.info.n_kv_heads
            lo, hi = max(g0, o0), min(g1, o1)
            if lo < hi:
                vt.vt_kv_copy_heads(og.kv, lo - o0, gs.kv, lo - g0, hi - lo, n_pos,
                                    side.cuda_stream)
        gs.kv.len = n_pos
    side.synchronize()

    kc1 = np.concatenate([kc, ref0["k_new"][:, None, :]], axis=1)
    vc1 = np.concatenate([vc, ref0["v_new"][:, None, :]], axis=1)
    ref1 = oracle.decode(W, d.n_heads, d.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, x1,
                         kc1, vc1, wl.ctx + 1)
    a1, h1, f1 = shards_step(new, x1, wl.ctx + 1)
    assert_close(a1, ref1["p_attn"], "token 1 attention (new partition)")
    assert_close(h1.astype(np.float64), ref1["h"], "token 1 h")
    # the FFN shards run on the aggregated h; the reference is the oracle's
    # FFN at the oracle's h rounded to fp16
    assert_close(f1, ffn_at_h16(W, d.rms_eps, ref1)["p_ffn"], "token 1 FFN (new partition)")


@pytest.mark.parametrize("dropped", [(1,), (0, 3), (2,)])
def test_pruned_shards_sum_to_pruned_layer(dropped):
    fr = (0.25, 0.25, 0.25, 0.25)
    wl = tiny_workload(431, 512, 8, 4, 64, 1376, fr, 0, 64)
    d = wl.dims
    li = LayerInputs(wl)
    kept = [GpuShard(wl, device=s, li=li) for s in range(4) if s not in dropped]
    keep_g = np.ones(d.n_kv_heads, bool)
    keep_c = np.ones(d.ffn, bool)
    for s in dropped:
        r = oracle.shard_ranges(d.n_heads, d.n_kv_heads, d.ffn, fr, fr, s)
        keep_g[r.kv_head_begin:r.kv_head_begin + r.n_kv_heads] = False
        keep_c[r.col_begin:r.col_begin + r.n_cols] = False
    Wp = pruned_weights(full_weights(li), d.head_dim, d.n_heads // d.n_kv_heads, keep_g, keep_c)
    x = li.x(0)
    kc, vc = li.kv_context_heads(0, d.n_kv_heads)
    ref = oracle.decode(Wp, d.n_heads, d.n_kv_heads, d.head_dim, d.rms_eps, d.rope_base, x, kc,
                        vc, wl.ctx)
    a, h, f = shards_step(kept, x, wl.ctx)
    assert_close(a, ref["p_attn"], "kept attention partials")
    assert_close(f, ffn_at_h16(Wp, d.rms_eps, ref)["p_ffn"], "kept FFN partials")
