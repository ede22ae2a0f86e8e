"""GPU parity of the MoE FFN shard (paper Sec. 2.1 FFN variants; Table 3's
MoE model) through vt_moe_ffn_decode against the fp64 oracle.moe:

* the selected experts equal the oracle's (bit-exact) wherever the gap
  between the k-th and (k+1)-th oracle logit is far above the rounding of
  the device's fp32 logits from fp16-rounded activations; inside that gap
  the device's choice must still be a valid top-k within it;
* probabilities, the partial sum and y match to the decode tolerance;
* the shards of a partition add up to the unsharded sub-layer;
* ragged column counts (one expert's share shorter than, equal to and
  longer than a 512-column segment), every expert selected, one expert,
  a shard with no columns, NaN in every row padding, and several tokens
  through one workspace.
"""
import functools

import numpy as np
import pytest
import torch

import oracle
from oracle.moe import moe_ffn
from paper_2607_07046_amd import pack
from paper_2607_07046_amd import voltron as vt
from synth.configs import MOE_WORKLOADS, MoEWorkload
from synth.gen import MoEInputs
from tests.common import assert_close
from tests.gpu_common import h16

pytestmark = pytest.mark.gpu

NAN16 = 0x7E00
# |logit error| of the device: fp16 rounding of w (2^-11 relative) through
# a router row, far below this gap
GAP = 1e-2


class CachedInputs:
    """MoEInputs with each expert tensor drawn once."""

    def __init__(self, wl):
        self.wl = wl
        self._mi = MoEInputs(wl)

    def g_ffn(self):
        return self._mi.g_ffn()

    def router(self):
        return self._mi.router()

    def h(self, token=0):
        return self._mi.h(token)

    @functools.lru_cache(maxsize=None)
    def expert(self, name, e):
        return self._mi.expert(name, e)


@functools.lru_cache(maxsize=None)
def workload_inputs(key):
    return CachedInputs(MOE_WORKLOADS[key])


def moe_spec(wl, device):
    dims = vt.vt_layer_dims(hidden=wl.hidden, n_heads=1, n_kv_heads=1, head_dim=64,
                            ffn=wl.expert_ffn, rms_eps=wl.rms_eps, rope_base=10000.0, window=0)
    spec = vt.vt_shard_spec_create(dims, wl.fracs, wl.fracs, device)
    _, info = vt.vt_shard_spec_query(spec)
    return spec, info


def oracle_shard(mi, c0, nc):
    E = mi.wl.n_experts
    wg = np.stack([mi.expert("wg", e)[c0:c0 + nc] for e in range(E)])
    wu = np.stack([mi.expert("wu", e)[c0:c0 + nc] for e in range(E)])
    wd = np.stack([mi.expert("wd", e)[:, c0:c0 + nc] for e in range(E)])
    return wg, wu, wd


class GpuMoE:
    def __init__(self, mi, device, ld_pad=0, nan_pad=False):
        wl = mi.wl
        self.wl = wl
        self.spec, self.info = moe_spec(wl, device)
        self.c0, self.nc = self.info.col_begin, self.info.n_cols
        self.w = pack.pack_moe_shard(mi, self.c0, self.nc, ld_pad=ld_pad)
        if nan_pad:  # every padding element of every row
            H = wl.hidden
            for name in ("wg", "wu"):
                t = self.w.tensors[name]
                if t.numel():
                    t[:, :, H:].view(torch.int16).fill_(NAN16)
            t = self.w.tensors["wd"]
            t[:, :, self.nc:].view(torch.int16).fill_(NAN16)
        self.ws_bytes = vt.vt_moe_workspace_size(self.spec, wl.n_experts, wl.top_k)
        self.ws = torch.zeros(self.ws_bytes, dtype=torch.uint8, device="cuda")

    def run(self, h, peer=None):
        H, k = self.wl.hidden, self.wl.top_k
        ht = h16(h)
        pt = h16(peer) if peer is not None else None
        p = torch.empty(H, dtype=torch.float16, device="cuda")
        y = torch.empty(H, dtype=torch.float16, device="cuda")
        sel = torch.full((k,), -1, dtype=torch.int32, device="cuda")
        prob = torch.full((k,), -1.0, dtype=torch.float32, device="cuda")
        io = vt.vt_layer_io(x=None, peer_attn=None, peer_ffn=pt.data_ptr() if pt is not None else None,
                            attn_partial=None, h=ht.data_ptr(), ffn_partial=p.data_ptr(),
                            y=y.data_ptr())
        vt.vt_moe_ffn_decode(self.spec, self.w.struct, self.wl.n_experts, k, io, sel.data_ptr(),
                             prob.data_ptr(), self.ws.data_ptr(), self.ws_bytes)
        torch.cuda.synchronize()
        return dict(p_ffn=p.float().cpu().numpy(), y=y.float().cpu().numpy(),
                    sel=sel.cpu().numpy(), probs=prob.cpu().numpy())


def check_selection(got_sel, ref, k):
    logits = ref["logits"]
    order = np.argsort(-logits, kind="stable")
    kth = logits[order[k - 1]]
    nxt = logits[order[k]] if k < len(logits) else -np.inf
    assert len(set(got_sel.tolist())) == k and np.all((got_sel >= 0) & (got_sel < len(logits)))
    if kth - nxt > GAP:
        assert np.array_equal(got_sel, ref["sel"]), (got_sel, ref["sel"])
        return True
    # inside the rounding gap: every chosen logit is within it of the k-th
    assert np.all(logits[got_sel] >= kth - GAP), (got_sel, ref["sel"])
    return False


def check_token(g, mi, h, peer=None):
    wl = g.wl
    out = g.run(h, peer)
    wg, wu, wd = oracle_shard(mi, g.c0, g.nc)
    ref = moe_ffn(mi.g_ffn(), mi.router(), wg, wu, wd, wl.rms_eps, h, wl.top_k, peer=peer)
    if check_selection(out["sel"], ref, wl.top_k):
        assert_close(out["probs"], ref["probs"], "probabilities")
        assert_close(out["p_ffn"], ref["p_ffn"], "p_ffn")
        assert_close(out["y"], ref["y"], "y")
    return out, ref


def small(seed, H, E, F, k, fracs, sigma=0.05, rsigma=0.2):
    return MoEWorkload(key=f"moe_{seed}", seed_id=seed, title="", hidden=H, n_experts=E,
                       expert_ffn=F, top_k=k, fracs=fracs, device=0, weight_sigma=sigma,
                       router_sigma=rsigma)


def test_moe_workload_device0_tokens():
    """Qwen1.5-MoE-A2.7B-shaped routed experts, device 0 of 4 (352 columns
    of each of 60 experts, top-4): three tokens through one workspace."""
    mi = workload_inputs("moe")
    wl = mi.wl
    g = GpuMoE(mi, wl.device)
    exact = 0
    for t in range(3):
        h = mi.h(t)
        peer = h16(np.asarray(MoEInputs(wl).h(100 + t), np.float32) * 0.1).cpu().numpy()
        out, ref = check_token(g, mi, h, peer)
        exact += check_selection(out["sel"], ref, wl.top_k)
    assert exact >= 2


def test_moe_partition_sums_to_layer():
    mi = workload_inputs("moe")
    wl = mi.wl
    h = mi.h(0)
    total = np.zeros(wl.hidden)
    for dev in range(len(wl.fracs)):
        g = GpuMoE(mi, dev)
        out, ref = check_token(g, mi, h)
        total += out["p_ffn"]
    E = wl.n_experts
    wg = np.stack([mi.expert("wg", e) for e in range(E)])
    wu = np.stack([mi.expert("wu", e) for e in range(E)])
    wd = np.stack([mi.expert("wd", e) for e in range(E)])
    full = moe_ffn(mi.g_ffn(), mi.router(), wg, wu, wd, wl.rms_eps, h, wl.top_k)
    assert_close(total, full["p_ffn"], "sum of the 4 shards' partials")


CASES = {
    # (H, E, F, top_k, fracs, device)
    "ragged_lt_seg": (264, 5, 1000, 2, (0.3, 0.7), 0),     # 300 columns
    "ragged_gt_seg": (264, 5, 1000, 2, (0.3, 0.7), 1),     # 700 columns
    "one_seg": (512, 7, 512, 3, (1.0,), 0),                # exactly 512
    "multi_seg": (1032, 4, 2600, 2, (1.0,), 0),            # 2600 columns, H past a segment
    "all_experts": (256, 6, 200, 6, (0.5, 0.5), 0),
    "one_expert": (256, 1, 200, 1, (1.0,), 0),
    "top1_of_256": (128, 256, 24, 1, (1.0,), 0),
    "top8": (512, 16, 96, 8, (0.25, 0.75), 1),
    # the largest expert count and top-k; router rows 1.5/sqrt(hidden): at the
    # default 0.2 the 8 largest of 256 logits reach about 10, where the
    # router's fp16 input alone moves the partial by 1.5e-3 normwise (a numpy
    # model of the rounding points gives the device's error to three digits)
    "top8_of_256": (512, 256, 64, 8, (0.5, 0.5), 1, 1.5 / 512 ** 0.5),
}


@pytest.mark.parametrize("case", CASES)
def test_moe_shapes(case):
    H, E, F, k, fr, dev, *rsigma = CASES[case]
    wl = small(900 + len(case), H, E, F, k, fr, **({"rsigma": rsigma[0]} if rsigma else {}))
    mi = CachedInputs(wl)
    g = GpuMoE(mi, dev)
    for t in range(2):
        check_token(g, mi, mi.h(t))


def _random_moe_shapes(n=6, seed=20261205):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        H = 8 * int(rng.integers(16, 513))
        E = int(rng.integers(1, 65))
        F = int(rng.integers(16, 2049))
        k = int(rng.integers(1, min(E, 8) + 1))
        ndev = int(rng.integers(1, 4))
        fr = rng.dirichlet(np.ones(ndev)) * 0.9 + 0.1 / ndev
        fr = tuple(float(round(f, 3)) for f in fr)
        fr = fr[:-1] + (round(1.0 - sum(fr[:-1]), 3),)
        out.append((930 + i, H, E, F, k, fr, float(1.0 / np.sqrt(H)), float(1.5 / np.sqrt(H))))
    return out


RANDOM_MOE = _random_moe_shapes()


@pytest.mark.parametrize("case", RANDOM_MOE,
                         ids=[f"H{c[1]}-E{c[2]}-F{c[3]}-k{c[4]}-n{len(c[5])}" for c in RANDOM_MOE])
def test_moe_random_shapes(case):
    """Seeded random MoE shards: hidden any multiple of 8 up to 4096, 1-64
    experts of 16-2048 columns, top-1..8, 1-3 devices (every device's shard
    checked); expert weights scaled 1/sqrt(hidden) and router rows
    1.5/sqrt(hidden), so the router logits keep a spread of about 1.5 at
    every hidden size (a fixed router scale of 0.2 gives logits of about 13
    at hidden 4056, where the probabilities' fp16 rounding error alone
    exceeds the normwise bar)."""
    seed, H, E, F, k, fr, sigma, rsigma = case
    wl = small(seed, H, E, F, k, fr, sigma=sigma, rsigma=rsigma)
    mi = CachedInputs(wl)
    for dev in range(len(fr)):
        g = GpuMoE(mi, dev)
        check_token(g, mi, mi.h(0))


def test_moe_nan_padding_never_read():
    wl = small(951, 264, 5, 1000, 2, (0.3, 0.7))
    mi = CachedInputs(wl)
    for dev in (0, 1):
        g = GpuMoE(mi, dev, ld_pad=8, nan_pad=True)
        out, _ = check_token(g, mi, mi.h(0))
        assert np.all(np.isfinite(out["p_ffn"]))


def test_moe_shard_without_columns():
    wl = small(953, 256, 4, 64, 2, (0.0, 1.0))
    mi = CachedInputs(wl)
    g = GpuMoE(mi, 0)
    assert g.nc == 0
    h = mi.h(0)
    peer = np.asarray(mi.h(1), np.float16)
    out = g.run(h, peer)
    assert np.all(out["p_ffn"] == 0)
    want = (np.asarray(h, np.float64) + peer.astype(np.float64)).astype(np.float16)
    assert np.array_equal(out["y"].astype(np.float16), want)
    wg, wu, wd = oracle_shard(mi, 0, 0)
    ref = moe_ffn(mi.g_ffn(), mi.router(), wg, wu, wd, wl.rms_eps, h, wl.top_k)
    check_selection(out["sel"], ref, wl.top_k)


class RouterOverride(CachedInputs):
    """A small workload whose router rows are set by the test."""

    def __init__(self, wl, router):
        super().__init__(wl)
        self._router = np.asarray(router, np.float16)

    def router(self):
        return self._router


@pytest.mark.parametrize("k", [1, 2, 3])
def test_moe_ties_go_to_the_lower_index(k):
    """Equal logits (identical router rows: the same fp32 sums on the device,
    the same fp64 sums in the oracle) are ordered by expert index."""
    wl = small(961, 256, 8, 64, k, (1.0,))
    base = CachedInputs(wl)
    r = base.router().copy()
    r[5] = r[2] = np.abs(r[2]) * np.sign(base.h(0) * base.g_ffn()).astype(np.float16)  # largest
    mi = RouterOverride(wl, r)
    g = GpuMoE(mi, 0)
    out, ref = check_token(g, mi, mi.h(0))
    assert out["sel"][0] == 2 and ref["sel"][0] == 2
    if k >= 2:
        assert out["sel"][1] == 5 and ref["sel"][1] == 5
        assert out["probs"][0] == out["probs"][1]


def test_moe_zero_logits_tie():
    """Zero router rows give logits of exactly zero (whatever their sign
    bit); every other expert's logit is negative, so the zero-logit experts
    are selected lowest index first."""
    wl = small(963, 256, 6, 64, 2, (1.0,))
    base = CachedInputs(wl)
    sgn = np.sign(base.h(0).astype(np.float32) * base.g_ffn().astype(np.float32))
    r = np.tile(-0.05 * sgn, (6, 1)).astype(np.float16)
    r[1] = 0
    r[3] = 0
    mi = RouterOverride(wl, r)
    g = GpuMoE(mi, 0)
    out, ref = check_token(g, mi, mi.h(0))
    assert list(out["sel"]) == [1, 3] and list(ref["sel"]) == [1, 3]
