"""Whole-layer GPU parity (moe_forward) against the CPU oracle on small and
adversarial layers: every intermediate the layer exposes bit-exact (expert
ids, counts, offsets, dispatch order), gates within 1e-6 and the output
within the layer tolerance.  The five workloads at full size are in
test_gpu_full_size.py."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2606_15177_amd import workloads as W
from tests.gpu_util import (assert_gates_close, assert_layer_close, dev, dev_weights, gating_cfg, host_bf16,
                            oracle_forward_cfg, oracle_route_cfg, workload)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def moe():
    from paper_2606_15177_amd import moe
    return moe


def _forward(moe, cfg, wl, counts=None, repeat=1):
    d = moe.dims_of(cfg)
    T, k = cfg.T, cfg.k
    taps_t = dict(topk_idx=torch.full((max(T, 1), k), -9, dtype=torch.int32, device="cuda"),
                  topk_w=torch.zeros((max(T, 1), k), dtype=torch.float32, device="cuda"),
                  expert_load=torch.full((cfg.E,), -9, dtype=torch.int32, device="cuda"),
                  offsets=torch.full((cfg.E_local + 1,), -9, dtype=torch.int32, device="cuda"),
                  perm_token=torch.full((max(T * k, 1),), -9, dtype=torch.int32, device="cuda"),
                  inv_pos=torch.full((max(T * k, 1),), -9, dtype=torch.int32, device="cuda"))
    taps = moe.make_taps(**taps_t)
    loc = None if wl["local_experts"] is None else dev(wl["local_experts"])
    gating, gate_bias = gating_cfg(moe, cfg, wl)
    layer = moe.MoeLayer(d, dev_weights(wl), loc, gating=gating)
    if counts is None:
        counts = torch.zeros((cfg.S, cfg.E), dtype=torch.int64, device="cuda")
    logits, src, x = dev(wl["logits"]), dev(wl["src"]), dev(wl["x"])
    outs = []
    for _ in range(repeat):
        out = torch.full((max(T, 1), cfg.H), 3.0, dtype=torch.bfloat16, device="cuda")
        layer.forward(logits, src, x, counts, out[:T] if T else None, taps)
        outs.append(out)
    torch.cuda.synchronize()
    res = {n: t.cpu().numpy() for n, t in taps_t.items()}
    res["counts"] = counts.cpu().numpy()
    res["outs"] = [host_bf16(o)[:T] for o in outs]
    return res


def _check_routing(cfg, wl, res, calls=1):
    T, k = cfg.T, cfg.k
    ridx, rw = oracle_route_cfg(cfg, wl)
    np.testing.assert_array_equal(res["topk_idx"][:T], ridx)
    assert_gates_close(res["topk_w"][:T], rw, cfg.name)
    rc, rl = oracle.route_stats(wl["src"], ridx, cfg.S, cfg.E)
    np.testing.assert_array_equal(res["counts"], calls * rc)
    np.testing.assert_array_equal(res["expert_load"], rl)
    off, perm, inv = oracle.permute(ridx, cfg.E, cfg.E_local, wl["local_experts"])
    np.testing.assert_array_equal(res["offsets"], off)
    np.testing.assert_array_equal(res["perm_token"][: off[-1]], perm)
    np.testing.assert_array_equal(res["inv_pos"][: T * k], inv)
    return ridx


def test_forward_tiny_all_tokens_and_determinism(moe):
    cfg = W.CONFIGS["tiny"]
    wl = workload("tiny")
    res = _forward(moe, cfg, wl, repeat=2)
    _check_routing(cfg, wl, res, calls=2)
    ref = oracle.forward_tokens(cfg.dims, np.arange(cfg.T), wl["logits"], wl["x"], wl["local_experts"], wl)
    assert_layer_close(res["outs"][0], ref, "tiny")
    np.testing.assert_array_equal(res["outs"][0], res["outs"][1])     # bitwise deterministic


@pytest.mark.parametrize("variant", [
    dict(T=1), dict(T=2, k=1), dict(T=64, E=16, k=4, E_local=5, local_layout="choice"),
    dict(T=63, H=136, I=200, n_shared=2, I_shared=72), dict(T=300, H=200, I=136, E=12, k=3, E_local=12),
    dict(T=777, E=33, k=5, E_local=7, local_layout="choice", n_shared=1, I_shared=64),
    dict(T=100, src_layout="blocks"), dict(T=100, src_layout="interleaved", S=3),
    # routing and dispatch in one launch (at most 512 pairs and four token
    # groups of the routing block) and just past its limits
    dict(T=128, k=4), dict(T=129, k=2), dict(T=128, E=8, k=5),
    dict(T=32, E=256, k=8, E_local=32, local_layout="choice", S=8),
    dict(T=16, E=1024, k=8, E_local=300, local_layout="choice", S=16),   # a 64 KB statistics histogram too
    # the largest k: routing block dispatching 512 pairs itself, and a
    # permute-path batch whose combine sums 32 pairs per token
    dict(T=16, E=64, k=32, E_local=64), dict(T=40, E=64, k=32, E_local=24, local_layout="choice", n_shared=1,
                                              I_shared=64),
])
def test_forward_variants(moe, variant):
    cfg = W.CONFIGS["tiny"].replace(name="variant", **variant)
    wl = W.make_workload(cfg, seed=2)
    res = _forward(moe, cfg, wl)
    _check_routing(cfg, wl, res)
    ref = oracle.forward_tokens(cfg.dims, np.arange(cfg.T), wl["logits"], wl["x"], wl["local_experts"], wl)
    assert_layer_close(res["outs"][0], ref, str(variant))


@pytest.mark.parametrize("variant,repeat", [
    (dict(T=600, E=64, k=4, E_local=64, S=5, src_layout="interleaved"), 2),
    (dict(T=900, E=128, k=8, E_local=16, local_layout="choice", S=8, src_layout="blocks"), 1),
    (dict(T=300, E=1024, k=2, E_local=40, local_layout="choice", S=17), 1),   # S*E past the LDS histogram
    # per-tile histograms summed by the scatter launch's extra blocks: more
    # tiles than bins (33 tiles, 32 bins), 32 tiles over 512 bins, a 64 KB
    # histogram in each of 4 tiles; and 258 tiles of 16384 bins, past the
    # rows' limit, flushed by atomics instead
    (dict(T=4100, E=16, k=4, E_local=16, S=2), 2),
    (dict(T=2000, E=64, k=8, E_local=64, S=8), 1),
    (dict(T=200, E=1024, k=8, E_local=64, local_layout="choice", S=16), 1),
    (dict(T=16500, E=1024, k=8, E_local=16, local_layout="choice", S=16), 2),
])
def test_forward_statistics_in_the_dispatch_count_pass(moe, variant, repeat):
    """Batches of more than 512 pairs count the source x expert statistics
    in the dispatch's count pass (over all E experts, local or not): counts
    accumulate over calls and expert_load is set, as when the router counts."""
    cfg = W.CONFIGS["tiny"].replace(name="stats", **variant)
    assert cfg.T * cfg.k > 512
    wl = W.make_workload(cfg, seed=4)
    res = _forward(moe, cfg, wl, repeat=repeat)
    _check_routing(cfg, wl, res, calls=repeat)


def test_forward_statistics_skip_bad_sources(moe):
    """Out-of-range source ids are skipped by the count pass: counts and
    expert_load are the oracle's over the tokens with valid sources, and the
    dispatch and output do not depend on the sources."""
    cfg = W.CONFIGS["tiny"].replace(name="badsrc", T=700, E=32, k=3, E_local=32, S=4)
    wl = W.make_workload(cfg, seed=6)
    src = wl["src"].copy()
    src[::7] = cfg.S + 3
    src[1::11] = -1
    wl_bad = dict(wl, src=src)
    res = _forward(moe, cfg, wl_bad)
    ridx, rw = oracle_route_cfg(cfg, wl)
    np.testing.assert_array_equal(res["topk_idx"][:cfg.T], ridx)
    ok = (src >= 0) & (src < cfg.S)
    rc, rl = oracle.route_stats(src[ok], ridx[ok], cfg.S, cfg.E)
    np.testing.assert_array_equal(res["counts"], rc)
    np.testing.assert_array_equal(res["expert_load"], rl)
    off, perm, inv = oracle.permute(ridx, cfg.E, cfg.E_local, wl["local_experts"])
    np.testing.assert_array_equal(res["offsets"], off)
    np.testing.assert_array_equal(res["perm_token"][: off[-1]], perm)
    ref = oracle.forward_tokens(cfg.dims, np.arange(cfg.T), wl["logits"], wl["x"], wl["local_experts"], wl)
    assert_layer_close(res["outs"][0], ref, "badsrc")


def test_forward_tokens_without_local_experts(moe):
    """Tokens none of whose experts are hosted here get only the shared part;
    without shared experts they get exact zeros."""
    cfg = W.CONFIGS["tiny"].replace(name="remote", E=16, k=2, E_local=2, local_layout="choice", T=200)
    wl = W.make_workload(cfg, seed=3)
    res = _forward(moe, cfg, wl)
    ridx = _check_routing(cfg, wl, res)
    local = set(wl["local_experts"].tolist())
    remote_tok = [t for t in range(cfg.T) if not (set(ridx[t].tolist()) & local)]
    assert remote_tok
    assert (res["outs"][0][remote_tok] == 0).all()
    ref = oracle.forward_tokens(cfg.dims, np.arange(cfg.T), wl["logits"], wl["x"], wl["local_experts"], wl)
    assert_layer_close(res["outs"][0], ref, "remote")


def test_forward_one_hot_gates_is_dense_ffn(moe):
    cfg = W.CONFIGS["tiny"].replace(name="onehot", T=100, E=8, k=2)
    wl = W.make_workload(cfg, seed=4)
    chosen = np.random.default_rng(0).integers(0, cfg.E, cfg.T)
    logits = np.full((cfg.T, cfg.E), -np.inf, np.float32)
    logits[np.arange(cfg.T), chosen] = 0.0
    wl["logits"] = logits
    res = _forward(moe, cfg, wl)
    ref = np.stack([oracle.swiglu_ffn(wl["x"][t], wl["w_gate"][e], wl["w_up"][e], wl["w_down"][e])
                    for t, e in enumerate(chosen)])
    assert_layer_close(res["outs"][0], ref, "one-hot")


def test_forward_empty_batch(moe):
    cfg = W.CONFIGS["tiny"].replace(name="empty", T=0)
    wl = W.make_workload(cfg, seed=0)
    d = moe.dims_of(cfg)
    layer = moe.MoeLayer(d, dev_weights(wl))
    counts = torch.zeros((cfg.S, cfg.E), dtype=torch.int64, device="cuda")
    moe.forward(d, None, None, None, None, layer._w, counts, None, layer.ws)
    torch.cuda.synchronize()
    assert counts.sum().item() == 0


@pytest.mark.parametrize("variant", [
    dict(gate=1),
    dict(gate=1, n_group=4, topk_group=2, routed_scale=2.0),
    dict(gate=2, gate_bias_std=0.05, routed_scale=2.5, n_group=4, topk_group=2),
    dict(gate=2, gate_bias_std=0.05, E=64, k=6, E_local=20, local_layout="choice", n_group=8, topk_group=3,
         n_shared=1, I_shared=128, T=513),
])
def test_forward_gated_routers(moe, variant):
    """The layer under each gating variant: routing bit-exact, output within
    the layer tolerance against the oracle's layer with the same router."""
    cfg = W.CONFIGS["tiny"].replace(**{**dict(name="gated", E=16, k=4, E_local=16, T=300), **variant})
    wl = W.make_workload(cfg, seed=7)
    res = _forward(moe, cfg, wl)
    _check_routing(cfg, wl, res)
    ref = oracle_forward_cfg(cfg, wl, np.arange(cfg.T))
    assert_layer_close(res["outs"][0], ref, str(variant))
