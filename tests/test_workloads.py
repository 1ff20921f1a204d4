"""The seeded input generator: determinism, shapes, bf16 rounding and the
skew structure each workload is meant to have.  CPU only."""
import numpy as np
import pytest
import torch

from paper_2606_15177_amd import workloads as W


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    a = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 0.02,
                        np.array([1.0, -0.0, 0.0, 1.00390625, 1.01171875, 3.0e38], np.float32)])
    ours = W.f32_to_bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    np.testing.assert_array_equal(W.bf16_bits_to_f32(ours),
                                  torch.from_numpy(a).to(torch.bfloat16).float().numpy())


def test_deterministic_and_independent_streams():
    cfg = W.CONFIGS["tiny"]
    a = W.make_workload(cfg, seed=3)
    b = W.make_workload(cfg, seed=3)
    for k in a:
        if a[k] is not None:
            np.testing.assert_array_equal(a[k], b[k])
    r = W.make_routing(cfg, seed=3)                 # routing alone draws the same values
    np.testing.assert_array_equal(r["logits"], a["logits"])
    c = W.make_workload(cfg, seed=4)
    assert not np.array_equal(a["logits"], c["logits"])
    # one expert's weights do not depend on which other experts are drawn
    one = W.make_weights(cfg, seed=3, experts=[5])
    np.testing.assert_array_equal(one["w_down"][0], a["w_down"][5])


@pytest.mark.parametrize("name", W.CONFIG_ORDER)
def test_routing_shapes(name):
    cfg = W.CONFIGS[name]
    r = W.make_routing(cfg, seed=0)
    assert r["src"].shape == (cfg.T,) and r["src"].dtype == np.int32
    assert r["src"].min() >= 0 and r["src"].max() < cfg.S
    assert r["logits"].shape == (cfg.T, cfg.E) and r["logits"].dtype == np.float32
    assert np.isfinite(r["logits"]).all()
    loc = r["local_experts"]
    if cfg.local_layout == "all":
        assert loc is None and cfg.E_local == cfg.E
    else:
        assert loc.shape == (cfg.E_local,) and len(set(loc.tolist())) == cfg.E_local
        assert loc.min() >= 0 and loc.max() < cfg.E


def test_weight_scale_and_layout():
    cfg = W.CONFIGS["tiny"]
    w = W.make_weights(cfg, seed=0)
    assert w["w_gate"].shape == (cfg.E_local, cfg.I, cfg.H)
    assert w["w_down"].shape == (cfg.E_local, cfg.H, cfg.I)
    v = W.bf16_bits_to_f32(w["w_up"]).astype(np.float64)
    assert abs(v.std() - 0.02) < 5e-4 and abs(v.mean()) < 5e-4
    sh = W.make_weights(W.CONFIGS["prefill_dsv2_lite"].replace(H=64, I=32, I_shared=32), seed=0)
    assert sh["sh_gate"].shape == (2, 32, 64) and sh["sh_down"].shape == (2, 64, 32)


def test_skews():
    # Zipf popularity: the argmax histogram is heavy-headed
    cfg = W.CONFIGS["prefill_dsv2_lite"]
    lg = W.make_routing(cfg, seed=0)["logits"]
    top1 = np.bincount(lg.argmax(1), minlength=cfg.E)
    assert top1.max() > 8 * np.median(top1)
    # contiguous source blocks for the expert-parallel share
    cfg5 = W.CONFIGS["ep_share_dsv3"]
    src = W.make_src(cfg5)
    assert (np.diff(src) >= 0).all() and np.bincount(src).tolist() == [cfg5.T // cfg5.S] * cfg5.S
    # per-source hot sets
    cfg4 = W.CONFIGS["prefill_qwen3_30b_a3b"]
    r = W.make_routing(cfg4, seed=0)
    top = r["logits"].argmax(1)
    for s in range(cfg4.S):
        hist = np.bincount(top[r["src"] == s], minlength=cfg4.E)
        assert np.sort(hist)[-8:].sum() > 0.5 * hist.sum()
