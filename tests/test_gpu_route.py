"""GPU parity of top-k gating and the source x expert statistics against the
CPU oracle: expert ids and counts bit-exact, gates within 1e-6."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2606_15177_amd import workloads as W
from tests.gpu_util import assert_gates_close, dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def moe():
    from paper_2606_15177_amd import moe
    return moe


def _route(moe, logits: np.ndarray, k: int):
    T, E = logits.shape
    d = moe.dims(T=T, H=8, E=E, k=k, I=8, S=1, E_local=E)
    idx = torch.full((T, k), -7, dtype=torch.int32, device="cuda")
    w = torch.full((T, k), -7.0, dtype=torch.float32, device="cuda")
    moe.route(d, dev(logits), idx, w)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), w.cpu().numpy()


@pytest.mark.parametrize("name", W.CONFIG_ORDER)
def test_route_configs(moe, name):
    cfg = W.CONFIGS[name]
    r = W.make_routing(cfg, seed=0)
    idx, w = _route(moe, r["logits"], cfg.k)
    ridx, rw = oracle.route(r["logits"], cfg.k)
    np.testing.assert_array_equal(idx, ridx)
    assert_gates_close(w, rw, name)


def _adversarial_rows(E: int, rng) -> np.ndarray:
    rows = [rng.standard_normal(E),
            np.round(rng.standard_normal(E) * 1.5),            # integer logits: many ties
            np.zeros(E),                                       # all equal
            np.where(rng.random(E) < 0.5, -0.0, 0.0),          # signed zeros only
            np.full(E, -np.inf)]
    r = rng.standard_normal(E)
    r[rng.random(E) < 0.2] = np.nan
    r[rng.random(E) < 0.1] = -np.inf
    r[rng.random(E) < 0.05] = np.inf
    rows.append(r)
    r = np.round(rng.standard_normal(E))
    r[rng.random(E) < 0.3] = -0.0
    r[rng.random(E) < 0.1] = np.nan
    rows.append(r)
    return np.stack(rows).astype(np.float32)


@pytest.mark.parametrize("E,k", [(1, 1), (2, 2), (3, 2), (8, 8), (13, 4), (33, 5), (64, 32), (65, 3),
                                 (100, 7), (256, 8), (511, 9), (1000, 32), (1024, 1)])
def test_route_adversarial(moe, E, k):
    rng = np.random.default_rng(E * 31 + k)
    logits = np.concatenate([_adversarial_rows(E, rng) for _ in range(6)])
    logits = np.concatenate([logits, rng.standard_normal((257, E)).astype(np.float32)])  # ragged tail
    idx, w = _route(moe, logits, k)
    ridx, rw = oracle.route(logits, k)
    np.testing.assert_array_equal(idx, ridx)
    assert_gates_close(w, rw, f"E={E} k={k}")


def test_route_empty_is_noop(moe):
    d = moe.dims(T=0, H=8, E=8, k=2, I=8, S=1, E_local=8)
    moe.route(d, None, None, None)
    torch.cuda.synchronize()


def _stats(moe, src, idx, S, E, counts=None, with_load=True):
    T, k = idx.shape
    d = moe.dims(T=T, H=8, E=E, k=k, I=8, S=S, E_local=E)
    c = torch.zeros((S, E), dtype=torch.int64, device="cuda") if counts is None else counts
    load = torch.full((E,), 12345, dtype=torch.int32, device="cuda") if with_load else None
    moe.route_stats(d, dev(src), dev(idx), c, load)
    torch.cuda.synchronize()
    return c, (load.cpu().numpy() if with_load else None)


@pytest.mark.parametrize("name", W.CONFIG_ORDER)
def test_stats_configs(moe, name):
    cfg = W.CONFIGS[name]
    r = W.make_routing(cfg, seed=0)
    ridx, _ = oracle.route(r["logits"], cfg.k)
    rc, rl = oracle.route_stats(r["src"], ridx, cfg.S, cfg.E)
    c, load = _stats(moe, r["src"], ridx, cfg.S, cfg.E)
    np.testing.assert_array_equal(c.cpu().numpy(), rc)
    np.testing.assert_array_equal(load, rl)
    # a second call accumulates the matrix and sets the load again
    c, load = _stats(moe, r["src"], ridx, cfg.S, cfg.E, counts=c)
    np.testing.assert_array_equal(c.cpu().numpy(), 2 * rc)
    np.testing.assert_array_equal(load, rl)


def test_stats_global_atomic_path_and_bad_ids(moe):
    """S*E beyond the LDS histogram (global atomics), and out-of-range source
    or expert ids, which are skipped: the expected counts are the oracle's over
    the valid pairs alone."""
    rng = np.random.default_rng(5)
    for S, E, T, k in ((40, 1000, 3000, 6), (4, 8, 3000, 3)):
        src = rng.integers(0, S, T).astype(np.int32)
        idx = np.stack([rng.choice(E, k, replace=False) for _ in range(T)]).astype(np.int32)
        rc, rl = oracle.route_stats(src, idx, S, E)
        c, load = _stats(moe, src, idx, S, E)
        np.testing.assert_array_equal(c.cpu().numpy(), rc)
        np.testing.assert_array_equal(load, rl)
        src[::7] = S + 3
        src[1::11] = -1
        idx[2::13, 0] = E
        idx[3::17, k - 1] = -5
        ok = ((src >= 0) & (src < S))[:, None] & (idx >= 0) & (idx < E)
        pair_src = np.repeat(src, k)[ok.ravel()]
        pair_idx = idx.ravel()[ok.ravel()][:, None]
        rc, rl = oracle.route_stats(pair_src, pair_idx, S, E)
        c, load = _stats(moe, src, idx, S, E)
        np.testing.assert_array_equal(c.cpu().numpy(), rc)
        np.testing.assert_array_equal(load, rl)


# ------------------------------------------------------ gating variants ---

def _route_gated(moe, logits, k, gate, bias=None, scale=1.0, n_group=0, topk_group=0):
    T, E = logits.shape
    d = moe.dims(T=T, H=8, E=E, k=k, I=8, S=1, E_local=E, flags=gate)
    b = None if bias is None else dev(bias)
    g = moe.gating(b, scale, n_group, topk_group)
    idx = torch.full((T, k), -7, dtype=torch.int32, device="cuda")
    w = torch.full((T, k), -7.0, dtype=torch.float32, device="cuda")
    moe.route(d, dev(logits), idx, w, gating=g)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), w.cpu().numpy()


GATED_CASES = [  # (E, k, gate, with bias, scale, n_group, topk_group)
    (8, 2, 1, False, 1.0, 0, 0), (64, 6, 1, False, 1.0, 0, 0), (256, 8, 1, False, 16.0, 8, 3),
    (8, 2, 2, True, 2.5, 4, 2), (64, 6, 2, True, 1.0, 8, 3), (256, 8, 2, True, 2.5, 8, 4),
    (256, 8, 2, False, 1.0, 0, 0), (160, 6, 2, True, 2.5, 5, 2), (1024, 16, 2, True, 1.0, 64, 8),
    (12, 3, 2, True, 1.0, 12, 3), (96, 4, 0, False, 3.0, 6, 2), (33, 5, 2, True, 1.0, 0, 0),
    # 8 and 4 lanes of a token's lane group scan each expert group
    (64, 4, 2, True, 1.0, 2, 1), (128, 8, 1, False, 1.0, 4, 2),
]


@pytest.mark.parametrize("E,k,gate,with_bias,scale,n_group,topk_group", GATED_CASES)
def test_route_gated_variants(moe, E, k, gate, with_bias, scale, n_group, topk_group):
    rng = np.random.default_rng(E * 31 + k * 7 + gate)
    T = 700
    logits = rng.standard_normal((T, E)).astype(np.float32) * 2
    logits[:100] = np.round(logits[:100])                       # ties
    logits[100:150, rng.integers(0, E, 3)] = np.nan
    logits[150:200, rng.integers(0, E, 3)] = -np.inf
    logits[200:220, rng.integers(0, E, 2)] = np.inf
    bias = (rng.standard_normal(E) * 0.05).astype(np.float32) if with_bias else None
    if with_bias:
        bias[:: max(1, E // 7)] = np.round(bias[:: max(1, E // 7)] * 8) / 8
    idx, w = _route_gated(moe, logits, k, gate, bias, scale, n_group, topk_group)
    ridx, rw = oracle.route_gated(logits, k, gate, bias, scale, n_group, topk_group)
    np.testing.assert_array_equal(idx, ridx)
    finite = np.isfinite(rw)
    np.testing.assert_array_equal(np.isfinite(w), finite)
    np.testing.assert_allclose(w[finite], rw[finite], rtol=0, atol=1e-6 * max(1.0, scale))


def test_route_v3_router_full_size(moe):
    """The DeepSeek-V3 router on the full 16384-token, 256-expert workload."""
    cfg = W.CONFIGS["ep_share_dsv3_v3router"]
    r = W.make_routing(cfg, seed=0)
    idx, w = _route_gated(moe, r["logits"], cfg.k, cfg.gate, r["gate_bias"], cfg.routed_scale, cfg.n_group,
                          cfg.topk_group)
    ridx, rw = oracle.route_gated(r["logits"], cfg.k, cfg.gate, r["gate_bias"], cfg.routed_scale, cfg.n_group,
                                  cfg.topk_group)
    np.testing.assert_array_equal(idx, ridx)
    np.testing.assert_allclose(w, rw, rtol=0, atol=1e-6 * cfg.routed_scale)
    # only 4 of the 8 groups per token
    assert (np.array([len(set(row // 32)) for row in idx]) <= 4).all()
