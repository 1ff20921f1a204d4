"""GPU parity of the window diagnostics (remote traffic per source, rank
loads, per-engine MoE pressure) against the CPU oracle: integers bit-exact,
pressures exact too (one IEEE division each on both sides)."""
import json
import os

import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2606_15177_amd import workloads as W
from tests.gpu_util import dev

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module")
def moe():
    from paper_2606_15177_amd import moe
    return moe


def _gpu(moe, A, x, home, G, B=None, engine=None, n_eng=None, pressure=True):
    L, S, E = A.shape
    n_eng = G if n_eng is None else n_eng
    wd = moe.MoeWindowDims(L, S, E, G, n_eng)
    remote = torch.full((max(L, 1), S), -7, dtype=torch.int64, device="cuda")
    total = torch.full((max(L, 1), S), -7, dtype=torch.int64, device="cuda")
    rank_load = torch.full((max(L, 1), G), -7, dtype=torch.int64, device="cuda")
    pr = torch.full((n_eng,), float("nan"), dtype=torch.float64, device="cuda") if pressure else None
    moe.window_stats(wd, dev(A) if L else None, dev(x) if L else None, dev(home), remote, total, rank_load,
                     B=None if B is None else dev(B), engine=None if engine is None else dev(engine), pressure=pr)
    torch.cuda.synchronize()
    return (remote.cpu().numpy()[:L], total.cpu().numpy()[:L], rank_load.cpu().numpy()[:L],
            None if pr is None else pr.cpu().numpy())


def _check(moe, A, x, home, G, **kw):
    got = _gpu(moe, A, x, home, G, **kw)
    ref = oracle.window_stats(A, x, home, G, B=kw.get("B"), engine=kw.get("engine"), n_eng=kw.get("n_eng"),
                              pressure=kw.get("pressure", True))
    for name, g, r in zip(("remote", "total", "rank_load", "pressure"), got, ref):
        if r is None:
            assert g is None
        else:
            np.testing.assert_array_equal(g, r, err_msg=name)
    return got


def test_window_worked_example(moe):
    with open(os.path.join(GOLDEN, "place_worked.json")) as f:
        g = json.load(f)
    w = g["window"]
    remote, total, rank_load, _ = _check(moe, np.array(g["A"], np.int64)[None], np.array([w["x"]], np.int32),
                                         np.array(w["home"], np.int32), 2, B=np.array([g["B"]], np.int64))
    assert remote[0].tolist() == w["remote"] and total[0].tolist() == w["total"]
    assert rank_load[0].tolist() == w["rank_load"]


@pytest.mark.parametrize("name", list(W.PLACE_CONFIGS))
def test_window_workloads_before_and_after_placement(moe, name):
    cfg = W.PLACE_CONFIGS[name]
    p = W.make_place_inputs(cfg, seed=0)
    home = (np.arange(cfg.S) * cfg.G // cfg.S).astype(np.int32)
    _check(moe, p["A"], p["x0"], home, cfg.G)
    x, _ = oracle.place_greedy(p["A"], p["D"], p["x0"], p["cap"], m_uniform=p["m_uniform"])
    _check(moe, p["A"], x, home, cfg.G)


@pytest.mark.parametrize("L,S,E,G,n_eng", [(1, 1, 1, 1, 1), (3, 5, 37, 6, 2), (2, 64, 8192, 4, 4),
                                           (2, 3, 300, 1024, 16), (4, 130, 64, 8, 3)])
@pytest.mark.parametrize("variant", ["plain", "B", "odd_ids"])
def test_window_shapes(moe, L, S, E, G, n_eng, variant):
    rng = np.random.default_rng(L * 7 + S * 131 + E + G)
    A = rng.integers(0, 10 ** 6, size=(L, S, E)).astype(np.int64)
    x = rng.integers(0, G, size=(L, E)).astype(np.int32)
    home = rng.integers(0, G, size=S).astype(np.int32)
    engine = rng.integers(0, n_eng, size=G).astype(np.int32) if n_eng != G else None
    B = rng.integers(0, 10 ** 7, size=(L, E)).astype(np.int64) if variant == "B" else None
    if variant == "odd_ids":
        x[rng.random((L, E)) < 0.2] = -1
        x[rng.random((L, E)) < 0.1] = G + 3
        home[rng.random(S) < 0.3] = -2
        if engine is not None:
            engine[rng.random(G) < 0.3] = n_eng + 1
    _check(moe, A, x, home, G, B=B, engine=engine, n_eng=n_eng)


def test_window_no_pressure_and_no_layers(moe):
    rng = np.random.default_rng(3)
    A = rng.integers(0, 50, size=(2, 3, 10)).astype(np.int64)
    x = rng.integers(0, 4, size=(2, 10)).astype(np.int32)
    _check(moe, A, x, np.array([0, 1, 2], np.int32), 4, pressure=False)
    _, _, _, pr = _check(moe, np.zeros((0, 3, 10), np.int64), np.zeros((0, 10), np.int32),
                         np.array([0, 1, 2], np.int32), 4)
    assert pr.tolist() == [0.0] * 4
