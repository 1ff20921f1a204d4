"""Pins for the CPU oracle: it is checked against hand-derived worked examples,
closed forms, brute force, textbook/library special cases and invariants,
never against itself or the HIP path.  CPU only."""
import itertools
import json
import math
import os

import numpy as np
import pytest

from paper_2606_15177_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _f32(vals):
    return np.array([float(v) for v in vals], dtype=np.float32)


def _bf16(a):
    return W.f32_to_bf16_bits(np.asarray(a, dtype=np.float32))


# ---------------------------------------------------------------- routing ---

def test_route_worked_example(oracle_mod):
    g = _load("route_worked.json")
    row = _f32(g["logits"])[None, :]
    for case in g["cases"]:
        idx, w = oracle_mod.route(row, case["k"])
        assert idx[0].tolist() == case["idx"], case
        if case["w"] is None:
            assert np.isnan(w).all()
        else:
            np.testing.assert_allclose(w[0], case["w"], rtol=0, atol=1e-15)
    for case in g["extra_rows"]:
        idx, w = oracle_mod.route(_f32(case["logits"])[None, :], case["k"])
        assert idx[0].tolist() == case["idx"], case["note"]
        np.testing.assert_allclose(w[0], case["w"], rtol=0, atol=1e-15)


def _sort_key(v, e):
    # the selection order spelled out as a tuple: numbers by value descending,
    # then index; NaN after all numbers.
    v = float(v)
    return (1, 0.0, e) if math.isnan(v) else (0, -v, e)


@pytest.mark.parametrize("E,k", [(5, 1), (6, 2), (7, 3), (8, 4), (10, 3), (12, 4), (9, 9)])
def test_route_brute_force_subsets(oracle_mod, E, k):
    """The selected set is the unique k-subset whose every member precedes
    every non-member; found by enumerating all C(E, k) subsets."""
    rng = np.random.default_rng(E * 100 + k)
    rows = []
    for _ in range(40):
        rows.append(rng.integers(-2, 3, size=E).astype(np.float32))      # heavy ties
    for _ in range(20):
        r = rng.standard_normal(E).astype(np.float32)
        r[rng.integers(0, E, size=2)] = rng.choice(np.array([np.nan, -np.inf, np.inf, -0.0, 0.0], np.float32), 2)
        rows.append(r)
    logits = np.stack(rows)
    idx, _ = oracle_mod.route(logits, k)
    for t in range(len(rows)):
        keys = [_sort_key(logits[t, e], e) for e in range(E)]
        winners = [s for s in itertools.combinations(range(E), k)
                   if max(keys[e] for e in s) < min((keys[e] for e in range(E) if e not in s),
                                                    default=(9, 0, 0))]
        assert len(winners) == 1
        assert set(idx[t].tolist()) == set(winners[0])
        # within the k slots: the selection order itself
        assert [keys[e] for e in idx[t]] == sorted(keys[e] for e in idx[t])


def test_route_matches_numpy_stable_argsort(oracle_mod):
    """Special cases reducing to library routines: k=E is a stable descending
    argsort, k=1 is argmax (first occurrence); signed zeros and NaNs included."""
    rng = np.random.default_rng(7)
    T, E = 300, 16
    logits = np.round(rng.standard_normal((T, E)) * 2).astype(np.float32)
    logits[rng.random((T, E)) < 0.05] = -0.0
    logits[rng.random((T, E)) < 0.02] = np.nan
    full, _ = oracle_mod.route(logits, E)
    np.testing.assert_array_equal(full, np.argsort(-logits, axis=1, kind="stable"))
    clean = np.where(np.isnan(logits), np.float32(-1e30), logits)
    top1, w1 = oracle_mod.route(clean, 1)
    np.testing.assert_array_equal(top1[:, 0], np.argmax(clean, axis=1))
    assert (w1 == 1.0).all()


def test_route_gate_closed_forms(oracle_mod):
    rng = np.random.default_rng(3)
    logits = rng.standard_normal((500, 32)).astype(np.float32) * 3
    idx, w = oracle_mod.route(logits, 2)
    l0 = logits[np.arange(500), idx[:, 0]].astype(np.float64)
    l1 = logits[np.arange(500), idx[:, 1]].astype(np.float64)
    np.testing.assert_allclose(w[:, 0], 1.0 / (1.0 + np.exp(l1 - l0)), rtol=0, atol=1e-15)
    idx8, w8 = oracle_mod.route(logits, 8)
    np.testing.assert_allclose(w8.sum(1), 1.0, atol=1e-14)
    assert (np.diff(w8, axis=1) <= 0).all()      # gates follow the selection order
    # softmax over all experts, restricted to the top-k and renormalised, is the same thing
    p = np.exp(logits.astype(np.float64) - logits.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    sel = np.take_along_axis(p, idx8, 1)
    np.testing.assert_allclose(w8, sel / sel.sum(1, keepdims=True), rtol=1e-12)


# ------------------------------------------------------------------ stats ---

def test_stats_worked_example(oracle_mod):
    g = _load("dispatch_worked.json")
    counts, load = oracle_mod.route_stats(np.array(g["src"]), np.array(g["topk_idx"]), g["S"], g["E"])
    assert counts.tolist() == g["counts"]
    assert load.tolist() == g["expert_load"]


def test_stats_invariants_and_accumulation(oracle_mod):
    cfg = W.CONFIGS["prefill_qwen3_30b_a3b"].replace(T=1000)
    r = W.make_routing(cfg, seed=5)
    idx, _ = oracle_mod.route(r["logits"], cfg.k)
    counts, load = oracle_mod.route_stats(r["src"], idx, cfg.S, cfg.E)
    assert counts.sum() == cfg.T * cfg.k
    for s in range(cfg.S):
        assert counts[s].sum() == cfg.k * int((r["src"] == s).sum())
    np.testing.assert_array_equal(counts.sum(0), np.bincount(idx.ravel(), minlength=cfg.E))
    np.testing.assert_array_equal(load, counts.sum(0))
    counts2, load2 = oracle_mod.route_stats(r["src"], idx, cfg.S, cfg.E, counts=counts.copy())
    np.testing.assert_array_equal(counts2, 2 * counts)      # += over a profiling window
    np.testing.assert_array_equal(load2, load)              # = per call
    # source hotspots of this workload show up in A: each source's hot set dominates its row
    assert (counts.max(1) > 3 * counts.mean(1)).all()


def test_stats_rejects_bad_ids(oracle_mod):
    with pytest.raises(oracle_mod.OracleError):
        oracle_mod.route_stats(np.array([0, 2]), np.array([[0], [1]]), 2, 4)
    with pytest.raises(oracle_mod.OracleError):
        oracle_mod.route_stats(np.array([0, 1]), np.array([[0], [4]]), 2, 4)


# ---------------------------------------------------------------- permute ---

def test_permute_worked_example(oracle_mod):
    g = _load("dispatch_worked.json")
    off, perm, inv = oracle_mod.permute(np.array(g["topk_idx"]), g["E"], 2, np.array(g["local_experts"]))
    assert off.tolist() == g["offsets"]
    assert perm.tolist() == g["perm_token"]
    assert inv.tolist() == g["inv_pos"]


@pytest.mark.parametrize("name", ["tiny", "prefill_dsv2_lite", "ep_share_dsv3"])
def test_permute_is_stable_sort_bijection(oracle_mod, name):
    cfg = W.CONFIGS[name]
    cfg = cfg.replace(T=min(cfg.T, 2048))
    r = W.make_routing(cfg, seed=1)
    idx, _ = oracle_mod.route(r["logits"], cfg.k)
    loc = r["local_experts"]
    off, perm, inv = oracle_mod.permute(idx, cfg.E, cfg.E_local, loc)
    slot_of = np.full(cfg.E, -1, np.int64)
    slot_of[np.arange(cfg.E) if loc is None else loc] = np.arange(cfg.E_local)
    slot = slot_of[idx.ravel()]
    local = np.nonzero(slot >= 0)[0]
    R = len(local)
    assert off[-1] == R and off[0] == 0
    np.testing.assert_array_equal(np.diff(off), np.bincount(slot[local], minlength=cfg.E_local))
    order = local[np.argsort(slot[local], kind="stable")]
    np.testing.assert_array_equal(perm, order // cfg.k)
    # bijection between local pairs and rows, and inv_pos inverts perm_token
    assert sorted(inv[local].tolist()) == list(range(R))
    assert (inv[slot < 0] == -1).all()
    np.testing.assert_array_equal(perm[inv[local]], local // cfg.k)
    # every row of segment s belongs to slot s
    row_slot = np.repeat(np.arange(cfg.E_local), np.diff(off))
    np.testing.assert_array_equal(row_slot[inv[local]], slot[local])


def test_permute_rejects_bad_placement(oracle_mod):
    idx = np.array([[0, 1]], np.int32)
    with pytest.raises(oracle_mod.OracleError):
        oracle_mod.permute(idx, 4, 2, np.array([1, 1]))
    with pytest.raises(oracle_mod.OracleError):
        oracle_mod.permute(idx, 4, 2, np.array([1, 4]))


def test_gather_rows(oracle_mod):
    x = np.arange(12, dtype=np.uint16).reshape(4, 3)
    np.testing.assert_array_equal(oracle_mod.gather_rows(x, np.array([3, 0, 3])), x[[3, 0, 3]])


# -------------------------------------------------------------------- FFN ---

def test_ffn_worked_example(oracle_mod):
    g = _load("ffn_worked.json")
    x, wg, wu, wd = (_bf16(g[n]) for n in ("x", "w_gate", "w_up", "w_down"))
    h = oracle_mod.swiglu_hidden(x, wg, wu)
    np.testing.assert_allclose(h, g["h"], rtol=1e-15, atol=1e-15)
    y = oracle_mod.swiglu_ffn(x, wg, wu, wd)
    np.testing.assert_allclose(y, g["y"], rtol=1e-15)


def test_ffn_worked_layer(oracle_mod):
    g = _load("ffn_worked.json")
    L = g["layer"]
    x, wg, wu, wd = (_bf16(g[n]) for n in ("x", "w_gate", "w_up", "w_down"))
    rng = np.random.default_rng(0)
    w = {"w_gate": np.stack([wg, wg, _bf16(rng.standard_normal((3, 2)))]),
         "w_up": np.stack([wu, wu, _bf16(rng.standard_normal((3, 2)))]),
         "w_down": np.stack([wd, _bf16(2 * W.bf16_bits_to_f32(wd)), _bf16(rng.standard_normal((2, 3)))])}
    dims = dict(T=1, H=2, E=3, k=L["k"], I=3, S=1, E_local=3)
    logits = _f32(L["logits"])[None, :]
    out = oracle_mod.forward_tokens(dims, [0], logits, x[None, :], None, w)
    np.testing.assert_allclose(out[0], L["out_all"], rtol=1e-14)
    for loc, key in (([1], "out_only_e1"), ([2], "out_only_e2")):
        sub = {n: v[loc] for n, v in w.items()}
        out = oracle_mod.forward_tokens(dict(dims, E_local=1), [0], logits, x[None, :], np.array(loc), sub)
        np.testing.assert_allclose(out[0], L[key], rtol=1e-14, atol=1e-300)


def _small_expert(rng, H, I, std=0.3):
    return (_bf16(rng.standard_normal((I, H)) * std), _bf16(rng.standard_normal((I, H)) * std),
            _bf16(rng.standard_normal((H, I)) * std))


def test_ffn_linearity_and_gate_up_roles(oracle_mod):
    rng = np.random.default_rng(11)
    H, I = 24, 40                       # H != I: a transposed operand cannot line up
    wg, wu, wd = _small_expert(rng, H, I)
    x = _bf16(rng.standard_normal(H))
    y = oracle_mod.swiglu_ffn(x, wg, wu, wd)
    dbl = lambda a: _bf16(2 * W.bf16_bits_to_f32(a))          # exact in bf16
    np.testing.assert_array_equal(oracle_mod.swiglu_ffn(x, wg, dbl(wu), wd), 2 * y)
    np.testing.assert_array_equal(oracle_mod.swiglu_ffn(x, wg, wu, dbl(wd)), 2 * y)
    # the gate goes through silu, so doubling it is not a doubling of the output
    assert not np.allclose(oracle_mod.swiglu_ffn(x, dbl(wg), wu, wd), 2 * y, rtol=1e-3)
    # relabelling the intermediate units consistently leaves the output unchanged ...
    p = rng.permutation(I)
    np.testing.assert_allclose(oracle_mod.swiglu_ffn(x, wg[p], wu[p], wd[:, p]), y, rtol=1e-12, atol=1e-15)
    # ... and inconsistently does not
    assert not np.allclose(oracle_mod.swiglu_ffn(x, wg[p], wu, wd[:, p]), y, rtol=1e-3)


def _dense_swiglu_numpy(x, wg, wu, wd):
    f = W.bf16_bits_to_f32
    xv = f(x).astype(np.float64)
    g = f(wg).astype(np.float64) @ xv
    u = f(wu).astype(np.float64) @ xv
    return f(wd).astype(np.float64) @ (g / (1.0 + np.exp(-g)) * u)


def test_ffn_matches_numpy_matmul(oracle_mod):
    rng = np.random.default_rng(12)
    H, I = 64, 96
    wg, wu, wd = _small_expert(rng, H, I)
    for _ in range(5):
        x = _bf16(rng.standard_normal(H))
        np.testing.assert_allclose(oracle_mod.swiglu_ffn(x, wg, wu, wd), _dense_swiglu_numpy(x, wg, wu, wd),
                                   rtol=1e-12, atol=1e-14)


def _tiny_layer(rng, T=12, H=16, E=6, k=2, I=24, n_sh=0, I_sh=0):
    dims = dict(T=T, H=H, E=E, k=k, I=I, S=2, E_local=E, n_shared=n_sh, I_shared=I_sh)
    ws = [_small_expert(rng, H, I) for _ in range(E)]
    w = {"w_gate": np.stack([a for a, _, _ in ws]), "w_up": np.stack([b for _, b, _ in ws]),
         "w_down": np.stack([c for _, _, c in ws])}
    if n_sh:
        sh = [_small_expert(rng, H, I_sh) for _ in range(n_sh)]
        w.update(sh_gate=np.stack([a for a, _, _ in sh]), sh_up=np.stack([b for _, b, _ in sh]),
                 sh_down=np.stack([c for _, _, c in sh]))
    x = _bf16(rng.standard_normal((T, H)))
    logits = rng.standard_normal((T, E)).astype(np.float32)
    return dims, w, x, logits


def test_forward_one_hot_gates_is_dense_ffn(oracle_mod):
    rng = np.random.default_rng(13)
    dims, w, x, _ = _tiny_layer(rng)
    T, E = dims["T"], dims["E"]
    chosen = rng.integers(0, E, T)
    logits = np.full((T, E), -np.inf, np.float32)
    logits[np.arange(T), chosen] = 0.0
    out = oracle_mod.forward_tokens(dims, np.arange(T), logits, x, None, w)
    for t in range(T):
        e = chosen[t]
        ref = _dense_swiglu_numpy(x[t], w["w_gate"][e], w["w_up"][e], w["w_down"][e])
        np.testing.assert_allclose(out[t], ref, rtol=1e-12, atol=1e-14)


def test_forward_identical_experts_is_dense_ffn(oracle_mod):
    rng = np.random.default_rng(14)
    dims, w, x, logits = _tiny_layer(rng, k=3)
    E = dims["E"]
    same = {n: np.stack([v[0]] * E) for n, v in w.items()}
    out = oracle_mod.forward_tokens(dims, np.arange(dims["T"]), logits, x, None, same)
    for t in range(dims["T"]):
        ref = _dense_swiglu_numpy(x[t], same["w_gate"][0], same["w_up"][0], same["w_down"][0])
        np.testing.assert_allclose(out[t], ref, rtol=1e-12, atol=1e-14)


def test_forward_placements_add_up(oracle_mod):
    """Expert parallelism: the outputs of GPUs that split the experts between
    them add up to the output of one GPU hosting all of them."""
    rng = np.random.default_rng(15)
    dims, w, x, logits = _tiny_layer(rng, E=7, k=3)
    toks = np.arange(dims["T"])
    full = oracle_mod.forward_tokens(dims, toks, logits, x, None, w)
    parts = [np.array([4, 0, 6]), np.array([2, 5]), np.array([1, 3])]
    acc = np.zeros_like(full)
    for loc in parts:
        sub = {n: v[loc] for n, v in w.items()}
        acc += oracle_mod.forward_tokens(dict(dims, E_local=len(loc)), toks, logits, x, loc, sub)
    np.testing.assert_allclose(acc, full, rtol=1e-12, atol=1e-14)


def test_forward_shared_experts_add(oracle_mod):
    rng = np.random.default_rng(16)
    dims, w, x, logits = _tiny_layer(rng, n_sh=2, I_sh=20)
    toks = np.arange(dims["T"])
    with_sh = oracle_mod.forward_tokens(dims, toks, logits, x, None, w)
    routed = oracle_mod.forward_tokens(dict(dims, n_shared=0, I_shared=0), toks, logits, x, None, w)
    for t in toks:
        ref = sum(_dense_swiglu_numpy(x[t], w["sh_gate"][q], w["sh_up"][q], w["sh_down"][q]) for q in range(2))
        np.testing.assert_allclose(with_sh[t] - routed[t], ref, rtol=1e-11, atol=1e-13)


def test_permuted_pipeline_equals_direct_definition(oracle_mod):
    """route -> permute -> gather -> per-row FFN -> weighted sum reproduces the
    token-by-token definition (which never permutes)."""
    rng = np.random.default_rng(17)
    dims, w, x, logits = _tiny_layer(rng, T=20, E=8, k=3)
    loc = np.array([5, 1, 7, 2])
    sub = {n: v[loc] for n, v in w.items()}
    d = dict(dims, E_local=4)
    idx, gates = oracle_mod.route(logits, d["k"])
    off, perm, inv = oracle_mod.permute(idx, d["E"], 4, loc)
    xp = oracle_mod.gather_rows(x, perm)
    slots = np.repeat(np.arange(4), np.diff(off)).astype(np.int32)
    y = oracle_mod.ffn_rows(xp, slots, sub["w_gate"], sub["w_up"], sub["w_down"])
    out = np.zeros((d["T"], d["H"]))
    for t in range(d["T"]):
        for j in range(d["k"]):
            r = inv[t * d["k"] + j]
            if r >= 0:
                out[t] += gates[t, j] * y[r]
    ref = oracle_mod.forward_tokens(d, np.arange(d["T"]), logits, x, loc, sub)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-14)


def test_combine_definition(oracle_mod):
    rng = np.random.default_rng(18)
    T, k, H, R = 9, 3, 8, 14
    y = _bf16(rng.standard_normal((R, H)))
    ysh = _bf16(rng.standard_normal((T, H)))
    inv = np.full(T * k, -1, np.int32)
    inv[rng.permutation(T * k)[:R]] = np.arange(R)
    w = rng.random((T, k)).astype(np.float32)
    f = lambda a: W.bf16_bits_to_f32(a).astype(np.float64)
    out = oracle_mod.combine(y, inv, w, ysh)
    ref = f(ysh).copy()
    for p in range(T * k):
        if inv[p] >= 0:
            ref[p // k] += float(w.reshape(-1)[p]) * f(y[inv[p]])
    np.testing.assert_allclose(out, ref, rtol=1e-14, atol=1e-15)
    # one-hot gates make it a pure gather; nothing local and no shared part gives zeros
    one = np.zeros((T, k), np.float32)
    one[:, 0] = 1.0
    inv0 = np.arange(T * k, dtype=np.int32) % R
    np.testing.assert_array_equal(oracle_mod.combine(y, inv0, one), f(y[inv0.reshape(T, k)[:, 0]]))
    assert (oracle_mod.combine(y, np.full(T * k, -1, np.int32), w) == 0).all()


def test_forward_tiny_config_matches_numpy_rederivation(oracle_mod):
    """The whole tiny workload against an fp64 numpy re-derivation that uses
    library argsort / matmul for every step."""
    cfg = W.CONFIGS["tiny"]
    wl = W.make_workload(cfg, seed=0)
    toks = np.arange(cfg.T)
    out = oracle_mod.forward_tokens(cfg.dims, toks, wl["logits"], wl["x"], wl["local_experts"], wl)
    f = lambda a: W.bf16_bits_to_f32(a).astype(np.float64)
    order = np.argsort(-wl["logits"], axis=1, kind="stable")[:, : cfg.k]
    sel = np.take_along_axis(wl["logits"].astype(np.float64), order, 1)
    gates = np.exp(sel - sel[:, :1])
    gates /= gates.sum(1, keepdims=True)
    X = f(wl["x"])
    ref = np.zeros((cfg.T, cfg.H))
    for e in range(cfg.E):
        g = X @ f(wl["w_gate"][e]).T
        u = X @ f(wl["w_up"][e]).T
        y = (g / (1 + np.exp(-g)) * u) @ f(wl["w_down"][e]).T
        ref += ((order == e) * gates).sum(1)[:, None] * y
    err = np.abs(out - ref).max() / np.abs(ref).max()
    assert err < 1e-12, err


# ------------------------------------------------------ gating variants ---

def _gcase_arrays(case):
    logits = _f32(case["logits"])[None, :]
    bias = None if case["bias"] is None else _f32(case["bias"])
    return logits, bias


def test_route_gated_worked_examples(oracle_mod):
    g = _load("route_worked.json")
    for case in g["gated_cases"]:
        logits, bias = _gcase_arrays(case)
        idx, w = oracle_mod.route_gated(logits, case["k"], case["gate"], bias, case["scale"],
                                        case["n_group"], case["topk_group"])
        assert idx[0].tolist() == case["idx"], case["note"]
        np.testing.assert_allclose(w[0], case["w"], rtol=0, atol=1e-15, err_msg=case["note"])


def _sigmoid_f32(logits):
    """fp32 rounding of the fp64 logistic function (scipy's expit)."""
    from scipy.special import expit
    return expit(logits.astype(np.float64)).astype(np.float32)


def _unique_top_set(keys, allowed, k):
    """The unique k-subset of allowed ids preceding every other allowed id in
    the total order of the keys (tuples, smaller first): brute force."""
    ids = [e for e in range(len(keys)) if allowed[e]]
    found = [s for s in itertools.combinations(ids, k)
             if max(keys[e] for e in s) < min((keys[e] for e in ids if e not in s), default=(9, 0, 0))]
    assert len(found) == 1
    return set(found[0])


@pytest.mark.parametrize("E,k,n_group,topk_group", [(8, 2, 4, 2), (12, 3, 4, 2), (12, 4, 3, 1), (10, 3, 5, 3),
                                                    (12, 2, 12, 3), (9, 3, 0, 0)])
def test_route_sigmoid_grouped_brute_force(oracle_mod, E, k, n_group, topk_group):
    """Kept groups and selected experts by subset enumeration, on tie-heavy
    rows (quantised logits and biases) with NaN and infinities."""
    rng = np.random.default_rng(E * 1000 + k * 10 + n_group)
    rows = []
    for _ in range(30):
        rows.append((rng.integers(-2, 3, size=E) * 0.5).astype(np.float32))
    for _ in range(15):
        r = rng.standard_normal(E).astype(np.float32)
        r[rng.integers(0, E, size=2)] = rng.choice(np.array([np.nan, -np.inf, np.inf], np.float32), 2)
        rows.append(r)
    logits = np.stack(rows)
    bias = (rng.integers(-2, 3, size=E) * 0.125).astype(np.float32)
    idx, w = oracle_mod.route_gated(logits, k, oracle_mod.GATE_SIGMOID, bias, 2.5, n_group, topk_group)
    s = _sigmoid_f32(logits)
    c = s + bias
    gsz = E // n_group if n_group > 1 else E
    for t in range(len(rows)):
        keys = [_sort_key(c[t, e], e) for e in range(E)]
        allowed = [True] * E
        if n_group > 1:
            gs = []
            for q in range(n_group):
                members = sorted(range(q * gsz, (q + 1) * gsz), key=lambda e: keys[e])
                top = [c[t, e] for e in members[:2]]
                gs.append(np.float32(top[0] + top[1]) if len(top) == 2 else top[0])
            gkeys = [_sort_key(gs[q], q) for q in range(n_group)]
            kept = _unique_top_set(gkeys, [True] * n_group, topk_group)
            allowed = [e // gsz in kept for e in range(E)]
        assert set(idx[t].tolist()) == _unique_top_set(keys, allowed, k)
        assert [keys[e] for e in idx[t]] == sorted(keys[e] for e in idx[t])
        sel = s[t, idx[t]].astype(np.float64)
        if np.isfinite(sel).all() and sel.sum() > 0:
            np.testing.assert_allclose(w[t], 2.5 * sel / sel.sum(), rtol=1e-15)


def test_route_softmax_full_is_library_softmax(oracle_mod):
    from scipy.special import softmax
    rng = np.random.default_rng(11)
    logits = (rng.standard_normal((300, 24)) * 2).astype(np.float32)
    logits[rng.random((300, 24)) < 0.05] = -np.inf
    idx, w = oracle_mod.route_gated(logits, 5, oracle_mod.GATE_SOFTMAX)
    np.testing.assert_array_equal(idx, np.argsort(-logits, axis=1, kind="stable")[:, :5])
    full = softmax(logits.astype(np.float64), axis=1)
    np.testing.assert_allclose(w, np.take_along_axis(full, idx, axis=1), rtol=1e-13, atol=1e-300)
    _, w_all = oracle_mod.route_gated(logits, 24, oracle_mod.GATE_SOFTMAX)
    np.testing.assert_allclose(w_all.sum(axis=1), 1.0, rtol=1e-13)
    assert (w.sum(axis=1) < 1.0 + 1e-12).all()


def test_route_bias_moves_selection_not_gates(oracle_mod):
    """A large bias on a cold expert selects it; its gate stays its sigmoid
    share of the selected scores."""
    logits = np.array([[2.0, 1.0, -6.0, 0.5]], np.float32)
    idx, w = oracle_mod.route_gated(logits, 2, oracle_mod.GATE_SIGMOID)
    assert idx[0].tolist() == [0, 1]
    bias = np.array([0.0, 0.0, 5.0, 0.0], np.float32)
    idx, w = oracle_mod.route_gated(logits, 2, oracle_mod.GATE_SIGMOID, bias)
    assert idx[0].tolist() == [2, 0]
    s = _sigmoid_f32(logits[0]).astype(np.float64)
    np.testing.assert_allclose(w[0], [s[2] / (s[2] + s[0]), s[0] / (s[2] + s[0])], rtol=1e-15)


def test_route_group_limit_special_cases(oracle_mod):
    """One group, or keeping every group, is the ungrouped selection."""
    rng = np.random.default_rng(12)
    logits = np.round(rng.standard_normal((200, 16)) * 3).astype(np.float32)
    bias = (rng.integers(-3, 4, size=16) * 0.25).astype(np.float32)
    ref, wref = oracle_mod.route_gated(logits, 4, oracle_mod.GATE_SIGMOID, bias)
    for n_group, topk_group in ((1, 1), (4, 4), (16, 16), (2, 2)):
        idx, w = oracle_mod.route_gated(logits, 4, oracle_mod.GATE_SIGMOID, bias, 1.0, n_group, topk_group)
        np.testing.assert_array_equal(idx, ref)
        np.testing.assert_array_equal(w, wref)
    # softmax gates under a group limit still take their values from the full softmax
    from scipy.special import softmax
    idx, w = oracle_mod.route_gated(logits, 4, oracle_mod.GATE_SOFTMAX, None, 1.0, 4, 2)
    full = softmax(logits.astype(np.float64), axis=1)
    np.testing.assert_allclose(w, np.take_along_axis(full, idx, axis=1), rtol=1e-13)
    assert ((idx // 4)[:, :, None] == (idx // 4)[:, None, :]).any(axis=2).all()


def test_route_gated_rejects(oracle_mod):
    logits = np.zeros((2, 8), np.float32)
    for args in [dict(gate=3), dict(gate=0, bias=np.zeros(8, np.float32)), dict(gate=2, n_group=3, topk_group=1),
                 dict(gate=2, n_group=4, topk_group=5), dict(gate=2, n_group=4, topk_group=1, k=3)]:
        k = args.pop("k", 2)
        with pytest.raises(oracle_mod.OracleError):
            oracle_mod.route_gated(logits, k, **args)
