"""Pins for the placement oracle (Sec. 5.2 objective, Sec. 5.3 greedy): a hand-
worked instance built from the paper's example statistics, brute-force
minimisation of the objective where the greedy is provably optimal, the
textbook LPT list schedule that the load term reduces to, an identity tying
the greedy's per-step scores to the objective, and the tie rules.  Never
checked against itself or the HIP path.  CPU only."""
import heapq
import itertools
import json
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
PAPER_WEIGHTS = (1.0, 0.0025, 1.0)  # (alpha, beta, gamma), Sec. 6


def _golden():
    with open(os.path.join(GOLDEN, "place_worked.json")) as f:
        return json.load(f)


def _random_instance(rng, L, S, E, G, hot=1000, home_ok=True, with_m=True):
    A = rng.integers(0, hot, size=(L, S, E)).astype(np.int64)
    D = rng.uniform(0.0, 2.0, size=(S, G))
    M = rng.uniform(0.0, 50.0, size=(L, E, G)) if with_m else None
    x0 = rng.integers(0, G, size=(L, E)).astype(np.int32)
    if not home_ok:
        x0[rng.random(size=(L, E)) < 0.3] = -1
    return A, D, M, x0


# ------------------------------------------------------- worked example ----

def test_objective_worked_example(oracle_mod):
    g = _golden()
    for case in g["objective_cases"]:
        terms = oracle_mod.place_objective(np.array(g["A"]), np.array(g["D"]), np.array(case["x"]),
                                           np.array(g["x0"]), B=np.array(g["B"]),
                                           m_uniform=g["m_uniform"])
        assert terms[0].tolist() == case["terms"], case["derivation"]


def test_greedy_worked_example(oracle_mod):
    g = _golden()
    a, b, c = g["weights"]
    x, score = oracle_mod.place_greedy(np.array(g["A"]), np.array(g["D"]), np.array(g["x0"]),
                                       np.array(g["cap"]), B=np.array(g["B"]), m_uniform=g["m_uniform"],
                                       alpha=a, beta=b, gamma=c)
    assert x[0].tolist() == g["greedy"]["x"], g["greedy"]["derivation"]
    # first step, rank 1: 478 + 0.0025 * (-22413928284) + 2 (hand arithmetic)
    assert score[0][0] == pytest.approx(478 - 56034820.71 + 2, abs=1e-6)


# ------------------------------------------- objective closed forms ---------

def test_objective_balanced_and_unmoved_are_zero(oracle_mod):
    A = np.array([[[3, 0, 5, 1]]], np.int64)
    B = np.array([[7, 7, 4, 10]], np.int64)   # {7, 7} | {4, 10}: equal loads
    D = np.zeros((1, 2))
    x = np.array([[0, 0, 1, 1]], np.int32)
    t = oracle_mod.place_objective(A, D, x, x, B=B)
    assert t[0].tolist() == [0.0, 0.0, 0.0]


def test_objective_uniform_migration_counts_moves(oracle_mod):
    rng = np.random.default_rng(7)
    for _ in range(20):
        E, G = 9, 4
        x0 = rng.integers(0, G, size=(1, E)).astype(np.int32)
        x = rng.integers(0, G, size=(1, E)).astype(np.int32)
        t = oracle_mod.place_objective(np.zeros((1, 1, E), np.int64), np.zeros((1, G)), x, x0,
                                       m_uniform=3.5)
        assert t[0, 2] == 2 * 3.5 * int((x != x0).sum())


def test_objective_load_variance_closed_form(oracle_mod):
    """C_load = G * population variance of the rank loads (numpy)."""
    rng = np.random.default_rng(8)
    for _ in range(20):
        E, G = 11, 3
        B = rng.integers(0, 10**6, size=(1, E)).astype(np.int64)
        x = rng.integers(0, G, size=(1, E)).astype(np.int32)
        loads = np.bincount(x[0], weights=B[0].astype(np.float64), minlength=G)
        t = oracle_mod.place_objective(np.zeros((1, 1, E), np.int64), np.zeros((1, G)), x, x, B=B)
        assert t[0, 1] == pytest.approx(G * np.var(loads), rel=1e-12)


def test_objective_comm_is_traffic_to_remote_ranks(oracle_mod):
    """With D = 1 - [rank g is source s's own], C_comm counts the tokens that
    leave their source's rank (the traffic of Fig. 4)."""
    rng = np.random.default_rng(9)
    S = G = 4
    A = rng.integers(0, 100, size=(1, S, 10)).astype(np.int64)
    x = rng.integers(0, G, size=(1, 10)).astype(np.int32)
    D = 1.0 - np.eye(S)
    remote = sum(int(A[0, s, e]) for s in range(S) for e in range(10) if x[0, e] != s)
    t = oracle_mod.place_objective(A, D, x, x, B=np.zeros((1, 10), np.int64))
    assert t[0, 0] == remote


# -------------------------------------------- greedy vs brute force ---------

def _brute_force_min(oracle_mod, A, B, D, M, x0, cap, w):
    E = A.shape[2]
    G = D.shape[1]
    best = None
    for assign in itertools.product(range(G), repeat=E):
        counts = np.bincount(assign, minlength=G)
        if (counts > cap).any():
            continue
        x = np.array([assign], np.int32)
        t = oracle_mod.place_objective(A, D, x, x0, B=B, M=M)[0]
        f = w[0] * t[0] + w[1] * t[1] + w[2] * t[2]
        if best is None or f < best:
            best = f
    return best


@pytest.mark.parametrize("seed", range(6))
def test_greedy_optimal_when_objective_separates(oracle_mod, seed):
    """beta = 0 with capacities that never bind: the objective is a sum of
    per-expert terms, so placing each expert at its own best rank (the greedy)
    reaches the brute-force minimum over all G^E placements."""
    rng = np.random.default_rng(100 + seed)
    E, G, S = 6, 3, 3
    A, D, M, x0 = _random_instance(rng, 1, S, E, G, home_ok=seed % 2 == 0)
    cap = np.full(G, E, np.int32)
    w = (1.0, 0.0, 1.0)
    x, _ = oracle_mod.place_greedy(A, D, x0, cap, M=M, alpha=w[0], beta=w[1], gamma=w[2])
    t = oracle_mod.place_objective(A, D, x, x0, M=M)[0]
    got = w[0] * t[0] + w[2] * t[2]
    assert got == pytest.approx(_brute_force_min(oracle_mod, A, None, D, M, x0, cap, w), rel=1e-12, abs=1e-9)


@pytest.mark.parametrize("E,G", [(6, 2), (6, 3), (8, 4), (9, 3)])
def test_greedy_balances_equal_loads(oracle_mod, E, G):
    """Equal loads, load term only, capacity E/G: the greedy fills every rank
    with E/G experts, the brute-force optimum (C_load = 0)."""
    rng = np.random.default_rng(E * 10 + G)
    B = np.full((1, E), 1234, np.int64)
    A = rng.integers(0, 50, size=(1, 2, E)).astype(np.int64)
    x0 = rng.integers(0, G, size=(1, E)).astype(np.int32)
    cap = np.full(G, E // G, np.int32)
    x, _ = oracle_mod.place_greedy(A, np.ones((2, G)), x0, cap, B=B, alpha=0.0, beta=1.0, gamma=0.0)
    assert np.bincount(x[0], minlength=G).tolist() == [E // G] * G
    t = oracle_mod.place_objective(A, np.ones((2, G)), x, x0, B=B)[0]
    assert t[1] == 0.0 == _brute_force_min(oracle_mod, A, B, np.ones((2, G)), None, x0, cap, (0.0, 1.0, 0.0))


@pytest.mark.parametrize("seed", range(4))
def test_greedy_never_beats_brute_force(oracle_mod, seed):
    rng = np.random.default_rng(200 + seed)
    E, G, S = 6, 3, 2
    A, D, M, x0 = _random_instance(rng, 1, S, E, G)
    cap = np.array([2, 3, 2], np.int32)
    x, _ = oracle_mod.place_greedy(A, D, x0, cap, M=M, alpha=1.0, beta=1e-4, gamma=1.0)
    t = oracle_mod.place_objective(A, D, x, x0, M=M)[0]
    got = t[0] + 1e-4 * t[1] + t[2]
    assert got >= _brute_force_min(oracle_mod, A, None, D, M, x0, cap, (1.0, 1e-4, 1.0)) - 1e-9


# ------------------------------------------------ textbook reduction --------

def _lpt(loads, G):
    """Graham's LPT list schedule: jobs by size descending (then index), each
    to the machine with the least load so far (then the lower index)."""
    heap = [(0, g) for g in range(G)]
    out = [None] * len(loads)
    for e in sorted(range(len(loads)), key=lambda e: (-loads[e], e)):
        load, g = heapq.heappop(heap)
        out[e] = g
        heapq.heappush(heap, (load + loads[e], g))
    return out


@pytest.mark.parametrize("E,G", [(10, 3), (32, 4), (64, 8), (40, 7)])
def test_load_term_alone_is_lpt(oracle_mod, E, G):
    """alpha = gamma = 0, no capacity limit, nothing placed before: the load
    term B (2 (L_g - Lbar) + B) is smallest on the least-loaded rank, so the
    greedy is LPT scheduling (loads of at least 1000 and below 2^26 keep
    rounding far below the smallest gap between two ranks' scores)."""
    rng = np.random.default_rng(E + 1000 * G)
    B = rng.choice(np.arange(1000, 10**6), size=E, replace=False).astype(np.int64)[None]
    A = np.zeros((1, 1, E), np.int64)
    x0 = np.full((1, E), -1, np.int32)
    x, _ = oracle_mod.place_greedy(A, np.zeros((1, G)), x0, np.full(G, E, np.int32), B=B,
                                   alpha=0.0, beta=1.0, gamma=0.0)
    assert x[0].tolist() == _lpt(B[0].tolist(), G)


# ------------------------------------------------- telescoping identity -----

@pytest.mark.parametrize("seed", range(8))
def test_step_scores_add_up_to_objective(oracle_mod, seed):
    """Every per-step term is the growth of its objective term when the expert
    joins its rank, so the winning scores add up to
    alpha C_comm + beta (C_load - G Lbar^2) + gamma C_mig of the result."""
    rng = np.random.default_rng(300 + seed)
    L, S, E, G = 3, 4, 24, 5
    A, D, M, x0 = _random_instance(rng, L, S, E, G, home_ok=seed % 2 == 1, with_m=seed % 3 != 0)
    B = None if seed % 2 else rng.integers(0, 5000, size=(L, E)).astype(np.int64)
    cap = np.array([5, 6, 4, 5, 7], np.int32)
    a, b, c = (1.0, 0.003, 0.7)
    x, score = oracle_mod.place_greedy(A, D, x0, cap, B=B, M=M, m_uniform=2.5, alpha=a, beta=b, gamma=c)
    t = oracle_mod.place_objective(A, D, x, x0, B=B, M=M, m_uniform=2.5)
    for l in range(L):
        bl = A[l].sum(0) if B is None else B[l]
        mean = bl.sum() / G
        want = a * t[l, 0] + b * (t[l, 1] - G * mean * mean) + c * t[l, 2]
        assert score[l].sum() == pytest.approx(want, rel=1e-9, abs=1e-6)


# ----------------------------------------------- order, ties, capacity ------

def test_hottest_expert_gets_the_cheap_rank(oracle_mod):
    """Capacity 1 per rank and rank 0 free for every source: the hotter expert
    (more aggregate load; equal load -> more source volume; then lower index)
    is placed first and takes rank 0."""
    D = np.array([[0.0, 5.0]])
    x0 = np.full((1, 2), -1, np.int32)
    cap = np.array([1, 1], np.int32)
    cases = [  # (B, A row), expected hotter expert
        (([10, 20], [1, 1]), 1),
        (([20, 10], [1, 1]), 0),
        (([20, 20], [3, 4]), 1),   # equal B: more source volume
        (([20, 20], [4, 4]), 0),   # all equal: lower index
    ]
    for (b, a_row), hot in cases:
        x, _ = oracle_mod.place_greedy(np.array([[a_row]], np.int64), D, x0, cap,
                                       B=np.array([b], np.int64), alpha=1.0, beta=0.0, gamma=0.0)
        assert x[0, hot] == 0 and x[0, 1 - hot] == 1, (b, a_row)


def test_ties_prefer_home_then_fewer_then_lower_rank(oracle_mod):
    """All scores zero: each expert stays on its current rank while it has
    room; otherwise it goes to the rank with fewest experts, then the lower
    index (worked by hand, experts visited 0..5 since all are equally hot)."""
    E, G = 6, 3
    x0 = np.array([[2, 2, 2, -1, -1, 0]], np.int32)
    x, score = oracle_mod.place_greedy(np.zeros((1, 1, E), np.int64), np.zeros((1, G)), x0,
                                       np.full(G, 2, np.int32), M=np.zeros((1, E, G)),
                                       alpha=1.0, beta=1.0, gamma=1.0)
    assert x[0].tolist() == [2, 2, 0, 1, 0, 1]
    assert (score == 0).all()


def test_migration_weight_keeps_current_placement(oracle_mod):
    """A migration cost far above the other terms keeps every expert home."""
    rng = np.random.default_rng(11)
    E, G = 16, 4
    A, D, _, _ = _random_instance(rng, 1, 2, E, G)
    x0 = np.repeat(np.arange(G, dtype=np.int32), E // G)[None]
    x, _ = oracle_mod.place_greedy(A, D, x0, np.full(G, E // G, np.int32), m_uniform=1e12,
                                   alpha=1.0, beta=1e-6, gamma=1.0)
    assert (x == x0).all()


def test_nan_score_loses_to_any_number(oracle_mod):
    """A NaN score counts as +inf: the rank with a finite score wins."""
    D = np.array([[np.nan, 7.0]])
    x, _ = oracle_mod.place_greedy(np.array([[[3]]], np.int64), D, np.array([[0]], np.int32),
                                   np.array([1, 1], np.int32), alpha=1.0, beta=0.0, gamma=0.0)
    assert x[0, 0] == 1


@pytest.mark.parametrize("seed", range(5))
def test_capacity_and_bijection(oracle_mod, seed):
    rng = np.random.default_rng(400 + seed)
    L, S, E, G = 4, 3, 37, 6
    A, D, M, x0 = _random_instance(rng, L, S, E, G, home_ok=False)
    cap = rng.integers(0, 12, size=G).astype(np.int32)
    cap[0] = max(cap[0], E - int(np.minimum(cap[1:], E).sum()))
    x, _ = oracle_mod.place_greedy(A, D, x0, cap, M=M, alpha=1.0, beta=1e-5, gamma=1.0)
    for l in range(L):
        assert ((x[l] >= 0) & (x[l] < G)).all()
        assert (np.bincount(x[l], minlength=G) <= cap).all()


def test_infeasible_capacity_is_rejected(oracle_mod):
    with pytest.raises(oracle_mod.OracleError):
        oracle_mod.place_greedy(np.zeros((1, 1, 5), np.int64), np.zeros((1, 2)), np.zeros((1, 5), np.int32),
                                np.array([2, 2], np.int32))


# ------------------------------------------------- window diagnostics -------

def test_window_worked_example(oracle_mod):
    g = _golden()
    w = g["window"]
    remote, total, rank_load, pressure = oracle_mod.window_stats(
        np.array(g["A"]), np.array(w["x"]), np.array(w["home"]), 2, B=np.array(g["B"]))
    assert remote[0].tolist() == w["remote"], w["derivation"]
    assert total[0].tolist() == w["total"]
    assert rank_load[0].tolist() == w["rank_load"]
    assert pressure.tolist() == pytest.approx([a / b for a, b in w["pressure_fraction"]], rel=1e-15)


@pytest.mark.parametrize("seed", range(4))
def test_window_remote_is_objective_comm(oracle_mod, seed):
    """With D_{s,g} = [g is not source s's rank], the remote tokens of all
    sources add up to the objective's C_comm (an independent function)."""
    rng = np.random.default_rng(500 + seed)
    L, S, E, G = 3, 6, 20, 4
    A = rng.integers(0, 1000, size=(L, S, E)).astype(np.int64)
    x = rng.integers(0, G, size=(L, E)).astype(np.int32)
    home = rng.integers(0, G, size=S).astype(np.int32)
    D = np.ones((S, G))
    D[np.arange(S), home] = 0.0
    remote, total, _, _ = oracle_mod.window_stats(A, x, home, G)
    terms = oracle_mod.place_objective(A, D, x, x)
    assert remote.sum(axis=1).tolist() == terms[:, 0].tolist()
    assert (total == A.sum(axis=2)).all()


@pytest.mark.parametrize("seed", range(4))
def test_window_loads_and_pressure(oracle_mod, seed):
    rng = np.random.default_rng(600 + seed)
    L, S, E, G = 4, 3, 24, 6
    A = rng.integers(0, 500, size=(L, S, E)).astype(np.int64)
    B = rng.integers(0, 9000, size=(L, E)).astype(np.int64) if seed % 2 else None
    x = rng.integers(0, G, size=(L, E)).astype(np.int32)
    _, _, rank_load, pressure = oracle_mod.window_stats(A, x, np.zeros(S, np.int32), G, B=B)
    load = A.sum(axis=1) if B is None else B
    assert (rank_load.sum(axis=1) == load.sum(axis=1)).all()
    for l in range(L):
        assert rank_load[l].tolist() == np.bincount(x[l], weights=load[l], minlength=G).astype(np.int64).tolist()
    assert pressure.mean() == pytest.approx(1.0, rel=1e-12)
    assert pressure.tolist() == pytest.approx((rank_load.sum(0) / rank_load.sum(0).mean()).tolist(), rel=1e-15)
    # two engines of three ranks each (TP groups): pressure of the sums
    engine = np.array([0, 0, 0, 1, 1, 1], np.int32)
    _, _, _, p2 = oracle_mod.window_stats(A, x, np.zeros(S, np.int32), G, B=B, engine=engine, n_eng=2)
    per = rank_load.sum(0)
    eng = np.array([per[:3].sum(), per[3:].sum()], np.float64)
    assert p2.tolist() == pytest.approx((eng / eng.mean()).tolist(), rel=1e-15)


def test_window_all_experts_home(oracle_mod):
    """Every expert on source 2's rank: nothing of source 2 is remote, all of
    every other source is; only that rank carries load."""
    rng = np.random.default_rng(7)
    L, S, E, G = 2, 4, 10, 4
    A = rng.integers(1, 100, size=(L, S, E)).astype(np.int64)
    home = np.arange(S, dtype=np.int32)
    remote, total, rank_load, pressure = oracle_mod.window_stats(A, np.full((L, E), 2, np.int32), home, G)
    assert (remote[:, 2] == 0).all()
    assert (remote[:, [0, 1, 3]] == total[:, [0, 1, 3]]).all()
    assert (rank_load[:, [0, 1, 3]] == 0).all()
    assert pressure.tolist() == [0.0, 0.0, 4.0, 0.0]


def test_window_unplaced_and_homeless(oracle_mod):
    """An expert hosted nowhere is remote for every source and loads no rank;
    a source without a rank has all of its traffic remote; no load at all
    gives zero pressure."""
    A = np.array([[[5, 7, 11]]], np.int64)
    remote, total, rank_load, pressure = oracle_mod.window_stats(A, np.array([[0, -1, 9]]), np.array([0]), 2)
    assert remote.tolist() == [[18]] and total.tolist() == [[23]] and rank_load.tolist() == [[5, 0]]
    remote, _, _, _ = oracle_mod.window_stats(A, np.array([[0, 0, 1]]), np.array([-3]), 2)
    assert remote.tolist() == [[23]]
    _, _, _, pressure = oracle_mod.window_stats(np.zeros((1, 1, 3), np.int64), np.array([[0, 1, 1]]),
                                                np.array([0]), 2)
    assert pressure.tolist() == [0.0, 0.0]
