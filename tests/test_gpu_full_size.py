"""Full-size parity of the layer over every tile of the expert GEMMs.

At each workload's full size, in the launch configuration the benchmark
times, the GPU results are compared with the CPU oracle:
  - moe_forward: every routing intermediate over all tokens, bit-exact, and
    the layer output of a token set that covers every (local expert, m-tile)
    of the routed GEMMs (a token of one row of each tile, plus each expert's
    first and last rows), every 256-token m-tile of the shared experts, and
    tokens none of whose experts are hosted here;
  - moe_expert_ffn on the oracle's own dispatch: the rows of the same tile
    cover, each against the oracle's per-row FFN, and the shared experts'
    output on one token of every m-tile.
The per-row oracle runs in host threads (the C oracle is reentrant; ctypes
releases the interpreter lock), each on a disjoint slice of the rows."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2606_15177_amd import workloads as W
from tests.gpu_util import (assert_gates_close, assert_layer_close, dev, dev_weights, gating_cfg, host_bf16,
                            oracle_route_cfg, parallel_rows)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

M_TILE = 256      # token rows of an m-tile of the tiled grouped GEMM
CHUNK = 32        # token rows of a chunk of the weight-streaming GEMM
NAMES = W.CONFIG_ORDER + ["ep_share_dsv3_v3router"]


def tile_rows(off, tile: int, seed: int) -> np.ndarray:
    """One row of every (group, m-tile) -- a random row inside the tile --
    plus the first and last row of every group."""
    rng = np.random.default_rng(seed)
    rows = []
    for s in range(len(off) - 1):
        a, b = int(off[s]), int(off[s + 1])
        for m0 in range(a, b, tile):
            rows.append(int(rng.integers(m0, min(m0 + tile, b))))
        if b > a:
            rows += [a, b - 1]
    return np.unique(np.asarray(rows, np.int64))


def shared_tile_tokens(T: int, seed: int) -> np.ndarray:
    """One token of every 256-token m-tile of the shared experts, plus the
    first and last token."""
    rng = np.random.default_rng(seed)
    toks = [int(rng.integers(m0, min(m0 + M_TILE, T))) for m0 in range(0, T, M_TILE)]
    return np.unique(np.asarray(toks + [0, T - 1], np.int64))


@pytest.fixture(scope="module", params=NAMES)
def full(request):
    name = request.param
    cfg = W.CONFIGS[name]
    wl = W.make_workload(cfg, 0)
    ridx, rw = oracle_route_cfg(cfg, wl)
    off, perm, inv = oracle.permute(ridx, cfg.E, cfg.E_local, wl["local_experts"])
    # small batches are checked row by row; otherwise one row per tile of the
    # tiled kernel (above 64 rows per expert) or the weight-streaming one
    tile = 1 if off[-1] <= 1024 else (CHUNK if cfg.T <= 64 else M_TILE)
    yield dict(cfg=cfg, wl=wl, ridx=ridx, rw=rw, off=off, perm=perm, inv=inv, tile=tile)


def _oracle_forward(cfg, wl, toks):
    def one(part):
        return oracle.forward_tokens(cfg.dims, part.astype(np.int32), wl["logits"], wl["x"],
                                     wl["local_experts"], wl, gate=cfg.gate, bias=wl.get("gate_bias"),
                                     scale=cfg.routed_scale, n_group=cfg.n_group, topk_group=cfg.topk_group)
    return parallel_rows(one, toks)


def test_forward_every_tile(full):
    from paper_2606_15177_amd import moe
    cfg, wl, off, perm = full["cfg"], full["wl"], full["off"], full["perm"]
    T, k = cfg.T, cfg.k
    d = moe.dims_of(cfg)
    taps_t = dict(topk_idx=torch.full((T, k), -9, dtype=torch.int32, device="cuda"),
                  topk_w=torch.zeros((T, k), dtype=torch.float32, device="cuda"),
                  expert_load=torch.full((cfg.E,), -9, dtype=torch.int32, device="cuda"),
                  offsets=torch.full((cfg.E_local + 1,), -9, dtype=torch.int32, device="cuda"),
                  perm_token=torch.full((T * k,), -9, dtype=torch.int32, device="cuda"),
                  inv_pos=torch.full((T * k,), -9, dtype=torch.int32, device="cuda"))
    loc = None if wl["local_experts"] is None else dev(wl["local_experts"])
    gating, _bias = gating_cfg(moe, cfg, wl)
    layer = moe.MoeLayer(d, dev_weights(wl), loc, gating=gating)
    counts = torch.zeros((cfg.S, cfg.E), dtype=torch.int64, device="cuda")
    out = torch.full((T, cfg.H), 3.0, dtype=torch.bfloat16, device="cuda")
    layer.forward(dev(wl["logits"]), dev(wl["src"]), dev(wl["x"]), counts, out, moe.make_taps(**taps_t))
    torch.cuda.synchronize()
    res = {n: t.cpu().numpy() for n, t in taps_t.items()}

    # routing, statistics and dispatch: bit-exact over all tokens
    np.testing.assert_array_equal(res["topk_idx"], full["ridx"])
    assert_gates_close(res["topk_w"], full["rw"], cfg.name)
    rc, rl = oracle.route_stats(wl["src"], full["ridx"], cfg.S, cfg.E)
    np.testing.assert_array_equal(counts.cpu().numpy(), rc)
    np.testing.assert_array_equal(res["expert_load"], rl)
    np.testing.assert_array_equal(res["offsets"], off)
    np.testing.assert_array_equal(res["perm_token"][: off[-1]], perm)
    np.testing.assert_array_equal(res["inv_pos"], full["inv"])

    # output: tokens covering every routed tile, every shared m-tile and the
    # tokens with no local expert
    toks = set(perm[tile_rows(off, full["tile"], seed=1)].tolist()) if off[-1] else set()
    if T <= 256:
        toks = set(range(T))
    if cfg.n_shared:
        toks |= set(shared_tile_tokens(T, seed=2).tolist())
    no_local = np.flatnonzero((full["inv"].reshape(T, k) < 0).all(axis=1))
    toks |= set(no_local[:4].tolist())
    toks = np.array(sorted(toks), np.int64)
    ref = _oracle_forward(cfg, wl, toks)
    e = assert_layer_close(host_bf16(out)[toks], ref, cfg.name)
    print(f"{cfg.name}: {len(toks)} tokens, rel {e['rel']:.2e} rel_mae {e['rel_mae']:.2e}")


def test_expert_ffn_every_tile(full):
    """moe_expert_ffn on the oracle's dispatch (the rows already gathered):
    one row of every (local expert, m-tile) against the oracle's per-row FFN."""
    from paper_2606_15177_amd import moe
    cfg, wl, off, perm = full["cfg"], full["wl"], full["off"], full["perm"]
    R, cap = int(off[-1]), cfg.T * cfg.k
    xp = oracle.gather_rows(wl["x"], perm)
    x_perm = torch.zeros((cap, cfg.H), dtype=torch.bfloat16, device="cuda")
    if R:
        x_perm[:R] = dev(xp)
    y_perm = torch.full((cap, cfg.H), 5.0, dtype=torch.bfloat16, device="cuda")
    ysh = torch.full((cfg.T, cfg.H), 5.0, dtype=torch.bfloat16, device="cuda") if cfg.n_shared else None
    d = moe.dims_of(cfg)
    ws = moe.workspace(d, moe.ENTRY_EXPERT_FFN)
    moe.expert_ffn(d, x_perm, dev(off), dev_weights(wl), dev(wl["x"]) if cfg.n_shared else None, y_perm, ysh, ws)
    torch.cuda.synchronize()

    rows = tile_rows(off, full["tile"], seed=3)
    slots = np.repeat(np.arange(cfg.E_local, dtype=np.int32), np.diff(off))

    def per_rows(part):
        return oracle.ffn_rows(xp[part], slots[part], wl["w_gate"], wl["w_up"], wl["w_down"])
    ref = parallel_rows(per_rows, rows)
    e = assert_layer_close(host_bf16(y_perm)[rows], ref, f"{cfg.name} y_perm")
    print(f"{cfg.name}: {len(rows)} routed rows, rel {e['rel']:.2e}")

    if cfg.n_shared:
        toks = shared_tile_tokens(cfg.T, seed=4)

        def per_tok(part):
            y = np.zeros((len(part), cfg.H))
            for i, t in enumerate(part):
                for q in range(cfg.n_shared):
                    y[i] += oracle.swiglu_ffn(wl["x"][t], wl["sh_gate"][q], wl["sh_up"][q], wl["sh_down"][q])
            return y
        ref_sh = parallel_rows(per_tok, toks)
        e = assert_layer_close(host_bf16(ysh)[toks], ref_sh, f"{cfg.name} y_shared")
        print(f"{cfg.name}: {len(toks)} shared rows, rel {e['rel']:.2e}")
