"""GPU parity of the dispatch (offsets, perm_token, inv_pos, x_perm) against the
CPU oracle, bit-exact, including the degenerate placements."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2606_15177_amd import workloads as W
from tests.gpu_util import dev, host_bf16

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def moe():
    from paper_2606_15177_amd import moe
    return moe


def _permute(moe, idx, E, E_local, local, x=None):
    T, k = idx.shape
    H = 8 if x is None else x.shape[1]
    d = moe.dims(T=T, H=H, E=E, k=k, I=8, S=1, E_local=E_local)
    cap = max(T * k, 1)
    offsets = torch.full((E_local + 1,), -9, dtype=torch.int32, device="cuda")
    perm = torch.full((cap,), -9, dtype=torch.int32, device="cuda")
    inv = torch.full((cap,), -9, dtype=torch.int32, device="cuda")
    x_d = None if x is None else dev(x)
    xp = None if x is None else torch.zeros((cap, H), dtype=torch.bfloat16, device="cuda")
    ws = moe.workspace(d, moe.ENTRY_PERMUTE)
    moe.permute(d, dev(idx) if T else None, None if local is None else dev(local), x_d, offsets,
                perm if T else None, inv if T else None, xp, ws)
    torch.cuda.synchronize()
    off = offsets.cpu().numpy()
    R = int(off[-1])
    out = (off, perm.cpu().numpy()[:R], inv.cpu().numpy()[:T * k])
    if x is not None:
        out = out + (host_bf16(xp)[:R],)
    return out


def _check(moe, idx, E, E_local, local, x=None):
    got = _permute(moe, idx, E, E_local, local, x)
    off, perm, inv = oracle.permute(idx, E, E_local, local)
    np.testing.assert_array_equal(got[0], off)
    np.testing.assert_array_equal(got[1], perm)
    np.testing.assert_array_equal(got[2], inv)
    if x is not None:
        np.testing.assert_array_equal(got[3], oracle.gather_rows(x, perm))


@pytest.mark.parametrize("name", W.CONFIG_ORDER)
def test_permute_configs(moe, name):
    cfg = W.CONFIGS[name]
    r = W.make_routing(cfg, seed=0)
    idx, _ = oracle.route(r["logits"], cfg.k)
    x = W.make_x(cfg.replace(H=64), seed=0) if cfg.H > 64 else W.make_x(cfg, seed=0)
    _check(moe, idx, cfg.E, cfg.E_local, r["local_experts"], x)


def test_permute_full_width_gather(moe):
    """x_perm at the full hidden size of the expert-parallel share."""
    cfg = W.CONFIGS["ep_share_dsv3"]
    r = W.make_routing(cfg, seed=0)
    idx, _ = oracle.route(r["logits"], cfg.k)
    _check(moe, idx, cfg.E, cfg.E_local, r["local_experts"], W.make_x(cfg, seed=0))


def _rand_idx(rng, T, E, k):
    return np.stack([rng.choice(E, k, replace=False) for _ in range(T)]).astype(np.int32) \
        if T else np.zeros((0, k), np.int32)


@pytest.mark.parametrize("T,E,k,E_local", [
    (1, 8, 2, 8), (1, 8, 2, 3), (3, 4, 4, 4), (255, 16, 2, 5), (257, 64, 6, 64), (1000, 128, 8, 17),
    (4097, 256, 8, 32), (20000, 1024, 7, 1024), (513, 1024, 32, 1),
    # tiles x slots at and just past the bound of the scatter pass's own
    # slot sums, one slot per 4-slot load, and 1024 slots over few tiles
    (8192, 128, 8, 128), (8193, 128, 8, 128), (16384, 8, 2, 4), (300, 1024, 8, 1024),
])
def test_permute_shapes(moe, T, E, k, E_local):
    rng = np.random.default_rng(T + E + k)
    idx = _rand_idx(rng, T, E, k)
    local = None if E_local == E and T % 2 else rng.choice(E, E_local, replace=False).astype(np.int32)
    _check(moe, idx, E, E_local, local, rng.integers(0, 65535, (T, 16)).astype(np.uint16))


def test_permute_degenerate(moe):
    rng = np.random.default_rng(1)
    T, E, k = 700, 16, 2
    # every token on the same two experts
    idx = np.tile(np.array([[3, 11]], np.int32), (T, 1))
    _check(moe, idx, E, E, None)
    _check(moe, idx, E, 4, np.array([11, 0, 1, 3], np.int32))
    # hosted experts that receive no token, and a GPU that receives none at all
    _check(moe, idx, E, 3, np.array([5, 6, 7], np.int32))
    _check(moe, _rand_idx(rng, T, E, k), E, 1, np.array([9], np.int32))
    # expert ids out of range are treated as remote: the oracle sees them as one
    # extra expert (id E) that this GPU does not host
    bad = _rand_idx(rng, T, E, k)
    bad[::5, 1] = E + 2
    bad[1::9, 0] = -4
    got = _permute(moe, bad, E, E, None)
    mapped = np.where((bad < 0) | (bad >= E), E, bad).astype(np.int32)
    off, perm, inv = oracle.permute(mapped, E + 1, E, np.arange(E, dtype=np.int32))
    np.testing.assert_array_equal(got[0], off)
    np.testing.assert_array_equal(got[1], perm)
    np.testing.assert_array_equal(got[2], inv)


def test_permute_empty(moe):
    d = moe.dims(T=0, H=8, E=8, k=2, I=8, S=1, E_local=8)
    offsets = torch.full((9,), -9, dtype=torch.int32, device="cuda")
    ws = moe.workspace(d, moe.ENTRY_PERMUTE)
    moe.permute(d, None, None, None, offsets, None, None, None, ws)
    torch.cuda.synchronize()
    assert (offsets.cpu().numpy() == 0).all()
