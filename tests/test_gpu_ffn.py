"""GPU parity of the expert FFN grouped GEMMs (weight-streaming path for
decode-sized batches, LDS-tiled MFMA path for larger ones) and of the combine
kernel against the CPU oracle."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2606_15177_amd import workloads as W
from tests.gpu_util import assert_layer_close, bf16_f64, dev, dev_weights, host_bf16, parallel_rows

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def moe():
    from paper_2606_15177_amd import moe
    return moe


def _case(T, H, E, k, I, E_local, n_sh=0, I_sh=0, seed=0, idx=None, local=None):
    cfg = W.MoeConfig("t", T=T, H=H, E=E, k=k, I=I, S=2, E_local=E_local, n_shared=n_sh,
                      I_shared=I_sh, local_layout="all" if E_local == E else "choice")
    wl = W.make_workload(cfg, seed)
    if local is not None:
        wl["local_experts"] = np.asarray(local, np.int32)
        wl.update(W.make_weights(cfg, seed, experts=local))
    if idx is None:
        idx, _ = oracle.route(wl["logits"], k)
    return cfg, wl, idx


def _run_ffn(moe, cfg, wl, idx):
    """Dispatch with the oracle, run moe_expert_ffn, compare every row."""
    off, perm, inv = oracle.permute(idx, cfg.E, cfg.E_local, wl["local_experts"])
    R = int(off[-1])
    xp = oracle.gather_rows(wl["x"], perm)
    cap = cfg.T * cfg.k
    x_perm = torch.zeros((cap, cfg.H), dtype=torch.bfloat16, device="cuda")
    if R:
        x_perm[:R] = dev(xp)
    y_perm = torch.zeros((cap, cfg.H), dtype=torch.bfloat16, device="cuda")
    d = moe.dims_of(cfg)
    ysh = torch.zeros((cfg.T, cfg.H), dtype=torch.bfloat16, device="cuda") if cfg.n_shared else None
    ws = moe.workspace(d, moe.ENTRY_EXPERT_FFN)
    moe.expert_ffn(d, x_perm, dev(off), dev_weights(wl), dev(wl["x"]) if cfg.n_shared else None,
                   y_perm, ysh, ws)
    torch.cuda.synchronize()
    slots = np.repeat(np.arange(cfg.E_local), np.diff(off)).astype(np.int32)
    if R:
        ref = parallel_rows(lambda p: oracle.ffn_rows(xp[p], slots[p], wl["w_gate"], wl["w_up"], wl["w_down"]),
                            np.arange(R))
        assert_layer_close(host_bf16(y_perm)[:R], ref, "y_perm")
    if cfg.n_shared:
        def shared_rows(part):
            y = np.zeros((len(part), cfg.H))
            for i, t in enumerate(part):
                for q in range(cfg.n_shared):
                    y[i] += oracle.swiglu_ffn(wl["x"][t], wl["sh_gate"][q], wl["sh_up"][q], wl["sh_down"][q])
            return y
        ref_sh = parallel_rows(shared_rows, np.arange(cfg.T))
        assert_layer_close(host_bf16(ysh), ref_sh, "y_shared")
    return R


@pytest.mark.parametrize("T,H,E,k,I,E_local,n_sh,I_sh", [
    # weight-streaming path (T <= 64)
    (16, 256, 8, 2, 512, 8, 0, 0),
    (64, 136, 4, 2, 200, 4, 0, 0),           # K and N not multiples of the tile
    (40, 512, 8, 2, 256, 3, 2, 72),          # remote experts, shared experts over a split K
    (1, 128, 8, 2, 128, 8, 1, 64),
    # LDS-tiled path
    (300, 256, 8, 2, 384, 8, 0, 0),
    (257, 200, 6, 3, 136, 6, 0, 0),          # ragged K, N and M
    (200, 128, 16, 4, 256, 5, 2, 200),       # shared experts over a split K
    (1500, 512, 64, 6, 192, 64, 1, 192),     # many groups, a few rows each
    # K >= 4096: the half tail tiles (128 x 256), gate/up and down
    (500, 4096, 3, 2, 256, 3, 0, 0),
    (500, 256, 3, 2, 4096, 3, 0, 0),
    (500, 4096, 3, 2, 200, 3, 0, 0),         # ... with ragged N
    (500, 200, 3, 2, 4096, 3, 0, 0),
    # the shared experts' tiles in the routed launch, groups with short
    # remainders (whole tiles there), short and long K
    (500, 256, 3, 2, 256, 3, 1, 256),
    (500, 4096, 3, 2, 256, 3, 1, 200),
    (500, 200, 3, 2, 4096, 3, 1, 4096),
    # the tiled kernel's group lookup holds 1, 4 or 16 prefix entries per lane
    (2048, 128, 128, 8, 128, 128, 0, 0),     # 65..256 groups
    (4096, 128, 300, 8, 128, 300, 0, 0),     # 257..1024 groups
    (8192, 64, 1024, 8, 64, 1024, 0, 0),     # the largest group count
    (600, 16, 4, 2, 8, 4, 0, 0),             # one partial K stage, a partial column tile
    (520, 24, 2, 1, 24, 2, 1, 16),           # small shared expert next to the routed ones
])
def test_ffn_paths(moe, T, H, E, k, I, E_local, n_sh, I_sh):
    cfg, wl, idx = _case(T, H, E, k, I, E_local, n_sh, I_sh)
    _run_ffn(moe, cfg, wl, idx)


@pytest.mark.parametrize("T", [48, 500])
def test_ffn_one_hot_expert_and_empty_experts(moe, T):
    """All rows on one expert; the other hosted experts get none."""
    cfg, wl, _ = _case(T, 256, 8, 2, 256, 8)
    idx = np.tile(np.array([[5, 2]], np.int32), (T, 1))
    assert _run_ffn(moe, cfg, wl, idx) == 2 * T
    cfg, wl, _ = _case(T, 256, 8, 2, 256, 3, local=[6, 7, 0])
    assert _run_ffn(moe, cfg, wl, idx) == 0


def test_ffn_group_larger_than_batch(moe):
    """Duplicate expert ids give one expert more rows than there are tokens:
    the weight-streaming kernel then walks the rows in several passes."""
    T = 50
    cfg, wl, _ = _case(T, 128, 4, 2, 128, 4)
    idx = np.tile(np.array([[1, 1]], np.int32), (T, 1))
    assert _run_ffn(moe, cfg, wl, idx) == 2 * T


def test_ffn_tile_boundaries(moe):
    """Groups of 1, 127..129, 255..257 and 511..513 rows: one row, half and
    whole 256-row m-tiles, and one row past them, side by side in one launch."""
    sizes = [1, 127, 128, 129, 255, 256, 257, 511, 512, 513, 65]
    T = sum(sizes)
    cfg, wl, _ = _case(T, 136, len(sizes), 1, 200, len(sizes))
    idx = np.repeat(np.arange(len(sizes), dtype=np.int32), sizes)[np.random.default_rng(3).permutation(T)]
    assert _run_ffn(moe, cfg, wl, idx.reshape(T, 1)) == T


@pytest.mark.parametrize("I_sh", [1024, 960])
def test_ffn_shared_experts_with_or_without_the_routed_launch(moe, I_sh):
    """4096 tokens and two shared experts: 2 x 1024 shared columns make 16 x 16 = 256
    gate/up tiles, whole rounds on 256 CUs, so the shared GEMMs keep their own launches;
    2 x 960 make 240 tiles, which run inside the routed experts' launch."""
    cfg, wl, idx = _case(4096, 128, 16, 2, 128, 16, 2, I_sh)
    _run_ffn(moe, cfg, wl, idx)


@pytest.mark.parametrize("T,H,I_sh,which", [
    (1000, 128, 8192, "up"),       # 4 m-tiles x 64 column tiles: all tiles past the last whole block
    (2900, 128, 8192, "up"),       # 12 m-tiles: one whole block of 8, then the remainder of 4
    (1000, 16376, 64, "down"),     # the down projection's 64 column tiles (H = 16376)
    (2900, 16376, 64, "down"),
])
def test_ffn_shared_blocked_order_remainder(moe, T, H, I_sh, which):
    """A launch of the shared experts alone (their tiles fill whole rounds of
    the 256 compute units) orders its tiles in blocks of 8 m-tiles; these
    shapes have m-tile counts that are not multiples of 8, so the tiles past
    the last whole block take the remainder order.  Every row is checked."""
    if torch.cuda.get_device_properties(0).multi_processor_count != 256:
        pytest.skip("the shapes fill whole rounds of 256 compute units")
    cfg, wl, idx = _case(T, H, 8, 2, 64, 8, 1, I_sh)
    _run_ffn(moe, cfg, wl, idx)


def _combine(moe, T, k, H, R, with_shared, seed):
    rng = np.random.default_rng(seed)
    y = W.f32_to_bf16_bits(rng.standard_normal((max(R, 1), H)).astype(np.float32))
    inv = np.full(T * k, -1, np.int32)
    inv[rng.permutation(T * k)[:R]] = np.arange(R, dtype=np.int32)
    w = rng.random((T, k)).astype(np.float32)
    ysh = W.f32_to_bf16_bits(rng.standard_normal((T, H)).astype(np.float32)) if with_shared else None
    d = moe.dims(T=T, H=H, E=max(k, 8), k=k, I=8, S=1, E_local=max(k, 8))
    out = torch.full((T, H), 7.0, dtype=torch.bfloat16, device="cuda")
    moe.combine(d, dev(y), dev(inv), dev(w), None if ysh is None else dev(ysh), out)
    torch.cuda.synchronize()
    got = bf16_f64(host_bf16(out))
    ref = oracle.combine(y[:R] if R else y[:0], inv, w, ysh, H=H)
    # bf16 rounding of the result plus fp32 accumulation of the terms
    mag = np.zeros((T, H))
    for p in range(T * k):
        if inv[p] >= 0:
            mag[p // k] += abs(float(w.reshape(-1)[p])) * np.abs(bf16_f64(y[inv[p]]))
    if ysh is not None:
        mag += np.abs(bf16_f64(ysh))
    # bf16 unit roundoff is 2^-8; fp32 accumulation of at most 33 terms stays below 2^-16 of their magnitude
    assert (np.abs(got - ref) <= 1.01 * 2.0 ** -8 * np.abs(ref) + 2.0 ** -16 * mag + 1e-30).all()


@pytest.mark.parametrize("T,k,H,R,sh", [(1, 1, 8, 1, False), (7, 2, 136, 9, True), (64, 2, 4096, 128, False),
                                        (300, 8, 2048, 1700, True), (500, 6, 256, 0, True),
                                        (500, 6, 256, 0, False), (33, 32, 64, 1000, False)])
def test_combine(moe, T, k, H, R, sh):
    _combine(moe, T, k, H, R, sh, seed=T + k + H)
