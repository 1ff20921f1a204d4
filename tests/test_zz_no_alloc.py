"""moe_forward_noalloc, the layer with the library's own scratch array as
its workspace, against moe_forward with a caller workspace: two calls in a
row on one device, the second with a smaller batch, each bit-identical to
moe_forward on the same inputs (the same kernels run on the same data) and
within the layer tolerance of the CPU oracle."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2606_15177_amd import workloads as W
from tests.gpu_util import assert_layer_close, dev, dev_weights, host_bf16

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def moe():
    from paper_2606_15177_amd import moe
    return moe


def _taps(moe, cfg):
    T, k = cfg.T, cfg.k
    t = dict(topk_idx=torch.full((T, k), -9, dtype=torch.int32, device="cuda"),
             topk_w=torch.zeros((T, k), dtype=torch.float32, device="cuda"),
             offsets=torch.full((cfg.E_local + 1,), -9, dtype=torch.int32, device="cuda"),
             perm_token=torch.full((T * k,), -9, dtype=torch.int32, device="cuda"),
             inv_pos=torch.full((T * k,), -9, dtype=torch.int32, device="cuda"))
    return t, moe.make_taps(**t)


def _both(moe, cfg, wl, w, loc):
    """(moe_forward results, moe_forward_noalloc results) on the same inputs."""
    d = moe.dims_of(cfg)
    assert moe.workspace_bytes(d, moe.ENTRY_FORWARD) <= 32 << 20
    logits, src, x = dev(wl["logits"]), dev(wl["src"]), dev(wl["x"])
    res = []
    for noalloc in (False, True):
        counts = torch.zeros((cfg.S, cfg.E), dtype=torch.int64, device="cuda")
        out = torch.full((cfg.T, cfg.H), 7.0, dtype=torch.bfloat16, device="cuda")
        t, taps = _taps(moe, cfg)
        if noalloc:
            moe.forward_noalloc(d, logits, src, x, loc, w, counts, out, taps)
        else:
            ws = moe.workspace(d, moe.ENTRY_FORWARD)
            moe.forward(d, logits, src, x, loc, w, counts, out, ws, taps)
        torch.cuda.synchronize()
        r = {n: v.cpu().numpy() for n, v in t.items()}
        r["counts"] = counts.cpu().numpy()
        r["out"] = host_bf16(out)
        res.append(r)
    return res


def test_noalloc_two_calls_match_forward(moe):
    # a prefill-sized call (tiled GEMMs, shared expert), then a decode-sized
    # one (weight-streaming GEMMs, chunk-blocked intermediate) on the same
    # layer: the second finds the first one's data in the scratch array
    base = W.MoeConfig("noalloc", T=300, H=256, E=16, k=4, I=512, S=3, E_local=8, n_shared=1, I_shared=256,
                       local_layout="choice")
    wl_big = W.make_workload(base, seed=11)
    wdev = dev_weights(wl_big)          # keeps the device weights alive while w points at them
    w = moe.make_weights(wdev)
    loc = dev(wl_big["local_experts"])
    for T, seed in ((300, 11), (48, 12)):
        cfg = base.replace(T=T)
        wl = W.make_workload(cfg, seed=seed, weights=False)
        wl.update({k: wl_big[k] for k in ("w_gate", "w_up", "w_down", "sh_gate", "sh_up", "sh_down",
                                          "local_experts")})
        ref, got = _both(moe, cfg, wl, w, loc)
        for name in ref:
            np.testing.assert_array_equal(got[name], ref[name], err_msg=f"T={T}: {name}")
        expect = oracle.forward_tokens(cfg.dims, np.arange(T), wl["logits"], wl["x"], wl["local_experts"], wl)
        assert_layer_close(got["out"], expect, f"noalloc T={T}")


def test_noalloc_rejects_sizes_beyond_the_scratch(moe):
    """The DeepSeek-V3 share needs 2.7 GB of workspace: refused on the host,
    nothing enqueued."""
    import ctypes as C
    d = moe.dims_of(W.CONFIGS["ep_share_dsv3"])
    w = moe.MoeWeights(256, 256, 256, 256, 256, 256)
    rc = moe._lib.moe_forward_noalloc(C.byref(d), None, 256, 256, 256, 256, C.byref(w), None, 256, None, None)
    assert rc == moe.MOE_ERR_WORKSPACE
