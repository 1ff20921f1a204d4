"""The C-ABI library without a GPU: it loads, exports every function that
include/moe.h declares, and its host-side checks return the documented codes
before touching the device."""
import ctypes as C
import subprocess

import pytest

from paper_2606_15177_amd import workloads as W


@pytest.fixture(scope="module")
def moe():
    from paper_2606_15177_amd import moe
    return moe


def test_exports_every_declared_function(moe):
    names = moe.header_functions()
    assert {"moe_route", "moe_route_stats", "moe_permute", "moe_expert_ffn", "moe_combine",
            "moe_forward", "moe_workspace_bytes", "moe_validate", "moe_strerror"} <= set(names)
    out = subprocess.run(["nm", "-D", "--defined-only", moe.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    for n in names:
        assert n in exported, n
    lib = C.CDLL(moe.LIB_PATH)
    for n in names:
        getattr(lib, n)


def test_abi_version_and_strerror(moe):
    assert moe._lib.moe_abi_version() == 2
    for code in (0, -1, -2, -3, -4, -5, -6):
        assert moe.strerror(code) and moe.strerror(code) != "unknown status"
    assert moe.strerror(-99) == "unknown status"


@pytest.mark.parametrize("name", W.CONFIG_ORDER)
def test_configs_validate(moe, name):
    d = moe.dims_of(W.CONFIGS[name])
    assert moe.validate(d) == moe.MOE_OK
    for entry in (moe.ENTRY_PERMUTE, moe.ENTRY_EXPERT_FFN, moe.ENTRY_FORWARD):
        need = moe.workspace_bytes(d, entry)
        assert need > 0 and need % 256 == 0
        assert moe.validate(d, entry, need) == moe.MOE_OK
        assert moe.validate(d, entry, need - 1) == moe.MOE_ERR_WORKSPACE


def test_forward_workspace_size(moe):
    cfg = W.CONFIGS["ep_share_dsv3"]
    d = moe.dims_of(cfg)
    rows = cfg.T * cfg.k
    # y_perm + h dominate (capacity T*k rows); there is no gathered copy of x,
    # the gate/up GEMM reads x through perm_token
    lower = rows * cfg.H * 2 + rows * cfg.I * 2
    assert lower <= moe.workspace_bytes(d, moe.ENTRY_FORWARD) < lower * 1.2


@pytest.mark.parametrize("change,code", [
    (dict(T=-1), -2), (dict(H=0), -2), (dict(k=0), -2), (dict(k=9), -2), (dict(S=0), -2),
    (dict(E_local=0), -2), (dict(E_local=9), -2), (dict(n_shared=-1), -2),
    (dict(n_shared=1, I_shared=0), -2), (dict(I=0), -2),
    (dict(H=12), -3), (dict(I=100), -3), (dict(n_shared=1, I_shared=36), -3),
    (dict(E=1025, E_local=8), -3), (dict(E=64, k=33), -3), (dict(flags=3), -3), (dict(flags=-1), -3),
    (dict(T=2 ** 30, k=2), -3),
])
def test_validate_rejects(moe, change, code):
    base = dict(T=16, H=64, E=8, k=2, I=64, S=2, E_local=8, n_shared=0, I_shared=0)
    base.update(change)
    flags = base.pop("flags", 0)
    d = moe.dims(**base, flags=flags)
    assert moe.validate(d) == code
    assert moe.workspace_bytes(d, moe.ENTRY_FORWARD) == 0


def test_entry_points_reject_before_launch(moe):
    """Errors are decided on the host; nothing reaches the device."""
    lib = moe._lib
    d = moe.dims(T=4, H=64, E=8, k=2, I=64, S=2, E_local=4)
    assert lib.moe_route(None, None, None, None, None, None) == moe.MOE_ERR_NULL
    assert lib.moe_route(C.byref(d), None, None, None, None, None) == moe.MOE_ERR_NULL
    assert lib.moe_route_stats(C.byref(d), None, None, None, None, None) == moe.MOE_ERR_NULL
    # no placement list while E_local < E
    assert lib.moe_permute(C.byref(d), 16, None, None, 16, 16, 16, None, None, 0, None) == moe.MOE_ERR_DIMS
    d8 = moe.dims(T=4, H=64, E=8, k=2, I=64, S=2, E_local=8)
    # x given without x_perm
    assert lib.moe_permute(C.byref(d8), 16, None, 16, 16, 16, 16, None, None, 0, None) == moe.MOE_ERR_NULL
    # misaligned x
    assert lib.moe_permute(C.byref(d8), 16, None, 24, 16, 16, 16, 32, None, 0, None) == moe.MOE_ERR_ALIGN
    # workspace too small
    assert lib.moe_permute(C.byref(d8), 16, None, 16, 16, 16, 16, 32, 256, 0, None) == moe.MOE_ERR_WORKSPACE
    w = moe.MoeWeights(None, None, None, None, None, None)
    assert lib.moe_expert_ffn(C.byref(d8), 16, 16, C.byref(w), None, 16, None, None, 0, None) == moe.MOE_ERR_NULL
    w = moe.MoeWeights(16, 16, 24, None, None, None)
    assert lib.moe_expert_ffn(C.byref(d8), 16, 16, C.byref(w), None, 16, None, None, 0, None) == moe.MOE_ERR_ALIGN
    w = moe.MoeWeights(16, 16, 16, None, None, None)
    dsh = moe.dims(T=4, H=64, E=8, k=2, I=64, S=2, E_local=8, n_shared=1, I_shared=64)
    assert lib.moe_expert_ffn(C.byref(dsh), 16, 16, C.byref(w), None, 16, None, None, 0, None) == moe.MOE_ERR_NULL
    assert lib.moe_combine(C.byref(d8), None, 16, 16, None, 16, None) == moe.MOE_ERR_NULL
    assert lib.moe_forward(C.byref(d8), None, 16, None, 16, None, C.byref(w), 16, 16, None, None, 0,
                           None) == moe.MOE_ERR_NULL       # counts without src
    ws_need = moe.workspace_bytes(d8, moe.ENTRY_FORWARD)
    assert lib.moe_forward(C.byref(d8), None, 16, 16, 16, None, C.byref(w), 16, 16, None, 256, ws_need - 1,
                           None) == moe.MOE_ERR_WORKSPACE
    assert lib.moe_forward(C.byref(d8), None, 16, 16, 16, None, C.byref(w), 16, 16, None, 128, ws_need,
                           None) == moe.MOE_ERR_ALIGN      # workspace not 256-byte aligned


# ------------------------------------------------------------ placement ----

def _cap(vals):
    import numpy as np
    a = np.ascontiguousarray(vals, dtype=np.int32)
    return a, a.ctypes.data_as(C.c_void_p)


def test_place_slots(moe):
    lib = moe._lib
    pd = moe.place_dims(L=2, S=2, E=10, G=3)
    assert moe.place_slots(pd, [4, 4, 4]) == 4
    assert moe.place_slots(pd, [0, 25, 3]) == 10      # a rank never holds more than E
    assert moe.place_slots(pd, [-3, 5, 5]) == 5
    assert lib.moe_place_slots(None, None) == 0


@pytest.mark.parametrize("change,cap,code", [
    (dict(), [4, 4], -1),                    # A missing (see below: all pointers NULL)
    (dict(L=-1), [4, 4], -2), (dict(S=0), [4, 4], -2), (dict(E=0), [4, 4], -2),
    (dict(G=0), [], -2),
    (dict(), [4, 3], -2),                    # 7 places for 8 experts
    (dict(), [-1, 9], -2),                   # negative capacity
    (dict(E=1025), [1025, 1025], -3), (dict(G=65), [1] * 65, -3),
    (dict(S=2049), [8, 8], -3),              # S*G > 4096
])
def test_place_rejects_before_launch(moe, change, cap, code):
    base = dict(L=2, S=2, E=8, G=2)
    base.update(change)
    pd = moe.place_dims(**base)
    cap_a, cap_p = _cap(cap)
    rc = moe._lib.moe_place_experts(C.byref(pd), cap_p, None, None, None, None, None, None, None, None, None)
    assert rc == code


def test_place_checks_alignment_and_noop(moe):
    lib = moe._lib
    pd = moe.place_dims(L=2, S=2, E=8, G=2)
    cap_a, cap_p = _cap([4, 4])
    assert lib.moe_place_experts(None, cap_p, 16, None, 16, None, 16, 16, None, None, None) == moe.MOE_ERR_NULL
    assert lib.moe_place_experts(C.byref(pd), None, 16, None, 16, None, 16, 16, None, None, None) == moe.MOE_ERR_NULL
    assert lib.moe_place_experts(C.byref(pd), cap_p, 12, None, 16, None, 16, 16, None, None, None) == moe.MOE_ERR_ALIGN
    assert lib.moe_place_experts(C.byref(pd), cap_p, 16, None, 16, 20, 16, 16, None, None, None) == moe.MOE_ERR_ALIGN
    assert lib.moe_place_experts(C.byref(pd), cap_p, 16, None, 16, None, 18, 16, None, None, None) == moe.MOE_ERR_ALIGN
    # L = 0: nothing to place, nothing launched, no pointer needed
    pd0 = moe.place_dims(L=0, S=2, E=8, G=2)
    assert lib.moe_place_experts(C.byref(pd0), cap_p, None, None, None, None, None, None, None, None,
                                 None) == moe.MOE_OK


@pytest.mark.parametrize("change,engine,code", [
    (dict(L=-1), False, -2), (dict(S=0), False, -2), (dict(E=0), False, -2), (dict(G=0, n_engines=0), False, -2),
    (dict(n_engines=0), True, -2),
    (dict(n_engines=3), False, -2),          # no engine map: engines must be the ranks
    (dict(E=8193), False, -3), (dict(G=1025, n_engines=1025), False, -3), (dict(n_engines=1025), True, -3),
    (dict(), False, -1),                     # outputs missing
])
def test_window_rejects_before_launch(moe, change, engine, code):
    base = dict(L=2, S=2, E=8, G=4, n_engines=4)
    base.update(change)
    wd = moe.MoeWindowDims(**base)
    rc = moe._lib.moe_window_stats(C.byref(wd), None, None, None, None, 16 if engine else None, None, None, None,
                                   None, None)
    assert rc == code


def test_window_alignment_and_empty(moe):
    lib = moe._lib
    wd = moe.MoeWindowDims(L=2, S=2, E=8, G=4, n_engines=4)
    assert lib.moe_window_stats(None, 16, None, 16, 16, None, 16, 16, 16, None, None) == moe.MOE_ERR_NULL
    assert lib.moe_window_stats(C.byref(wd), 20, None, 16, 16, None, 16, 16, 16, None, None) == moe.MOE_ERR_ALIGN
    assert lib.moe_window_stats(C.byref(wd), 16, None, 18, 16, None, 16, 16, 16, None, None) == moe.MOE_ERR_ALIGN
    assert lib.moe_window_stats(C.byref(wd), 16, None, 16, 16, None, 16, 16, 16, 12, None) == moe.MOE_ERR_ALIGN
    wd0 = moe.MoeWindowDims(L=0, S=2, E=8, G=4, n_engines=4)
    assert lib.moe_window_stats(C.byref(wd0), None, None, None, None, None, None, None, None, None,
                                None) == moe.MOE_OK


@pytest.mark.parametrize("flags,g,code", [
    (0, dict(bias=16), -2),                           # a bias needs sigmoid gates
    (2, dict(bias=18), -6),                           # misaligned bias
    (2, dict(n_group=3, topk_group=1), -2),           # 8 experts do not split into 3 groups
    (2, dict(n_group=4, topk_group=0), -2),
    (2, dict(n_group=4, topk_group=5), -2),
    (2, dict(n_group=4, topk_group=1), -2),           # k=4 > 1 group of 2 experts
    (2, dict(n_group=-1), -2),
    (2, dict(n_group=128, topk_group=1), -3),
    (1, dict(n_group=4, topk_group=2), -1),           # valid: fails later on the NULL logits
    (2, dict(bias=16, n_group=2, topk_group=2, routed_scale=2.5), -1),
])
def test_gating_rejects_before_launch(moe, flags, g, code):
    d = moe.dims(T=4, H=64, E=8, k=4, I=64, S=2, E_local=8, flags=flags)
    n_group = g.get("n_group", 0)
    if n_group == 128:
        d = moe.dims(T=4, H=64, E=256, k=4, I=64, S=2, E_local=256, flags=flags)
    gat = moe.MoeGating(g.get("bias"), g.get("routed_scale", 1.0), n_group, g.get("topk_group", 0))
    assert moe._lib.moe_route(C.byref(d), C.byref(gat), None, None, None, None) == code


# ------------------------------------------------------- kernel limits ----

def test_kernel_limits_decided_on_the_host(moe):
    """The tiled gate/up GEMM of moe_forward reads token rows through the
    dispatch list with 32-bit byte offsets from the start of x, so T*H*2 must
    stay below 2^31 (T >= 149,797 at H = 7168 does not).  moe_validate and
    moe_forward say so before anything is enqueued; moe_expert_ffn, which
    reads a gathered copy tile by tile, takes the same sizes."""
    import numpy as np
    lib = moe._lib
    big = moe.dims(T=150000, H=7168, E=256, k=8, I=2048, S=8, E_local=32, n_shared=1, I_shared=2048)
    assert moe.validate(big, moe.ENTRY_FORWARD) == moe.MOE_ERR_UNSUPPORTED
    assert moe.validate(big) == moe.MOE_ERR_UNSUPPORTED                  # entry 0: every entry point
    assert moe.workspace_bytes(big, moe.ENTRY_FORWARD) == 0
    assert moe.validate(big, moe.ENTRY_EXPERT_FFN, 1 << 62) == moe.MOE_OK
    assert moe.validate(big, moe.ENTRY_PERMUTE, 1 << 62) == moe.MOE_OK
    ok = moe.dims(T=149000, H=7168, E=256, k=8, I=2048, S=8, E_local=32, n_shared=1, I_shared=2048)
    assert moe.validate(ok, moe.ENTRY_FORWARD, 1 << 62) == moe.MOE_OK
    # moe_forward returns the same code with nothing launched: host buffers
    # stand in for every device pointer (nothing may touch them) and the
    # counts matrix stays as it was
    counts = np.arange(8 * 256, dtype=np.int64)
    before = counts.copy()
    buf = np.zeros(1 << 12, dtype=np.uint8)
    p = buf.ctypes.data + (-buf.ctypes.data) % 256
    w = moe.MoeWeights(p, p, p, p, p, p)
    rc = lib.moe_forward(C.byref(big), None, p, p, p, p, C.byref(w), counts.ctypes.data, p, None, p,
                         1 << 62, None)
    assert rc == moe.MOE_ERR_UNSUPPORTED
    assert np.array_equal(counts, before)


@pytest.mark.parametrize("change", [
    dict(T=1024, H=8, E=8, k=2, I=2 ** 22, E_local=8),               # a tiled tile's output rows: 257*I*2 >= 2^31
    dict(T=16, H=2 ** 16, E=8, k=2, I=2 ** 15, E_local=8),           # streamed weights of one expert: I*H*2 >= 2^31
])
def test_kernel_limits_of_each_gemm(moe, change):
    d = moe.dims(S=2, **change)
    assert moe.validate(d, moe.ENTRY_EXPERT_FFN, 1 << 62) == moe.MOE_ERR_UNSUPPORTED
    assert moe.validate(d, moe.ENTRY_FORWARD, 1 << 62) == moe.MOE_ERR_UNSUPPORTED
    assert moe.validate(d, moe.ENTRY_PERMUTE, 1 << 62) == moe.MOE_OK


def test_forward_noalloc_rejects_on_the_host(moe):
    """moe_forward_noalloc's workspace is the library's 32 MiB scratch array:
    larger layers are refused before anything is enqueued."""
    lib = moe._lib
    w = moe.MoeWeights(256, 256, 256, 256, 256, 256)
    assert lib.moe_forward_noalloc(None, None, 256, 256, 256, 256, C.byref(w), None, 256, None,
                                   None) == moe.MOE_ERR_NULL
    big = moe.dims_of(W.CONFIGS["ep_share_dsv3"])
    assert moe.workspace_bytes(big, moe.ENTRY_FORWARD) > 32 << 20
    assert lib.moe_forward_noalloc(C.byref(big), None, 256, 256, 256, 256, C.byref(w), None, 256, None,
                                   None) == moe.MOE_ERR_WORKSPACE
    decode = moe.dims_of(W.CONFIGS["decode_mixtral"])
    assert moe.workspace_bytes(decode, moe.ENTRY_FORWARD) <= 32 << 20
