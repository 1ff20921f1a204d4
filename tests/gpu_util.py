"""Helpers of the GPU parity tests: device transfer, tolerance checks and
cached workloads.  Inputs come from the seeded generator only; expected
values come from the CPU oracle only."""
from __future__ import annotations

import concurrent.futures as cf
import functools
import os

import numpy as np
import torch

from paper_2606_15177_amd import workloads as W

# Layer-output tolerance: bf16 inputs, fp32 accumulation, bf16 intermediates,
# against the fp64 oracle.  rel is normwise (max error over max |ref|); the
# 1e-3 absolute MAE bound is vacuous at these output scales, so the mean
# error is also bounded relative to the mean |ref|.
REL_TOL = 2e-2
MAE_TOL = 1e-3
REL_MAE_TOL = 1e-2
GATE_ATOL = 1e-6


def dev(a: np.ndarray) -> torch.Tensor:
    """numpy -> contiguous CUDA tensor; uint16 arrays become bfloat16 bits."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(a).cuda()


def host_bf16(t: torch.Tensor) -> np.ndarray:
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


def bf16_f64(a: np.ndarray) -> np.ndarray:
    return W.bf16_bits_to_f32(a).astype(np.float64)


def layer_errors(got_bf16: np.ndarray, ref: np.ndarray) -> dict:
    g = bf16_f64(got_bf16)
    diff = np.abs(g - ref)
    scale = float(np.abs(ref).max()) if ref.size else 0.0
    mean_ref = float(np.abs(ref).mean()) if ref.size else 0.0
    return dict(rel=float(diff.max()) / scale if scale > 0 else float(diff.max()),
                mae=float(diff.mean()) if ref.size else 0.0,
                rel_mae=float(diff.mean()) / mean_ref if mean_ref > 0 else float(diff.mean()),
                scale=scale)


def assert_layer_close(got_bf16: np.ndarray, ref: np.ndarray, what: str = "") -> dict:
    e = layer_errors(got_bf16, ref)
    if e["scale"] == 0.0:
        assert (bf16_f64(got_bf16) == 0).all(), f"{what}: expected exact zeros"
        return e
    assert e["rel"] <= REL_TOL, f"{what}: normwise rel err {e['rel']:.3e} > {REL_TOL}"
    assert e["mae"] <= MAE_TOL, f"{what}: MAE {e['mae']:.3e} > {MAE_TOL}"
    assert e["rel_mae"] <= REL_MAE_TOL, f"{what}: relative MAE {e['rel_mae']:.3e} > {REL_MAE_TOL}"
    return e


def assert_gates_close(got: np.ndarray, ref: np.ndarray, what: str = "") -> None:
    finite = np.isfinite(ref)
    assert np.array_equal(np.isnan(got), np.isnan(ref)), f"{what}: NaN pattern differs"
    if finite.any():
        err = np.abs(got[finite].astype(np.float64) - ref[finite]).max()
        assert err <= GATE_ATOL, f"{what}: gate error {err:.3e}"


@functools.lru_cache(maxsize=2)
def workload(name: str, seed: int = 0) -> dict:
    return W.make_workload(W.CONFIGS[name], seed)


def dev_weights(wl: dict) -> dict:
    return {k: dev(wl[k]) for k in ("w_gate", "w_up", "w_down", "sh_gate", "sh_up", "sh_down") if k in wl}


def sample_tokens(T: int, n: int, seed: int = 0, extra=()) -> np.ndarray:
    rng = np.random.default_rng(seed)
    pick = set(rng.choice(T, size=min(n, T), replace=False).tolist()) | {0, T - 1} | set(extra)
    return np.array(sorted(pick), dtype=np.int32)


def oracle_route_cfg(cfg, wl):
    """The oracle's routing of a workload under its router's gate function."""
    from oracle import oracle
    if not cfg.gated:
        return oracle.route(wl["logits"], cfg.k)
    return oracle.route_gated(wl["logits"], cfg.k, cfg.gate, wl.get("gate_bias"), cfg.routed_scale,
                              cfg.n_group, cfg.topk_group)


def oracle_forward_cfg(cfg, wl, tokens):
    from oracle import oracle
    return oracle.forward_tokens(cfg.dims, tokens, wl["logits"], wl["x"], wl["local_experts"], wl,
                                 gate=cfg.gate, bias=wl.get("gate_bias"), scale=cfg.routed_scale,
                                 n_group=cfg.n_group, topk_group=cfg.topk_group)


def gating_cfg(moe, cfg, wl, keep=None):
    """(MoeGating or None, the device bias tensor it points to) for a workload."""
    if not cfg.gated:
        return None, None
    b = wl.get("gate_bias")
    bias = None if b is None else dev(b)
    return moe.gating(bias, cfg.routed_scale, cfg.n_group, cfg.topk_group), bias


def host_threads() -> int:
    """Worker threads for the oracle: the CPUs this process may use, at most 16."""
    return max(1, min(16, len(os.sched_getaffinity(0))))


def parallel_rows(fn, items):
    """fn(items[a:b]) over disjoint slices in host threads, results stacked in
    order.  The C oracle is reentrant and ctypes releases the interpreter lock
    during the call, so the slices run in parallel."""
    items = np.asarray(items)
    if len(items) == 0:
        return fn(items)
    parts = np.array_split(items, min(host_threads(), len(items)))
    with cf.ThreadPoolExecutor(len(parts)) as ex:
        res = list(ex.map(fn, parts))
    return np.concatenate(res, axis=0)
