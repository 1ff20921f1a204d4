"""Python access to the plain-C CPU oracle of the MoE-layer hot path.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's CPU
baseline may use this module; the product path never imports it.  It only
marshals numpy arrays into ``moe_oracle.c`` (the layer) and ``place_oracle.c``
(source-aware expert placement), where all the arithmetic lives (fp64,
single-threaded, written from the definitions).  Shares nothing with the HIP
library.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRCS = [os.path.join(_HERE, "moe_oracle.c"), os.path.join(_HERE, "place_oracle.c")]
# MOE_ORACLE_LIB lets the mutation test load a deliberately broken build.
LIB = os.environ.get("MOE_ORACLE_LIB") or os.path.join(_HERE, "libmoe_oracle.so")

_i32p = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(dtype=np.int64, flags="C_CONTIGUOUS")
_u16p = np.ctypeslib.ndpointer(dtype=np.uint16, flags="C_CONTIGUOUS")
_f32p = np.ctypeslib.ndpointer(dtype=np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(dtype=np.float64, flags="C_CONTIGUOUS")
_vp = C.c_void_p


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain -O2: no fast-math, no host-specific
    ISA, no contraction into fused multiply-adds, so every fp64 operation
    rounds as written)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fPIC", "-shared",
                               "-Wall", "-Wextra", *SRCS, "-o", tmp, "-lm"])
        os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build(force=False)
        L = C.CDLL(LIB)
        L.oracle_route.argtypes = [C.c_int, C.c_int, C.c_int, _f32p, _i32p, _f64p]
        L.oracle_route_gated.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, _f32p, _vp, C.c_double, C.c_int,
                                         C.c_int, _i32p, _f64p]
        L.oracle_route_stats.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, _i32p, _i32p, _i64p, _vp]
        L.oracle_permute.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, _vp, _i32p, _i32p, _i32p, _i32p]
        L.oracle_gather_rows.argtypes = [C.c_int, C.c_int, _i32p, _u16p, _u16p]
        L.oracle_swiglu_hidden.argtypes = [C.c_int, C.c_int, _u16p, _u16p, _u16p, _f64p]
        L.oracle_linear.argtypes = [C.c_int, C.c_int, _u16p, _f64p, _f64p]
        L.oracle_swiglu_ffn.argtypes = [C.c_int, C.c_int, _u16p, _u16p, _u16p, _u16p, _f64p]
        L.oracle_ffn_rows.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, _i32p, _u16p, _u16p, _u16p, _u16p, _f64p]
        L.oracle_combine.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, _u16p, _i32p, _f32p, _vp, _f64p]
        L.oracle_forward_tokens.argtypes = [_i32p, C.c_int, _i32p, _f32p, _u16p, _vp, _u16p, _u16p, _u16p,
                                            _vp, _vp, _vp, _vp, C.c_double, C.c_int, C.c_int, _f64p]
        L.oracle_place_objective.argtypes = [C.c_int] * 4 + [_i64p, _vp, _f64p, _vp, C.c_double, _i32p,
                                                             _i32p, _f64p]
        L.oracle_place_greedy.argtypes = [C.c_int] * 4 + [_i64p, _vp, _f64p, _vp, C.c_double, _i32p, _i32p,
                                                          C.c_double, C.c_double, C.c_double, _i32p, _vp]
        L.oracle_window_stats.argtypes = [C.c_int] * 4 + [_i64p, _vp, _i32p, _i32p, _vp, C.c_int, _i64p, _i64p,
                                                          _i64p, _vp]
        for name in ("oracle_route_gated", "oracle_window_stats", "oracle_place_objective", "oracle_place_greedy", "oracle_route", "oracle_route_stats", "oracle_permute", "oracle_gather_rows",
                     "oracle_swiglu_hidden", "oracle_linear", "oracle_swiglu_ffn", "oracle_ffn_rows",
                     "oracle_combine", "oracle_forward_tokens"):
            getattr(L, name).restype = C.c_int
        _lib = L
    return _lib


class OracleError(RuntimeError):
    pass


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise OracleError(f"{what} returned {rc}")


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def route(logits: np.ndarray, k: int):
    """Top-k expert ids [T, k] int32 and softmax-over-top-k gates [T, k] fp64."""
    logits = _c(logits, np.float32)
    T, E = logits.shape
    idx = np.empty((T, k), np.int32)
    w = np.empty((T, k), np.float64)
    _check(lib().oracle_route(T, E, k, logits, idx, w), "oracle_route")
    return idx, w


GATE_SOFTMAX_TOPK, GATE_SOFTMAX, GATE_SIGMOID = 0, 1, 2


def route_gated(logits: np.ndarray, k: int, gate: int = GATE_SOFTMAX_TOPK, bias=None, scale: float = 1.0,
                n_group: int = 0, topk_group: int = 0):
    """Top-k ids [T, k] int32 and gates [T, k] fp64 under a gating variant."""
    logits = _c(logits, np.float32)
    T, E = logits.shape
    b = None if bias is None else _c(bias, np.float32)
    idx = np.empty((max(T, 1), k), np.int32)
    w = np.empty((max(T, 1), k), np.float64)
    _check(lib().oracle_route_gated(T, E, k, gate, logits, _ptr(b), float(scale), n_group, topk_group, idx, w),
           "oracle_route_gated")
    return idx[:T], w[:T]


def route_stats(src: np.ndarray, topk_idx: np.ndarray, S: int, E: int, counts=None):
    """Accumulate the S x E source/expert counts; return (counts, expert_load)."""
    src = _c(src, np.int32)
    topk_idx = _c(topk_idx, np.int32)
    T, k = topk_idx.shape
    counts = np.zeros((S, E), np.int64) if counts is None else counts
    assert counts.dtype == np.int64 and counts.flags.c_contiguous
    load = np.empty(E, np.int32)
    _check(lib().oracle_route_stats(T, k, S, E, src, topk_idx, counts, _ptr(load)), "oracle_route_stats")
    return counts, load


def permute(topk_idx: np.ndarray, E: int, E_local: int, local_experts=None):
    """(offsets [E_local+1], perm_token [R], inv_pos [T*k]) of the stable dispatch sort."""
    topk_idx = _c(topk_idx, np.int32)
    T, k = topk_idx.shape
    loc = None if local_experts is None else _c(local_experts, np.int32)
    offsets = np.empty(E_local + 1, np.int32)
    perm = np.empty(max(T * k, 1), np.int32)
    inv = np.empty(T * k, np.int32)
    _check(lib().oracle_permute(T, k, E, E_local, _ptr(loc), topk_idx, offsets, perm, inv), "oracle_permute")
    return offsets, perm[: offsets[-1]].copy(), inv


def gather_rows(x: np.ndarray, perm_token: np.ndarray) -> np.ndarray:
    x = _c(x, np.uint16)
    perm_token = _c(perm_token, np.int32)
    R, H = len(perm_token), x.shape[1]
    out = np.empty((max(R, 1), H), np.uint16)
    _check(lib().oracle_gather_rows(R, H, perm_token, x, out), "oracle_gather_rows")
    return out[:R]


def swiglu_hidden(x_row, w_gate, w_up) -> np.ndarray:
    w_gate = _c(w_gate, np.uint16)
    I, H = w_gate.shape
    h = np.empty(I, np.float64)
    _check(lib().oracle_swiglu_hidden(H, I, _c(x_row, np.uint16), w_gate, _c(w_up, np.uint16), h),
           "oracle_swiglu_hidden")
    return h


def linear(w, v) -> np.ndarray:
    w = _c(w, np.uint16)
    n_out, n_in = w.shape
    y = np.empty(n_out, np.float64)
    _check(lib().oracle_linear(n_out, n_in, w, _c(v, np.float64), y), "oracle_linear")
    return y


def swiglu_ffn(x_row, w_gate, w_up, w_down) -> np.ndarray:
    w_gate = _c(w_gate, np.uint16)
    I, H = w_gate.shape
    y = np.empty(H, np.float64)
    _check(lib().oracle_swiglu_ffn(H, I, _c(x_row, np.uint16), w_gate, _c(w_up, np.uint16),
                                   _c(w_down, np.uint16), y), "oracle_swiglu_ffn")
    return y


def ffn_rows(x_rows, slots, w_gate, w_up, w_down) -> np.ndarray:
    """y[r] = FFN_{slots[r]}(x_rows[r]) with weights stacked by local slot."""
    x_rows = _c(x_rows, np.uint16)
    slots = _c(slots, np.int32)
    w_gate = _c(w_gate, np.uint16)
    E_local, I, H = w_gate.shape
    n = len(slots)
    y = np.empty((max(n, 1), H), np.float64)
    _check(lib().oracle_ffn_rows(n, H, I, E_local, slots, x_rows, w_gate, _c(w_up, np.uint16),
                                 _c(w_down, np.uint16), y), "oracle_ffn_rows")
    return y[:n]


def combine(y_perm, inv_pos, topk_w, y_shared=None, H=None) -> np.ndarray:
    """out[t] = sum_j w[t,j] y_perm[inv_pos[t,j]] (+ y_shared[t]), fp64."""
    topk_w = _c(topk_w, np.float32)
    T, k = topk_w.shape
    y_perm = _c(y_perm, np.uint16)
    H = y_perm.shape[1] if H is None else H
    R = y_perm.shape[0]
    if R == 0:
        y_perm = np.zeros((1, H), np.uint16)
    ysh = None if y_shared is None else _c(y_shared, np.uint16)
    out = np.empty((max(T, 1), H), np.float64)
    _check(lib().oracle_combine(T, k, H, R, y_perm, _c(inv_pos, np.int32).reshape(-1), topk_w,
                                _ptr(ysh), out), "oracle_combine")
    return out[:T]


def forward_tokens(dims: dict, tokens, logits, x, local_experts, weights: dict, gate: int = 0, bias=None,
                   scale: float = 1.0, n_group: int = 0, topk_group: int = 0) -> np.ndarray:
    """Layer output [len(tokens), H] in fp64 for the listed tokens, from the definition."""
    d = np.array([dims["T"], dims["H"], dims["E"], dims["k"], dims["I"], dims["S"],
                  dims["E_local"], dims.get("n_shared", 0), dims.get("I_shared", 0), gate], np.int32)
    tokens = _c(tokens, np.int32)
    loc = None if local_experts is None else _c(local_experts, np.int32)
    n_sh = dims.get("n_shared", 0)
    shg = _c(weights["sh_gate"], np.uint16) if n_sh else None
    shu = _c(weights["sh_up"], np.uint16) if n_sh else None
    shd = _c(weights["sh_down"], np.uint16) if n_sh else None
    b = None if bias is None else _c(bias, np.float32)
    out = np.empty((max(len(tokens), 1), dims["H"]), np.float64)
    _check(lib().oracle_forward_tokens(d, len(tokens), tokens, _c(logits, np.float32), _c(x, np.uint16),
                                       _ptr(loc), _c(weights["w_gate"], np.uint16),
                                       _c(weights["w_up"], np.uint16), _c(weights["w_down"], np.uint16),
                                       _ptr(shg), _ptr(shu), _ptr(shd), _ptr(b), float(scale), n_group,
                                       topk_group, out), "oracle_forward_tokens")
    return out[: len(tokens)]


# ---- source-aware expert placement (Sec. 5.2 objective, Sec. 5.3 greedy) ----

def _place_inputs(A, B, D, M, x0):
    A = _c(A, np.int64)
    if A.ndim == 2:
        A = A[None]
    L, S, E = A.shape
    D = _c(D, np.float64)
    G = D.shape[1]
    assert D.shape == (S, G)
    B = None if B is None else _c(B, np.int64).reshape(L, E)
    M = None if M is None else _c(M, np.float64).reshape(L, E, G)
    x0 = _c(x0, np.int32).reshape(L, E)
    return A, B, D, M, x0, (L, S, E, G)


def place_objective(A, D, x, x0, B=None, M=None, m_uniform: float = 1.0) -> np.ndarray:
    """[L, 3] = (C_comm, C_load, C_mig) of placement x (rank per expert, [L, E])."""
    A, B, D, M, x0, (L, S, E, G) = _place_inputs(A, B, D, M, x0)
    x = _c(x, np.int32).reshape(L, E)
    terms = np.empty((max(L, 1), 3), np.float64)
    _check(lib().oracle_place_objective(L, S, E, G, A, _ptr(B), D, _ptr(M), float(m_uniform), x0, x, terms),
           "oracle_place_objective")
    return terms[:L]


def place_greedy(A, D, x0, cap, B=None, M=None, m_uniform: float = 1.0,
                 alpha: float = 1.0, beta: float = 0.0025, gamma: float = 1.0):
    """(x [L, E] rank per expert, step_score [L, E]) of the online greedy."""
    A, B, D, M, x0, (L, S, E, G) = _place_inputs(A, B, D, M, x0)
    cap = _c(cap, np.int32)
    assert cap.shape == (G,)
    x = np.empty((max(L, 1), E), np.int32)
    score = np.empty((max(L, 1), E), np.float64)
    _check(lib().oracle_place_greedy(L, S, E, G, A, _ptr(B), D, _ptr(M), float(m_uniform), x0, cap,
                                     float(alpha), float(beta), float(gamma), x, _ptr(score)),
           "oracle_place_greedy")
    return x[:L], score[:L]


def window_stats(A, x, home, G, B=None, engine=None, n_eng=None, pressure=True):
    """(remote [L,S], total [L,S], rank_load [L,G], pressure [n_eng] or None)."""
    A = _c(A, np.int64)
    if A.ndim == 2:
        A = A[None]
    L, S, E = A.shape
    x = _c(x, np.int32).reshape(L, E)
    home = _c(home, np.int32)
    B = None if B is None else _c(B, np.int64).reshape(L, E)
    eng = None if engine is None else _c(engine, np.int32)
    n_eng = G if n_eng is None else n_eng
    remote = np.empty((max(L, 1), S), np.int64)
    total = np.empty((max(L, 1), S), np.int64)
    rank_load = np.empty((max(L, 1), G), np.int64)
    pr = np.empty(n_eng, np.float64) if pressure else None
    _check(lib().oracle_window_stats(L, S, E, G, A, _ptr(B), x, home, _ptr(eng), n_eng, remote, total,
                                     rank_load, _ptr(pr)), "oracle_window_stats")
    return remote[:L], total[:L], rank_load[:L], pr
