"""CPU oracle for the ECOKV eviction pass -- TEST INFRASTRUCTURE ONLY.

Python marshalling around ``ecokv_oracle.c`` (plain C, double precision).  Only
``tests/``, ``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline`` leg
may import this package; the HIP product path never does.  Nothing here
imports the HIP package, and the C source shares nothing with it.

Functions follow the paper's steps (see ``ecokv_oracle.c`` for citations):
``score_unit`` (Sec. 3 and Sec. 5, Eqs. (1)-(7), Algorithm 1; with V, the
value-norm importance of Sec. 5.2; the alternatives of Sec. 6.3 / Table 4,
Appendix D and Appendix B.6 through ``Params``), ``score`` (all units of a
tensor), ``select`` (Sec. 3 selection; AdaKV layer-flat budget and budgets
per layer and head, Appendix A.1), ``pyramid_budgets`` (PyramidKV's layer
schedule, Appendix A.1), ``compact`` (gather of the kept rows) and
``decode`` (attention of one query per head over the compressed cache).
Every one is pinned by ``tests/test_oracle_pins.py``.
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ecokv_oracle.c")
_LIB = os.path.join(_HERE, "libecokv_oracle.so")

NSTATS = 12
STAT = dict(lambda_=0, rC=1, rE=2, DE=3, dmin=4, dmax=5, sdmin=6, sdmax=7,
            imp_mean=8, sbar_mean=9, mu_norm2=10, scale=11)
PER_HEAD, LAYER_FLAT, HEAD_BUDGETS = 0, 1, 2
IMP_ATTN, IMP_ATTN_VNORM = 0, 1
NORM_MINMAX, NORM_WINSOR, NORM_MAD = 0, 1, 2
RED_EUCLID, RED_STD = 0, 1
CENTROID_ALL, CENTROID_PREFIX = 0, 1
BF16, F32 = 0, 1


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (double precision, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fopenmp",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class _Params(ctypes.Structure):
    _fields_ = [("alpha", ctypes.c_double), ("beta", ctypes.c_double), ("eps", ctypes.c_double),
                ("tau", ctypes.c_double), ("pool_kernel", ctypes.c_int), ("causal", ctypes.c_int),
                ("lambda_override", ctypes.c_double), ("imp_mode", ctypes.c_int), ("norm_mode", ctypes.c_int),
                ("winsor_q", ctypes.c_double), ("mad_tau", ctypes.c_double), ("redundancy", ctypes.c_int),
                ("centroid_scope", ctypes.c_int)]


_TRACE_FIELDS = ["a", "imp", "dE", "cosmu", "sC", "sE", "sdiv", "sbar", "stilde", "kbar", "mu", "rowmass"]


class _Trace(ctypes.Structure):
    _fields_ = [(n, ctypes.POINTER(ctypes.c_double)) for n in _TRACE_FIELDS]


@dataclasses.dataclass
class Params:
    alpha: float = 0.8            # Table 6
    beta: float = 0.6             # Table 6
    eps: float = 1e-6
    tau: float = 0.0              # <= 0 -> sqrt(D)  (Sec. 5.2)
    pool_kernel: int = 5          # Table 6
    causal: bool = True
    lambda_override: float = math.nan
    imp_mode: int = IMP_ATTN       # IMP_ATTN_VNORM: times the value norm (Sec. 5.2)
    norm_mode: int = NORM_MINMAX   # s_E normalisation (Sec. 6.3, Table 4)
    winsor_q: float = 0.01
    mad_tau: float = 1.0
    redundancy: int = RED_EUCLID   # RED_STD: r_std (Appendix D)
    centroid_scope: int = CENTROID_ALL  # CENTROID_PREFIX: Appendix B.6

    def c(self) -> _Params:
        return _Params(self.alpha, self.beta, self.eps, self.tau, int(self.pool_kernel),
                       int(bool(self.causal)), self.lambda_override, int(self.imp_mode), int(self.norm_mode),
                       float(self.winsor_q), float(self.mad_tau), int(self.redundancy),
                       int(self.centroid_scope))


_lib = None
_lib_path = _LIB  # the build lib() loads


def use_library(path: str) -> None:
    """Load the routines from another build of this source from now on: the
    planted-mistake test builds altered copies and checks that the pins
    fail on each."""
    global _lib, _lib_path
    _lib, _lib_path = None, path


def lib():
    global _lib
    if _lib is None:
        if _lib_path == _LIB and not os.path.exists(_LIB):
            build(force=False)
        L = ctypes.CDLL(_lib_path)
        vp, i32p, dp = ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_double)
        L.ora_score_unit_v.argtypes = [vp, vp, vp, ctypes.c_size_t, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                       ctypes.c_int, ctypes.c_int, ctypes.POINTER(_Params), dp, dp,
                                       ctypes.POINTER(_Trace)]
        L.ora_score_v.argtypes = [vp, vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                  ctypes.c_int, i32p, ctypes.c_int, ctypes.c_int, ctypes.POINTER(_Params), dp,
                                  dp, ctypes.c_int]
        L.ora_select_unit.argtypes = [dp, ctypes.c_int, ctypes.c_int, ctypes.c_int, i32p]
        L.ora_select_flat.argtypes = [dp, ctypes.c_size_t, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                      ctypes.c_int, i32p, i32p]
        L.ora_select.argtypes = [dp, ctypes.c_int, ctypes.c_int, ctypes.c_int, i32p, ctypes.c_int, i32p,
                                 ctypes.c_int, i32p, i32p, i32p, ctypes.c_int]
        L.ora_compact.argtypes = [vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, i32p,
                                  ctypes.c_int, i32p, i32p, i32p, vp, vp]
        L.ora_prefill_unit.argtypes = [vp, vp, ctypes.c_size_t, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                       ctypes.c_int, ctypes.c_int, ctypes.c_int, dp]
        L.ora_prefill_sums.argtypes = [vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                       ctypes.c_int, i32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, dp, ctypes.c_int]
        L.ora_decode.argtypes = [vp, vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                 ctypes.c_int, i32p, i32p, dp, dp]
        _lib = L
    return _lib


def _dp(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _ip(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.uint16:
        return BF16
    if a.dtype == np.float32:
        return F32
    raise TypeError("oracle inputs are bf16 bit patterns (uint16) or float32")


def score_unit(K: np.ndarray, Q: np.ndarray, w: int, params: Optional[Params] = None,
               trace: bool = False, V: Optional[np.ndarray] = None) -> dict:
    """Score one (layer, KV head, sequence) unit.

    K: [T, D] keys (uint16 bf16 bits or float32).  Q: [G, w, D] window queries of
    the G query heads sharing this KV head.  V: [T, D] values of the unit's
    tokens (needed with imp_mode IMP_ATTN_VNORM).  Returns ``S`` [P] (float64),
    ``stats`` [NSTATS] and, with ``trace``, every intermediate of the paper's
    steps (a, imp, dE, cosmu, sC, sE, sdiv, sbar, stilde, kbar, mu, rowmass).
    """
    p = params or Params()
    K = np.ascontiguousarray(K)
    Q = np.ascontiguousarray(Q)
    code = _dtype_code(K)
    assert _dtype_code(Q) == code and K.ndim == 2 and Q.ndim == 3
    T, D = K.shape
    G = Q.shape[0]
    assert Q.shape[1] == w and Q.shape[2] == D
    P = T - w
    S = np.zeros(max(P, 0), np.float64)
    stats = np.zeros(NSTATS, np.float64)
    out = {"S": S, "stats": stats}
    tr_ptr = None
    if trace:
        sizes = dict(a=P, imp=P, dE=T, cosmu=P, sC=P, sE=P, sdiv=P, sbar=P, stilde=P, kbar=D, mu=D,
                     rowmass=G * w)
        arrs = {k: np.zeros(v, np.float64) for k, v in sizes.items()}
        tr = _Trace(*[_dp(arrs[n]) for n in _TRACE_FIELDS])
        tr_ptr = ctypes.byref(tr)
        out.update(arrs)
    pc = p.c()
    if V is not None:
        V = np.ascontiguousarray(V)
        assert V.shape == K.shape and _dtype_code(V) == code
    rc = lib().ora_score_unit_v(K.ctypes.data, None if V is None else V.ctypes.data, Q.ctypes.data, w * D,
                                code, T, D, G, w, ctypes.byref(pc), _dp(S), _dp(stats), tr_ptr)
    if rc != 0:
        raise ValueError(f"oracle rejected the unit (rc={rc})")
    return out


def score(K, Q, L, Hq, Hkv, cu_seqlens, D, w, params: Optional[Params] = None, nthreads: int = 1, V=None):
    """Score every unit.  K [L][Hkv][Ttot][D], Q [L][Hq][B][w][D], V like K
    (needed with imp_mode IMP_ATTN_VNORM).

    Returns S [L][Hkv][Ptot] (float64) and stats [L][Hkv][B][NSTATS]."""
    p = params or Params()
    K = np.ascontiguousarray(K)
    Q = np.ascontiguousarray(Q)
    if V is not None:
        V = np.ascontiguousarray(V)
        assert V.shape == K.shape and V.dtype == K.dtype
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    B = len(cu) - 1
    Ptot = int(cu[-1]) - B * w
    S = np.zeros((L, Hkv, Ptot), np.float64)
    stats = np.zeros((L, Hkv, B, NSTATS), np.float64)
    pc = p.c()
    rc = lib().ora_score_v(K.ctypes.data, None if V is None else V.ctypes.data, Q.ctypes.data, _dtype_code(K),
                           L, Hq, Hkv, B, _ip(cu), D, w, ctypes.byref(pc), _dp(S), _dp(stats), nthreads)
    if rc != 0:
        raise ValueError(f"oracle rejected the shape (rc={rc})")
    return S, stats


def prefill_unit(K: np.ndarray, Q: np.ndarray, w: int, causal: bool = True) -> np.ndarray:
    """The first sweep's results of one unit as a prefill hands them to the
    pass: [2D + 2R] = sum k, sum k/|k|, per window row r = g w + j the largest
    visible logit q.k/sqrt(D) and the sum of exp(logit - largest).
    K: [T, D], Q: [G, w, D] (uint16 bf16 bits or float32)."""
    K = np.ascontiguousarray(K)
    Q = np.ascontiguousarray(Q)
    code = _dtype_code(K)
    assert _dtype_code(Q) == code and K.ndim == 2 and Q.ndim == 3 and Q.shape[1] == w
    T, D = K.shape
    G = Q.shape[0]
    out = np.zeros(2 * D + 2 * G * w, np.float64)
    rc = lib().ora_prefill_unit(K.ctypes.data, Q.ctypes.data, w * D, code, T, D, G, w, int(bool(causal)), _dp(out))
    if rc != 0:
        raise ValueError(f"oracle rejected the unit (rc={rc})")
    return out


def prefill_sums(K, Q, L, Hq, Hkv, cu_seqlens, D, w, causal: bool = True, nthreads: int = 1) -> np.ndarray:
    """prefill_unit over every unit: K [L][Hkv][Ttot][D], Q [L][Hq][B][w][D];
    returns [L][Hkv][B][2D + 2R] (float64)."""
    K = np.ascontiguousarray(K)
    Q = np.ascontiguousarray(Q)
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    B = len(cu) - 1
    R = (Hq // Hkv) * w
    out = np.zeros((L, Hkv, B, 2 * D + 2 * R), np.float64)
    rc = lib().ora_prefill_sums(K.ctypes.data, Q.ctypes.data, _dtype_code(K), L, Hq, Hkv, B, _ip(cu), D, w,
                                int(bool(causal)), _dp(out), nthreads)
    if rc != 0:
        raise ValueError(f"oracle rejected the shape (rc={rc})")
    return out


def select_unit(S: np.ndarray, T: int, w: int, b: int) -> np.ndarray:
    S = np.ascontiguousarray(S, dtype=np.float64)
    out = np.zeros(min(b, T), np.int32)
    n = lib().ora_select_unit(_dp(S), T, w, b, _ip(out))
    if n < 0:
        raise ValueError("invalid selection arguments")
    return out


def select_flat(S_heads: np.ndarray, T: int, w: int, b: int):
    """S_heads [H][P]: returns (idx packed head-major, counts [H])."""
    S_heads = np.ascontiguousarray(S_heads, dtype=np.float64)
    H = S_heads.shape[0]
    out = np.zeros(H * min(b, T), np.int32)
    counts = np.zeros(H, np.int32)
    n = lib().ora_select_flat(_dp(S_heads), S_heads.shape[1], H, T, w, b, _ip(out), _ip(counts))
    if n < 0:
        raise ValueError("invalid selection arguments")
    return out, counts


def index_count(L, Hkv, cu_seqlens, budget, mode=PER_HEAD) -> int:
    """Entries of idx: budget[s] per sequence, or budget[l][h] with mode HEAD_BUDGETS."""
    B = len(cu_seqlens) - 1
    lens = [int(cu_seqlens[s + 1] - cu_seqlens[s]) for s in range(B)]
    if mode == HEAD_BUDGETS:
        b = np.asarray(budget).reshape(-1)
        return sum(min(int(b[lh]), lens[s]) for lh in range(L * Hkv) for s in range(B))
    return L * Hkv * sum(min(int(budget[s]), lens[s]) for s in range(B))


def pyramid_budgets(m: int, total, beta) -> list:
    """PyramidKV's layer schedule (Appendix A.1) in exact rational arithmetic:
    b^{m-1} = total / (beta m), b^0 = 2 total / m - b^{m-1}, the layers between
    on the straight line from b^0 to b^{m-1}; one layer gets the total.  Each
    value is rounded down.  `total` and `beta` are taken exactly (a float is
    its binary value)."""
    from fractions import Fraction
    tot, bet = Fraction(total), Fraction(beta)
    if m == 1:
        return [math.floor(tot)]
    last = tot / (bet * m)
    first = 2 * tot / m - last
    return [math.floor(first - (first - last) * l / (m - 1)) for l in range(m)]


def select(S, L, Hkv, cu_seqlens, w, budget, mode=PER_HEAD, nthreads: int = 1):
    """Select over every unit; returns idx (packed), counts [L][Hkv][B], offsets [L][Hkv][B].
    `budget` has one entry per sequence, or [L][Hkv] entries with mode HEAD_BUDGETS."""
    S = np.ascontiguousarray(S, dtype=np.float64)
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    bud = np.ascontiguousarray(np.asarray(budget).reshape(-1), dtype=np.int32)
    B = len(cu) - 1
    idx = np.zeros(index_count(L, Hkv, cu, bud, mode), np.int32)
    counts = np.zeros((L, Hkv, B), np.int32)
    offsets = np.zeros((L, Hkv, B), np.int32)
    rc = lib().ora_select(_dp(S), L, Hkv, B, _ip(cu), w, _ip(bud), mode, _ip(idx), _ip(counts),
                          _ip(offsets), nthreads)
    if rc != 0:
        raise ValueError("invalid selection arguments")
    return idx, counts, offsets


def compact(K, V, L, Hkv, cu_seqlens, D, idx, counts, offsets):
    """Gather the kept rows of K and V (exact byte copies)."""
    K = np.ascontiguousarray(K)
    V = np.ascontiguousarray(V)
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    B = len(cu) - 1
    n = int(np.asarray(idx).size)
    Kc = np.zeros((n, D), K.dtype)
    Vc = np.zeros((n, D), V.dtype)
    rc = lib().ora_compact(K.ctypes.data, V.ctypes.data, K.dtype.itemsize, L, Hkv, B, _ip(cu), D,
                           _ip(np.ascontiguousarray(idx, np.int32)),
                           _ip(np.ascontiguousarray(counts, np.int32)),
                           _ip(np.ascontiguousarray(offsets, np.int32)), Kc.ctypes.data, Vc.ctypes.data)
    if rc != 0:
        raise ValueError("index out of range")
    return Kc, Vc


def decode(Q, Kc, Vc, L, Hq, Hkv, B, D, counts, offsets):
    """Decode attention of one query per (layer, query head, sequence) over the
    compressed cache.  Q [L][Hq][B][D] (uint16 bf16 bits or float32), Kc / Vc
    [entries][D] as written by compact, counts / offsets [L][Hkv][B].
    Returns O [L][Hq][B][D] and lse [L][Hq][B] (float64)."""
    Q = np.ascontiguousarray(Q)
    Kc = np.ascontiguousarray(Kc)
    Vc = np.ascontiguousarray(Vc)
    code = _dtype_code(Q)
    assert _dtype_code(Kc) == code and _dtype_code(Vc) == code
    O = np.zeros((L, Hq, B, D), np.float64)
    lse = np.zeros((L, Hq, B), np.float64)
    rc = lib().ora_decode(Q.ctypes.data, Kc.ctypes.data, Vc.ctypes.data, code, L, Hq, Hkv, B, D,
                          _ip(np.ascontiguousarray(counts, np.int32)), _ip(np.ascontiguousarray(offsets, np.int32)),
                          _dp(O), _dp(lse))
    if rc != 0:
        raise ValueError("invalid decode arguments")
    return O, lse
