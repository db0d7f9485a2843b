"""Thin Python binding of libecokv.so (argument marshalling only).

Every step of the eviction pass runs in the HIP kernels behind the C ABI
declared in ``include/ecokv.h``; this module turns torch tensors into device
pointers, the current HIP stream into a handle, and error codes into
exceptions.  PyTorch provides device memory and streams only.  If the built
library is missing, importing this module raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence

import torch

# ECOKV_LIBRARY names another build of the library to load instead of the
# in-tree one (for instance one whose host code is built with sanitizers).
_LIB_PATH = os.environ.get("ECOKV_LIBRARY") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libecokv.so")

OK, EINVAL, EWORKSPACE, EUNSUPPORTED, EHIP, ETIMEOUT = 0, -1, -2, -3, -4, -5
BF16, F32 = 0, 1
PER_HEAD, LAYER_FLAT, HEAD_BUDGETS = 0, 1, 2
IMP_ATTN, IMP_ATTN_VNORM = 0, 1
NORM_MINMAX, NORM_WINSOR, NORM_MAD = 0, 1, 2
RED_EUCLID, RED_STD = 0, 1
CENTROID_ALL, CENTROID_PREFIX = 0, 1
MAX_SEQS, MAX_ROWS = 64, 64
NSTATS = 12
STAT = dict(lambda_=0, rC=1, rE=2, DE=3, dmin=4, dmax=5, sdmin=6, sdmax=7, imp_mean=8, sbar_mean=9,
            mu_norm2=10, scale=11)

EXPORTS = ["ecokv_default_params", "ecokv_workspace_size", "ecokv_workspace_status", "ecokv_score", "ecokv_score_v",
           "ecokv_score_pre", "ecokv_score_noalloc", "ecokv_prefill_workspace_size", "ecokv_prefill_write",
           "ecokv_index_count",
           "ecokv_index_count_mode", "ecokv_select_workspace_size", "ecokv_select", "ecokv_compact",
           "ecokv_pyramid_budgets",
           "ecokv_decode_workspace_size", "ecokv_decode",
           "ecokv_last_error", "ecokv_stage_times"]


class _StageTime(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("ms", ctypes.c_double), ("launches", ctypes.c_int64)]


class EcoKVError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libecokv error {code}: {msg}")
        self.code = code


class _Shape(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("window", ctypes.c_int32), ("num_seqs", ctypes.c_int32),
                ("cu_seqlens", ctypes.POINTER(ctypes.c_int32))]


class Params(ctypes.Structure):
    """ecokv_params; defaults are the paper's (Table 6)."""
    _fields_ = [("alpha", ctypes.c_float), ("beta", ctypes.c_float), ("eps", ctypes.c_float),
                ("tau", ctypes.c_float), ("pool_kernel", ctypes.c_int32), ("causal", ctypes.c_int32),
                ("lambda_override", ctypes.c_float), ("imp_mode", ctypes.c_int32),
                ("norm_mode", ctypes.c_int32), ("winsor_q", ctypes.c_float), ("mad_tau", ctypes.c_float),
                ("redundancy", ctypes.c_int32), ("centroid_scope", ctypes.c_int32)]

    def __init__(self, alpha=0.8, beta=0.6, eps=1e-6, tau=0.0, pool_kernel=5, causal=True,
                 lambda_override=math.nan, imp_mode=IMP_ATTN, norm_mode=NORM_MINMAX, winsor_q=0.01,
                 mad_tau=1.0, redundancy=RED_EUCLID, centroid_scope=CENTROID_ALL):
        super().__init__(alpha, beta, eps, tau, int(pool_kernel), int(bool(causal)), lambda_override,
                         int(imp_mode), int(norm_mode), winsor_q, mad_tau, int(redundancy), int(centroid_scope))


class Shape:
    """ecokv_shape plus the host array of sequence offsets it points to."""

    def __init__(self, num_layers: int, num_q_heads: int, num_kv_heads: int, head_dim: int, window: int,
                 cu_seqlens: Sequence[int]):
        self.cu = (ctypes.c_int32 * len(cu_seqlens))(*[int(x) for x in cu_seqlens])
        self.c = _Shape(num_layers, num_q_heads, num_kv_heads, head_dim, window, len(cu_seqlens) - 1,
                        ctypes.cast(self.cu, ctypes.POINTER(ctypes.c_int32)))

    @property
    def cu_seqlens(self):
        return list(self.cu)

    # element counts of the tensors of a call, for the binding's checks
    @property
    def units(self) -> int:
        c = self.c
        return c.num_layers * c.num_kv_heads * c.num_seqs

    @property
    def ttot(self) -> int:
        return int(self.cu[self.c.num_seqs])

    @property
    def ptot(self) -> int:
        return self.ttot - self.c.num_seqs * self.c.window

    def kv_numel(self) -> int:
        c = self.c
        return c.num_layers * c.num_kv_heads * self.ttot * c.head_dim

    def q_numel(self) -> int:
        c = self.c
        return c.num_layers * c.num_q_heads * c.num_seqs * c.window * c.head_dim

    def score_numel(self) -> int:
        return self.c.num_layers * self.c.num_kv_heads * self.ptot


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is not built; run `python paper_2609_06663_amd/build.py`")
    lib = ctypes.CDLL(_LIB_PATH)
    vp, sp, pp = ctypes.c_void_p, ctypes.POINTER(_Shape), ctypes.POINTER(Params)
    i32p = ctypes.POINTER(ctypes.c_int32)
    lib.ecokv_default_params.argtypes = [pp]
    lib.ecokv_workspace_size.argtypes = [sp, pp, ctypes.POINTER(ctypes.c_size_t)]
    lib.ecokv_workspace_status.argtypes = [vp, vp]
    lib.ecokv_score.argtypes = [vp, vp, ctypes.c_int, sp, pp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.ecokv_score_v.argtypes = [vp, vp, vp, ctypes.c_int, sp, pp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.ecokv_score_pre.argtypes = [vp, vp, vp, ctypes.c_int, sp, pp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.ecokv_score_noalloc.argtypes = [vp, vp, vp, ctypes.c_int, sp, pp, vp, vp, vp, vp, vp]
    lib.ecokv_prefill_workspace_size.argtypes = [sp, ctypes.POINTER(ctypes.c_size_t)]
    lib.ecokv_prefill_write.argtypes = [vp, vp, vp, ctypes.c_int, sp, pp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.ecokv_index_count.argtypes = [sp, i32p, ctypes.POINTER(ctypes.c_int64)]
    lib.ecokv_index_count_mode.argtypes = [sp, ctypes.c_int, i32p, ctypes.POINTER(ctypes.c_int64)]
    lib.ecokv_decode_workspace_size.argtypes = [sp, ctypes.c_int32, ctypes.POINTER(ctypes.c_size_t)]
    lib.ecokv_decode.argtypes = [vp, vp, vp, ctypes.c_int, sp, vp, vp, ctypes.c_int32, vp, vp, vp,
                                 ctypes.c_size_t, vp]
    lib.ecokv_pyramid_budgets.argtypes = [ctypes.c_int, ctypes.c_double, ctypes.c_double, ctypes.c_int, i32p]
    lib.ecokv_select_workspace_size.argtypes = [sp, ctypes.c_int, ctypes.POINTER(ctypes.c_size_t)]
    lib.ecokv_select.argtypes = [vp, sp, ctypes.c_int, i32p, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.ecokv_compact.argtypes = [vp, vp, ctypes.c_int, sp, ctypes.c_int, i32p, vp, vp, vp, vp, vp, vp]
    lib.ecokv_last_error.restype = ctypes.c_char_p
    lib.ecokv_stage_times.argtypes = [ctypes.POINTER(_StageTime), ctypes.c_int, ctypes.POINTER(ctypes.c_int)]
    for name in EXPORTS:
        if name != "ecokv_last_error":
            getattr(lib, name).restype = ctypes.c_int
    return lib


lib = _load()


def _check(rc: int):
    if rc != OK:
        raise EcoKVError(rc, lib.ecokv_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libecokv must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


_ELEM = {torch.bfloat16: "bf16", torch.float32: "float32", torch.int32: "int32", torch.uint8: "uint8"}


def _arg(t: Optional[torch.Tensor], name: str, dtypes, numel: int, device, optional: bool = False):
    """Device pointer of `t` after checking that it is a contiguous tensor on
    `device` with an allowed element type and at least `numel` elements: the
    kernels trust these sizes, so a mismatch is refused here rather than read
    or written out of bounds on the GPU."""
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor (got {t.device})")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, the call's tensors on {device}")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} must be {' or '.join(_ELEM.get(d, str(d)) for d in dtypes)} (got {t.dtype})")
    if t.numel() < numel:
        raise ValueError(f"{name} has {t.numel()} elements, the call needs {numel}")
    return _ptr(t)


_KV_TYPES = (torch.bfloat16, torch.float32)
_F32 = (torch.float32,)
_I32 = (torch.int32,)
_U8 = (torch.uint8,)


def _workspace(workspace: Optional[torch.Tensor], nbytes: int, device, stream):
    """The caller's workspace, or a zero-filled one allocated here; a tensor
    allocated here is recorded on `stream`, so that torch's allocator does not
    hand its memory out again before the work queued there has used it."""
    if workspace is not None:
        return workspace
    ws = torch.zeros(max(nbytes, 256), dtype=torch.uint8, device=device)
    if stream is not None:
        ws.record_stream(stream)
    return ws


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported element type {t.dtype} (bf16 or fp32)")


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _flat_ints(x) -> list:
    if hasattr(x, "reshape"):  # numpy array or tensor
        x = x.reshape(-1).tolist()
    out = []
    for v in x:
        if isinstance(v, (list, tuple)):
            out.extend(_flat_ints(v))
        else:
            out.append(int(v))
    return out


def _budget(shape: Shape, budget, mode: int = PER_HEAD):
    """Host budget array: one per sequence, or [L][H_kv] for HEAD_BUDGETS."""
    vals = _flat_ints(budget)
    c = shape.c
    n = c.num_layers * c.num_kv_heads if mode == HEAD_BUDGETS else c.num_seqs
    if len(vals) != n:
        raise ValueError("HEAD_BUDGETS takes one budget per (layer, KV head)" if mode == HEAD_BUDGETS
                         else "one budget per sequence")
    return (ctypes.c_int32 * max(n, 1))(*vals)


def ecokv_default_params() -> Params:
    p = Params()
    _check(lib.ecokv_default_params(ctypes.byref(p)))
    return p


def ecokv_workspace_size(shape: Shape, params: Optional[Params] = None) -> int:
    n = ctypes.c_size_t(0)
    _check(lib.ecokv_workspace_size(ctypes.byref(shape.c), ctypes.byref(params or Params()), ctypes.byref(n)))
    return n.value


def _score_args(K, V, Q_win, shape: Shape, p: Params, scores, lambda_, stats, workspace, stream, pre=None):
    """Checked pointers of a score call, in the order of ecokv_score_pre."""
    L = shape.c.num_layers
    if L == 0:  # nothing is read or written
        return [_ptr(K), _ptr(V), _ptr(Q_win), _dtype_code(K) if K is not None else BF16, ctypes.byref(shape.c),
                ctypes.byref(p), _ptr(pre), _ptr(scores), _ptr(lambda_), _ptr(stats), _ptr(workspace),
                0 if workspace is None else workspace.numel(), _stream(stream)]
    dev = K.device if isinstance(K, torch.Tensor) else None
    kp = _arg(K, "K", _KV_TYPES, shape.kv_numel(), dev)
    if Q_win.dtype != K.dtype or (V is not None and V.dtype != K.dtype):
        raise TypeError("K, V and Q_win must have the same element type")
    vp = _arg(V, "V", _KV_TYPES, shape.kv_numel(), dev, optional=p.imp_mode != IMP_ATTN_VNORM)
    qp = _arg(Q_win, "Q_win", _KV_TYPES, shape.q_numel(), dev)
    R = shape.c.num_q_heads // shape.c.num_kv_heads * shape.c.window
    pp = _arg(pre, "pre", _F32, shape.units * (2 * shape.c.head_dim + 2 * R), dev, optional=True)
    sp_ = _arg(scores, "scores", _F32, shape.score_numel(), dev)
    lp = _arg(lambda_, "lambda", _F32, shape.units, dev, optional=True)
    stp = _arg(stats, "stats", _F32, shape.units * NSTATS, dev, optional=True)
    need = ecokv_workspace_size(shape, p)
    workspace = _workspace(workspace, need, dev, stream)
    wp = _arg(workspace, "workspace", _U8, need, dev)
    return [kp, vp, qp, _dtype_code(K), ctypes.byref(shape.c), ctypes.byref(p), pp, sp_, lp, stp, wp,
            workspace.numel(), _stream(stream)]


def ecokv_score(K: torch.Tensor, Q_win: torch.Tensor, shape: Shape, params: Optional[Params],
                scores: torch.Tensor, lambda_: Optional[torch.Tensor] = None,
                stats: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                stream=None) -> None:
    """Enqueue ecokv_score.  `workspace` (uint8, >= ecokv_workspace_size bytes,
    zero-filled before its first use) is allocated here when not given."""
    p = params or Params()
    a = _score_args(K, None, Q_win, shape, p, scores, lambda_, stats, workspace, stream)
    del a[1], a[5]  # no V, no pre
    _check(lib.ecokv_score(*a))


def ecokv_score_v(K: torch.Tensor, V: Optional[torch.Tensor], Q_win: torch.Tensor, shape: Shape,
                  params: Optional[Params], scores: torch.Tensor, lambda_: Optional[torch.Tensor] = None,
                  stats: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                  stream=None) -> None:
    """Enqueue ecokv_score_v (V is read with imp_mode IMP_ATTN_VNORM)."""
    p = params or Params()
    a = _score_args(K, V, Q_win, shape, p, scores, lambda_, stats, workspace, stream)
    del a[6]  # no pre
    _check(lib.ecokv_score_v(*a))


def ecokv_score_pre(K: torch.Tensor, V: Optional[torch.Tensor], Q_win: torch.Tensor, shape: Shape,
                    params: Optional[Params], pre: torch.Tensor, scores: torch.Tensor,
                    lambda_: Optional[torch.Tensor] = None, stats: Optional[torch.Tensor] = None,
                    workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    """Enqueue ecokv_score_pre: `pre` (float32 [L][Hkv][B][2D + 2R]) holds the
    key sums and window softmax statistics a prefill produced."""
    p = params or Params()
    if pre is not None and pre.dtype != torch.float32:
        raise TypeError("pre is float32")
    a = _score_args(K, V, Q_win, shape, p, scores, lambda_, stats, workspace, stream, pre=pre)
    _check(lib.ecokv_score_pre(*a))


def ecokv_prefill_workspace_size(shape: Shape) -> int:
    n = ctypes.c_size_t(0)
    _check(lib.ecokv_prefill_workspace_size(ctypes.byref(shape.c), ctypes.byref(n)))
    return n.value


def ecokv_prefill_write(K_new: torch.Tensor, V_new: Optional[torch.Tensor], Q_win: torch.Tensor, shape: Shape,
                        params: Optional[Params], K_cache: torch.Tensor, V_cache: Optional[torch.Tensor],
                        pre: torch.Tensor, workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    """Enqueue ecokv_prefill_write: K_new / V_new token-major ([L][T_total][Hkv][D])
    into K_cache / V_cache (the pass's [L][Hkv][T_total][D]), and `pre` (float32
    [L][Hkv][B][2D + 2R]) for ecokv_score_pre.  V_new and V_cache: both or neither."""
    p = params or Params()
    if shape.c.num_layers == 0:
        return
    if (V_new is None) != (V_cache is None):
        raise ValueError("V_new and V_cache: both or neither")
    dev = K_new.device
    kn = _arg(K_new, "K_new", _KV_TYPES, shape.kv_numel(), dev)
    for t, n in ((Q_win, "Q_win"), (K_cache, "K_cache"), (V_new, "V_new"), (V_cache, "V_cache")):
        if t is not None and t.dtype != K_new.dtype:
            raise TypeError(f"{n} must have the element type of K_new")
    vn = _arg(V_new, "V_new", _KV_TYPES, shape.kv_numel(), dev, optional=True)
    qp = _arg(Q_win, "Q_win", _KV_TYPES, shape.q_numel(), dev)
    kc = _arg(K_cache, "K_cache", _KV_TYPES, shape.kv_numel(), dev)
    vc = _arg(V_cache, "V_cache", _KV_TYPES, shape.kv_numel(), dev, optional=True)
    R = shape.c.num_q_heads // shape.c.num_kv_heads * shape.c.window
    pp = _arg(pre, "pre", _F32, shape.units * (2 * shape.c.head_dim + 2 * R), dev)
    need = ecokv_prefill_workspace_size(shape)
    workspace = _workspace(workspace, need, dev, stream)
    wp = _arg(workspace, "workspace", _U8, need, dev)
    _check(lib.ecokv_prefill_write(kn, vn, qp, _dtype_code(K_new), ctypes.byref(shape.c), ctypes.byref(p), kc, vc, pp,
                                   wp, workspace.numel(), _stream(stream)))


def ecokv_score_noalloc(K: torch.Tensor, V: Optional[torch.Tensor], Q_win: torch.Tensor, shape: Shape,
                        params: Optional[Params], pre: Optional[torch.Tensor], scores: torch.Tensor,
                        lambda_: Optional[torch.Tensor] = None, stats: Optional[torch.Tensor] = None,
                        stream=None) -> None:
    """Enqueue ecokv_score_noalloc: ecokv_score_pre (pre may be None) with the
    library's own per-device scratch; nothing is allocated here either."""
    p = params or Params()
    if pre is not None and pre.dtype != torch.float32:
        raise TypeError("pre is float32")
    if shape.c.num_layers == 0:
        return
    dev = K.device
    kp = _arg(K, "K", _KV_TYPES, shape.kv_numel(), dev)
    if Q_win.dtype != K.dtype or (V is not None and V.dtype != K.dtype):
        raise TypeError("K, V and Q_win must have the same element type")
    vp = _arg(V, "V", _KV_TYPES, shape.kv_numel(), dev, optional=p.imp_mode != IMP_ATTN_VNORM)
    qp = _arg(Q_win, "Q_win", _KV_TYPES, shape.q_numel(), dev)
    R = shape.c.num_q_heads // shape.c.num_kv_heads * shape.c.window
    prp = _arg(pre, "pre", _F32, shape.units * (2 * shape.c.head_dim + 2 * R), dev, optional=True)
    _check(lib.ecokv_score_noalloc(kp, vp, qp, _dtype_code(K), ctypes.byref(shape.c), ctypes.byref(p), prp,
                                   _arg(scores, "scores", _F32, shape.score_numel(), dev),
                                   _arg(lambda_, "lambda", _F32, shape.units, dev, optional=True),
                                   _arg(stats, "stats", _F32, shape.units * NSTATS, dev, optional=True),
                                   _stream(stream)))


def ecokv_workspace_status(workspace: torch.Tensor, stream=None) -> None:
    """Synchronise `stream` and raise EcoKVError (code ETIMEOUT) if a score call
    on `workspace` since the last query had a wait between blocks give up (its
    lambda and scores of the affected units are then NaN); clears the record."""
    _check(lib.ecokv_workspace_status(_arg(workspace, "workspace", _U8, 4, None), _stream(stream)))


def ecokv_index_count(shape: Shape, budget: Sequence[int]) -> int:
    n = ctypes.c_int64(0)
    _check(lib.ecokv_index_count(ctypes.byref(shape.c), _budget(shape, budget), ctypes.byref(n)))
    return n.value


def ecokv_index_count_mode(shape: Shape, mode: int, budget) -> int:
    n = ctypes.c_int64(0)
    _check(lib.ecokv_index_count_mode(ctypes.byref(shape.c), int(mode), _budget(shape, budget, mode),
                                      ctypes.byref(n)))
    return n.value


def ecokv_pyramid_budgets(num_layers: int, total: float, beta: float, window: int) -> list:
    out = (ctypes.c_int32 * max(int(num_layers), 1))()
    _check(lib.ecokv_pyramid_budgets(int(num_layers), float(total), float(beta), int(window), out))
    return [int(v) for v in out[:num_layers]]


def ecokv_select_workspace_size(shape: Shape, mode: int) -> int:
    n = ctypes.c_size_t(0)
    _check(lib.ecokv_select_workspace_size(ctypes.byref(shape.c), int(mode), ctypes.byref(n)))
    return n.value


def ecokv_select(scores: torch.Tensor, shape: Shape, mode: int, budget, idx: torch.Tensor,
                 counts: Optional[torch.Tensor] = None, offsets: Optional[torch.Tensor] = None,
                 workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    """Enqueue ecokv_select.  `workspace` (uint8, >= ecokv_select_workspace_size
    bytes, zero-filled before its first use) is allocated here when not given."""
    bud = _budget(shape, budget, mode)
    if shape.c.num_layers == 0:
        _check(lib.ecokv_select(_ptr(scores), ctypes.byref(shape.c), int(mode), bud, _ptr(idx), _ptr(counts),
                                _ptr(offsets), _ptr(workspace), 0 if workspace is None else workspace.numel(),
                                _stream(stream)))
        return
    n = ecokv_index_count_mode(shape, mode, budget)
    dev = scores.device if isinstance(scores, torch.Tensor) else None
    flat = int(mode) == LAYER_FLAT
    sp_ = _arg(scores, "scores", _F32, shape.score_numel(), dev)
    ip = _arg(idx, "idx", _I32, n, dev)
    cp = _arg(counts, "counts", _I32, shape.units, dev, optional=not flat)
    op = _arg(offsets, "offsets", _I32, shape.units, dev, optional=not flat)
    need = ecokv_select_workspace_size(shape, mode)
    workspace = _workspace(workspace, need, dev, stream)
    _check(lib.ecokv_select(sp_, ctypes.byref(shape.c), int(mode), bud, ip, cp, op,
                            _arg(workspace, "workspace", _U8, need, dev), workspace.numel(), _stream(stream)))


def ecokv_compact(K: torch.Tensor, V: torch.Tensor, shape: Shape, mode: int, budget,
                  idx: torch.Tensor, counts: Optional[torch.Tensor], offsets: Optional[torch.Tensor],
                  Kc: torch.Tensor, Vc: torch.Tensor, stream=None) -> None:
    if V.dtype != K.dtype or Kc.dtype != K.dtype or Vc.dtype != K.dtype:
        raise TypeError("K, V, Kc and Vc must share one element type")
    bud = _budget(shape, budget, mode)
    if shape.c.num_layers == 0:
        _check(lib.ecokv_compact(_ptr(K), _ptr(V), _dtype_code(K), ctypes.byref(shape.c), int(mode), bud,
                                 _ptr(idx), _ptr(counts), _ptr(offsets), _ptr(Kc), _ptr(Vc), _stream(stream)))
        return
    n = ecokv_index_count_mode(shape, mode, budget)
    dev = K.device
    flat = int(mode) == LAYER_FLAT
    D = shape.c.head_dim
    _check(lib.ecokv_compact(_arg(K, "K", _KV_TYPES, shape.kv_numel(), dev),
                             _arg(V, "V", _KV_TYPES, shape.kv_numel(), dev), _dtype_code(K), ctypes.byref(shape.c),
                             int(mode), bud, _arg(idx, "idx", _I32, n, dev),
                             _arg(counts, "counts", _I32, shape.units, dev, optional=True),
                             _arg(offsets, "offsets", _I32, shape.units, dev, optional=not flat),
                             _arg(Kc, "Kc", _KV_TYPES, n * D, dev), _arg(Vc, "Vc", _KV_TYPES, n * D, dev),
                             _stream(stream)))


def ecokv_decode_workspace_size(shape: Shape, max_count: int) -> int:
    n = ctypes.c_size_t(0)
    _check(lib.ecokv_decode_workspace_size(ctypes.byref(shape.c), int(max_count), ctypes.byref(n)))
    return n.value


def ecokv_decode(Q_dec: torch.Tensor, Kc: torch.Tensor, Vc: torch.Tensor, shape: Shape, counts: torch.Tensor,
                 offsets: torch.Tensor, max_count: int, O: torch.Tensor, lse: Optional[torch.Tensor] = None,
                 workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    """Enqueue ecokv_decode (attention of one query per head over the compressed cache).
    The rows each unit reads (offsets[u] .. + counts[u]) are device values the
    binding cannot see; the caller guarantees they lie inside Kc and Vc, as
    ecokv_select writes them for a cache that ecokv_compact filled."""
    if Kc.dtype != Q_dec.dtype or Vc.dtype != Q_dec.dtype:
        raise TypeError("Q_dec, Kc and Vc must share one element type")
    c = shape.c
    need = ecokv_decode_workspace_size(shape, max_count)
    if c.num_layers == 0:
        return
    dev = Q_dec.device
    D = c.head_dim
    nq = c.num_layers * c.num_q_heads * c.num_seqs
    if Kc.numel() % D or Vc.numel() != Kc.numel():
        raise ValueError("Kc and Vc must hold the same whole number of rows of head_dim elements")
    workspace = _workspace(workspace, need, dev, stream)
    _check(lib.ecokv_decode(_arg(Q_dec, "Q_dec", _KV_TYPES, nq * D, dev), _arg(Kc, "Kc", _KV_TYPES, D, dev),
                            _arg(Vc, "Vc", _KV_TYPES, D, dev), _dtype_code(Q_dec), ctypes.byref(shape.c),
                            _arg(counts, "counts", _I32, shape.units, dev),
                            _arg(offsets, "offsets", _I32, shape.units, dev), int(max_count),
                            _arg(O, "O", _F32, nq * D, dev), _arg(lse, "lse", _F32, nq, dev, optional=True),
                            _arg(workspace, "workspace", _U8, need, dev), workspace.numel(), _stream(stream)))


def ecokv_last_error() -> str:
    return lib.ecokv_last_error().decode()


def ecokv_stage_times(max_entries: int = 32) -> dict:
    """Per-kernel times recorded while ECOKV_STAGE_TIMING=1: {name: (ms, launches)}; clears the record."""
    arr = (_StageTime * max_entries)()
    n = ctypes.c_int(0)
    _check(lib.ecokv_stage_times(arr, int(max_entries), ctypes.byref(n)))
    return {arr[i].name.decode(): (arr[i].ms, int(arr[i].launches)) for i in range(n.value)}
