"""Helpers of the GPU-vs-oracle parity tests.

Tolerances (fp32 accumulation of bf16/fp32 inputs against the fp64 oracle):
  scores   |S_g(i) - S_o(i)| <= 2e-3 * max(|S_o(i)|, mean_P |S_o|, mean_P S_imp)
           The floor mean_P S_imp is the common magnitude of both terms of
           Eq. (7) (the diversity term is rescaled to it), so a head whose
           scores are all (near) zero is still compared at its natural scale.
  stats    2e-3 relative (distance statistics: with an absolute floor of
           2e-3 * D_E for near-zero values; the S_div extrema with a floor of
           2e-3 * max S_div, the scale of S_div, which Eq. (3) keeps in [0, 1]).
  indices  |sel_g| = |sel_o|, window present, ascending and unique; every
           disagreement lies in the oracle near-tie band |S_o - theta| <=
           2e-3 * max(|theta|, floor) around the k-th largest oracle score
           theta; and the GPU set is exactly the top-k of the GPU's own fp32
           scores under the tie rule (larger first, then smaller position).
  compact  bit-exact: Kc == K[idx_g], Vc == V[idx_g].
"""
from __future__ import annotations

import numpy as np
import torch

import oracle
import workloads as W

RTOL = 2e-3


def dev(a: np.ndarray, dtype: str) -> torch.Tensor:
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def host_bits(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def gpu_pass(wl: W.Workload, params=None, mode=None, budget=None, pre=None):
    """Run score -> select -> compact through the C ABI; returns numpy outputs.
    `budget` overrides the workload's per-sequence budgets (e.g. [L][Hkv]
    budgets with mode HEAD_BUDGETS)."""
    import paper_2609_06663_amd as P
    from paper_2609_06663_amd.pipeline import EvictionPass
    shape = P.Shape(wl.L, wl.Hq, wl.Hkv, wl.D, wl.w, wl.cu_seqlens)
    m = mode if mode is not None else (P.LAYER_FLAT if wl.mode == "layer_flat" else P.PER_HEAD)
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    ep = EvictionPass(shape, wl.budget if budget is None else budget, m, params or P.Params(), tdt)
    K, V, Q = dev(wl.K, wl.dtype), dev(wl.V, wl.dtype), dev(wl.Q, wl.dtype)
    ep.run(K, V, Q, pre=None if pre is None else torch.from_numpy(np.ascontiguousarray(pre, np.float32)).cuda())
    torch.cuda.synchronize()
    U = wl.L * wl.Hkv * wl.B
    out = dict(
        scores=ep.scores.cpu().numpy().reshape(wl.L, wl.Hkv, -1),
        lambda_=ep.lambda_.cpu().numpy().reshape(wl.L, wl.Hkv, wl.B),
        stats=ep.stats.cpu().numpy().reshape(wl.L, wl.Hkv, wl.B, P.NSTATS),
        idx=ep.idx[:ep.n_idx].cpu().numpy(),
        counts=ep.counts[:U].cpu().numpy().reshape(wl.L, wl.Hkv, wl.B),
        offsets=ep.offsets[:U].cpu().numpy().reshape(wl.L, wl.Hkv, wl.B),
        Kc=host_bits(ep.Kc[:ep.n_idx]),
        Vc=host_bits(ep.Vc[:ep.n_idx]),
    )
    return out


def oracle_params(p=None):
    import math
    if p is None:
        return oracle.Params()
    lo = float(p.lambda_override)
    return oracle.Params(alpha=float(np.float32(p.alpha)), beta=float(np.float32(p.beta)),
                         eps=float(np.float32(p.eps)), tau=float(np.float32(p.tau)),
                         pool_kernel=int(p.pool_kernel), causal=bool(p.causal),
                         lambda_override=lo if not math.isnan(lo) else math.nan,
                         imp_mode=int(p.imp_mode), norm_mode=int(p.norm_mode),
                         winsor_q=float(np.float32(p.winsor_q)), mad_tau=float(np.float32(p.mad_tau)),
                         redundancy=int(p.redundancy), centroid_scope=int(p.centroid_scope))


def unit_slices(wl: W.Workload, s: int):
    cu = wl.cu_seqlens
    T = cu[s + 1] - cu[s]
    off = cu[s] - s * wl.w
    return T, off


def oracle_all(wl: W.Workload, params=None):
    """Oracle scores [L][Hkv][Ptot] and statistics [L][Hkv][B][NSTATS] of every
    unit, on all host threads."""
    import os
    vn = params is not None and params.imp_mode
    return oracle.score(wl.K, wl.Q, wl.L, wl.Hq, wl.Hkv, wl.cu_seqlens, wl.D, wl.w, oracle_params(params),
                        nthreads=os.cpu_count() or 1, V=wl.V if vn else None)


def oracle_unit(wl: W.Workload, l: int, h: int, s: int, params=None):
    cu = wl.cu_seqlens
    K = wl.K[l, h, cu[s]:cu[s + 1]]
    Q = wl.Q[l, h * wl.G:(h + 1) * wl.G, s]
    V = wl.V[l, h, cu[s]:cu[s + 1]] if params is not None and params.imp_mode else None
    return oracle.score_unit(K, Q, wl.w, oracle_params(params), V=V)


def check_scores(Sg: np.ndarray, So: np.ndarray, imp_mean: float, what: str = ""):
    floor = max(float(np.mean(np.abs(So))), float(imp_mean))
    scale = np.maximum(np.abs(So), floor)
    err = np.abs(Sg.astype(np.float64) - So)
    bad = err > RTOL * scale
    assert not bad.any(), (f"{what}: {int(bad.sum())} scores off; worst rel "
                           f"{float((err / scale).max()):.3e} at {int(np.argmax(err / scale))}")
    return floor


STAT_NAMES = ["lambda", "r_C", "r_E", "D_E", "dmin", "dmax", "sdiv_min", "sdiv_max", "imp_mean",
              "sbar_mean", "mu_norm2", "scale"]


def check_stats(sg: np.ndarray, so: np.ndarray, what: str = "", skip=()):
    for k, name in enumerate(STAT_NAMES):
        if name in skip:
            continue
        floor = abs(so[3]) if name in ("D_E", "dmin", "dmax") else 0.0
        if name in ("sdiv_min", "sdiv_max"):
            floor = abs(so[7])
        tol = RTOL * max(abs(so[k]), floor, 1e-30)
        assert abs(float(sg[k]) - so[k]) <= tol, f"{what}: stat {name} gpu {sg[k]!r} oracle {so[k]!r}"


def topk_rule(S: np.ndarray, k: int) -> np.ndarray:
    """Positions of the k largest (larger first, then smaller position), ascending."""
    if k == 0:
        return np.zeros(0, np.int64)
    S = np.asarray(S, dtype=np.float64)
    key = np.where(np.isnan(S), -np.inf, S)
    order = np.lexsort((np.arange(len(S)), -key))
    return np.sort(order[:k])


def check_unit_selection(idx_g: np.ndarray, Sg: np.ndarray, So: np.ndarray, T: int, w: int, b: int,
                         floor: float, what: str = ""):
    P = T - w
    beff = min(b, T)
    assert len(idx_g) == beff, f"{what}: {len(idx_g)} entries, want {beff}"
    if b >= T:
        np.testing.assert_array_equal(idx_g, np.arange(T), err_msg=what)
        return 0
    k = b - w
    np.testing.assert_array_equal(idx_g[k:], np.arange(P, T), err_msg=f"{what}: window")
    sel = idx_g[:k]
    assert np.all(np.diff(sel) > 0) if k > 1 else True, f"{what}: not ascending"
    assert k == 0 or (sel[0] >= 0 and sel[-1] < P), f"{what}: position out of range"
    np.testing.assert_array_equal(sel, topk_rule(Sg, k), err_msg=f"{what}: not the top-k of the GPU scores")
    if k == 0:
        return 0
    sel_o = topk_rule(So, k)
    theta = np.sort(So)[::-1][k - 1]
    band = RTOL * max(abs(theta), floor)
    diff = np.setxor1d(sel, sel_o)
    far = [i for i in diff if abs(So[i] - theta) > band]
    assert not far, f"{what}: {len(far)} disagreements outside the near-tie band (e.g. {far[:5]})"
    return len(diff)
