"""Seeded synthetic inputs for the ECOKV prefill eviction pass.

This module only draws random tensors and lays them out; it holds none of the
eviction method's arithmetic. Both the CPU oracle (through the tests and the
benchmark's CPU leg) and the HIP library consume the exact bytes produced here.

Shapes and statistics stand in for the multimodal-LLM key caches the paper
evaluates on (Qwen2-VL-7B and LLaVA-NeXT-Mistral-7B on document/VQA benchmarks,
Sec. 6): long runs of near-duplicate "visual" patch keys followed by "text"
keys, all sharing an anisotropic offset so that the mean pairwise cosine is
high, as the paper observes in every layer (Sec. 4, cosine-similarity
paragraph, Fig. 2).  Layouts:

* K, V: ``[L][H_kv][sum_s T_s][D]`` row-major; sequences of a varlen batch are
  packed per head, delimited by ``cu_seqlens``.
* Q_win (the last ``w`` query rows of every query head, per sequence):
  ``[L][H_q][B][w][D]``.
* bf16 tensors are stored as ``uint16`` bit patterns (round-to-nearest-even
  from float32); fp32 tensors as ``float32``.

Every unit (layer, KV head) draws from its own ``SeedSequence([seed, tag, l, h])``
stream so a single unit can be regenerated without generating the rest.
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import List, Optional

import numpy as np

__all__ = [
    "Workload", "to_bf16_bits", "bf16_bits_to_f32",
    "tiny", "layer7b", "stack28", "mha64k", "varlen", "custom", "CONFIG_BUILDERS",
]


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit pattern (uint16), round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + r) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit pattern -> float32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclasses.dataclass
class Workload:
    name: str
    L: int
    Hq: int
    Hkv: int
    D: int
    w: int
    cu_seqlens: List[int]
    dtype: str                 # "bf16" | "f32"
    K: np.ndarray              # [L][Hkv][Ttot][D]  uint16 bits or float32
    V: np.ndarray              # same
    Q: np.ndarray              # [L][Hq][B][w][D]   uint16 bits or float32
    budget: List[int]          # per sequence: tokens kept per head, window included
    mode: str                  # "per_head" | "layer_flat"
    seed: int
    meta: dict

    @property
    def B(self) -> int:
        return len(self.cu_seqlens) - 1

    @property
    def seqlens(self) -> List[int]:
        c = self.cu_seqlens
        return [c[i + 1] - c[i] for i in range(self.B)]

    @property
    def Ttot(self) -> int:
        return self.cu_seqlens[-1]

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    def f32(self, a: np.ndarray) -> np.ndarray:
        return bf16_bits_to_f32(a) if self.dtype == "bf16" else np.asarray(a, np.float32)


def _encode(x: np.ndarray, dtype: str) -> np.ndarray:
    return to_bf16_bits(x) if dtype == "bf16" else x.astype(np.float32)


def _rng(seed: int, tag: int, *ix: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, tag, *ix]))


def _unit_dir(rng: np.random.Generator, D: int) -> np.ndarray:
    u = rng.standard_normal(D)
    return (u / np.linalg.norm(u)).astype(np.float32)


_TAG_K, _TAG_Q, _TAG_V, _TAG_LAYER = 1, 2, 3, 4


def _mllm_unit_keys(rng, T, D, n_visual, group, sigmas, offset):
    """Visual prefix of near-duplicate groups + i.i.d. text tokens, plus a shared offset.

    Visual token t in group g: centre_g + sigma_g * n_t + offset, centre_g ~ N(0, I).
    Text token: n_t + offset.  ``sigmas`` has one entry per group.
    """
    K = rng.standard_normal((T, D), dtype=np.float32)
    ng = len(sigmas)
    centres = rng.standard_normal((ng, D), dtype=np.float32)
    for g in range(ng):
        a, b = g * group, min((g + 1) * group, n_visual)
        K[a:b] *= np.float32(sigmas[g])
        K[a:b] += centres[g]
    K += offset[None, :]
    return K


def _gqa_generate(name, seed, L, Hq, Hkv, D, w, seqlens, dtype, budget, mode,
                  visual_frac, group, sigma_fn, strength_fn, meta, query_offset=True):
    """Generic generator for the MLLM-shaped configurations."""
    B = len(seqlens)
    cu = [0]
    for t in seqlens:
        cu.append(cu[-1] + t)
    Ttot = cu[-1]
    edt = np.uint16 if dtype == "bf16" else np.float32
    K = np.empty((L, Hkv, Ttot, D), dtype=edt)
    V = np.empty((L, Hkv, Ttot, D), dtype=edt)
    Q = np.empty((L, Hq, B, w, D), dtype=edt)
    G = Hq // Hkv
    strengths = [float(strength_fn(_rng(seed, _TAG_LAYER, l))) for l in range(L)]

    def one_unit(lhs):
        l, h, s = lhs
        T = seqlens[s]
        rk = _rng(seed, _TAG_K, l, h, s)
        u = _unit_dir(rk, D)
        off = np.float32(strengths[l] * math.sqrt(D)) * u
        nv = (int(visual_frac * T) // group) * group if visual_frac < 1 else T
        ngroups = (nv + group - 1) // group
        sig = sigma_fn(rk, ngroups)
        K[l, h, cu[s]:cu[s + 1]] = _encode(_mllm_unit_keys(rk, T, D, nv, group, sig, off), dtype)
        rv = _rng(seed, _TAG_V, l, h, s)
        V[l, h, cu[s]:cu[s + 1]] = _encode(rv.standard_normal((T, D), dtype=np.float32), dtype)
        rq = _rng(seed, _TAG_Q, l, h, s)
        Qg = rq.standard_normal((G, w, D), dtype=np.float32)
        if query_offset:
            Qg += off[None, None, :]
        Q[l, h * G:(h + 1) * G, s] = _encode(Qg, dtype)

    units = [(l, h, s) for l in range(L) for h in range(Hkv) for s in range(B)]
    # Units draw from independent streams, so the thread schedule cannot change the bytes.
    with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
        list(ex.map(one_unit, units))
    meta = dict(meta)
    meta["strength_per_layer"] = strengths
    return Workload(name, L, Hq, Hkv, D, w, cu, dtype, K, V, Q, list(budget), mode, seed, meta)


def tiny(seed: int = 0) -> Workload:
    """1 layer, 2 KV heads (MHA), D=128, T=512, fp32, w=8, budget 128 per head.

    Per head: a unit direction u; base key = s * (4 u + n), n ~ N(0, I),
    s ~ LogNormal(0, 0.3).  Positions [0, 128) hold 4 clusters x 32 near
    duplicates: member = centre + 0.05 N(0, I), centre drawn as a base key.
    Window queries are base keys of the same head (independent draws); V ~ N(0, 1).
    """
    L, H, D, T, w, b = 1, 2, 128, 512, 8, 128
    K = np.empty((L, H, T, D), np.float32)
    V = np.empty((L, H, T, D), np.float32)
    Q = np.empty((L, H, 1, w, D), np.float32)
    for h in range(H):
        rk = _rng(seed, _TAG_K, 0, h, 0)
        u = _unit_dir(rk, D)

        def base(n):
            s = rk.lognormal(0.0, 0.3, size=(n, 1)).astype(np.float32)
            return s * (np.float32(4.0) * u[None, :] + rk.standard_normal((n, D), dtype=np.float32))

        Kh = base(T)
        centres = base(4)
        for r in range(4):
            Kh[r * 32:(r + 1) * 32] = centres[r][None, :] + np.float32(0.05) * rk.standard_normal((32, D), dtype=np.float32)
        K[0, h] = Kh
        Q[0, h, 0] = base(w)
        V[0, h] = _rng(seed, _TAG_V, 0, h, 0).standard_normal((T, D), dtype=np.float32)
    meta = {"recipe": "shared direction norm 4 + N(0,1), lognormal(0,0.3) scale, 4x32 duplicates sigma 0.05"}
    return Workload("tiny", L, H, H, D, w, [0, T], "f32", K, V, Q, [b], "per_head", seed, meta)


def layer7b(seed: int = 1, T: int = 8192) -> Workload:
    """One 7B-shaped layer: 28 query / 4 KV heads, D=128, bf16, T=8192, w=8, budget 20 %.

    Visual [0, 0.75 T) in 256-token groups, member = centre + 0.1 N(0, I) + o;
    text = N(0, I) + o;  o = 1.5 sqrt(D) u (anisotropic shared offset).
    """
    b = int(0.2 * T)
    return _gqa_generate("layer7b", seed, 1, 28, 4, 128, 8, [T], "bf16", [b], "per_head",
                         0.75, 256, lambda r, n: np.full(n, 0.1), lambda r: 1.5,
                         {"visual_frac": 0.75, "group": 256, "sigma": 0.1, "strength": 1.5})


def stack28(seed: int = 2, T: int = 32768, budget_frac: float = 0.2, L: int = 28) -> Workload:
    """28 layers of the 7B GQA shape at T=32768, bf16, w=4, budget 10/20/40 % per head.

    Per-layer offset strength a_l ~ U[0.5, 3] (offset norm a_l sqrt(D)), 75 % visual
    tokens in 256-token groups with sigma 0.1, 25 % text.
    """
    b = int(budget_frac * T)
    return _gqa_generate("stack28", seed, L, 28, 4, 128, 4, [T], "bf16", [b], "per_head",
                         0.75, 256, lambda r, n: np.full(n, 0.1), lambda r: r.uniform(0.5, 3.0),
                         {"visual_frac": 0.75, "group": 256, "sigma": 0.1, "strength": "U[0.5,3]",
                          "budget_frac": budget_frac})


def mha64k(seed: int = 3, T: int = 65536, Hkv: int = 32, L: int = 1) -> Workload:
    """32-head MHA, D=128, bf16, T=65536, w=8, budget 2048 per head.

    56000 visual tokens in 256-token groups (218 full + one of 192) with a per-group
    sigma log-uniform in [0.02, 0.5]; 9536 text tokens; offset strength 1.5.
    """
    nvis = 56000 if T == 65536 else (int(0.8545 * T) // 256) * 256
    return _mha_exact(seed, L, Hkv, T, nvis)


def _mha_exact(seed, L, H, T, nvis):
    D, w = 128, 8
    K = np.empty((L, H, T, D), np.uint16)
    V = np.empty((L, H, T, D), np.uint16)
    Q = np.empty((L, H, 1, w, D), np.uint16)
    for l in range(L):
        for h in range(H):
            rk = _rng(seed, _TAG_K, l, h, 0)
            u = _unit_dir(rk, D)
            off = np.float32(1.5 * math.sqrt(D)) * u
            ng = (nvis + 255) // 256
            sig = np.exp(rk.uniform(math.log(0.02), math.log(0.5), size=ng))
            K[l, h] = to_bf16_bits(_mllm_unit_keys(rk, T, D, nvis, 256, sig, off))
            V[l, h] = to_bf16_bits(_rng(seed, _TAG_V, l, h, 0).standard_normal((T, D), dtype=np.float32))
            rq = _rng(seed, _TAG_Q, l, h, 0)
            Q[l, h, 0] = to_bf16_bits(rq.standard_normal((w, D), dtype=np.float32) + off[None, :])
    meta = {"visual_tokens": nvis, "group": 256, "sigma": "loguniform[0.02,0.5]", "strength": 1.5}
    return Workload("mha64k", L, H, H, D, w, [0, T], "bf16", K, V, Q, [2048], "per_head", seed, meta)


def varlen(seed: int = 4, nseq: int = 8, tmin: int = 4096, tmax: int = 32768,
           budget_frac: float = 0.15) -> Workload:
    """Head-adaptive budget batch: 8 sequences, T_s ~ U_int[4096, 32768], 28q/4kv,
    D=128, bf16, 75 % visual as in the 7B layer, w=4, layer-flat selection with
    a layer budget of H_kv * floor(0.15 T_s) per sequence.
    """
    r = _rng(seed, 0)
    seqlens = [int(t) for t in r.integers(tmin, tmax + 1, size=nseq)]
    budget = [int(budget_frac * t) for t in seqlens]
    return _gqa_generate("varlen", seed, 1, 28, 4, 128, 4, seqlens, "bf16", budget, "layer_flat",
                         0.75, 256, lambda rr, n: np.full(n, 0.1), lambda rr: 1.5,
                         {"visual_frac": 0.75, "group": 256, "sigma": 0.1, "strength": 1.5,
                          "budget_frac": budget_frac})


def custom(seed: int, L: int, Hq: int, Hkv: int, D: int, w: int, seqlens: List[int],
           dtype: str = "bf16", budget: Optional[List[int]] = None, mode: str = "per_head",
           visual_frac: float = 0.75, group: int = 256, sigma: float = 0.1,
           strength: float = 1.5, query_offset: bool = True) -> Workload:
    """Any shape with the MLLM recipe (used for ragged / edge-case parity tests).
    With query_offset False the window queries are plain N(0, I) draws instead
    of sharing the keys' offset: with a strong offset the keys then share a
    common direction while the window logits stay of ordinary size."""
    if budget is None:
        budget = [max(w, int(0.2 * t)) for t in seqlens]
    return _gqa_generate("custom", seed, L, Hq, Hkv, D, w, list(seqlens), dtype, budget, mode,
                         visual_frac, group, lambda r, n: np.full(n, sigma), lambda r: strength,
                         {"visual_frac": visual_frac, "group": group, "sigma": sigma,
                          "strength": strength, "query_offset": query_offset}, query_offset=query_offset)


CONFIG_BUILDERS = {
    "tiny": tiny,
    "layer7b": layer7b,
    "stack28": stack28,
    "mha64k": mha64k,
    "varlen": varlen,
}
