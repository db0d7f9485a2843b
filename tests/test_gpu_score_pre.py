"""GPU parity of ecokv_score_pre: the pass with the first sweep's sums
supplied by the caller (key sums and window softmax statistics, as a prefill
can produce them), so that K is read once.  The sums are computed here from
their definitions in float64 (numpy) and handed over as float32; the scores
are compared with the oracle's to the tolerances of parity_utils.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity_utils import gpu_pass
from test_gpu_parity import check_compact, check_per_head

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_06663_amd  # noqa: F401  (fails loudly if the library is not built)
    oracle.build(force=False)


def say(msg):
    print(f"[gpu-score-pre] {msg}", file=sys.stderr, flush=True)


def prefill_sums(wl, causal=True, lse=False):
    """[L][Hkv][B][2D + 2R]: sum k, sum k/|k|, per window row max logit and sum exp(logit - max)
    (with lse, each row's log-sum-exp and 1, the pair a flash-attention epilogue has)."""
    G, w, D = wl.G, wl.w, wl.D
    R = G * w
    out = np.zeros((wl.L, wl.Hkv, wl.B, 2 * D + 2 * R), np.float64)
    cu = wl.cu_seqlens
    for l in range(wl.L):
        for h in range(wl.Hkv):
            for s in range(wl.B):
                K = wl.f32(wl.K[l, h, cu[s]:cu[s + 1]]).astype(np.float64)
                Q = wl.f32(wl.Q[l, h * G:(h + 1) * G, s]).astype(np.float64).reshape(R, D)
                T = K.shape[0]
                n = np.maximum(np.sqrt((K * K).sum(axis=1)), 1e-12)
                out[l, h, s, :D] = K.sum(axis=0)
                out[l, h, s, D:2 * D] = (K / n[:, None]).sum(axis=0)
                x = Q @ K.T / np.sqrt(D)
                for r in range(R):
                    j = r % w
                    last = T - w + j if causal else T - 1
                    xr = x[r, :last + 1]
                    m = xr.max()
                    z = np.exp(xr - m).sum()
                    out[l, h, s, 2 * D + r] = m + np.log(z) if lse else m
                    out[l, h, s, 2 * D + R + r] = 1.0 if lse else z
    return out


@pytest.mark.parametrize("dtype,D,Hq,Hkv,w", [("bf16", 128, 28, 4, 4), ("bf16", 128, 8, 2, 8), ("f32", 64, 4, 2, 8),
                                              ("bf16", 64, 8, 2, 4)])
def test_score_pre_matches_oracle(dtype, D, Hq, Hkv, w):
    wl = W.custom(91, L=2, Hq=Hq, Hkv=Hkv, D=D, w=w, seqlens=[1500, 333, 70], dtype=dtype, budget=[300, 60, 9],
                  group=64)
    say(f"{dtype} D={D} Hq={Hq} Hkv={Hkv} w={w}: first-sweep sums supplied")
    g = gpu_pass(wl, pre=prefill_sums(wl))
    check_per_head(wl, g)
    check_compact(wl, g)


def test_score_pre_log_sum_exp_pairs():
    # each window row handed over as (log-sum-exp, 1): the form a prefill's
    # flash attention produces, above the row's largest logit by up to log T
    wl = W.custom(93, L=2, Hq=28, Hkv=4, D=128, w=4, seqlens=[3000, 640], dtype="bf16", budget=[600, 128],
                  group=64)
    say("window rows handed over as (log-sum-exp, 1)")
    g = gpu_pass(wl, pre=prefill_sums(wl, lse=True))
    check_per_head(wl, g)
    check_compact(wl, g)


def test_score_pre_with_options():
    import paper_2609_06663_amd as P
    wl = W.custom(92, L=1, Hq=8, Hkv=2, D=128, w=4, seqlens=[2100, 257], dtype="bf16", budget=[400, 60], group=64)
    for p in (P.Params(causal=False), P.Params(centroid_scope=P.CENTROID_PREFIX, redundancy=P.RED_STD),
              P.Params(norm_mode=P.NORM_MAD, imp_mode=P.IMP_ATTN_VNORM)):
        say(f"supplied sums with causal {p.causal}, centroid {p.centroid_scope}, norm {p.norm_mode}")
        g = gpu_pass(wl, params=p, pre=prefill_sums(wl, causal=bool(p.causal)))
        check_per_head(wl, g, params=p)


def test_score_pre_stack28():
    wl = W.stack28(L=4)
    say("four layers of the benchmark stack (T = 32768) with supplied sums")
    g = gpu_pass(wl, pre=prefill_sums(wl))
    check_per_head(wl, g)
