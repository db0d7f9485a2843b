"""ecokv_score_noalloc (the score call with the library's own scratch, for
callers that cannot allocate) against ecokv_score_pre with a caller
workspace: two calls in a row, the second with a smaller input, through the
C ABI; and the refusal of a call whose scratch would not fit."""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from parity_utils import check_scores, check_stats, dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_06663_amd  # noqa: F401  (fails loudly if the library is not built)


def say(msg):
    print(f"[gpu-noalloc] {msg}", file=sys.stderr, flush=True)


def _both(wl, params):
    import paper_2609_06663_amd as P
    shape = P.Shape(wl.L, wl.Hq, wl.Hkv, wl.D, wl.w, wl.cu_seqlens)
    K, V, Q = dev(wl.K, wl.dtype), dev(wl.V, wl.dtype), dev(wl.Q, wl.dtype)
    U, Ptot = shape.units, shape.ptot
    out = {}
    for name in ("workspace", "noalloc"):
        S = torch.full((wl.L * wl.Hkv * Ptot,), float("nan"), device="cuda")
        lam = torch.full((U,), float("nan"), device="cuda")
        st = torch.full((U * P.NSTATS,), float("nan"), device="cuda")
        if name == "workspace":
            P.ecokv_score_pre(K, V, Q, shape, params, None, S, lam, st)
        else:
            P.ecokv_score_noalloc(K, V, Q, shape, params, None, S, lam, st)
        torch.cuda.synchronize()
        out[name] = (S.cpu().numpy().reshape(wl.L, wl.Hkv, -1), lam.cpu().numpy(),
                     st.cpu().numpy().reshape(U, P.NSTATS))
    return out


def _compare(wl, out):
    Sw, lw, sw = out["workspace"]
    Sn, ln, sn = out["noalloc"]
    assert np.isfinite(Sn).all() and np.isfinite(ln).all()
    for l in range(wl.L):
        for h in range(wl.Hkv):
            for s in range(wl.B):
                u = (l * wl.Hkv + h) * wl.B + s
                T = wl.cu_seqlens[s + 1] - wl.cu_seqlens[s]
                off = wl.cu_seqlens[s] - s * wl.w
                ref = Sw[l, h, off:off + T - wl.w].astype(np.float64)
                check_scores(Sn[l, h, off:off + T - wl.w], ref, sw[u, 8], f"noalloc unit {u}")
                check_stats(sn[u], sw[u].astype(np.float64), f"noalloc unit {u}")
    np.testing.assert_allclose(ln, lw, rtol=2e-3)


def test_noalloc_matches_workspace_call_twice_second_smaller():
    import paper_2609_06663_amd as P
    big = W.stack28(L=4)
    say("noalloc call 1: 4 layers x 4 KV heads x 32768 tokens")
    _compare(big, _both(big, P.Params()))
    small = W.custom(52, L=1, Hq=8, Hkv=2, D=128, w=4, seqlens=[5003, 700], dtype="bf16")
    say("noalloc call 2 (smaller): 1 layer, sequences [5003, 700]")
    _compare(small, _both(small, P.Params()))


def test_noalloc_refuses_a_call_past_its_scratch():
    import paper_2609_06663_amd as P
    L = 64
    shape = P.Shape(L, 28, 4, 128, 4, [0, 32768])   # ~140 MiB of scratch
    assert P.ecokv_workspace_size(shape) > 96 << 20
    K = torch.zeros(L * 4 * 32768 * 128, dtype=torch.bfloat16, device="cuda")
    Q = torch.zeros(L * 28 * 4 * 128, dtype=torch.bfloat16, device="cuda")
    S = torch.full((L * 4 * 32764,), -1.0, device="cuda")
    with pytest.raises(P.EcoKVError) as e:
        P.ecokv_score_noalloc(K, None, Q, shape, None, None, S)
    assert e.value.code == P.EWORKSPACE and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert bool((S == -1.0).all())  # refused before anything was enqueued
