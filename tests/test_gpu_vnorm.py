"""GPU parity of the value-norm importance (imp_mode IMP_ATTN_VNORM, Sec. 5.2:
S_imp(i) = pool(a)(i) * |v_i|_2) through ecokv_score_v, against the oracle
given the same V bytes, to the tolerances of parity_utils.  Covers every
(element type, head_dim) instantiation of the value pass, a wider pool, the
two epilogue forms (one launch per unit and the split one for sequences over
32768 + w tokens), a one-row window and the full-size stack.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity_utils import gpu_pass
from test_gpu_parity import check_all_selections_valid, check_compact, check_per_head

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_06663_amd  # noqa: F401  (fails loudly if the library is not built)
    oracle.build(force=False)


def say(msg):
    print(f"[gpu-vnorm] {msg}", file=sys.stderr, flush=True)


def vparams(**kw):
    import paper_2609_06663_amd as P
    return P.Params(imp_mode=P.IMP_ATTN_VNORM, **kw)


@pytest.mark.parametrize("dtype,D", [("bf16", 128), ("bf16", 64), ("f32", 128), ("f32", 64)])
def test_value_norm_small(dtype, D):
    wl = W.custom(61, L=2, Hq=8, Hkv=2, D=D, w=4, seqlens=[1500, 333, 70], dtype=dtype, budget=[300, 60, 9],
                  group=64)
    say(f"value-norm importance, {dtype} head_dim {D}, ragged sequences")
    p = vparams()
    g = gpu_pass(wl, params=p)
    check_per_head(wl, g, params=p)
    check_compact(wl, g)


def test_value_norm_wide_pool_and_noncausal():
    wl = W.custom(62, L=1, Hq=28, Hkv=4, D=128, w=4, seqlens=[3000], dtype="bf16", budget=[500], group=128)
    for p in (vparams(pool_kernel=7), vparams(causal=False, pool_kernel=1)):
        say(f"value-norm importance, pool {p.pool_kernel}, causal {p.causal}")
        g = gpu_pass(wl, params=p)
        check_per_head(wl, g, params=p)


def test_value_norm_long_sequence_split_epilogue():
    # 40000 tokens: beyond the one-launch epilogue, so the split epilogue reads the importance
    wl = W.custom(63, L=1, Hq=4, Hkv=1, D=128, w=4, seqlens=[40000], dtype="bf16", budget=[4000], group=256)
    say("value-norm importance, one 40000-token sequence (split epilogue)")
    p = vparams()
    g = gpu_pass(wl, params=p)
    check_per_head(wl, g, params=p)


def test_value_norm_one_row_window():
    wl = W.custom(64, L=2, Hq=28, Hkv=4, D=128, w=1, seqlens=[5003, 1200], dtype="bf16", budget=[700, 100],
                  group=128)
    say("value-norm importance with a one-row window")
    p = vparams()
    g = gpu_pass(wl, params=p)
    check_per_head(wl, g, params=p)


def test_value_norm_stack28_full_size():
    wl = W.stack28()
    say("stack28 with the value-norm importance (every unit against the oracle)")
    p = vparams()
    g = gpu_pass(wl, params=p)
    check_all_selections_valid(wl, g)
    check_compact(wl, g)
    check_per_head(wl, g, params=p)
