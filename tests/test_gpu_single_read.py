"""GPU parity of the single-read score path (ECOKV_SCORE_PATH=single).

The single-read kernel keeps every key on chip between the two sweeps and
publishes per-slice partials (224-key slices) and per-unit constants between
blocks (bf16, head_dim 128, G*w <= 28).  The cases below run it against the CPU oracle with
the tolerances of parity_utils, plus: it is bit-reproducible, and it agrees
with the two-sweep path to the score tolerance.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity_utils import RTOL, gpu_pass
from test_gpu_parity import (check_all_selections_valid, check_compact, check_layer_flat, check_per_head)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_06663_amd  # noqa: F401  (fails loudly if the library is not built)
    oracle.build(force=False)


@pytest.fixture(autouse=True)
def _single_path(monkeypatch):
    monkeypatch.setenv("ECOKV_SCORE_PATH", "single")


def say(msg):
    print(f"[gpu-single] {msg}", file=sys.stderr, flush=True)


def test_stack28_full_size_sampled():
    wl = W.stack28()
    say("stack28: 28 layers, 28q/4kv, T=32768, w=4 (single-read path)")
    g = gpu_pass(wl)
    check_all_selections_valid(wl, g)
    check_compact(wl, g)
    check_per_head(wl, g, units=[(0, 0, 0), (7, 1, 0), (13, 2, 0), (27, 3, 0)])


def test_mha64k_full_size_sampled():
    wl = W.mha64k()
    say("mha64k: 32 MHA heads, T=65536, w=8 (single-read path, 293 slices per unit)")
    g = gpu_pass(wl)
    check_all_selections_valid(wl, g)
    check_per_head(wl, g, units=[(0, 0, 0), (0, 31, 0)])


def test_varlen_layer_flat():
    wl = W.varlen()
    say("varlen: 8 sequences, layer-flat budget (single-read path)")
    g = gpu_pass(wl)
    check_layer_flat(wl, g)
    check_compact(wl, g)


@pytest.mark.parametrize("seqlens", [[5003], [300, 2100, 257, 4096], [40, 224, 223, 225, 449]])
def test_ragged_lengths(seqlens):
    # slice boundaries: shorter than one slice, exactly one, one key short, one over, many
    wl = W.custom(21, L=2, Hq=8, Hkv=2, D=128, w=4, seqlens=seqlens, dtype="bf16", group=64)
    say(f"ragged sequences {seqlens} (single-read path)")
    g = gpu_pass(wl)
    check_per_head(wl, g)
    check_compact(wl, g)


def test_window_rows_28_and_1():
    for (Hq, w) in [(28, 1), (7, 4), (1, 1)]:
        wl = W.custom(22, L=1, Hq=Hq, Hkv=1, D=128, w=w, seqlens=[1500], dtype="bf16", group=32)
        say(f"G*w = {Hq * w} window rows (single-read path)")
        g = gpu_pass(wl)
        check_per_head(wl, g)


def test_identical_and_zero_keys():
    wl = W.custom(15, L=1, Hq=4, Hkv=2, D=128, w=4, seqlens=[600], dtype="bf16", budget=[100], group=32)
    wl.K[0, 0, :] = wl.K[0, 0, 17]
    wl.K[0, 1, 5:9] = 0
    wl.K[0, 1, 300] = 0
    say("identical keys in head 0, zero keys in head 1 (single-read path)")
    g = gpu_pass(wl)
    check_per_head(wl, g, units=[(0, 0, 0)], stat_skip=("dmin", "dmax", "D_E", "sdiv_min", "sdiv_max",
                                                       "sbar_mean", "scale"))
    check_per_head(wl, g, units=[(0, 1, 0)])


def test_rising_logits():
    wl = W.custom(18, L=1, Hq=8, Hkv=2, D=128, w=4, seqlens=[5003, 2100], dtype="bf16", budget=[700, 300],
                  group=64)
    cu = wl.cu_seqlens
    for s in range(wl.B):
        n = cu[s + 1] - cu[s]
        ramp = np.exp(np.linspace(0.0, np.log(8.0), n)).astype(np.float32)
        k = W.bf16_bits_to_f32(wl.K[0, :, cu[s]:cu[s + 1]]) * ramp[None, :, None]
        wl.K[0, :, cu[s]:cu[s + 1]] = W.to_bf16_bits(k)
    say("rising logits (single-read path)")
    g = gpu_pass(wl)
    check_per_head(wl, g)


@pytest.mark.parametrize("variant", ["noncausal", "lambda0", "mixkv", "pool7", "tau"])
def test_parameter_variants(variant):
    import paper_2609_06663_amd as P
    p = {
        "noncausal": P.Params(causal=False),
        "lambda0": P.Params(lambda_override=0.0),
        "mixkv": P.Params(alpha=0.0, beta=0.0),
        "pool7": P.Params(pool_kernel=7),
        "tau": P.Params(tau=3.0),
    }[variant]
    wl = W.custom(16, L=1, Hq=8, Hkv=2, D=128, w=4, seqlens=[900, 333], dtype="bf16", budget=[150, 60],
                  group=64)
    say(f"parameter variant {variant} (single-read path)")
    g = gpu_pass(wl, params=p)
    check_per_head(wl, g, params=p)


def test_deterministic_and_matches_two_sweep(monkeypatch):
    wl = W.custom(23, L=3, Hq=28, Hkv=4, D=128, w=4, seqlens=[8192, 3000], dtype="bf16", group=256)
    say("single-read path: two runs bit-identical; two-sweep path within the score tolerance")
    g1 = gpu_pass(wl)
    g2 = gpu_pass(wl)
    for k in ("scores", "lambda_", "stats", "idx", "counts", "offsets"):
        np.testing.assert_array_equal(g1[k], g2[k], err_msg=k)
    monkeypatch.setenv("ECOKV_SCORE_PATH", "two-sweep")
    g3 = gpu_pass(wl)
    a, b = g1["scores"].astype(np.float64), g3["scores"].astype(np.float64)
    floor = np.maximum(np.abs(b).mean(axis=-1, keepdims=True), 1e-30)
    assert np.all(np.abs(a - b) <= RTOL * np.maximum(np.abs(b), floor))
