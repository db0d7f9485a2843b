"""LayerwiseEviction (one call per layer, alternating over two streams with a
workspace each) gives bit for bit the outputs of the same single-layer calls
issued one after another on one stream: the kernels are deterministic, and
the two streams must neither race on a workspace nor reorder a layer before
its inputs.  Four layers of the benchmark stack's shape.
"""
import sys

import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_06663_amd  # noqa: F401  (fails loudly if the library is not built)


def test_two_streams_match_one_stream():
    import paper_2609_06663_amd as P
    from paper_2609_06663_amd.pipeline import EvictionPass, LayerwiseEviction
    wl = W.stack28(L=4)
    print("[gpu-layerwise] 4 layers of 28q/4kv x 32768 tokens, two streams vs one", file=sys.stderr, flush=True)
    to = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    K, V, Q = to(wl.K), to(wl.V), to(wl.Q)
    shape1 = P.Shape(1, wl.Hq, wl.Hkv, wl.D, wl.w, wl.cu_seqlens)
    ref = [EvictionPass(shape1, wl.budget) for _ in range(wl.L)]
    for l in range(wl.L):
        ref[l].run(K[l:l + 1], V[l:l + 1], Q[l:l + 1])
    lw = LayerwiseEviction(shape1, wl.budget, wl.L)
    for rep in range(2):  # the second round reuses the workspaces and outputs
        if rep == 0:
            for l in range(wl.L):
                lw.run_layer(l, K[l:l + 1], V[l:l + 1], Q[l:l + 1])
        else:
            lw.run_layers(range(wl.L), [K[l:l + 1] for l in range(wl.L)], [V[l:l + 1] for l in range(wl.L)],
                          [Q[l:l + 1] for l in range(wl.L)])
        lw.wait()
        torch.cuda.synchronize()
        for l in range(wl.L):
            a, b = ref[l], lw.passes[l]
            for name in ("scores", "lambda_", "stats", "idx", "counts", "offsets"):
                assert torch.equal(getattr(a, name), getattr(b, name)), (rep, l, name)
            assert torch.equal(a.Kc.view(torch.int16), b.Kc.view(torch.int16)), (rep, l, "Kc")
            assert torch.equal(a.Vc.view(torch.int16), b.Vc.view(torch.int16)), (rep, l, "Vc")


def test_groups_of_layers_on_two_streams_match_one_stream():
    # a call per group of 2 consecutive layers (views of the layer-major cache)
    import paper_2609_06663_amd as P
    from paper_2609_06663_amd.pipeline import EvictionPass, LayerwiseEviction
    wl = W.stack28(L=4)
    print("[gpu-layerwise] 4 layers in groups of 2, two streams vs one", file=sys.stderr, flush=True)
    to = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    K, V, Q = to(wl.K), to(wl.V), to(wl.Q)
    k = 2
    shape2 = P.Shape(k, wl.Hq, wl.Hkv, wl.D, wl.w, wl.cu_seqlens)
    calls = wl.L // k
    ref = [EvictionPass(shape2, wl.budget) for _ in range(calls)]
    for c in range(calls):
        ref[c].run(K[c * k:(c + 1) * k], V[c * k:(c + 1) * k], Q[c * k:(c + 1) * k])
    lw = LayerwiseEviction(shape2, wl.budget, wl.L)
    with pytest.raises(ValueError):
        lw.run_layer(0, K[:1], V[:1], Q[:1])
    for c in range(calls):
        lw.run_group(c, K[c * k:(c + 1) * k], V[c * k:(c + 1) * k], Q[c * k:(c + 1) * k])
    lw.wait()
    torch.cuda.synchronize()
    lw.check()
    for c in range(calls):
        a, b = ref[c], lw.passes[c]
        for name in ("scores", "lambda_", "stats", "idx", "counts", "offsets"):
            assert torch.equal(getattr(a, name), getattr(b, name)), (c, name)
        assert torch.equal(a.Kc.view(torch.int16), b.Kc.view(torch.int16)), (c, "Kc")
        assert torch.equal(a.Vc.view(torch.int16), b.Vc.view(torch.int16)), (c, "Vc")
    with pytest.raises(ValueError):
        LayerwiseEviction(P.Shape(3, wl.Hq, wl.Hkv, wl.D, wl.w, wl.cu_seqlens), wl.budget, wl.L)
