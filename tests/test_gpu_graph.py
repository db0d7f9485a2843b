"""The pass captured in a HIP graph (torch.cuda.CUDAGraph) and replayed on
changing inputs: every replay must reproduce, bit for bit, the eager pass on
the same inputs, over shapes that take each selection form and the split
epilogue; the no-alloc entry point is captured too.
"""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from parity_utils import dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_06663_amd  # noqa: F401  (fails loudly if the library is not built)


def say(msg):
    print(f"[gpu-graph] {msg}", file=sys.stderr, flush=True)


OUTS = ("scores", "lambda_", "stats", "idx", "counts", "offsets")


# shape cases: the epilogue split over blocks that exchange sums with a
# one-block selection; layer-flat groups past 32 Ki keys (the five-launch
# multi-block selection, whose workspace must end zero-filled after every
# replay); a long single head with a small budget (the two-stage selection)
CASES = {
    "per_head": dict(L=1, Hq=8, Hkv=2, seqlens=[9000, 3000], budget=[900, 300], mode="per_head"),
    "flat_multiblock": dict(L=1, Hq=8, Hkv=4, seqlens=[12000, 9500], budget=[1800, 1400], mode="layer_flat"),
    "two_stage": dict(L=1, Hq=4, Hkv=1, seqlens=[40000], budget=[1024], mode="per_head"),
}


def _inputs(seed, case):
    c = CASES[case]
    wl = W.custom(seed, L=c["L"], Hq=c["Hq"], Hkv=c["Hkv"], D=128, w=4, seqlens=c["seqlens"], dtype="bf16",
                  budget=c["budget"], mode=c["mode"])
    return wl, (dev(wl.K, "bf16"), dev(wl.V, "bf16"), dev(wl.Q, "bf16"))


def _snapshot(ep):
    out = {n: getattr(ep, n).clone() for n in OUTS}
    out["Kc"] = ep.Kc.view(torch.int16).clone()
    out["Vc"] = ep.Vc.view(torch.int16).clone()
    return out


def _same(a, b, what):
    for n in a:
        assert torch.equal(a[n], b[n]), f"{what}: {n} differs"


@pytest.mark.parametrize("case,noalloc", [("per_head", False), ("per_head", True), ("flat_multiblock", False),
                                          ("two_stage", False)])
def test_graph_replays_match_eager(case, noalloc):
    import paper_2609_06663_amd as P
    from paper_2609_06663_amd.pipeline import EvictionPass
    wl1, in1 = _inputs(61, case)
    wl2, in2 = _inputs(62, case)
    shape = P.Shape(wl1.L, wl1.Hq, wl1.Hkv, wl1.D, wl1.w, wl1.cu_seqlens)
    mode = P.LAYER_FLAT if wl1.mode == "layer_flat" else P.PER_HEAD

    def run(ep, K, V, Q, stream=None):
        if noalloc:
            P.ecokv_score_noalloc(K, V, Q, ep.shape, ep.params, None, ep.scores, ep.lambda_, ep.stats, stream)
            ep.select(stream)
            ep.compact(K, V, stream)
        else:
            ep.run(K, V, Q, stream)

    say(f"{case}: eager passes on two inputs (noalloc={noalloc})")
    ep_e = EvictionPass(shape, wl1.budget, mode, P.Params(), torch.bfloat16)
    eager = []
    for K, V, Q in (in1, in2):
        run(ep_e, K, V, Q)
        torch.cuda.synchronize()
        eager.append(_snapshot(ep_e))

    ep_g = EvictionPass(shape, wl1.budget, mode, P.Params(), torch.bfloat16)
    Ks, Vs, Qs = (t.clone() for t in in1)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(2):
            run(ep_g, Ks, Vs, Qs)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    say("capture")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run(ep_g, Ks, Vs, Qs)
    torch.cuda.synchronize()
    for rep, which in enumerate([0, 1, 1, 0, 1, 0]):
        src = (in1, in2)[which]
        for dst, s in zip((Ks, Vs, Qs), src):
            dst.copy_(s)
        # eager work of the program's own between replays
        run(ep_e, *src)
        g.replay()
        torch.cuda.synchronize()
        say(f"replay {rep} on input {which + 1}")
        _same(_snapshot(ep_g), eager[which], f"replay {rep} (input {which + 1})")
        _same(_snapshot(ep_e), eager[which], f"eager pass beside replay {rep}")
    if not noalloc:
        ep_g.check()


def test_graph_replays_read_once_flow():
    # the prefill's cache write with the first sweep's sums, the pass on them,
    # then decode attention over the compressed cache: all captured in one graph
    import paper_2609_06663_amd as P
    from paper_2609_06663_amd.pipeline import EvictionPass
    wl1, in1 = _inputs(63, "per_head")
    wl2, in2 = _inputs(64, "per_head")
    shape = P.Shape(wl1.L, wl1.Hq, wl1.Hkv, wl1.D, wl1.w, wl1.cu_seqlens)
    L, Hq, Hkv, D, B, w = wl1.L, wl1.Hq, wl1.Hkv, wl1.D, wl1.B, wl1.w
    R = Hq // Hkv * w
    max_count = max(wl1.budget)
    gen = torch.Generator(device="cuda").manual_seed(65)
    inputs = []
    for K, V, Q in (in1, in2):
        Kn, Vn = K.transpose(1, 2).contiguous(), V.transpose(1, 2).contiguous()  # token-major new rows
        Qd = torch.randn((L, Hq, B, D), generator=gen, device="cuda").to(torch.bfloat16)
        inputs.append((Kn, Vn, Q, Qd))

    class Flow:
        def __init__(self):
            self.ep = EvictionPass(shape, wl1.budget, P.PER_HEAD, P.Params(), torch.bfloat16)
            self.Kcache = torch.empty_like(in1[0])
            self.Vcache = torch.empty_like(in1[1])
            self.pre = torch.empty(L * Hkv * B * (2 * D + 2 * R), dtype=torch.float32, device="cuda")
            self.ws_p = torch.zeros(P.ecokv_prefill_workspace_size(shape), dtype=torch.uint8, device="cuda")
            self.ws_d = torch.zeros(max(P.ecokv_decode_workspace_size(shape, max_count), 256), dtype=torch.uint8,
                                    device="cuda")
            self.O = torch.empty((L, Hq, B, D), dtype=torch.float32, device="cuda")
            self.lse = torch.empty((L, Hq, B), dtype=torch.float32, device="cuda")

        def __call__(self, Kn, Vn, Q, Qd):
            P.ecokv_prefill_write(Kn, Vn, Q, shape, P.Params(), self.Kcache, self.Vcache, self.pre, self.ws_p)
            self.ep.run(self.Kcache, self.Vcache, Q, pre=self.pre)
            P.ecokv_decode(Qd, self.ep.Kc, self.ep.Vc, shape, self.ep.counts, self.ep.offsets, max_count, self.O,
                           self.lse, self.ws_d)

        def snapshot(self):
            out = _snapshot(self.ep)
            out.update(pre=self.pre.clone(), Kcache=self.Kcache.view(torch.int16).clone(),
                       Vcache=self.Vcache.view(torch.int16).clone(), O=self.O.clone(), lse=self.lse.clone())
            return out

    say("read-once flow: eager on two inputs")
    fe = Flow()
    eager = []
    for x in inputs:
        fe(*x)
        torch.cuda.synchronize()
        eager.append(fe.snapshot())
    fg = Flow()
    static = [t.clone() for t in inputs[0]]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(2):
            fg(*static)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    say("read-once flow: capture")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fg(*static)
    torch.cuda.synchronize()
    for rep, which in enumerate([0, 1, 1, 0, 1]):
        for dst, s in zip(static, inputs[which]):
            dst.copy_(s)
        fe(*inputs[which])
        g.replay()
        torch.cuda.synchronize()
        say(f"read-once flow: replay {rep} on input {which + 1}")
        _same(fg.snapshot(), eager[which], f"replay {rep} (input {which + 1})")
        _same(fe.snapshot(), eager[which], f"eager flow beside replay {rep}")
    fg.ep.check()
