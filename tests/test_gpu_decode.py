"""GPU parity of ecokv_decode (attention of one new query per head over the
compressed cache, Sec. 3) against the oracle on seeded synthetic caches:
packed Kc / Vc rows with ragged per-unit counts, as ecokv_select and
ecokv_compact lay them out.

Tolerance (fp32 accumulation of bf16 / fp32 inputs against fp64):
|O_g - O_o| <= 1e-4 * max |Vc| over the unit's rows, |lse_g - lse_o| <= 1e-4 * max(1, |lse_o|).
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from parity_utils import dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_06663_amd  # noqa: F401  (fails loudly if the library is not built)
    oracle.build(force=False)


def say(msg):
    print(f"[gpu-decode] {msg}", file=sys.stderr, flush=True)


def make_cache(seed, L, Hq, Hkv, B, D, counts, dtype, kscale=1.0):
    r = np.random.default_rng(seed)
    counts = np.asarray(counts, np.int32).reshape(L, Hkv, B)
    offsets = np.concatenate([[0], np.cumsum(counts.reshape(-1))[:-1]]).reshape(L, Hkv, B).astype(np.int32)
    n = int(counts.sum())

    def arr(shape, scale):
        x = (r.standard_normal(shape) * scale).astype(np.float32)
        if dtype == "bf16":
            return (x.view(np.uint32) >> 16).astype(np.uint16)  # truncation: any bf16 values will do
        return x

    return dict(Q=arr((L, Hq, B, D), 1.0), Kc=arr((n, D), kscale), Vc=arr((n, D), 1.0), counts=counts,
                offsets=offsets)


def run(c, L, Hq, Hkv, B, D, dtype, max_count=None):
    import paper_2609_06663_amd as P
    shape = P.Shape(L, Hq, Hkv, D, 1, [0] + list(np.cumsum([2] * B)))
    mc = int(c["counts"].max()) if max_count is None else max_count
    O = torch.full((L, Hq, B, D), -7.0, device="cuda")
    lse = torch.full((L, Hq, B), -7.0, device="cuda")
    P.ecokv_decode(dev(c["Q"], dtype), dev(c["Kc"], dtype), dev(c["Vc"], dtype), shape,
                   torch.from_numpy(c["counts"].reshape(-1)).cuda(), torch.from_numpy(c["offsets"].reshape(-1)).cuda(),
                   mc, O, lse)
    torch.cuda.synchronize()
    return O.cpu().numpy(), lse.cpu().numpy()


def check(c, O, lse, L, Hq, Hkv, B, D, dtype):
    Oo, lo = oracle.decode(c["Q"], c["Kc"], c["Vc"], L, Hq, Hkv, B, D, c["counts"], c["offsets"])
    G = Hq // Hkv
    V = c["Vc"].astype(np.float32) if dtype == "f32" else (c["Vc"].astype(np.uint32) << 16).view(np.float32)
    for l in range(L):
        for q in range(Hq):
            for s in range(B):
                o, n = c["offsets"][l, q // G, s], c["counts"][l, q // G, s]
                vmax = float(np.abs(V[o:o + n]).max())
                err = np.abs(O[l, q, s] - Oo[l, q, s]).max()
                assert err <= 1e-4 * vmax, f"O (l={l}, q={q}, s={s}, n={n}): error {err:.3e}, max|V| {vmax:.3e}"
                assert abs(lse[l, q, s] - lo[l, q, s]) <= 1e-4 * max(1.0, abs(lo[l, q, s])), (l, q, s)


@pytest.mark.parametrize("dtype,D,Hq,Hkv", [("bf16", 128, 28, 4), ("bf16", 64, 8, 8), ("f32", 128, 8, 4),
                                            ("f32", 64, 12, 4), ("bf16", 128, 32, 2), ("bf16", 128, 24, 2)])
def test_decode_ragged(dtype, D, Hq, Hkv):
    # G = 7, 1, 2, 3, 16 (two blocks of 8 query heads), 12 (8 + 4)
    L, B = 2, 3
    r = np.random.default_rng(100 + Hq)
    counts = r.integers(1, 2600, size=(L, Hkv, B))
    counts.reshape(-1)[0] = 1                     # one row
    counts.reshape(-1)[-1] = 1024                 # exactly one chunk
    if counts.size > 2:
        counts.reshape(-1)[1] = 257               # one row past a wave's share
    c = make_cache(7, L, Hq, Hkv, B, D, counts, dtype, kscale=2.0)
    say(f"{dtype} D={D} Hq={Hq} Hkv={Hkv}: ragged counts up to {int(counts.max())}")
    O, lse = run(c, L, Hq, Hkv, B, D, dtype)
    check(c, O, lse, L, Hq, Hkv, B, D, dtype)


def test_decode_large_logits_and_a_loose_max_count():
    # keys scaled up: logits span hundreds, the online maxima move often; a
    # max_count far above every count only adds empty chunks
    L, Hq, Hkv, B, D = 1, 8, 2, 2, 128
    counts = [[[3000, 77], [1, 2049]]]
    c = make_cache(8, L, Hq, Hkv, B, D, counts, "bf16", kscale=30.0)
    say("large logits, max_count 9000")
    O, lse = run(c, L, Hq, Hkv, B, D, "bf16", max_count=9000)
    check(c, O, lse, L, Hq, Hkv, B, D, "bf16")


def test_decode_count_above_max_count_is_nan():
    L, Hq, Hkv, B, D = 1, 4, 2, 1, 64
    c = make_cache(9, L, Hq, Hkv, B, D, [[[100], [300]]], "f32")
    say("a unit with more rows than max_count")
    O, lse = run(c, L, Hq, Hkv, B, D, "f32", max_count=200)
    assert np.isnan(O[0, 2:]).all() and np.isnan(lse[0, 2:]).all()   # KV head 1's query heads
    Oo, lo = oracle.decode(c["Q"], c["Kc"], c["Vc"], L, Hq, Hkv, B, D, c["counts"], c["offsets"])
    np.testing.assert_allclose(O[0, :2], Oo[0, :2], atol=1e-4 * np.abs(c["Vc"][:100]).max())


def test_decode_stack28_sized_cache():
    # the compressed cache of the 28-layer benchmark stack at 20 %: 6553 rows per head
    L, Hq, Hkv, B, D = 28, 28, 4, 1, 128
    counts = np.full((L, Hkv, B), 6553)
    c = make_cache(10, L, Hq, Hkv, B, D, counts, "bf16")
    say("28 layers x 4 KV heads x 6553 rows, 28 query heads")
    O, lse = run(c, L, Hq, Hkv, B, D, "bf16")
    check(c, O, lse, L, Hq, Hkv, B, D, "bf16")


def test_decode_many_units_ragged():
    # 224 units of up to 6000 rows (more blocks than the device holds at once);
    # the counts are ragged, so chunks and 16-row tiles end inside and past units
    L, Hq, Hkv, B, D = 28, 28, 4, 2, 128
    r = np.random.default_rng(11)
    counts = r.integers(1, 6000, size=(L, Hkv, B))
    counts.reshape(-1)[3] = 6000
    counts.reshape(-1)[4] = 1
    counts.reshape(-1)[7] = 16
    counts.reshape(-1)[8] = 17
    c = make_cache(12, L, Hq, Hkv, B, D, counts, "bf16")
    say(f"224 units, ragged counts up to 6000, {int(counts.sum())} rows")
    O, lse = run(c, L, Hq, Hkv, B, D, "bf16", max_count=6000)
    check(c, O, lse, L, Hq, Hkv, B, D, "bf16")
