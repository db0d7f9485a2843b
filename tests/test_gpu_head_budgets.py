"""GPU parity of ECOKV_HEAD_BUDGETS: a budget per (layer, KV head), as the
PyramidKV layer schedule and the SparseMM head budgets assign them
(Appendix A.1).  Selection is compared bit-exactly with the oracle on
identical fp32 scores; the whole pass (score -> select -> compact) is compared
with the oracle's units to the tolerances of parity_utils; compaction is
bit-exact.  Cases cover budgets equal to the window, at or above T_s, ragged
sequences, and more (layer, head) pairs than one launch's table holds.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity_utils import check_scores, check_stats, check_unit_selection, gpu_pass, oracle_unit, topk_rule, \
    unit_slices

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_06663_amd  # noqa: F401  (fails loudly if the library is not built)
    oracle.build(force=False)


def say(msg):
    print(f"[gpu-head-budgets] {msg}", file=sys.stderr, flush=True)


def select_and_compact(S, L, Hkv, D, w, cu, bud, K=None, V=None):
    """ecokv_select (+ ecokv_compact when K, V are given) in HEAD_BUDGETS mode."""
    import paper_2609_06663_amd as P
    shape = P.Shape(L, Hkv, Hkv, D, w, cu)
    n = P.ecokv_index_count_mode(shape, P.HEAD_BUDGETS, bud)
    U = L * Hkv * (len(cu) - 1)
    idx = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    counts = torch.full((U,), -7, dtype=torch.int32, device="cuda")
    offsets = torch.full((U,), -7, dtype=torch.int32, device="cuda")
    P.ecokv_select(torch.from_numpy(np.ascontiguousarray(S, np.float32)).cuda(), shape, P.HEAD_BUDGETS, bud,
                   idx, counts, offsets)
    out = {}
    if K is not None:
        Kd = torch.from_numpy(K.view(np.int16)).cuda()
        Vd = torch.from_numpy(V.view(np.int16)).cuda()
        Kc = torch.empty((n, D), dtype=torch.int16, device="cuda")
        Vc = torch.empty((n, D), dtype=torch.int16, device="cuda")
        # counts and offsets are not needed by the gather in this mode
        P.ecokv_compact(Kd.view(torch.bfloat16), Vd.view(torch.bfloat16), shape, P.HEAD_BUDGETS, bud, idx,
                        None, None, Kc.view(torch.bfloat16), Vc.view(torch.bfloat16))
        out["Kc"] = Kc.cpu().numpy().view(np.uint16)
        out["Vc"] = Vc.cpu().numpy().view(np.uint16)
    torch.cuda.synchronize()
    out.update(idx=idx.cpu().numpy(), counts=counts.cpu().numpy().reshape(L, Hkv, -1),
               offsets=offsets.cpu().numpy().reshape(L, Hkv, -1))
    return out


def check_against_oracle(S, L, Hkv, w, cu, bud, g, K=None, V=None, D=None):
    ref_idx, ref_c, ref_o = oracle.select(S.astype(np.float64), L, Hkv, cu, w, bud, oracle.HEAD_BUDGETS)
    np.testing.assert_array_equal(g["idx"], ref_idx)
    np.testing.assert_array_equal(g["counts"], ref_c)
    np.testing.assert_array_equal(g["offsets"], ref_o)
    if K is not None:
        Kc, Vc = oracle.compact(K, V, L, Hkv, cu, D, ref_idx, ref_c, ref_o)
        np.testing.assert_array_equal(g["Kc"], Kc)
        np.testing.assert_array_equal(g["Vc"], Vc)


def test_select_bit_exact_with_ties_and_edges():
    rng = np.random.default_rng(41)
    seqlens = [3000, 70, 1025, 9]
    cu = np.concatenate([[0], np.cumsum(seqlens)]).tolist()
    L, Hkv, w = 3, 4, 3
    Ptot = cu[-1] - len(seqlens) * w
    S = rng.integers(0, 40, size=(L, Hkv, Ptot)).astype(np.float32) * np.float32(0.25) - np.float32(2.0)
    S[0, 0, :50] = np.nan
    S[1, 2, 10:20] = -0.0
    S[1, 2, 20:30] = 0.0
    bud = rng.integers(w, 3100, size=(L, Hkv)).astype(np.int32)
    bud[0, 1] = w          # the window only
    bud[2, 3] = 5000       # every token of every sequence
    bud[1, 1] = 1024       # T - 1 of the third sequence
    say(f"select-only bit-exact, budgets {bud.tolist()}")
    g = select_and_compact(S, L, Hkv, 128, w, cu, bud)
    check_against_oracle(S, L, Hkv, w, cu, bud, g)


def test_long_sequences_two_stage_and_multi_block():
    # sequences past 32768 keys: small per-head budgets take the two-stage
    # selection (every head's candidates fit one block), one large budget in
    # the second call sends the whole call to the multi-block form
    rng = np.random.default_rng(43)
    seqlens = [50004, 2000]
    cu = np.concatenate([[0], np.cumsum(seqlens)]).tolist()
    L, Hkv, w = 2, 3, 4
    Ptot = cu[-1] - len(seqlens) * w
    S = rng.integers(0, 300, size=(L, Hkv, Ptot)).astype(np.float32) * np.float32(0.125)
    S[0, 1, 9000:9100] = np.nan
    bud = rng.integers(w, 3000, size=(L, Hkv)).astype(np.int32)
    bud[1, 2] = w          # the window only
    bud[0, 2] = 60000      # every token
    say(f"two-stage: budgets {bud.tolist()}")
    check_against_oracle(S, L, Hkv, w, cu, bud, select_and_compact(S, L, Hkv, 128, w, cu, bud))
    bud[1, 0] = 30000
    say(f"multi-block: budgets {bud.tolist()}")
    check_against_oracle(S, L, Hkv, w, cu, bud, select_and_compact(S, L, Hkv, 128, w, cu, bud))


def test_more_pairs_than_one_table():
    # 40 layers x 8 KV heads = 320 (layer, head) pairs: two launches of the table
    rng = np.random.default_rng(42)
    seqlens = [300, 131]
    cu = np.concatenate([[0], np.cumsum(seqlens)]).tolist()
    L, Hkv, w, D = 40, 8, 2, 128
    Ptot = cu[-1] - len(seqlens) * w
    S = rng.standard_normal((L, Hkv, Ptot)).astype(np.float32)
    bud = rng.integers(w, 320, size=(L, Hkv)).astype(np.int32)
    K = rng.integers(0, 1 << 16, size=(L, Hkv, cu[-1], D), dtype=np.uint16)
    V = rng.integers(0, 1 << 16, size=(L, Hkv, cu[-1], D), dtype=np.uint16)
    say("320 (layer, head) pairs, two sequences: select and compact against the oracle")
    g = select_and_compact(S, L, Hkv, D, w, cu, bud, K, V)
    check_against_oracle(S, L, Hkv, w, cu, bud, g, K, V, D)


def check_units(wl, g, bud, units):
    for (l, h, s) in units:
        T, off = unit_slices(wl, s)
        P = T - wl.w
        r = oracle_unit(wl, l, h, s)
        Sg = g["scores"][l, h, off:off + P]
        what = f"{wl.name} unit (l={l}, h={h}, s={s}), budget {int(bud[l][h])}"
        floor = check_scores(Sg, r["S"], r["stats"][8], what)
        check_stats(g["stats"][l, h, s], r["stats"], what)
        o, n = int(g["offsets"][l, h, s]), int(g["counts"][l, h, s])
        check_unit_selection(g["idx"][o:o + n], Sg, r["S"], T, wl.w, int(bud[l][h]), floor, what)


def check_all_units_valid(wl, g, bud):
    """Every unit: its count, the window, ascending order and the top-k of the GPU scores; compaction."""
    cu = wl.cu_seqlens
    o = 0
    for l in range(wl.L):
        for h in range(wl.Hkv):
            for s in range(wl.B):
                T, off = unit_slices(wl, s)
                P, b = T - wl.w, int(bud[l][h])
                n = min(b, T)
                assert int(g["offsets"][l, h, s]) == o and int(g["counts"][l, h, s]) == n
                idx = g["idx"][o:o + n]
                if b >= T:
                    np.testing.assert_array_equal(idx, np.arange(T))
                else:
                    k = b - wl.w
                    np.testing.assert_array_equal(idx[k:], np.arange(P, T))
                    np.testing.assert_array_equal(idx[:k], topk_rule(g["scores"][l, h, off:off + P], k))
                np.testing.assert_array_equal(g["Kc"][o:o + n], wl.K[l, h, cu[s] + idx])
                np.testing.assert_array_equal(g["Vc"][o:o + n], wl.V[l, h, cu[s] + idx])
                o += n
    assert o == len(g["idx"])


def test_stack28_pyramid_schedule():
    import paper_2609_06663_amd as P
    wl = W.stack28()
    per_layer = P.ecokv_pyramid_budgets(wl.L, wl.L * wl.budget[0], 20.0, wl.w)
    bud = [[b] * wl.Hkv for b in per_layer]
    say(f"stack28 with the PyramidKV schedule (beta 20): {per_layer[0]} .. {per_layer[-1]} tokens per head")
    g = gpu_pass(wl, mode=P.HEAD_BUDGETS, budget=bud)
    check_all_units_valid(wl, g, bud)
    check_units(wl, g, bud, [(0, 0, 0), (14, 1, 0), (27, 3, 0)])


def test_layer7b_sparsemm_like_head_budgets():
    # SparseMM assigns each head the window, a uniform share and a head-specific
    # share; here the head-specific share is random (the visual-head scores
    # come from a benchmark run outside this library)
    import paper_2609_06663_amd as P
    wl = W.custom(43, L=2, Hq=28, Hkv=4, D=128, w=8, seqlens=[4096, 1500], dtype="bf16", group=128)
    rng = np.random.default_rng(43)
    bud = (8 + 64 + rng.integers(0, 2000, size=(wl.L, wl.Hkv))).astype(np.int32)
    bud[1, 2] = 8
    say(f"two layers, SparseMM-like head budgets {bud.tolist()}")
    g = gpu_pass(wl, mode=P.HEAD_BUDGETS, budget=bud)
    check_all_units_valid(wl, g, bud)
    check_units(wl, g, bud, [(l, h, s) for l in range(wl.L) for h in range(wl.Hkv) for s in range(wl.B)])
