"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Every case draws seeded synthetic inputs (workloads/), runs score -> select ->
compact on the GPU and compares with the oracle on the same bytes, to the
tolerances stated in parity_utils.  Every unit of every shape is compared,
the full-size ones (28 layers x 32k tokens, 32 heads x 64k tokens) included,
with the oracle on all host threads.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity_utils import (check_scores, check_stats, check_unit_selection, dev, gpu_pass, oracle_all,
                          oracle_params, oracle_unit, topk_rule, unit_slices, RTOL)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_06663_amd  # noqa: F401  (fails loudly if the library is not built)
    oracle.build(force=False)


def say(msg):
    print(f"[gpu-parity] {msg}", file=sys.stderr, flush=True)


def check_compact(wl, g):
    cu = wl.cu_seqlens
    for l in range(wl.L):
        for h in range(wl.Hkv):
            for s in range(wl.B):
                o, n = int(g["offsets"][l, h, s]), int(g["counts"][l, h, s])
                rows = g["idx"][o:o + n]
                np.testing.assert_array_equal(g["Kc"][o:o + n], wl.K[l, h, cu[s] + rows])
                np.testing.assert_array_equal(g["Vc"][o:o + n], wl.V[l, h, cu[s] + rows])


def check_per_head(wl, g, units=None, params=None, stat_skip=()):
    """Every unit (or the listed ones) against the oracle: scores, statistics, selection."""
    if units is None:
        units = [(l, h, s) for l in range(wl.L) for h in range(wl.Hkv) for s in range(wl.B)]
        So_all, st_all = oracle_all(wl, params)
    else:
        So_all = st_all = None
    ties = 0
    for (l, h, s) in units:
        T, off = unit_slices(wl, s)
        P = T - wl.w
        if So_all is None:
            r = oracle_unit(wl, l, h, s, params)
            So, sto = r["S"], r["stats"]
        else:
            So, sto = So_all[l, h, off:off + P], st_all[l, h, s]
        Sg = g["scores"][l, h, off:off + P]
        what = f"{wl.name} unit (l={l}, h={h}, s={s})"
        floor = check_scores(Sg, So, sto[8], what)
        check_stats(g["stats"][l, h, s], sto, what, skip=stat_skip)
        assert g["lambda_"][l, h, s] == g["stats"][l, h, s, 0]
        o, n = int(g["offsets"][l, h, s]), int(g["counts"][l, h, s])
        ties += check_unit_selection(g["idx"][o:o + n], Sg, So, T, wl.w, wl.budget[s], floor, what)
    return ties


def check_all_selections_valid(wl, g):
    """Properties that hold for every unit: count, window, order, range, top-k of the GPU scores."""
    for l in range(wl.L):
        for h in range(wl.Hkv):
            for s in range(wl.B):
                T, off = unit_slices(wl, s)
                P, b = T - wl.w, wl.budget[s]
                o, n = int(g["offsets"][l, h, s]), int(g["counts"][l, h, s])
                assert n == min(b, T)
                idx = g["idx"][o:o + n]
                if b >= T:
                    np.testing.assert_array_equal(idx, np.arange(T))
                    continue
                k = b - wl.w
                np.testing.assert_array_equal(idx[k:], np.arange(P, T))
                Sg = g["scores"][l, h, off:off + P]
                np.testing.assert_array_equal(idx[:k], topk_rule(Sg, k))


def test_tiny_full():
    wl = W.tiny()
    say("tiny: 1 layer, 2 heads, T=512, fp32")
    g = gpu_pass(wl)
    check_per_head(wl, g)
    check_compact(wl, g)


def test_layer7b_full():
    wl = W.layer7b()
    say("layer7b: 28q/4kv, T=8192, bf16, w=8, b=1638")
    g = gpu_pass(wl)
    check_per_head(wl, g)
    check_compact(wl, g)


def test_stack28_full_size():
    wl = W.stack28()
    say("stack28: 28 layers, 28q/4kv, T=32768, bf16, w=4, b=6553 (every unit against the oracle)")
    g = gpu_pass(wl)
    check_all_selections_valid(wl, g)
    check_compact(wl, g)
    check_per_head(wl, g)
    # every lambda is a blend of two redundancies in [-1/(T-1), 1]
    assert np.all(g["lambda_"] <= 1.0 + 1e-6) and np.all(g["lambda_"] > -1e-3)


@pytest.mark.parametrize("frac", [0.1, 0.4])
def test_stack_other_budgets(frac):
    # the stack's other two per-head budgets, on its first two layers
    wl = W.stack28(L=2, budget_frac=frac)
    say(f"stack, 2 layers, budget {frac:.0%} per head ({wl.budget[0]} tokens)")
    g = gpu_pass(wl)
    check_all_selections_valid(wl, g)
    check_compact(wl, g)
    check_per_head(wl, g)


def test_mha64k_full_size():
    wl = W.mha64k()
    say("mha64k: 32 MHA heads, T=65536, bf16, w=8, b=2048 (every unit against the oracle)")
    g = gpu_pass(wl)
    check_all_selections_valid(wl, g)
    check_compact(wl, g)
    check_per_head(wl, g)


@pytest.mark.parametrize("strength", [10.0, 30.0, 100.0])
@pytest.mark.parametrize("form", ["stream", "block", "generic"])
def test_high_anisotropy(strength, form):
    # A shared offset of norm a sqrt(D) over unit-variance keys gives a mean key
    # cosine of about a^2 / (1 + a^2): 0.99, 0.9989, 0.9999 -- the regime the
    # paper reports for the first layer (Sec. 4).  The distance to the centroid
    # is then a small difference of large vectors.  Three sweep forms: bf16 /
    # D 128 with one 32-row window operand (w 4, G 7), with several (w 8, G 7),
    # and fp32 / D 64.  The window queries are plain N(0, I) draws: were they
    # to share the offset too, the logits would reach a^2 D / sqrt(D) ~ 1e5 at
    # a = 100, where fp32 rounding of q.k alone exceeds the score tolerance.
    kw = dict(strength=strength, query_offset=False)
    if form == "stream":
        wl = W.custom(31, L=2, Hq=28, Hkv=4, D=128, w=4, seqlens=[6000, 2500], dtype="bf16", **kw)
    elif form == "block":
        wl = W.custom(32, L=1, Hq=28, Hkv=4, D=128, w=8, seqlens=[8192], dtype="bf16", **kw)
    else:
        wl = W.custom(33, L=1, Hq=8, Hkv=2, D=64, w=4, seqlens=[3000], dtype="f32", **kw)
    say(f"high anisotropy a={strength}, {form} sweeps: sequences {wl.seqlens}")
    g = gpu_pass(wl)
    check_per_head(wl, g)
    check_compact(wl, g)


@pytest.mark.parametrize("case", ["rows28_short_keys", "rows29", "rows30"])
def test_stream_key_norms(case):
    # The streaming sweep 2 at the edges of its 32-row operand (window rows
    # G w = 29 and 30 beside the two rows of mu), and with keys far shorter
    # than the centroid among strongly aligned ones, where k.mu / |k| and
    # |k - kbar| are each computed from a short key.
    if case == "rows28_short_keys":
        wl = W.custom(34, L=1, Hq=28, Hkv=4, D=128, w=4, seqlens=[3000, 1100], dtype="bf16",
                      strength=10.0, query_offset=False)
        rng = np.random.default_rng(35)
        K = W.bf16_bits_to_f32(wl.K)
        for h in range(wl.Hkv):
            rows = rng.choice(wl.cu_seqlens[-1], size=150, replace=False)
            K[0, h, rows] *= rng.uniform(0.0, 0.2, size=(150, 1)).astype(np.float32)
        wl.K[...] = W.to_bf16_bits(K)
    elif case == "rows29":
        wl = W.custom(36, L=1, Hq=29, Hkv=1, D=128, w=1, seqlens=[2500, 700], dtype="bf16")
    else:
        wl = W.custom(37, L=1, Hq=10, Hkv=2, D=128, w=6, seqlens=[4100], dtype="bf16")
    say(f"streaming sweep 2 key norms: {case}, G*w = {wl.Hq // wl.Hkv * wl.w}, sequences {wl.seqlens}")
    g = gpu_pass(wl)
    check_per_head(wl, g)
    check_compact(wl, g)


def check_layer_flat(wl, g, params=None):
    cu = wl.cu_seqlens
    for l in range(wl.L):
        for s in range(wl.B):
            T, off = unit_slices(wl, s)
            P, b = T - wl.w, wl.budget[s]
            H = wl.Hkv
            So = np.zeros((H, P))
            Sg = g["scores"][l, :, off:off + P]
            floor = 0.0
            for h in range(H):
                r = oracle_unit(wl, l, h, s, params)
                So[h] = r["S"]
                f = check_scores(Sg[h], r["S"], r["stats"][8], f"{wl.name} (l={l}, h={h}, s={s})")
                check_stats(g["stats"][l, h, s], r["stats"], f"{wl.name} (l={l}, h={h}, s={s})")
                floor = max(floor, f)
            counts = g["counts"][l, :, s]
            offs = g["offsets"][l, :, s]
            assert counts.sum() == H * min(b, T)
            if b >= T:
                for h in range(H):
                    np.testing.assert_array_equal(g["idx"][offs[h]:offs[h] + counts[h]], np.arange(T))
                continue
            assert np.all(offs[1:] == offs[:-1] + counts[:-1])
            chosen_g = []
            for h in range(H):
                ent = g["idx"][offs[h]:offs[h] + counts[h]]
                np.testing.assert_array_equal(ent[-wl.w:], np.arange(P, T))
                sel = ent[:-wl.w]
                assert np.all(np.diff(sel) > 0)
                chosen_g += [h * P + i for i in sel]
            ktot = H * (b - wl.w)
            chosen_g = np.array(sorted(chosen_g), dtype=np.int64)
            np.testing.assert_array_equal(chosen_g, topk_rule(Sg.reshape(-1), ktot))
            flat_o = So.reshape(-1)
            chosen_o = topk_rule(flat_o, ktot)
            if ktot:
                theta = np.sort(flat_o)[::-1][ktot - 1]
                band = RTOL * max(abs(theta), floor)
                far = [v for v in np.setxor1d(chosen_g, chosen_o) if abs(flat_o[v] - theta) > band]
                assert not far, f"layer-flat (l={l}, s={s}): {len(far)} disagreements outside the band"


def test_varlen_layer_flat_full():
    wl = W.varlen()
    say(f"varlen layer-flat: 8 sequences {wl.seqlens}, 28q/4kv, bf16, w=4")
    g = gpu_pass(wl)
    check_layer_flat(wl, g)
    check_compact(wl, g)


# ---------------------------------------------------------------------------
# edge cases
# ---------------------------------------------------------------------------

def test_ragged_varlen_per_head():
    wl = W.custom(11, L=2, Hq=6, Hkv=2, D=128, w=3, seqlens=[129, 1000, 257, 4, 130], dtype="bf16",
                  budget=[40, 300, 400, 3, 3 + 127], group=64)
    say("ragged varlen per-head: seqlens [129, 1000, 257, 4, 130]")
    g = gpu_pass(wl)
    check_per_head(wl, g)
    check_compact(wl, g)


def test_head_dim_64_fp32_window_1():
    wl = W.custom(12, L=1, Hq=8, Hkv=2, D=64, w=1, seqlens=[700], dtype="f32", budget=[97], group=32)
    say("D=64 fp32 w=1 G=4")
    g = gpu_pass(wl)
    check_per_head(wl, g)
    check_compact(wl, g)


def test_head_dim_64_bf16_gqa():
    wl = W.custom(18, L=2, Hq=12, Hkv=3, D=64, w=5, seqlens=[611, 90], dtype="bf16", budget=[120, 40], group=32)
    say("D=64 bf16 G=4 w=5 (generic sweep)")
    g = gpu_pass(wl)
    check_per_head(wl, g)
    check_compact(wl, g)


def test_max_window_rows():
    wl = W.custom(13, L=1, Hq=16, Hkv=2, D=128, w=8, seqlens=[300], dtype="bf16", budget=[60], group=16)
    say("G*w = 64 window rows")
    g = gpu_pass(wl)
    check_per_head(wl, g)


def test_long_ragged_single_sequence():
    wl = W.custom(14, L=1, Hq=4, Hkv=1, D=128, w=4, seqlens=[5003], dtype="bf16", budget=[777], group=128)
    say("T=5003 single head")
    g = gpu_pass(wl)
    check_per_head(wl, g)
    check_compact(wl, g)


def test_identical_and_zero_keys():
    # head 0: every key identical (zero diversity, lambda = 1); head 1: some zero keys.
    wl = W.custom(15, L=1, Hq=4, Hkv=2, D=128, w=4, seqlens=[600], dtype="bf16", budget=[100], group=32)
    wl.K[0, 0, :] = wl.K[0, 0, 17]
    wl.K[0, 1, 5:9] = 0
    wl.K[0, 1, 300] = 0
    say("identical keys in head 0, zero keys in head 1")
    g = gpu_pass(wl)
    check_per_head(wl, g, units=[(0, 0, 0)], stat_skip=("dmin", "dmax", "D_E", "sdiv_min", "sdiv_max",
                                                       "sbar_mean", "scale"))
    check_per_head(wl, g, units=[(0, 1, 0)])
    check_compact(wl, g)


def test_rising_logits():
    # key magnitudes ramp up along each sequence (x1 -> x8), so the window
    # logits (about 45 in log2 units at the start, 360 at the end) keep
    # setting new maxima far above the earlier ones: the running softmax
    # statistics must move their reference many times inside a block.  (A much
    # steeper ramp makes the logits so large that fp32 rounding of q.k alone
    # exceeds the score tolerance.)
    wl = W.custom(18, L=1, Hq=8, Hkv=2, D=128, w=4, seqlens=[5003, 2100], dtype="bf16", budget=[700, 300],
                  group=64)
    cu = wl.cu_seqlens
    for s in range(wl.B):
        n = cu[s + 1] - cu[s]
        ramp = np.exp(np.linspace(0.0, np.log(8.0), n)).astype(np.float32)
        k = W.bf16_bits_to_f32(wl.K[0, :, cu[s]:cu[s + 1]]) * ramp[None, :, None]
        wl.K[0, :, cu[s]:cu[s + 1]] = W.to_bf16_bits(k)
    say("rising logits: keys scaled x1..x8 along the sequence")
    g = gpu_pass(wl)
    check_per_head(wl, g)
    check_compact(wl, g)


@pytest.mark.parametrize("variant", ["noncausal", "lambda0", "lambda1_alpha1", "mixkv", "pool1", "pool7",
                                     "pool9", "pool11", "tau"])
def test_parameter_variants(variant):
    import paper_2609_06663_amd as P
    p = {
        "noncausal": P.Params(causal=False),
        "lambda0": P.Params(lambda_override=0.0),
        "lambda1_alpha1": P.Params(lambda_override=1.0, alpha=1.0),
        "mixkv": P.Params(alpha=0.0, beta=0.0),
        "pool1": P.Params(pool_kernel=1),
        "pool7": P.Params(pool_kernel=7),
        "pool9": P.Params(pool_kernel=9),    # widest pooling of the one-launch epilogue
        "pool11": P.Params(pool_kernel=11),  # wider: the two-launch epilogue
        "tau": P.Params(tau=3.0),
    }[variant]
    wl = W.custom(16, L=1, Hq=8, Hkv=2, D=128, w=4, seqlens=[900, 333], dtype="bf16", budget=[150, 60],
                  group=64)
    say(f"parameter variant {variant}")
    g = gpu_pass(wl, params=p)
    check_per_head(wl, g, params=p)


@pytest.mark.parametrize("seqlens", [[4100], [4101, 4100], [8196, 8197, 30], [16388, 16389], [32772], [32773],
                                     [100, 32772], [2052, 255], [65540], [65541], [32773, 40000, 700]])
def test_epilogue_unit_bounds(seqlens):
    # The one-launch epilogue spreads a unit's P non-window keys over 1, 2, 4
    # or 8 blocks of 4096 keys up to P = 32768, over 8 blocks of 8192 up to
    # P = 65536, and past that the two-launch epilogue takes over: P at each
    # boundary and one past it (window w = 4); short units leave most of a
    # block's keys, or whole blocks, past P
    wl = W.custom(24, L=1, Hq=8, Hkv=2, D=128, w=4, seqlens=seqlens, dtype="bf16", group=128)
    say(f"epilogue bounds: sequences {seqlens}")
    g = gpu_pass(wl)
    check_per_head(wl, g)
    check_compact(wl, g)


def test_budget_edges_per_head_and_flat():
    import paper_2609_06663_amd as P
    wl = W.custom(17, L=2, Hq=4, Hkv=2, D=128, w=5, seqlens=[300, 200, 150], dtype="bf16",
                  budget=[5, 400, 149], group=32)
    say("budgets b == w, b >= T, b = T - 1")
    g = gpu_pass(wl, mode=P.PER_HEAD)
    check_per_head(wl, g)
    check_compact(wl, g)
    wl.mode = "layer_flat"
    g = gpu_pass(wl, mode=P.LAYER_FLAT)
    check_layer_flat(wl, g)
    check_compact(wl, g)


def test_empty_layers_is_a_noop():
    import paper_2609_06663_amd as P
    shape = P.Shape(0, 4, 2, 128, 4, [0, 100])
    x = torch.zeros(16, device="cuda")
    P.ecokv_score(x, x, shape, None, x, workspace=torch.empty(256, dtype=torch.uint8, device="cuda"))
    P.ecokv_select(x, shape, P.PER_HEAD, [10], x)
    torch.cuda.synchronize()
    assert torch.all(x == 0)


def test_deterministic():
    wl = W.layer7b(seed=21, T=4096)
    say("determinism: two identical runs")
    g1 = gpu_pass(wl)
    g2 = gpu_pass(wl)
    for k in ("scores", "stats", "idx", "Kc"):
        np.testing.assert_array_equal(g1[k], g2[k])


# ---------------------------------------------------------------------------
# selection alone: bit-exact against the oracle on identical fp32 scores
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("mode", ["per_head", "layer_flat"])
def test_select_bit_exact_with_ties(mode):
    import paper_2609_06663_amd as P
    rng = np.random.default_rng(5)
    seqlens = [3000, 70, 1025, 9]
    cu = np.concatenate([[0], np.cumsum(seqlens)]).tolist()
    L, Hkv, w = 3, 4, 3
    budget = [500, 71, 1025 // 2, 3]
    Ptot = cu[-1] - len(seqlens) * w
    S = rng.integers(0, 40, size=(L, Hkv, Ptot)).astype(np.float32) * np.float32(0.25) - np.float32(2.0)
    S[0, 0, :50] = np.nan
    S[1, 2, 10:20] = -0.0
    S[1, 2, 20:30] = 0.0
    m = P.PER_HEAD if mode == "per_head" else P.LAYER_FLAT
    shape = P.Shape(L, 4 * Hkv, Hkv, 128, w, cu)
    n = P.ecokv_index_count(shape, budget)
    idx = torch.empty(n, dtype=torch.int32, device="cuda")
    counts = torch.empty(L * Hkv * len(seqlens), dtype=torch.int32, device="cuda")
    offsets = torch.empty_like(counts)
    say(f"select-only bit-exact ({mode})")
    P.ecokv_select(torch.from_numpy(S).cuda(), shape, m, budget, idx, counts, offsets)
    torch.cuda.synchronize()
    ref_idx, ref_c, ref_o = oracle.select(S.astype(np.float64), L, Hkv, cu, w, budget,
                                          oracle.PER_HEAD if m == P.PER_HEAD else oracle.LAYER_FLAT)
    np.testing.assert_array_equal(idx.cpu().numpy(), ref_idx)
    np.testing.assert_array_equal(counts.cpu().numpy(), ref_c.reshape(-1))
    np.testing.assert_array_equal(offsets.cpu().numpy(), ref_o.reshape(-1))


def _digit_case(case, rng, P=32000):
    """Scores of one P-key unit shaped for a path of the register radix select
    (counts scaled from the 32000-key form)."""
    f = P / 32000
    spread = np.exp(rng.uniform(np.log(1e-3), np.log(100.0), size=P)).astype(np.float32)
    if case == "prefix_overflow":
        # 31000 of 32000 keys in [1, 1.0001): one first digit (the exponent)
        # holds more keys than the stage can gather, so the later digits count
        # the registers (at smaller sizes the cluster fits the stage)
        S = spread.copy()
        nc = int(31000 * f)
        S[:nc] = 1.0 + rng.uniform(0, 1e-4, size=nc).astype(np.float32)
        k = int(12000 * f)
    elif case == "prefix_fits":
        S = spread.copy()
        nc = int(12000 * f)
        S[:nc] = 1.0 + rng.uniform(0, 1e-4, size=nc).astype(np.float32)
        k = int(9000 * f)
    elif case == "one_digit":
        # keys that differ only in their low 8 bits: a single radix digit
        S = (np.float32(1.0).view(np.uint32) + rng.integers(0, 200, size=P).astype(np.uint32)).view(np.float32)
        k = int(7000 * f)
    else:  # "cluster_ties": 64 values inside the cluster, many equal to the threshold
        S = spread.copy()
        nc = int(13000 * f)
        S[:nc] = 1.0 + rng.integers(0, 64, size=nc).astype(np.float32) * np.float32(1e-6)
        k = int(11000 * f)
    rng.shuffle(S)
    return S.astype(np.float32), k


@pytest.mark.parametrize("keys", [32000, 16000, 8000])  # 32, 16 and 8 keys per thread
@pytest.mark.parametrize("case", ["prefix_overflow", "prefix_fits", "one_digit", "cluster_ties"])
def test_select_register_digit_paths(case, keys):
    import paper_2609_06663_amd as P
    rng = np.random.default_rng({"prefix_overflow": 61, "prefix_fits": 62, "one_digit": 63, "cluster_ties": 64}[case]
                                + keys)
    w = 4
    S1, k = _digit_case(case, rng, keys)
    S2, _ = _digit_case(case, rng, keys)
    L, Hkv = 1, 2
    cu = [0, len(S1) + w]
    S = np.stack([S1, S2])[None]  # [L][Hkv][P]
    budget = [k + w]
    shape = P.Shape(L, Hkv, Hkv, 128, w, cu)
    n = P.ecokv_index_count(shape, budget)
    idx = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    counts = torch.full((L * Hkv,), -7, dtype=torch.int32, device="cuda")
    offsets = torch.full_like(counts, -7)
    say(f"select-only bit-exact, {case}: {keys} keys, k = {k}")
    P.ecokv_select(torch.from_numpy(np.ascontiguousarray(S)).cuda(), shape, P.PER_HEAD, budget, idx, counts, offsets)
    torch.cuda.synchronize()
    ref_idx, ref_c, ref_o = oracle.select(S.astype(np.float64), L, Hkv, cu, w, budget, oracle.PER_HEAD)
    np.testing.assert_array_equal(idx.cpu().numpy(), ref_idx)
    np.testing.assert_array_equal(counts.cpu().numpy(), ref_c.reshape(-1))
    np.testing.assert_array_equal(offsets.cpu().numpy(), ref_o.reshape(-1))


@pytest.mark.parametrize("case", ["list_fits", "list_overflows", "ties_in_list"])
def test_select_flat_large_group_paths(case):
    # layer-flat groups of 4 x 32000 keys: past the register select, so the
    # streaming select runs; its later digits count a gathered list of the keys
    # that keep the first digit's prefix (up to 32768 of them), or every key
    import paper_2609_06663_amd as P
    rng = np.random.default_rng({"list_fits": 71, "list_overflows": 72, "ties_in_list": 73}[case])
    L, Hkv, w, Pn = 1, 4, 4, 32000
    S = np.exp(rng.uniform(np.log(1e-3), np.log(100.0), size=(L, Hkv, Pn))).astype(np.float32)
    if case == "list_fits":
        S[..., :6000] = 1.0 + rng.uniform(0, 1e-4, size=(L, Hkv, 6000)).astype(np.float32)
    elif case == "list_overflows":
        S[..., :31000] = 1.0 + rng.uniform(0, 1e-4, size=(L, Hkv, 31000)).astype(np.float32)
    else:
        S[..., :6000] = 1.0 + rng.integers(0, 64, size=(L, Hkv, 6000)).astype(np.float32) * np.float32(1e-6)
    for h in range(Hkv):
        rng.shuffle(S[0, h])
    cu = [0, Pn + w]
    budget = [12000 + w]
    shape = P.Shape(L, Hkv, Hkv, 128, w, cu)
    n = P.ecokv_index_count(shape, budget)
    idx = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    counts = torch.full((L * Hkv,), -7, dtype=torch.int32, device="cuda")
    offsets = torch.full_like(counts, -7)
    say(f"layer-flat select-only bit-exact, {case}: 4 x 32000 keys, {Hkv * 12000} places")
    P.ecokv_select(torch.from_numpy(np.ascontiguousarray(S)).cuda(), shape, P.LAYER_FLAT, budget, idx, counts, offsets)
    torch.cuda.synchronize()
    ref_idx, ref_c, ref_o = oracle.select(S.astype(np.float64), L, Hkv, cu, w, budget, oracle.LAYER_FLAT)
    np.testing.assert_array_equal(idx.cpu().numpy(), ref_idx)
    np.testing.assert_array_equal(counts.cpu().numpy(), ref_c.reshape(-1))
    np.testing.assert_array_equal(offsets.cpu().numpy(), ref_o.reshape(-1))


@pytest.mark.parametrize("case", ["fits", "overflows"])
def test_select_register_64_keys_per_thread(case):
    # 60000-key units: 64 keys per thread; the later digits count the gathered
    # keys that keep the first digit's prefix, or every key when they overflow
    import paper_2609_06663_amd as P
    rng = np.random.default_rng({"fits": 81, "overflows": 82}[case])
    L, Hkv, w, Pn = 1, 2, 4, 60000
    S = np.exp(rng.uniform(np.log(1e-3), np.log(100.0), size=(L, Hkv, Pn))).astype(np.float32)
    nc = 10000 if case == "fits" else 55000
    S[..., :nc] = 1.0 + rng.uniform(0, 1e-4, size=(L, Hkv, nc)).astype(np.float32)
    for h in range(Hkv):
        rng.shuffle(S[0, h])
    cu = [0, Pn + w]
    budget = [20000 + w]
    shape = P.Shape(L, Hkv, Hkv, 128, w, cu)
    n = P.ecokv_index_count(shape, budget)
    idx = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    counts = torch.full((L * Hkv,), -7, dtype=torch.int32, device="cuda")
    offsets = torch.full_like(counts, -7)
    say(f"select-only bit-exact, 60000-key units, gathered list {case}")
    P.ecokv_select(torch.from_numpy(np.ascontiguousarray(S)).cuda(), shape, P.PER_HEAD, budget, idx, counts, offsets)
    torch.cuda.synchronize()
    ref_idx, ref_c, ref_o = oracle.select(S.astype(np.float64), L, Hkv, cu, w, budget, oracle.PER_HEAD)
    np.testing.assert_array_equal(idx.cpu().numpy(), ref_idx)
    np.testing.assert_array_equal(counts.cpu().numpy(), ref_c.reshape(-1))
    np.testing.assert_array_equal(offsets.cpu().numpy(), ref_o.reshape(-1))


# ---------------------------------------------------------------------------
# selection of groups past 32768 keys: shapes for each path of the
# multi-block form, and (per head, small budgets) of the two-stage form,
# bit-exact against the oracle
# ---------------------------------------------------------------------------

def _select_case(name, rng):
    """(L, Hkv, w, seqlens, budget, mode, scores[L][Hkv][Ptot] float32) for one case."""
    if name == "ties_across_slices":
        # 3 values over 40000 keys: the threshold class spans many slices
        L, Hkv, w, lens, bud = 1, 2, 4, [40004], [15004]
        S = rng.integers(0, 3, size=(L, Hkv, 40000)).astype(np.float32)
    elif name == "bin_taken_whole":
        # the k largest are exactly the keys of one top-digit bin and above
        L, Hkv, w, lens, bud = 1, 2, 4, [40004], [10004]
        S = rng.uniform(0.0, 0.5, size=(L, Hkv, 40000)).astype(np.float32)
        for h in range(Hkv):
            top = rng.choice(40000, 10000, replace=False)
            S[0, h, top] = rng.uniform(4.0, 8.0, size=10000).astype(np.float32)
    elif name == "flat_tiny_heads":
        # layer-flat groups of 256 short heads (P = 5 and 140): slices span many heads
        L, Hkv, w, lens, bud = 2, 256, 3, [8, 143], [5, 40]
        S = rng.integers(0, 5, size=(L, Hkv, 5 + 140)).astype(np.float32) * np.float32(0.5)
    elif name == "flat_long":
        L, Hkv, w, lens, bud = 1, 4, 4, [70004, 9000], [10504, 1350]
        S = rng.standard_normal((L, Hkv, 70000 + 8996)).astype(np.float32)
    elif name == "many_groups_16_per_thread":
        # 160 groups of 9 slices each: the 16-keys-per-thread form
        L, Hkv, w, lens, bud = 40, 4, 4, [33004], [6604]
        S = np.exp(rng.uniform(-8, 2, size=(L, Hkv, 33000))).astype(np.float32)
    elif name == "nan_and_signed_zero":
        L, Hkv, w, lens, bud = 1, 3, 2, [36002, 500], [15000, 300]
        S = rng.integers(-3, 3, size=(L, Hkv, 36000 + 498)).astype(np.float32) * np.float32(0.0) + \
            rng.integers(0, 4, size=(L, Hkv, 36498)).astype(np.float32)
        S[0, 0, :400] = np.nan
        S[0, 1, 100:900] = -0.0
        S[0, 2, 50:70] = np.inf
        S[0, 2, 70:90] = -np.inf
    elif name == "two_stage_normal":
        # per head: 8 slices of 8192 keys, k = 2048 (the two-stage form)
        L, Hkv, w, lens, bud = 1, 4, 4, [65540], [2052]
        S = rng.standard_normal((L, Hkv, 65536)).astype(np.float32)
    elif name == "two_stage_ties":
        # 7 values over 50000 keys, k = 1000: the threshold class spans every slice
        L, Hkv, w, lens, bud = 1, 2, 4, [50004], [1004]
        S = rng.integers(0, 7, size=(L, Hkv, 50000)).astype(np.float32)
    elif name == "two_stage_nan_inf_zero":
        L, Hkv, w, lens, bud = 1, 3, 2, [40002], [802]
        S = rng.integers(0, 5, size=(L, Hkv, 40000)).astype(np.float32)
        S[0, 0, 8000:8500] = np.nan
        S[0, 1, 100:20000] = -0.0
        S[0, 1, 30000:30010] = 0.0
        S[0, 2, 16380:16390] = np.inf
        S[0, 2, 70:90] = -np.inf
    elif name == "two_stage_short_tail":
        # 33000 keys: the fifth slice has 232, fewer than k = 1000 (all of them candidates)
        L, Hkv, w, lens, bud = 1, 2, 4, [33004], [1004]
        S = rng.standard_normal((L, Hkv, 33000)).astype(np.float32)
    elif name == "two_stage_ragged":
        # sequences of 70000, 9000 and 40000 keys (9, 2 and 5 slices), one kept whole
        L, Hkv, w, lens, bud = 2, 2, 4, [70004, 9004, 40004, 300], [3004, 504, 3004, 400]
        S = np.exp(rng.uniform(-6, 3, size=(L, Hkv, 70000 + 9000 + 40000 + 296))).astype(np.float32)
    else:
        raise ValueError(name)
    return L, Hkv, w, lens, bud, S


@pytest.mark.parametrize("mode", ["per_head", "layer_flat"])
@pytest.mark.parametrize("name", ["ties_across_slices", "bin_taken_whole", "flat_tiny_heads", "flat_long",
                                  "many_groups_16_per_thread", "nan_and_signed_zero", "two_stage_normal",
                                  "two_stage_ties", "two_stage_nan_inf_zero", "two_stage_short_tail",
                                  "two_stage_ragged"])
def test_select_multiblock_bit_exact(name, mode):
    import paper_2609_06663_amd as P
    import zlib
    rng = np.random.default_rng(zlib.crc32(f"{name}/{mode}".encode()))
    L, Hkv, w, lens, bud, S = _select_case(name, rng)
    cu = np.concatenate([[0], np.cumsum(lens)]).tolist()
    m = P.PER_HEAD if mode == "per_head" else P.LAYER_FLAT
    shape = P.Shape(L, Hkv, Hkv, 128, w, cu)
    n = P.ecokv_index_count(shape, bud)
    idx = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    counts = torch.full((L * Hkv * len(lens),), -7, dtype=torch.int32, device="cuda")
    offsets = torch.full_like(counts, -7)
    ws = torch.zeros(P.ecokv_select_workspace_size(shape, m), dtype=torch.uint8, device="cuda")
    say(f"multi-block select {name} ({mode}): {L} layers x {Hkv} heads, sequences {lens}")
    Sd = torch.from_numpy(np.ascontiguousarray(S)).cuda()
    ref_idx, ref_c, ref_o = oracle.select(S.astype(np.float64), L, Hkv, cu, w, bud,
                                          oracle.PER_HEAD if m == P.PER_HEAD else oracle.LAYER_FLAT)
    for rep in range(2):  # the same workspace twice: the calls leave it as they found it
        P.ecokv_select(Sd, shape, m, bud, idx, counts, offsets, ws)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(idx.cpu().numpy(), ref_idx)
        np.testing.assert_array_equal(counts.cpu().numpy(), ref_c.reshape(-1))
        np.testing.assert_array_equal(offsets.cpu().numpy(), ref_o.reshape(-1))
        idx.fill_(-7)
