"""The C ABI library loads and exports every entry point of include/ecokv.h,
and its host-side argument checks reject bad calls before any device work.
No GPU needed: every call here returns from host validation."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = []
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            names += re.findall(r"^(?:int|const char \*|size_t)\s*\*?\s*(ecokv_\w+)\s*\(", text, re.M)
    return sorted(set(names))


@pytest.fixture(scope="module")
def P():
    import paper_2609_06663_amd as P
    return P


def test_header_declares_the_three_calls():
    names = declared_functions()
    for n in ("ecokv_score", "ecokv_select", "ecokv_compact", "ecokv_workspace_size", "ecokv_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol(P):
    from paper_2609_06663_amd import ecokv
    lib = ctypes.CDLL(ecokv._LIB_PATH)
    for n in declared_functions():
        assert hasattr(lib, n), f"{n} is declared but not exported"
    assert set(declared_functions()) == set(ecokv.EXPORTS)


def test_default_params(P):
    p = P.ecokv_default_params()
    assert p.alpha == pytest.approx(0.8) and p.beta == pytest.approx(0.6)
    assert p.pool_kernel == 5 and p.causal == 1 and p.lambda_override != p.lambda_override


def test_workspace_and_index_count(P):
    s = P.Shape(28, 28, 4, 128, 4, [0, 32768])
    assert P.ecokv_workspace_size(s) > 0
    assert P.ecokv_index_count(s, [6553]) == 28 * 4 * 6553
    s2 = P.Shape(2, 8, 2, 64, 3, [0, 10, 15])
    assert P.ecokv_index_count(s2, [4, 100]) == 2 * 2 * (4 + 5)


@pytest.mark.parametrize("args,code", [
    ((1, 4, 2, 96, 4, [0, 100]), -3),      # head_dim unsupported
    ((1, 5, 2, 128, 4, [0, 100]), -1),     # H_q not a multiple of H_kv
    ((1, 4, 2, 128, 0, [0, 100]), -1),     # window < 1
    ((1, 4, 2, 128, 100, [0, 100]), -1),   # window >= T
    ((1, 4, 2, 128, 4, [1, 100]), -1),     # cu_seqlens[0] != 0
    ((1, 4, 2, 128, 4, [0, 50, 52]), -1),  # a sequence not longer than the window
    ((-1, 4, 2, 128, 4, [0, 100]), -1),    # negative layers
    ((1, 64, 2, 128, 4, [0, 100]), -3),    # (H_q/H_kv)*w = 128 rows > max
])
def test_bad_shapes_rejected(P, args, code):
    with pytest.raises(P.EcoKVError) as e:
        P.ecokv_workspace_size(P.Shape(*args))
    assert e.value.code == code
    assert P.ecokv_last_error()


def test_too_many_sequences(P):
    cu = list(range(0, 10 * 66, 10))
    with pytest.raises(P.EcoKVError):
        P.ecokv_workspace_size(P.Shape(1, 4, 2, 128, 4, cu))


@pytest.mark.parametrize("field,value", [("pool_kernel", 4), ("pool_kernel", 0), ("eps", -1.0),
                                         ("causal", 2), ("alpha", float("inf"))])
def test_bad_params_rejected(P, field, value):
    p = P.Params()
    setattr(p, field, value)
    with pytest.raises(P.EcoKVError) as e:
        P.ecokv_workspace_size(P.Shape(1, 4, 2, 128, 4, [0, 100]), p)
    assert e.value.code == -1


def test_calls_fail_before_device_work(P):
    """Null pointers, a short workspace, budgets below the window: rejected on the host."""
    from paper_2609_06663_amd import ecokv as E
    s = P.Shape(1, 4, 2, 128, 4, [0, 100])
    p = P.Params()
    ws = P.ecokv_workspace_size(s, p)
    lib = E.lib
    fake = ctypes.c_void_p(256)
    # NULL K
    rc = lib.ecokv_score(None, fake, 0, ctypes.byref(s.c), ctypes.byref(p), fake, None, None, fake, ws, None)
    assert rc == -1
    # workspace too small
    rc = lib.ecokv_score(fake, fake, 0, ctypes.byref(s.c), ctypes.byref(p), fake, None, None, fake, ws - 1, None)
    assert rc == -2
    # misaligned workspace
    rc = lib.ecokv_score(fake, fake, 0, ctypes.byref(s.c), ctypes.byref(p), fake, None, None,
                         ctypes.c_void_p(260), ws, None)
    assert rc == -1
    # unsupported dtype
    rc = lib.ecokv_score(fake, fake, 7, ctypes.byref(s.c), ctypes.byref(p), fake, None, None, fake, ws, None)
    assert rc == -3
    bud = (ctypes.c_int32 * 1)(3)   # below the window
    rc = lib.ecokv_select(fake, ctypes.byref(s.c), 0, bud, fake, None, None, fake, 1 << 30, None)
    assert rc == -1
    bud = (ctypes.c_int32 * 1)(10)
    rc = lib.ecokv_select(fake, ctypes.byref(s.c), 1, bud, fake, None, None, fake, 1 << 30, None)   # flat without counts
    assert rc == -1
    rc = lib.ecokv_select(fake, ctypes.byref(s.c), 5, bud, fake, None, None, fake, 1 << 30, None)   # bad mode
    assert rc == -1
    # layer-flat scores of a layer beyond 2^31 bytes (8 heads x 67.1 M tokens)
    big = P.Shape(1, 8, 8, 128, 4, [0, 1 << 26, (1 << 26) + 200000])
    bud2 = (ctypes.c_int32 * 2)(10, 10)
    rc = lib.ecokv_select(fake, ctypes.byref(big.c), 1, bud2, fake, fake, fake, fake, 1 << 30, None)
    assert rc == -3 and b"2^31" in lib.ecokv_last_error()
    rc = lib.ecokv_compact(fake, None, 0, ctypes.byref(s.c), 0, bud, fake, None, None, fake, fake, None)
    assert rc == -1
    rc = lib.ecokv_compact(fake, fake, 0, ctypes.byref(s.c), 1, bud, fake, None, None, fake, fake, None)
    assert rc == -1   # flat without offsets


def test_empty_call_is_ok_without_device(P):
    # L = 0: nothing to enqueue, success, no device access.
    from paper_2609_06663_amd import ecokv as E
    s = P.Shape(0, 4, 2, 128, 4, [0, 100])
    p = P.Params()
    rc = E.lib.ecokv_score(None, None, 0, ctypes.byref(s.c), ctypes.byref(p), None, None, None, None, 0, None)
    assert rc == 0


@pytest.mark.parametrize("m", [1, 2, 3, 4, 5, 7, 28, 32, 80])
@pytest.mark.parametrize("total,beta", [(4096, 2.0), (1000, 4.0), (183484, 20.0), (1234.5, 2.5), (900, 1.5),
                                        (4096, 1.0), (300, 0.75)])
def test_pyramid_budgets_match_oracle(P, m, total, beta):
    import oracle
    want = oracle.pyramid_budgets(m, total, beta)
    w = 4
    if min(want) < w:
        with pytest.raises(P.EcoKVError) as e:
            P.ecokv_pyramid_budgets(m, total, beta, w)
        assert e.value.code == -1
    else:
        assert P.ecokv_pyramid_budgets(m, total, beta, w) == want


@pytest.mark.parametrize("args", [(0, 100.0, 2.0, 1), (3, 0.0, 2.0, 1), (3, 100.0, -1.0, 1), (3, float("nan"), 2.0, 1),
                                  (3, 100.0, 2.0, 0), (2, 1e12, 2.0, 1)])
def test_pyramid_budgets_rejects(P, args):
    with pytest.raises(P.EcoKVError) as e:
        P.ecokv_pyramid_budgets(*args)
    assert e.value.code == -1


def test_head_budget_index_count(P):
    import oracle
    cu = [0, 10, 25, 27]
    s = P.Shape(2, 6, 3, 128, 1, cu)
    bud = [[1, 5, 30], [10, 15, 2]]
    want = oracle.index_count(2, 3, cu, bud, oracle.HEAD_BUDGETS)
    assert want == sum(min(b, T) for row in bud for b in row for T in (10, 15, 2))
    assert P.ecokv_index_count_mode(s, P.HEAD_BUDGETS, bud) == want
    assert P.ecokv_index_count_mode(s, P.PER_HEAD, [3, 4, 1]) == P.ecokv_index_count(s, [3, 4, 1])
    with pytest.raises(ValueError):
        P.ecokv_index_count_mode(s, P.HEAD_BUDGETS, [1, 2, 3])   # one per sequence is the wrong shape
    with pytest.raises(P.EcoKVError):
        P.ecokv_index_count_mode(s, 7, [1, 2, 3])


def test_head_budget_calls_fail_before_device_work(P):
    from paper_2609_06663_amd import ecokv as E
    s = P.Shape(2, 4, 2, 128, 4, [0, 100])
    lib = E.lib
    fake = ctypes.c_void_p(256)
    bud = (ctypes.c_int32 * 4)(10, 20, 3, 50)   # pair (1, 0) below the window
    assert lib.ecokv_select(fake, ctypes.byref(s.c), 2, bud, fake, None, None, fake, 1 << 30, None) == -1
    assert "below the window" in P.ecokv_last_error()
    assert lib.ecokv_compact(fake, fake, 0, ctypes.byref(s.c), 2, bud, fake, None, None, fake, fake, None) == -1
    bud = (ctypes.c_int32 * 4)(10, 20, 30, 50)
    assert lib.ecokv_select(None, ctypes.byref(s.c), 2, bud, fake, None, None, fake, 1 << 30, None) == -1   # NULL scores
    assert lib.ecokv_compact(fake, None, 0, ctypes.byref(s.c), 2, bud, fake, None, None, fake, fake, None) == -1
    s0 = P.Shape(0, 4, 2, 128, 4, [0, 100])
    assert lib.ecokv_select(None, ctypes.byref(s0.c), 2, None, None, None, None, None, 0, None) == 0   # nothing to do


def test_value_norm_mode_checks(P):
    from paper_2609_06663_amd import ecokv as E
    s = P.Shape(2, 8, 2, 128, 4, [0, 1000])
    p0, p1 = P.Params(), P.Params(imp_mode=P.IMP_ATTN_VNORM)
    assert P.ecokv_default_params().imp_mode == P.IMP_ATTN
    # one float per non-window key of the workspace holds the finished importance
    assert P.ecokv_workspace_size(s, p1) >= P.ecokv_workspace_size(s, p0) + 4 * 2 * 2 * 996
    bad = P.Params(imp_mode=5)
    with pytest.raises(P.EcoKVError):
        P.ecokv_workspace_size(s, bad)
    fake = ctypes.c_void_p(256)
    ws = P.ecokv_workspace_size(s, p1)
    lib = E.lib
    # ecokv_score has no V: the value-norm mode is refused there
    rc = lib.ecokv_score(fake, fake, 0, ctypes.byref(s.c), ctypes.byref(p1), fake, None, None, fake, ws, None)
    assert rc == -1 and "ecokv_score_v" in P.ecokv_last_error()
    # ecokv_score_v needs V in that mode
    rc = lib.ecokv_score_v(fake, None, fake, 0, ctypes.byref(s.c), ctypes.byref(p1), fake, None, None, fake, ws,
                           None)
    assert rc == -1
    # the value-norm workspace is larger (fp32 keys: the larger of the two layouts)
    ws0 = P.ecokv_workspace_size(s, p0)
    rc = lib.ecokv_score_v(fake, fake, fake, 1, ctypes.byref(s.c), ctypes.byref(p1), fake, None, None, fake, ws0,
                           None)
    assert rc == -2


def test_alternative_options_defaults_and_checks(P):
    d = P.ecokv_default_params()
    assert (d.norm_mode, d.redundancy, d.centroid_scope) == (P.NORM_MINMAX, P.RED_EUCLID, P.CENTROID_ALL)
    assert d.winsor_q == pytest.approx(0.01) and d.mad_tau == 1.0
    s = P.Shape(1, 4, 2, 128, 4, [0, 100])
    for kw in (dict(norm_mode=3), dict(norm_mode=-1), dict(winsor_q=0.5), dict(winsor_q=-0.1),
               dict(mad_tau=0.0), dict(mad_tau=float("inf")), dict(redundancy=2), dict(centroid_scope=2)):
        with pytest.raises(P.EcoKVError) as e:
            P.ecokv_workspace_size(s, P.Params(**kw))
        assert e.value.code == -1, kw
    for kw in (dict(norm_mode=P.NORM_WINSOR, winsor_q=0.0), dict(norm_mode=P.NORM_MAD, mad_tau=2.0),
               dict(redundancy=P.RED_STD), dict(centroid_scope=P.CENTROID_PREFIX)):
        assert P.ecokv_workspace_size(s, P.Params(**kw)) > 0


def test_decode_checks_before_device_work(P):
    from paper_2609_06663_amd import ecokv as E
    s = P.Shape(2, 8, 2, 128, 4, [0, 100])
    assert P.ecokv_decode_workspace_size(s, 768) == 4 * 2 * 8 * 1 * 1 * 130
    assert P.ecokv_decode_workspace_size(s, 769) == 4 * 2 * 8 * 1 * 2 * 130
    with pytest.raises(P.EcoKVError):
        P.ecokv_decode_workspace_size(s, 0)
    lib = E.lib
    fake = ctypes.c_void_p(256)
    ws = P.ecokv_decode_workspace_size(s, 100)
    args = lambda **kw: [kw.get("Q", fake), fake, fake, kw.get("dtype", 0), ctypes.byref(s.c), fake, fake,
                         kw.get("mc", 100), kw.get("O", fake), None, kw.get("ws", fake), kw.get("wsb", ws), None]
    assert lib.ecokv_decode(*args(Q=None)) == -1
    assert lib.ecokv_decode(*args(O=None)) == -1
    assert lib.ecokv_decode(*args(dtype=5)) == -3
    assert lib.ecokv_decode(*args(mc=0)) == -1
    assert lib.ecokv_decode(*args(wsb=ws - 1)) == -2
    assert lib.ecokv_decode(*args(ws=ctypes.c_void_p(260))) == -1
    assert lib.ecokv_decode(*args(Q=ctypes.c_void_p(264))) == -1   # not 16-byte aligned


def test_workspace_status_checks_before_device_work(P):
    from paper_2609_06663_amd import ecokv as E
    assert E.lib.ecokv_workspace_status(None, None) == -1
    assert E.lib.ecokv_workspace_status(ctypes.c_void_p(260), None) == -1
    assert P.ETIMEOUT == -5


def test_binding_refuses_host_tensors(P):
    # the binding checks device, element type and size before calling the
    # library: a host tensor never reaches a kernel
    import torch
    s = P.Shape(1, 4, 2, 128, 4, [0, 100])
    K = torch.zeros(2 * 100 * 128, dtype=torch.bfloat16)
    Q = torch.zeros(4 * 4 * 128, dtype=torch.bfloat16)
    out = torch.zeros(2 * 96)
    with pytest.raises(ValueError, match="GPU tensor"):
        P.ecokv_score(K, Q, s, None, out, workspace=torch.zeros(1 << 20, dtype=torch.uint8))
    with pytest.raises(ValueError, match="GPU tensor"):
        P.ecokv_select(out, s, P.PER_HEAD, [10], torch.zeros(20, dtype=torch.int32))


def test_select_workspace_checks(P):
    from paper_2609_06663_amd import ecokv as E
    s = P.Shape(2, 8, 2, 128, 4, [0, 1000, 5000])
    fake = ctypes.c_void_p(256)
    bud = (ctypes.c_int32 * 2)(100, 200)
    for mode in (P.PER_HEAD, P.LAYER_FLAT, P.HEAD_BUDGETS):
        assert P.ecokv_select_workspace_size(s, mode) > 0
    need = P.ecokv_select_workspace_size(s, P.PER_HEAD)
    lib = E.lib
    assert lib.ecokv_select(fake, ctypes.byref(s.c), 0, bud, fake, None, None, None, need, None) == -1   # NULL
    assert lib.ecokv_select(fake, ctypes.byref(s.c), 0, bud, fake, None, None, ctypes.c_void_p(260), need,
                            None) == -1   # misaligned
    assert lib.ecokv_select(fake, ctypes.byref(s.c), 0, bud, fake, None, None, fake, need - 1, None) == -2
    # a layer-flat group holds every head's keys of a (layer, sequence): more slices per group
    assert P.ecokv_select_workspace_size(P.Shape(1, 8, 8, 128, 4, [0, 32768]), P.LAYER_FLAT) > \
        P.ecokv_select_workspace_size(P.Shape(1, 8, 8, 128, 4, [0, 32768]), P.PER_HEAD) // 8


def test_prefill_write_fails_before_device_work(P):
    """NULL, unpaired, misaligned or overlapping buffers, a short workspace and an
    unsupported element type are refused on the host; L = 0 enqueues nothing."""
    from paper_2609_06663_amd import ecokv as E
    s = P.Shape(1, 4, 2, 128, 4, [0, 100])
    p = P.Params()
    lib = E.lib
    n = ctypes.c_size_t(0)
    assert lib.ecokv_prefill_workspace_size(ctypes.byref(s.c), ctypes.byref(n)) == 0 and n.value > 0
    ws = n.value
    assert P.ecokv_prefill_workspace_size(s) == ws
    # fake device addresses far apart (51200 bytes of rows each), never dereferenced
    kn, kc, q, pre, wsp = (ctypes.c_void_p(1 << b) for b in (20, 30, 34, 38, 36))

    def call(K_new=kn, V_new=None, K_cache=kc, V_cache=None, dtype=0, w=wsp, nbytes=ws):
        return lib.ecokv_prefill_write(K_new, V_new, q, dtype, ctypes.byref(s.c), ctypes.byref(p), K_cache, V_cache,
                                       pre, w, nbytes, None)

    assert call(K_new=None) == -1
    assert call(K_cache=None) == -1
    assert call(V_cache=ctypes.c_void_p(1 << 39)) == -1                  # V_cache without V_new
    assert call(K_cache=kn) == -1                                         # the cache on the new rows
    assert "overlap" in P.ecokv_last_error()
    assert call(K_cache=ctypes.c_void_p((1 << 20) + 4096)) == -1          # ... partly
    assert call(K_new=ctypes.c_void_p((1 << 20) + 8)) == -1               # misaligned rows
    assert call(w=ctypes.c_void_p((1 << 36) + 16)) == -1                  # misaligned workspace
    assert call(nbytes=ws - 1) == -2
    assert call(dtype=7) == -3
    empty = P.Shape(0, 4, 2, 128, 4, [0, 100])
    assert lib.ecokv_prefill_write(None, None, None, 0, ctypes.byref(empty.c), ctypes.byref(p), None, None, None, None,
                                   0, None) == 0
