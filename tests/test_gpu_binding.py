"""The binding's checks with GPU tensors of the wrong type or size (refused
before any launch), and the workspace status after a bounded wait that the
host makes give up at once (every kernel still ends normally)."""
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
    print(f"[gpu-binding] {msg}", file=sys.stderr, flush=True)


def test_wrong_types_and_sizes_are_refused():
    import paper_2609_06663_amd as P
    say("binding checks: wrong element types and short buffers")
    s = P.Shape(2, 8, 2, 128, 4, [0, 300])
    K = torch.zeros(2 * 2 * 300 * 128, dtype=torch.bfloat16, device="cuda")
    Q = torch.zeros(2 * 8 * 4 * 128, dtype=torch.bfloat16, device="cuda")
    S = torch.zeros(2 * 2 * 296, dtype=torch.float32, device="cuda")
    with pytest.raises(ValueError, match="K has"):
        P.ecokv_score(K[:-1], Q, s, None, S)
    with pytest.raises(ValueError, match="Q_win has"):
        P.ecokv_score(K, Q[:-128], s, None, S)
    with pytest.raises(ValueError, match="scores has"):
        P.ecokv_score(K, Q, s, None, S[:-1])
    with pytest.raises(TypeError, match="scores must be float32"):
        P.ecokv_score(K, Q, s, None, S.to(torch.bfloat16))
    with pytest.raises(ValueError, match="workspace has"):
        P.ecokv_score(K, Q, s, None, S, workspace=torch.zeros(1024, dtype=torch.uint8, device="cuda"))
    n = P.ecokv_index_count(s, [40])
    idx = torch.zeros(n, dtype=torch.int32, device="cuda")
    with pytest.raises(ValueError, match="idx has"):
        P.ecokv_select(S, s, P.PER_HEAD, [40], idx[:-1])
    with pytest.raises(TypeError, match="idx must be int32"):
        P.ecokv_select(S, s, P.PER_HEAD, [40], idx.to(torch.int64))
    with pytest.raises(ValueError, match="counts is required"):
        P.ecokv_select(S, s, P.LAYER_FLAT, [40], idx)
    Kc = torch.zeros(n * 128, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ValueError, match="Vc has"):
        P.ecokv_compact(K, K, s, P.PER_HEAD, [40], idx, None, None, Kc, Kc[:-1])
    torch.cuda.synchronize()


def test_forced_wait_timeout_is_reported(monkeypatch):
    import paper_2609_06663_amd as P
    from paper_2609_06663_amd.pipeline import EvictionPass
    # 8996 non-window keys: four blocks of 4096 keys per unit, which exchange sums
    wl = W.custom(41, L=1, Hq=8, Hkv=2, D=128, w=4, seqlens=[9000], dtype="bf16", budget=[900])
    shape = P.Shape(wl.L, wl.Hq, wl.Hkv, wl.D, wl.w, wl.cu_seqlens)
    ep = EvictionPass(shape, wl.budget, P.PER_HEAD, P.Params(), torch.bfloat16)
    K, V, Q = dev(wl.K, "bf16"), dev(wl.V, "bf16"), dev(wl.Q, "bf16")
    say("split epilogue with a spin limit of 0: its wait gives up at once")
    monkeypatch.setenv("ECOKV_SPIN_LIMIT", "0")
    ep.score(K, Q)
    with pytest.raises(P.EcoKVError) as e:
        ep.check()
    assert e.value.code == P.ETIMEOUT
    lam = ep.lambda_.cpu().numpy()
    assert np.isnan(lam).all() and np.isnan(ep.scores.cpu().numpy()).all()
    say("the query cleared the record; a normal call then reports nothing")
    monkeypatch.delenv("ECOKV_SPIN_LIMIT")
    ep.check()
    ep.score(K, Q)
    ep.check()
    assert np.isfinite(ep.lambda_.cpu().numpy()).all() and np.isfinite(ep.scores.cpu().numpy()).all()


def test_forced_wait_timeout_long_units(monkeypatch):
    # units of 32769 to 65536 non-window keys: eight blocks of 8192 keys per unit exchange sums
    import paper_2609_06663_amd as P
    from paper_2609_06663_amd.pipeline import EvictionPass
    wl = W.custom(42, L=1, Hq=4, Hkv=1, D=128, w=4, seqlens=[40000], dtype="bf16", budget=[4000])
    shape = P.Shape(wl.L, wl.Hq, wl.Hkv, wl.D, wl.w, wl.cu_seqlens)
    ep = EvictionPass(shape, wl.budget, P.PER_HEAD, P.Params(), torch.bfloat16)
    K, Q = dev(wl.K, "bf16"), dev(wl.Q, "bf16")
    say("eight-block epilogue with a spin limit of 0: its waits give up at once")
    monkeypatch.setenv("ECOKV_SPIN_LIMIT", "0")
    ep.score(K, Q)
    with pytest.raises(P.EcoKVError) as e:
        ep.check()
    assert e.value.code == P.ETIMEOUT
    assert np.isnan(ep.lambda_.cpu().numpy()).all() and np.isnan(ep.scores.cpu().numpy()).all()
    monkeypatch.delenv("ECOKV_SPIN_LIMIT")
    ep.score(K, Q)
    ep.check()
    assert np.isfinite(ep.lambda_.cpu().numpy()).all() and np.isfinite(ep.scores.cpu().numpy()).all()
