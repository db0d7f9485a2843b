"""GPU parity of ecokv_prefill_write: the KV-cache write of a prefill with the
first sweep over K as its by-product (Sec. 3 window attention; Eq. (1)
centroid; Appendix A.1 mu).

  cache   bit-exact: K_cache / V_cache are the new token-major rows moved to
          the head-major layout of the pass.
  pre     against the oracle's prefill_sums (float64):
            key sums     |g - o| <= 2e-3 max(|o|, m / sqrt(T)), m the column's
                         absolute mass sum_i |x_i| (a sum of T terms whose
                         cancellation leaves |o| far below its terms is held to
                         the scale of its terms over sqrt(T));
            row reference m_r + log(z_r), the row's log-sum-exp (all the
                         pass uses): |g - o| <= 2e-3 max(|o|, 1);
            row reference m_r: at most the row's largest logit (the oracle's
                         m_r) and within 16 ln 2 of it, each to 2e-3 max(|o|, 1)
                         (the streaming sweep moves its reference lazily).
  pass    ecokv_score_pre on the written cache with the written pre: scores,
          statistics and selections against the oracle's pass (parity_utils).
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity_utils import dev, gpu_pass, host_bits
from test_gpu_parity import check_compact, check_per_head

pytestmark = pytest.mark.gpu

RTOL = 2e-3


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_06663_amd  # noqa: F401  (fails loudly if the library is not built)
    oracle.build(force=False)


def say(msg):
    print(f"[gpu-prefill] {msg}", file=sys.stderr, flush=True)


def token_major(a: np.ndarray) -> np.ndarray:
    """[L][Hkv][Ttot][D] -> [L][Ttot][Hkv][D] (the layout a projection writes)."""
    return np.ascontiguousarray(np.swapaxes(a, 1, 2))


def run_prefill(wl, params=None, with_v=True):
    import paper_2609_06663_amd as P
    shape = P.Shape(wl.L, wl.Hq, wl.Hkv, wl.D, wl.w, wl.cu_seqlens)
    Kn, Vn, Q = dev(token_major(wl.K), wl.dtype), dev(token_major(wl.V), wl.dtype), dev(wl.Q, wl.dtype)
    # the cache in the pass's head-major shape, filled with 7s (every row must be written)
    Kc = torch.full(wl.K.shape, 7, dtype=Kn.dtype, device="cuda")
    Vc = torch.full(wl.V.shape, 7, dtype=Vn.dtype, device="cuda")
    R = wl.G * wl.w
    pre = torch.full((wl.L * wl.Hkv * wl.B * (2 * wl.D + 2 * R),), float("nan"), device="cuda")
    P.ecokv_prefill_write(Kn, Vn if with_v else None, Q, shape, params or P.Params(), Kc, Vc if with_v else None, pre)
    torch.cuda.synchronize()
    return host_bits(Kc), host_bits(Vc), pre.cpu().numpy().astype(np.float64).reshape(wl.L, wl.Hkv, wl.B, -1)


def check_pre(wl, pre_g, causal=True, what=""):
    D, R, cu = wl.D, wl.G * wl.w, wl.cu_seqlens
    pre_o = oracle.prefill_sums(wl.K, wl.Q, wl.L, wl.Hq, wl.Hkv, cu, D, wl.w, causal=causal,
                                nthreads=__import__("os").cpu_count() or 1)
    assert np.isfinite(pre_g).all(), f"{what}: pre has non-finite entries"
    for l in range(wl.L):
        for h in range(wl.Hkv):
            for s in range(wl.B):
                K = wl.f32(wl.K[l, h, cu[s]:cu[s + 1]]).astype(np.float64)
                T = K.shape[0]
                kh = K / np.maximum(np.linalg.norm(K, axis=1, keepdims=True), 1e-12)
                mass = np.concatenate([np.abs(K).sum(axis=0), np.abs(kh).sum(axis=0)])
                g, o = pre_g[l, h, s], pre_o[l, h, s]
                tol = RTOL * np.maximum(np.abs(o[:2 * D]), mass / np.sqrt(T))
                bad = np.abs(g[:2 * D] - o[:2 * D]) > tol
                assert not bad.any(), f"{what} unit {(l, h, s)}: key sums off at columns {np.nonzero(bad)[0][:8]}"
                mg, mo = g[2 * D:2 * D + R], o[2 * D:2 * D + R]
                slack = RTOL * np.maximum(np.abs(mo), 1.0)
                assert ((mg <= mo + slack) & (mg >= mo - 16 * np.log(2.0) - slack)).all(), \
                    f"{what} unit {(l, h, s)}: row reference {mg} vs largest logit {mo}"
                lg, lo = mg + np.log(g[2 * D + R:]), mo + np.log(o[2 * D + R:])
                assert (np.abs(lg - lo) <= RTOL * np.maximum(np.abs(lo), 1.0)).all(), \
                    f"{what} unit {(l, h, s)}: row log-sum-exp {lg} vs {lo}"


def check_cache(wl, Kc, Vc, with_v=True):
    np.testing.assert_array_equal(Kc, wl.K)
    if with_v:
        np.testing.assert_array_equal(Vc, wl.V)
    else:  # untouched
        seven = host_bits(torch.full((1,), 7, dtype=torch.bfloat16 if wl.dtype == "bf16" else torch.float32))
        assert (Vc == seven[0]).all()


@pytest.mark.parametrize("dtype,D,Hq,Hkv,w,seqlens", [
    ("bf16", 128, 28, 4, 4, [3000, 517, 1200]),   # streaming sweep with the cache write (512-key blocks)
    ("bf16", 128, 8, 8, 8, [4100]),               # one query head per KV head, R = 8
    ("bf16", 128, 32, 4, 8, [2100, 700]),         # R = 64: copy, then the block sweep
    ("f32", 64, 4, 2, 8, [1500, 333, 70]),        # fp32 keys
    ("bf16", 64, 8, 2, 4, [2000, 9]),             # head_dim 64; a sequence just past the window
])
def test_prefill_write_matches_oracle(dtype, D, Hq, Hkv, w, seqlens):
    wl = W.custom(93, L=2, Hq=Hq, Hkv=Hkv, D=D, w=w, seqlens=seqlens, dtype=dtype,
                  budget=[max(w, t // 5) for t in seqlens], group=64)
    say(f"{dtype} D={D} Hq={Hq} Hkv={Hkv} w={w} T={seqlens}: cache write with the first sweep")
    Kc, Vc, pre = run_prefill(wl)
    check_cache(wl, Kc, Vc)
    check_pre(wl, pre, what=f"{dtype} D{D}")
    say("  the pass on the written cache with the written sums")
    g = gpu_pass(wl, pre=pre)
    check_per_head(wl, g)
    check_compact(wl, g)


def test_prefill_write_keys_only_and_non_causal():
    import paper_2609_06663_amd as P
    wl = W.custom(94, L=1, Hq=8, Hkv=2, D=128, w=4, seqlens=[2100, 257], dtype="bf16", budget=[400, 60], group=64)
    say("keys only (no V), non-causal window rows")
    Kc, Vc, pre = run_prefill(wl, params=P.Params(causal=False), with_v=False)
    check_cache(wl, Kc, Vc, with_v=False)
    check_pre(wl, pre, causal=False, what="non-causal")
    p = P.Params(causal=False)
    g = gpu_pass(wl, params=p, pre=pre)
    check_per_head(wl, g, params=p)


def test_prefill_write_full_length():
    # 64 units of 32768 keys, 64 blocks each
    wl = W.custom(95, L=8, Hq=56, Hkv=8, D=128, w=4, seqlens=[32768], dtype="bf16", budget=[6553], group=256)
    say("8 layers x 8 KV heads x 32768 tokens")
    Kc, Vc, pre = run_prefill(wl)
    check_cache(wl, Kc, Vc)
    check_pre(wl, pre, what="T=32768")
    g = gpu_pass(wl, pre=pre)
    check_per_head(wl, g)


def test_prefill_write_refusals_leave_outputs_alone():
    import paper_2609_06663_amd as P
    wl = W.custom(96, L=1, Hq=4, Hkv=2, D=128, w=4, seqlens=[300], dtype="bf16")
    shape = P.Shape(wl.L, wl.Hq, wl.Hkv, wl.D, wl.w, wl.cu_seqlens)
    Kn, Q = dev(token_major(wl.K), "bf16"), dev(wl.Q, "bf16")
    pre = torch.zeros(wl.L * wl.Hkv * wl.B * (2 * wl.D + 2 * wl.G * wl.w), device="cuda")
    # the cache on top of the new rows: refused before anything is enqueued
    with pytest.raises(P.EcoKVError) as e:
        P.ecokv_prefill_write(Kn, None, Q, shape, P.Params(), Kn, None, pre)
    assert e.value.code == P.EINVAL
    torch.cuda.synchronize()
    assert (pre == 0).all()


def test_score_pre_takes_log_sum_exp_pairs():
    # any pair with the row's log-sum-exp as m_r + log z_r: here (lse, 1), as a
    # flash-attention prefill outputs it
    wl = W.custom(97, L=1, Hq=28, Hkv=4, D=128, w=4, seqlens=[2500, 700], dtype="bf16", budget=[500, 140], group=64)
    D, R = wl.D, wl.G * wl.w
    pre = oracle.prefill_sums(wl.K, wl.Q, wl.L, wl.Hq, wl.Hkv, wl.cu_seqlens, D, wl.w)
    pre[..., 2 * D:2 * D + R] += np.log(pre[..., 2 * D + R:])
    pre[..., 2 * D + R:] = 1.0
    say("window rows handed over as (log-sum-exp, 1)")
    g = gpu_pass(wl, pre=pre)
    check_per_head(wl, g)
