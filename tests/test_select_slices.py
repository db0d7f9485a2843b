"""The premise of the library's two-stage selection of long single-head units
(CPU): the chosen keys of a unit, restricted to one slice of it, are that
slice's own largest keys under the same order (score descending, position
ascending), so the union of every slice's min(k, slice) largest holds them
all, and choosing k among that union, taken in position order, gives the
unit's selection (Sec. 3 selection rule; ties favour the smaller position).
Checked against the oracle's selection on random, tied, NaN and signed-zero
scores, with slices shorter than k too."""
import numpy as np
import pytest

import oracle


@pytest.fixture(scope="module", autouse=True)
def _build():
    oracle.build(force=False)


def top_in_order(S, k):
    """Positions of the k largest of S (the oracle's order), ascending."""
    w = 1  # a one-key window that is never among the candidates
    return oracle.select_unit(S, len(S) + w, w, k + w)[:k]


def two_stage(S, k, slice_len):
    cand = []
    for s0 in range(0, len(S), slice_len):
        seg = S[s0:s0 + slice_len]
        cand.extend((top_in_order(seg, min(k, len(seg))) + s0).tolist())
    cand = np.asarray(cand, np.int64)
    assert (np.diff(cand) > 0).all()  # position order
    chosen = top_in_order(S[cand], k)
    return cand[chosen]


def cases():
    rng = np.random.default_rng(71)
    yield "normal", rng.standard_normal(5000)
    yield "ties", rng.integers(0, 4, 5000).astype(np.float64)
    s = rng.integers(0, 3, 4000).astype(np.float64)
    s[100:400] = np.nan
    s[500:900] = -0.0
    s[1000:1010] = np.inf
    yield "nan_zero_inf", s


@pytest.mark.parametrize("name,S", list(cases()))
@pytest.mark.parametrize("slice_len", [7, 64, 1000])
@pytest.mark.parametrize("k", [1, 37, 500, 2100])
def test_slices_hold_the_selection(name, S, slice_len, k):
    ref = top_in_order(S, k)
    np.testing.assert_array_equal(two_stage(S, k, slice_len), ref)
