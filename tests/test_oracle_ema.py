"""Pins of the oracle's planner statistics: the EMA update of counts
(Section 3.2, Stage 1 and Stage 2) and the Ochiai similarity (Section 1,
the footnote on Fig. 3)."""
import numpy as np
import pytest

import oracle

F32_EPS = 2.0 ** -23


def test_init_and_the_two_extreme_decays_are_exact():
    rng = np.random.default_rng(1)
    x = rng.integers(0, 2**31, size=1000).astype(np.uint32)
    ema, _ = oracle.count_ema(x, 0.9, init=True)
    assert np.array_equal(ema, x.astype(np.float32))          # init: m = x
    m0 = rng.random(1000).astype(np.float32) * 1e6
    ema, _ = oracle.count_ema(x, 1.0, ema=m0.copy())
    assert np.array_equal(ema, m0)                            # decay 1: unchanged
    ema, _ = oracle.count_ema(x, 0.0, ema=m0.copy())
    assert np.array_equal(ema, x.astype(np.float32))          # decay 0: the new count


@pytest.mark.parametrize("decay", [0.5, 0.9, 0.99])
def test_constant_input_follows_the_closed_form(decay):
    """From 0, k updates with the same count x give x (1 - decay^k)."""
    x = np.full(4, 1000, np.uint32)
    ema = np.zeros(4, np.float32)
    for k in range(1, 61):
        oracle.count_ema(x, decay, ema=ema)
        exact = 1000.0 * (1.0 - float(np.float32(decay)) ** k)
        # each update rounds at most three times: 1.5 ulp, accumulated k times
        assert abs(float(ema[0]) - exact) <= 1.5 * k * F32_EPS * 1000.0 + 1e-30


def test_matches_the_weighted_sum_of_past_counts():
    """m_k = b^k m_0 + (1 - b) sum_i b^(k-i) x_i, evaluated in fp64."""
    rng = np.random.default_rng(2)
    b = 0.8
    bf = float(np.float32(b))
    gain = float(np.float32(1.0) - np.float32(b))
    m0 = (rng.random(64) * 5000).astype(np.float32)
    xs = [rng.integers(0, 10**5, size=64).astype(np.uint32) for _ in range(30)]
    ema = m0.copy()
    for x in xs:
        oracle.count_ema(x, b, ema=ema)
    k = len(xs)
    exact = bf ** k * m0.astype(np.float64)
    for i, x in enumerate(xs, start=1):
        exact += gain * bf ** (k - i) * x.astype(np.float64)
    scale = np.maximum(m0, 10**5)
    assert np.all(np.abs(ema - exact) <= 1.5 * k * F32_EPS * scale)


def test_clear_zeroes_the_counts_after_reading():
    x = np.arange(10, dtype=np.uint32)
    ema, c = oracle.count_ema(x, 0.5, clear=True)
    assert not x.any() and c is x
    assert np.array_equal(ema, 0.5 * np.arange(10, dtype=np.float32))


@pytest.mark.parametrize("decay", [-0.1, 1.5, float("nan")])
def test_rejects_decay_outside_the_unit_interval(decay):
    with pytest.raises(oracle.OracleError):
        oracle.count_ema(np.zeros(3, np.uint32), decay)


def _sets(T, E, K, rng):
    """Random top-K selections and the token set A_e of each expert."""
    D = np.stack([rng.choice(E, size=K, replace=False) for _ in range(T)])
    A = [set(np.nonzero((D == e).any(1))[0].tolist()) for e in range(E)]
    return D, A


def test_ochiai_equals_the_set_definition():
    """O_ij = |A_i & A_j| / sqrt(|A_i| |A_j|) over the token sets, in fp64,
    against the oracle's fp32 value from counts (three roundings: 2 ulp)."""
    rng = np.random.default_rng(3)
    T, E, K = 400, 24, 4
    D, A = _sets(T, E, K, rng)
    coact = np.zeros((E, E), np.uint32)
    count = np.array([len(a) for a in A], np.uint32)
    for i in range(E):
        for j in range(E):
            if i != j:
                coact[i, j] = len(A[i] & A[j])
    got = oracle.ochiai(coact, count)
    for i in range(E):
        for j in range(E):
            inter = len(A[i] & A[j])
            want = inter / np.sqrt(len(A[i]) * len(A[j])) if inter else 0.0
            assert abs(float(got[i, j]) - want) <= 2 * F32_EPS * max(want, 1e-30)
    assert np.array_equal(got, got.T)
    assert got.max() <= 1.0


def test_ochiai_special_cases():
    # experts 0 and 1 selected by the same 9 tokens; 2 by 4 of those;
    # 3 by 5 other tokens; 4 by none
    count = np.array([9, 9, 4, 5, 0], np.uint32)
    coact = np.zeros((5, 5), np.uint32)
    coact[0, 1] = coact[1, 0] = 9
    coact[0, 2] = coact[2, 0] = coact[1, 2] = coact[2, 1] = 4
    O = oracle.ochiai(coact, count)
    assert O[0, 1] == 1.0                                  # identical sets
    assert abs(O[0, 2] - np.sqrt(4 / 9)) <= F32_EPS        # subset: sqrt(|A|/|B|)
    assert O[0, 3] == 0.0 and O[2, 3] == 0.0               # disjoint
    assert np.array_equal(np.diag(O), [1, 1, 1, 1, 0])    # inactive expert: 0
    assert not O[4].any() and not O[:, 4].any()
