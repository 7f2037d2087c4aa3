"""The native TeaCache gate (host code behind dit_teacache_gate) against the oracle's gate: the
hand-worked sequence, random sequences with rescale polynomials (decisions exact, accumulator to
1e-15), and argument errors. No GPU."""
import numpy as np
import pytest

from oracle import dit_oracle as O


@pytest.fixture(scope="module")
def d():
    from paper_2606_19004_amd import ditstep
    return ditstep


def _past_first(st):
    st.has_prev, st.has_residual = 1, 1


def test_hand_sequence(d):
    st = d.teacache_state(0.3)
    assert d.dit_teacache_gate(st, 0.5) is True          # no previous input yet: run
    _past_first(st)
    assert [d.dit_teacache_gate(st, r) for r in (0.1, 0.15, 0.1, 0.02, 0.25)] == [False, False, True, False, False]
    assert st.accumulated == pytest.approx(0.27)
    assert d.dit_teacache_gate(st, 0.01, force=True) is True and st.accumulated == 0.0
    st2 = d.teacache_state(0.3, coef=[2.0, 0.0])
    _past_first(st2)
    assert [d.dit_teacache_gate(st2, r) for r in (0.1, 0.1, 0.05)] == [False, True, False]


@pytest.mark.parametrize("seed", range(5))
def test_random_sequences_match_oracle(d, seed):
    rng = np.random.default_rng(seed)
    coef = [] if seed == 0 else rng.uniform(-2, 2, rng.integers(1, 6)).tolist()
    thr = float(rng.uniform(0.05, 1.5))
    nat, ref = d.teacache_state(thr, coef), O.TeaCacheState(thr, coef)
    _past_first(nat)
    ref.h_prev, ref.residual = 1, 1
    for _ in range(400):
        rel = float(rng.uniform(0, 0.4))
        force = bool(rng.random() < 0.05)
        assert d.dit_teacache_gate(nat, rel, force) == ref.gate(rel, force)
        assert abs(nat.accumulated - ref.accumulated) <= 1e-12 * max(1.0, abs(ref.accumulated))


def test_init_errors(d):
    for args in [(-0.1, ()), (0.1, tuple(range(9))), (float("nan"), ())]:
        with pytest.raises(d.DitError):
            d.teacache_state(*args)
    st = d.teacache_state(0.2)
    _past_first(st)
    with pytest.raises(d.DitError):
        d.dit_teacache_gate(st, float("nan"))
