"""Pins for the oracle's stochastic acceptance (Preliminaries, "Speculative
Decoding": under sampling the standard acceptance-rejection rule keeps the
target distribution).

* sample_index: on a uniform grid of u every index is drawn with frequency
  w_i / sum(w) (to the grid's resolution); zero weights are never drawn.
* The rule itself: for one draft position, the distribution of the
  committed token, integrated over the draft sample, the acceptance test and
  the resample on fine grids, equals the verifier's p to the grid's
  resolution; the same computation with a plausible mistake (resampling from
  p instead of max(0, p - q), or testing p/q the wrong way round) is far off.
* T -> 0: the sampled round is the greedy round (same drafts, A and state).
"""
import numpy as np
import pytest

from oracle import decode as od
from tests.test_oracle_model import _clone, _prefilled

N_GRID = 4000


def _grid():
    return (np.arange(N_GRID) + 0.5) / N_GRID


def test_sample_index_frequencies():
    rng = np.random.default_rng(0)
    w = rng.random(7)
    w[3] = 0.0
    counts = np.bincount([od.sample_index(w, u) for u in _grid()], minlength=7)
    np.testing.assert_allclose(counts / N_GRID, w / w.sum(), atol=2.0 / N_GRID)
    assert counts[3] == 0
    assert od.sample_index(np.array([0.0, 0.0, 2.0, 1.0]), 0.0) == 2


def _committed_distribution(p, q, resample, accept):
    """Exact-to-grid distribution of the committed token at one position."""
    V = len(p)
    out = np.zeros(V)
    grid = _grid()
    res = np.bincount([od.sample_index(resample(p, q), u) for u in grid], minlength=V) / N_GRID
    for d in range(V):
        acc = np.mean([accept(p, q, d, u) for u in grid])
        out += q[d] * (acc * np.eye(V)[d] + (1 - acc) * res)
    return out


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_acceptance_rule_preserves_target_distribution(seed):
    rng = np.random.default_rng(seed)
    V = 6
    p = od.softmax_t(rng.standard_normal(V) * 1.5, 1.0)
    q = od.softmax_t(rng.standard_normal(V) * 1.5, 1.0)

    def accept(p_, q_, d, u):
        return od.stochastic_accept(p_[None], q_[None], np.array([d]), np.array([u])) == 1

    got = _committed_distribution(p, q, lambda a, b: od.resample_weights(a, b), accept)
    np.testing.assert_allclose(got, p, atol=5.0 / N_GRID)
    # plausible mistakes are caught
    wrong_res = _committed_distribution(p, q, lambda a, b: od.resample_weights(a, None), accept)
    wrong_acc = _committed_distribution(
        p, q, lambda a, b: od.resample_weights(a, b),
        lambda p_, q_, d, u: u * p_[d] < q_[d])
    assert np.abs(wrong_res - p).max() > 0.01
    assert np.abs(wrong_acc - p).max() > 0.01
    # after full acceptance the final token is drawn from p itself
    np.testing.assert_array_equal(od.resample_weights(p, None), p)


@pytest.mark.parametrize("seed,B", [(40, 4), (41, 3)])
def test_zero_temperature_limit_is_the_greedy_round(seed, B):
    m, st = _prefilled(seed, B=B, n_causal=B + 1)
    rng = np.random.default_rng(seed)
    a, sa = _clone(m), st.copy()
    b, sb = _clone(m), st.copy()
    for _ in range(3):
        u = rng.random((sa.kv_len.shape[0], 2 * B + 2))
        A_g = a.literal_round(sa, B)[3]
        _, _, A_s, _, err = b.sampled_round(sb, B, 1e-4, u)
        assert err == 0
        np.testing.assert_array_equal(A_g, A_s)
        np.testing.assert_array_equal(sa.draft, sb.draft)
        np.testing.assert_array_equal(sa.out_tokens, sb.out_tokens)
        np.testing.assert_array_equal(sa.kv_len, sb.kv_len)
