"""Pins of the oracle's E-step sampler against what mathematics fixes.

The paper names no sampler; the library's normative definition (Philox4x32-10,
a uniform on a 2^-24 grid, a fixed float32 log, Gumbel-max) is checked here
against: the accuracy of the log versus float64 log on every input it can
ever see, the Gumbel law of -log(-log U) over the whole uniform grid, the
Gumbel-max theorem (draw frequencies = softmax(logit/T), chi-square), the
statistical quality of the Philox stream, and the tie rules.
"""
import math

import numpy as np
import pytest
from scipy import stats

from oracle import sampler

GRID = np.arange(2 ** 23, dtype=np.int64)


def _all_u():
    return ((2 * GRID + 1).astype(np.float32) * np.float32(2.0 ** -24))


def _ulp_err(approx, exact):
    ulp = np.spacing(np.maximum(np.abs(exact), 1e-30).astype(np.float32)).astype(np.float64)
    return np.abs(approx.astype(np.float64) - exact) / ulp


def test_uniform_grid_is_exact_and_symmetric():
    u = _all_u()
    assert u.dtype == np.float32
    assert np.all(np.diff(u) > 0) and u[0] == np.float32(2.0 ** -24) and u[-1] == np.float32(1 - 2.0 ** -24)
    # every word maps onto the grid through its top 23 bits
    w = np.array([0, 511, 512, 0xFFFFFFFF], dtype=np.uint32)
    assert list(sampler.uniform_from_word(w)) == [u[0], u[0], u[1], u[-1]]
    np.testing.assert_array_equal(u + u[::-1], np.ones_like(u))


def test_spec_log_within_two_ulp_on_every_uniform():
    u = _all_u()
    lu = sampler.spec_log(u)
    assert _ulp_err(lu, np.log(u.astype(np.float64))).max() <= 2.0


def test_spec_log_within_two_ulp_on_every_exponential():
    e = -sampler.spec_log(_all_u())
    assert e.min() > 0 and np.all(np.isfinite(e))
    le = sampler.spec_log(e)
    assert _ulp_err(le, np.log(e.astype(np.float64))).max() <= 2.0


def test_spec_log_special_values():
    x = np.array([1.0, 2.0, 0.5, 2.0 ** -24, 2.0 ** 20, math.e, 10.0], dtype=np.float32)
    got = sampler.spec_log(x).astype(np.float64)
    ref = np.log(x.astype(np.float64))
    assert got[0] == 0.0
    assert np.all(_ulp_err(got.astype(np.float32), ref) <= 1.0)
    # across the range split at sqrt(2): continuous and increasing
    m = np.nextafter(np.float32(1.41421354), np.float32(0))
    pts = np.array([m, np.float32(1.41421354), np.nextafter(np.float32(1.41421354), np.float32(2))], dtype=np.float32)
    assert np.all(np.diff(sampler.spec_log(pts)) >= 0)


def test_gumbel_law_over_the_whole_grid():
    """-log(-log U) with U uniform on the grid has the Gumbel(0,1) moments:
    mean = Euler-Mascheroni gamma, variance = pi^2/6 (up to grid truncation)."""
    words = (GRID.astype(np.uint64) << np.uint64(9)).astype(np.uint32)
    g = sampler.gumbel_from_word(words).astype(np.float64)
    assert abs(g.mean() - np.euler_gamma) < 1e-5
    assert abs(g.var() - math.pi ** 2 / 6) < 1e-4
    # CDF at a few points: P(G <= t) = exp(-exp(-t))
    for t in (-1.0, 0.0, 1.0, 3.0):
        assert abs((g <= t).mean() - math.exp(-math.exp(-t))) < 1e-6


@pytest.mark.parametrize("temperature", [1.0, 0.5, 2.0])
def test_gumbel_max_draw_frequencies_match_softmax(temperature):
    """Gumbel-max theorem: argmax(logit/T + G) ~ softmax(logit/T)."""
    logits = np.array([0.0, 1.0, -0.5, 2.0, 0.3, -3.0], dtype=np.float32)
    n = 200_000
    rows = np.arange(n)
    keys = sampler.gumbel_keys(np.broadcast_to(logits, (n, logits.size)), rows, 0, temperature, seed=7, offset=3)
    z = sampler.first_argmax(keys)
    counts = np.bincount(z, minlength=logits.size)
    lg = logits.astype(np.float64) / temperature
    p = np.exp(lg - lg.max())
    p /= p.sum()
    _, pval = stats.chisquare(counts, p * n)
    assert pval > 1e-4, (counts, p * n)


def test_philox_words_are_uniform_and_bits_balanced():
    n_calls = 1 << 18
    w = np.stack(sampler.philox4x32_10(np.arange(n_calls), 5, 1, 9, seed=0x1234_5678_9ABC_DEF0)).reshape(-1)
    top = (w >> np.uint32(24)).astype(np.int64)
    _, pval = stats.chisquare(np.bincount(top, minlength=256))
    assert pval > 1e-4
    ones = np.array([((w >> np.uint32(b)) & np.uint32(1)).sum() for b in range(32)])
    n = w.size
    assert np.all(np.abs(ones - n / 2) < 5 * math.sqrt(n / 4))


def test_philox_avalanche_on_every_counter_and_key_word():
    """Flipping one input bit flips about half of the 128 output bits."""
    base = sampler.philox4x32_10(11, 22, 33, 44, seed=99)
    base_bits = np.concatenate([np.unpackbits(np.array([x], dtype='>u4').view(np.uint8)) for x in base])
    flips = []
    for word in range(4):
        for bit in (0, 7, 19, 31):
            c = [11, 22, 33, 44]
            c[word] ^= 1 << bit
            out = sampler.philox4x32_10(*c, seed=99)
            bits = np.concatenate([np.unpackbits(np.array([x], dtype='>u4').view(np.uint8)) for x in out])
            flips.append((bits != base_bits).sum())
    for kbit in (0, 31, 32, 63):
        out = sampler.philox4x32_10(11, 22, 33, 44, seed=99 ^ (1 << kbit))
        bits = np.concatenate([np.unpackbits(np.array([x], dtype='>u4').view(np.uint8)) for x in out])
        flips.append((bits != base_bits).sum())
    flips = np.array(flips)
    assert flips.min() > 40 and flips.max() < 88 and abs(flips.mean() - 64) < 8


def test_streams_differ_by_row_family_seed_offset_and_repeat_exactly():
    a = sampler.random_words([3], 0, 64, seed=1, offset=0)
    assert np.array_equal(a, sampler.random_words([3], 0, 64, seed=1, offset=0))
    for other in (sampler.random_words([4], 0, 64, seed=1, offset=0),
                  sampler.random_words([3], 1, 64, seed=1, offset=0),
                  sampler.random_words([3], 0, 64, seed=2, offset=0),
                  sampler.random_words([3], 0, 64, seed=1, offset=1),
                  sampler.random_words([3], 0, 64, seed=1 << 32, offset=0)):
        assert (a != other).mean() > 0.95


def test_word_selection_uses_v_div_4_and_v_mod_4():
    w = sampler.random_words([5], 1, 10, seed=3, offset=2)[0]
    for v in range(10):
        words = sampler.philox4x32_10(v >> 2, 5, 1, 2, seed=3)
        assert w[v] == words[v & 3]


def test_argmax_ties_go_to_the_smallest_index():
    a = np.array([[1.0, 3.0, 3.0, 2.0], [5.0, 5.0, 5.0, 5.0]])
    assert list(sampler.first_argmax(a)) == [1, 0]


def test_greedy_token_is_the_first_maximum_of_the_mapped_target():
    x = np.zeros((1, 4), dtype=np.float32)
    y_mapped = np.array([[0.5, 2.0, 2.0, -1.0]], dtype=np.float32)
    _, _, zg = sampler.sample_rows(x, y_mapped, np.array([0]), 1.0, 1.0, 0, 0)
    assert zg[0] == 1


def test_key_arithmetic_is_float32_throughout():
    keys = sampler.gumbel_keys(np.array([[0.1, -2.5, 7.25]], dtype=np.float32), [0], 0, 0.7, 0, 0)
    assert keys.dtype == np.float32
    inv_t = np.float32(1) / np.float32(0.7)
    g = sampler.gumbel_from_word(sampler.random_words([0], 0, 3, 0, 0))
    manual = np.array([[0.1, -2.5, 7.25]], dtype=np.float32) * inv_t + g
    np.testing.assert_array_equal(keys, manual)
