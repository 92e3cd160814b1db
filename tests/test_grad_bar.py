"""The gradient parity bar rejects the mistakes the absolute 2e-3 bar cannot
see and accepts a correctly rounded result (CPU only).

The reference is the oracle's gradient (derivative of Eq. advance) on a
small batch whose rows span a few thousand entries, so that almost every
entry is far below 2e-3, as on the 32k-128k rows of the real workloads.
"""
import numpy as np
import pytest
import torch

from oracle import reference
from tests import grad_bar

V = 4000
N, L = 4, 3


@pytest.fixture(scope="module")
def case():
    rng = np.random.default_rng(7)
    npos = 2
    Y = rng.normal(0.0, 3.0, size=(npos * N * L, V))
    X = 0.8 * Y + rng.normal(0.0, 1.5, size=Y.shape)
    X = torch.as_tensor(X, dtype=torch.float32).to(torch.bfloat16).float().numpy()
    Y = torch.as_tensor(Y, dtype=torch.float32).to(torch.bfloat16).float().numpy()
    depth = np.array([[3, 1, 2, 3], [2, 3, 3, 1]])
    p = dict(temp_draft=0.7, temp_target=1.0, loss_scale=0.5)
    ora = reference.run_positions(X, Y, None, depth, [0, 1], N, L, p)
    m, rel = grad_bar.summand_magnitude(X, ora["lse_q"], ora["coef_a"], ora["coef_b"], ora["tok_draft"],
                                        ora["tok_target"], p["temp_draft"], p["loss_scale"])
    live = np.nonzero((ora["coef_a"] != 0) | (ora["coef_b"] != 0))[0]
    assert live.size > 4
    return ora["grad"], m, rel, live


def _bf16(a):
    return torch.as_tensor(np.asarray(a, dtype=np.float32)).to(torch.bfloat16).float().numpy()


def _truncate_bf16(a):
    bits = np.asarray(a, dtype=np.float32).view(np.uint32) & np.uint32(0xFFFF0000)
    return bits.view(np.float32).astype(np.float64)


def _rejects(got, ref, m, rel, bf16=True):
    e, r = grad_bar.violations(got, ref, m, rel, bf16)
    return bool(e.any() or r.any())


def test_most_entries_are_below_the_absolute_bar(case):
    ref, _, _, live = case
    assert np.mean(np.abs(ref[live]) < 2e-3) > 0.99


def test_accepts_round_to_nearest_bf16(case):
    ref, m, rel, _ = case
    assert not _rejects(_bf16(ref), ref, m, rel)


def test_accepts_float32_rounding_noise(case):
    ref, m, rel, _ = case
    rng = np.random.default_rng(1)
    got = (ref * (1.0 + 4e-6 * rng.standard_normal(ref.shape))).astype(np.float32)
    assert not _rejects(got, ref, m, rel, bf16=False)
    assert not _rejects(_bf16(got), ref, m, rel)


def test_rejects_a_zeroed_tail_chunk(case):
    ref, m, rel, live = case
    got = _bf16(ref)
    got[live[0], V - 64:] = 0.0
    assert np.all(np.abs(got - ref) <= 2e-3), "the absolute bar alone does not see it"
    assert _rejects(got, ref, m, rel)


def test_rejects_a_one_element_shift(case):
    ref, m, rel, live = case
    got = _bf16(ref)
    got[live[1], 1:] = got[live[1], :-1].copy()
    assert _rejects(got, ref, m, rel)


def test_rejects_truncating_rounding(case):
    ref, m, rel, _ = case
    got = _truncate_bf16(ref)
    assert np.all(np.abs(got - ref) <= 2e-3)
    assert _rejects(got, ref, m, rel)


def test_rejects_a_stale_normaliser(case):
    ref, m, rel, live = case
    got = _bf16(ref)
    r = live[2]
    got[r] = _bf16(ref[r] * 1.01)  # q formed with a log-sum-exp off by 0.01
    assert np.all(np.abs(got - ref) <= 2e-3)
    assert _rejects(got, ref, m, rel)


def test_rejects_writes_into_a_zero_row(case):
    ref, m, rel, _ = case
    dead = np.nonzero(np.all(ref == 0.0, axis=1))[0]
    assert dead.size > 0
    got = _bf16(ref)
    got[dead[0], 5] = 1e-9
    assert _rejects(got, ref, m, rel)


def test_one_token_vocabulary_cancellation_is_accepted():
    """V = 1: q = 1 and g = s/T ((a + b) - a - b) = 0 exactly; a float32
    kernel leaves rounding residue of the summands' size, which the bar
    admits, while a write into a row with a = b = 0 is still rejected."""
    X = np.zeros((3, 1))
    a = np.array([0.7, 0.0, 0.3])
    b = np.array([0.2, 0.0, 0.45])
    tok = np.array([0, -1, 0])
    m, rel = grad_bar.summand_magnitude(X, np.zeros(3), a, b, tok, tok, 1.0, 1.0)
    ref = np.zeros((3, 1))
    got = np.array([[6e-8], [0.0], [-3e-8]])
    e, r = grad_bar.violations(got, ref, m, rel, bf16=False)
    assert not e.any() and not r.any()
    got[1, 0] = 1e-9
    e, r = grad_bar.violations(got, ref, m, rel, bf16=False)
    assert e[1, 0] and r[1]
