"""Conformance of the oracle's Philox4x32-10 to an independent implementation
(CPU only).

The normative sampler draws its random words from Philox4x32 with ten rounds
(Salmon et al., SC'11).  The oracle implements the generator from that
definition; here its blocks are compared, word for word, with those of
rocRAND's engine (built from its header as a host program, `philox_ref.py`)
on edge counters and keys (all zeros, all ones, key words that wrap when the
Weyl increments are added) and on 4096 random ones.  A wrong multiplier,
Weyl constant, round count or output-word order changes every block.
"""
import numpy as np
import pytest

from oracle import sampler
from tests import philox_ref

pytestmark = pytest.mark.skipif(not philox_ref.available(), reason="hipcc or the rocRAND header is missing")

M32 = 0xFFFFFFFF


def _cases():
    edge_c = [(0, 0, 0, 0), (M32, M32, M32, M32), (1, 0, 0, 0), (0, 0, 0, 1), (0x243F6A88, 0x85A308D3, 0x13198A2E,
                                                                              0x03707344)]
    edge_k = [(0, 0), (M32, M32), (M32 - 0x9E3779B9 + 1, M32 - 0xBB67AE85 + 1), (0xA4093822, 0x299F31D0)]
    cs, ks = [], []
    for c in edge_c:
        for k in edge_k:
            cs.append(c)
            ks.append(k)
    rng = np.random.default_rng(2024)
    cs += [tuple(int(v) for v in rng.integers(0, 1 << 32, 4, dtype=np.uint64)) for _ in range(4096)]
    ks += [tuple(int(v) for v in rng.integers(0, 1 << 32, 2, dtype=np.uint64)) for _ in range(4096)]
    return np.array(cs, dtype=np.uint64), np.array(ks, dtype=np.uint64)


def oracle_blocks(S, counters, keys):
    out = np.empty_like(counters)
    for j, (c, k) in enumerate(zip(counters, keys)):
        seed = int(k[0]) | (int(k[1]) << 32)
        out[j] = [int(w) for w in S.philox4x32_10(*(int(v) for v in c), seed=seed)]
    return out


def test_oracle_philox_blocks_equal_rocrand_engine():
    counters, keys = _cases()
    ref = philox_ref.blocks(counters, keys)
    got = oracle_blocks(sampler, counters, keys)
    bad = np.nonzero(np.any(got != ref, axis=1))[0]
    assert bad.size == 0, f"{bad.size} blocks differ, first counter {counters[bad[0]]} key {keys[bad[0]]}"


def test_vectorised_counters_equal_scalar_calls():
    """The sampler calls the generator on arrays of counters (one per group
    of four vocabulary entries); the array form gives the scalar blocks."""
    counters, keys = _cases()
    seed = int(keys[7][0]) | (int(keys[7][1]) << 32)
    c = counters[:512]
    arr = np.stack(sampler.philox4x32_10(c[:, 0], c[:, 1], c[:, 2], c[:, 3], seed=seed), axis=1)
    ref = philox_ref.blocks(c, np.broadcast_to(keys[7], (512, 2)))
    assert np.array_equal(arr.astype(np.uint64), ref)
