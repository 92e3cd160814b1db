"""E-step sampler of the oracle (test infrastructure; see the package header).

The paper draws z~ ~ q_psi and z' ~ p_theta (Alg. 1, E-step) and the greedy
reference z-bar from the greedy target policy (Alg. 2), but names no sampler.
This module implements, from its written definition, the library's normative
sampler: Philox4x32-10 counter-based random words (Salmon et al., SC'11), a
uniform on a 2^-24 grid, a Gumbel variate through a fixed float32 logarithm,
and the Gumbel-max rule (argmax of logit/T + G samples softmax(logit/T)).

Every floating-point step is a separate float32 numpy operation, so each is
rounded to nearest-even exactly once, as the definition requires.
"""
import numpy as np

F32 = np.float32

# Philox4x32 constants (SC'11): round multipliers and Weyl key increments.
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
_MASK32 = 0xFFFFFFFF


def philox4x32_10(c0, c1, c2, c3, seed):
    """Philox4x32 with 10 rounds on counter (c0,c1,c2,c3), key from `seed`.

    Counters are integer arrays (broadcast together); the key is
    (low 32 bits, high 32 bits) of the 64-bit seed.  Round j (0-based) uses
    key (k0 + j*W0, k1 + j*W1) mod 2^32 and maps (c0,c1,c2,c3) to
    (hi(M1*c2)^c1^k0, lo(M1*c2), hi(M0*c0)^c3^k1, lo(M0*c0)).
    Returns four uint32 arrays.
    """
    c0, c1, c2, c3 = np.broadcast_arrays(*(np.asarray(c, dtype=np.uint64) for c in (c0, c1, c2, c3)))
    x0, x1, x2, x3 = (c & np.uint64(_MASK32) for c in (c0, c1, c2, c3))
    seed = int(seed)
    k0, k1 = seed & _MASK32, (seed >> 32) & _MASK32
    m0, m1 = np.uint64(PHILOX_M0), np.uint64(PHILOX_M1)
    for j in range(10):
        rk0 = np.uint64((k0 + j * PHILOX_W0) & _MASK32)
        rk1 = np.uint64((k1 + j * PHILOX_W1) & _MASK32)
        p0 = m0 * x0  # both factors < 2^32: the 64-bit product is exact
        p1 = m1 * x2
        hi0, lo0 = p0 >> np.uint64(32), p0 & np.uint64(_MASK32)
        hi1, lo1 = p1 >> np.uint64(32), p1 & np.uint64(_MASK32)
        x0, x1, x2, x3 = hi1 ^ x1 ^ rk0, lo1, hi0 ^ x3 ^ rk1, lo0
    return tuple(x.astype(np.uint32) for x in (x0, x1, x2, x3))


def uniform_from_word(w):
    """u = float(2*(w >> 9) + 1) * 2^-24: 2^23 equally spaced values in (0,1)."""
    k = (np.asarray(w, dtype=np.uint32) >> np.uint32(9)).astype(np.int64)
    return (2 * k + 1).astype(F32) * F32(2.0 ** -24)


# Constants of the normative logarithm, each the float32 nearest its value.
_SQRT2 = np.uint32(0x3FB504F3).view(F32)
_C9 = F32(1.0 / 9.0)
_C7 = F32(1.0 / 7.0)
_C5 = F32(1.0 / 5.0)
_C3 = F32(1.0 / 3.0)
_LN2_HI = np.uint32(0x3F317200).view(F32)
_LN2_LO = np.uint32(0x35BFBE8E).view(F32)


def spec_log(x):
    """The normative float32 natural logarithm of positive normal floats.

    x = 2^e * m with m in (sqrt(1/2), sqrt(2)]; log m = 2 atanh(s) with
    s = (m-1)/(m+1) = f/(2+f), summed as 2s + 2s*z*(1/3 + z/5 + z^2/7 + z^3/9),
    z = s^2 (Horner, one rounding per operation); log x = e*ln2 + log m with
    ln2 split into an exact-product high part and a low part.
    """
    x = np.asarray(x, dtype=F32)
    assert np.all(np.isfinite(x)) and np.all(x >= np.finfo(F32).tiny), "normal positive inputs only"
    bits = x.view(np.uint32)
    e = ((bits >> np.uint32(23)) & np.uint32(0xFF)).astype(np.int32) - 127
    m = ((bits & np.uint32(0x7FFFFF)) | np.uint32(0x3F800000)).view(F32)
    big = m > _SQRT2
    m = np.where(big, m * F32(0.5), m).astype(F32)
    e = e + big.astype(np.int32)
    f = m - F32(1.0)
    s = f / (F32(2.0) + f)
    z = s * s
    p = np.full_like(z, _C9)
    p = _C7 + z * p
    p = _C5 + z * p
    p = _C3 + z * p
    t2 = s + s
    lm = t2 + t2 * (z * p)
    ef = e.astype(F32)
    out = ef * _LN2_HI + (lm + ef * _LN2_LO)
    assert out.dtype == F32
    return out


def gumbel_from_word(w):
    """G = -Lambda(-Lambda(u)) for the uniform u of word w (float32)."""
    u = uniform_from_word(w)
    e = -spec_log(u)
    return -spec_log(e)


def random_words(rows, family, n_vocab, seed, offset):
    """Philox word for every (row, vocabulary index) pair: counter
    (v >> 2, row, family, offset), word v & 3.  Returns uint32 [len(rows), n_vocab]."""
    rows = np.asarray(rows, dtype=np.uint64).reshape(-1, 1)
    n_calls = (n_vocab + 3) // 4
    c0 = np.arange(n_calls, dtype=np.uint64).reshape(1, -1)
    words = philox4x32_10(c0, rows, np.uint64(family), np.uint64(offset), seed)
    stacked = np.stack(words, axis=-1).reshape(rows.shape[0], 4 * n_calls)
    return stacked[:, :n_vocab]


def gumbel_keys(logits, rows, family, temperature, seed, offset):
    """key[v] = float32(logit[v] * float32(1/T)) + G[v]  (float32, [nrows, V])."""
    logits = np.asarray(logits, dtype=F32)
    inv_t = F32(1.0) / F32(temperature)
    g = gumbel_from_word(random_words(rows, family, logits.shape[1], seed, offset))
    keys = logits * inv_t + g
    assert keys.dtype == F32
    return keys


def first_argmax(a):
    """Index of the largest entry of each row; ties go to the smallest index."""
    return np.argmax(a, axis=1).astype(np.int64)


def sample_rows(draft_rows, target_rows_mapped, rows, temp_draft, temp_target, seed, offset):
    """Draw (z~, z', z-bar) for a set of rows.

    draft_rows          [n, V_d]  exact draft logits X_r
    target_rows_mapped  [n, V_d]  target logits at the mapped indices Y_r[d2t[v]]
    rows                [n]       global row indices (Philox counter word 1)
    """
    k_draft = gumbel_keys(draft_rows, rows, 0, temp_draft, seed, offset)
    k_target = gumbel_keys(target_rows_mapped, rows, 1, temp_target, seed, offset)
    return (first_argmax(k_draft), first_argmax(k_target),
            first_argmax(np.asarray(target_rows_mapped, dtype=np.float64)))


def sample_rows_ctx(draft_rows, target_rows_mapped, greedy_rows_mapped, rows, temp_draft, temp_target, seed, offset):
    """Draw (z~, z', z-bar) when each family has its own rows (exact context):
    z~ from the draft rows along z~, z' from the target rows along z', z-bar
    the first argmax of the target rows along z-bar.  The Philox counters are
    those of sample_rows, so equal rows give equal tokens."""
    k_draft = gumbel_keys(draft_rows, rows, 0, temp_draft, seed, offset)
    k_target = gumbel_keys(target_rows_mapped, rows, 1, temp_target, seed, offset)
    return (first_argmax(k_draft), first_argmax(k_target),
            first_argmax(np.asarray(greedy_rows_mapped, dtype=np.float64)))
