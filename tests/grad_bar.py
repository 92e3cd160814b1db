"""The gradient parity bar (test infrastructure, plain numpy: no GPU needed).

The gradient of the weighted log-likelihood with respect to the draft logits
(derivative of Eq. advance) is, per row r and vocabulary index v,

    g[v] = s/T (c q(v) - a [v = z~] - b [v = z'])  (+ the top-K KL term's
                                                     sparse part, Eq. klv)

with c = a + b, q = softmax(X/T) and s the loss scale.  Three bounds hold for
a correct kernel and are checked element by element or row by row:

1. The benchmark spec's absolute bar: |got - ref| <= 2e-3.
2. An element bound from the arithmetic.  The kernel forms q(v) in float32
   from exp of (X[v]/T - lse); the exponent's argument carries rounding
   errors of a few float32 ulps of |X[v]/T| + |lse|, so q(v), and every term
   built from it, has a relative error below
       rel(v) = 16 * 2^-24 * (|X[v]/T| + |lse|) + 1e-5,
   and the float32 gradient differs from the exact one by at most rel(v)
   times the magnitude of its summands,
       m(v) = |s|/T ((|a| + |b| + 1e-6) q(v) + |a| [v = z~] + |b| [v = z'])
              + |s| lambda / (N T) * 2 [v in Omega]
   (1e-6: the coefficients' own float32 error; the KL part's q_hat and
   p_hat are at most 1).  A bf16 output then adds its round-to-nearest-even
   error, at most 2^-8 of the value:
       |got - ref| <= 2^-8 |ref| + (1 + 2^-8) rel(v) m(v) + 1e-37
   (1e-37: float32 values below the normal range may be flushed to zero).
   Unlike the absolute bar this reaches the ~1e-8 entries that make up
   almost all of a 32k-128k row.
3. A per-row L2 bound: ||got - ref|| <= 1e-2 ||ref|| + (1 + 2^-8) ||rel m||.
   The second term is the summands' float32 error of bound 2: it matters
   only in rows whose gradient is a cancellation, e.g. a peaked row whose
   draft token holds nearly all of q, where g[z~] = s/T a (q(z~) - 1) and
   every other entry is tiny, or a one-token vocabulary, where g = 0
   exactly.  Rows with a = b = 0 (masked slots among them) keep only the
   1e-6 q part of m, so they must be written as zeros to within ~1e-11.
"""
import numpy as np

ABS_BAR = 2e-3
ROW_REL_L2 = 1e-2
BF16_REL = 2.0 ** -8
FLUSH_FLOOR = 1e-37


def summand_magnitude(X, lse, coef_a, coef_b, tok_draft, tok_target, temp, loss_scale,
                      kl_idx=None, kl_weight=0.0, n_paths=1):
    """m(v) and rel(v) of the element bound for rows X [n, V] (float64
    arrays from the oracle's inputs and outputs; tokens -1 on masked rows).
    Returns (m, rel), both [n, V]."""
    X = np.asarray(X, dtype=np.float64)
    lse = np.asarray(lse, dtype=np.float64)[:, None]
    a = np.asarray(coef_a, dtype=np.float64)[:, None]
    b = np.asarray(coef_b, dtype=np.float64)[:, None]
    inv_t = 1.0 / float(temp)
    arg = X * inv_t - lse
    with np.errstate(over="ignore", invalid="ignore"):
        q = np.where(np.isfinite(arg), np.exp(np.minimum(arg, 0.0)), 0.0)
    s = abs(float(loss_scale)) * inv_t
    m = s * (np.abs(a) + np.abs(b) + 1e-6) * q
    rows = np.arange(X.shape[0])
    for tok, coef in ((tok_draft, a[:, 0]), (tok_target, b[:, 0])):
        tok = np.asarray(tok)
        live = tok >= 0
        m[rows[live], tok[live]] += s * np.abs(coef[live])
    if kl_idx is not None and kl_weight > 0.0:
        kl_idx = np.asarray(kl_idx)
        r, k = np.nonzero(kl_idx >= 0)
        m[r, kl_idx[r, k]] += 2.0 * s * float(kl_weight) / float(n_paths)
    with np.errstate(invalid="ignore"):
        mag_arg = np.where(np.isfinite(X), np.abs(X * inv_t), 0.0) + np.abs(lse)
    rel = 16.0 * 2.0 ** -24 * mag_arg + 1e-5
    return m, rel


def violations(got, ref, m, rel, bf16):
    """Boolean [n, V] mask of elements outside bounds 1 and 2, and the [n]
    mask of rows outside bound 3."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    err = np.abs(got - ref)
    tol = (1.0 + BF16_REL) * rel * m + FLUSH_FLOOR
    if bf16:
        tol = tol + BF16_REL * np.abs(ref)
    bad_elem = (err > ABS_BAR) | (err > tol) | ~np.isfinite(got)
    nref = np.sqrt(np.sum(ref * ref, axis=1))
    nerr = np.sqrt(np.sum(err * err, axis=1))
    f32 = (1.0 + BF16_REL) * rel * m
    nf32 = np.sqrt(np.sum(f32 * f32, axis=1))
    bad_row = nerr > ROW_REL_L2 * nref + nf32
    return bad_elem, bad_row


def margin_used(got, ref, m, rel, bf16):
    """Largest fraction of the element bound used (diagnostic)."""
    err = np.abs(np.asarray(got, dtype=np.float64) - np.asarray(ref, dtype=np.float64))
    tol = (1.0 + BF16_REL) * rel * m + FLUSH_FLOOR
    if bf16:
        tol = tol + BF16_REL * np.abs(ref)
    return float(np.max(err / tol)) if err.size else 0.0
