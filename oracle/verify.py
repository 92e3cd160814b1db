"""Decode-time verification of draft paths (test infrastructure; see the
package header).

Speculative decoding checks a draft path token by token (Sec. "Preliminary",
Eq. acc): the draft token z_i, drawn from q, is kept with probability
alpha_i = min(1, p(z_i) / q(z_i)); at the first rejection a replacement is
drawn from the residual distribution norm(max(0, p - q)) and the path ends.
The number of kept tokens is the accepted length whose conditional mean given
the path is sum_k S_k (Eq. accepted_len_cond); no bonus token is drawn after a
fully kept path (there is no row for it).  With a vocabulary map the residual
runs over the whole target vocabulary: q(t) = q(v) for t = d2t[v] and 0 for
target tokens the draft cannot propose.

Random numbers follow the library's sampler definition (oracle.sampler):
  * the acceptance uniform of slot r is u from word 0 of Philox counter
    (0, r, 2, offset); the token is kept iff Lambda(u) < log alpha, with
    Lambda the normative float32 logarithm (u < alpha up to its rounding);
  * the residual draw at slot r is the Gumbel-max of log(max(0, p - q)) over
    target indices t, G_t from Philox counter (t >> 2, r, 3, offset), word
    t & 3; entries with p <= q never win.
"""
import numpy as np

from . import paths, sampler

FAMILY_ACCEPT = 2
FAMILY_RESIDUAL = 3


def acceptance_log_uniform(rows, seed, offset):
    """Lambda(u) (float32) of the acceptance uniform of each row."""
    w = sampler.random_words(np.asarray(rows), FAMILY_ACCEPT, 1, seed, offset)[:, 0]
    return sampler.spec_log(sampler.uniform_from_word(w))


def residual_draw(x, y, d2t, lse_q, lse_p, row, temp_draft, temp_target, seed, offset):
    """(token, key gap) of the residual draw of one row: x [V_d] draft logits,
    y [V_t] target logits.  The gap between the two largest keys tells how
    close the draw was to a tie."""
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    Vd, Vt = x.size, y.size
    d2t = np.arange(Vd) if d2t is None else np.asarray(d2t, dtype=np.int64)
    p = np.exp(y / temp_target - lse_p)
    q = np.zeros(Vt)
    q[d2t] = np.exp(x / temp_draft - lse_q)
    res = np.maximum(0.0, p - q)
    g = sampler.gumbel_from_word(sampler.random_words([row], FAMILY_RESIDUAL, Vt, seed, offset)[0])
    with np.errstate(divide="ignore"):
        keys = np.where(res > 0.0, np.log(res) + g.astype(np.float64), -np.inf)
    top = int(np.argmax(keys))
    second = np.max(np.delete(keys, top)) if Vt > 1 else -np.inf
    return top, keys[top] - second


def verify_position(X, Y, d2t, depth, tok_d, first_row, temp_draft=1.0, temp_target=1.0, seed=0, offset=0):
    """Verify the N draft paths of one position.

    X [N, L, V_d], Y [N, L, V_t], depth [N], tok_d [N, L] (the draft path),
    first_row = global row of slot (0, 1).  Returns accept_len [N] int,
    resample_tok [N] int (target index; -1 when every token was kept), the
    margin |Lambda(u) - log alpha| of each path's deciding comparisons (the
    smallest over its tested slots) and the residual's key gap (inf if none).
    """
    X = np.asarray(X, dtype=np.float64)
    Y = np.asarray(Y, dtype=np.float64)
    N, L, Vd = X.shape
    d2t_arr = np.arange(Vd) if d2t is None else np.asarray(d2t, dtype=np.int64)
    accept = np.zeros(N, dtype=np.int64)
    resample = np.full(N, -1, dtype=np.int64)
    margin = np.full(N, np.inf)
    gap = np.full(N, np.inf)
    for s in range(N):
        for i in range(int(depth[s])):
            r = first_row + s * L + i
            lse_q = paths.log_softmax_normaliser(X[s, i], temp_draft)
            lse_p = paths.log_softmax_normaliser(Y[s, i], temp_target)
            z = int(tok_d[s, i])
            log_alpha = min(0.0, (Y[s, i, d2t_arr[z]] / temp_target - lse_p) - (X[s, i, z] / temp_draft - lse_q))
            lu = float(acceptance_log_uniform([r], seed, offset)[0])
            margin[s] = min(margin[s], abs(lu - log_alpha))
            if lu < log_alpha:
                accept[s] += 1
                continue
            resample[s], gap[s] = residual_draw(X[s, i], Y[s, i], d2t, lse_q, lse_p, r, temp_draft, temp_target,
                                                seed, offset)
            break
    return accept, resample, margin, gap
