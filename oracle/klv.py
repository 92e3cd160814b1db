"""Top-K renormalised KL term of the VSD (KL) variant (test infrastructure;
see the package header).

The paper's KL variant replaces the divergence term of its objective with a
token-level distillation loss over the K tokens the target model finds most
likely (Appendix on the MLLM experiments, Eq. klv).  Per row, with the target
logits over the mapped draft vocabulary y_v = Y[d2t[v]] and the draft logits
x_v:

  Omega     = the K draft indices with the largest y_v (equal values: the
              smaller index first), among those with a finite y_v: a token
              of zero target probability (y_v = -inf, a masked vocabulary
              entry) is not one of the target's likely tokens, so a row with
              fewer than K finite mapped logits has fewer than K members
              (none: the row's term is 0)
  p_hat(v)  = exp(y_v / T_p) / sum_{u in Omega} exp(y_u / T_p)
  q_hat(v)  = exp(x_v / T_q) / sum_{u in Omega} exp(x_u / T_q)
  L_topK    = - sum_{v in Omega} p_hat(v) log q_hat(v)

and its derivative with respect to the draft logits is (q_hat - p_hat) / T_q
on Omega (p_hat sums to one) and zero elsewhere.  Per position the term is
averaged over the N sampled paths and summed over their live slots,
KL_x = (1/N) sum_{live (s, i)} L_topK(s, i): by the chain rule the path-level
divergence is the expected sum of the per-step ones, estimated over the N
paths; the E-step draws are held fixed, as for the rest of the M-step.
"""
import numpy as np


def topk_set(y, K):
    """Indices of the K largest finite entries of y (fewer if y has fewer),
    largest first, equal values in increasing index order."""
    y = np.asarray(y, dtype=np.float64)
    order = np.lexsort((np.arange(y.size), -y))
    order = order[np.isfinite(y[order])]
    return order[:K]


def row_term(x, y_mapped, K, temp_draft=1.0, temp_target=1.0):
    """(omega, p_hat, q_hat, L) of one row; x, y_mapped over the draft vocabulary."""
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y_mapped, dtype=np.float64)
    omega = topk_set(y, K)
    if omega.size == 0:
        return omega, np.zeros(0), np.zeros(0), 0.0
    a = y[omega] / temp_target
    p_hat = np.exp(a - a.max())
    p_hat /= p_hat.sum()
    b = x[omega] / temp_draft
    log_q_hat = b - (b.max() + np.log(np.exp(b - b.max()).sum()))
    L = -np.sum(p_hat * log_q_hat)
    return omega, p_hat, np.exp(log_q_hat), L


def position_terms(X, Y, d2t, depth, K, temp_draft=1.0, temp_target=1.0):
    """Per-slot terms of one position: X [N, L, V_d], Y [N, L, V_t].

    Returns L_row [N, L] (0 on masked slots), omega [N, L, K] (-1 on masked
    slots and past the members of a smaller set), dLrow_dx [N, L, K] =
    (q_hat - p_hat) / T_q on omega (0 past the members), and KL_x."""
    X = np.asarray(X, dtype=np.float64)
    Y = np.asarray(Y, dtype=np.float64)
    N, L, Vd = X.shape
    d2t_arr = np.arange(Vd) if d2t is None else np.asarray(d2t, dtype=np.int64)
    L_row = np.zeros((N, L))
    omega = np.full((N, L, K), -1, dtype=np.int64)
    dx = np.zeros((N, L, K))
    for s in range(N):
        for i in range(int(depth[s])):
            om, p_hat, q_hat, Lr = row_term(X[s, i], Y[s, i][d2t_arr], K, temp_draft, temp_target)
            L_row[s, i] = Lr
            omega[s, i, :om.size] = om
            dx[s, i, :om.size] = (q_hat - p_hat) / temp_draft
    return L_row, omega, dx, L_row.sum() / N
