"""Path scoring and M-step weights of the oracle, in float64 (test infrastructure).

One training position (prefix x) at a time, following the paper's order:

  row statistics     q = softmax(X/T_q), p = softmax(Y/T_p) (Sec. "Preliminary")
  acceptance         alpha_i = min(1, p/q), kept as log alpha (Eq. acc)
  survival           S_k = prod_{i<=k} alpha_i, kappa = S_l (Eqs. kappa,
                     survival_def); E[A|x,z] = sum_k S_k (Eq. accepted_len_cond)
  oracle gate        o = w(l) [log kappa(z) >= log kappa(z-bar)] (Alg. 2)
  correction         z = z~ if the gate passes, else z' (Alg. 1, E-step)
  ARW                beta (Eq. beta_update, leave-one-out)
  CAR                zeta (Eq. zeta_update, softmax at temperature tau)
  loss               Eq. advance (or Eq. basic when c = 0)
  gradient           d loss / d X from the loss written per row

Readings where the paper leaves a choice (each also listed in the design notes):
  * level l uses the length-l prefix of the depth-L path of slot s; the
    correction path is the length-l prefix of slot s's target path;
  * all three families at slot (s,i) read the same logit rows, unless each
    family's own context rows are given (exact context: X, Y with a leading
    family axis, the rows of the conditionals along z~, z' and z-bar);
  * the oracle's indicator in beta's numerator is the binary gate I~, o' keeps
    the weight w(l) (so w cancels and beta is a local acceptance rate);
  * beta = 0 when no other live path has o' > 0;
  * zeta's softmax runs over the paths alive at level l; Q is the path
    probability (product of tempered token probabilities) by default;
  * o', beta, zeta and the tokens are constants of the M-step (Theorem 3 fixes
    the E-step quantities during the update), so the gradient flows only
    through log q;
  * the loss of a position is divided by W = sum o' (0 when W = 0) and the
    batch loss is loss_scale times the sum over positions;
  * with a vocabulary map d2t, p(v) = p_target(d2t[v]) with the target softmax
    over the whole target vocabulary;
  * slot (s,i) exists iff i <= d_s (ragged depths); masked slots contribute
    nothing and their outputs are zero.
"""
import numpy as np

MODE_BASIC, MODE_ARW, MODE_ARW_CAR = 0, 1, 2
CAR_PROB, CAR_LOGPROB = 0, 1

DEFAULT_PARAMS = dict(temp_draft=1.0, temp_target=1.0, w_base=1.05, car_tau=0.2,
                      mode=MODE_ARW_CAR, car_input=CAR_PROB, loss_scale=1.0,
                      kl_weight=0.0, kl_topk=10)


def log_softmax_normaliser(logits, temperature):
    """log sum_v exp(logit_v / T) in float64 (max-shifted)."""
    z = np.asarray(logits, dtype=np.float64) / float(temperature)
    m = z.max(axis=-1, keepdims=True)
    return (m + np.log(np.exp(z - m).sum(axis=-1, keepdims=True)))[..., 0]


def length_weight(level, w_base):
    """w(l) = w_base^l, l = 1..L (the paper fixes w(l) = 1.05^l)."""
    return float(w_base) ** int(level)


def score_position(X, Y, d2t, depth, tok_d, tok_t, tok_g, params=None):
    """Score the N paths of one position.

    X      [N, L, V_d]  draft logits of each slot's row, or [3, N, L, V_d]:
                        the rows along each family's own path (z~, z', z-bar)
    Y      [N, L, V_t]  target logits of each slot's row, or [3, N, L, V_t]
    d2t    [V_d] int or None (identity)
    depth  [N]   valid depth d_s in [1, L]
    tok_*  [N, L] tokens of the three families (draft-index space; -1 masked)
    Returns a dict of float64 / bool arrays indexed [s, i-1] (rows) or [s];
    lse_q / lse_p are those of the z~ rows, and with per-family rows
    lse_q_ctx [N, L, 3] holds the draft normaliser of every family's row.
    """
    p = dict(DEFAULT_PARAMS)
    if params:
        p.update(params)
    X = np.asarray(X)
    Y = np.asarray(Y)
    ctx = X.ndim == 4
    if not ctx:  # one row per slot, read by every family
        X = X[None]
        Y = Y[None]
    N, L, Vd = X.shape[1:]
    d2t = np.arange(Vd) if d2t is None else np.asarray(d2t)
    depth = np.asarray(depth, dtype=np.int64)
    toks = [np.asarray(t, dtype=np.int64) for t in (tok_d, tok_t, tok_g)]
    Tq, Tp = float(p["temp_draft"]), float(p["temp_target"])
    live = np.arange(L)[None, :] < depth[:, None]          # [N, L]

    # Row statistics and per-token log probabilities (Sec. "Preliminary"),
    # family f on its own row (row set f, or the shared one).
    nrow = X.shape[0]
    lse_q = np.zeros((nrow, N, L))
    lse_p = np.zeros((nrow, N, L))
    log_q = np.zeros((3, N, L))
    log_ratio = np.zeros((3, N, L))
    for s in range(N):
        for i in range(depth[s]):
            for k in range(nrow):
                lse_q[k, s, i] = log_softmax_normaliser(X[k, s, i], Tq)
                lse_p[k, s, i] = log_softmax_normaliser(Y[k, s, i], Tp)
            for f in range(3):
                k = f if ctx else 0
                z = toks[f][s, i]
                x, y = float(X[k, s, i, z]), float(Y[k, s, i, d2t[z]])
                log_q[f, s, i] = x / Tq - lse_q[k, s, i]
                # log p - log q, grouped as (y/T_p - x/T_q) - (lse_p - lse_q):
                # tokens of one row with equal y/T_p - x/T_q (common with
                # bf16 logits) then get bitwise equal values, so the gate
                # below sees their exact tie (equality accepts)
                log_ratio[f, s, i] = (y / Tp - x / Tq) - (lse_p[k, s, i] - lse_q[k, s, i])
    # Eq. acc: alpha = min(1, p/q)  <=>  log alpha = min(0, log p - log q).
    log_alpha = np.where(live[None], np.minimum(0.0, log_ratio), 0.0)

    # Prefix sums over depth: log S_k (Eq. survival_def) and log-likelihoods.
    LS = np.zeros((3, N, L))
    LQ = np.zeros((3, N, L))
    for s in range(N):
        acc = np.zeros(3)
        accq = np.zeros(3)
        for i in range(depth[s]):
            acc = acc + log_alpha[:, s, i]
            accq = accq + log_q[:, s, i]
            LS[:, s, i] = acc
            LQ[:, s, i] = accq
    survival = np.where(live, np.exp(LS[0]), 0.0)            # S_k of z~
    exp_accept_len = survival.sum(axis=1)                     # Eq. accepted_len_cond

    # Alg. 2 gate and Alg. 1 correction, for each level l = i (1-based i+1).
    acc_flag = np.zeros((N, L), dtype=bool)   # I~ : oracle passes z~
    val_flag = np.zeros((N, L), dtype=bool)   # I' : oracle passes the used path z
    o_prime = np.zeros((N, L))
    for s in range(N):
        for i in range(depth[s]):
            acc_flag[s, i] = LS[0, s, i] >= LS[2, s, i]
            corrected_ok = LS[1, s, i] >= LS[2, s, i]
            val_flag[s, i] = acc_flag[s, i] or corrected_ok
            o_prime[s, i] = length_weight(i + 1, p["w_base"]) * val_flag[s, i]

    # ARW (Eq. beta_update) and CAR (Eq. zeta_update), per level over live paths.
    beta = np.zeros((N, L))
    zeta = np.zeros((N, L))
    for i in range(L):
        alive = [s for s in range(N) if live[s, i]]
        if not alive:
            continue
        for s in alive:
            num = sum(o_prime[j, i] * acc_flag[j, i] for j in alive if j != s)
            den = sum(o_prime[j, i] for j in alive if j != s)
            beta[s, i] = num / den if den > 0 else 0.0
        if p["car_input"] == CAR_PROB:
            conf = np.array([np.exp(LQ[0, s, i]) for s in alive])   # path probability
        else:
            conf = np.array([LQ[0, s, i] for s in alive])           # its logarithm
        e = np.exp((conf - conf.max()) / float(p["car_tau"]))
        for k, s in enumerate(alive):
            zeta[s, i] = e[k] / e.sum()
    if p["mode"] == MODE_ARW_CAR:
        c = beta * zeta
    elif p["mode"] == MODE_ARW:
        c = beta.copy()
    else:
        c = np.zeros_like(beta)

    # Eq. advance: L_x = -(1/W) sum_{l,s} o' [log q(z) - c log q(z~)].
    W = o_prime.sum()
    loss = 0.0
    if W > 0:
        total = 0.0
        for s in range(N):
            for i in range(depth[s]):
                lq_used = LQ[0, s, i] if acc_flag[s, i] else LQ[1, s, i]
                total += o_prime[s, i] * (lq_used - c[s, i] * LQ[0, s, i])
        loss = -total / W

    # The same loss per row: L_x = -sum_{s,i} [a log q(z~_i) + b log q(z'_i)],
    # a_{s,i} = (1/W) sum_{l>=i} o'(I~ - c), b_{s,i} = (1/W) sum_{l>=i} o'(1 - I~).
    coef_a = np.zeros((N, L))
    coef_b = np.zeros((N, L))
    if W > 0:
        for s in range(N):
            for i in range(depth[s]):
                for lev in range(i, depth[s]):
                    coef_a[s, i] += o_prime[s, lev] * (acc_flag[s, lev] - c[s, lev])
                    coef_b[s, i] += o_prime[s, lev] * (1.0 - acc_flag[s, lev])
        coef_a /= W
        coef_b /= W

    out = {}
    if ctx:
        out["lse_q_ctx"] = np.moveaxis(np.where(live[None], lse_q, 0.0), 0, -1)
    return dict(out, lse_q=np.where(live, lse_q[0], 0.0), lse_p=np.where(live, lse_p[0], 0.0),
                log_alpha=np.moveaxis(log_alpha, 0, -1),
                log_q=np.moveaxis(np.where(live[None], log_q, 0.0), 0, -1),
                survival=survival, exp_accept_len=exp_accept_len,
                accept_flag=acc_flag, valid_flag=val_flag, o_prime=o_prime,
                beta=np.where(live, beta, 0.0), zeta=np.where(live, zeta, 0.0),
                c=np.where(live, c, 0.0), W=W, loss=loss,
                coef_a=coef_a, coef_b=coef_b, LS=np.moveaxis(LS, 0, -1))


def grad_position(X, lse_q, tok_d, tok_t, coef_a, coef_b, temp_draft=1.0, loss_scale=1.0):
    """d(loss_scale * L_x)/dX for every row of one position, float64 [N, L, V_d].

    Per row, d(-log q(z))/dX_v = (q(v) - [v = z]) / T_q, so with the row's
    coefficients a (for z~) and b (for z'):
      g_v = loss_scale / T_q * ((a + b) q(v) - a [v = z~] - b [v = z']).
    With per-family rows z~ and z' sit on different rows: the gradient on the
    z~ rows is this with b = 0, on the z' rows with a = 0 (grad_position_ctx).
    """
    X = np.asarray(X, dtype=np.float64)
    N, L, Vd = X.shape
    g = np.zeros((N, L, Vd))
    for s in range(N):
        for i in range(L):
            a, b = coef_a[s, i], coef_b[s, i]
            if a == 0.0 and b == 0.0:
                continue
            q = np.exp(X[s, i] / temp_draft - lse_q[s, i])
            row = (a + b) * q
            row[tok_d[s, i]] -= a
            row[tok_t[s, i]] -= b
            g[s, i] = loss_scale / temp_draft * row
    return g


def grad_position_ctx(X_draft_path, X_corr_path, lse_draft_path, lse_corr_path, tok_d, tok_t, coef_a, coef_b,
                      temp_draft=1.0, loss_scale=1.0):
    """Gradients with per-family rows: (d/dX along z~, d/dX along z'), each
    [N, L, V_d]; the rows along z-bar only gate and get none."""
    zero = np.zeros_like(np.asarray(coef_a, dtype=np.float64))
    g_d = grad_position(X_draft_path, lse_draft_path, tok_d, tok_t, coef_a, zero, temp_draft, loss_scale)
    g_c = grad_position(X_corr_path, lse_corr_path, tok_d, tok_t, zero, coef_b, temp_draft, loss_scale)
    return g_d, g_c


def loss_from_logits(X, Y, d2t, depth, tok_d, tok_t, tok_g, frozen, params=None):
    """L_x recomputed from logits with the E-step quantities (flags, o', c) frozen.

    Used by the finite-difference pin: the derivative of this function with
    respect to X must equal grad_position (the M-step treats o', beta, zeta
    and the tokens as constants).
    """
    p = dict(DEFAULT_PARAMS)
    if params:
        p.update(params)
    X = np.asarray(X, dtype=np.float64)
    Xd, Xc = (X[0], X[1]) if X.ndim == 4 else (X, X)   # rows along z~ and along z'
    N, L, Vd = Xd.shape
    Tq = float(p["temp_draft"])
    W = frozen["o_prime"].sum()
    if W == 0:
        return 0.0
    total = 0.0
    for s in range(N):
        lq_d = 0.0
        lq_t = 0.0
        for i in range(depth[s]):
            lq_d += Xd[s, i, tok_d[s, i]] / Tq - log_softmax_normaliser(Xd[s, i], Tq)
            lq_t += Xc[s, i, tok_t[s, i]] / Tq - log_softmax_normaliser(Xc[s, i], Tq)
            used = lq_d if frozen["accept_flag"][s, i] else lq_t
            total += frozen["o_prime"][s, i] * (used - frozen["c"][s, i] * lq_d)
    return -total / W


def loss_with_klv(X, Y, d2t, depth, tok_d, tok_t, tok_g, frozen, params=None):
    """loss_from_logits plus kl_weight times the position's top-K term
    (oracle.klv), the E-step quantities frozen; its derivative with respect to
    X is what grad_position plus the KL rows give."""
    from . import klv
    p = dict(DEFAULT_PARAMS)
    if params:
        p.update(params)
    base = loss_from_logits(X, Y, d2t, depth, tok_d, tok_t, tok_g, frozen, p)
    if p["kl_weight"] == 0.0:
        return base
    if np.ndim(X) == 4:  # per-family rows: the term is taken on the rows along z~
        X, Y = X[0], Y[0]
    KL = klv.position_terms(X, Y, d2t, depth, int(p["kl_topk"]), p["temp_draft"], p["temp_target"])[3]
    return base + p["kl_weight"] * KL
