"""Seeded generators for the workload recipes in configs.py.

Device-side generation uses torch.Generator(device).manual_seed(cfg.seed) with a
fixed call order, so the same config, device type and torch version always give
the same tensors.  C1 also has a pure-numpy generator (PCG64, seed 0) so CPU
tests can use it without torch.

Logit arrays are [R, ld] with ld = v rounded up to a 16-byte multiple; the
padding columns [v, ld) hold PAD_VALUE, a large finite logit that would
visibly corrupt any softmax or argmax that wrongly read it.
"""
import math

import numpy as np
import torch

PAD_VALUE = 30000.0


def _dtype(cfg):
    return torch.float32 if cfg.dtype == "f32" else torch.bfloat16


def positions_rows(cfg, positions):
    """Row indices (int64 numpy) of all N*L rows of the given positions."""
    positions = np.asarray(positions, dtype=np.int64)
    per = cfg.N * cfg.L
    return (positions[:, None] * per + np.arange(per)[None, :]).reshape(-1)


def _padded(cfg, values, v, device):
    """Place [R, v] values into an [R, ld] array of the config's dtype."""
    ld = cfg.ld(v)
    if ld == v:
        return values.to(_dtype(cfg)).contiguous()
    out = torch.full((values.shape[0], ld), PAD_VALUE, dtype=_dtype(cfg), device=device)
    out[:, :v] = values.to(_dtype(cfg))
    return out


def _draft_map(cfg):
    """Injective, ascending draft->target map: the first v_draft entries of a
    seeded permutation of the target vocabulary, sorted."""
    g = torch.Generator(device="cpu").manual_seed(cfg.seed * 7919 + 1)
    perm = torch.randperm(cfg.v_target, generator=g)
    return torch.sort(perm[: cfg.v_draft]).values.to(torch.int32)


def _peaked_scale(g_rows, top1, iters=60):
    """Per-row c > 0 with max_v softmax(c * g)_v = top1 (bisection in float64)."""
    g = g_rows.double()
    gap = g - g.max(dim=1, keepdim=True).values          # <= 0
    lo = torch.zeros(g.shape[0], 1, dtype=torch.float64, device=g.device)
    hi = torch.full_like(lo, 4096.0)
    target = top1.double().view(-1, 1)
    for _ in range(iters):
        mid = 0.5 * (lo + hi)
        pmax = 1.0 / torch.exp(mid * gap).sum(dim=1, keepdim=True)
        too_low = pmax < target
        lo = torch.where(too_low, mid, lo)
        hi = torch.where(too_low, hi, mid)
    return 0.5 * (lo + hi)


def make_inputs(cfg, device="cuda", chunk_rows=8192):
    """Generate every input array of `cfg` on `device`.

    Returns a dict with X [R, ld_d], Y [R, ld_t] (absent for the fused recipe),
    d2t [v_draft] int32 or None, valid_depth [B, T, N] int32 or None, and for
    the fused recipe Hd, Ht [R, H] and Wd [v_draft, H], Wt [v_target, H].
    """
    dev = torch.device(device)
    gen = torch.Generator(device=dev).manual_seed(cfg.seed)
    R, Vd, Vt = cfg.R, cfg.v_draft, cfg.v_target
    out = {"d2t": None, "valid_depth": None}
    if cfg.mapped:
        out["d2t"] = _draft_map(cfg).to(dev)
    if cfg.ragged:
        out["valid_depth"] = torch.randint(1, cfg.L + 1, (cfg.B, cfg.T, cfg.N), generator=gen,
                                           device=dev, dtype=torch.int64).to(torch.int32)

    if cfg.kind == "fused":
        H = cfg.hidden
        bf = torch.bfloat16
        out["Hd"] = torch.randn(R, H, generator=gen, device=dev, dtype=torch.float32).to(bf)
        out["Ht"] = torch.randn(R, H, generator=gen, device=dev, dtype=torch.float32).to(bf)
        out["Wd"] = (cfg.w_std * torch.randn(Vd, H, generator=gen, device=dev)).to(bf)
        out["Wt"] = (cfg.w_std * torch.randn(Vt, H, generator=gen, device=dev)).to(bf)
        return out

    X = torch.empty(R, cfg.ld(Vd), dtype=_dtype(cfg), device=dev)
    Y = torch.empty(R, cfg.ld(Vt), dtype=_dtype(cfg), device=dev)
    if cfg.ld(Vd) != Vd:
        X[:, Vd:] = PAD_VALUE
    if cfg.ld(Vt) != Vt:
        Y[:, Vt:] = PAD_VALUE
    d2t_long = out["d2t"].long() if cfg.mapped else None
    for r0 in range(0, R, chunk_rows):
        r1 = min(R, r0 + chunk_rows)
        n = r1 - r0
        if cfg.kind == "gauss_shared":            # C1 recipe
            x = 2.0 * torch.randn(n, Vd, generator=gen, device=dev)
            y = x + torch.randn(n, Vd, generator=gen, device=dev)
        elif cfg.kind == "gauss_corr":            # C2 recipe
            y = 3.0 * torch.randn(n, Vt, generator=gen, device=dev)
            y = y.to(_dtype(cfg)).float()
            x = 0.8 * y + 1.5 * torch.randn(n, Vd, generator=gen, device=dev)
        elif cfg.kind == "mapped_corr":           # C3 recipe
            y = 3.0 * torch.randn(n, Vt, generator=gen, device=dev)
            y = y.to(_dtype(cfg)).float()
            ym = y[:, d2t_long] if d2t_long is not None else y
            x = 0.7 * ym + math.sqrt(0.51) * 3.0 * torch.randn(n, Vd, generator=gen, device=dev)
        elif cfg.kind == "peaked_ragged":         # C4 recipe
            g = torch.randn(n, Vt, generator=gen, device=dev)
            top1 = 0.85 + 0.14 * torch.rand(n, generator=gen, device=dev)
            c = _peaked_scale(g, top1).float()
            y = (c * g).to(_dtype(cfg)).float()
            x = 0.8 * y + 1.5 * torch.randn(n, Vd, generator=gen, device=dev)
        else:
            raise ValueError(f"unknown recipe {cfg.kind}")
        X[r0:r1, :Vd] = x.to(_dtype(cfg))
        Y[r0:r1, :Vt] = y.to(_dtype(cfg))
    out["X"] = X
    out["Y"] = Y
    return out


def make_inputs_numpy_c1(cfg):
    """The C1 recipe on the host with numpy PCG64(seed): float32 [R, V] arrays."""
    rng = np.random.Generator(np.random.PCG64(cfg.seed))
    X = rng.normal(0.0, 2.0, size=(cfg.R, cfg.v_draft))
    Y = X + rng.normal(0.0, 1.0, size=(cfg.R, cfg.v_draft))
    return {"X": X.astype(np.float32), "Y": Y.astype(np.float32), "d2t": None, "valid_depth": None}


def rows_to_host(t, rows, v):
    """float32 numpy copy of rows `rows`, columns [0, v), of a device array."""
    idx = torch.as_tensor(np.asarray(rows, dtype=np.int64), device=t.device)
    return t.index_select(0, idx)[:, :v].float().cpu().numpy()
