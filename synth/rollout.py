"""A token-dependent toy model for rollouts with exact context (inputs only).

Real draft and target models give, at depth i of a path, logits conditioned
on that path's own prefix.  This stand-in makes such rows from a recipe's
ordinary rows (`base`, one per slot) and a seeded table of M shift rows:

    row at depth i along a path whose token at depth i-1 is z
        = base[slot at depth i] + table[z mod M]      (no shift at depth 0)

in float32, rounded once to the logit dtype.  At depth 0 every family shares
the prefix, so its rows are the base rows.  The same torch operations run on
the host and on the device, so equal tokens give identical rows on both
sides.  This module holds none of the method's arithmetic.
"""
import torch

M_SHIFTS = 61


def make_tables(cfg, device, scale=1.0, m=M_SHIFTS):
    """(table_d [m, ld_d], table_t [m, ld_t]) float32 shift rows, N(0, scale^2),
    zero in the padding columns; seeded by the config."""
    gen = torch.Generator(device=device).manual_seed(cfg.seed * 31 + 7)
    td = torch.zeros(m, cfg.ld(cfg.v_draft), dtype=torch.float32, device=device)
    tt = torch.zeros(m, cfg.ld(cfg.v_target), dtype=torch.float32, device=device)
    tt[:, :cfg.v_target] = scale * torch.randn(m, cfg.v_target, generator=gen, device=device)
    td[:, :cfg.v_draft] = scale * torch.randn(m, cfg.v_draft, generator=gen, device=device)
    return td, tt


def context_rows(base, table, prev):
    """Rows [n, ld] in base's dtype: base + table[prev mod m] where prev >= 0,
    base where prev < 0 (depth 0)."""
    prev = prev.long()
    shift = table[prev.clamp(min=0) % table.shape[0]] * (prev >= 0).to(torch.float32)[:, None]
    return (base.float() + shift).to(base.dtype)


def depth_view(t, n_paths, L, step):
    """The rows of depth `step` of every path in an [n_paths*L, ld] tensor,
    as a strided [n_paths, ld] view (row stride L*ld)."""
    return t.view(n_paths, L, t.shape[1])[:, step]
