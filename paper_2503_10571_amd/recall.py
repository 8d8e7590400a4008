"""Recall diagnostics: Radar's segment selection against the exact search.

Radar ranks segments by the random-feature estimate of Eq. 6; the exact
segment search (the selector of the ablation in Section 3.3) ranks them by
beta_s, the summed unnormalised attention weights of the segment's keys.
Theorem 2 bounds when the estimate recovers the top segment; these helpers
measure how much of the exact selection, and of the attention mass, Radar
keeps as n and k vary (the quantities behind the n / k study of Section 3.3,
here on any keys the caller supplies):

  set_recall   |S_radar ∩ S_exact| / |S_exact| per query head;
  mass_ratio   attention mass of Radar's segments over that of the exact
               top-k (<= 1: the exact top-k maximises the mass);
  captured_mass  share of the full softmax kept by the selected segments
               plus the window;
  sweep        both, plus each selector's output error against full
               attention, over a grid of (n, k).

Selections, outputs, full attention and the exact segment masses come from
the library's own calls (radar_decode, radar_decode_exact,
radar_segment_mass); this module only compares and normalises them.
"""
from __future__ import annotations

import dataclasses

import torch

from . import Config, build_index, decode, decode_exact, new_summaries
from . import segment_mass as _segment_mass


def set_recall(sel: torch.Tensor, ref: torch.Tensor) -> torch.Tensor:
    """sel, ref: [B][Hq][k] segment ids, -1 padded. Fraction of ref's ids
    that sel also holds, per (b, q head); 1 where ref is empty."""
    hit = (sel.unsqueeze(-1) == ref.unsqueeze(-2)) & (sel.unsqueeze(-1) >= 0)
    found = hit.any(dim=-2).sum(-1).float()
    size = (ref >= 0).sum(-1).float()
    return torch.where(size > 0, found / size.clamp(min=1), torch.ones_like(size))


def segment_mass(cfg: Config, q: torch.Tensor, K: torch.Tensor, t: int,
                 n_cand: int) -> torch.Tensor:
    """Softmax attention mass of each candidate segment, [B][Hq][n_cand]
    fp32: the segment's share of the softmax over all t tokens. The exact
    masses come from the library (radar_segment_mass: ln(beta) of every
    candidate and of the window and sinks); here they are only normalised
    over those n_cand + 1 parts."""
    ln = _segment_mass(cfg, q, K, t)[..., :n_cand + 1]
    return torch.softmax(ln, dim=-1)[..., :n_cand]


def mass_ratio(sel: torch.Tensor, ref: torch.Tensor,
               mass: torch.Tensor) -> torch.Tensor:
    """Attention mass of sel's segments over that of ref's, per (b, q head);
    1 where ref selects nothing."""
    def total(s):
        m = torch.gather(mass, 2, s.clamp(min=0).long())
        return torch.where(s >= 0, m, torch.zeros_like(m)).sum(-1)
    den = total(ref)
    return torch.where(den > 0, total(sel) / den.clamp(min=1e-30),
                       torch.ones_like(den))


def captured_mass(sel: torch.Tensor, mass: torch.Tensor) -> torch.Tensor:
    """Share of the full softmax that attention over sel's segments plus the
    window keeps, per (b, q head): the selected segments' mass plus the
    mass outside every candidate segment (the window). The output error of
    attention restricted to these tokens is at most 2 (1 - captured) max|v|."""
    m = torch.gather(mass, 2, sel.clamp(min=0).long())
    picked = torch.where(sel >= 0, m, torch.zeros_like(m)).sum(-1)
    return picked + (1.0 - mass.sum(-1)).clamp(min=0)


def _rel_err(x: torch.Tensor, ref: torch.Tensor) -> torch.Tensor:
    """max_i |x_i - ref_i| / max_i |ref_i| per (b, q head)."""
    x, ref = x.float(), ref.float()
    return (x - ref).abs().amax(-1) / ref.abs().amax(-1).clamp(min=1e-30)


def sweep(cfg: Config, q: torch.Tensor, K: torch.Tensor, V: torch.Tensor,
          t: int, omegas: dict, ks) -> list:
    """Radar vs exact segment search at context length t for every n in
    omegas (n -> Omega [n][d] fp32) and every k in ks. Returns one dict per
    (n, k) with the mean / minimum set recall and mass ratio over the query
    heads and the mean output error of both selectors against full
    attention."""
    c, w = cfg.seg_len, cfg.window
    ws = c * (max(0, t - w) // c)
    n_cand = ws // c
    mass = segment_mass(cfg, q, K, t, n_cand) if n_cand else None
    # full attention: a window that covers the whole context (no candidate
    # segment, so the summaries and Omega are not read)
    n0, om0 = next(iter(omegas.items()))
    full_cfg = dataclasses.replace(cfg, window=cfg.capacity, n_features=n0)
    full = decode(full_cfg, q, K, V, om0, new_summaries(full_cfg, q.device),
                  t, 1)
    rows = []
    B, Hq = q.shape[0], q.shape[1]

    def ids(k):
        return torch.empty(B, Hq, k, dtype=torch.int32, device=q.device)
    exact = {}
    for k in ks:
        se = ids(k)
        out_e = decode_exact(cfg, q, K, V, t, k, selected=se)
        exact[k] = (se, _rel_err(out_e, full))
    for n, omega in omegas.items():
        ncfg = dataclasses.replace(cfg, n_features=n)
        summ = new_summaries(ncfg, q.device)
        build_index(ncfg, K, omega, t, summ)
        for k in ks:
            sr = ids(k)
            out_r = decode(ncfg, q, K, V, omega, summ, t, k, selected=sr)
            se, err_e = exact[k]
            rec = set_recall(sr, se)
            one = torch.ones_like(rec)
            mr = mass_ratio(sr, se, mass) if mass is not None else one
            cr = captured_mass(sr, mass) if mass is not None else one
            ce = captured_mass(se, mass) if mass is not None else one
            err_r = _rel_err(out_r, full)
            rows.append({
                "n": n, "k": k, "n_cand": n_cand,
                "recall_mean": float(rec.mean()), "recall_min": float(rec.min()),
                "mass_ratio_mean": float(mr.mean()),
                "mass_ratio_min": float(mr.min()),
                "captured_radar": float(cr.mean()),
                "captured_exact": float(ce.mean()),
                "out_err_radar": float(err_r.mean()),
                "out_err_exact": float(err_e.mean()),
            })
    return rows
