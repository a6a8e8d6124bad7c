"""Shared test helpers: build a problem (tables, parameters, batch) from a
configuration and hand it to the CPU checker in its plain-array form."""
from __future__ import annotations

import dataclasses

import numpy as np

from paper_2007_16122_amd import synth


def dims_of(cfg: synth.ColdConfig) -> dict:
    return dict(n_user=cfg.n_user, n_seq=cfg.n_seq, n_ad=cfg.n_ad, n_cross=cfg.n_cross,
                emb_dim=cfg.emb_dim, se_hidden=cfg.se_hidden, dtype=cfg.dtype,
                hashed=cfg.hashed, linear_log=cfg.linear_log, topk_k=cfg.topk_k,
                widths=list(cfg.widths), cross_pairs=[list(p) for p in cfg.cross_pairs],
                se_form=1 if cfg.se_form == "literal" else 0)


def tiny(name: str, **kw) -> synth.ColdConfig:
    """A small version of a named configuration: few rows, small tables."""
    base = synth.CONFIGS[name]
    small = dict(vocab=min(base.vocab, 257), n_requests=min(base.n_requests, 3),
                 cand_per_request=min(base.cand_per_request, 11), seq_len_max=7)
    if base.n_groups > 20:
        small.update(n_user=3, n_ad=5, n_cross=3)
        if base.n_seq:
            small["n_seq"] = 2
    if base.topk_k:
        small["topk_k"] = 5
    small.update(kw)
    cfg = synth.config(name, **small)
    if cfg.widths[0] != cfg.d_in or len(cfg.widths) > 4:
        w = (cfg.d_in, 24, 16, cfg.widths[-1]) if "widths" not in kw else cfg.widths
        cfg = dataclasses.replace(cfg, widths=w)
    return cfg


def stored_params(cfg, params: dict) -> dict:
    out = dict(params)
    out["mlp_w"] = [synth.mlp_weight_stored(w, cfg.dtype) for w in params["mlp_w"]]
    return out


def problem(cfg, seed=None, cand=None, scheme=None, params=None):
    tables = [synth.table_numpy(cfg, g, seed=seed, scheme=scheme) for g in range(cfg.n_groups)]
    params = synth.make_params(cfg, seed) if params is None else params
    batch = synth.make_batch(cfg, seed, cand)
    return tables, params, batch


def table_f64(cfg, t: np.ndarray) -> np.ndarray:
    """Stored table -> float64 (bf16 bit patterns widened to fp32 first)."""
    if cfg.dtype == "bf16":
        return (t.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return t.astype(np.float64)
