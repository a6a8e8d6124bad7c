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


def problem(cfg, seed=None, cand=None, scheme=None, params=None, model_seed=None):
    """Tables, parameters and a batch of a configuration.  The batch comes
    from `seed`; the model (tables and parameters) from `model_seed` when it
    is given (cfg.seed: the configured model itself), else from `seed`."""
    ms = seed if model_seed is None else model_seed
    tables = [synth.table_numpy(cfg, g, seed=ms, scheme=scheme) for g in range(cfg.n_groups)]
    params = synth.make_params(cfg, ms) if params is None else params
    batch = synth.make_batch(cfg, seed, cand)
    return tables, params, batch


def table_f64(cfg, t: np.ndarray) -> np.ndarray:
    """Stored table -> float64 (bf16 bit patterns widened to fp32 first)."""
    if cfg.dtype == "bf16":
        return (t.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return t.astype(np.float64)


def se_weight_bound(params: dict, z: np.ndarray, s: np.ndarray, floor: float = 2e-6) -> np.ndarray:
    """Per-element bound on |s_fp32 - s| for the squeeze-excitation weights
    (Eq. 2: h = ReLU(W1 z + b1), s = sigmoid(W2 h + b2)) evaluated in fp32
    by sequential sums that start from the bias and add the terms in index
    order (the order the gather kernel uses).

    The synthetic tables hold multiples of a power of two with few
    significant bits and d is a power of two, so the squeeze z is exact in
    fp32 (callers check this).  Each dot product is then off by at most
    u * (sum_k |S_k| + sum_k |p_k|), u = 2^-24, over its partial sums S_k and
    products p_k (running error analysis: one rounding per product and one
    per addition, so fused or not); the hidden error passes through the ReLU
    unamplified and into the logit through |W2|; the sigmoid's slope over
    the logit's error interval scales the result, and `floor` covers the
    sigmoid's own evaluation.  z: [n][M], s: [n][M] (fp64 reference).
    """
    u = 2.0 ** -24
    w1, b1, w2, b2 = (np.asarray(params[k], np.float64) for k in ("se_w1", "se_b1", "se_w2", "se_b2"))

    def dot_and_error(x, w, b):
        p = x[:, None, :] * w[None, :, :]                  # [n][out][in]
        partial = b[None, :, None] + np.cumsum(p, axis=2)
        err = u * (np.abs(b)[None, :] + np.abs(partial).sum(axis=2) + np.abs(p).sum(axis=2))
        return partial[:, :, -1], err * (1.0 + 4 * x.shape[1] * u)

    a, da = dot_and_error(z, w1, b1)
    h = np.maximum(a, 0.0)
    logit, dl = dot_and_error(h, w2, b2)
    dl = dl + da @ np.abs(w2).T
    # steepest sigmoid slope on [logit - dl, logit + dl]
    x = np.maximum(np.abs(logit) - dl, 0.0)
    sx = 1.0 / (1.0 + np.exp(-x))
    slope = sx * (1.0 - sx)
    assert s.shape == dl.shape
    return slope * dl + floor


def assert_se_weights_close(params: dict, got: np.ndarray, o: dict) -> None:
    """fp32 SE weights against the checker's, within se_weight_bound."""
    z = o["z"]
    assert np.array_equal(z.astype(np.float32).astype(np.float64), z), "squeeze not exact in fp32"
    bound = se_weight_bound(params, z, o["s"])
    err = np.abs(np.asarray(got, np.float64) - o["s"])
    worst = np.unravel_index(np.argmax(err - bound), err.shape) if err.size else None
    assert np.all(err <= bound), (f"SE weight off by {err[worst]:.3e} at {worst}, "
                                  f"bound {bound[worst]:.3e}")
