"""Helpers for the GPU parity tests: run the HIP path through the C ABI and
the CPU checker on the same seeded inputs, and compare."""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

import oracle
from paper_2007_16122_amd import binding, synth
from tests.common import dims_of, stored_params

TOL = {"f32": 1e-5, "bf16": 2e-3, "f16": 2e-3}


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def device_table_from_numpy(t: np.ndarray, dtype: str, device):
    import torch
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(t).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(t)).to(device)


def needed_rows(cfg, batch, sample, whole_requests=False):
    """Per group, the table rows the checker will read for the sampled rows
    (all rows of their requests when whole_requests)."""
    req_off = batch["req_off"]
    q_n = len(req_off) - 1
    reqs = np.unique(np.searchsorted(req_off, sample, side="right") - 1)
    if whole_requests:
        sample = np.concatenate([np.arange(req_off[q], req_off[q + 1]) for q in reqs])
    out = []
    for g in range(cfg.n_groups):
        kind = cfg.group_kind(g)
        if kind == "user":
            ids = batch["user_ids"][g][reqs]
        elif kind == "seq":
            f = g - cfg.n_user
            so = batch["seq_off"]
            ids = np.concatenate([batch["seq_ids"][so[f * q_n + q]:so[f * q_n + q + 1]] for q in reqs])
        elif kind == "ad":
            ids = batch["ad_ids"][g - cfg.n_user - cfg.n_seq][sample]
        else:
            ids = batch["cross_ids"][g - cfg.n_user - cfg.n_seq - cfg.n_ad][sample]
        if cfg.hashed:
            rows = np.array([oracle.hash_row(int(v), g, cfg.vocab) for v in np.unique(ids)], np.int64)
        else:
            rows = ids.astype(np.int64)
        out.append(np.unique(rows))
    return out


def sparse_host_tables(cfg, batch, sample, seed=None, scheme=None, whole_requests=False):
    """Full-shape host tables holding only the rows the checker reads (the
    rest stays untouched zero pages); the values come from the numpy twin of
    the generator that filled the device tables."""
    np_dt = {"f32": np.float32, "f16": np.float16, "bf16": np.uint16}[cfg.dtype]
    tabs = []
    for g, rows in enumerate(needed_rows(cfg, batch, sample, whole_requests)):
        t = np.zeros((cfg.vocab, cfg.emb_dim), np_dt)
        if rows.size:
            t[rows] = synth.table_rows_numpy(cfg, g, rows, seed=seed, scheme=scheme)
        tabs.append(t)
    return tabs


class GpuScorer:
    """A model loaded on the GPU for one configuration."""

    def __init__(self, cfg, tables_dev, params, device="cuda"):
        import torch
        self.torch = torch
        self.cfg = cfg
        self.device = torch.device(device)
        self.model = binding.ColdModel(cfg, device=self.device)
        self.params_dev = binding.params_to_device(params, cfg.dtype, self.device)
        self.tables_dev = tables_dev
        self.model.load(tables_dev, self.params_dev)

    def score(self, batch_np, want_rows=False, want_s=False, want_mask=False, want_x=False,
              validate=True):
        torch = self.torch
        cfg = self.cfg
        b = binding.batch_to_device(batch_np, self.device)
        r_n, q_n = batch_np["n_rows"], len(batch_np["req_off"]) - 1
        m = cfg.n_groups
        rows = torch.full((m, max(r_n, 1)), -7, dtype=torch.int32, device=self.device) if want_rows else None
        imp = torch.zeros((max(r_n, 1), m), dtype=torch.float32, device=self.device) if want_s else None
        mask = torch.zeros((max(q_n, 1), m), dtype=torch.uint8, device=self.device) if want_mask else None
        xdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[cfg.dtype]
        x = torch.full((max(r_n, 1), cfg.d_in), float("nan"), dtype=xdt, device=self.device) \
            if want_x else None
        scores = self.model.score(b, importance=imp, group_mask=mask, rows_out=rows, x_out=x,
                                  validate=validate)
        torch.cuda.synchronize(self.device)
        out = {"scores": scores.cpu().numpy().astype(np.float64)}
        if want_rows:
            out["rows"] = rows.cpu().numpy()[:, :r_n]
        if want_s:
            out["s"] = imp.cpu().numpy()[:r_n]
        if want_mask:
            out["mask"] = mask.cpu().numpy()[:q_n]
        if want_x:
            out["x"] = x[:r_n].to(torch.float32).cpu().numpy().astype(np.float64)
        return out

    def close(self):
        self.model.close()


def run_oracle(cfg, tables, params, batch, sample=None, **kw):
    t0 = time.time()
    o = oracle.score(dims_of(cfg), tables, stored_params(cfg, params), batch, sample=sample, **kw)
    o["seconds"] = time.time() - t0
    return o


def record(entry: dict) -> None:
    """Append one JSON line to the file COLD_PARITY_LOG names (if set)."""
    path = os.environ.get("COLD_PARITY_LOG")
    if path:
        with open(path, "a") as fh:
            fh.write(json.dumps(entry) + "\n")


def compare_scores(cfg, got, want, label=""):
    """|GPU - checker| CTR statistics, asserted within the tolerance of the
    model's dtype.  With COLD_PARITY_LOG set, each comparison is also
    appended to that file as one JSON line."""
    d = np.abs(got - want)
    tol = TOL[cfg.dtype]
    stats = dict(max=float(d.max()) if d.size else 0.0,
                 p99=float(np.quantile(d, 0.99)) if d.size else 0.0,
                 mean=float(d.mean()) if d.size else 0.0, n=int(d.size))
    log(f"[{label}] |dCTR| max {stats['max']:.3e} p99 {stats['p99']:.3e} "
        f"mean {stats['mean']:.3e} over {stats['n']} rows (tol {tol:g})")
    record(dict(stats, label=label, workload=cfg.name, dtype=cfg.dtype, tol=tol,
                ctr_mean=float(np.mean(want)) if d.size else 0.0,
                ctr_std=float(np.std(want)) if d.size else 0.0))
    assert np.all(np.isfinite(got)), "non-finite GPU score"
    assert stats["max"] <= tol, stats
    return stats


def request_slice(cfg, batch, q, q_end=None):
    """Requests q .. q_end - 1 (default: request q alone) of a host batch as
    a batch of their own."""
    q_end = q + 1 if q_end is None else q_end
    off = batch["req_off"]
    lo, hi = int(off[q]), int(off[q_end])
    Q = len(off) - 1
    out = dict(req_off=(off[q:q_end + 1] - lo).astype(np.int32),
               user_ids=np.ascontiguousarray(batch["user_ids"][:, q:q_end]),
               ad_ids=np.ascontiguousarray(batch["ad_ids"][:, lo:hi]),
               cross_ids=np.ascontiguousarray(batch["cross_ids"][:, lo:hi]),
               n_rows=hi - lo, n_requests=q_end - q)
    if cfg.n_seq:
        so = batch["seq_off"]
        segs = [batch["seq_ids"][so[f * Q + qq]:so[f * Q + qq + 1]]
                for f in range(cfg.n_seq) for qq in range(q, q_end)]
        out["seq_off"] = np.concatenate([[0], np.cumsum([len(x) for x in segs])]).astype(np.int32)
        out["seq_ids"] = np.concatenate(segs)
    else:
        out["seq_off"] = np.zeros(1, np.int32)
        out["seq_ids"] = np.zeros(0, batch["ad_ids"].dtype)
    return out


def with_empty_sequences(cfg, batch, empties):
    """The batch with the behaviour sequences (field f, request q) in
    `empties` emptied (Section 3.3: an empty sequence pools to zero)."""
    q_n = len(batch["req_off"]) - 1
    so, ids = batch["seq_off"], batch["seq_ids"]
    segs = []
    for f in range(cfg.n_seq):
        for q in range(q_n):
            seg = ids[so[f * q_n + q]:so[f * q_n + q + 1]]
            segs.append(seg[:0] if (f, q) in empties else seg)
    out = dict(batch)
    out["seq_off"] = np.concatenate([[0], np.cumsum([len(x) for x in segs])]).astype(np.int32)
    out["seq_ids"] = np.concatenate(segs) if segs else ids[:0]
    return out


def half_ulp(x, dtype):
    """The spacing of the model dtype's values at |x| (the unit in the last
    place of the rounded network input): fp16 10 fraction bits with
    subnormals below 2^-14, bf16 7 fraction bits."""
    ax = np.abs(np.asarray(x, np.float64))
    if dtype == "f16":
        e = np.floor(np.log2(np.maximum(ax, 2.0 ** -14)))
        return 2.0 ** (e - 10)
    if dtype == "bf16":
        e = np.floor(np.log2(np.maximum(ax, 2.0 ** -126)))
        return 2.0 ** (e - 7)
    e = np.floor(np.log2(np.maximum(ax, 2.0 ** -126)))
    return 2.0 ** (e - 23)
