"""An independent numpy fp64 formulation of the COLD scoring path for tiny
inputs, used to pin the C checker.

Where the checker walks rows and loops, this writes every step as dense
matrix algebra over the whole batch: embedding lookup and sum-pooling as
(multi-)hot count matrices times the table, the squeeze as a block-averaging
matrix, the SE block and the network as matrix products, the per-request
importance as a request-averaging matrix, and the two-way softmax head as
sigmoid(z1 - z0).  Hashed ids use Python integers.
"""
from __future__ import annotations

import numpy as np

MASK64 = (1 << 64) - 1


def mix64_int(z: int) -> int:
    """SplitMix64's output function on Python integers."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def hashed_row(raw: int, g: int, rows: int) -> int:
    salt = ((g + 1) * 0x9E3779B97F4A7C15) & MASK64
    return mix64_int(int(raw) ^ salt) % rows


def _row_of(ids, g, rows, hashed):
    if hashed:
        return np.array([hashed_row(int(v), g, rows) for v in np.ravel(ids)], np.int64)
    return np.asarray(ids, np.int64).ravel()


def forward(dims, tables_f64, se, mlp_w_f64, mlp_b, batch):
    """Returns dict(scores, s, x, rows, importance, mask) for every row."""
    nu, ns, na, nx = dims["n_user"], dims["n_seq"], dims["n_ad"], dims["n_cross"]
    m = nu + ns + na + nx
    d = dims["emb_dim"]
    hashed = bool(dims["hashed"])
    req_off = np.asarray(batch["req_off"], np.int64)
    q_n = len(req_off) - 1
    r_n = int(req_off[-1])
    # membership matrix A[q, r] = 1 if row r belongs to request q
    member = np.zeros((q_n, r_n))
    for q in range(q_n):
        member[q, req_off[q]:req_off[q + 1]] = 1.0
    req_of_row = member.argmax(axis=0) if r_n else np.zeros(0, np.int64)

    blocks, rows_cols = [], []
    user_ids = np.asarray(batch["user_ids"]).reshape(nu, q_n)
    for f in range(nu):
        g = f
        rows_q = _row_of(user_ids[f], g, tables_f64[g].shape[0], hashed)
        count = np.zeros((r_n, tables_f64[g].shape[0]))
        count[np.arange(r_n), rows_q[req_of_row]] = 1.0
        blocks.append(count @ tables_f64[g])
        rows_cols.append(rows_q[req_of_row])
    seq_off = np.asarray(batch.get("seq_off", np.zeros(1)), np.int64)
    seq_ids = np.asarray(batch.get("seq_ids", np.zeros(0)))
    for f in range(ns):
        g = nu + f
        v = tables_f64[g].shape[0]
        per_req = np.zeros((q_n, v))          # multi-hot counts per request
        for q in range(q_n):
            lo, hi = seq_off[f * q_n + q], seq_off[f * q_n + q + 1]
            for rr in _row_of(seq_ids[lo:hi], g, v, hashed):
                per_req[q, rr] += 1.0
        blocks.append((member.T @ per_req) @ tables_f64[g])
        rows_cols.append(np.full(r_n, -1, np.int64))
    pairs = dims.get("cross_pairs") or None
    ad_all = np.asarray(batch["ad_ids"]).reshape(na, r_n)
    for name, count_f, base in (("ad_ids", na, nu + ns), ("cross_ids", nx, nu + ns + na)):
        if name == "cross_ids" and pairs:
            ids = None
        else:
            ids = np.asarray(batch[name]).reshape(count_f, r_n)
        for f in range(count_f):
            g = base + f
            v = tables_f64[g].shape[0]
            if ids is None:
                # cross value from a user field and an ad field:
                # key = mix64(user id) ^ ad id on unsigned integers, then hashed
                uf, af = pairs[f]
                width = 64 if hashed else 32
                unsigned = lambda x: int(x) & ((1 << width) - 1)
                rr = np.array([hashed_row(mix64_int(unsigned(user_ids[uf][req_of_row[i]]))
                                          ^ unsigned(ad_all[af][i]), g, v)
                               for i in range(r_n)], np.int64)
            else:
                rr = _row_of(ids[f], g, v, hashed)
            onehot = np.zeros((r_n, v))
            onehot[np.arange(r_n), rr] = 1.0
            blocks.append(onehot @ tables_f64[g])
            rows_cols.append(rr)
    e = np.concatenate(blocks, axis=1)                     # [R][M*d]
    avg = np.kron(np.eye(m), np.full((d, 1), 1.0 / d))     # [M*d][M]
    if int(dims.get("se_form", 0)) == 1:
        # Eq. 2 as printed: one dense layer from the concatenation to M logits
        s = 1.0 / (1.0 + np.exp(-(e @ se["se_w1"].astype(np.float64).T + se["se_b1"])))
    else:
        z = e @ avg
        h = np.maximum(z @ se["se_w1"].astype(np.float64).T + se["se_b1"], 0.0)
        s = 1.0 / (1.0 + np.exp(-(h @ se["se_w2"].astype(np.float64).T + se["se_b2"])))
    k = int(dims.get("topk_k", 0))
    importance = mask = None
    keep = np.ones_like(s)
    if k > 0:
        counts = member.sum(axis=1, keepdims=True)
        importance = (member @ s) / np.maximum(counts, 1.0)
        mask = np.zeros((q_n, m), np.uint8)
        for q in range(q_n):
            order = sorted(range(m), key=lambda g: (-importance[q, g], g))
            mask[q, order[:k]] = 1
        keep = mask[req_of_row].astype(np.float64)
    expand = np.kron(np.eye(m), np.ones((1, d)))           # [M][M*d]
    x = ((s * keep) @ expand) * e
    if dims["linear_log"]:
        ax = np.maximum(np.abs(x), 1.0)
        x = np.where(np.abs(x) <= 1.0, x, np.sign(x) * (1.0 + np.log(ax)))
    a = x
    n_layers = len(mlp_w_f64)
    for li in range(n_layers):
        a = a @ mlp_w_f64[li].T + mlp_b[li]
        if li < n_layers - 1:
            a = np.maximum(a, 0.0)
    if a.shape[1] == 1:
        scores = 1.0 / (1.0 + np.exp(-a[:, 0]))
    else:
        scores = 1.0 / (1.0 + np.exp(-(a[:, 1] - a[:, 0])))
    return dict(scores=scores, s=s, x=x, rows=np.stack(rows_cols, axis=1),
                importance=importance, mask=mask)
