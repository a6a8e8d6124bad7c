"""CPU checker for the COLD scoring path -- test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It wraps ``cold_oracle.c`` (plain
double-precision C, see that file for the steps and the paper passages they
follow) with ctypes, takes plain numpy arrays, and shares no code with the
HIP library.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcold_oracle.so")
SRC_PATH = os.path.join(_HERE, "cold_oracle.c")

DTYPES = {"f32": 0, "bf16": 1, "f16": 2}


def build(force: bool = True) -> str:
    """Compile the checker with gcc (-O2, no fast-math, OpenMP)."""
    if force or not os.path.exists(LIB_PATH):
        tmp = LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                               "-Wall", "-Wextra", "-o", tmp, SRC_PATH, "-lm"])
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


class _Problem(ctypes.Structure):
    _fields_ = [
        ("n_requests", ctypes.c_int64), ("n_rows", ctypes.c_int64),
        ("n_user", ctypes.c_int32), ("n_seq", ctypes.c_int32),
        ("n_ad", ctypes.c_int32), ("n_cross", ctypes.c_int32),
        ("emb_dim", ctypes.c_int32), ("se_hidden", ctypes.c_int32),
        ("dtype", ctypes.c_int32), ("hashed", ctypes.c_int32),
        ("linear_log", ctypes.c_int32), ("topk_k", ctypes.c_int32),
        ("n_layers", ctypes.c_int32),
        ("widths", ctypes.c_void_p), ("table_rows", ctypes.c_void_p),
        ("tables", ctypes.c_void_p),
        ("se_w1", ctypes.c_void_p), ("se_b1", ctypes.c_void_p),
        ("se_w2", ctypes.c_void_p), ("se_b2", ctypes.c_void_p),
        ("mlp_w", ctypes.c_void_p), ("mlp_b", ctypes.c_void_p),
        ("req_off", ctypes.c_void_p), ("user_ids", ctypes.c_void_p),
        ("ad_ids", ctypes.c_void_p), ("cross_ids", ctypes.c_void_p),
        ("seq_off", ctypes.c_void_p), ("seq_ids", ctypes.c_void_p),
        ("n_seq_ids", ctypes.c_int64),
        ("cross_pairs", ctypes.c_void_p),
        ("se_form", ctypes.c_int32),
    ]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        L.orc_score.restype = ctypes.c_int
        L.orc_score.argtypes = [ctypes.POINTER(_Problem), ctypes.c_void_p, ctypes.c_int64,
                                ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                ctypes.c_void_p, ctypes.c_int]
        L.orc_linear_log.restype = ctypes.c_double
        L.orc_linear_log.argtypes = [ctypes.c_double]
        L.orc_mix64.restype = ctypes.c_uint64
        L.orc_mix64.argtypes = [ctypes.c_uint64]
        L.orc_hash_row.restype = ctypes.c_uint64
        L.orc_hash_row.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_uint64]
        L.orc_cross_key.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        L.orc_cross_key.restype = ctypes.c_uint64
        L.orc_decode_stored.restype = ctypes.c_int
        L.orc_decode_stored.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64,
                                        ctypes.c_void_p]
        _lib = L
    return _lib


class OracleError(RuntimeError):
    pass


_ERRORS = {-1: "bad argument", -2: "id out of range", -3: "out of memory"}


def _ptr(a):
    return None if a is None else a.ctypes.data


def linear_log(x: float) -> float:
    return lib().orc_linear_log(float(x))


def mix64(z: int) -> int:
    return int(lib().orc_mix64(z & 0xFFFFFFFFFFFFFFFF))


def hash_row(raw: int, g: int, rows: int) -> int:
    return int(lib().orc_hash_row(raw & 0xFFFFFFFFFFFFFFFF, g, rows))


def cross_key(user_id: int, ad_id: int) -> int:
    """64-bit key of a user x ad cross value (see orc_cross_key)."""
    return int(lib().orc_cross_key(user_id & 0xFFFFFFFFFFFFFFFF, ad_id & 0xFFFFFFFFFFFFFFFF))


def decode_stored(dtype: str, values: np.ndarray) -> np.ndarray:
    """The checker's decoder of stored parameters (fp32, bf16 bit patterns
    as uint16, or fp16) to float64."""
    src = np.ascontiguousarray(values)
    out = np.zeros(src.size, np.float64)
    st = lib().orc_decode_stored(DTYPES[dtype], src.ctypes.data, src.size, out.ctypes.data)
    if st != 0:
        raise OracleError(_ERRORS.get(st, f"status {st}"))
    return out


def score(dims: dict, tables, params: dict, batch: dict, sample=None, *,
          want_rows=False, want_s=False, want_x=False, want_z=False,
          n_threads=None) -> dict:
    """Score rows of a batch.

    dims: n_user, n_seq, n_ad, n_cross, emb_dim, se_hidden, dtype ('f32' |
      'bf16' | 'f16'), hashed, linear_log, topk_k, widths, and optionally
      cross_pairs ([n_cross][2] user field, ad field: cross ids are then
      built from the pairs and batch['cross_ids'] is not read) and se_form
      (0: squeeze/excitation SE; 1: one FC over the concatenated embeddings,
      se_w1 [M][M*d], se_b1 [M], se_w2/se_b2 unused).
    tables: list of M arrays [rows][d] in stored form (float32, float16, or
      uint16 bf16 bit patterns).
    params: se_w1 [H][M], se_b1, se_w2 [M][H], se_b2 (float32); mlp_w list of
      [out][in] arrays in stored form; mlp_b list of float32 [out].
    batch: req_off, user_ids, ad_ids, cross_ids, seq_off, seq_ids.
    sample: row indices to score (default: every row).

    Returns a dict with 'scores' and, on request, 'rows', 's', 'x', 'z' (the
    SE squeeze, zero for the one-layer form), and (when topk_k > 0)
    'importance' and 'mask' per request.
    """
    L = lib()
    m = dims["n_user"] + dims["n_seq"] + dims["n_ad"] + dims["n_cross"]
    d = dims["emb_dim"]
    hashed = bool(dims["hashed"])
    id_dt = np.uint64 if hashed else np.int32
    keep = []

    def arr(a, dt):
        a = np.ascontiguousarray(a, dtype=dt)
        keep.append(a)
        return a

    widths = arr(dims["widths"], np.int32)
    n_layers = len(widths) - 1
    req_off = arr(batch["req_off"], np.int32)
    q = len(req_off) - 1
    r = int(req_off[-1])
    tabs = [np.ascontiguousarray(t) for t in tables]
    keep.extend(tabs)
    assert len(tabs) == m
    for t in tabs:
        assert t.ndim == 2 and t.shape[1] == d
    table_rows = arr([t.shape[0] for t in tabs], np.int64)
    table_ptrs = arr([t.ctypes.data for t in tabs], np.uint64)
    mlp_w = [np.ascontiguousarray(w) for w in params["mlp_w"]]
    mlp_b = [np.ascontiguousarray(b, dtype=np.float32) for b in params["mlp_b"]]
    keep.extend(mlp_w)
    keep.extend(mlp_b)
    w_ptrs = arr([w.ctypes.data for w in mlp_w], np.uint64)
    b_ptrs = arr([b.ctypes.data for b in mlp_b], np.uint64)
    se_w1 = arr(params["se_w1"], np.float32)
    se_b1 = arr(params["se_b1"], np.float32)
    se_w2 = arr(params["se_w2"], np.float32)
    se_b2 = arr(params["se_b2"], np.float32)
    user_ids = arr(np.asarray(batch["user_ids"]).reshape(dims["n_user"], q), id_dt)
    ad_ids = arr(np.asarray(batch["ad_ids"]).reshape(dims["n_ad"], r), id_dt)
    pairs = dims.get("cross_pairs") or None
    cross_pairs = None if pairs is None else arr(np.asarray(pairs).reshape(-1), np.int32)
    if pairs is None:
        cross_ids = arr(np.asarray(batch["cross_ids"]).reshape(dims["n_cross"], r), id_dt)
    else:
        cross_ids = None      # built from the user/ad id pairs
    seq_off = arr(batch.get("seq_off", np.zeros(1, np.int32)), np.int32)
    seq_ids = arr(batch.get("seq_ids", np.zeros(0, id_dt)), id_dt)
    if seq_ids.size == 0:
        seq_ids = arr(np.zeros(1, id_dt), id_dt)
        n_seq_ids = 0
    else:
        n_seq_ids = seq_ids.size
    prob = _Problem(
        n_requests=q, n_rows=r, n_user=dims["n_user"], n_seq=dims["n_seq"],
        n_ad=dims["n_ad"], n_cross=dims["n_cross"], emb_dim=d,
        se_hidden=dims["se_hidden"], dtype=DTYPES[dims["dtype"]], hashed=int(hashed),
        linear_log=int(bool(dims["linear_log"])), topk_k=int(dims.get("topk_k", 0)),
        n_layers=n_layers, widths=_ptr(widths), table_rows=_ptr(table_rows),
        tables=_ptr(table_ptrs), se_w1=_ptr(se_w1), se_b1=_ptr(se_b1), se_w2=_ptr(se_w2),
        se_b2=_ptr(se_b2), mlp_w=_ptr(w_ptrs), mlp_b=_ptr(b_ptrs), req_off=_ptr(req_off),
        user_ids=_ptr(user_ids), ad_ids=_ptr(ad_ids), cross_ids=_ptr(cross_ids),
        seq_off=_ptr(seq_off), seq_ids=_ptr(seq_ids), n_seq_ids=n_seq_ids,
        cross_pairs=_ptr(cross_pairs), se_form=int(dims.get("se_form", 0)))
    sample = arr(np.arange(r) if sample is None else sample, np.int64)
    n = sample.size
    out = {"scores": np.zeros(n, np.float64)}
    if want_rows:
        out["rows"] = np.zeros((n, m), np.int64)
    if want_s:
        out["s"] = np.zeros((n, m), np.float64)
    if want_x:
        out["x"] = np.zeros((n, m * d), np.float64)
    if want_z:
        out["z"] = np.zeros((n, m), np.float64)
    topk = int(dims.get("topk_k", 0)) > 0
    if topk:
        out["importance"] = np.zeros((q, m), np.float64)
        out["mask"] = np.zeros((q, m), np.uint8)
    if n_threads is None:
        n_threads = len(os.sched_getaffinity(0))
    st = L.orc_score(ctypes.byref(prob), _ptr(sample), n, _ptr(out["scores"]),
                     _ptr(out.get("rows")), _ptr(out.get("s")), _ptr(out.get("x")),
                     _ptr(out.get("z")), _ptr(out.get("importance")), _ptr(out.get("mask")), int(n_threads))
    if st != 0:
        raise OracleError(_ERRORS.get(st, f"status {st}"))
    out["n_threads"] = n_threads
    return out


# ----------------------------------------------------------------------------
# Top-n selection by eCPM (Section 2 and its footnote: the pre-ranking stage
# passes on the N candidates of a request with the highest eCPM, where
# eCPM = pCTR * bid for CPC bidding).  Plain numpy, one request at a time.
# ----------------------------------------------------------------------------
def total_order_key(x32: np.ndarray) -> np.ndarray:
    """IEEE-754 totalOrder position of fp32 values as int64 (larger = later
    in the order): a non-negative value keeps its magnitude bits, a value
    with the sign bit set becomes -(magnitude bits) - 1, which puts -0 just
    below +0, larger negative magnitudes lower, and NaNs beyond the
    infinities on the side of their sign."""
    bits = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32).astype(np.int64)
    mag = bits & 0x7FFFFFFF
    return np.where(bits >> 31 == 1, -mag - 1, mag)


def select_topn(scores, bids, req_off, n_top: int):
    """Per request q: eCPM = scores * bids (one fp32 multiplication per row),
    rows ordered by eCPM descending under totalOrder, ties by ascending row
    index, the first n_top kept.  Returns (rows int32 [Q][n_top], ecpm fp32
    [Q][n_top]); a request with fewer rows pads with -1 and -inf."""
    scores = np.asarray(scores, dtype=np.float32)
    bids = np.asarray(bids, dtype=np.float32)
    req_off = np.asarray(req_off, dtype=np.int64)
    n_req = req_off.size - 1
    r_total = scores.size
    rows = np.full((n_req, n_top), -1, dtype=np.int32)
    ecpm = np.full((n_req, n_top), -np.inf, dtype=np.float32)
    for q in range(n_req):
        lo = min(max(int(req_off[q]), 0), r_total)
        hi = min(max(int(req_off[q + 1]), lo), r_total)
        if hi == lo:
            continue
        e = scores[lo:hi] * bids[lo:hi]                  # float32 * float32 -> float32
        idx = np.arange(lo, hi, dtype=np.int64)
        order = np.lexsort((idx, -total_order_key(e)))  # last key is the primary one
        k = min(n_top, hi - lo)
        rows[q, :k] = idx[order[:k]]
        ecpm[q, :k] = e[order[:k]]
    return rows, ecpm


def recall_at(pre_rows, rank_rows) -> float:
    """Eq. 4 of Section 4.1: |top-k by the pre-ranking model ∩ top-m by the
    ranking model| / |top-m by the ranking model|, pooled over requests
    (padding -1 entries are ignored)."""
    hit = tot = 0
    for a, b in zip(pre_rows, rank_rows):
        ref = set(int(v) for v in b if v >= 0)
        hit += len(ref & set(int(v) for v in a if v >= 0))
        tot += len(ref)
    return hit / tot if tot else 1.0
