"""ctypes binding of libcold.so (include/cold.h).

Argument marshalling only: every step of the scoring path runs in the HIP
kernels of libcold.so.  The functions keep the C names; :class:`ColdModel`
strings them together with torch providing device memory and the stream.
If the library is missing this module raises -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libcold.so")

COLD_OK = 0
COLD_ERR_INVALID_ARG = -1
COLD_ERR_SHAPE = -2
COLD_ERR_DTYPE = -3
COLD_ERR_NOT_LOADED = -4
COLD_ERR_WORKSPACE = -5
COLD_ERR_HIP = -6
COLD_ERR_ID_RANGE = -7
COLD_F32, COLD_BF16, COLD_F16 = 0, 1, 2
COLD_IDS_DIRECT_I32, COLD_IDS_HASHED_U64 = 0, 1
COLD_SCORE_VALIDATE = 1
DTYPES = {"f32": COLD_F32, "bf16": COLD_BF16, "f16": COLD_F16}

EXPORTS = ("cold_create_model", "cold_destroy_model", "cold_weight_arena_bytes",
           "cold_workspace_bytes", "cold_load_weights", "cold_score",
           "cold_status_string", "cold_last_error", "cold_profile_enable",
           "cold_profile_read", "cold_select_topn", "cold_score_noalloc")
COLD_NOALLOC_WORKSPACE_BYTES = 96 * 1024 * 1024
COLD_TOPN_MAX = 1024
COLD_SE_SQUEEZE, COLD_SE_LITERAL = 0, 1


class ColdError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


class cold_model_desc(ctypes.Structure):
    _fields_ = [("n_user", ctypes.c_int32), ("n_seq", ctypes.c_int32),
                ("n_ad", ctypes.c_int32), ("n_cross", ctypes.c_int32),
                ("emb_dim", ctypes.c_int32), ("id_kind", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("se_reduction", ctypes.c_int32),
                ("n_layers", ctypes.c_int32),
                ("widths", ctypes.POINTER(ctypes.c_int32)),
                ("table_rows", ctypes.POINTER(ctypes.c_int64)),
                ("linear_log", ctypes.c_int32), ("topk_k", ctypes.c_int32),
                ("cross_pairs", ctypes.POINTER(ctypes.c_int32)),
                ("se_form", ctypes.c_int32)]


class cold_weights(ctypes.Structure):
    _fields_ = [("tables", ctypes.POINTER(ctypes.c_void_p)),
                ("se_w1", ctypes.c_void_p), ("se_b1", ctypes.c_void_p),
                ("se_w2", ctypes.c_void_p), ("se_b2", ctypes.c_void_p),
                ("mlp_w", ctypes.POINTER(ctypes.c_void_p)),
                ("mlp_b", ctypes.POINTER(ctypes.c_void_p))]


class cold_batch(ctypes.Structure):
    _fields_ = [("n_requests", ctypes.c_int64), ("n_rows", ctypes.c_int64),
                ("n_seq_ids", ctypes.c_int64), ("req_off", ctypes.c_void_p),
                ("user_ids", ctypes.c_void_p), ("ad_ids", ctypes.c_void_p),
                ("cross_ids", ctypes.c_void_p), ("seq_off", ctypes.c_void_p),
                ("seq_ids", ctypes.c_void_p)]


_lib = None


def lib():
    """The loaded libcold.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2007_16122_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        L.cold_create_model.argtypes = [ctypes.POINTER(cold_model_desc), ctypes.POINTER(vp)]
        L.cold_create_model.restype = ctypes.c_int
        L.cold_destroy_model.argtypes = [vp]
        L.cold_destroy_model.restype = None
        L.cold_weight_arena_bytes.argtypes = [vp]
        L.cold_weight_arena_bytes.restype = sz
        L.cold_workspace_bytes.argtypes = [vp, i64, i64]
        L.cold_workspace_bytes.restype = sz
        L.cold_load_weights.argtypes = [vp, ctypes.POINTER(cold_weights), vp, sz, vp]
        L.cold_load_weights.restype = ctypes.c_int
        L.cold_score.argtypes = [vp, ctypes.POINTER(cold_batch), vp, sz, vp, vp, vp, vp, vp, i32, vp]
        L.cold_score.restype = ctypes.c_int
        L.cold_score_noalloc.argtypes = [vp, ctypes.POINTER(cold_batch), vp, vp, vp, vp, vp, i32, vp]
        L.cold_score_noalloc.restype = ctypes.c_int
        L.cold_status_string.argtypes = [ctypes.c_int]
        L.cold_status_string.restype = ctypes.c_char_p
        L.cold_last_error.argtypes = [vp]
        L.cold_last_error.restype = ctypes.c_char_p
        L.cold_profile_enable.argtypes = [vp, i32]
        L.cold_profile_enable.restype = ctypes.c_int
        L.cold_profile_read.argtypes = [vp, i32, vp, vp, ctypes.POINTER(i32), ctypes.POINTER(i32)]
        L.cold_profile_read.restype = ctypes.c_int
        L.cold_select_topn.argtypes = [vp, vp, vp, i64, i64, i32, vp, vp, vp]
        L.cold_select_topn.restype = ctypes.c_int
        _lib = L
    return _lib


# ---------------------------------------------------------------- C names
def cold_create_model(desc: cold_model_desc):
    h = ctypes.c_void_p()
    st = lib().cold_create_model(ctypes.byref(desc), ctypes.byref(h))
    if st != COLD_OK:
        raise ColdError(st, "cold_create_model: " + cold_status_string(st))
    return h


def cold_destroy_model(h) -> None:
    lib().cold_destroy_model(h)


def cold_weight_arena_bytes(h) -> int:
    return int(lib().cold_weight_arena_bytes(h))


def cold_workspace_bytes(h, max_rows: int, max_requests: int) -> int:
    return int(lib().cold_workspace_bytes(h, max_rows, max_requests))


def cold_load_weights(h, w: cold_weights, arena: int, arena_bytes: int, stream: int) -> int:
    return lib().cold_load_weights(h, ctypes.byref(w), arena, arena_bytes, stream)


def cold_score(h, b: cold_batch, workspace: int, ws_bytes: int, scores: int,
               importance: Optional[int], group_mask: Optional[int], rows_out: Optional[int],
               x_out: Optional[int], flags: int, stream: int) -> int:
    return lib().cold_score(h, ctypes.byref(b), workspace, ws_bytes, scores, importance,
                            group_mask, rows_out, x_out, flags, stream)


def cold_score_noalloc(h, b: cold_batch, scores: int, importance: Optional[int],
                       group_mask: Optional[int], rows_out: Optional[int], x_out: Optional[int],
                       flags: int, stream: int) -> int:
    return lib().cold_score_noalloc(h, ctypes.byref(b), scores, importance, group_mask, rows_out,
                                    x_out, flags, stream)


def cold_status_string(st: int) -> str:
    return lib().cold_status_string(st).decode()


def cold_last_error(h) -> str:
    return lib().cold_last_error(h).decode()


def cold_profile_enable(h, enable: bool) -> int:
    return lib().cold_profile_enable(h, int(bool(enable)))


def cold_profile_read(h, max_stages: int = 32):
    """Per-stage summed milliseconds of the profiled calls since the last
    read: (list of (name, ms), n_calls)."""
    names = (ctypes.c_char * 32 * max_stages)()
    total = (ctypes.c_float * max_stages)()
    ns, nc = ctypes.c_int32(), ctypes.c_int32()
    st = lib().cold_profile_read(h, max_stages, ctypes.addressof(names), ctypes.addressof(total),
                                 ctypes.byref(ns), ctypes.byref(nc))
    if st != COLD_OK:
        raise ColdError(st, "cold_profile_read: " + cold_last_error(h))
    out = [(bytes(names[i]).split(b"\0")[0].decode(), float(total[i]))
           for i in range(min(ns.value, max_stages))]
    return out, nc.value


def cold_select_topn(scores: int, bids: int, req_off: int, n_requests: int, n_rows: int,
                     n_top: int, top_rows: int, top_ecpm: Optional[int], stream: int) -> int:
    return lib().cold_select_topn(scores, bids, req_off, n_requests, n_rows, n_top, top_rows,
                                  top_ecpm, stream)


def select_topn(scores, bids, req_off, n_top: int, with_ecpm: bool = True):
    """Top-n rows of every request by eCPM = score * bid on the current
    stream: returns (rows int32 [Q][n_top], ecpm fp32 [Q][n_top] or None)."""
    import torch
    n_req = req_off.numel() - 1
    rows = torch.empty((max(n_req, 0), n_top), dtype=torch.int32, device=scores.device)
    ecpm = torch.empty((max(n_req, 0), n_top), dtype=torch.float32, device=scores.device) \
        if with_ecpm else None
    st = cold_select_topn(_ptr(scores), _ptr(bids), _ptr(req_off), n_req, scores.numel(), n_top,
                          _ptr(rows), _ptr(ecpm), torch.cuda.current_stream().cuda_stream)
    if st != COLD_OK:
        raise ColdError(st, "cold_select_topn: " + cold_status_string(st))
    return rows, ecpm


def make_desc(n_user, n_seq, n_ad, n_cross, emb_dim, dtype, se_reduction,
              widths: Sequence[int], table_rows: Sequence[int], hashed=False,
              linear_log=False, topk_k=0, cross_pairs=None, se_form=0):
    """A cold_model_desc plus the arrays it points to (keep both alive).
    cross_pairs: None, or (user field, ad field) per cross field."""
    w = (ctypes.c_int32 * len(widths))(*widths)
    r = (ctypes.c_int64 * len(table_rows))(*table_rows)
    flat = [v for pr in (cross_pairs or ()) for v in pr]
    cp = (ctypes.c_int32 * len(flat))(*flat) if flat else None
    d = cold_model_desc(n_user=n_user, n_seq=n_seq, n_ad=n_ad, n_cross=n_cross,
                        emb_dim=emb_dim,
                        id_kind=COLD_IDS_HASHED_U64 if hashed else COLD_IDS_DIRECT_I32,
                        dtype=DTYPES[dtype] if isinstance(dtype, str) else dtype,
                        se_reduction=se_reduction, n_layers=len(widths) - 1,
                        widths=w, table_rows=r, linear_log=int(bool(linear_log)),
                        topk_k=topk_k,
                        cross_pairs=ctypes.cast(cp, ctypes.POINTER(ctypes.c_int32)) if cp else None,
                        se_form=se_form)
    return d, (w, r, cp)


# ---------------------------------------------------------------- wrapper
def _ptr(t) -> Optional[int]:
    return None if t is None else int(t.data_ptr())


class ColdModel:
    """One model on one device: torch supplies the arena, workspace and the
    current stream; libcold.so does the work."""

    def __init__(self, cfg, device="cuda"):
        import torch
        self.torch = torch
        self.cfg = cfg
        self.device = torch.device(device)
        self.desc, self._desc_keep = make_desc(
            cfg.n_user, cfg.n_seq, cfg.n_ad, cfg.n_cross, cfg.emb_dim, cfg.dtype,
            cfg.se_reduction, cfg.widths, [cfg.vocab] * cfg.n_groups, hashed=cfg.hashed,
            linear_log=cfg.linear_log, topk_k=cfg.topk_k,
            cross_pairs=getattr(cfg, "cross_pairs", None) or None,
            se_form=COLD_SE_LITERAL if getattr(cfg, "se_form", "squeeze") == "literal"
            else COLD_SE_SQUEEZE)
        self.h = cold_create_model(self.desc)
        self.arena = torch.empty(cold_weight_arena_bytes(self.h), dtype=torch.uint8,
                                 device=self.device)
        self.workspace = None
        self._keep = None

    def close(self):
        if getattr(self, "h", None) is not None:
            cold_destroy_model(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _stream(self) -> int:
        return int(self.torch.cuda.current_stream(self.device).cuda_stream)

    def load(self, tables, params) -> None:
        """tables: list of device tensors [rows][d]; params: dict with se_w1,
        se_b1, se_w2, se_b2 (fp32) and mlp_w (dtype), mlp_b (fp32) lists of
        device tensors."""
        tabs = (ctypes.c_void_p * len(tables))(*[_ptr(t) for t in tables])
        ws = (ctypes.c_void_p * len(params["mlp_w"]))(*[_ptr(t) for t in params["mlp_w"]])
        bs = (ctypes.c_void_p * len(params["mlp_b"]))(*[_ptr(t) for t in params["mlp_b"]])
        def opt(t):   # an empty tensor (unused SE parameters) travels as NULL
            return None if t.numel() == 0 else _ptr(t)
        w = cold_weights(tables=tabs, se_w1=_ptr(params["se_w1"]), se_b1=_ptr(params["se_b1"]),
                         se_w2=opt(params["se_w2"]), se_b2=opt(params["se_b2"]),
                         mlp_w=ws, mlp_b=bs)
        st = cold_load_weights(self.h, w, _ptr(self.arena), self.arena.numel(), self._stream())
        if st != COLD_OK:
            raise ColdError(st, "cold_load_weights: " + cold_last_error(self.h))
        self._keep = (tables, params)

    def ensure_workspace(self, n_rows: int, n_requests: int):
        need = cold_workspace_bytes(self.h, n_rows, n_requests)
        if self.workspace is None or self.workspace.numel() < need:
            self.workspace = self.torch.empty(max(need, 256), dtype=self.torch.uint8,
                                              device=self.device)
        return self.workspace

    @staticmethod
    def make_batch_struct(batch: dict) -> cold_batch:
        """batch: dict of device tensors req_off, user_ids, ad_ids, cross_ids,
        seq_off, seq_ids (as produced by :func:`batch_to_device`)."""
        req_off = batch["req_off"]
        return cold_batch(n_requests=req_off.numel() - 1, n_rows=int(batch["n_rows"]),
                          n_seq_ids=int(batch["seq_ids"].numel()) if batch.get("seq_ids") is not None else 0,
                          req_off=_ptr(req_off), user_ids=_ptr(batch["user_ids"]),
                          ad_ids=_ptr(batch["ad_ids"]), cross_ids=_ptr(batch["cross_ids"]),
                          seq_off=_ptr(batch.get("seq_off")), seq_ids=_ptr(batch.get("seq_ids")))

    def prepare(self, batch: dict, scores, importance=None, group_mask=None, rows_out=None,
                validate=False, workspace=None, x_out=None) -> "ScoreCall":
        """The same call as score() on fixed device buffers, on the current
        stream, prepared once: calling the result enqueues it (for serving
        loops that reuse their input and output buffers; the buffers must
        stay alive and in place)."""
        return ScoreCall(self, batch, scores, importance, group_mask, rows_out, workspace, x_out,
                         validate, self._stream())

    def score(self, batch: dict, scores=None, importance=None, group_mask=None, rows_out=None,
              validate=False, workspace=None, x_out=None):
        """Score every row; returns the fp32 score tensor (asynchronous on
        the current stream unless validate).  Concurrent calls on different
        streams pass distinct `workspace` tensors (uint8, device, at least
        cold_workspace_bytes); by default the model's own workspace is used."""
        torch = self.torch
        b = self.make_batch_struct(batch)
        ws = self.ensure_workspace(b.n_rows, b.n_requests) if workspace is None else workspace
        if scores is None:
            scores = torch.empty(b.n_rows, dtype=torch.float32, device=self.device)
        st = cold_score(self.h, b, _ptr(ws), ws.numel(), _ptr(scores), _ptr(importance),
                        _ptr(group_mask), _ptr(rows_out), _ptr(x_out),
                        COLD_SCORE_VALIDATE if validate else 0, self._stream())
        if st != COLD_OK:
            raise ColdError(st, "cold_score: " + cold_last_error(self.h))
        return scores


class ScoreCall:
    """One cold_score call on fixed buffers, ready to enqueue again and
    again (see ColdModel.prepare): the batch struct, the pointers and the
    stream are resolved once, so a call costs the C function alone."""

    def __init__(self, model, batch, scores, importance, group_mask, rows_out, workspace, x_out,
                 validate, stream):
        self._keep = (model, batch, scores, importance, group_mask, rows_out, workspace, x_out)
        self._b = model.make_batch_struct(batch)
        ws = (model.ensure_workspace(self._b.n_rows, self._b.n_requests)
              if workspace is None else workspace)
        self._ws = ws
        vp = ctypes.c_void_p
        self._fn = lib().cold_score
        self._h = model.h
        self._args = (model.h, ctypes.byref(self._b), vp(_ptr(ws)), ctypes.c_size_t(ws.numel()),
                      vp(_ptr(scores)), vp(_ptr(importance)), vp(_ptr(group_mask)),
                      vp(_ptr(rows_out)), vp(_ptr(x_out)),
                      ctypes.c_int32(COLD_SCORE_VALIDATE if validate else 0), vp(stream))
        self.scores = scores

    def __call__(self):
        st = self._fn(*self._args)
        if st != COLD_OK:
            raise ColdError(st, "cold_score: " + cold_last_error(self._h))
        return self.scores


def batch_to_device(batch: dict, device="cuda") -> dict:
    """Move a numpy batch (see synth.make_batch) to device tensors; uint64 ids
    travel as int64 with the same bits."""
    import torch

    def t(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint64:
            a = a.view(np.int64)
        if a.size == 0:
            a = np.zeros(1, a.dtype)
        return torch.from_numpy(a).to(device)

    out = {k: t(batch[k]) for k in ("req_off", "user_ids", "ad_ids", "cross_ids",
                                      "seq_off", "seq_ids")}
    out["n_rows"] = int(batch["n_rows"])
    if np.asarray(batch["seq_ids"]).size == 0:
        out["seq_ids"] = None
    return out


def params_to_device(params: dict, dtype: str, device="cuda") -> dict:
    """SE parameters as fp32 and MLP weights in the model dtype (the values
    are exact in it), biases fp32."""
    import torch
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype]
    out = {k: torch.from_numpy(np.ascontiguousarray(params[k], np.float32)).to(device)
           for k in ("se_w1", "se_b1", "se_w2", "se_b2")}
    out["mlp_w"] = []
    for w in params["mlp_w"]:
        tw = torch.from_numpy(np.ascontiguousarray(w, np.float32))
        cw = tw.to(tdt)
        if not torch.equal(cw.to(torch.float32), tw):
            raise ValueError("MLP weight not exact in " + dtype)
        out["mlp_w"].append(cw.contiguous().to(device))
    out["mlp_b"] = [torch.from_numpy(np.ascontiguousarray(b, np.float32)).to(device)
                    for b in params["mlp_b"]]
    return out
