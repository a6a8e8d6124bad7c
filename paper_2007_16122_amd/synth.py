"""Seeded synthetic inputs for the COLD scoring path.

This module draws the inputs that both the HIP path and the CPU checker consume:
request batches (id columns, request offsets, behaviour sequences), embedding
tables and model parameters.  It holds none of the scoring arithmetic (no id
hashing, pooling, squeeze-excitation, normalisation or MLP).

The paper's workload is production traffic of an advertising system
(Section 4.1), which is not public; the configurations below stand in for it
with the shapes of the paper's model (embedding dim 16, FCN widths
D_in x 1024 x 512 x 256 x 128 x 64 x 2, Section 4.1) and candidate sets of
thousands of ads per request (Section 2).

Every value that lands in an embedding table or an MLP weight is a small
integer times a power of two, so it is exactly representable in fp32, bf16 and
fp16; all consumers therefore see identical parameters with no conversion
ambiguity.  Table values come from a counter-based 32-bit hash (MurmurHash3's
fmix32 finaliser) of (table key, row, element), implemented twice below, once
for numpy and once for torch, with bit-identical results, so a large table can
be generated on the GPU while the CPU checker regenerates exactly the rows it
needs.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

__all__ = [
    "ColdConfig", "CONFIGS", "config", "make_batch", "make_params",
    "table_numpy", "table_torch", "table_rows_numpy", "zipf_ranks", "make_bids",
]

MASK32 = 0xFFFFFFFF


# ----------------------------------------------------------------------------
# Configurations
# ----------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class ColdConfig:
    """Shape of one scoring workload.

    Groups are ordered user single-valued, user sequence, ad, cross.  Every
    field is one feature group with its own table of ``vocab`` rows.
    """
    name: str
    n_requests: int
    cand_per_request: int
    n_user: int
    n_seq: int
    n_ad: int
    n_cross: int
    emb_dim: int
    vocab: int
    zipf_s: float
    dtype: str                 # "f32" | "bf16" | "f16"
    se_reduction: int
    widths: tuple              # (D_in, hidden..., n_out)
    head: str                  # "sigmoid1" | "softmax2"
    linear_log: bool = False
    hashed: bool = False       # raw uint64 ids hashed into the tables
    topk_k: int = 0            # 0: no group mask
    emit_importance: bool = False
    seq_len_max: int = 50
    init: str = "he"           # "normal005" | "he"
    seq_table: str = "tri"     # value scheme of the sequence tables
    out_gain: float = 15.0     # output-layer scale relative to He init ("he" init)
    out_bias: float = -2.0     # output-layer bias of the click class ("he" init)
    seed: int = 2007_16122
    # () : cross ids come with the batch; else ((user field, ad field), ...)
    # per cross field, and the cross ids are built on the GPU from the pair
    cross_pairs: tuple = ()
    # "squeeze": SE as squeeze -> FC -> ReLU -> FC -> sigmoid; "literal": one
    # FC from the concatenated embeddings to the M weights (Eq. 2 as printed)
    se_form: str = "squeeze"

    @property
    def n_groups(self) -> int:
        return self.n_user + self.n_seq + self.n_ad + self.n_cross

    @property
    def d_in(self) -> int:
        return self.n_groups * self.emb_dim

    @property
    def se_hidden(self) -> int:
        return max(1, self.n_groups // self.se_reduction)

    @property
    def n_rows(self) -> int:
        return self.n_requests * self.cand_per_request

    def group_kind(self, g: int) -> str:
        if g < self.n_user:
            return "user"
        if g < self.n_user + self.n_seq:
            return "seq"
        if g < self.n_user + self.n_seq + self.n_ad:
            return "ad"
        return "cross"

    def table_scheme(self, g: int) -> str:
        return self.seq_table if self.group_kind(g) == "seq" else "tri"


def _mlp(d_in):
    return (d_in, 1024, 512, 256, 128, 64, 2)


CONFIGS = {
    # 1 request x 512 ads, 4/8/4 single-valued fields, vocab 10k, d = 8.
    "tiny_fp32": ColdConfig(
        name="tiny_fp32", n_requests=1, cand_per_request=512,
        n_user=4, n_seq=0, n_ad=8, n_cross=4, emb_dim=8, vocab=10_000,
        zipf_s=1.1, dtype="f32", se_reduction=4, widths=(128, 64, 32, 1),
        head="sigmoid1", init="normal005", seed=2007_16122 + 0),
    # 32 requests x 2000 ads, 12/24/12 fields, 1M-row tables, bf16.
    "serving_bf16": ColdConfig(
        name="serving_bf16", n_requests=32, cand_per_request=2000,
        n_user=12, n_seq=0, n_ad=24, n_cross=12, emb_dim=16, vocab=1_000_000,
        zipf_s=1.05, dtype="bf16", se_reduction=4, widths=_mlp(48 * 16),
        head="softmax2", seed=2007_16122 + 1),
    # as serving, plus 6 sum-pooled behaviour sequences; fp16 + linear_log.
    "multivalued_fp16_ll": ColdConfig(
        name="multivalued_fp16_ll", n_requests=32, cand_per_request=2000,
        n_user=12, n_seq=6, n_ad=24, n_cross=12, emb_dim=16, vocab=1_000_000,
        zipf_s=1.05, dtype="f16", se_reduction=4, widths=_mlp(54 * 16),
        head="softmax2", linear_log=True, seq_table="big", out_gain=0.19,
        seed=2007_16122 + 2),
    # 128 requests x 10k ads, 64 fields with 10M-row hashed tables, fp16.
    "large_fp16_ll": ColdConfig(
        name="large_fp16_ll", n_requests=128, cand_per_request=10_000,
        n_user=16, n_seq=0, n_ad=32, n_cross=16, emb_dim=16, vocab=10_000_000,
        zipf_s=1.0, dtype="f16", se_reduction=4, widths=_mlp(64 * 16),
        head="softmax2", linear_log=True, hashed=True, seed=2007_16122 + 3),
    # 1 request x 5000 ads, 200 fields; SE importance + top-k group mask.
    "wide_prune_bf16": ColdConfig(
        name="wide_prune_bf16", n_requests=1, cand_per_request=5000,
        n_user=50, n_seq=0, n_ad=100, n_cross=50, emb_dim=16,
        vocab=1_000_000, zipf_s=1.05, dtype="bf16", se_reduction=4,
        widths=_mlp(200 * 16), head="softmax2", topk_k=100,
        emit_importance=True, seed=2007_16122 + 4),
}


def config(name: str, **overrides) -> ColdConfig:
    """A named configuration, optionally with fields replaced (e.g. a smaller
    vocabulary or fewer requests for a quick test).  ``widths[0]`` follows the
    group count and embedding dim unless given explicitly."""
    cfg = CONFIGS[name]
    if overrides:
        cfg = dataclasses.replace(cfg, **overrides)
        if "widths" not in overrides and cfg.widths[0] != cfg.d_in:
            cfg = dataclasses.replace(cfg, widths=(cfg.d_in,) + tuple(cfg.widths[1:]))
    return cfg


# ----------------------------------------------------------------------------
# Ids: bounded Zipf ranks (inverse CDF), scattered over the id space
# ----------------------------------------------------------------------------
_CDF_CACHE: dict = {}


def _zipf_cdf(n: int, s: float) -> np.ndarray:
    key = (n, s)
    if key not in _CDF_CACHE:
        w = np.arange(1, n + 1, dtype=np.float64) ** (-s)
        c = np.cumsum(w)
        c /= c[-1]
        _CDF_CACHE.clear()
        _CDF_CACHE[key] = c
    return _CDF_CACHE[key]


_TORCH_CDF: dict = {}


def zipf_ranks(rng: np.random.Generator, n: int, s: float, size: int,
               device=None) -> np.ndarray:
    """0-based ranks k with P(k) proportional to (k+1)^(-s), k < n.  Bounded,
    so any s > 0 (including s <= 1) is valid.  With ``device`` the inverse-CDF
    search runs in torch there; the comparisons are exact fp64 either way, so
    the ranks are identical."""
    cdf = _zipf_cdf(n, s)
    u = rng.random(size)
    if device is None or size < (1 << 20):
        k = np.searchsorted(cdf, u, side="right")
    else:
        import torch
        key = (n, s, str(device))
        if key not in _TORCH_CDF:
            _TORCH_CDF.clear()
            _TORCH_CDF[key] = torch.from_numpy(cdf).to(device)
        k = torch.searchsorted(_TORCH_CDF[key], torch.from_numpy(u).to(device),
                               right=True).cpu().numpy()
    return np.minimum(k, n - 1).astype(np.int64)


def _coprime_multiplier(rng: np.random.Generator, n: int) -> int:
    while True:
        a = int(rng.integers(1, n))
        if math.gcd(a, n) == 1:
            return a


def _ids_for_field(rng, cfg: ColdConfig, size: int, device=None) -> np.ndarray:
    """Ids of one field: Zipf ranks mapped to ids by a per-field bijection so
    the hot ids are scattered over the table (direct ids, int32) or over the
    64-bit raw id space (hashed ids, uint64)."""
    ranks = zipf_ranks(rng, cfg.vocab, cfg.zipf_s, size, device)
    if not cfg.hashed:
        a = _coprime_multiplier(rng, cfg.vocab)
        b = int(rng.integers(0, cfg.vocab))
        return ((ranks * a + b) % cfg.vocab).astype(np.int32)
    # raw ids: an odd multiplier is a bijection of Z / 2^64
    a = np.uint64(int(rng.integers(0, 2**62)) * 2 + 1)
    b = np.uint64(int(rng.integers(0, 2**63)))
    with np.errstate(over="ignore"):
        return ranks.astype(np.uint64) * a + b


def make_bids(cfg: ColdConfig, n_rows: int, seed: Optional[int] = None) -> np.ndarray:
    """CPC bids of the candidate rows (fp32, whole cents, log-normal around
    0.50 and clipped to 0.01 .. 50.00).  The paper's selection metric is
    eCPM = pCTR * bid (Section 2); its bids are not published."""
    seed = cfg.seed if seed is None else seed
    rng = np.random.default_rng(np.random.SeedSequence([seed, 0xB1D5]))
    cents = np.rint(np.exp(rng.normal(np.log(50.0), 0.7, size=n_rows)))
    return (np.clip(cents, 1, 5000) / 100.0).astype(np.float32)


def make_batch(cfg: ColdConfig, seed: Optional[int] = None,
               cand_per_request=None, device=None) -> dict:
    """One request batch in the column (field-major) layout.

    Returns numpy arrays::

        req_off   int32 [Q+1]            rows of request q: req_off[q]..req_off[q+1]
        user_ids  [n_user][Q]            int32 (direct) or uint64 (hashed)
        ad_ids    [n_ad][R]
        cross_ids [n_cross][R]
        seq_off   int32 [n_seq*Q + 1]    ids of (field f, request q) at entry f*Q+q
        seq_ids   [total]

    ``cand_per_request`` may be a list of per-request candidate counts
    (ragged batches, empty requests allowed).  ``device`` (e.g. "cuda")
    only speeds up the Zipf inverse-CDF search; the result is the same.
    """
    seed = cfg.seed if seed is None else seed
    ss = np.random.SeedSequence([seed, 0xB47C])
    rngs = [np.random.default_rng(s) for s in ss.spawn(4 + cfg.n_groups)]
    q_count = cfg.n_requests
    if cand_per_request is None:
        cands = np.full(q_count, cfg.cand_per_request, dtype=np.int64)
    else:
        cands = np.asarray(cand_per_request, dtype=np.int64)
        q_count = len(cands)
    req_off = np.zeros(q_count + 1, dtype=np.int32)
    req_off[1:] = np.cumsum(cands)
    n_rows = int(req_off[-1])
    id_dtype = np.uint64 if cfg.hashed else np.int32
    g = 0
    user_ids = np.zeros((cfg.n_user, q_count), dtype=id_dtype)
    for f in range(cfg.n_user):
        user_ids[f] = _ids_for_field(rngs[4 + g], cfg, q_count)
        g += 1
    seq_len_rng = rngs[0]
    lens = seq_len_rng.integers(1, cfg.seq_len_max + 1, size=cfg.n_seq * q_count)
    seq_off = np.zeros(cfg.n_seq * q_count + 1, dtype=np.int32)
    seq_off[1:] = np.cumsum(lens)
    seq_ids = np.zeros(int(seq_off[-1]), dtype=id_dtype)
    for f in range(cfg.n_seq):
        lo, hi = seq_off[f * q_count], seq_off[(f + 1) * q_count]
        seq_ids[lo:hi] = _ids_for_field(rngs[4 + g], cfg, int(hi - lo))
        g += 1
    ad_ids = np.zeros((cfg.n_ad, n_rows), dtype=id_dtype)
    for f in range(cfg.n_ad):
        ad_ids[f] = _ids_for_field(rngs[4 + g], cfg, n_rows, device)
        g += 1
    if cfg.cross_pairs:      # built from the user and ad ids by the scorer
        cross_ids = np.zeros((cfg.n_cross, 0), dtype=id_dtype)
    else:
        cross_ids = np.zeros((cfg.n_cross, n_rows), dtype=id_dtype)
        for f in range(cfg.n_cross):
            cross_ids[f] = _ids_for_field(rngs[4 + g], cfg, n_rows, device)
            g += 1
    return dict(req_off=req_off, user_ids=user_ids, ad_ids=ad_ids,
                cross_ids=cross_ids, seq_off=seq_off, seq_ids=seq_ids,
                n_requests=q_count, n_rows=n_rows)


# ----------------------------------------------------------------------------
# Embedding tables: counter-based values, identical in numpy and torch
# ----------------------------------------------------------------------------
_C1, _C2, _GOLD = 0x85EBCA6B, 0xC2B2AE35, 0x9E3779B9


def table_keys(cfg: ColdConfig, g: int, seed: Optional[int] = None):
    seed = cfg.seed if seed is None else seed
    k = np.random.SeedSequence([seed, 0x7AB1E, g]).generate_state(2)
    return int(k[0]), int(k[1])


def _mul32(x, c: int):
    """(x * c) mod 2^32 for 0 <= x < 2^32 held in int64, without int64
    overflow: the constant is split in 16-bit halves."""
    lo, hi = c & 0xFFFF, c >> 16
    return (x * lo + (((x * hi) & 0xFFFF) << 16)) & MASK32


def _fmix32(h):
    h = h ^ (h >> 16)
    h = _mul32(h, _C1)
    h = h ^ (h >> 13)
    h = _mul32(h, _C2)
    return h ^ (h >> 16)


def _hash_elems(rows, elem, k0: int, k1: int):
    """32-bit hash of (row, element) under the table keys; rows and elem are
    broadcastable int64 arrays/tensors with values < 2^32."""
    h = _fmix32(rows ^ k0)
    return _fmix32(h ^ _mul32(elem + 1, _GOLD) ^ k1)


def _values_from_hash(h, scheme: str):
    """Small integer k and the power-of-two scale: value = k * 2^scale."""
    if scheme == "tri":      # triangular on [-255, 255] * 2^-11, std ~0.051
        return ((h & 0xFF) + ((h >> 8) & 0xFF) - 255), -11
    if scheme == "big":      # uniform on [-1024, 1023] * 16 (|v| <= 16384)
        return (((h >> 16) & 0x7FF) - 1024), 4
    if scheme == "int":      # small integers [-8, 7]
        return ((h & 0xF) - 8), 0
    raise ValueError(scheme)


def _np_store(vals_f32: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return vals_f32.astype(np.float32)
    if dtype == "f16":
        out = vals_f32.astype(np.float16)
        assert np.array_equal(out.astype(np.float32), vals_f32)
        return out
    if dtype == "bf16":
        bits = vals_f32.astype(np.float32).view(np.uint32)
        assert not np.any(bits & 0xFFFF), "value not exact in bf16"
        return (bits >> 16).astype(np.uint16)
    raise ValueError(dtype)


def table_rows_numpy(cfg: ColdConfig, g: int, rows: np.ndarray,
                     seed: Optional[int] = None, scheme: Optional[str] = None) -> np.ndarray:
    """Rows ``rows`` of table g as stored: float32, float16, or uint16 bf16
    bit patterns; shape [len(rows)][emb_dim]."""
    k0, k1 = table_keys(cfg, g, seed)
    r = np.asarray(rows, dtype=np.int64)[:, None]
    e = np.arange(cfg.emb_dim, dtype=np.int64)[None, :]
    kk, sc = _values_from_hash(_hash_elems(r, e, k0, k1),
                               scheme or cfg.table_scheme(g))
    vals = np.ldexp(kk.astype(np.float64), sc).astype(np.float32)
    return _np_store(vals, cfg.dtype)


def table_numpy(cfg: ColdConfig, g: int, seed: Optional[int] = None,
                scheme: Optional[str] = None) -> np.ndarray:
    return table_rows_numpy(cfg, g, np.arange(cfg.vocab), seed, scheme)


def table_torch(cfg: ColdConfig, g: int, device="cpu", seed: Optional[int] = None,
                scheme: Optional[str] = None, chunk_rows: int = 1 << 22):
    """The same table as :func:`table_numpy`, built with torch ops on
    ``device``; bfloat16 tables come back as torch.bfloat16."""
    import torch
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[cfg.dtype]
    k0, k1 = table_keys(cfg, g, seed)
    out = torch.empty((cfg.vocab, cfg.emb_dim), dtype=tdt, device=device)
    e = torch.arange(cfg.emb_dim, dtype=torch.int64, device=device)[None, :]
    for lo in range(0, cfg.vocab, chunk_rows):
        hi = min(cfg.vocab, lo + chunk_rows)
        r = torch.arange(lo, hi, dtype=torch.int64, device=device)[:, None]
        kk, sc = _values_from_hash(_hash_elems(r, e, k0, k1),
                                   scheme or cfg.table_scheme(g))
        out[lo:hi] = (kk.to(torch.float32) * (2.0 ** sc)).to(tdt)
    return out


# ----------------------------------------------------------------------------
# Model parameters
# ----------------------------------------------------------------------------
def _quantised_normal(rng, sigma: float, shape) -> np.ndarray:
    """N(0, sigma) rounded to k * 2^-e with |k| <= 255 (exact in bf16/fp16),
    e chosen so that sigma * 2^e is about 48."""
    e = int(round(math.log2(48.0 / sigma)))
    k = np.clip(np.round(rng.normal(0.0, sigma, shape) * 2.0 ** e), -255, 255)
    return np.ldexp(k, -e).astype(np.float32)


def make_params(cfg: ColdConfig, seed: Optional[int] = None) -> dict:
    """SE block and MLP parameters (float32 values; MLP weights are exact in
    the config's dtype).

    ``normal005``: every parameter N(0, 0.05) (the tiny fp32 workload).
    ``he``: SE W1 ~ N(0, 10/sqrt(M)), b1 ~ N(0, 0.1), W2 ~ N(0, 1/sqrt(H)),
    b2 ~ N(0, 1) (so groups differ in importance); hidden MLP layers
    N(0, sqrt(2/fan_in)) with biases N(0, 0.01); the output layer at
    ``out_gain`` (15) times that scale with bias ``out_bias`` (-2) on the
    click class.  The behaviour-sequence workload, whose linear_log'd pooled
    groups are about 300 times larger than an embedding, takes the gain that
    gives its logit the spread of the serving workload's at 15 (0.19).
    Its SE W1 columns of the pooled groups are scaled by 2^-20 (see below).
    """
    seed = cfg.seed if seed is None else seed
    rng = np.random.default_rng(np.random.SeedSequence([seed, 0x5E, 0x3A]))
    m, h = cfg.n_groups, cfg.se_hidden
    f32 = np.float32
    if cfg.init == "normal005":
        se_w1 = rng.normal(0, 0.05, (h, m)).astype(f32)
        se_b1 = rng.normal(0, 0.05, h).astype(f32)
        se_w2 = rng.normal(0, 0.05, (m, h)).astype(f32)
        se_b2 = rng.normal(0, 0.05, m).astype(f32)
    else:
        se_w1 = rng.normal(0, 10.0 / math.sqrt(m), (h, m)).astype(f32)
        se_b1 = rng.normal(0, 0.1, h).astype(f32)
        se_w2 = rng.normal(0, 1.0 / math.sqrt(h), (m, h)).astype(f32)
        se_b2 = rng.normal(0, 1.0, m).astype(f32)
        if cfg.n_seq and cfg.seq_table == "big":
            # the squeeze of a pooled large-value sequence group is about
            # 2^20 times that of an embedding group (std ~1.2e4 against
            # ~0.013); its W1 columns are scaled by 2^-20 so that it moves
            # the SE logits as much as any other group, instead of driving
            # every weight to 0 or 1
            se_w1[:, cfg.n_user:cfg.n_user + cfg.n_seq] *= f32(2.0 ** -20)
    if cfg.se_form == "literal":
        # se_w1 [M][D_in], se_b1 [M]; drawn from a stream of their own so the
        # network weights are those of the squeeze form of the same workload
        lrng = np.random.default_rng(np.random.SeedSequence([seed, 0x5E, 0x1E]))
        se_w1 = lrng.normal(0, 30.0 / math.sqrt(cfg.d_in), (m, cfg.d_in)).astype(f32)
        se_b1 = lrng.normal(0, 0.5, m).astype(f32)
        se_w2 = np.zeros((m, 0), f32)
        se_b2 = np.zeros(0, f32)
    ws, bs = [], []
    n_layers = len(cfg.widths) - 1
    for li in range(n_layers):
        fi, fo = cfg.widths[li], cfg.widths[li + 1]
        last = li == n_layers - 1
        if cfg.init == "normal005":
            w = rng.normal(0, 0.05, (fo, fi)).astype(f32)
            b = rng.normal(0, 0.05, fo).astype(f32)
            if cfg.dtype != "f32":
                w = _quantised_normal(rng, 0.05, (fo, fi))
        else:
            sig = math.sqrt(2.0 / fi) * (cfg.out_gain if last else 1.0)
            w = _quantised_normal(rng, sig, (fo, fi))
            if last:
                b = np.zeros(fo, f32)
                b[-1] = cfg.out_bias
            else:
                b = rng.normal(0, 0.01, fo).astype(f32)
        ws.append(w)
        bs.append(b)
    return dict(se_w1=se_w1, se_b1=se_b1, se_w2=se_w2, se_b2=se_b2,
                mlp_w=ws, mlp_b=bs)


def mlp_weight_stored(w: np.ndarray, dtype: str) -> np.ndarray:
    """An MLP weight matrix in its stored form (float32, float16 or bf16 bits)."""
    return _np_store(np.asarray(w, np.float32), dtype)
