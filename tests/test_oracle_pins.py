"""Pins of the CPU checker against things other than itself: values fixed by
the paper's equations (golden files), published test vectors, closed forms,
invariants of the method, and an independent dense numpy formulation on tiny
inputs.  No GPU needed."""
import math
import os

import numpy as np
import pytest

import oracle
from paper_2007_16122_amd import synth
from tests import bruteforce
from tests.common import dims_of, problem, stored_params, table_f64, tiny

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
CONFIG_NAMES = list(synth.CONFIGS)


def _read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.split("#")[0].strip()
            if line:
                rows.append(line.split())
    return rows


def _parse_x(tok):
    sign = -1.0 if tok.startswith("-") else 1.0
    tok = tok.lstrip("-")
    if tok.startswith("e^"):
        return sign * math.exp(float(tok[2:]))
    return sign * float(tok)


def run_oracle(cfg, tables, params, batch, **kw):
    return oracle.score(dims_of(cfg), tables, stored_params(cfg, params), batch, **kw)


def run_brute(cfg, tables, params, batch):
    return bruteforce.forward(dims_of(cfg), [table_f64(cfg, t) for t in tables], params,
                              [np.asarray(w, np.float64) for w in params["mlp_w"]],
                              [np.asarray(b, np.float64) for b in params["mlp_b"]], batch)


# ------------------------------------------------- stored-value decoding
def _same_f64(got, want):
    """Equal as float64 bit patterns, except that any NaN matches any NaN."""
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan].view(np.uint64), want[~nan].view(np.uint64))


def test_decode_f16_every_pattern():
    """The checker's binary16 decoder on all 65,536 bit patterns (normals,
    subnormals, signed zeros, infinities, NaNs) against numpy's own
    float16 -> float64 widening."""
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    want = bits.view(np.float16).astype(np.float64)
    got = oracle.decode_stored("f16", bits.view(np.float16))
    _same_f64(got, want)
    # the classes the synthetic inputs never produce are really covered
    assert np.sum(np.isnan(want)) == 2 * 1023 and np.sum(np.isinf(want)) == 2
    assert np.sum((want != 0) & (np.abs(want) < 2.0 ** -14)) == 2 * 1023


def test_decode_bf16_every_pattern():
    """bfloat16 patterns against the upper half of a binary32 pattern
    widened by numpy."""
    bits = np.arange(1 << 16, dtype=np.uint32)
    want = (bits << 16).astype(np.uint32).view(np.float32).astype(np.float64)
    got = oracle.decode_stored("bf16", bits.astype(np.uint16))
    _same_f64(got, want)


def test_decode_f32_passthrough():
    v = np.array([0.0, -0.0, 1.5, -3.25e-41, np.inf, -np.inf, 3.4e38], np.float32)
    _same_f64(oracle.decode_stored("f32", v), v.astype(np.float64))


# --------------------------------------------------------------- Eq. 3
def test_linear_log_golden():
    for x_tok, want in _read_golden("linear_log.txt"):
        x = _parse_x(x_tok)
        assert oracle.linear_log(x) == pytest.approx(float(want), abs=1e-12), x_tok


def test_linear_log_c1_and_odd():
    # C^1 at the joins: one-sided slopes at +-1 equal 1 (Eq. 3 claim)
    for x0 in (1.0, -1.0):
        for hh in (1e-6, -1e-6):
            slope = (oracle.linear_log(x0 + hh) - oracle.linear_log(x0)) / hh
            assert slope == pytest.approx(1.0, abs=1e-5)
    xs = np.concatenate([np.linspace(-50, 50, 1001), [65504.0, -65504.0, 1e30]])
    for x in xs:
        assert oracle.linear_log(-x) == -oracle.linear_log(x)
    ys = [oracle.linear_log(x) for x in np.sort(xs)]
    assert all(b >= a for a, b in zip(ys, ys[1:]))        # monotone


# ----------------------------------------------------- hashed id rows
def test_mix64_published_vector():
    rows = _read_golden("splitmix64.txt")
    seed = int(rows[0][1])
    want = [int(r[0]) for r in rows[1:]]
    state = seed
    for w in want:
        state = (state + 0x9E3779B97F4A7C15) & bruteforce.MASK64
        assert oracle.mix64(state) == w
        assert bruteforce.mix64_int(state) == w


def test_hash_row_matches_integer_definition():
    rng = np.random.default_rng(5)
    for _ in range(200):
        raw = int(rng.integers(0, 2**63)) * 2 + int(rng.integers(0, 2))
        g = int(rng.integers(0, 300))
        rows = int(rng.integers(1, 10**8))
        assert oracle.hash_row(raw, g, rows) == bruteforce.hashed_row(raw, g, rows)


def test_cross_key_matches_integer_definition():
    rng = np.random.default_rng(6)
    for _ in range(200):
        u = int(rng.integers(0, 2**63)) * 2 + int(rng.integers(0, 2))
        a = int(rng.integers(0, 2**63)) * 2 + int(rng.integers(0, 2))
        assert oracle.cross_key(u, a) == bruteforce.mix64_int(u) ^ a
    # the mixing function fixes 0, so a zero user id leaves the ad id as is
    assert oracle.cross_key(0, 12345) == 12345


@pytest.mark.parametrize("name,hashed", [("serving_bf16", False), ("large_fp16_ll", True)])
def test_oracle_gpu_cross_features_match_bruteforce(name, hashed):
    """Cross ids built from (user field, ad field) pairs: rows and scores
    against the dense formulation, which derives the rows with Python
    integers."""
    base = tiny(name)
    pairs = tuple((f % base.n_user, (3 * f + 1) % base.n_ad) for f in range(base.n_cross))
    cfg = tiny(name, cross_pairs=pairs)
    assert cfg.hashed == hashed
    tables, params, batch = problem(cfg, seed=12, cand=[5, 0, 7])
    assert batch["cross_ids"].shape[1] == 0
    o = run_oracle(cfg, tables, params, batch, want_rows=True, want_x=True)
    b = run_brute(cfg, tables, params, batch)
    assert np.array_equal(o["rows"], b["rows"])
    np.testing.assert_allclose(o["x"], b["x"], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(o["scores"], b["scores"], rtol=1e-11, atol=1e-13)


@pytest.mark.parametrize("name", ["tiny_fp32", "serving_bf16", "multivalued_fp16_ll",
                                  "wide_prune_bf16"])
def test_oracle_literal_se_matches_bruteforce(name):
    """Eq. 2 as printed (one FC over the concatenated embeddings): importance
    weights, network input and scores against the dense formulation."""
    cfg = tiny(name, se_form="literal")
    tables, params, batch = problem(cfg, seed=13, cand=[4, 0, 9])
    assert params["se_w1"].shape == (cfg.n_groups, cfg.d_in)
    o = run_oracle(cfg, tables, params, batch, want_s=True, want_x=True)
    b = run_brute(cfg, tables, params, batch)
    np.testing.assert_allclose(o["s"], b["s"], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(o["x"], b["x"], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(o["scores"], b["scores"], rtol=1e-11, atol=1e-13)
    if cfg.topk_k:
        assert np.array_equal(o["mask"], b["mask"])


def test_literal_se_closed_forms():
    """W = 0 gives s = sigmoid(b) for every row; a W that averages each
    group's own block gives s_g = sigmoid(z_g + b_g), z_g the group mean."""
    cfg = tiny("serving_bf16", se_form="literal")
    tables, params, batch = problem(cfg, seed=14)
    m, d = cfg.n_groups, cfg.emb_dim
    p0 = dict(params, se_w1=np.zeros_like(params["se_w1"]))
    o = run_oracle(cfg, tables, p0, batch, want_s=True)
    want = 1.0 / (1.0 + np.exp(-params["se_b1"].astype(np.float64)))
    np.testing.assert_allclose(o["s"], np.broadcast_to(want, o["s"].shape), rtol=0, atol=1e-15)
    wavg = np.zeros((m, m * d), np.float32)
    for g in range(m):
        wavg[g, g * d:(g + 1) * d] = 1.0 / d          # exact in fp32 (d a power of two)
    o = run_oracle(cfg, tables, dict(params, se_w1=wavg), batch, want_s=True, want_x=True)
    s = o["s"]
    e = o["x"].reshape(-1, m, d) / s[:, :, None]       # x = s * e
    z = e.mean(axis=2)
    np.testing.assert_allclose(s, 1.0 / (1.0 + np.exp(-(z + params["se_b1"]))), rtol=1e-12)


# ----------------------------------------- whole path vs dense formulation
@pytest.mark.parametrize("name", CONFIG_NAMES)
def test_oracle_matches_bruteforce(name):
    cfg = tiny(name)
    tables, params, batch = problem(cfg, seed=11)
    o = run_oracle(cfg, tables, params, batch, want_rows=True, want_s=True, want_x=True)
    b = run_brute(cfg, tables, params, batch)
    assert np.array_equal(o["rows"], b["rows"])
    np.testing.assert_allclose(o["s"], b["s"], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(o["x"], b["x"], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(o["scores"], b["scores"], rtol=1e-11, atol=1e-13)
    if cfg.topk_k:
        assert np.array_equal(o["mask"], b["mask"])
        np.testing.assert_allclose(o["importance"], b["importance"], rtol=1e-12)


@pytest.mark.parametrize("name", ["serving_bf16", "multivalued_fp16_ll"])
def test_oracle_bruteforce_ragged(name):
    """Ragged requests, an empty request, and an empty behaviour sequence."""
    cfg = tiny(name, n_requests=4)
    tables, params, batch = problem(cfg, seed=3, cand=[5, 0, 1, 9])
    if cfg.n_seq:
        # empty the first sequence of request 0
        off = batch["seq_off"].copy()
        cut = off[1] - off[0]
        batch["seq_ids"] = batch["seq_ids"][cut:]
        off[1:] -= cut
        batch["seq_off"] = off
    o = run_oracle(cfg, tables, params, batch, want_x=True)
    b = run_brute(cfg, tables, params, batch)
    np.testing.assert_allclose(o["x"], b["x"], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(o["scores"], b["scores"], rtol=1e-11, atol=1e-13)


# -------------------------------------------------------- closed forms
@pytest.mark.parametrize("name", CONFIG_NAMES)
def test_zero_se_gives_half(name):
    """W1 = b1 = W2 = b2 = 0  =>  s = sigmoid(0) = 1/2 exactly, x = e/2."""
    cfg = tiny(name, linear_log=False)
    tables, params, batch = problem(cfg, seed=2)
    for k in ("se_w1", "se_b1", "se_w2", "se_b2"):
        params[k] = np.zeros_like(params[k])
    o = run_oracle(cfg, tables, params, batch, want_s=True, want_x=True, want_rows=True)
    assert np.all(o["s"] == 0.5)
    b = run_brute(cfg, tables, params, batch)
    if not cfg.topk_k:   # with all s equal, the mask keeps the first k groups
        np.testing.assert_allclose(o["x"], b["x"], rtol=0, atol=0)


def test_w1_zero_gives_sigmoid_b2():
    cfg = tiny("serving_bf16")
    tables, params, batch = problem(cfg, seed=4)
    params["se_w1"] = np.zeros_like(params["se_w1"])
    params["se_b1"] = np.zeros_like(params["se_b1"])
    o = run_oracle(cfg, tables, params, batch, want_s=True)
    want = 1.0 / (1.0 + np.exp(-params["se_b2"].astype(np.float64)))
    np.testing.assert_allclose(o["s"], np.broadcast_to(want, o["s"].shape), rtol=1e-15)


@pytest.mark.parametrize("head", ["sigmoid1", "softmax2"])
def test_constant_network_head(head):
    """All weights zero, output bias c  =>  CTR = sigmoid(c) (one output) or
    sigmoid(c1 - c0) (two outputs, class 1 = click)."""
    n_out = 1 if head == "sigmoid1" else 2
    base = tiny("serving_bf16")
    cfg = tiny("serving_bf16", head=head, widths=(base.d_in, 8, n_out))
    tables, params, batch = problem(cfg, seed=6)
    params["mlp_w"] = [np.zeros_like(w) for w in params["mlp_w"]]
    c = np.array([0.3, -1.7][:n_out], np.float32)
    params["mlp_b"] = [np.zeros(8, np.float32), c]
    o = run_oracle(cfg, tables, params, batch)
    want = 1 / (1 + math.exp(-float(c[0]))) if n_out == 1 else \
        1 / (1 + math.exp(-(float(c[1]) - float(c[0]))))
    np.testing.assert_allclose(o["scores"], want, rtol=1e-15)


def test_integer_tables_pool_exactly():
    """Small-integer tables: gathered and sum-pooled values are integers, so
    x = e/2 (zero SE) is exact and equals a plain integer sum of table rows."""
    cfg = tiny("multivalued_fp16_ll", linear_log=False)
    tables, params, batch = problem(cfg, seed=8, scheme="int")
    for k in ("se_w1", "se_b1", "se_w2", "se_b2"):
        params[k] = np.zeros_like(params[k])
    o = run_oracle(cfg, tables, params, batch, want_x=True)
    q_n = batch["n_requests"]
    d = cfg.emb_dim
    for r in range(batch["n_rows"]):
        q = int(np.searchsorted(batch["req_off"], r, side="right") - 1)
        for f in range(cfg.n_seq):
            g = cfg.n_user + f
            lo, hi = batch["seq_off"][f * q_n + q], batch["seq_off"][f * q_n + q + 1]
            tot = np.zeros(d, np.int64)
            for i in batch["seq_ids"][lo:hi]:
                tot += tables[g][i].astype(np.int64)
            assert np.array_equal(o["x"][r, g * d:(g + 1) * d] * 2, tot)


def test_linear_log_inside_path():
    """Zero SE (s = 1/2) on integer tables: x = LL(e/2) elementwise."""
    cfg = tiny("multivalued_fp16_ll")
    tables, params, batch = problem(cfg, seed=9, scheme="int")
    for k in ("se_w1", "se_b1", "se_w2", "se_b2"):
        params[k] = np.zeros_like(params[k])
    o = run_oracle(cfg, tables, params, batch, want_x=True, want_rows=True)
    d = cfg.emb_dim
    for r in range(3):
        for g in range(cfg.n_groups):
            if cfg.group_kind(g) == "seq":
                continue
            e = tables[g][o["rows"][r, g]].astype(np.float64)
            for k in range(d):
                v = e[k] / 2
                want = v if abs(v) <= 1 else math.copysign(1 + math.log(abs(v)), v)
                assert o["x"][r, g * d + k] == pytest.approx(want, abs=1e-15)


def test_sequence_workload_inputs_exercise_se_and_linear_log():
    """The behaviour-sequence workload's inputs are shaped so that its
    parity checks reach both parts of the method they exist for: the SE
    weights (Section 3.2, Eq. 2) of every group, pooled ones included, stay
    fractional rather than saturating at 0 or 1, and pooled values still
    pass the fp16 range before linear_log (Section 3.3, Eq. 3)."""
    cfg = synth.config("multivalued_fp16_ll", vocab=4000)
    tables, params, batch = problem(cfg, seed=5, cand=[300, 200, 1, 250])
    o = run_oracle(cfg, tables, params, batch, want_s=True, want_x=True)
    s = o["s"]
    saturated = (s < 1e-6) | (s > 1.0 - 1e-6)
    seq = slice(cfg.n_user, cfg.n_user + cfg.n_seq)
    assert saturated.mean() < 0.01 and saturated[:, seq].mean() < 0.01, saturated.mean()
    # every pooled group's weight varies across rows (requests)
    assert np.all(s[:, seq].std(axis=0) > 1e-3)
    # |s e| > 65504 for some pooled coordinates: x = LL(s e) > 1 + ln 65504
    d = cfg.emb_dim
    xs = o["x"][:, cfg.n_user * d:(cfg.n_user + cfg.n_seq) * d]
    frac = np.mean(np.abs(xs) > 1.0 + math.log(65504.0))
    assert frac > 0.001, frac


# ----------------------------------------------------------- invariants
@pytest.mark.parametrize("name", ["tiny_fp32", "serving_bf16", "multivalued_fp16_ll",
                                  "large_fp16_ll"])
def test_permutation_invariance(name):
    """Scores are per-ad independent (Section 3.3): permuting the candidates of
    each request and the order of requests permutes the scores exactly."""
    cfg = tiny(name, n_requests=3)
    tables, params, batch = problem(cfg, seed=12, cand=[4, 7, 6])
    base = run_oracle(cfg, tables, params, batch)["scores"]
    rng = np.random.default_rng(0)
    q_n = batch["n_requests"]
    order_q = rng.permutation(q_n)
    off = batch["req_off"]
    perm_rows, new_off = [], [0]
    for q in order_q:
        rows = np.arange(off[q], off[q + 1])
        perm_rows.append(rng.permutation(rows))
        new_off.append(new_off[-1] + len(rows))
    perm = np.concatenate(perm_rows)
    nb = dict(batch)
    nb["req_off"] = np.asarray(new_off, np.int32)
    nb["user_ids"] = batch["user_ids"][:, order_q]
    nb["ad_ids"] = batch["ad_ids"][:, perm]
    nb["cross_ids"] = batch["cross_ids"][:, perm]
    if cfg.n_seq:
        so, si = batch["seq_off"], batch["seq_ids"]
        offs, ids = [0], []
        for f in range(cfg.n_seq):
            for q in order_q:
                seg = si[so[f * q_n + q]:so[f * q_n + q + 1]]
                ids.append(seg)
                offs.append(offs[-1] + len(seg))
        nb["seq_off"] = np.asarray(offs, np.int32)
        nb["seq_ids"] = np.concatenate(ids)
    got = run_oracle(cfg, tables, params, nb)["scores"]
    assert np.array_equal(got, base[perm])


def split_into_single_row_requests(cfg, batch):
    """Each row becomes its own request carrying a copy of its request's user
    ids and behaviour sequences."""
    q_n, r_n = batch["n_requests"], batch["n_rows"]
    off = batch["req_off"]
    req_of_row = np.searchsorted(off, np.arange(r_n), side="right") - 1
    nb = dict(batch)
    nb["req_off"] = np.arange(r_n + 1, dtype=np.int32)
    nb["user_ids"] = batch["user_ids"][:, req_of_row]
    nb["n_requests"] = r_n
    if cfg.n_seq:
        so, si = batch["seq_off"], batch["seq_ids"]
        offs, ids = [0], []
        for f in range(cfg.n_seq):
            for r in range(r_n):
                q = req_of_row[r]
                seg = si[so[f * q_n + q]:so[f * q_n + q + 1]]
                ids.append(seg)
                offs.append(offs[-1] + len(seg))
        nb["seq_off"] = np.asarray(offs, np.int32)
        nb["seq_ids"] = np.concatenate(ids)
    return nb


@pytest.mark.parametrize("name", ["serving_bf16", "multivalued_fp16_ll", "large_fp16_ll"])
def test_user_broadcast_equals_per_row(name):
    """User-side features shared by a request's candidates (Section 3.3): the
    batched request scores exactly as one-row requests with copied user ids."""
    cfg = tiny(name)
    tables, params, batch = problem(cfg, seed=13)
    base = run_oracle(cfg, tables, params, batch)["scores"]
    got = run_oracle(cfg, tables, params, split_into_single_row_requests(cfg, batch))["scores"]
    assert np.array_equal(got, base)


def test_topk_mask_ties_prefer_lower_group():
    """W1 = 0 makes s_g = sigmoid(b2_g) for every row; with tied b2 the mask
    must keep the lower group index (sorted by (-importance, g))."""
    cfg = tiny("wide_prune_bf16", topk_k=4)
    tables, params, batch = problem(cfg, seed=14)
    params["se_w1"] = np.zeros_like(params["se_w1"])
    params["se_b1"] = np.zeros_like(params["se_b1"])
    m = cfg.n_groups
    b2 = np.zeros(m, np.float32)
    b2[[1, 3, 6, 8]] = 0.5        # four tied at the top
    b2[[0, 2]] = 0.25             # next
    b2[[5, 9, 10]] = 1.0          # highest three
    params["se_b2"] = b2
    o = run_oracle(cfg, tables, params, batch)
    want = sorted(range(m), key=lambda g: (-float(b2[g]), g))[:4]
    assert sorted(np.flatnonzero(o["mask"][0]).tolist()) == sorted(want)
    assert sorted(want) == [1, 5, 9, 10]


def test_topk_k_at_least_m_keeps_all():
    cfg = tiny("wide_prune_bf16", topk_k=1000)
    tables, params, batch = problem(cfg, seed=15)
    o = run_oracle(cfg, tables, params, batch, want_x=True)
    assert np.all(o["mask"] == 1)
    cfg0 = tiny("wide_prune_bf16", topk_k=0)
    o0 = run_oracle(cfg0, tables, params, batch, want_x=True)
    assert np.array_equal(o["x"], o0["x"])


def test_direct_id_out_of_range_is_an_error():
    cfg = tiny("serving_bf16")
    tables, params, batch = problem(cfg, seed=16)
    batch["ad_ids"] = batch["ad_ids"].copy()
    batch["ad_ids"][2, 3] = cfg.vocab
    with pytest.raises(oracle.OracleError):
        run_oracle(cfg, tables, params, batch)


def test_sample_subset_equals_full():
    cfg = tiny("serving_bf16")
    tables, params, batch = problem(cfg, seed=17)
    full = run_oracle(cfg, tables, params, batch)["scores"]
    idx = np.array([5, 0, 3, batch["n_rows"] - 1])
    part = run_oracle(cfg, tables, params, batch, sample=idx)["scores"]
    assert np.array_equal(part, full[idx])
