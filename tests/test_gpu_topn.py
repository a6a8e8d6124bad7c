"""GPU top-n selection by eCPM (cold_select_topn, through the C ABI) against
the checker's selection on the same fp32 scores and bids: row indices and
eCPM bit-exact, since both sides decide in fp32 (one multiplication, then a
totalOrder comparison).  Plus Eq. 4 recall between the top-n lists of the
GPU-scored and checker-scored serving batch."""
import numpy as np
import pytest

import oracle
from paper_2007_16122_amd import binding, synth
from tests.common import problem
from tests.gpu_common import GpuScorer, device_table_from_numpy, log, run_oracle

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda"


def gpu_select(scores, bids, req_off, n_top):
    s = torch.from_numpy(np.ascontiguousarray(scores, np.float32)).to(DEV)
    b = torch.from_numpy(np.ascontiguousarray(bids, np.float32)).to(DEV)
    o = torch.from_numpy(np.ascontiguousarray(req_off, np.int32)).to(DEV)
    rows, ecpm = binding.select_topn(s, b, o, n_top)
    torch.cuda.synchronize()
    return rows.cpu().numpy(), ecpm.cpu().numpy()


def check(scores, bids, req_off, n_top, label):
    log(f"[{label}] Q={len(req_off) - 1} R={len(scores)} n={n_top}")
    g_rows, g_ecpm = gpu_select(scores, bids, req_off, n_top)
    o_rows, o_ecpm = oracle.select_topn(scores, bids, req_off, n_top)
    assert np.array_equal(g_rows, o_rows), f"{label}: selected rows differ"
    assert np.array_equal(g_ecpm.view(np.uint32), o_ecpm.view(np.uint32)), f"{label}: eCPM bits differ"


def ragged(counts):
    return np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)


def test_topn_serving_shape():
    cfg = synth.config("serving_bf16")
    rng = np.random.default_rng(11)
    req_off = ragged([2000] * 32)
    scores = rng.random(64000).astype(np.float32)
    check(scores, synth.make_bids(cfg, 64000), req_off, 200, "serving 32x2000 n=200")


def test_topn_ties_and_ragged_requests():
    rng = np.random.default_rng(12)
    counts = [0, 1, 5, 200, 1023, 1024, 1025, 3000, 0, 17]
    req_off = ragged(counts)
    r = int(req_off[-1])
    scores = rng.choice(np.array([0.125, 0.25, 0.5], np.float32), size=r)
    bids = rng.choice(np.array([1.0, 2.0, 4.0], np.float32), size=r)
    for n in (1, 7, 300, 1024):
        check(scores, bids, req_off, n, f"ties n={n}")


@pytest.mark.parametrize("c", [8191, 8192, 8193, 10_000])
def test_topn_long_requests(c):
    """Around the LDS key cache (8,192 rows) and the large workload's 10,000
    candidates per request."""
    rng = np.random.default_rng(c)
    req_off = ragged([c, 3, c])
    r = int(req_off[-1])
    scores = rng.random(r).astype(np.float32)
    scores[::97] = scores[5]                 # a few exact ties
    check(scores, synth.make_bids(synth.config("large_fp16_ll"), r), req_off, 500, f"C={c}")


def test_topn_special_values():
    vals = np.array([1.0, np.nan, -0.0, -np.inf, 0.0, -np.nan, np.inf, -1.0, 0.5, 0.5], np.float32)
    check(vals, np.ones(vals.size, np.float32), ragged([vals.size]), 10, "special values")
    check(vals, np.ones(vals.size, np.float32), ragged([vals.size]), 3, "special values n=3")


def test_topn_no_rows():
    req_off = ragged([0, 0, 0])
    g_rows, g_ecpm = gpu_select(np.zeros(1, np.float32), np.zeros(1, np.float32), req_off, 4)
    assert np.all(g_rows == -1) and np.all(g_ecpm == -np.inf)


def test_recall_of_gpu_scores_against_checker_scores():
    """Eq. 4 with k = m = 200: the top-200 by eCPM of the GPU-scored serving
    batch against the top-200 of the checker-scored one (same bids)."""
    base = synth.CONFIGS["serving_bf16"]
    cfg = synth.config("serving_bf16", vocab=20_000)
    tables, params, batch = problem(cfg, seed=31, cand=[2000] * 4, model_seed=cfg.seed)
    run = GpuScorer(cfg, [device_table_from_numpy(t, cfg.dtype, DEV) for t in tables], params, DEV)
    try:
        g = run.score(batch)
    finally:
        run.close()
    o = run_oracle(cfg, tables, params, batch)
    bids = synth.make_bids(base, batch["n_rows"], seed=31)
    g_rows, _ = gpu_select(g["scores"].astype(np.float32), bids, batch["req_off"], 200)
    o_rows, _ = oracle.select_topn(o["scores"].astype(np.float32), bids, batch["req_off"], 200)
    rec = oracle.recall_at(g_rows, o_rows)
    log(f"Eq. 4 recall@200 (GPU vs checker scores): {rec:.4f}")
    assert rec >= 0.98
