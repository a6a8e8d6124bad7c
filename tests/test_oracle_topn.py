"""Pins of the checker's top-n selection by eCPM (Section 2 and its
footnote: eCPM = pCTR * bid; the pre-ranking stage passes on the top N
candidates of each request) and of the recall metric of Eq. 4 (Section 4.1).
Each pin comes from outside the checker: a hand-worked example, a different
selection algorithm (heapq over Python floats), or a property of the result."""
import heapq
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_topn():
    rows, expected = [], {}
    req_off = None
    with open(os.path.join(GOLDEN, "topn_example.txt")) as fh:
        for line in fh:
            body = line.split("#", 1)[0].split()
            text = line.strip()
            if body:
                rows.append((int(body[0]), float(body[1]), float(body[2])))
            elif text.startswith("# req_off:"):
                req_off = [int(v) for v in text.split(":", 1)[1].split()]
            elif text.startswith("# q") and ":" in text:
                q = int(text[3:text.index(":")])
                toks = text.split(":", 1)[1].split()
                expected[q] = ([int(v) for v in toks[:4]],
                               [float(v.replace("inf", "Infinity")) for v in toks[4:]])
    rows.sort()
    pctr = np.array([r[1] for r in rows], np.float32)
    bid = np.array([r[2] for r in rows], np.float32)
    return pctr, bid, np.array(req_off, np.int32), expected


def test_topn_golden_example():
    pctr, bid, req_off, expected = _golden_topn()
    assert len(expected) == 3
    rows, ecpm = oracle.select_topn(pctr, bid, req_off, 4)
    for q, (want_rows, want_ecpm) in expected.items():
        assert rows[q].tolist() == want_rows
        assert ecpm[q].tolist() == want_ecpm


@pytest.mark.parametrize("seed", range(6))
def test_topn_matches_heap_selection(seed):
    rng = np.random.default_rng(seed)
    counts = rng.integers(0, 40, size=7)
    req_off = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    r = int(req_off[-1])
    # few distinct values, so ties are common; no NaN or signed zero (Python
    # float order is totalOrder on the rest)
    pctr = rng.choice(np.array([0.125, 0.25, 0.5, 0.75], np.float32), size=r)
    bid = rng.choice(np.array([0.5, 1.0, 2.0, 3.0], np.float32), size=r)
    n = int(rng.integers(1, 12))
    rows, ecpm = oracle.select_topn(pctr, bid, req_off, n)
    for q in range(counts.size):
        lo, hi = int(req_off[q]), int(req_off[q + 1])
        e = [float(np.float32(pctr[i]) * np.float32(bid[i])) for i in range(lo, hi)]
        best = heapq.nsmallest(n, range(lo, hi), key=lambda i: (-e[i - lo], i))
        want = best + [-1] * (n - len(best))
        assert rows[q].tolist() == want
        got_e = [v for v in ecpm[q].tolist() if v != -np.inf]
        assert got_e == [e[i - lo] for i in best]


def test_topn_total_order_of_special_values():
    vals = np.array([1.0, np.nan, -0.0, -np.inf, 0.0, -np.nan, np.inf, -1.0], np.float32)
    rows, _ = oracle.select_topn(vals, np.ones(8, np.float32), [0, 8], 8)
    # +NaN > +inf > 1 > +0 > -0 > -1 > -inf > -NaN (IEEE-754 totalOrder)
    assert rows[0].tolist() == [1, 6, 0, 4, 2, 7, 3, 5]


def test_topn_selected_dominate_the_rest():
    rng = np.random.default_rng(7)
    r = 3000
    pctr = rng.random(r).astype(np.float32)
    bid = (rng.integers(1, 300, size=r) / 100.0).astype(np.float32)
    rows, ecpm = oracle.select_topn(pctr, bid, [0, r], 250)
    e = pctr * bid
    chosen = set(rows[0].tolist())
    worst_chosen = min(e[i] for i in chosen)
    assert all(e[i] <= worst_chosen for i in range(r) if i not in chosen)
    assert np.all(np.diff(ecpm[0].astype(np.float64)) <= 0)


def test_recall_eq4_hand_example():
    # top-3 of the pre-ranking model {1, 2, 3}; top-4 of the ranking model
    # {2, 3, 4, 5}: two of four found -> 0.5; a second request adds 1 of 1
    assert oracle.recall_at([[1, 2, 3]], [[2, 3, 4, 5]]) == 0.5
    assert oracle.recall_at([[1, 2, 3], [9, -1, -1]], [[2, 3, 4, 5], [9, -1, -1]]) == 3 / 5
