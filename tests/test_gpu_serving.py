"""Serving-shaped use of the C ABI on the GPU (the paper's concurrent
serving, Section 3.3: several requests in flight on one GPU): scoring
captured in a HIP graph and replayed, and concurrent calls on several
streams with distinct workspaces, each against eager single-stream scoring
bit for bit and against the checker within the dtype's tolerance."""
import numpy as np
import pytest

from paper_2007_16122_amd import binding as B
from paper_2007_16122_amd import synth
from tests.common import problem
from tests.gpu_common import (compare_scores, device_table_from_numpy, log, request_slice,
                              run_oracle)

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda"


def _setup(name, cand, seed):
    base = synth.CONFIGS[name]
    cfg = synth.config(name, vocab=20_000, seq_len_max=base.seq_len_max)
    tables, params, batch = problem(cfg, seed=seed, cand=cand, model_seed=cfg.seed)
    model = B.ColdModel(cfg, device=DEV)
    model.load([device_table_from_numpy(t, cfg.dtype, DEV) for t in tables],
               B.params_to_device(params, cfg.dtype, DEV))
    return cfg, tables, params, batch, model


def _requests(cfg, batch, q0, q1):
    """Requests q0 .. q1-1 of a batch without behaviour sequences as a batch
    of their own."""
    off = batch["req_off"]
    lo, hi = int(off[q0]), int(off[q1])
    return dict(req_off=(off[q0:q1 + 1] - lo).astype(np.int32),
                user_ids=np.ascontiguousarray(batch["user_ids"][:, q0:q1]),
                ad_ids=np.ascontiguousarray(batch["ad_ids"][:, lo:hi]),
                cross_ids=np.ascontiguousarray(batch["cross_ids"][:, lo:hi]),
                seq_off=np.zeros(1, np.int32), seq_ids=np.zeros(0, batch["ad_ids"].dtype),
                n_rows=hi - lo, n_requests=q1 - q0)


def _copy_batch_into(dst: dict, src_np: dict):
    """Overwrite the device tensors of a batch (same shapes) with another
    batch's values, so that a captured graph reads the new ids."""
    new = B.batch_to_device(src_np, DEV)
    for k in ("req_off", "user_ids", "ad_ids", "cross_ids", "seq_off", "seq_ids"):
        if dst.get(k) is not None:
            assert dst[k].shape == new[k].shape, k
            dst[k].copy_(new[k])


@pytest.mark.parametrize("name,entry", [("serving_bf16", "cold_score"),
                                        ("multivalued_fp16_ll", "cold_score"),
                                        ("wide_prune_bf16", "cold_score"),
                                        ("serving_bf16", "cold_score_noalloc"),
                                        ("wide_prune_bf16", "cold_score_noalloc")])
def test_graph_replay_equals_eager(name, entry):
    """One 2,000-ad request's scoring call captured in a graph: every replay,
    with eager work and synchronisations between replays and the request's
    ids replaced in place between them, gives bit for bit the scores of
    eager scoring of the same ids, which match the checker (on the top-k
    model each replay forms its request's mask, kept-group list, weight
    columns and row-tile table on the device)."""
    cfg, tables, params, batch, model = _setup(name, [2000, 2000, 2000], seed=61)
    try:
        reqs = [request_slice(cfg, batch, q) for q in range(3)]
        if cfg.n_seq:   # the captured graph keeps the sequence-id count fixed
            n = min(len(r["seq_ids"]) for r in reqs)
            for r in reqs:
                r["seq_ids"] = r["seq_ids"][:n].copy()
                r["seq_off"] = np.minimum(r["seq_off"], n).astype(np.int32)
        eager = []
        for r in reqs:
            sc = model.score(B.batch_to_device(r, DEV))
            torch.cuda.synchronize()
            eager.append(sc.cpu().numpy())
        dev_req = B.batch_to_device(reqs[0], DEV)
        scores = torch.empty(2000, dtype=torch.float32, device=DEV)
        ws = model.ensure_workspace(2000, 1)
        b = B.ColdModel.make_batch_struct(dev_req)

        def call():
            stream = torch.cuda.current_stream().cuda_stream
            if entry == "cold_score":
                st = B.cold_score(model.h, b, B._ptr(ws), ws.numel(), B._ptr(scores), None, None,
                                  None, None, 0, stream)
            else:
                st = B.cold_score_noalloc(model.h, b, B._ptr(scores), None, None, None, None, 0,
                                          stream)
            assert st == B.COLD_OK, B.cold_last_error(model.h)

        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            call()                                   # warm-up outside the capture
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            call()
        junk = torch.randn(1 << 20, device=DEV)
        for rep in range(6):
            q = rep % 3
            _copy_batch_into(dev_req, reqs[q])
            scores.fill_(-1.0)
            junk.mul_(1.0001)                        # eager work between replays
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            got = scores.cpu().numpy()
            assert np.array_equal(got.view(np.uint32), eager[q].view(np.uint32)), \
                f"replay {rep} (request {q}) differs from eager scoring"
        log(f"{name} {entry}: 6 replays bit-identical to eager scoring")
        for q, r in enumerate(reqs):
            o = run_oracle(cfg, tables, params, r)
            compare_scores(cfg, eager[q].astype(np.float64), o["scores"], f"graph {name} req {q}")
        del g
    finally:
        model.close()


def test_concurrent_streams_with_distinct_workspaces():
    """Four streams, each with its own workspace and output buffer, score
    four different batches concurrently (eager calls and graph replays,
    several rounds): every result equals the same batch scored alone on one
    stream, bit for bit."""
    cfg, tables, params, batch, model = _setup("serving_bf16", [2000] * 4 + [700] * 4, seed=62)
    try:
        # three single requests and the 4-request tail of the batch
        subs = [request_slice(cfg, batch, q) for q in range(3)]
        subs.append(_requests(cfg, batch, 4, 8))
        alone = []
        for s in subs:
            sc = model.score(B.batch_to_device(s, DEV))
            torch.cuda.synchronize()
            alone.append(sc.cpu().numpy())
        streams = [torch.cuda.Stream() for _ in range(4)]
        jobs = []
        for s in subs:
            db = B.batch_to_device(s, DEV)
            ws = torch.empty(B.cold_workspace_bytes(model.h, db["n_rows"], db["req_off"].numel() - 1),
                             dtype=torch.uint8, device=DEV)
            jobs.append((db, ws, torch.empty(db["n_rows"], dtype=torch.float32, device=DEV)))
        torch.cuda.synchronize()
        for rnd in range(5):
            for (db, ws, sc), st in zip(jobs, streams):
                sc.fill_(-1.0)
            torch.cuda.synchronize()
            for (db, ws, sc), st in zip(jobs, streams):
                with torch.cuda.stream(st):
                    model.score(db, scores=sc, workspace=ws)
            torch.cuda.synchronize()
            for i, (db, ws, sc) in enumerate(jobs):
                assert np.array_equal(sc.cpu().numpy().view(np.uint32), alone[i].view(np.uint32)), \
                    f"round {rnd} stream {i}"
        # the same four calls as graphs replayed concurrently
        graphs = []
        for (db, ws, sc), st in zip(jobs, streams):
            st.wait_stream(torch.cuda.current_stream())
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=st):
                model.score(db, scores=sc, workspace=ws)
            graphs.append(g)
        torch.cuda.synchronize()
        for rnd in range(5):
            for db, ws, sc in jobs:
                sc.fill_(-1.0)
            torch.cuda.synchronize()
            for g, st in zip(graphs, streams):
                with torch.cuda.stream(st):
                    g.replay()
            torch.cuda.synchronize()
            for i, (db, ws, sc) in enumerate(jobs):
                assert np.array_equal(sc.cpu().numpy().view(np.uint32), alone[i].view(np.uint32)), \
                    f"graph round {rnd} stream {i}"
        log("4 concurrent streams: eager and graph rounds bit-identical to scoring alone")
        o = run_oracle(cfg, tables, params, subs[0])
        compare_scores(cfg, alone[0].astype(np.float64), o["scores"], "streams request 0")
        del graphs
    finally:
        model.close()


def test_prepared_call_equals_score():
    """A prepared call (binding.ColdModel.prepare: the batch struct,
    pointers and stream resolved once) enqueued repeatedly, with the
    request's ids replaced in place between calls, gives bit for bit the
    scores of score() on the same ids."""
    cfg, tables, params, batch, model = _setup("serving_bf16", [700, 0, 300, 1000], seed=61)
    try:
        a_np, b_np = _requests(cfg, batch, 0, 2), _requests(cfg, batch, 2, 4)
        b_np = dict(b_np, ad_ids=b_np["ad_ids"][:, :a_np["n_rows"]],
                    cross_ids=b_np["cross_ids"][:, :a_np["n_rows"]],
                    req_off=np.array([0, 350, a_np["n_rows"]], np.int32), n_rows=a_np["n_rows"])
        dev = B.batch_to_device(a_np, DEV)
        scores = torch.empty(a_np["n_rows"], dtype=torch.float32, device=DEV)
        call = model.prepare(dev, scores)
        for src in (a_np, b_np, a_np):
            _copy_batch_into(dev, src)
            want = model.score(B.batch_to_device(src, DEV)).clone()
            call()
            torch.cuda.synchronize()
            assert torch.equal(scores.view(torch.int32), want.view(torch.int32))
    finally:
        model.close()
