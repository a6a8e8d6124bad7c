"""cold_score_noalloc, the entry point for callers that cannot allocate
device memory, against cold_score on the same inputs through the C ABI:
bit-identical scores, SE weights, group masks, gather rows and network
input, on two calls in a row, the second smaller (it runs on what the first
left in the library's array), scores within the dtype's tolerance of the
checker, and the size limit."""
import numpy as np
import pytest

from paper_2007_16122_amd import binding as B
from paper_2007_16122_amd import synth
from tests.common import problem
from tests.gpu_common import compare_scores, device_table_from_numpy, log, run_oracle

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda"


def _model(cfg, tables, params):
    m = B.ColdModel(cfg, device=DEV)
    m.load([device_table_from_numpy(t, cfg.dtype, DEV) for t in tables],
           B.params_to_device(params, cfg.dtype, DEV))
    return m


def _outputs(cfg, n_rows, n_req):
    xdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[cfg.dtype]
    r = max(n_rows, 1)
    return dict(scores=torch.full((r,), -1.0, dtype=torch.float32, device=DEV),
                importance=torch.full((r, cfg.n_groups), -1.0, dtype=torch.float32, device=DEV),
                mask=torch.full((max(n_req, 1), cfg.n_groups), 7, dtype=torch.uint8, device=DEV),
                rows=torch.full((cfg.n_groups, r), -7, dtype=torch.int32, device=DEV),
                x=torch.full((r, cfg.d_in), -1.0, dtype=xdt, device=DEV))


def _score_both(model, cfg, batch_np):
    """The batch through cold_score (its own workspace) and through
    cold_score_noalloc; returns both sets of outputs on the host."""
    dev_batch = B.batch_to_device(batch_np, DEV)
    b = B.ColdModel.make_batch_struct(dev_batch)
    n_rows, n_req = int(batch_np["n_rows"]), len(batch_np["req_off"]) - 1
    stream = torch.cuda.current_stream().cuda_stream
    mask_on = cfg.topk_k > 0
    got = []
    for noalloc in (False, True):
        o = _outputs(cfg, n_rows, n_req)
        args = (B._ptr(o["scores"]), B._ptr(o["importance"]),
                B._ptr(o["mask"]) if mask_on else None, B._ptr(o["rows"]), B._ptr(o["x"]))
        if noalloc:
            st = B.cold_score_noalloc(model.h, b, *args, B.COLD_SCORE_VALIDATE, stream)
        else:
            ws = model.ensure_workspace(n_rows, n_req)
            st = B.cold_score(model.h, b, B._ptr(ws), ws.numel(), *args, B.COLD_SCORE_VALIDATE,
                              stream)
        assert st == B.COLD_OK, B.cold_last_error(model.h)
        torch.cuda.synchronize()
        got.append({k: v.cpu() for k, v in o.items()})
    return got


def _same_bits(a, b, what):
    assert a.dtype == b.dtype and a.shape == b.shape, what
    if a.dtype.is_floating_point:
        a = a.view(torch.int16 if a.element_size() == 2 else torch.int32)
        b = b.view(torch.int16 if b.element_size() == 2 else torch.int32)
    assert torch.equal(a, b), what


@pytest.mark.parametrize("name,cands", [("wide_prune_bf16", ([333, 0, 150], [100])),
                                        ("wide_prune_bf16", ([5000], [333, 0, 150])),
                                        ("multivalued_fp16_ll", ([257, 0, 1, 500], [40, 3])),
                                        ("serving_bf16", ([2000], [700]))])
def test_noalloc_matches_cold_score(name, cands):
    base = synth.CONFIGS[name]
    cfg = synth.config(name, vocab=20_000, seq_len_max=base.seq_len_max)
    first = problem(cfg, seed=51, cand=cands[0], model_seed=cfg.seed)
    tables, params, _ = first
    model = _model(cfg, tables, params)
    try:
        for i, cand in enumerate(cands):
            _, _, batch = problem(cfg, seed=51 + i, cand=cand, model_seed=cfg.seed)
            log(f"noalloc {name} call {i}: {cand}")
            ref, got = _score_both(model, cfg, batch)
            n = int(batch["n_rows"])
            for k in ("scores", "importance", "rows", "x") + (("mask",) if cfg.topk_k else ()):
                _same_bits(got[k], ref[k], f"{name} call {i}: {k}")
            o = run_oracle(cfg, tables, params, batch)
            compare_scores(cfg, got["scores"][:n].numpy().astype(np.float64), o["scores"],
                           f"noalloc {name} call {i}")
    finally:
        model.close()


def test_noalloc_rejects_batches_beyond_its_array():
    cfg = synth.config("serving_bf16", vocab=20_000)
    tables, params, batch = problem(cfg, seed=52, cand=[2000] * 12, model_seed=cfg.seed)
    model = _model(cfg, tables, params)
    try:
        need = B.cold_workspace_bytes(model.h, int(batch["n_rows"]), 12)
        assert need > B.COLD_NOALLOC_WORKSPACE_BYTES
        b = B.ColdModel.make_batch_struct(B.batch_to_device(batch, DEV))
        sc = torch.full((int(batch["n_rows"]),), -1.0, dtype=torch.float32, device=DEV)
        st = B.cold_score_noalloc(model.h, b, B._ptr(sc), None, None, None, None, 0,
                                  torch.cuda.current_stream().cuda_stream)
        assert st == B.COLD_ERR_WORKSPACE
        msg = B.cold_last_error(model.h)
        assert "cold_score_noalloc" in msg and str(need) in msg, msg
        torch.cuda.synchronize()
        assert bool((sc == -1.0).all())      # nothing was enqueued
        # eight 2,000-ad requests fit, nine do not
        _, _, small = problem(cfg, seed=53, cand=[2000] * 8, model_seed=cfg.seed)
        assert B.cold_workspace_bytes(model.h, 16000, 8) <= B.COLD_NOALLOC_WORKSPACE_BYTES
        assert B.cold_workspace_bytes(model.h, 18000, 9) > B.COLD_NOALLOC_WORKSPACE_BYTES
        ref, got = _score_both(model, cfg, small)
        _same_bits(got["scores"], ref["scores"], "eight requests")
    finally:
        model.close()
