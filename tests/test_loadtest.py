"""Load-test procedures (Sec. III-C): the batch-weight search and corner-case
batches on the host, and on the GPU the closed-loop characterization and the
search's budget checked against engine creation."""
import numpy as np
import pytest

from oracle import serving as S
from paper_2410_02425_amd import loadtest, lp, synth


@pytest.mark.parametrize("name,gb", [("8b", 40), ("8b", 100), ("8b", 250), ("7b", 60), ("tiny", 1)])
def test_search_max_batch_weight_is_the_largest_fitting_budget(name, gb):
    shape, wl = synth.SHAPES[name], synth.WORKLOADS[name]
    cfg = lp.make_config(shape)
    opt = loadtest._options(wl, wl.max_batch)
    arena = int(gb * 2**30)
    w = loadtest.search_max_batch_weight(cfg, opt, arena)
    assert w > 0 and w % loadtest.KV_BLOCK == 0

    def need(x):
        return lp.arena_bytes(cfg, lp.EngineOptions(opt.max_batch, opt.max_seq_len, x, opt.max_prefill_tokens, 0, 0))

    assert need(w) <= arena < need(w + loadtest.KV_BLOCK)
    # the KV pool grows by exactly the cache bytes of the added tokens
    assert need(w + loadtest.KV_BLOCK) - need(w) == loadtest.KV_BLOCK * loadtest.kv_bytes_per_token(cfg)


def test_search_reports_zero_when_weights_do_not_fit():
    cfg = lp.make_config(synth.SHAPES["8b"])
    assert loadtest.search_max_batch_weight(cfg, loadtest._options(synth.WORKLOADS["8b"], 64), 8 * 2**30) == 0


@pytest.mark.parametrize("weight,max_batch", [(100000, 64), (20000, 4), (5120, 8), (3000, 8), (10**7, 64)])
def test_corner_case_batch(weight, max_batch):
    reqs = loadtest.corner_case_requests(weight, max_batch, 5120, 1000)
    total = sum(r.in_len + r.out_len for r in reqs)
    assert 1 <= len(reqs) <= max_batch and total <= max(weight, 5120)
    if weight >= 5120:
        assert all(r.in_len + r.out_len == 5120 for r in reqs)
        assert len(reqs) == min(max_batch, weight // 5120)
    else:
        assert len(reqs) == 1 and total == weight


# ------------------------------------------------------------------ GPU

@pytest.mark.gpu
def test_characterize_tiny_matches_oracle_accounting():
    import torch
    torch.cuda.set_device(0)
    shape, wl = synth.SHAPES["tiny"], synth.WORKLOADS["tiny"]
    cfg = lp.make_config(shape)
    eng = lp.Engine(cfg, lp.EngineOptions(4, 64, 0, 4096, 0, 0))
    eng.init_weights_random(3, 0.02)
    # 8 and 16 users on 4 slots: the users beyond the running batch queue
    rows = loadtest.characterize(eng, wl, shape.vocab, [1, 2, 4, 8, 16], requests_per_user=2)
    assert [r["users"] for r in rows] == [1, 2, 4, 8, 16]
    for r in rows:
        U = r["users"]
        # replay the last run (U users) through the oracle's accounting
        reqs = synth.make_requests(wl, shape.vocab, max(2 * U, 4))
        eng.submit(reqs)
        eng.run(lp.LP_CLOSED_LOOP, U)
        # the schedule is the oracle's closed-loop policy on the recorded step times
        log = eng.step_log()
        sreqs = [S.SimRequest(q.id, q.in_len, q.out_len) for q in reqs]
        tr = S.simulate(sreqs, 4, eng.max_batch_weight(), 4096, True, U, [st["end_ns"] for st in log])
        assert [(st.kind, st.ids, st.slots) for st in tr.steps] == [(st["kind"], st["ids"], st["slots"])
                                                                    for st in log]
        got = eng.latency_summary()
        res = {q.id: eng.result(q.id) for q in reqs}
        toks = {q.id: eng.token_times(q.id).tolist() for q in reqs}
        exp = S.summarize({q.id: res[q.id]["arrival_ns"] for q in reqs}, toks, {q.id: q.in_len for q in reqs})
        for k in ("ttft_p50_ns", "nttft_p50_ns", "itl_p50_ns", "e2e_p50_ns", "itl_p90_ns", "output_tokens",
                  "throughput_tok_s"):
            assert got[k] == exp[k], (U, k)
        assert max(st["n_rows"] for st in log) <= min(U, 4)
        if U > 4:  # more users than slots: the running batch is full
            assert max(st["n_rows"] for st in log if st["kind"] == "decode") == 4
        assert r["output_tokens"] == sum(q.out_len for q in reqs)
    eng.close()


@pytest.mark.gpu
def test_searched_budget_runs_and_one_block_more_does_not_fit():
    import torch
    torch.cuda.set_device(0)
    cfg = lp.make_config(synth.SHAPES["tiny"])
    opt = lp.EngineOptions(4, 96, 0, 4096, 0, 0)
    arena = lp.arena_bytes(cfg, lp.EngineOptions(4, 96, 640, 4096, 0, 0)) + 1000
    w = loadtest.search_max_batch_weight(cfg, opt, arena)
    assert w == 640
    ok, msg = loadtest.verify_batch_weight(cfg, opt, w, arena)
    assert ok, msg
    ok, msg = loadtest.verify_batch_weight(cfg, opt, w + loadtest.KV_BLOCK, arena)
    assert not ok and "-2" in msg  # LP_ENOMEM


def test_generated_requests_follow_the_samples():
    model = lp.RequestModel(synth.trace_records(5, 20000))
    rng = np.random.default_rng(0)
    corpus = rng.integers(0, 1000, size=600).astype(np.int32)
    u = rng.random(300)
    vals, _ = model.sample(u)
    reqs = loadtest.generated_requests(model, u, 1000, 500, 100, corpus)
    assert len(reqs) == int(np.clip(np.rint(vals[:, 2]), 1, 64).sum())
    k = 0
    for row in vals:
        for _ in range(int(np.rint(row[2]))):
            r = reqs[k]
            assert r.in_len == int(np.clip(np.rint(row[0]), 1, 500)) and r.out_len == int(np.clip(np.rint(row[1]), 1, 100))
            assert np.array_equal(r.prompt, corpus[:r.in_len])
            k += 1
    ind = loadtest.generated_requests(model, rng.random((300, 6)), 1000, 500, 100, corpus, independent=True)
    assert all(1 <= r.in_len <= 500 and 1 <= r.out_len <= 100 for r in ind)


@pytest.mark.gpu
def test_generator_comparison_tiny():
    import torch
    torch.cuda.set_device(0)
    shape = synth.SHAPES["tiny"]
    eng = lp.Engine(lp.make_config(shape), lp.EngineOptions(4, 128, 0, 4096, 0, 0))
    eng.init_weights_random(5, 0.02)
    model = lp.RequestModel(synth.trace_records(6, 5000), 64)
    rows = loadtest.generator_comparison(eng, model, [1, 4], 2, 7)
    assert [(r["mode"], r["users"]) for r in rows] == [("joint", 1), ("independent", 1), ("joint", 4),
                                                        ("independent", 4)]
    for r in rows:
        assert r["output_tokens"] >= r["n_requests"] >= r["generated"]
        assert r["throughput_tok_s"] > 0
    eng.close()
