"""Load tests of the serving engine, the way LLM-Pilot characterizes an
inference service (Sec. III-C).

* ``characterize``: closed-loop load tests at a range of concurrent users
  (Sec. III-C-3): for each user count U, U users send requests back to back
  (zero think time) and the test reports median TTFT, nTTFT, ITL and
  end-to-end latency and the output-token throughput.
* ``search_max_batch_weight`` / ``verify_batch_weight``: the maximum batch
  weight of Sec. III-C-2 as the largest token budget whose KV blocks fit the
  memory given to the engine, found by bisection and checked with a
  corner-case batch of maximal-length requests that fills the budget.
* ``batch_weight_sweep``: end-to-end latency and throughput of one load test
  run under a range of batch-weight budgets.
* ``generated_requests`` / ``generator_comparison``: requests from the
  workload generator's joint request model (Sec. III-B), or with every
  parameter drawn from its own marginal, and the load tests of the two
  (the comparison of Sec. V-A).

Every step of a test runs in the engine behind the C ABI (scheduling, the
GPU serving step, timestamps and the latency summary); this module only
chooses the experiments and collects their results.
"""
from __future__ import annotations

import argparse
import json
import sys

import numpy as np

from . import lp, synth

KV_BLOCK = 64  # tokens per KV-cache block of the engine


def _options(wl: synth.Workload, max_batch: int, max_batch_weight: int = 0, flags: int = 0) -> lp.EngineOptions:
    return lp.EngineOptions(max_batch, wl.in_range[1] + wl.out_range[1], max_batch_weight, 65536, 0, flags)


def characterize(eng: lp.Engine, wl: synth.Workload, vocab: int, users, requests_per_user: int = 2,
                 min_requests: int = 4, sampling=None):
    """Closed-loop load test at each user count in ``users`` over the first
    max(requests_per_user * U, min_requests) requests of the workload's
    seeded stream; ``sampling`` = (temperature, top_k, top_p) applies to
    every request (seeded by its id), None keeps them greedy.  User counts
    above the engine's slot count are allowed: the users beyond the running
    batch wait in the admission queue, and their waiting counts in TTFT, as a
    client of the paper's load test sees it.  Returns one metrics dict per
    user count."""
    rows = []
    for U in users:
        if U < 1:
            raise ValueError(f"user count {U} < 1")
        reqs = synth.make_requests(wl, vocab, max(requests_per_user * U, min_requests))
        eng.submit(reqs)
        if sampling is not None:
            for r in reqs:
                eng.set_sampling(r.id, *sampling, seed=1000 + r.id)
        eng.run(lp.LP_CLOSED_LOOP, U)
        rows.append({"users": U, **eng.latency_summary()})
    return rows


def kv_bytes_per_token(cfg: lp.ModelConfig) -> int:
    """KV-cache bytes one token holds (K and V of every layer and KV head)."""
    esz = 4 if cfg.dtype == lp.LP_F32 else 2
    return 2 * cfg.n_layers * cfg.n_kv_heads * (cfg.d_model // cfg.n_heads) * esz


def search_max_batch_weight(cfg: lp.ModelConfig, opt: lp.EngineOptions, arena_bytes: int) -> int:
    """Largest max_batch_weight (a multiple of the KV block) whose engine
    needs at most ``arena_bytes``; 0 if not even one block fits."""
    def fits(w):
        o = lp.EngineOptions(opt.max_batch, opt.max_seq_len, w, opt.max_prefill_tokens, opt.hbm_reserve_bytes,
                             opt.flags)
        return lp.arena_bytes(cfg, o) <= arena_bytes

    if not fits(KV_BLOCK):
        return 0
    lo, hi = 1, max(2, arena_bytes // (kv_bytes_per_token(cfg) * KV_BLOCK) + 2)  # in blocks; fits(lo)
    while not fits(hi * KV_BLOCK) and hi - lo > 1:
        mid = (lo + hi) // 2
        if fits(mid * KV_BLOCK):
            lo = mid
        else:
            hi = mid
    if fits(hi * KV_BLOCK):
        lo = hi
    return lo * KV_BLOCK


def corner_case_requests(weight: int, max_batch: int, max_seq_len: int, vocab: int, n_out: int = 8, seed: int = 0):
    """The heaviest batch the budget admits at once: requests of the longest
    prompt the engine accepts (max_seq_len - n_out tokens, n_out outputs),
    as many as the budget and max_batch allow; a budget below one such
    request gets one request of exactly that weight."""
    rng = np.random.default_rng(seed)
    per = max_seq_len
    n = min(max_batch, weight // per)
    shapes = [(per - n_out, n_out)] * n if n else [(max(1, weight - n_out), min(n_out, weight - 1))]
    return [synth.Request(k, rng.integers(0, vocab, size=a).astype(np.int32), b) for k, (a, b) in
            enumerate(shapes)]


def verify_batch_weight(cfg: lp.ModelConfig, opt: lp.EngineOptions, weight: int, arena_bytes: int):
    """Creates an engine with the given budget in ``arena_bytes`` of device
    memory and runs its corner-case batch.  Returns (ok, message)."""
    o = lp.EngineOptions(opt.max_batch, opt.max_seq_len, weight, opt.max_prefill_tokens, opt.hbm_reserve_bytes,
                         opt.flags)
    try:
        eng = lp.Engine(cfg, o, arena_bytes)
    except lp.LPError as err:
        _release()
        return False, str(err)
    try:
        eng.init_weights_random(1, 0.02)
        reqs = corner_case_requests(weight, o.max_batch, o.max_seq_len, cfg.vocab)
        eng.submit(reqs)
        eng.run(lp.LP_CLOSED_LOOP, len(reqs))
        return True, f"{len(reqs)} requests of {reqs[0].in_len}+{reqs[0].out_len} tokens"
    except lp.LPError as err:
        return False, str(err)
    finally:
        eng.close()
        _release()


def _release():
    import torch
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def batch_weight_sweep(cfg: lp.ModelConfig, wl: synth.Workload, weights, users: int, n_requests: int,
                       seed: int = 1):
    """One closed-loop load test (``users`` users, the first ``n_requests``
    requests of the workload) per batch-weight budget."""
    rows = []
    reqs = synth.make_requests(wl, cfg.vocab, n_requests)
    for w in weights:
        if w < max(r.in_len + r.out_len for r in reqs):
            raise ValueError(f"budget {w} is below the heaviest request")
        eng = lp.Engine(cfg, _options(wl, users, w))
        try:
            eng.init_weights_random(seed, 0.02)
            eng.submit(reqs)
            eng.run(lp.LP_CLOSED_LOOP, users)
            rows.append({"max_batch_weight": w, "users": users, **eng.latency_summary()})
        finally:
            eng.close()
            _release()
    return rows


def generated_requests(model: lp.RequestModel, uniforms, vocab: int, max_in: int, max_out: int, corpus,
                       independent: bool = False):
    """Engine requests from workload-generator samples (columns as
    synth.TRACE_COLUMNS).  Token counts are the sampled interval centres
    rounded to the nearest integer (ties to even) and clipped to the engine's
    limits; the prompt is the corpus truncated to that length (Sec. III-B); a
    request with batch size b becomes b sequences submitted together.  The
    sampling parameters are carried by the model but the engine decodes
    greedily."""
    vals = model.sample_independent(uniforms) if independent else model.sample(uniforms)[0]
    reqs = []
    for row in vals:
        n_in = int(np.clip(np.rint(row[0]), 1, max_in))
        n_out = int(np.clip(np.rint(row[1]), 1, max_out))
        for _ in range(int(np.clip(np.rint(row[2]), 1, 64))):
            reqs.append(synth.Request(len(reqs), np.ascontiguousarray(corpus[:n_in]), n_out))
    return reqs


def generator_comparison(eng: lp.Engine, model: lp.RequestModel, users, n_per_user: int, seed: int):
    """Closed-loop load tests with requests from the joint model and from
    independent marginals, the same number of generated requests for both."""
    rng = np.random.default_rng(seed)
    corpus = rng.integers(0, eng.cfg.vocab, size=eng.opt.max_seq_len).astype(np.int32)
    max_out = min(1500, eng.opt.max_seq_len // 2)  # the traces' output range (Table II)
    max_in = eng.opt.max_seq_len - max_out
    rows = []
    for U in users:
        n = max(n_per_user * U, 4)
        u_joint = rng.random(n)
        u_ind = rng.random((n, model.n_params))
        for mode, reqs in (("joint", generated_requests(model, u_joint, eng.cfg.vocab, max_in, max_out, corpus)),
                           ("independent", generated_requests(model, u_ind, eng.cfg.vocab, max_in, max_out, corpus,
                                                              independent=True))):
            eng.submit(reqs)
            eng.run(lp.LP_CLOSED_LOOP, U)
            rows.append({"mode": mode, "users": U, "generated": n, **eng.latency_summary()})
    return rows


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    c = sub.add_parser("characterize", help="closed-loop load tests over a range of user counts")
    c.add_argument("--config", default="8b")
    c.add_argument("--users", default="1,2,4,8,16,32,64,128")
    c.add_argument("--max-batch", type=int, default=64, help="running-batch slots (users beyond them queue)")
    c.add_argument("--requests-per-user", type=int, default=2)
    c.add_argument("--sampling", default="", help="temperature,top_k,top_p for every request (default greedy)")
    b = sub.add_parser("batch-weight", help="search the maximum batch weight, then sweep budgets")
    b.add_argument("--config", default="8b")
    b.add_argument("--users", type=int, default=64)
    b.add_argument("--requests", type=int, default=128)
    b.add_argument("--weights", default="8192,16384,32768,65536,131072,max",
                   help="budgets in tokens; 'max' is the searched maximum")
    b.add_argument("--arena-gb", type=float, default=0.0, help="memory budget (default: 85%% of free HBM)")
    o = sub.add_parser("open", help="open-loop run of a Poisson-arrival workload (e.g. 8b-poisson)")
    o.add_argument("--config", default="8b-poisson")
    o.add_argument("--requests", type=int, default=0, help="first N requests of the workload (default: all)")
    g = sub.add_parser("generator", help="joint vs independent request parameters (workload generator)")
    g.add_argument("--config", default="8b")
    g.add_argument("--users", default="4,16,64")
    g.add_argument("--requests-per-user", type=int, default=2)
    g.add_argument("--trace-records", type=int, default=200000)
    args = ap.parse_args(argv)

    import torch
    torch.cuda.set_device(0)
    wl = synth.WORKLOADS[args.config]
    shape = synth.SHAPES[args.config.split("-")[0]]
    cfg = lp.make_config(shape)
    key = synth.workload_seeds(wl.base_seed)[0]
    if args.cmd == "open":
        reqs = synth.make_requests(wl, shape.vocab, args.requests or None)
        eng = lp.Engine(cfg, _options(wl, wl.max_batch))
        eng.init_weights_random(key, 0.02)
        eng.submit(reqs)
        eng.run(lp.LP_OPEN_LOOP, wl.max_batch)
        log = eng.step_log()
        dec = [st for st in log if st["kind"] == "decode"]
        print(json.dumps({"config": args.config, "rate_per_s": wl.rate_per_s, "max_batch": wl.max_batch,
                          "arrival_span_s": reqs[-1].arrival_ns / 1e9, "decode_steps": len(dec),
                          "mean_decode_rows": float(np.mean([st["n_rows"] for st in dec])) if dec else 0.0,
                          "max_decode_rows": max((st["n_rows"] for st in dec), default=0),
                          **eng.latency_summary()}), flush=True)
        eng.close()
        return 0
    if args.cmd == "generator":
        import time
        recs = synth.trace_records(wl.base_seed, args.trace_records)
        t0 = time.perf_counter()
        model = lp.RequestModel(recs, 64)
        t_fit = time.perf_counter() - t0
        u = np.random.default_rng(0).random(1000)
        t0 = time.perf_counter()
        model.sample(u)
        t_draw = time.perf_counter() - t0
        print(json.dumps({"config": args.config, "trace_records": args.trace_records,
                          "joint_bins_nonempty": model.n_joint_bins(),
                          "joint_bins_possible": int(np.prod([len(model.bins(p)[1]) for p in range(model.n_params)])),
                          "fit_s": round(t_fit, 4), "draw_1000_ms": round(t_draw * 1e3, 4)}), flush=True)
        users = [int(x) for x in args.users.split(",")]
        eng = lp.Engine(cfg, lp.EngineOptions(max(users), 4096 + 1500, 0, 65536, 0, 0))
        eng.init_weights_random(key, 0.02)
        for row in generator_comparison(eng, model, users, args.requests_per_user, wl.base_seed):
            print(json.dumps({"config": args.config, **row}), flush=True)
        eng.close()
        return 0
    if args.cmd == "characterize":
        users = [int(u) for u in args.users.split(",")]
        eng = lp.Engine(cfg, _options(wl, min(max(users), args.max_batch)))
        eng.init_weights_random(key, 0.02)
        smp = None
        if args.sampling:
            t, k, p = args.sampling.split(",")
            smp = (float(t), int(k), float(p))
        for row in characterize(eng, wl, shape.vocab, users, args.requests_per_user, sampling=smp):
            print(json.dumps({"config": args.config, "sampling": args.sampling or "greedy", **row}), flush=True)
        eng.close()
        return 0
    opt = _options(wl, args.users)
    free = torch.cuda.mem_get_info()[0]
    arena = int(args.arena_gb * 2**30) if args.arena_gb else int(free * 0.85)
    w_max = search_max_batch_weight(cfg, opt, arena)
    ok, msg = verify_batch_weight(cfg, opt, w_max, arena)
    ok_over, msg_over = verify_batch_weight(cfg, opt, w_max + KV_BLOCK, arena)
    print(json.dumps({"config": args.config, "arena_bytes": arena, "max_batch_weight": w_max,
                      "slots_hold_tokens": opt.max_batch * opt.max_seq_len, "corner_case_ok": ok,
                      "corner_case": msg, "one_block_more_ok": ok_over, "one_block_more": msg_over}), flush=True)
    heaviest = max(r.in_len + r.out_len for r in synth.make_requests(wl, shape.vocab, args.requests))
    weights = sorted({w_max if x == "max" else max(heaviest, int(x)) for x in args.weights.split(",")})
    weights = [w for w in weights if w <= w_max]
    for row in batch_weight_sweep(cfg, wl, weights, args.users, args.requests, key):
        print(json.dumps({"config": args.config, **row}), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
