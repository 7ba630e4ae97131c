"""End-to-end parity of the serving step on the GPU through the C ABI.

* tiny config (fp32 path): greedy tokens bit-exact vs the oracle for every
  request, logits within 1e-4, from host-loaded and device-generated weights;
* bf16 path: teacher-forced logits within 2e-2 of the oracle (tiny shape, and
  the 8B shape truncated to 2 layers at full width on sampled vocabulary rows);
* the run's schedule and token timestamps replayed through the oracle's
  scheduler; per-request latency accounting identities.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import serving as S
from oracle import transformer as T
from paper_2410_02425_amd import lp, synth

pytestmark = pytest.mark.gpu


def cfg_dict(shape):
    return dict(n_layers=shape.n_layers, d_model=shape.d_model, n_heads=shape.n_heads,
                n_kv_heads=shape.n_kv_heads, ffn_dim=shape.ffn_dim, vocab=shape.vocab,
                rope_theta=shape.rope_theta, norm_eps=shape.norm_eps)


def engine_for(shape, max_batch, max_seq, flags=lp.LP_FLAG_KEEP_LOGITS, max_prefill=4096, weight=0):
    """Engine for `shape`; bf16 models compute with fp16 GEMM inputs unless
    flags has LP_FLAG_BF16_ACTIVATIONS."""
    cfg = lp.make_config(shape)
    opt = lp.EngineOptions(max_batch, max_seq, weight, max_prefill, 0, flags)
    return lp.Engine(cfg, opt)


def check_accounting(eng, reqs):
    for r in reqs:
        res = eng.result(r.id)
        times = eng.token_times(r.id)
        ttft, itl, e2e = S.request_latencies(res["arrival_ns"], times)
        assert res["ttft_ns"] == ttft and list(res["itl_ns"]) == itl and res["e2e_ns"] == e2e
        assert e2e == ttft + sum(itl) and len(itl) == r.out_len - 1
        assert ttft > 0 and all(x > 0 for x in itl)


@pytest.mark.parametrize("source", ["blob", "device"])
def test_tiny_fp32_greedy_bit_exact(source):
    shape = synth.SHAPES["tiny"]
    wl = synth.WORKLOADS["tiny"]
    key = synth.workload_seeds(wl.base_seed)[0]
    reqs = synth.make_requests(wl, shape.vocab)
    w = synth.model_weights(shape, key)
    eng = engine_for(shape, 4, 48)
    if source == "blob":
        eng.load_weights(synth.weights_blob(shape, w))
    else:
        eng.init_weights_random(key, 0.02)
    eng.submit(reqs)
    eng.run(lp.LP_CLOSED_LOOP, 4)
    m = T.Model(cfg_dict(shape), w)
    min_margin = np.inf
    for r in reqs:
        toks, logits = T.generate(m, r.prompt, r.out_len)
        res = eng.result(r.id)
        got_logits = np.stack([eng.logits(r.id, k) for k in range(r.out_len)])
        assert np.max(np.abs(got_logits - logits)) <= 1e-4
        np.testing.assert_array_equal(res["tokens"], toks)
        srt = np.sort(logits, axis=1)
        min_margin = min(min_margin, float(np.min(srt[:, -1] - srt[:, -2])))
    print(f"oracle minimum top-1/top-2 margin over all tokens: {min_margin:.3e}")
    check_accounting(eng, reqs)


def test_tiny_fp32_random_gains_mixed_lengths():
    shape = synth.SHAPES["tiny"]
    w = synth.model_weights(shape, 99, std=0.05, gain_std=0.3)
    rng = np.random.default_rng(5)
    reqs = [synth.Request(i, rng.integers(0, shape.vocab, size=n).astype(np.int32), o)
            for i, (n, o) in enumerate([(1, 9), (70, 3), (5, 1), (130, 12), (64, 7), (2, 20)])]
    eng = engine_for(shape, 3, 160, max_prefill=200)
    eng.load_weights(synth.weights_blob(shape, w))
    eng.submit(reqs)
    eng.run(lp.LP_CLOSED_LOOP, 3)
    m = T.Model(cfg_dict(shape), w)
    for r in reqs:
        toks, logits = T.generate(m, r.prompt, r.out_len)
        got = np.stack([eng.logits(r.id, k) for k in range(r.out_len)])
        assert np.max(np.abs(got - logits)) <= 1e-4
        np.testing.assert_array_equal(eng.result(r.id)["tokens"], toks)
    # the schedule is the oracle's policy replayed on the recorded step times
    log = eng.step_log()
    sreqs = [S.SimRequest(r.id, r.in_len, r.out_len) for r in reqs]
    tr = S.simulate(sreqs, 3, eng.max_batch_weight(), 200, True, 3, [s["end_ns"] for s in log])
    assert [(s.kind, s.ids, s.slots) for s in tr.steps] == [(s["kind"], s["ids"], s["slots"]) for s in log]
    for r in reqs:
        assert list(eng.token_times(r.id)) == tr.token_ns[r.id]
    check_accounting(eng, reqs)


def test_tiny_degenerate_requests():
    """Edges of the serving step: a run with nothing submitted is refused
    (LP_ESTATE), a request longer than max_seq_len is refused at submission
    (LP_EINVAL); a one-token prompt with one output token and a request whose
    in_len + out_len is exactly max_seq_len match the oracle bit for bit."""
    shape = synth.SHAPES["tiny"]
    w = synth.model_weights(shape, 7)
    eng = engine_for(shape, 2, 48, max_prefill=64)
    eng.load_weights(synth.weights_blob(shape, w))
    with pytest.raises(lp.LPError) as err:
        eng.run(lp.LP_CLOSED_LOOP, 2)
    assert err.value.code == lp.LP_ESTATE
    rng = np.random.default_rng(11)
    too_long = [synth.Request(0, rng.integers(0, shape.vocab, size=41).astype(np.int32), 8)]
    with pytest.raises(lp.LPError) as err:
        eng.submit(too_long)
    assert err.value.code == lp.LP_EINVAL
    reqs = [synth.Request(0, rng.integers(0, shape.vocab, size=1).astype(np.int32), 1),
            synth.Request(1, rng.integers(0, shape.vocab, size=40).astype(np.int32), 8)]
    eng.submit(reqs)
    eng.run(lp.LP_CLOSED_LOOP, 2)
    m = T.Model(cfg_dict(shape), w)
    for r in reqs:
        toks, logits = T.generate(m, r.prompt, r.out_len)
        got = np.stack([eng.logits(r.id, k) for k in range(r.out_len)])
        assert np.max(np.abs(got - logits)) <= 1e-4
        np.testing.assert_array_equal(eng.result(r.id)["tokens"], toks)
    check_accounting(eng, reqs)


def mixed_requests(vocab, n, seed, max_in=130, min_out=8, max_out=20):
    """n requests with prompts of 1..max_in tokens (a third of them above 64,
    so prefill rows span several tiles) and min_out..max_out output tokens,
    except every eleventh request, which wants a single token (decided by
    prefill alone)."""
    rng = np.random.default_rng(seed)
    reqs = []
    for i in range(n):
        n_in = int(rng.integers(65, max_in + 1)) if i % 3 == 0 else int(rng.integers(1, 65))
        n_out = 1 if i % 11 == 5 else int(rng.integers(min_out, max_out + 1))
        reqs.append(synth.Request(i, rng.integers(0, vocab, size=n_in).astype(np.int32), n_out))
    return reqs


def test_tiny_fp32_64_slots_closed_loop():
    """The benchmark's batch configuration at the tiny shape: 64 slots, 64
    closed-loop users, 168 requests of mixed lengths (Sec. II-B: one running
    batch, refilled as requests finish).  Every step has up to 64 decode rows
    and prefill steps pack up to 64 prompts.  Greedy tokens bit-exact and
    logits within 1e-4 of the oracle for every request; the schedule and every
    token time replay through the oracle's scheduler."""
    shape = synth.SHAPES["tiny"]
    w = synth.model_weights(shape, 21)
    reqs = mixed_requests(shape.vocab, 168, 64)
    eng = engine_for(shape, 64, 160)
    eng.load_weights(synth.weights_blob(shape, w))
    eng.submit(reqs)
    eng.run(lp.LP_CLOSED_LOOP, 64)
    log = eng.step_log()
    assert max(s["n_rows"] for s in log if s["kind"] == "decode") == 64  # full 64-row decode steps ran
    assert max(s["n_rows"] for s in log if s["kind"] == "prefill") >= 32  # and wide packed prefills
    m = T.Model(cfg_dict(shape), w)
    min_margin = np.inf
    for r in reqs:
        toks, logits = T.generate(m, r.prompt, r.out_len)
        got = np.stack([eng.logits(r.id, k) for k in range(r.out_len)])
        assert np.max(np.abs(got - logits)) <= 1e-4, r.id
        np.testing.assert_array_equal(eng.result(r.id)["tokens"], toks)
        srt = np.sort(logits, axis=1)
        min_margin = min(min_margin, float(np.min(srt[:, -1] - srt[:, -2])))
    print(f"oracle minimum top-1/top-2 margin over all tokens: {min_margin:.3e}")
    sreqs = [S.SimRequest(r.id, r.in_len, r.out_len) for r in reqs]
    tr = S.simulate(sreqs, 64, eng.max_batch_weight(), 4096, True, 64, [s["end_ns"] for s in log])
    assert [(s.kind, s.ids, s.slots) for s in tr.steps] == [(s["kind"], s["ids"], s["slots"]) for s in log]
    for r in reqs:
        assert list(eng.token_times(r.id)) == tr.token_ns[r.id]
    check_accounting(eng, reqs)


def test_tiny_bf16_64_slots_teacher_forced():
    """The 16-bit kernels at 64 rows through the engine (decode GEMMs with four
    16-row tiles and split K, 64-row decode attention, a 64-prompt packed
    prefill) at the tiny shape with one KV head per two query heads; teacher
    forced, logits within 2e-2 of the oracle."""
    shape = synth.ModelShape("tiny-bf16", 2, 256, 4, 2, 688, 1024)
    w = synth.model_weights(shape, 12)
    reqs = mixed_requests(shape.vocab, 80, 65, min_out=4, max_out=8)
    eng = engine_for(shape, 64, 160)
    eng.load_weights(synth.weights_blob(shape, w))
    eng.submit(reqs)
    m = T.Model(cfg_dict(shape), w)
    ref = {}
    for r in reqs:
        toks, logits = T.generate(m, r.prompt, r.out_len)
        ref[r.id] = logits
        eng.set_forced_tokens(r.id, toks[:-1])
    eng.run(lp.LP_CLOSED_LOOP, 64)
    assert max(s["n_rows"] for s in eng.step_log() if s["kind"] == "decode") == 64
    for r in reqs:
        got = np.stack([eng.logits(r.id, k) for k in range(r.out_len)])
        assert np.max(np.abs(got - ref[r.id])) <= 2e-2, r.id
    check_accounting(eng, reqs)


def test_tiny_open_loop_replay():
    shape = synth.SHAPES["tiny"]
    w = synth.model_weights(shape, 3)
    rng = np.random.default_rng(8)
    reqs = []
    t = 0
    for i in range(12):
        t += int(rng.integers(0, 3_000_000))
        reqs.append(synth.Request(i, rng.integers(0, shape.vocab, size=int(rng.integers(1, 40))).astype(np.int32),
                                  int(rng.integers(1, 8)), t))
    eng = engine_for(shape, 2, 64, flags=0, max_prefill=64, weight=100)
    eng.load_weights(synth.weights_blob(shape, w))
    eng.submit(reqs)
    eng.run(lp.LP_OPEN_LOOP, 0)
    log = eng.step_log()
    # replay with the recorded planning times of each iteration
    plan = []
    for s in log:
        if not plan or s["plan_ns"] != plan[-1]:
            plan.append(s["plan_ns"])
    sreqs = [S.SimRequest(r.id, r.in_len, r.out_len, r.arrival_ns) for r in reqs]
    tr = S.simulate(sreqs, 2, 100, 64, False, 0, [s["end_ns"] for s in log], plan_ns=plan)
    assert [(s.kind, s.ids, s.slots) for s in tr.steps] == [(s["kind"], s["ids"], s["slots"]) for s in log]
    check_accounting(eng, reqs)
    m = T.Model(cfg_dict(shape), w)
    for r in reqs[:4]:
        np.testing.assert_array_equal(eng.result(r.id)["tokens"], T.generate(m, r.prompt, r.out_len)[0])


# Logit tolerance of the bf16 model path.  fp16 GEMM inputs / KV cache: the
# stated 2e-2.  bf16 GEMM inputs / KV cache: rounding 8x coarser; replaying the
# bf16 rounding points in float64 on the 2-layer 8B-shape case gives 5.2e-2,
# so that mode is held to 8e-2.
TOL = {0: 2e-2, lp.LP_FLAG_BF16_ACTIVATIONS: 8e-2}


@pytest.mark.parametrize("kv_heads", [4, 1])
@pytest.mark.parametrize("source", ["blob", "device"])
@pytest.mark.parametrize("act", [0, lp.LP_FLAG_BF16_ACTIVATIONS])
def test_tiny_bf16_teacher_forced_logits(act, source, kv_heads):
    """ffn_dim 688 is not a multiple of 32: the down projection's weight tiles
    carry zero padding, written by the host tiling (blob) or left by the
    engine's clearing of the weight region (device generator).  With one KV
    head, k and v are 64-row pieces of the fused QKV matrix beside a 256-row
    q, placed by the host's strided copy or generated in place."""
    shape = synth.ModelShape("tiny-bf16", 2, 256, 4, kv_heads, 688, 1024)
    w = synth.model_weights(shape, 11)
    rng = np.random.default_rng(2)
    reqs = [synth.Request(i, rng.integers(0, 1024, size=n).astype(np.int32), 6) for i, n in enumerate([32, 1, 70])]
    eng = engine_for(shape, 4, 96, flags=lp.LP_FLAG_KEEP_LOGITS | act)
    if source == "blob":
        eng.load_weights(synth.weights_blob(shape, w))
    else:
        eng.init_weights_random(11, 0.02)
    eng.submit(reqs)
    m = T.Model(cfg_dict(shape), w)
    ref = {}
    for r in reqs:
        toks, logits = T.generate(m, r.prompt, r.out_len)
        ref[r.id] = logits
        eng.set_forced_tokens(r.id, toks[:-1])
    eng.run(lp.LP_CLOSED_LOOP, 4)
    for r in reqs:
        got = np.stack([eng.logits(r.id, k) for k in range(r.out_len)])
        assert np.max(np.abs(got - ref[r.id])) <= TOL[act]


# Full-width shapes of every bf16 configuration at reduced depth: 8B (GQA,
# 4 query heads per KV head), 7B and 13B (MHA: one), 70B (8 per KV head,
# d = 8192).  Two layers, so that the first layer's down-projection partials
# are folded into the second layer's attention norm at every width.
# (name, layers, prompt lengths, activation flags).
FULL_WIDTH_CASES = [
    ("8b", 2, [67, 1, 300], 0),
    ("8b", 2, [67, 1, 300], lp.LP_FLAG_BF16_ACTIVATIONS),
    ("7b", 2, [67, 1, 130], 0),
    ("13b", 2, [40, 1, 90], 0),
    ("70b", 2, [40, 1, 90], 0),
]

_LAYER_CACHE = {}


def full_width_layers(shape, seed):
    """Host values of every layer tensor of `shape` (device generator's
    definition), kept for the cases that share a shape."""
    key = (shape.name, shape.n_layers, seed)
    if key not in _LAYER_CACHE:
        _LAYER_CACHE.clear()
        w = {}
        for nm, tid, (rows, cols) in synth.tensor_shapes(shape):
            if nm in ("embed", "lm_head"):
                continue
            v = synth.tensor_values(seed, tid, np.arange(rows), cols, 0.02, shape.dtype, gain=synth.is_gain(nm))
            w[nm] = v.reshape(cols) if rows == 1 else v
        _LAYER_CACHE[key] = w
    return _LAYER_CACHE[key]


def full_width_check(shape, reqs, forced, act, max_batch, max_seq=512, max_prefill=1024, n_vocab_rows=2048):
    """Runs `reqs` teacher-forced with `forced` tokens on device-generated
    weights, then compares the logits of every output position with the
    oracle's on n_vocab_rows sampled vocabulary rows plus the GPU's argmax
    (teacher forcing keeps both on one sequence).  Returns the max error."""
    seed = 0x8B8B
    rng = np.random.default_rng(4)
    eng = engine_for(shape, max_batch, max_seq, flags=lp.LP_FLAG_KEEP_LOGITS | act, max_prefill=max_prefill)
    eng.init_weights_random(seed, 0.02)
    eng.submit(reqs)
    for r in reqs:
        eng.set_forced_tokens(r.id, forced[r.id])
    eng.run(lp.LP_CLOSED_LOOP, max_batch)
    log = eng.step_log()
    decode_rows = max(s["n_rows"] for s in log if s["kind"] == "decode")
    full_width_check.max_prefill_tokens = max(s["n_tokens"] for s in log if s["kind"] == "prefill")
    got_all = {r.id: np.stack([eng.logits(r.id, k) for k in range(r.out_len)]) for r in reqs}
    eng.close()
    # oracle weights: every layer tensor, the embedding rows used (token ids
    # remapped below), sampled LM-head rows
    names = synth.tensor_shapes(shape)
    w = dict(full_width_layers(shape, seed))
    vocab_rows = np.unique(np.concatenate([rng.integers(0, shape.vocab, n_vocab_rows), [0, shape.vocab - 1]]))
    used = np.unique(np.concatenate([r.prompt for r in reqs] + [np.array(forced[r.id], dtype=np.int64)
                                                                 for r in reqs]))
    w["embed"] = synth.tensor_values(seed, names[0][1], used, shape.d_model, 0.02, shape.dtype)
    gpu_top = {rid: np.argmax(g, axis=1) for rid, g in got_all.items()}
    extra = np.unique(np.concatenate(list(gpu_top.values())))
    rows_needed = np.unique(np.concatenate([vocab_rows, extra]))
    w["lm_head"] = np.zeros((1, shape.d_model), dtype=np.float32)  # replaced below
    m = T.Model(cfg_dict(shape), w)
    m.w["lm_head"] = synth.tensor_values(seed, names[-1][1], rows_needed, shape.d_model, 0.02,
                                         shape.dtype).astype(np.float64)
    worst = 0.0
    for r in reqs:
        toks_in = np.searchsorted(used, np.concatenate([r.prompt, np.array(forced[r.id], dtype=np.int64)]))
        ref = T.forward(m, toks_in, T.KVCache(m), "all")[r.in_len - 1:]
        got = got_all[r.id][:, rows_needed]
        err = float(np.max(np.abs(got - ref)))
        worst = max(worst, err)
        assert err <= TOL[act], (r.id, err)
        # the GPU's greedy choice is (within tolerance) the oracle's best among the sampled rows
        pos = np.searchsorted(rows_needed, gpu_top[r.id])
        assert np.all(ref[np.arange(len(pos)), pos] >= ref.max(axis=1) - 2 * TOL[act])
    print(f"{shape.name} x{shape.n_layers}: {len(reqs)} requests, decode steps up to {decode_rows} rows, "
          f"max |logit error| on {rows_needed.size} rows = {worst:.3e}")
    return worst, decode_rows


def test_8b_two_layers_64_slots_teacher_forced():
    """The benchmark's configuration (8B shape, 64 slots) at two layers: 64
    concurrent requests with 1..48-token prompts and 2..4 output tokens, so
    the first prefill packs 64 prompts and every decode step runs the 64-row
    launches of the benchmark (QKV and O split K, the sixteen-wave LM head
    with four row tiles, 64-row decode attention).  Logits within 2e-2 of the
    oracle on sampled vocabulary rows (Sec. II-A: prefill, then decode in one
    running batch, Sec. II-B)."""
    shape = synth.SHAPES["8b"].with_layers(2)
    rng = np.random.default_rng(64)
    reqs, forced = [], {}
    for i in range(64):
        n_in, n_out = int(rng.integers(1, 49)), int(rng.integers(2, 5))
        reqs.append(synth.Request(i, rng.integers(0, shape.vocab, size=n_in).astype(np.int32), n_out))
        forced[i] = rng.integers(0, shape.vocab, size=n_out - 1).tolist()
    _, rows = full_width_check(shape, reqs, forced, 0, 64, max_seq=64, max_prefill=4096, n_vocab_rows=1024)
    assert rows == 64


@pytest.mark.parametrize("lo,hi,seed,paired", [(60, 73, 4300, ("O",)), (44, 51, 3000, ("QKV", "gate/up"))])
def test_8b_two_layers_large_prefill_two_workgroups_per_cu(lo, hi, seed, paired):
    """A packed prefill of 64 prompts (about 4,250 or 3,000 tokens) at the 8B
    shape (two layers): the projections the planner gives two 128-row
    workgroups per CU run that kernel with their engine epilogues (the
    residual add of O in the first case; RoPE and the KV append of QKV and
    the SiLU gate of gate/up in the second), the others their own plans
    (256-row tiles, K splits folded by the next RMSNorm); then decode steps
    at 64 rows.  Logits within 2e-2 of the oracle on sampled vocabulary rows
    (Sec. II-A)."""
    shape = synth.SHAPES["8b"].with_layers(2)
    rng = np.random.default_rng(seed)
    reqs, forced = [], {}
    for i in range(64):
        n_in, n_out = int(rng.integers(lo, hi)), int(rng.integers(2, 4))
        reqs.append(synth.Request(i, rng.integers(0, shape.vocab, size=n_in).astype(np.int32), n_out))
        forced[i] = rng.integers(0, shape.vocab, size=n_out - 1).tolist()
    M = sum(r.in_len for r in reqs)
    d, F, hd = shape.d_model, shape.ffn_dim, shape.head_dim
    names = ["QKV", "O", "gate/up", "down"]
    plans = dict(zip(names, [lp.op_gemm_plan(M, N, K, 0) for N, K in
                             [((shape.n_heads + 2 * shape.n_kv_heads) * hd, d), (d, shape.n_heads * hd), (2 * F, d),
                              (d, F)]]))
    assert [nm for nm in names if plans[nm][0] == "prefill_pair"] == list(paired), (M, plans)
    _, rows = full_width_check(shape, reqs, forced, 0, 64, max_seq=80, max_prefill=8192, n_vocab_rows=1024)
    assert rows == 64 and full_width_check.max_prefill_tokens == M  # all 64 prompts in one prefill step


@pytest.mark.parametrize("name,layers,lens,act", FULL_WIDTH_CASES)
def test_full_width_teacher_forced(name, layers, lens, act):
    """A configuration's shape at full width and reduced depth."""
    shape = synth.SHAPES[name].with_layers(layers)
    rng = np.random.default_rng(4)
    outs = [3, 3, 2]
    reqs = [synth.Request(i, rng.integers(0, shape.vocab, size=n).astype(np.int32), o)
            for i, (n, o) in enumerate(zip(lens, outs))]
    forced = {0: [5, shape.vocab - 1], 1: [99, 1], 2: [42]}
    full_width_check(shape, reqs, forced, act, 4)
