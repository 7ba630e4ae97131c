"""CPU oracle for the serving step's scheduling and latency accounting:
TEST INFRASTRUCTURE ONLY (tests, the smoke check and the benchmark's CPU leg).

Scheduling follows the paper's description of an inference server (Sec. II-B):
one running batch under continuous batching -- finished requests leave, queued
requests join between iterations -- bounded by the maximum batch weight, the
total number of input plus output tokens of all requests in the batch at any
time.  Readings where the paper is silent:

* A request reserves in_len + out_len tokens of batch weight when admitted and
  releases them when its last token is produced.
* Strict first-come-first-served admission ordered by (arrival, request id):
  admission stops at the first arrived request that does not fit (no free
  slot, batch weight or prompt-token limit of one prefill step).
* Each iteration: admit, then one prefill step over all admitted requests
  (producing each one's first token), then one decode step over every active
  request that still owes tokens (producing one token each).  Rows of a decode
  step are ordered by slot; a request takes the lowest free slot.
* Closed loop with U users and zero think time: the first U requests arrive at
  time 0; when a request finishes, the next unsent request arrives at that time
  and may join at the next iteration.

Latency accounting follows the load-testing metrics of Sec. III-C-3: TTFT
(includes queueing and prompt processing), nTTFT = TTFT / input tokens, ITL
between consecutive output tokens excluding the first, and throughput = output
tokens / duration.  Times are int64 nanoseconds.
"""
from __future__ import annotations

from dataclasses import dataclass, field
import numpy as np


@dataclass
class SimRequest:
    id: int
    in_len: int
    out_len: int
    arrival_ns: int = 0


@dataclass
class Step:
    kind: str            # "prefill" or "decode"
    ids: list            # request ids, in row order
    slots: list          # slot of each row
    ctx: list            # tokens in the KV cache after the step, per row
    plan_ns: int = 0     # when the iteration holding this step was planned
    end_ns: int = 0


@dataclass
class Trace:
    steps: list = field(default_factory=list)
    token_ns: dict = field(default_factory=dict)     # id -> list of token times
    arrival_ns: dict = field(default_factory=dict)   # id -> arrival time


def simulate(requests, max_batch: int, max_batch_weight: int, max_prefill_tokens: int,
             closed_loop: bool, concurrency: int, step_ns, plan_ns=None) -> Trace:
    """Run the admission policy.

    ``step_ns(kind, n_rows, n_tokens, sum_ctx)`` gives each step's duration.
    To replay a recorded run, ``step_ns`` is instead the list of recorded step
    end times, and ``plan_ns`` (open loop only) the list of times at which each
    iteration was planned; without it an iteration is planned when the previous
    step ends.
    """
    reqs = list(requests)
    for r in reqs:
        if r.in_len < 1 or r.out_len < 1 or r.in_len + r.out_len > max_batch_weight \
                or r.in_len > max_prefill_tokens:
            raise ValueError(f"request {r.id} can never be admitted")
    order = {r.id: i for i, r in enumerate(reqs)}
    tr = Trace()
    pending = []                     # arrived-or-future requests not yet admitted
    next_unsent = 0
    if closed_loop:
        for r in reqs[:concurrency]:
            tr.arrival_ns[r.id] = 0
            pending.append(r)
        next_unsent = min(concurrency, len(reqs))
    else:
        for r in reqs:
            tr.arrival_ns[r.id] = int(r.arrival_ns)
            pending.append(r)
    active = {}                      # slot -> [req, emitted]
    weight = 0
    now = 0
    it = 0
    step_idx = 0
    replay = plan_ns is not None
    recorded = not callable(step_ns)
    done = 0
    while done < len(reqs):
        if replay:
            now = int(plan_ns[it])
        pending.sort(key=lambda r: (tr.arrival_ns[r.id], order[r.id]))
        if not active and pending and tr.arrival_ns[pending[0].id] > now:
            if replay:
                raise AssertionError("replayed plan time precedes every arrival")
            now = tr.arrival_ns[pending[0].id]
        admitted, tokens = [], 0
        while pending:
            r = pending[0]
            if tr.arrival_ns[r.id] > now or len(active) + len(admitted) >= max_batch:
                break
            if weight + r.in_len + r.out_len > max_batch_weight:
                break
            if tokens + r.in_len > max_prefill_tokens:
                break
            pending.pop(0)
            admitted.append(r)
            tokens += r.in_len
            weight += r.in_len + r.out_len
        it += 1
        retired = []
        plan_t = now

        def run_step(kind, rows, n_tokens):
            nonlocal now, step_idx
            sum_ctx = sum(c for _, c in rows)
            if recorded:
                end = int(step_ns[step_idx])
            else:
                end = now + int(step_ns(kind, len(rows), n_tokens, sum_ctx))
            st = Step(kind, [r.id for r, _ in rows], [], [c for _, c in rows], plan_ns=plan_t, end_ns=end)
            step_idx += 1
            now = end
            return st

        if admitted:
            rows, slots = [], []
            for r in admitted:
                slot = min(s for s in range(max_batch) if s not in active)
                active[slot] = [r, 1]
                slots.append(slot)
                rows.append((r, r.in_len))
            st = run_step("prefill", rows, tokens)
            st.slots = slots
            tr.steps.append(st)
            for r in admitted:
                tr.token_ns[r.id] = [st.end_ns]
            for s in slots:
                if active[s][0].out_len == 1:
                    retired.append((s, st.end_ns))
            for s, _ in retired:
                r = active.pop(s)[0]
                weight -= r.in_len + r.out_len
                done += 1
        dec = [s for s in sorted(active) if active[s][1] < active[s][0].out_len]
        if dec:
            rows = [(active[s][0], active[s][0].in_len + active[s][1]) for s in dec]
            st = run_step("decode", rows, len(dec))
            st.slots = dec
            tr.steps.append(st)
            fin = []
            for s in dec:
                r = active[s][0]
                active[s][1] += 1
                tr.token_ns[r.id].append(st.end_ns)
                if active[s][1] == r.out_len:
                    fin.append(s)
            for s in fin:
                r = active.pop(s)[0]
                weight -= r.in_len + r.out_len
                done += 1
                retired.append((s, st.end_ns))
        if closed_loop:
            for _, t in retired:
                if next_unsent < len(reqs):
                    nr = reqs[next_unsent]
                    next_unsent += 1
                    tr.arrival_ns[nr.id] = t
                    pending.append(nr)
    return tr


# ------------------------------------------------------------------ metrics

def request_latencies(arrival_ns: int, token_ns):
    """(TTFT, ITL list, e2e) of one request from its token arrival times."""
    t = [int(x) for x in token_ns]
    ttft = t[0] - int(arrival_ns)
    itl = [t[k + 1] - t[k] for k in range(len(t) - 1)]
    return ttft, itl, t[-1] - int(arrival_ns)


def median(values):
    """Median; the mean of the two middle values for an even count."""
    v = sorted(values)
    n = len(v)
    if n == 0:
        return float("nan")
    if n % 2:
        return float(v[n // 2])
    return (v[n // 2 - 1] + v[n // 2]) / 2.0


def summarize(arrivals: dict, token_ns: dict, in_lens: dict):
    """Median TTFT, nTTFT, pooled ITL and end-to-end latency, tail
    percentiles, and throughput over one experiment (Sec. III-C-3)."""
    ttfts, nttfts, itls, e2es = [], [], [], []
    n_tokens = 0
    for rid, times in token_ns.items():
        ttft, itl, e2e = request_latencies(arrivals[rid], times)
        ttfts.append(ttft)
        nttfts.append(ttft / in_lens[rid])
        itls.extend(itl)
        e2es.append(e2e)
        n_tokens += len(times)
    start = min(arrivals.values())
    end = max(max(t) for t in token_ns.values())
    return {
        "ttft_p50_ns": median(ttfts),
        "nttft_p50_ns": median(nttfts),
        "itl_p50_ns": median(itls),
        "e2e_p50_ns": median(e2es),
        "ttft_p90_ns": percentile_nearest_rank(ttfts, 90),
        "itl_p90_ns": percentile_nearest_rank(itls, 90),
        "itl_p99_ns": percentile_nearest_rank(itls, 99),
        "throughput_tok_s": n_tokens / ((end - start) * 1e-9) if end > start else float("inf"),
        "output_tokens": n_tokens,
        "n_requests": len(token_ns),
        "itl_count": len(itls),
    }


def percentile_nearest_rank(values, p: float):
    """p-th percentile by the nearest-rank rule (used only for reporting tails)."""
    v = sorted(values)
    if not v:
        return float("nan")
    k = max(1, int(np.ceil(p / 100.0 * len(v))))
    return float(v[k - 1])
