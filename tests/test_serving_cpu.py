"""Continuous batching with preemption and the serving simulation: the
oracle pinned to the paper's toy example and to hand-derived preemption
cases, then the native engine (queue-only contexts, through the C ABI)
compared with the oracle event for event."""
import json
import os
import random
from fractions import Fraction

import numpy as np
import pytest

from oracle import queue as Q
from oracle import serving as S

asr = pytest.importorskip("paper_2603_11273_amd.asr")
from paper_2603_11273_amd import synth  # noqa: E402

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "toy_example.json")
SR = 16000


def _toy():
    return json.load(open(GOLDEN))


def _ctx(policy, n_slots, max_admit=1, kv_capacity=0, cross_tokens=0, tok_num=27, tok_den=10,
         max_queue=4096):
    cfg = asr.model_cfg(synth.SHAPES["tiny"], max_slots=n_slots, max_prefill=max_admit,
                        max_decode=min(n_slots, 128), max_queue=max_queue)
    c = asr.Context(cfg, device=-1)
    c.set_policy(policy)
    c.serve_config(kv_capacity=kv_capacity, cross_tokens=cross_tokens, max_admit=max_admit,
                   tok_num=tok_num, tok_den=tok_den)
    return c


# --------------------------------------------------------------------------- oracle pins
@pytest.mark.parametrize("policy,key", [(Q.FCFS, "fcfs_completion_s"), (Q.SJF, "sjf_completion_s"),
                                        (Q.HRRN, "sjf_completion_s")])
def test_oracle_toy_example(policy, key):
    """Figure 1: one request at a time, 1 s encoder + 10 tokens/s decoding,
    5 tokens per audio-second; completion times 5/8/10 s (FCFS) and 2/5/10 s
    (SJF; HRRN orders the same three requests identically: all ratios are 1
    at t = 0 and the shorter job has the higher ratio at t = 2 s)."""
    g = _toy()
    eng = S.Engine(policy, n_slots=1, max_admit=1, kv_capacity=0, cross_tokens=0, tok_num=5,
                   tok_den=1)
    for r in g["requests"]:
        eng.submit(r["id"], r["duration_s"] * SR, SR, arrival_us=0)
    info, t_end = S.simulate(eng, S.Cost(prefill_us=g["encoder_s"] * 10**6,
                                         step_us=10**6 // g["decode_tokens_per_s"], row_us=0))
    for r in g["requests"]:
        d = info[r["id"]]
        assert d["n_tokens"] == r["tokens"]
        assert d["finish_us"] == g[key][str(r["id"])] * 10**6
    num, den = g["fcfs_mean_num_den" if key.startswith("fcfs") else "sjf_mean_num_den"]
    assert Fraction(sum(d["finish_us"] for d in info.values()), 3 * 10**6) == Fraction(num, den)


def test_oracle_token_counts():
    # round-half-up of 2.7 tokens per second, clamped to [1, min(448, max_tokens)]
    assert S.tokens_for(SR, SR, 448, 27, 10) == 3                    # 2.7 -> 3
    assert S.tokens_for(SR * 5 // 2, SR, 448, 27, 10) == 7           # 6.75 -> 7
    assert S.tokens_for(SR * 30, SR, 448, 27, 10) == 81
    assert S.tokens_for(1, SR, 448, 27, 10) == 1
    assert S.tokens_for(SR * 30, SR, 448, 100, 1) == 448
    assert S.tokens_for(SR * 30, SR, 50, 27, 10) == 50
    assert S.tokens_for(5 * SR, SR, 448, 1, 2) == 3                  # 2.5 rounds up


def test_oracle_preemption_rule_by_hand():
    """Hand-built pressure: A (3 s, arrives at 0 us), B (1 s, at 1 us), C
    (2 s, at 2 us); 10 tokens per audio-second (30, 10, 20 tokens; each fits
    the pool alone), cross share 4 positions, pool 40, one admission per step,
    steps at t = 0, 1, 2, ... us.  Before the step at t >= 2 the three hold t,
    t-1, t-2 tokens (B, with 10, is still running at t = 10), so the step
    needs 3*4 + (t+1) + t + (t-1) = 12 + 3t positions: first above 40 at
    t = 10, where exactly one request must go (evicting any one brings the
    need to at most 28).  SJF evicts the longest job (A), FCFS the last
    admitted (C), HRRN the lowest (wait + job) / job -- A, with the ratios
    written out below."""
    def run(policy):
        eng = S.Engine(policy, n_slots=3, max_admit=1, kv_capacity=40, cross_tokens=4,
                       tok_num=10, tok_den=1)
        eng.submit(1, 3 * SR, SR, 0)        # 30 tokens
        eng.submit(2, 1 * SR, SR, 1)        # 10 tokens
        eng.submit(3, 2 * SR, SR, 2)        # 20 tokens
        for t in range(12):
            res = eng.step(t)
            if res.preempted:
                return t, res.preempted
        return None
    assert run(Q.SJF) == (10, [1])          # largest job: A
    assert run(Q.FCFS) == (10, [3])         # last admitted: C
    # HRRN at t = 10 us: ratios (w + e) / e with e = duration in us
    r = {1: Fraction(10 + 3_000_000, 3_000_000), 2: Fraction(9 + 1_000_000, 1_000_000),
         3: Fraction(8 + 2_000_000, 2_000_000)}
    assert min(r, key=lambda k: r[k]) == 1 and run(Q.HRRN) == (10, [1])


def test_oracle_pool_never_exceeded_and_all_finish():
    rng = random.Random(5)
    for policy in (Q.FCFS, Q.SJF, Q.HRRN):
        eng = S.Engine(policy, n_slots=8, max_admit=2, kv_capacity=1500 + 448 + 600,
                       cross_tokens=300, tok_num=27, tok_den=10)
        n = 40
        for i in range(n):
            eng.submit(i, rng.randrange(SR, 30 * SR), SR, rng.randrange(0, 2_000_000))
        done, t = set(), 0
        while len(done) < n:
            res = eng.step(t)
            held = sum(eng.cross_tokens + r.generated for r in eng.running)
            assert held <= eng.kv_capacity
            done.update(res.finished)
            t += 50_000
        assert not eng.running and not eng.queue.reqs


def test_percentile_nearest_rank_matches_numpy():
    rng = np.random.default_rng(3)
    for n in (1, 2, 7, 100):
        v = rng.integers(0, 10**6, n).tolist()
        for p in (50, 90):
            assert S.percentile_nearest_rank(v, p) == int(np.percentile(v, p, method="inverted_cdf"))


def test_oracle_dynamic_rule_by_hand():
    """The switching rule on hand-built queues at now = 10 s (depth_low 2,
    starvation threshold ratio 3): two eligible requests -> FCFS whatever
    their waits; three short waits -> SJF; one request waiting 9 s for a 4 s
    job (ratio (9 + 4) / 4 = 3.25 > 3) -> HRRN; a request not yet arrived
    counts for nothing."""
    R = lambda rid, arr_s, dur_s: Q.Req(rid, int(arr_s * 1e6), 0, SR, int(dur_s * 1e6), 448)  # noqa: E731
    now = 10_000_000
    three = Fraction(3)
    assert S.dynamic_policy([R(1, 0, 1), R(2, 1, 9)], now, 2, three) == Q.FCFS
    assert S.dynamic_policy([R(1, 0, 1), R(2, 1, 9), R(3, 12, 1)], now, 2, three) == Q.FCFS
    assert S.dynamic_policy([R(1, 9, 1), R(2, 9.5, 2), R(3, 8, 5)], now, 2, three) == Q.SJF
    # ratios: (1 + 1)/1 = 2, (0.5 + 2)/2 = 1.25, (2 + 5)/5 = 1.4 -> no starvation
    assert S.dynamic_policy([R(1, 9, 1), R(2, 9.5, 2), R(3, 1, 4)], now, 2, three) == Q.HRRN
    # the boundary is strict: ratio exactly 3 ((8 + 4)/4) stays SJF
    assert S.dynamic_policy([R(1, 9, 1), R(2, 9.5, 2), R(3, 2, 4)], now, 2, three) == Q.SJF


# --------------------------------------------------------------------------- native vs oracle
def test_native_toy_example():
    g = _toy()
    for policy, key in ((asr.FCFS, "fcfs_completion_s"), (asr.SJF, "sjf_completion_s"),
                        (asr.HRRN, "sjf_completion_s")):
        c = _ctx(policy, n_slots=1, tok_num=5, tok_den=1)
        ids = []
        for r in g["requests"]:
            c.submit(r["id"], None, n_samples=r["duration_s"] * SR, arrival_us=0)
            ids.append(r["id"])
        info, _ = c.serve_simulate(ids, prefill_us=10**6, step_us=100_000, row_us=0)
        for r in g["requests"]:
            assert info[r["id"]]["finish_us"] == g[key][str(r["id"])] * 10**6
            assert info[r["id"]]["n_tokens"] == r["tokens"]


def _workload(seed, n, rate, uniform=False, burst=False):
    durs = synth.durations_uniform(seed, n) if uniform else synth.durations_lognormal(seed, n)
    ns = synth.n_samples_of(durs)
    arr = np.zeros(n, np.int64) if burst else synth.poisson_arrivals_us(seed, n, rate)
    return [int(x) for x in ns], [int(a) for a in arr]


CASES = [
    # policy, slots, admit, capacity, cross, n, rate, uniform, burst
    (Q.FCFS, 16, 4, 0, 1500, 120, 20.0, False, False),
    (Q.SJF, 16, 4, 0, 1500, 120, 20.0, False, False),
    (Q.HRRN, 16, 4, 0, 1500, 120, 20.0, True, False),
    # pool pressure: a small cross share lets many requests in, whose growth
    # then overflows the pool
    (Q.FCFS, 16, 4, 8 * 100 + 448, 100, 120, 25.0, False, False),
    (Q.SJF, 16, 4, 8 * 100 + 448, 100, 120, 25.0, True, False),
    (Q.HRRN, 16, 4, 8 * 100 + 448, 100, 120, 25.0, False, False),
    (Q.HRRN, 32, 8, 12 * 100 + 448, 100, 200, 0.0, False, True),
    (Q.SJF, 32, 8, 12 * 100 + 448, 100, 200, 0.0, True, True),
    (Q.FCFS, 32, 8, 12 * 100 + 448, 100, 200, 0.0, True, True),
]


DYN = dict(dynamic=True, depth_low=4, starve=(3, 1))
CASES_DYN = [
    (Q.FCFS, 16, 4, 0, 1500, 200, 60.0, False, False),
    (Q.SJF, 16, 4, 8 * 100 + 448, 100, 200, 80.0, True, False),
    (Q.HRRN, 32, 8, 12 * 100 + 448, 100, 300, 0.0, False, True),
]


def _engines(case, seed, dyn=None):
    policy, slots, admit, cap, cross, n, rate, uniform, burst = case
    ns, arr = _workload(seed + n, n, rate, uniform, burst)
    c = _ctx(policy, n_slots=slots, max_admit=admit, kv_capacity=cap, cross_tokens=cross)
    kw = {}
    if dyn:
        c.serve_config(kv_capacity=cap, cross_tokens=cross, max_admit=admit, **dyn)
        kw = dict(dynamic=True, depth_low=dyn["depth_low"], starve=Fraction(*dyn["starve"]))
    eng = S.Engine(policy, n_slots=slots, max_admit=admit, kv_capacity=cap, cross_tokens=cross,
                   **kw)
    for i in range(n):
        c.submit(i, None, n_samples=ns[i], arrival_us=arr[i])
        eng.submit(i, ns[i], SR, arr[i])
    return c, eng, n


@pytest.mark.parametrize("case", CASES[3:6])
def test_native_deferred_first_token_matches_oracle(case):
    """Overlapped-prefill schedule: admitted requests decode from the next
    step on (pool pressure cases)."""
    policy, slots, admit, cap, cross, n, rate, uniform, burst = case
    ns, arr = _workload(20260360 + n, n, rate, uniform, burst)
    c = _ctx(policy, n_slots=slots, max_admit=admit, kv_capacity=cap, cross_tokens=cross)
    c.serve_config(kv_capacity=cap, cross_tokens=cross, max_admit=admit, overlap=True)
    eng = S.Engine(policy, n_slots=slots, max_admit=admit, kv_capacity=cap, cross_tokens=cross,
                   defer_first=True)
    for i in range(n):
        c.submit(i, None, n_samples=ns[i], arrival_us=arr[i])
        eng.submit(i, ns[i], SR, arr[i])
    t, done = 0, 0
    while done < n:
        got = c.serve_plan(t)
        ref = eng.step(t)
        assert got["preempted"] == ref.preempted, t
        assert list(zip(got["admitted"], got["admitted_slot"])) == ref.admitted, t
        assert got["decoded"] == ref.decoded, t
        assert not set(got["decoded"]) & set(got["admitted"])
        assert got["finished"] == ref.finished, t
        done += len(ref.finished)
        t += 40_000


@pytest.mark.parametrize("case", CASES_DYN)
def test_native_dynamic_steps_match_oracle(case):
    c, eng, n = _engines(case, 20260350, DYN)
    t, done, seen = 0, 0, set()
    while done < n:
        got = c.serve_plan(t)
        ref = eng.step(t)
        assert got["policy"] == ref.policy, t
        assert got["preempted"] == ref.preempted, t
        assert list(zip(got["admitted"], got["admitted_slot"])) == ref.admitted, t
        assert got["decoded"] == ref.decoded, t
        assert got["finished"] == ref.finished, t
        done += len(ref.finished)
        seen.add(ref.policy)
        t += 40_000
    assert c.serve_stats() == eng.steps_by_policy
    assert len(seen) >= 2, "the case was meant to switch policies"


@pytest.mark.parametrize("case", CASES)
def test_native_steps_match_oracle(case):
    policy, slots, admit, cap, cross, n, rate, uniform, burst = case
    ns, arr = _workload(20260320 + n, n, rate, uniform, burst)
    c = _ctx(policy, n_slots=slots, max_admit=admit, kv_capacity=cap, cross_tokens=cross)
    eng = S.Engine(policy, n_slots=slots, max_admit=admit, kv_capacity=cap, cross_tokens=cross)
    for i in range(n):
        c.submit(i, None, n_samples=ns[i], arrival_us=arr[i])
        eng.submit(i, ns[i], SR, arr[i])
    t, done, n_pre = 0, 0, 0
    while done < n:
        got = c.serve_plan(t)
        ref = eng.step(t)
        assert got["preempted"] == ref.preempted, t
        assert list(zip(got["admitted"], got["admitted_slot"])) == ref.admitted, t
        assert got["decoded"] == ref.decoded, t
        assert got["finished"] == ref.finished, t
        done += len(ref.finished)
        n_pre += len(ref.preempted)
        t += 40_000
    if cap > 0:
        assert n_pre > 0, "the case was meant to exercise preemption"


@pytest.mark.parametrize("case", CASES)
def test_native_simulation_matches_oracle(case):
    policy, slots, admit, cap, cross, n, rate, uniform, burst = case
    ns, arr = _workload(20260330 + n, n, rate, uniform, burst)
    c = _ctx(policy, n_slots=slots, max_admit=admit, kv_capacity=cap, cross_tokens=cross)
    eng = S.Engine(policy, n_slots=slots, max_admit=admit, kv_capacity=cap, cross_tokens=cross)
    for i in range(n):
        c.submit(i, None, n_samples=ns[i], arrival_us=arr[i])
        eng.submit(i, ns[i], SR, arr[i])
    cost = dict(prefill_us=3300, step_us=9000, row_us=25)
    got, t_end = c.serve_simulate(list(range(n)), **cost)
    ref, t_ref = S.simulate(eng, S.Cost(**cost))
    assert t_end == t_ref
    for i in range(n):
        for k in ("first_us", "finish_us", "n_tokens", "n_preempt", "token_us"):
            assert got[i][k] == ref[i][k], (i, k)


def test_native_rejects_misuse():
    c = _ctx(asr.SJF, n_slots=4)
    with pytest.raises(asr.AsrError):
        c.pop_batch(0, 1)                     # manual API is off in serve mode
    with pytest.raises(asr.AsrError):
        c.serve_tokens(99)                    # unknown request
    c3 = _ctx(asr.SJF, n_slots=4, kv_capacity=1550, cross_tokens=1500)
    c3.submit(1, None, n_samples=30 * SR // 10)          # 8 tokens: fits
    with pytest.raises(asr.AsrError):
        c3.submit(2, None, n_samples=30 * SR)            # 81 tokens + 1500 > 1550
    cfg = asr.model_cfg(synth.SHAPES["tiny"], max_slots=4, max_prefill=1, max_decode=4)
    c2 = asr.Context(cfg, device=-1)
    c2.submit(7, None, n_samples=30 * SR)
    with pytest.raises(asr.AsrError):
        c2.serve_config(kv_capacity=1550, cross_tokens=1500)   # a waiting request cannot fit
    with pytest.raises(asr.AsrError):
        c2.serve_plan(0)                      # not configured
