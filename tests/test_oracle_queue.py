"""Pins for the queue oracle: the paper's worked example, closed forms of the
HRRN ratio and brute force over all service orders."""
import itertools
import json
import os
import random
from fractions import Fraction

import pytest

from oracle import queue as Q

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "toy_example.json")


def _toy():
    with open(GOLDEN) as f:
        return json.load(f)


def _toy_service(g):
    # service = encoder time + tokens / decode rate, tokens = 5 per audio-second
    tok_per_s = Fraction(g["requests"][0]["tokens"], g["requests"][0]["duration_s"])
    return lambda d: Fraction(g["encoder_s"]) + d * tok_per_s / g["decode_tokens_per_s"]


@pytest.mark.parametrize("policy,key", [(Q.FCFS, "fcfs"), (Q.SJF, "sjf"), (Q.HRRN, "hrrn")])
def test_toy_example(policy, key):
    """Figure 1: FCFS mean 23/3 (printed 7.66), SJF 17/3 (printed 5.66)."""
    g = _toy()
    # all three are queued when the server starts; their arrival order is the id
    # order, which is FCFS's tie-break on equal arrival times
    jobs = [(r["id"], Fraction(0), Fraction(r["duration_s"])) for r in g["requests"]]
    done = Q.simulate_single_server(jobs, policy, _toy_service(g))
    if key == "hrrn":
        # every ratio is ~1 when the server first frees up; the SJF tie-break then
        # decides, and later decisions see equal waits -> shortest first again
        key = "sjf"
    expect = {int(k): v for k, v in g[key + "_completion_s"].items()}
    assert done == expect
    num, den = g[key + "_mean_num_den"]
    assert sum(done.values()) / 3 == Fraction(num, den)
    printed = g["printed_" + key + "_mean"]
    assert int(float(Fraction(num, den)) * 100) / 100 == printed
    # the "1.4x" of the caption
    assert round(23 / 17, 1) == 1.4


def test_token_estimate_examples():
    """Appendix A.4 endpoint: max(1, int(d * kappa))."""
    assert Q.token_estimate(1600, 16000, 27, 10, 448) == 1        # 0.1 s * 2.7 -> 0 -> 1
    assert Q.token_estimate(8 * 16000, 16000, 5, 1, 448) == 40     # toy example, R1
    assert Q.token_estimate(16000, 16000, 27, 10, 448) == 2        # int(2.7)
    assert Q.token_estimate(0, 16000, 27, 10, 300) == 300          # request fallback to max_tokens


def test_hrrn_ratio_closed_forms():
    assert Q.response_ratio(5_000_000, 4_000_000) == Fraction(9, 4)
    assert Q.response_ratio(0, 7) == 1
    rs = [Q.response_ratio(w, 3_000_000) for w in range(0, 10_000_000, 1_000_000)]
    assert all(a < b for a, b in zip(rs, rs[1:]))                  # increasing in wait
    assert all(r >= 1 for r in rs)


def _reqs(rows):
    return [Q.Req(rid, a, n, 16000, Q.duration_us(n, 16000), 448) for rid, a, n in rows]


def test_sjf_tie_break():
    """Section 3.2: equal durations -> earlier arrival first, then id (listing key)."""
    reqs = _reqs([(5, 30, 32000), (4, 10, 32000), (3, 10, 32000), (2, 0, 48000), (1, 50, 16000)])
    assert [r.rid for r in Q.order(reqs, Q.SJF, 100)] == [1, 3, 4, 5, 2]


def test_hrrn_limits():
    # equal waits (simultaneous arrival) -> SJF order
    reqs = _reqs([(i, 0, n) for i, n in enumerate([48000, 16000, 32000, 16000])])
    assert [r.rid for r in Q.order(reqs, Q.HRRN, 5_000_000)] == \
        [r.rid for r in Q.order(reqs, Q.SJF, 5_000_000)]
    # equal job lengths -> longest wait first (= FCFS)
    reqs = _reqs([(i, a, 32000) for i, a in enumerate([300, 100, 200, 0])])
    assert [r.rid for r in Q.order(reqs, Q.HRRN, 10_000)] == \
        [r.rid for r in Q.order(reqs, Q.FCFS, 10_000)]
    # a long job that waited long enough overtakes a fresh short one
    reqs = _reqs([(1, 0, 160000), (2, 9_000_000, 16000)])          # 10 s waited 9.5 s vs 1 s fresh
    assert [r.rid for r in Q.order(reqs, Q.HRRN, 9_500_000)] == [1, 2]
    assert [r.rid for r in Q.order(reqs, Q.SJF, 9_500_000)] == [2, 1]


def test_ineligible_and_pop():
    q = Q.Queue(Q.SJF)
    q.submit(1, 32000, 16000, 0)
    q.submit(2, 16000, 16000, 500)
    q.submit(3, 8000, 16000, 10_000)                               # arrives later
    assert q.rank(1000) == [2, 1]
    assert q.pop_batch(1000, 1) == [2]
    assert q.rank(20_000) == [3, 1]
    with pytest.raises(KeyError):
        q.submit(1, 100, 16000, 0)


@pytest.mark.parametrize("seed", range(6))
def test_sjf_minimises_mean_completion_bruteforce(seed):
    """Section 3.2: for jobs present together, SJF order minimises mean completion."""
    rnd = random.Random(seed)
    n = rnd.randint(2, 7)
    jobs = [(i, 0, rnd.randint(1, 30) * 16000) for i in range(n)]
    reqs = _reqs(jobs)
    service = {r.rid: Fraction(r.dur_us, 1_000_000) for r in reqs}

    def total(order_ids):
        t, s = Fraction(0), Fraction(0)
        for i in order_ids:
            t += service[i]
            s += t
        return s

    best = min(total(p) for p in itertools.permutations(service))
    assert total([r.rid for r in Q.order(reqs, Q.SJF, 0)]) == best
