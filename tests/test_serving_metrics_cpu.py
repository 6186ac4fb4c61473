"""The paper's serving metrics (Section 4.1: P50 / P90 TTFT and E2EL; the
burst appendix: TPOT and inter-token latency; throughput).

The oracle's metrics() is pinned to a schedule worked out by hand and to the
Figure 1 toy example; the library-side implementation the benchmark uses is
then checked against it on native serving simulations."""
import json
import os

import pytest

from oracle import queue as Q
from oracle import serving as S

from paper_2603_11273_amd import serving_metrics as SM
from paper_2603_11273_amd import synth

asr = pytest.importorskip("paper_2603_11273_amd.asr")

SR = 16000
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "toy_example.json")


def _info(reqs):
    return {rid: {"arrival_us": a, "first_us": t[0], "finish_us": t[-1], "n_tokens": len(t),
                  "token_us": list(t), "n_preempt": p}
            for rid, (a, t, p) in reqs.items()}


HAND = {
    # id: (arrival, token emission times, preemptions)
    1: (0, [100, 150, 250], 1),
    2: (50, [900], 0),
    3: (100, [200, 260, 320, 380], 0),
}


def test_metrics_hand_schedule():
    """Three requests, run ending at t = 1000 us.

    TTFT: 100 - 0 = 100, 900 - 50 = 850, 200 - 100 = 100 -> sorted
      [100, 100, 850]; nearest rank P50 = 2nd (ceil 1.5) = 100, P90 = 3rd = 850.
    E2EL: 250, 850, 280 -> sorted [250, 280, 850]: P50 = 280, P90 = 850.
    TPOT: request 1 (250 - 100) / (3 - 1) = 75, request 3 (380 - 200) / 3 =
      60, request 2 has one token and no TPOT -> mean 67.5 (dividing by the
      token count instead would give 47.5).
    ITL: gaps inside a request only: 50, 100 (request 1), 60, 60, 60
      (request 3) -> sorted [50, 60, 60, 60, 100]; P50 = 3rd = 60, P90 =
      5th (ceil 4.5) = 100 (gaps across requests, 250 -> 900 and 900 -> 200,
      would make the P90 650).
    Throughput over 0 .. 1000 us: 3 requests -> 3000 /s, 8 tokens -> 8000 /s."""
    m = S.metrics(_info(HAND), t_end=1000)
    assert m["ttft_p50_us"] == 100 and m["ttft_p90_us"] == 850
    assert m["e2el_p50_us"] == 280 and m["e2el_p90_us"] == 850
    assert m["tpot_mean_us"] == 67.5
    assert m["itl_p50_us"] == 60 and m["itl_p90_us"] == 100
    assert m["req_per_s"] == pytest.approx(3000.0) and m["tok_per_s"] == pytest.approx(8000.0)
    assert m["preemptions"] == 1


@pytest.mark.parametrize("policy,first_s,finish_s", [
    # Figure 1 under this engine's step model: 1 s prefill, then 0.1 s per
    # decode step, the first token in the admitting step.  FCFS: R1's first
    # token at 1.1 s, R2's at 5 + 1.1, R3's at 8 + 1.1; SJF serves R3, R2, R1.
    (Q.FCFS, {1: 1.1, 2: 6.1, 3: 9.1}, {1: 5, 2: 8, 3: 10}),
    (Q.SJF, {3: 1.1, 2: 3.1, 1: 6.1}, {3: 2, 2: 5, 1: 10}),
])
def test_metrics_toy_example(policy, first_s, finish_s):
    """The toy example (Figure 1): completion times 5 / 8 / 10 s (FCFS) and
    2 / 5 / 10 s (SJF).  E2EL percentiles are the middle and last
    completion; every inter-token gap is the 0.1-s decode step, so TPOT and
    ITL are 100000 us exactly; 70 tokens and 3 requests in 10 s."""
    g = json.load(open(GOLDEN))
    eng = S.Engine(policy, n_slots=1, max_admit=1, kv_capacity=0, cross_tokens=0, tok_num=5,
                   tok_den=1)
    for r in g["requests"]:
        eng.submit(r["id"], r["duration_s"] * SR, SR, arrival_us=0)
    info, t_end = S.simulate(eng, S.Cost(prefill_us=10**6, step_us=10**5, row_us=0))
    for rid in first_s:
        assert info[rid]["first_us"] == round(first_s[rid] * 10**6)
        assert info[rid]["finish_us"] == finish_s[rid] * 10**6
    m = S.metrics(info, t_end)
    fin = sorted(finish_s.values())
    fst = sorted(first_s.values())
    assert m["e2el_p50_us"] == fin[1] * 10**6 and m["e2el_p90_us"] == fin[2] * 10**6
    assert m["ttft_p50_us"] == round(fst[1] * 10**6) and m["ttft_p90_us"] == round(fst[2] * 10**6)
    assert m["tpot_mean_us"] == pytest.approx(1e5, abs=1e-6)
    assert m["itl_p50_us"] == m["itl_p90_us"] == 10**5
    assert m["req_per_s"] == pytest.approx(0.3) and m["tok_per_s"] == pytest.approx(7.0)


def test_library_metrics_match_oracle_on_hand_schedule():
    info = _info(HAND)
    ids = sorted(info)
    m = SM.latency_metrics([info[i]["arrival_us"] for i in ids], [info[i]["first_us"] for i in ids],
                           [info[i]["finish_us"] for i in ids], [info[i]["n_tokens"] for i in ids],
                           [t for i in ids for t in info[i]["token_us"]], 1000)
    ref = S.metrics(info, 1000)
    for k in m:
        assert m[k] == pytest.approx(ref[k]), k


@pytest.mark.parametrize("policy,burst,kv", [(asr.FCFS, True, 0), (asr.SJF, False, 0),
                                             (asr.HRRN, False, 0), (asr.SJF, True, 1500 + 900)])
def test_library_metrics_match_oracle_on_native_simulation(policy, burst, kv):
    """A native virtual-clock run (queue-only context): the benchmark's
    metric code and the oracle's metrics() give the same numbers from the
    same per-token emission times (one case under pool pressure, with
    preemptions and recomputation)."""
    n = 300
    cfg = asr.model_cfg(synth.SHAPES["large-v3"], max_slots=32, max_prefill=8, max_decode=32,
                        max_queue=n + 1)
    q = asr.Context(cfg, device=-1)
    q.set_policy(policy)
    q.serve_config(kv_capacity=kv, cross_tokens=150 if kv else 1500, max_admit=8)
    seed = 77
    ns = synth.n_samples_of(synth.durations_lognormal(seed, n))
    arr = [0] * n if burst else synth.poisson_arrivals_us(seed, n, 40.0).tolist()
    for i in range(n):
        q.submit(i, None, n_samples=int(ns[i]), arrival_us=int(arr[i]))
    info, t_end = q.serve_simulate(list(range(n)), prefill_us=3000, step_us=3000, row_us=60)
    if kv:
        assert sum(d["n_preempt"] for d in info.values()) > 0
    for i in range(n):
        info[i]["arrival_us"] = int(arr[i])
    ref = S.metrics(info, t_end)
    m = SM.latency_metrics(arr, [info[i]["first_us"] for i in range(n)],
                           [info[i]["finish_us"] for i in range(n)],
                           [info[i]["n_tokens"] for i in range(n)],
                           [t for i in range(n) for t in info[i]["token_us"]], t_end)
    for k in m:
        assert m[k] == pytest.approx(ref[k], rel=1e-12), k
