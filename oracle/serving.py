"""Oracle for continuous batching with preemption and for the serving
simulation built on it (test infrastructure only).

What it follows:
* Section 4.1 (setup): requests arrive as a Poisson stream into an engine that
  batches running requests (continuous batching) and prefills new ones as
  slots free up; the evaluation metrics are end-to-end latency (arrival to
  completion) and time to first token, reported at P50 and P90 (the burst
  appendix adds time per output token and inter-token latency).
* The implementation appendix, preemption paragraph: under memory pressure
  SJF evicts the running request with the largest estimated length, HRRN the
  one with the lowest current response ratio.  FCFS evicts the most recently
  admitted request (the serving engines' recompute-on-preemption default,
  which the paper leaves in place for FCFS).
* Figure 1's toy: encoder cost 1 s per request, 10 output tokens per second
  of decoding, 5 output tokens per audio-second, one request at a time.

Readings where the paper is silent (the same ones the engine takes):
* memory is a pool of token positions: a running request holds a fixed
  cross-attention share plus one position per generated token, and every
  running request grows by one position per step;
* a preempted request drops its tokens, keeps its arrival time and keys, and
  is not re-admitted in the step that evicted it;
* admission stops at the first request the pool cannot hold; a request that
  could not fit the pool even alone is refused at submission (it could never
  finish);
* an admitted request is prefilled and produces its first token in the step
  that admits it (or, with overlapped prefill, in the next step);
* tokens per request: round-half-up(duration * rate), clamped to
  [1, min(448, max_tokens)];
* a token position that a recomputed request produces again is not emitted
  again: emission times (TTFT, inter-token gaps) count each position once.

Everything is integer (microseconds, token counts), so the engine and this
oracle can be compared event for event.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from fractions import Fraction

from . import queue as Q


def tokens_for(n_samples: int, sample_rate: int, max_tokens: int, tok_num: int,
               tok_den: int) -> int:
    """round-half-up(n / sr * tok_num / tok_den), clamped to [1, min(448, max_tokens)]."""
    den = sample_rate * tok_den
    t = (2 * n_samples * tok_num + den) // (2 * den)
    cap = min(448, max_tokens if max_tokens > 0 else 448)
    return max(1, min(t, cap))


@dataclass
class Running:
    req: Q.Req
    job: int
    slot: int
    total: int
    admit_seq: int
    generated: int = 0


def victim_key(r: Running, policy: int, now_us: int):
    """Key whose MAXIMUM over the running set is the request to evict."""
    sjf_worst = (r.job, r.req.arrival_us, r.req.rid)
    if policy == Q.FCFS:
        return (r.admit_seq, r.req.rid)
    if policy == Q.SJF:
        return sjf_worst
    # HRRN: the lowest response ratio is evicted first; ties by the SJF order reversed
    return (-Q.response_ratio(now_us - r.req.arrival_us, r.job), sjf_worst)


@dataclass
class StepResult:
    policy: int
    preempted: list
    admitted: list            # (id, slot)
    decoded: list             # ids, in decode-row order
    generated: dict           # id -> tokens held after the step
    finished: list


def dynamic_policy(waiting, now_us, depth_low, starve, kappa_num=0, kappa_den=0):
    """Dynamic switching (Section 5, future work: watch queue depth and
    starvation, switch among FCFS, SJF and HRRN) as this build reads it:
    FCFS while at most depth_low requests are eligible (all of them are about
    to be admitted, so the order costs nothing); otherwise HRRN when some
    eligible request's response ratio exceeds `starve` (a Fraction), else
    SJF."""
    elig = [r for r in waiting if r.arrival_us <= now_us]
    if len(elig) <= depth_low:
        return Q.FCFS
    top = max(Q.response_ratio(now_us - r.arrival_us, Q.job_length(r, kappa_num, kappa_den))
              for r in elig)
    return Q.HRRN if top > starve else Q.SJF


@dataclass
class Engine:
    policy: int
    n_slots: int
    max_admit: int
    kv_capacity: int          # <= 0: unlimited
    cross_tokens: int
    tok_num: int = 27
    tok_den: int = 10
    kappa_num: int = 0
    kappa_den: int = 0
    dynamic: bool = False
    depth_low: int = 0
    starve: Fraction = Fraction(0)
    defer_first: bool = False     # admitted requests start decoding in the next step
    queue: Q.Queue = None
    known: dict = field(default_factory=dict)
    running: list = field(default_factory=list)
    seq: int = 0
    steps_by_policy: list = field(default_factory=lambda: [0, 0, 0])

    def __post_init__(self):
        self.queue = Q.Queue(self.policy, self.kappa_num, self.kappa_den)

    def submit(self, rid, n_samples, sample_rate, arrival_us, duration_us=0, max_tokens=0):
        mt = max_tokens if max_tokens > 0 else Q.MAX_TOKENS
        need = self.cross_tokens + tokens_for(n_samples, sample_rate, mt, self.tok_num, self.tok_den)
        if self.kv_capacity > 0 and need > self.kv_capacity:
            raise ValueError(f"request {rid} can never fit the KV pool")
        self.queue.submit(rid, n_samples, sample_rate, arrival_us, duration_us, max_tokens)
        self.known[rid] = self.queue.reqs[rid]

    def total_of(self, rid):
        r = self.known[rid]
        return tokens_for(r.n_samples, r.sample_rate, r.max_tokens, self.tok_num, self.tok_den)

    def step(self, now_us: int) -> StepResult:
        if self.dynamic:
            self.policy = dynamic_policy(self.queue.reqs.values(), now_us, self.depth_low,
                                         self.starve, self.kappa_num, self.kappa_den)
            self.queue.policy = self.policy
        self.steps_by_policy[self.policy] += 1
        limited = self.kv_capacity > 0
        need = sum(self.cross_tokens + r.generated + 1 for r in self.running)
        preempted, requeue = [], []
        while limited and need > self.kv_capacity and self.running:
            v = max(self.running, key=lambda r: victim_key(r, self.policy, now_us))
            self.running.remove(v)
            need -= self.cross_tokens + v.generated + 1
            preempted.append(v.req.rid)
            requeue.append(v.req)
        used = {r.slot for r in self.running}
        free = [s for s in range(self.n_slots) if s not in used]
        admitted = []
        while len(admitted) < self.max_admit and free:
            if limited and need + self.cross_tokens + 1 > self.kv_capacity:
                break
            ids = self.queue.pop_batch(now_us, 1)
            if not ids:
                break
            req = self.known[ids[0]]
            job = Q.job_length(req, self.kappa_num, self.kappa_den)
            slot = free.pop(0)
            self.running.append(Running(req, job, slot, self.total_of(req.rid), self.seq))
            self.seq += 1
            need += self.cross_tokens + 1
            admitted.append((req.rid, slot))
        for req in requeue:
            self.queue.reqs[req.rid] = req
        new_ids = {rid for rid, _ in admitted} if self.defer_first else set()
        rows = [r for r in self.running if r.req.rid not in new_ids]
        decoded = [r.req.rid for r in rows]
        generated, finished = {}, []
        for r in rows:
            r.generated += 1
            generated[r.req.rid] = r.generated
            if r.generated >= r.total:
                self.running.remove(r)
                finished.append(r.req.rid)
        return StepResult(self.policy, preempted, admitted, decoded, generated, finished)


@dataclass
class Cost:
    """Virtual duration of one engine step, in microseconds."""
    prefill_us: int       # per admitted request
    step_us: int          # per step that decodes at least one row
    row_us: int           # per decode row

    def of(self, n_admitted: int, n_decoded: int) -> int:
        return (self.prefill_us * n_admitted
                + ((self.step_us + self.row_us * n_decoded) if n_decoded else 0))


def simulate(eng: Engine, cost: Cost, t0_us: int = 0):
    """Run the engine on a virtual clock until every submitted request
    finishes.  Returns ({id: {arrival_us, first_us, finish_us, n_tokens,
    n_preempt, token_us}}, end time)."""
    info = {rid: {"arrival_us": r.arrival_us, "n_preempt": 0, "token_us": []}
            for rid, r in eng.known.items()}
    pending = set(info)
    t = t0_us
    while pending:
        if not eng.running and not any(r.arrival_us <= t for r in eng.queue.reqs.values()):
            t = min(r.arrival_us for r in eng.queue.reqs.values())
            continue
        res = eng.step(t)
        t += cost.of(len(res.admitted), len(res.decoded))
        for rid in res.preempted:
            info[rid]["n_preempt"] += 1
        for rid in res.decoded:
            em = info[rid]["token_us"]
            while len(em) < res.generated[rid]:
                em.append(t)
        for rid in res.finished:
            info[rid]["finish_us"] = t
            pending.discard(rid)
    for d in info.values():
        d["first_us"] = d["token_us"][0]
        d["n_tokens"] = len(d["token_us"])
    return info, t


def percentile_nearest_rank(values, p):
    """Nearest-rank percentile (the smallest value with at least p% of the
    values at or below it) -- exact on integers."""
    v = sorted(values)
    k = max(1, -(-len(v) * p // 100))      # ceil(n p / 100)
    return v[k - 1]


def metrics(info: dict, t_end: int, t0_us: int = 0):
    """Paper metrics over a finished run: P50 / P90 of TTFT and E2EL, mean
    TPOT, P50 / P90 inter-token latency, request and token throughput."""
    ttft = [d["first_us"] - d["arrival_us"] for d in info.values()]
    e2el = [d["finish_us"] - d["arrival_us"] for d in info.values()]
    tpot = [(d["finish_us"] - d["first_us"]) / (d["n_tokens"] - 1)
            for d in info.values() if d["n_tokens"] > 1]
    itl = [b - a for d in info.values() for a, b in zip(d["token_us"], d["token_us"][1:])]
    span = t_end - min(d["arrival_us"] for d in info.values())
    n_tok = sum(d["n_tokens"] for d in info.values())
    return {
        "ttft_p50_us": percentile_nearest_rank(ttft, 50),
        "ttft_p90_us": percentile_nearest_rank(ttft, 90),
        "e2el_p50_us": percentile_nearest_rank(e2el, 50),
        "e2el_p90_us": percentile_nearest_rank(e2el, 90),
        "tpot_mean_us": sum(tpot) / len(tpot) if tpot else 0.0,
        "itl_p50_us": percentile_nearest_rank(itl, 50) if itl else 0,
        "itl_p90_us": percentile_nearest_rank(itl, 90) if itl else 0,
        "req_per_s": len(info) / (span * 1e-6) if span else 0.0,
        "tok_per_s": n_tok / (span * 1e-6) if span else 0.0,
        "preemptions": sum(d["n_preempt"] for d in info.values()),
    }
