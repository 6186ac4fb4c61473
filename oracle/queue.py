"""Oracle for the duration-aware waiting queue (test infrastructure only).

Follows the paper's methodology:
* Eq. 1 (Section 3.1): estimated output tokens n = d * kappa;
* Section 3.2: SJF (shortest first, earlier arrival wins ties) and HRRN
  (response ratio (wait + job time) / job time, highest first);
* Appendix A.4: the endpoint estimate max(1, int(duration * kappa)), the
  request-level fallback to max_tokens, the SJF key
  (estimate, arrival, id) and the HRRN ratio computed at every pop.

Integer keys only: durations in microseconds, kappa as a rational
kappa_num / kappa_den, ratios compared as exact fractions.  Readings where
the paper is silent: ties in HRRN fall back to the SJF key; only requests
whose arrival time is <= now are eligible; one `now` serves a whole
pop_batch call.
"""
from __future__ import annotations

from dataclasses import dataclass
from fractions import Fraction

FCFS, SJF, HRRN = 0, 1, 2
MAX_TOKENS = 448


@dataclass
class Req:
    rid: int
    arrival_us: int
    n_samples: int
    sample_rate: int
    dur_us: int
    max_tokens: int


def duration_us(n_samples: int, sample_rate: int) -> int:
    """Duration of the audio, len/sr (Appendix A.4 endpoint), in integer microseconds."""
    return (n_samples * 1_000_000) // sample_rate


def token_estimate(n_samples: int, sample_rate: int, kappa_num: int, kappa_den: int,
                   max_tokens: int) -> int:
    """Eq. 1 with the endpoint's clamp max(1, int(d * kappa)); falls back to
    max_tokens when the request carries no audio (Appendix A.4 request class)."""
    if n_samples <= 0:
        return max_tokens
    return max(1, (n_samples * kappa_num) // (sample_rate * kappa_den))


def job_length(r: Req, kappa_num: int, kappa_den: int) -> int:
    """Job-length proxy: the duration itself (Section 3.2, HRRN paragraph:
    only the relative order matters) or, with kappa given, the Eq. 1 estimate."""
    if kappa_den == 0:
        return r.dur_us
    return token_estimate(r.n_samples, r.sample_rate, kappa_num, kappa_den, r.max_tokens)


def response_ratio(wait_us: int, job: int) -> Fraction:
    """HRRN response ratio (waiting time + estimated job time) / estimated job
    time (Section 3.2), as an exact fraction."""
    return Fraction(wait_us + job, job)


def order(reqs, policy: int, now_us: int, kappa_num: int = 0, kappa_den: int = 0):
    """Eligible requests (arrival <= now) in service order under `policy`."""
    elig = [r for r in reqs if r.arrival_us <= now_us]
    if policy == FCFS:
        return sorted(elig, key=lambda r: (r.arrival_us, r.rid))
    if policy == SJF:
        return sorted(elig, key=lambda r: (job_length(r, kappa_num, kappa_den), r.arrival_us, r.rid))
    if policy == HRRN:
        def key(r):
            e = job_length(r, kappa_num, kappa_den)
            return (-response_ratio(now_us - r.arrival_us, e), e, r.arrival_us, r.rid)
        return sorted(elig, key=key)
    raise ValueError(policy)


class Queue:
    """Waiting queue with submit / rank / pop_batch, as the C ABI exposes it."""

    def __init__(self, policy: int = FCFS, kappa_num: int = 0, kappa_den: int = 0):
        self.policy, self.kn, self.kd = policy, kappa_num, kappa_den
        self.reqs: dict[int, Req] = {}

    def submit(self, rid, n_samples, sample_rate, arrival_us, duration_us_in=0, max_tokens=0):
        if rid in self.reqs:
            raise KeyError(rid)
        d = duration_us_in if duration_us_in > 0 else duration_us(n_samples, sample_rate)
        mt = max_tokens if max_tokens > 0 else MAX_TOKENS
        self.reqs[rid] = Req(rid, arrival_us, n_samples, sample_rate, d, mt)

    def rank(self, now_us):
        return [r.rid for r in order(self.reqs.values(), self.policy, now_us, self.kn, self.kd)]

    def pop_batch(self, now_us, k):
        ids = self.rank(now_us)[:k]
        for i in ids:
            del self.reqs[i]
        return ids


def simulate_single_server(jobs, policy, service_s, kappa_num=0, kappa_den=0):
    """Non-preemptive single server, as in the toy example of Figure 1.

    jobs: list of (rid, arrival_s as Fraction, duration_s as Fraction).
    service_s(duration) -> Fraction.  Returns {rid: completion time}.
    Time is kept as exact fractions; the queue's integer keys use microseconds.
    """
    pending = {rid: (Fraction(a), Fraction(d)) for rid, a, d in jobs}
    t = Fraction(0)
    done = {}
    while pending:
        arrived = [rid for rid, (a, _) in pending.items() if a <= t]
        if not arrived:
            t = min(a for a, _ in pending.values())
            continue
        reqs = []
        for rid in arrived:
            a, d = pending[rid]
            n = int(d * 16000)
            reqs.append(Req(rid, int(a * 1_000_000), n, 16000, duration_us(n, 16000), MAX_TOKENS))
        nxt = order(reqs, policy, int(t * 1_000_000), kappa_num, kappa_den)[0].rid
        a, d = pending.pop(nxt)
        t = t + service_s(d)
        done[nxt] = t
    return done
