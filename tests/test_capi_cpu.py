"""C ABI checks that need no GPU: exported symbols, argument validation, and
the host queue of a queue-only context against the queue oracle (bit-exact
pop sequences)."""
import ctypes
import os
import random
import re
import subprocess

import numpy as np
import pytest

from oracle import queue as Q

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

asr = pytest.importorskip("paper_2603_11273_amd.asr")


def _header_symbols():
    text = open(os.path.join(ROOT, "include", "asr.h")).read()
    return sorted(set(re.findall(r"\b(asr_[a-z_]+)\s*\(", text)) - {"asr_status"})


def test_library_exports_every_declared_symbol():
    declared = _header_symbols()
    assert len(declared) >= 20
    lib = ctypes.CDLL(asr.LIB_PATH)
    for name in declared:
        assert hasattr(lib, name), name
    assert sorted(asr.EXPORTED) == declared
    out = subprocess.run(["nm", "-D", "--defined-only", asr.LIB_PATH], capture_output=True,
                         text=True).stdout
    for name in declared:
        assert re.search(rf"\bT {name}$", out, re.M), name


def _tiny_cfg(**kw):
    from paper_2603_11273_amd import synth
    c = asr.model_cfg(synth.SHAPES["tiny"], max_slots=4, max_prefill=1, max_decode=4,
                      max_queue=kw.pop("max_queue", 64))
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def test_queue_only_context_refuses_gpu_calls():
    ctx = asr.Context(_tiny_cfg(), device=-1)
    with pytest.raises(asr.AsrError) as e:
        ctx.step(slots=[0], tokens=[1])
    assert e.value.status == asr.ASR_ENODEV
    with pytest.raises(asr.AsrError) as e:
        ctx.set_timing(True)
    assert e.value.status == asr.ASR_ENODEV
    assert ctx.workspace_size() > 0


@pytest.mark.parametrize("field,value", [("d_model", 100), ("n_head", 5), ("d_ffn", 100),
                                         ("max_decode", 9), ("max_queue", 0), ("dtype", 7)])
def test_create_rejects_bad_shapes(field, value):
    with pytest.raises(asr.AsrError) as e:
        asr.Context(_tiny_cfg(**{field: value}), device=-1)
    assert e.value.status == asr.ASR_EINVAL


def test_submit_validation():
    ctx = asr.Context(_tiny_cfg(max_queue=2), device=-1)
    pcm = np.zeros(1600, np.float32)
    ctx.submit(1, pcm)
    bad = [dict(rid=1, pcm=pcm),                                   # duplicate id
           dict(rid=2, pcm=pcm, sample_rate=8000),                 # no resampler
           dict(rid=3, pcm=np.zeros(480001, np.float32)),          # longer than 30 s
           dict(rid=4, pcm=pcm, max_tokens=449),
           dict(rid=5, pcm=None, n_samples=0)]                     # no samples, no duration
    for kw in bad:
        with pytest.raises(asr.AsrError) as e:
            ctx.submit(**kw)
        assert e.value.status == asr.ASR_EINVAL, kw
    ctx.submit(2, pcm)
    with pytest.raises(asr.AsrError) as e:
        ctx.submit(3, pcm)
    assert e.value.status == asr.ASR_EFULL
    with pytest.raises(asr.AsrError) as e:
        ctx.set_policy(3)
    assert e.value.status == asr.ASR_EINVAL


def _stream(seed, n):
    rnd = random.Random(seed)
    rows = []
    t = 0
    for i in range(n):
        t += rnd.choice([0, 0, 1, 5, 1000, 250_000])               # ties on purpose
        n_samples = rnd.choice([16000, 32000, rnd.randint(1, 480000)])
        rows.append((1000 + rnd.randint(0, 10**6) * 7 + i, t, n_samples))
    return rows


@pytest.mark.parametrize("policy", [Q.FCFS, Q.SJF, Q.HRRN])
@pytest.mark.parametrize("kappa", [(0, 0), (27, 10)])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_queue_matches_oracle_bit_exact(policy, kappa, seed):
    """Randomised submit / rank / pop_batch streams: identical id sequences."""
    rows = _stream(seed, 120)
    ctx = asr.Context(_tiny_cfg(max_queue=1000), device=-1)
    ctx.set_policy(policy, *kappa)
    ref = Q.Queue(policy, *kappa)
    rnd = random.Random(100 + seed)
    i = 0
    now = 0
    while i < len(rows) or ref.reqs:
        for _ in range(rnd.randint(0, 12)):
            if i < len(rows):
                rid, arr, n = rows[i]
                ctx.submit(rid, None if n % 5 == 0 else np.zeros(n, np.float32), n_samples=n,
                           arrival_us=arr, duration_us=(n * 10**6) // 16000 if n % 5 == 0 else 0)
                ref.submit(rid, n, 16000, arr)
                i += 1
        now += rnd.choice([0, 3, 700, 200_000])
        assert ctx.rank(now) == ref.rank(now)
        k = rnd.randint(0, 6)
        assert ctx.pop_batch(now, k) == ref.pop_batch(now, k)
        assert ctx.queue_len() == len(ref.reqs)
        if i >= len(rows) and not ctx.rank(now):
            now += 10**7


def test_policy_switch_reorders_waiting_requests():
    ctx = asr.Context(_tiny_cfg(), device=-1)
    for rid, n in [(1, 128000), (2, 64000), (3, 32000)]:
        ctx.submit(rid, np.zeros(n, np.float32), arrival_us=rid)
    assert ctx.rank(10) == [1, 2, 3]
    ctx.set_policy(asr.SJF)
    assert ctx.rank(10) == [3, 2, 1]
    ctx.set_policy(asr.HRRN)
    assert ctx.rank(10) == [3, 2, 1]
    # request 3 has not arrived at t=2; request 1 has waited 1 us, so its ratio
    # exceeds request 2's ratio of exactly 1
    assert ctx.rank(2) == [1, 2]
    assert Q.order([Q.Req(1, 1, 128000, 16000, 8_000_000, 448),
                    Q.Req(2, 2, 64000, 16000, 4_000_000, 448)], Q.HRRN, 2)[0].rid == 1
