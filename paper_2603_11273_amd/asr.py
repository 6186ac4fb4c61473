"""Thin ctypes binding of the C ABI in include/asr.h (argument marshalling only).

Every computation runs in the HIP library; this module only converts Python
values and torch/numpy buffers to pointers.  Importing it raises if the
library has not been built (python -m paper_2603_11273_amd.build).
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libasr_mi355x.so")

ASR_OK, ASR_EINVAL, ASR_ENOMEM, ASR_EFULL, ASR_ENOTFOUND, ASR_ESTATE, ASR_ENODEV, ASR_EDEVICE = range(8)
STATUS_NAMES = ["OK", "EINVAL", "ENOMEM", "EFULL", "ENOTFOUND", "ESTATE", "ENODEV", "EDEVICE"]
FCFS, SJF, HRRN = 0, 1, 2
F32, BF16 = 0, 1
(K_MEL, K_GEMM, K_ATTN, K_LN, K_DGEMM, K_DATTN, K_VOCAB, K_OTHER, K_PREFILL, K_DECODE,
 K_ENCODE, K_XKV) = range(12)
KERNEL_CLASSES = ["mel", "gemm", "attn", "ln", "dgemm", "dattn", "vocab", "other", "prefill",
                  "decode", "encode", "xkv"]
TIME_ALL = (1 << len(KERNEL_CLASSES)) - 1

EXPORTED = [
    "asr_create", "asr_destroy", "asr_last_error", "asr_workspace_size", "asr_bind",
    "asr_n_params", "asr_param_numel", "asr_load_weights", "asr_set_policy", "asr_submit",
    "asr_rank", "asr_pop_batch", "asr_queue_len", "asr_step", "asr_release_slot",
    "asr_slot_info", "asr_set_encoder_streams", "asr_set_decode_graphs", "asr_set_timing",
    "asr_get_timing",
    "asr_reset_timing",
    "asr_debug_logmel", "asr_debug_encode", "asr_debug_attention", "asr_debug_set_encoder_out",
    "asr_debug_get_kv",
    "asr_debug_set_self_kv", "asr_logmel_noalloc", "asr_serve_config", "asr_serve_step",
    "asr_serve_plan",
    "asr_serve_tokens", "asr_serve_simulate", "asr_serve_stats",
]


class ModelCfg(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "n_mels", "d_model", "n_enc", "n_dec", "n_head", "d_ffn", "vocab", "dtype",
        "max_slots", "max_prefill", "max_decode", "max_queue")]


class StepIn(C.Structure):
    _fields_ = [("n_prefill", C.c_int32), ("prefill_ids", C.POINTER(C.c_int64)),
                ("n_decode", C.c_int32), ("slots", C.POINTER(C.c_int32)),
                ("tokens", C.POINTER(C.c_int32)), ("logits", C.POINTER(C.c_float))]


class StepOut(C.Structure):
    _fields_ = [("slot_of", C.POINTER(C.c_int32)), ("argmax", C.POINTER(C.c_int32)),
                ("done", C.POINTER(C.c_int32))]


class ServeCfg(C.Structure):
    _fields_ = [("kv_capacity", C.c_int64), ("cross_tokens", C.c_int32),
                ("max_admit", C.c_int32), ("tok_num", C.c_int32), ("tok_den", C.c_int32),
                ("start_token", C.c_int32), ("dynamic", C.c_int32), ("depth_low", C.c_int32),
                ("starve_num", C.c_int64), ("starve_den", C.c_int64), ("overlap", C.c_int32)]


class ServeOut(C.Structure):
    _fields_ = [("cap", C.c_int32), ("policy", C.c_int32),
                ("preempted", C.POINTER(C.c_int64)), ("n_preempted", C.c_int32),
                ("admitted", C.POINTER(C.c_int64)), ("admitted_slot", C.POINTER(C.c_int32)),
                ("n_admitted", C.c_int32),
                ("decoded", C.POINTER(C.c_int64)), ("token", C.POINTER(C.c_int32)),
                ("n_decoded", C.c_int32),
                ("finished", C.POINTER(C.c_int64)), ("n_finished", C.c_int32)]


class SimCost(C.Structure):
    _fields_ = [("prefill_us", C.c_int64), ("step_us", C.c_int64), ("row_us", C.c_int64)]


class AsrError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES[status] if 0 <= status < 8 else status}: {msg}")
        self.status = status


def _load():
    # torch bundles its own HIP runtime (soname libamdhip64.so.7).  Loading it
    # first makes the library bind to that same runtime by soname, so device
    # pointers and streams from torch are valid here; loading the library
    # first would pull a second HIP runtime into the process.
    try:
        import torch  # noqa: F401
    except Exception:  # pragma: no cover - queue-only use without torch
        pass
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2603_11273_amd.build`")
    lib = C.CDLL(LIB_PATH)
    P, i32, i64, f, vp = C.POINTER, C.c_int32, C.c_int64, C.c_float, C.c_void_p
    sig = {
        "asr_create": [P(ModelCfg), i32, P(vp)],
        "asr_destroy": [vp],
        "asr_last_error": [],
        "asr_workspace_size": [vp, P(C.c_size_t)],
        "asr_bind": [vp, vp, C.c_size_t, vp],
        "asr_n_params": [vp, P(i32)],
        "asr_param_numel": [vp, i32, P(i64)],
        "asr_load_weights": [vp, P(vp), i32, i32],
        "asr_set_policy": [vp, i32, i32, i32],
        "asr_submit": [vp, i64, vp, i64, i32, i64, i64, i32, i32],
        "asr_rank": [vp, i64, P(i64), i32, P(i32)],
        "asr_pop_batch": [vp, i64, i32, P(i64), P(i32)],
        "asr_queue_len": [vp, P(i32)],
        "asr_step": [vp, P(StepIn), P(StepOut)],
        "asr_release_slot": [vp, i32],
        "asr_slot_info": [vp, i32, P(i32), P(i64), P(i32), P(i32)],
        "asr_set_encoder_streams": [vp, i32],
        "asr_set_decode_graphs": [vp, i32],
        "asr_set_timing": [vp, i32],
        "asr_get_timing": [vp, i32, P(C.c_double), P(i64), P(C.c_double), P(C.c_double)],
        "asr_reset_timing": [vp],
        "asr_debug_logmel": [vp, P(vp), P(i64), i32, i32, P(f)],
        "asr_debug_encode": [vp, P(vp), P(i64), i32, i32, P(f)],
        "asr_debug_attention": [vp, P(f), P(f), P(f), i32, P(f)],
        "asr_debug_set_encoder_out": [vp, P(i32), P(i64), P(i32), i32, vp, i32],
        "asr_debug_get_kv": [vp, i32, i32, P(f)],
        "asr_debug_set_self_kv": [vp, i32, vp, i32, i32],
        "asr_logmel_noalloc": [P(vp), P(i64), i32, i32, vp, vp],
        "asr_serve_config": [vp, P(ServeCfg)],
        "asr_serve_step": [vp, i64, P(ServeOut)],
        "asr_serve_plan": [vp, i64, P(ServeOut)],
        "asr_serve_tokens": [vp, i64, P(i32), i32, P(i32)],
        "asr_serve_stats": [vp, P(i64)],
        "asr_serve_simulate": [vp, P(SimCost), i64, i32, P(i64), P(i64), P(i64), P(i32),
                               P(i32), P(i64), i64, P(i64)],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = C.c_char_p if name == "asr_last_error" else C.c_int
    return lib


lib = _load()


def _check(status):
    if status != ASR_OK:
        raise AsrError(status, lib.asr_last_error().decode())


def _ptr(a):
    """Address of a torch tensor or numpy array (contiguous)."""
    if a is None:
        return None
    if hasattr(a, "data_ptr"):
        assert a.is_contiguous()
        return a.data_ptr()
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


def _i64(a):
    a = np.ascontiguousarray(a, dtype=np.int64)
    return a, a.ctypes.data_as(C.POINTER(C.c_int64))


def _i32(a):
    a = np.ascontiguousarray(a, dtype=np.int32)
    return a, a.ctypes.data_as(C.POINTER(C.c_int32))


def logmel_noalloc(clips, n_mels, out, stream=None):
    """asr_logmel_noalloc: normalised log-mel features of device clips (torch
    tensors, float32) into the device tensor out [n][3000][n_mels], on
    `stream` (torch.cuda.Stream; default: torch's current stream)."""
    import torch
    n = len(clips)
    for x in clips:
        if not (x.is_cuda and x.dtype == torch.float32):
            raise TypeError("clips must be float32 device tensors")
    if not (out.is_cuda and out.dtype == torch.float32 and tuple(out.shape) == (n, 3000, n_mels)):
        raise TypeError(f"out must be a float32 device tensor of shape ({n}, 3000, {n_mels})")
    ptrs = (C.c_void_p * n)(*[_ptr(x) for x in clips])
    ns = np.array([x.numel() for x in clips], np.int64)
    st = (stream or torch.cuda.current_stream()).cuda_stream
    _check(lib.asr_logmel_noalloc(ptrs, ns.ctypes.data_as(C.POINTER(C.c_int64)), n, n_mels,
                                  _ptr(out), st))


def model_cfg(shape, max_slots=8, max_prefill=1, max_decode=8, max_queue=4096) -> ModelCfg:
    """asr_model_cfg from a synth.ModelShape (or anything with the same fields)."""
    return ModelCfg(shape.n_mels, shape.d_model, shape.n_enc, shape.n_dec, shape.n_head,
                    shape.d_ffn, shape.vocab, BF16 if shape.dtype == "bf16" else F32,
                    max_slots, max_prefill, max_decode, max_queue)


class Context:
    """One asr_ctx.  device=-1 gives a queue-only context (no GPU calls)."""

    def __init__(self, cfg: ModelCfg, device: int = 0):
        self.cfg = cfg
        self.device = device
        h = C.c_void_p()
        _check(lib.asr_create(C.byref(cfg), device, C.byref(h)))
        self.h = h
        self._block = None
        self._keep = []
        self._serve_cap = max(cfg.max_slots, 1)

    def close(self):
        if self.h:
            lib.asr_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- memory ---------------------------------------------------------------
    def workspace_size(self) -> int:
        n = C.c_size_t()
        _check(lib.asr_workspace_size(self.h, C.byref(n)))
        return n.value

    def bind(self, block=None, stream=None):
        """Binds a device block (torch uint8 tensor; allocated here when None)."""
        import torch
        if block is None:
            block = torch.empty(self.workspace_size(), dtype=torch.uint8,
                                device=f"cuda:{self.device}")
        if stream is None:
            stream = torch.cuda.current_stream(self.device).cuda_stream
        _check(lib.asr_bind(self.h, C.c_void_p(block.data_ptr()), block.numel(),
                            C.c_void_p(stream)))
        self._block = block
        return block

    def n_params(self) -> int:
        n = C.c_int32()
        _check(lib.asr_n_params(self.h, C.byref(n)))
        return n.value

    def param_numel(self, i) -> int:
        n = C.c_int64()
        _check(lib.asr_param_numel(self.h, i, C.byref(n)))
        return n.value

    def load_weights(self, tensors, on_device: bool):
        arr = (C.c_void_p * len(tensors))(*[_ptr(t) for t in tensors])
        _check(lib.asr_load_weights(self.h, arr, len(tensors), int(on_device)))

    # -- queue ----------------------------------------------------------------
    def set_policy(self, policy, kappa_num=0, kappa_den=0):
        _check(lib.asr_set_policy(self.h, policy, kappa_num, kappa_den))

    def submit(self, rid, pcm, n_samples=None, sample_rate=16000, duration_us=0, arrival_us=0,
               max_tokens=0, on_device=False):
        if pcm is not None and n_samples is None:
            n_samples = pcm.numel() if hasattr(pcm, "numel") else len(pcm)
        if pcm is not None and not on_device:
            pcm = np.ascontiguousarray(pcm, dtype=np.float32)
        _check(lib.asr_submit(self.h, rid, _ptr(pcm) if pcm is not None else None, n_samples,
                              sample_rate, duration_us, arrival_us, max_tokens, int(on_device)))

    def rank(self, now_us, cap=1 << 20):
        n = C.c_int32()
        out = np.zeros(max(cap, 1), np.int64)
        _check(lib.asr_rank(self.h, now_us, out.ctypes.data_as(C.POINTER(C.c_int64)), cap,
                            C.byref(n)))
        return out[:n.value].tolist()

    def pop_batch(self, now_us, max_n):
        n = C.c_int32()
        out = np.zeros(max(max_n, 1), np.int64)
        _check(lib.asr_pop_batch(self.h, now_us, max_n,
                                 out.ctypes.data_as(C.POINTER(C.c_int64)), C.byref(n)))
        return out[:n.value].tolist()

    def queue_len(self):
        n = C.c_int32()
        _check(lib.asr_queue_len(self.h, C.byref(n)))
        return n.value

    # -- step -----------------------------------------------------------------
    def step(self, prefill_ids=(), slots=(), tokens=(), want_logits=False):
        """Returns dict(slot_of, argmax, done, logits)."""
        pids, p_pids = _i64(list(prefill_ids) or [0])
        sl, p_sl = _i32(list(slots) or [0])
        tk, p_tk = _i32(list(tokens) or [0])
        P, D = len(prefill_ids), len(slots)
        slot_of, p_so = _i32(np.zeros(max(P, 1)))
        am, p_am = _i32(np.zeros(max(D, 1)))
        done, p_dn = _i32(np.zeros(max(D, 1)))
        logits = None
        p_lg = None
        if want_logits and D > 0:
            logits = np.zeros((D, self.cfg.vocab), np.float32)
            p_lg = logits.ctypes.data_as(C.POINTER(C.c_float))
        sin = StepIn(P, p_pids, D, p_sl, p_tk, p_lg)
        sout = StepOut(p_so, p_am, p_dn)
        _check(lib.asr_step(self.h, C.byref(sin), C.byref(sout)))
        return {"slot_of": slot_of[:P].copy(), "argmax": am[:D].copy(),
                "done": done[:D].astype(bool), "logits": logits}

    def release_slot(self, slot):
        _check(lib.asr_release_slot(self.h, slot))

    # -- continuous batching ----------------------------------------------------
    def serve_config(self, kv_capacity=0, cross_tokens=1500, max_admit=1, tok_num=27,
                     tok_den=10, start_token=0, dynamic=False, depth_low=0, starve=(0, 1),
                     overlap=False):
        """starve = (num, den): the response-ratio threshold of the dynamic rule;
        overlap: prefill on a second stream beside the running rows' decode."""
        cfg = ServeCfg(kv_capacity, cross_tokens, max_admit, tok_num, tok_den, start_token,
                       int(dynamic), depth_low, starve[0], starve[1], int(overlap))  # >1: CUs kept free
        _check(lib.asr_serve_config(self.h, C.byref(cfg)))
        self._serve_cap = max(self.cfg.max_slots, 1)

    def _serve(self, fn, now_us):
        cap = self._serve_cap
        bufs = {k: np.zeros(cap, np.int64) for k in ("preempted", "admitted", "decoded", "finished")}
        slot = np.zeros(cap, np.int32)
        tok = np.zeros(cap, np.int32)
        p64 = lambda a: a.ctypes.data_as(C.POINTER(C.c_int64))  # noqa: E731
        p32 = lambda a: a.ctypes.data_as(C.POINTER(C.c_int32))  # noqa: E731
        out = ServeOut(cap, 0, p64(bufs["preempted"]), 0, p64(bufs["admitted"]), p32(slot), 0,
                       p64(bufs["decoded"]), p32(tok), 0, p64(bufs["finished"]), 0)
        _check(fn(self.h, now_us, C.byref(out)))
        return {"policy": out.policy,
                "preempted": bufs["preempted"][:out.n_preempted].tolist(),
                "admitted": bufs["admitted"][:out.n_admitted].tolist(),
                "admitted_slot": slot[:out.n_admitted].tolist(),
                "decoded": bufs["decoded"][:out.n_decoded].tolist(),
                "token": tok[:out.n_decoded].tolist(),
                "finished": bufs["finished"][:out.n_finished].tolist()}

    def serve_step(self, now_us):
        """One continuous-batching step on the GPU (see asr_serve_step)."""
        return self._serve(lib.asr_serve_step, now_us)

    def serve_plan(self, now_us):
        """The same schedule without the model (queue-only contexts)."""
        return self._serve(lib.asr_serve_plan, now_us)

    def serve_simulate(self, ids, prefill_us, step_us, row_us, t0_us=0, want_token_times=True,
                       token_cap=None):
        """Virtual-clock serving run (asr_serve_simulate).  Returns
        ({id: {first_us, finish_us, n_tokens, n_preempt, token_us}}, t_end_us)."""
        n = len(ids)
        ids_a = np.asarray(ids, np.int64)
        first = np.zeros(max(n, 1), np.int64)
        fin = np.zeros(max(n, 1), np.int64)
        ntok = np.zeros(max(n, 1), np.int32)
        npre = np.zeros(max(n, 1), np.int32)
        cap = token_cap if token_cap is not None else 448 * max(n, 1)
        tok = np.zeros(cap, np.int64) if want_token_times else None
        t_end = C.c_int64()
        p64 = lambda a: a.ctypes.data_as(C.POINTER(C.c_int64))  # noqa: E731
        p32 = lambda a: a.ctypes.data_as(C.POINTER(C.c_int32))  # noqa: E731
        cost = SimCost(prefill_us, step_us, row_us)
        _check(lib.asr_serve_simulate(self.h, C.byref(cost), t0_us, n, p64(ids_a), p64(first),
                                      p64(fin), p32(ntok), p32(npre),
                                      p64(tok) if tok is not None else None, cap,
                                      C.byref(t_end)))
        out, off = {}, 0
        for i, rid in enumerate(ids):
            k = int(ntok[i])
            out[int(rid)] = {"first_us": int(first[i]), "finish_us": int(fin[i]), "n_tokens": k,
                             "n_preempt": int(npre[i]),
                             "token_us": tok[off:off + k].tolist() if tok is not None else None}
            off += k
        return out, t_end.value

    def serve_stats(self):
        """Steps run under FCFS, SJF and HRRN since serve_config."""
        a = (C.c_int64 * 3)()
        _check(lib.asr_serve_stats(self.h, a))
        return list(a)

    def serve_tokens(self, rid):
        buf = np.zeros(448, np.int32)
        n = C.c_int32()
        _check(lib.asr_serve_tokens(self.h, rid, buf.ctypes.data_as(C.POINTER(C.c_int32)), 448,
                                    C.byref(n)))
        return buf[:n.value].tolist()

    def slot_info(self, slot):
        occ, rid, pos, left = C.c_int32(), C.c_int64(), C.c_int32(), C.c_int32()
        _check(lib.asr_slot_info(self.h, slot, C.byref(occ), C.byref(rid), C.byref(pos),
                                 C.byref(left)))
        return {"occupied": bool(occ.value), "id": rid.value, "position": pos.value,
                "steps_left": left.value}

    def set_encoder_streams(self, n):
        """Prefill clips in n groups whose encoder layers run on n streams."""
        _check(lib.asr_set_encoder_streams(self.h, int(n)))

    # -- timing ---------------------------------------------------------------
    def set_decode_graphs(self, on: bool):
        """Replay decode steps from HIP graphs (default) or launch directly."""
        _check(lib.asr_set_decode_graphs(self.h, int(bool(on))))

    def set_timing(self, classes=True):
        """True times every kernel class, False none; an int is a bit mask
        over the class numbers (K_MEL .. K_DECODE)."""
        if classes is True:
            classes = TIME_ALL
        elif classes is False:
            classes = 0
        _check(lib.asr_set_timing(self.h, int(classes)))

    def reset_timing(self):
        _check(lib.asr_reset_timing(self.h))

    def timing(self):
        out = {}
        for k, name in enumerate(KERNEL_CLASSES):
            ms, n, fl, by = C.c_double(), C.c_int64(), C.c_double(), C.c_double()
            _check(lib.asr_get_timing(self.h, k, C.byref(ms), C.byref(n), C.byref(fl),
                                      C.byref(by)))
            out[name] = {"ms": ms.value, "launches": n.value, "flops": fl.value,
                         "bytes": by.value}
        return out

    # -- debug / parity -------------------------------------------------------
    def _clip_args(self, clips, on_device):
        ptrs = (C.c_void_p * len(clips))(*[_ptr(x) for x in clips])
        ns = np.array([x.numel() if hasattr(x, "numel") else len(x) for x in clips], np.int64)
        return ptrs, ns

    def debug_logmel(self, clips, on_device=False):
        if not on_device:
            clips = [np.ascontiguousarray(x, np.float32) for x in clips]
        ptrs, ns = self._clip_args(clips, on_device)
        out = np.zeros((len(clips), 3000, self.cfg.n_mels), np.float32)
        _check(lib.asr_debug_logmel(self.h, ptrs, ns.ctypes.data_as(C.POINTER(C.c_int64)),
                                    len(clips), int(on_device),
                                    out.ctypes.data_as(C.POINTER(C.c_float))))
        return out

    def debug_encode(self, clips, on_device=False):
        if not on_device:
            clips = [np.ascontiguousarray(x, np.float32) for x in clips]
        ptrs, ns = self._clip_args(clips, on_device)
        out = np.zeros((len(clips), 1500, self.cfg.d_model), np.float32)
        _check(lib.asr_debug_encode(self.h, ptrs, ns.ctypes.data_as(C.POINTER(C.c_int64)),
                                    len(clips), int(on_device),
                                    out.ctypes.data_as(C.POINTER(C.c_float))))
        return out

    def debug_attention(self, q, k, v):
        """Encoder attention kernel on [n][1500][d] operands; q in the exp2
        domain (queries times 1/sqrt(64) log2(e))."""
        q, k, v = (np.ascontiguousarray(x, np.float32) for x in (q, k, v))
        assert q.shape == k.shape == v.shape and q.shape[1:] == (1500, self.cfg.d_model)
        out = np.zeros(q.shape, np.float32)
        fp = C.POINTER(C.c_float)
        _check(lib.asr_debug_attention(self.h, q.ctypes.data_as(fp), k.ctypes.data_as(fp),
                                       v.ctypes.data_as(fp), q.shape[0], out.ctypes.data_as(fp)))
        return out

    def debug_set_encoder_out(self, slots, ids, steps_left, E, on_device=False):
        sl, p_sl = _i32(slots)
        idv, p_id = _i64(ids)
        st, p_st = _i32(steps_left)
        if not on_device:
            E = np.ascontiguousarray(E, np.float32)
        _check(lib.asr_debug_set_encoder_out(self.h, p_sl, p_id, p_st, len(sl), _ptr(E),
                                             int(on_device)))

    def debug_get_kv(self, slot, which):
        H = self.cfg.n_head
        ctx = 448 if which == 0 else 1500
        out = np.zeros((self.cfg.n_dec, 2, H, ctx, 64), np.float32)
        _check(lib.asr_debug_get_kv(self.h, slot, which, out.ctypes.data_as(C.POINTER(C.c_float))))
        return out

    def debug_set_self_kv(self, slot, src, length, on_device=False):
        if not on_device:
            src = np.ascontiguousarray(src, np.float32)
        _check(lib.asr_debug_set_self_kv(self.h, slot, _ptr(src), length, int(on_device)))
