"""Python binding of libsara (ctypes, argument marshalling only).

Every step of the rollout-allocation hot path runs in the HIP kernels of
``libsara.so``; this module only converts arguments.  torch is used for device
memory and the stream.  Importing fails loudly when the library has not been
built (``python -m paper_2607_26253_amd.build``).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsara.so")

SARA_OK, SARA_EINVAL, SARA_ENOMEM, SARA_EHIP, SARA_ESTATE, SARA_EDEVICE = 0, -1, -2, -3, -4, -5
SARA_F32, SARA_BF16 = 0, 1
SARA_MODE_SARA, SARA_MODE_FIXED_K, SARA_MODE_SARA_THOMPSON = 0, 1, 2
_MODES = {"sara": SARA_MODE_SARA, "fixed_k": SARA_MODE_FIXED_K, "sara_thompson": SARA_MODE_SARA_THOMPSON}
SARA_COMMIT, SARA_ABANDON, SARA_CONTINUE = 1, 2, 3

EXPORTED = ["sara_init", "sara_begin_step", "sara_decode_step", "sara_posterior_decide",
            "sara_refill", "sara_run", "sara_query", "sara_finish_step", "sara_read_rollouts",
            "sara_read_logs", "sara_read_advantages", "sara_peff_batch", "grpo_group_advantages",
            "sara_sample_logits", "sara_sample_logits_noalloc", "sara_gumbel_fast_max_error", "sara_set_profiling", "sara_reset_profile",
            "sara_read_profile", "sara_set_warm_start", "sara_warm_start_update", "sara_poll",
            "sara_destroy",
            "sara_last_error"]


class sara_model_desc(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("d_ffn", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rope_theta", ctypes.c_float), ("rms_eps", ctypes.c_float),
                ("dtype", ctypes.c_int32), ("eos_id", ctypes.c_int32)]


class sara_alloc_desc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("k", ctypes.c_int32), ("n0", ctypes.c_int32),
                ("commit_min", ctypes.c_int32), ("tau_low", ctypes.c_double), ("alpha0", ctypes.c_double),
                ("beta0", ctypes.c_double), ("budget_N", ctypes.c_int64), ("pool_U", ctypes.c_int32),
                ("n_slots", ctypes.c_int32), ("kv_block", ctypes.c_int32), ("max_prompt", ctypes.c_int32),
                ("max_new", ctypes.c_int32), ("mode", ctypes.c_int32), ("temperature", ctypes.c_float),
                ("top_p", ctypes.c_float), ("forced_eos_u32", ctypes.c_uint32),
                ("prio_quant_bits", ctypes.c_int32), ("seed", ctypes.c_uint64)]


class sara_step_stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("done", "error", "decode_steps", "drawn", "committed",
                                              "abandoned", "active", "queued", "running", "pad_")] + \
               [(n, ctypes.c_int64) for n in ("budget_left", "rollouts", "tokens", "n_decisions",
                                              "n_draws", "n_assigns", "n_finishes")]


class sara_kernel_profile(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 40), ("launches", ctypes.c_int64), ("ms", ctypes.c_double),
                ("bytes", ctypes.c_double), ("flops", ctypes.c_double)]


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    if not os.path.exists(path):
        raise ImportError(f"libsara.so is not built ({path}); run `python -m paper_2607_26253_amd.build`")
    lib = ctypes.CDLL(path)
    P, I32, I64, U64, F32, F64 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64,
                                  ctypes.c_float, ctypes.c_double)
    sig = {
        "sara_init": [ctypes.POINTER(sara_model_desc), ctypes.POINTER(sara_alloc_desc),
                      ctypes.POINTER(P), I32, P, ctypes.POINTER(P)],
        "sara_begin_step": [P, P, P, P, P, I32],
        "sara_decode_step": [P, P, P, I32],
        "sara_posterior_decide": [P],
        "sara_refill": [P],
        "sara_run": [P, P, I32, I64, ctypes.POINTER(I64)],
        "sara_query": [P, ctypes.POINTER(sara_step_stats)],
        "sara_finish_step": [P, F32],
        "sara_read_rollouts": [P, P, P, P, P, P, P, P, P],
        "sara_read_logs": [P, P, I64, P, I64, P, I64, P, I64],
        "sara_read_advantages": [P, P, P, P, I32],
        "sara_peff_batch": [P, P, P, P, I32, I32, P, P],
        "sara_poll": [P, P],
        "grpo_group_advantages": [P, P, I32, F32, P, P],
        "sara_sample_logits": [P, I32, I32, P, P, U64, I32, F32, F32, I32, ctypes.c_uint32, P, P],
        "sara_sample_logits_noalloc": [P, I32, I32, P, P, U64, I32, F32, F32, I32, ctypes.c_uint32, P, P],
        "sara_gumbel_fast_max_error": [ctypes.POINTER(F64), P],
        "sara_set_profiling": [P, I32],
        "sara_reset_profile": [P],
        "sara_read_profile": [P, ctypes.POINTER(sara_kernel_profile), I32, ctypes.POINTER(I32)],
        "sara_set_warm_start": [P, P, P, P, I32],
        "sara_warm_start_update": [P, F64],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.sara_destroy.argtypes = [P]
    lib.sara_destroy.restype = None
    lib.sara_last_error.argtypes = []
    lib.sara_last_error.restype = ctypes.c_char_p
    return lib


_lib = load_library()


class SaraError(RuntimeError):
    def __init__(self, code, where):
        msg = _lib.sara_last_error().decode(errors="replace")
        super().__init__(f"{where} failed with {code}: {msg}")
        self.code = code


def _check(rc, where):
    if rc != SARA_OK:
        raise SaraError(rc, where)


def _ptr(t):
    """Device (torch tensor) or host (numpy array) pointer, or NULL."""
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        assert t.flags["C_CONTIGUOUS"]
        return t.ctypes.data
    assert t.is_contiguous(), "tensors passed to libsara must be contiguous"
    return t.data_ptr()


def _stream_handle(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def model_desc(model: dict) -> sara_model_desc:
    return sara_model_desc(model["n_layers"], model["d_model"], model["n_heads"], model["n_kv_heads"],
                           model["head_dim"], model["d_ffn"], model["vocab"], float(model["rope_theta"]),
                           float(model["rms_eps"]), SARA_BF16 if model["dtype"] == "bf16" else SARA_F32,
                           model["eos_id"])


def alloc_desc(alloc: dict, seed: int) -> sara_alloc_desc:
    return sara_alloc_desc(
        alloc["B"], alloc["k"], alloc["n0"], alloc["commit_min"], float(alloc["tau_low"]),
        float(alloc["alpha0"]), float(alloc["beta0"]), int(alloc["budget_N"]), alloc["pool_U"],
        alloc["n_slots"], alloc["kv_block"], alloc["max_prompt"], alloc["max_new"],
        _MODES[alloc["mode"]],
        float(alloc["temperature"]), float(alloc["top_p"]), int(alloc["forced_eos_u32"]),
        alloc["prio_quant_bits"], int(seed) & ((1 << 64) - 1))


def upload_weights(specs, weights: dict, device="cuda"):
    """Host weight arrays (fixed order) -> device tensors (bf16 bit patterns as int16)."""
    import torch
    out = []
    for name, _ in specs:
        a = weights[name]
        if a.dtype == np.uint16:
            t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device)
        else:
            t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)
        out.append(t)
    return out


class Sara:
    """One libsara context (one allocation problem on one stream)."""

    def __init__(self, model: dict, alloc: dict, seed: int, device_weights, stream=None):
        self.model, self.alloc = dict(model), dict(alloc)
        self.k, self.U, self.max_new = alloc["k"], alloc["pool_U"], alloc["max_new"]
        self._md, self._ad = model_desc(model), alloc_desc(alloc, seed)
        import torch
        arr = (ctypes.c_void_p * len(device_weights))(*[_ptr(t) for t in device_weights])
        # a stream of its own (graph capture is not allowed on the null stream),
        # ordered after the caller's current stream at every call
        self.stream = stream if stream is not None else torch.cuda.Stream()
        self._stream = self.stream.cuda_stream
        self._torch = torch
        self._in()
        h = ctypes.c_void_p()
        _check(_lib.sara_init(ctypes.byref(self._md), ctypes.byref(self._ad), arr, len(device_weights),
                              self._stream, ctypes.byref(h)), "sara_init")
        self.h = h
        self._keep = None
        self._out()

    def _in(self):
        self.stream.wait_stream(self._torch.cuda.current_stream())

    def _out(self):
        self._torch.cuda.current_stream().wait_stream(self.stream)

    def close(self):
        if self.h:
            _lib.sara_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- the hot path ----------------------------------------------------------
    def sara_begin_step(self, d_tokens, h_offsets, d_p, d_forced_len=None, step_index=0):
        h_off = np.ascontiguousarray(h_offsets, dtype=np.int32)
        self._keep = (d_tokens, h_off, d_p, d_forced_len)
        self._in()
        _check(_lib.sara_begin_step(self.h, _ptr(d_tokens), _ptr(h_off), _ptr(d_p), _ptr(d_forced_len),
                                    int(step_index)), "sara_begin_step")
        self._out()

    def sara_decode_step(self, d_forced_tok=None, d_logits=None, model_free=False):
        self._in()
        _check(_lib.sara_decode_step(self.h, _ptr(d_forced_tok), _ptr(d_logits), int(bool(model_free))),
               "sara_decode_step")
        self._out()

    def sara_posterior_decide(self):
        _check(_lib.sara_posterior_decide(self.h), "sara_posterior_decide")

    def sara_refill(self):
        _check(_lib.sara_refill(self.h), "sara_refill")

    def sara_run(self, d_forced_tok=None, graph_iters=16, max_iters=1 << 40):
        it = ctypes.c_int64(0)
        self._in()
        _check(_lib.sara_run(self.h, _ptr(d_forced_tok), int(graph_iters), int(max_iters), ctypes.byref(it)),
               "sara_run")
        self._out()
        return it.value

    def sara_query(self) -> dict:
        st = sara_step_stats()
        _check(_lib.sara_query(self.h, ctypes.byref(st)), "sara_query")
        return {f: getattr(st, f) for f, _ in sara_step_stats._fields_ if f != "pad_"}

    def sara_poll(self, h_pinned):
        """Enqueue the asynchronous poll: h_pinned (a pinned host int32 tensor
        of 2 elements) receives (done, device error word) when the stream
        reaches it; returns at once."""
        assert h_pinned.is_pinned() and h_pinned.numel() >= 2
        self._in()
        _check(_lib.sara_poll(self.h, _ptr(h_pinned)), "sara_poll")

    def sara_finish_step(self, eps=1e-6):
        self._in()
        _check(_lib.sara_finish_step(self.h, float(eps)), "sara_finish_step")
        self._out()

    def sara_set_warm_start(self, d_ids=None, d_a=None, d_b=None):
        """History warm start over a prompt set: d_ids [pool_U] int32 (set
        prompt of each pool prompt), d_a / d_b [n_store] fp64 pseudo-counts,
        all device tensors kept alive by the caller; d_ids=None turns it off."""
        n = 0 if d_ids is None else int(d_a.numel())
        self._warm = (d_ids, d_a, d_b)
        _check(_lib.sara_set_warm_start(self.h, _ptr(d_ids), _ptr(d_a), _ptr(d_b), n), "sara_set_warm_start")

    def sara_warm_start_update(self, lam):
        self._in()
        _check(_lib.sara_warm_start_update(self.h, float(lam)), "sara_warm_start_update")
        self._out()

    def sara_set_profiling(self, enable=True):
        _check(_lib.sara_set_profiling(self.h, int(bool(enable))), "sara_set_profiling")

    def sara_reset_profile(self):
        _check(_lib.sara_reset_profile(self.h), "sara_reset_profile")

    def sara_read_profile(self) -> list:
        arr = (sara_kernel_profile * 32)()
        n = ctypes.c_int32(0)
        _check(_lib.sara_read_profile(self.h, arr, 32, ctypes.byref(n)), "sara_read_profile")
        return [dict(name=arr[i].name.decode(), launches=arr[i].launches, ms=arr[i].ms,
                     bytes=arr[i].bytes, flops=arr[i].flops) for i in range(n.value)]

    # -- readback ---------------------------------------------------------------
    def read_rollouts(self) -> dict:
        nr, mn, U = self.U * self.k, self.max_new, self.U
        out = dict(tokens=np.empty((nr, mn), np.int32), sampled=np.empty((nr, mn), np.int32),
                   length=np.empty(nr, np.int32), reward=np.empty(nr, np.int32),
                   status=np.empty(U, np.int32), n=np.empty(U, np.int32), s=np.empty(U, np.int32),
                   p_eff=np.empty(U, np.float64))
        _check(_lib.sara_read_rollouts(self.h, *(out[k].ctypes.data for k in
                                                 ("tokens", "sampled", "length", "reward", "status", "n",
                                                  "s", "p_eff"))), "sara_read_rollouts")
        return out

    def read_logs(self) -> dict:
        q = self.sara_query()
        dec = np.zeros((q["n_decisions"], 6), np.int64)
        dr = np.zeros((q["n_draws"], 2), np.int64)
        asg = np.zeros((q["n_assigns"], 4), np.int64)
        fin = np.zeros((q["n_finishes"], 6), np.int64)
        _check(_lib.sara_read_logs(self.h, dec.ctypes.data, len(dec), dr.ctypes.data, len(dr),
                                   asg.ctypes.data, len(asg), fin.ctypes.data, len(fin)), "sara_read_logs")
        peff = dec[:, 5].copy().view(np.float64)
        return dict(decisions=dec, p_eff=peff, draws=dr, assigns=asg, finishes=fin)

    def read_advantages(self):
        cap = self.U * self.k
        off = np.zeros(self.U + 1, np.int32)
        r = np.zeros(cap, np.float32)
        a = np.zeros(cap, np.float32)
        _check(_lib.sara_read_advantages(self.h, off.ctypes.data, r.ctypes.data, a.ctypes.data, cap),
               "sara_read_advantages")
        n = int(self.sara_query()["committed"])
        off = off[:n + 1]
        return off, r[:off[-1]], a[:off[-1]]


# -- pure entry points ----------------------------------------------------------
def sara_peff_batch(d_alpha, d_beta, d_n, d_s, k, d_out, stream=None):
    """Eq. peff per prompt under its own prior Beta(d_alpha[i], d_beta[i])."""
    _check(_lib.sara_peff_batch(_ptr(d_alpha), _ptr(d_beta), _ptr(d_n), _ptr(d_s), int(k), int(d_n.numel()),
                                _ptr(d_out), _stream_handle(stream)), "sara_peff_batch")


def grpo_group_advantages(d_r, d_group_off, eps, d_adv, stream=None):
    _check(_lib.grpo_group_advantages(_ptr(d_r), _ptr(d_group_off), int(d_group_off.numel()) - 1, float(eps),
                                      _ptr(d_adv), _stream_handle(stream)), "grpo_group_advantages")


def sara_gumbel_fast_max_error(stream=None):
    out = ctypes.c_double(0.0)
    _check(_lib.sara_gumbel_fast_max_error(ctypes.byref(out), _stream_handle(stream)),
           "sara_gumbel_fast_max_error")
    return out.value


def sara_sample_logits(d_logits, d_rid, d_pos, seed, step_index, temperature, eos_id, forced_eos_u32,
                       d_tok, stream=None, top_p=1.0):
    n, V = d_logits.shape
    _check(_lib.sara_sample_logits(_ptr(d_logits), int(n), int(V), _ptr(d_rid), _ptr(d_pos),
                                   int(seed) & ((1 << 64) - 1), int(step_index), float(temperature),
                                   float(top_p), int(eos_id), int(forced_eos_u32), _ptr(d_tok), _stream_handle(stream)),
           "sara_sample_logits")


# limits of the allocation-free sampler (include/sara.h)
NOALLOC_MAX_ROWS, NOALLOC_MAX_TOPP_ROWS = 4096, 64


def sara_sample_logits_noalloc(d_logits, d_rid, d_pos, seed, step_index, temperature, eos_id, forced_eos_u32,
                               d_tok, stream=None, top_p=1.0):
    """The stand-alone sampler over the library's static scratch (no
    allocation, no synchronisation): enqueued on stream."""
    n, V = d_logits.shape
    _check(_lib.sara_sample_logits_noalloc(_ptr(d_logits), int(n), int(V), _ptr(d_rid), _ptr(d_pos),
                                           int(seed) & ((1 << 64) - 1), int(step_index), float(temperature),
                                           float(top_p), int(eos_id), int(forced_eos_u32), _ptr(d_tok),
                                           _stream_handle(stream)),
           "sara_sample_logits_noalloc")
