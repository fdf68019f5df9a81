"""ctypes binding of libpaci_stage.so (argument marshalling only).

Every step of the stage runs in the HIP library. This module only converts
configs to ``paci_shapes``, hands device pointers of torch tensors and the
current HIP stream to the C ABI, and turns negative status codes into
exceptions. Importing it raises if the library has not been built.
"""
import ctypes
import os
import re

import numpy as np

# torch ships its own HIP runtime. It must be loaded before the library so
# that the library's libamdhip64 dependency resolves to that same copy. Two
# runtimes in one process do not share device allocations.
import torch  # noqa: F401

from . import inputs

# PACI_STAGE_LIB: another build of the same library (e.g. one with host-side
# sanitizers for the host-only tests); the in-tree build otherwise
LIB_PATH = os.environ.get("PACI_STAGE_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                             "libpaci_stage.so")
HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "paci_stage.h")

OK, STEP_DUE = 0, 1
E_INVAL, E_UNSUPPORTED, E_NOMEM, E_ORDER, E_BACKPRESSURE, E_STEP_PENDING, E_NOT_DUE, E_HIP, E_SCRATCH = range(-1, -10, -1)
MIDDLE, FIRST, LAST = 0, 1, 2
FP32, BF16 = 0, 1
PARAMS, GRADS, EXP_AVG, EXP_AVG_SQ = 0, 1, 2, 3
KINDS = {"middle": MIDDLE, "first": FIRST, "last": LAST}
DTYPES = {"fp32": FP32, "bf16": BF16}


class PaciShapes(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("n_layers", "d_model", "n_heads", "head_dim", "d_ff", "seq",
                                              "micro_batch", "vocab", "max_pos", "kind", "dtype")] + \
               [(n, ctypes.c_float) for n in ("lr", "beta1", "beta2", "eps", "weight_decay", "ln_eps")] + \
               [("recompute", ctypes.c_int32), ("lr_warmup", ctypes.c_int32), ("lr_total", ctypes.c_int32),
                ("lr_min_ratio", ctypes.c_float), ("fused_head", ctypes.c_int32), ("dropout", ctypes.c_float),
                ("dropout_seed", ctypes.c_uint32), ("window", ctypes.c_int32)]


class PaciCounters(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("version", "c", "q", "next_f", "next_b", "K", "delay")]


class PaciParamInfo(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("rows", ctypes.c_int32), ("cols", ctypes.c_int32),
                ("offset", ctypes.c_int64), ("numel", ctypes.c_int64), ("decay", ctypes.c_int32)]


class PaciError(RuntimeError):
    def __init__(self, code, where="", hip=0):
        self.code = code
        self.hip = hip
        extra = f", hipError_t {hip}" if hip else ""
        super().__init__(f"{where}: {strerror(code)} ({code}{extra})")


def _load():
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_07881_amd.build` "
                           "(the stage has no fallback implementation)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I, I32P, I64, SZ = ctypes.c_void_p, ctypes.c_int, ctypes.POINTER(ctypes.c_int32), ctypes.c_int64, ctypes.c_size_t
    DP = ctypes.POINTER(ctypes.c_double)
    sig = {
        "paci_fsm_create": (I, [I, I, ctypes.POINTER(P)]),
        "paci_fsm_forward": (I, [P, I, ctypes.POINTER(I)]),
        "paci_fsm_backward": (I, [P, I, ctypes.POINTER(I)]),
        "paci_fsm_step": (I, [P, ctypes.POINTER(I)]),
        "paci_fsm_counters": (I, [P, ctypes.POINTER(PaciCounters)]),
        "paci_fsm_destroy": (I, [P]),
        "paci_schedule": (I, [I, I, I, I32P, I32P, I, ctypes.POINTER(I)]),
        "paci_schedule_flush": (I, [I, I, I, I32P, I32P, I, ctypes.POINTER(I)]),
        "paci_partition": (I, [I, I, DP, DP, DP, ctypes.c_double, I32P, DP, DP]),
        "paci_eta_flush": (ctypes.c_double, [ctypes.c_double, I]),
        "paci_eta_interleaved": (ctypes.c_double, [ctypes.c_double, I, I]),
        "paci_throughput_proxy": (ctypes.c_double, [ctypes.c_double, ctypes.c_double, I]),
        "paci_param_count": (I, [ctypes.POINTER(PaciShapes), ctypes.POINTER(I), ctypes.POINTER(I64)]),
        "paci_param_info_at": (I, [ctypes.POINTER(PaciShapes), I, ctypes.POINTER(PaciParamInfo)]),
        "paci_stage_arena_bytes": (I, [ctypes.POINTER(PaciShapes), I, I, ctypes.POINTER(SZ)]),
        "paci_stage_init": (I, [ctypes.POINTER(PaciShapes), I, I, P, SZ, P, ctypes.POINTER(P)]),
        "paci_stage_destroy": (I, [P]),
        "paci_stage_load": (I, [P, I, P, I64, I]),
        "paci_stage_read": (I, [P, I, P, I64, I]),
        "paci_stage_forward": (I, [P, I, P, P, P, ctypes.POINTER(I)]),
        "paci_stage_backward": (I, [P, I, P, P, ctypes.POINTER(I)]),
        "paci_stage_backward_static": (I, [P, I, P, P, ctypes.POINTER(I)]),
        "paci_stage_step": (I, [P, ctypes.POINTER(I)]),
        "paci_stage_run": (I, [P, I, P, P, P, P, P, I32P]),
        "paci_stage_run_events": (I, [P, I, I32P, I32P, P, P, P, P, P, I32P]),
        "paci_stage_reset_counters": (I, [P]),
        "paci_stage_updates": (I, [P, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32)]),
        "paci_stage_resume": (I, [P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]),
        "paci_stage_counters": (I, [P, ctypes.POINTER(PaciCounters)]),
        "paci_stage_sync": (I, [P]),
        "paci_last_hip_error": (I, [P]),
        "paci_strerror": (ctypes.c_char_p, [I]),
        "paci_kernel_family_count": (I, []),
        "paci_kernel_family_name": (ctypes.c_char_p, [I]),
        "paci_stage_set_timing": (I, [P, I]),
        "paci_stage_kernel_times": (I, [P, I, ctypes.POINTER(I64), ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_double)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()


def strerror(code):
    return lib.paci_strerror(code).decode()


def _check(code, where):
    if code < 0:
        raise PaciError(code, where)
    return code


def header_symbols():
    """Names of the functions include/paci_stage.h declares."""
    with open(HEADER) as fh:
        text = fh.read()
    return sorted(set(re.findall(r"\b(paci_[a-z_]+)\s*\(", text)))


def shapes(cfg):
    s = PaciShapes()
    for k in ("n_layers", "d_model", "n_heads", "head_dim", "d_ff", "seq", "micro_batch"):
        setattr(s, k, int(cfg[k]))
    s.vocab = int(cfg.get("vocab", 0))
    s.max_pos = int(cfg.get("max_pos", 0))
    s.kind = KINDS[cfg["kind"]]
    s.dtype = DTYPES[cfg["dtype"]]
    for k in ("lr", "beta1", "beta2", "eps", "weight_decay", "ln_eps"):
        setattr(s, k, float(cfg[k]))
    s.recompute = int(bool(cfg.get("recompute", False)))
    s.lr_warmup = int(cfg.get("lr_warmup", 0))
    s.lr_total = int(cfg.get("lr_total", 0))
    s.lr_min_ratio = float(cfg.get("lr_min_ratio", 0.1))
    s.fused_head = int(bool(cfg.get("fused_head", False)))
    s.dropout = float(cfg.get("dropout", 0.0))
    s.dropout_seed = int(cfg.get("dropout_seed", 0)) & 0xFFFFFFFF
    s.window = int(bool(cfg.get("window", False)))
    return s


# ---- host-only calls ----------------------------------------------------------------------
def partition(t, s, a, N, budget=float("inf")):
    """paci_partition: returns (cuts, max_time, max_overshoot); max_overshoot == 0
    exactly when every stage fits the budget."""
    t, s, a = (np.ascontiguousarray(x, np.float64) for x in (t, s, a))
    assert t.shape == s.shape == a.shape and t.ndim == 1
    cuts = np.zeros(max(N, 0) + 1, np.int32)
    mt, mo = ctypes.c_double(), ctypes.c_double()
    dp = ctypes.POINTER(ctypes.c_double)
    _check(lib.paci_partition(t.size, N, t.ctypes.data_as(dp), s.ctypes.data_as(dp), a.ctypes.data_as(dp),
                              float(budget), cuts.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                              ctypes.byref(mt), ctypes.byref(mo)), "paci_partition")
    return cuts, mt.value, mo.value


def schedule(M, K, delay, flush=False):
    """paci_schedule (asynchronous 1F1B) or, with ``flush``, paci_schedule_flush
    (synchronous 1F1B with a flush per window): returns (kinds, idx) int32
    arrays (0 = F, 1 = B, 2 = step)."""
    n = ctypes.c_int(0)
    cap = 2 * M + M // max(K, 1) + 1
    kinds = np.zeros(cap, np.int32)
    idx = np.zeros(cap, np.int32)
    name = "paci_schedule_flush" if flush else "paci_schedule"
    _check(getattr(lib, name)(M, K, delay, kinds.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                              idx.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), cap, ctypes.byref(n)), name)
    return kinds[:n.value].copy(), idx[:n.value].copy()


class Fsm:
    """The host-only protocol object (paci_fsm_*)."""

    def __init__(self, K, delay):
        self.h = ctypes.c_void_p()
        _check(lib.paci_fsm_create(K, delay, ctypes.byref(self.h)), "paci_fsm_create")

    def forward(self, mb):
        v = ctypes.c_int(-1)
        return lib.paci_fsm_forward(self.h, mb, ctypes.byref(v)), v.value

    def backward(self, mb):
        v = ctypes.c_int(-1)
        return lib.paci_fsm_backward(self.h, mb, ctypes.byref(v)), v.value

    def step(self):
        v = ctypes.c_int(-1)
        return lib.paci_fsm_step(self.h, ctypes.byref(v)), v.value

    def counters(self):
        c = PaciCounters()
        _check(lib.paci_fsm_counters(self.h, ctypes.byref(c)), "paci_fsm_counters")
        return {k: getattr(c, k) for k, _ in PaciCounters._fields_}

    def __del__(self):
        if getattr(self, "h", None) and lib is not None:
            lib.paci_fsm_destroy(self.h)
            self.h = None


def param_table(cfg):
    """paci_param_info_at for every tensor: list of dicts in canonical order."""
    s = shapes(cfg)
    n, tot = ctypes.c_int(0), ctypes.c_int64(0)
    _check(lib.paci_param_count(ctypes.byref(s), ctypes.byref(n), ctypes.byref(tot)), "paci_param_count")
    out = []
    for i in range(n.value):
        info = PaciParamInfo()
        _check(lib.paci_param_info_at(ctypes.byref(s), i, ctypes.byref(info)), "paci_param_info_at")
        out.append(dict(name=info.name.decode(), rows=info.rows, cols=info.cols, offset=info.offset,
                        numel=info.numel, decay=bool(info.decay)))
    return out


def arena_bytes(cfg, K=None, delay=None):
    s = shapes(cfg)
    b = ctypes.c_size_t(0)
    _check(lib.paci_stage_arena_bytes(ctypes.byref(s), cfg["K"] if K is None else K,
                                      cfg["delay"] if delay is None else delay, ctypes.byref(b)),
           "paci_stage_arena_bytes")
    return b.value


def kernel_families():
    return [lib.paci_kernel_family_name(i).decode() for i in range(lib.paci_kernel_family_count())]


# ---- the stage (device) --------------------------------------------------------------------
def _ptr(t):
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


class Stage:
    """stage_init(shapes, K, delay) on the current torch device and stream."""

    def __init__(self, cfg, K=None, delay=None, device="cuda"):
        import torch
        if not torch.cuda.is_available():
            raise RuntimeError("the PACI stage needs a HIP device")
        self.torch = torch
        self.cfg = dict(cfg)
        self.K = cfg["K"] if K is None else K
        self.delay = cfg["delay"] if delay is None else delay
        self.s = shapes(cfg)
        nbytes = arena_bytes(cfg, self.K, self.delay)
        self.arena = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
        base = self.arena.data_ptr()
        self.arena_ptr = (base + 255) // 256 * 256
        self.stream = torch.cuda.current_stream(self.arena.device)
        self.h = ctypes.c_void_p()
        r = lib.paci_stage_init(ctypes.byref(self.s), self.K, self.delay, ctypes.c_void_p(self.arena_ptr),
                                nbytes, ctypes.c_void_p(self.stream.cuda_stream), ctypes.byref(self.h))
        if r < 0:
            raise PaciError(r, "paci_stage_init", lib.paci_last_hip_error(None) if r == E_HIP else 0)
        self.n_params = sum(p["numel"] for p in param_table(cfg))
        self.act_dtype = torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32
        self.T = cfg["micro_batch"] * cfg["seq"]

    def close(self):
        if getattr(self, "h", None) and lib is not None:
            lib.paci_stage_destroy(self.h)
            self.h = None

    def __del__(self):
        self.close()

    # state transfer
    def load(self, what, values):
        """values: a float32 torch tensor on the device, or a numpy array on the host."""
        if isinstance(values, np.ndarray):
            a = np.ascontiguousarray(values, dtype=np.float32)
            _check(lib.paci_stage_load(self.h, what, ctypes.c_void_p(a.ctypes.data), a.size, 0), "paci_stage_load")
        else:
            assert values.dtype == self.torch.float32 and values.is_contiguous()
            _check(lib.paci_stage_load(self.h, what, _ptr(values), values.numel(), 1), "paci_stage_load")

    def load_params(self, params):
        self.load(PARAMS, inputs.flat_params(self.cfg, params))

    def read(self, what):
        out = np.empty(self.n_params, np.float32)
        _check(lib.paci_stage_read(self.h, what, ctypes.c_void_p(out.ctypes.data), out.size, 0), "paci_stage_read")
        return out

    # events of Alg. 1
    def forward(self, mb, inp, out, targets=None):
        v = ctypes.c_int(-1)
        _check(lib.paci_stage_forward(self.h, mb, _ptr(inp), _ptr(targets), _ptr(out), ctypes.byref(v)),
               "paci_stage_forward")
        return v.value

    def backward(self, mb, grad_out=None, grad_in=None):
        v = ctypes.c_int(-1)
        r = _check(lib.paci_stage_backward(self.h, mb, _ptr(grad_out), _ptr(grad_in), ctypes.byref(v)),
                   "paci_stage_backward")
        return v.value, r == STEP_DUE

    def backward_static(self, mb, grad_out=None, grad_in=None):
        """paci_stage_backward_static: the backward with its attention scratch in the
        library's static buffer (no allocation at call time)."""
        v = ctypes.c_int(-1)
        r = _check(lib.paci_stage_backward_static(self.h, mb, _ptr(grad_out), _ptr(grad_in), ctypes.byref(v)),
                   "paci_stage_backward_static")
        return v.value, r == STEP_DUE

    def step(self):
        v = ctypes.c_int(-1)
        _check(lib.paci_stage_step(self.h, ctypes.byref(v)), "paci_stage_step")
        return v.value

    def try_forward(self, mb, inp, out, targets=None):
        """Like forward but returns the raw status instead of raising."""
        v = ctypes.c_int(-1)
        return lib.paci_stage_forward(self.h, mb, _ptr(inp), _ptr(targets), _ptr(out), ctypes.byref(v))

    def try_backward(self, mb, grad_out=None, grad_in=None):
        v = ctypes.c_int(-1)
        return lib.paci_stage_backward(self.h, mb, _ptr(grad_out), _ptr(grad_in), ctypes.byref(v))

    def try_step(self):
        v = ctypes.c_int(-1)
        return lib.paci_stage_step(self.h, ctypes.byref(v))

    def run(self, M, in_all, grad_out_all=None, out_all=None, grad_in_all=None, targets_all=None):
        """paci_stage_run: replays the canonical order; returns stamps [M, 3] (t^F, t^B, Delta)."""
        stamps = np.zeros((M, 3), np.int32)
        _check(lib.paci_stage_run(self.h, M, _ptr(in_all), ctypes.cast(_ptr(targets_all), ctypes.POINTER(ctypes.c_int32)),
                                  _ptr(grad_out_all), _ptr(out_all), _ptr(grad_in_all),
                                  stamps.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))),
               "paci_stage_run")
        return stamps

    def run_events(self, kinds, idx, in_all, grad_out_all=None, out_all=None, grad_in_all=None, targets_all=None):
        """paci_stage_run_events: replays the (kinds, idx) list; returns stamps [M, 3]
        for micro-batch indices 0 .. max(idx)."""
        kinds = np.ascontiguousarray(kinds, np.int32)
        idx = np.ascontiguousarray(idx, np.int32)
        M = int(idx.max()) + 1 if idx.size else 0
        stamps = np.zeros((max(M, 1), 3), np.int32)
        i32 = ctypes.POINTER(ctypes.c_int32)
        _check(lib.paci_stage_run_events(self.h, kinds.size, kinds.ctypes.data_as(i32), idx.ctypes.data_as(i32),
                                         _ptr(in_all), ctypes.cast(_ptr(targets_all), i32), _ptr(grad_out_all),
                                         _ptr(out_all), _ptr(grad_in_all), stamps.ctypes.data_as(i32)),
               "paci_stage_run_events")
        return stamps[:M]

    def reset_counters(self):
        _check(lib.paci_stage_reset_counters(self.h), "paci_stage_reset_counters")

    def resume(self, version, next_mb, applied, skipped=0):
        """paci_stage_resume: continue a checkpoint of a drained stage."""
        _check(lib.paci_stage_resume(self.h, version, next_mb, applied, skipped), "paci_stage_resume")

    def updates(self):
        """(applied, skipped): updates the step applied and skipped (non-finite G)."""
        a, k = ctypes.c_int32(), ctypes.c_int32()
        _check(lib.paci_stage_updates(self.h, ctypes.byref(a), ctypes.byref(k)), "paci_stage_updates")
        return a.value, k.value

    def counters(self):
        c = PaciCounters()
        _check(lib.paci_stage_counters(self.h, ctypes.byref(c)), "paci_stage_counters")
        return {k: getattr(c, k) for k, _ in PaciCounters._fields_}

    def sync(self):
        _check(lib.paci_stage_sync(self.h), "paci_stage_sync")

    def set_timing(self, on):
        _check(lib.paci_stage_set_timing(self.h, 1 if on else 0), "paci_stage_set_timing")

    def kernel_times(self):
        out = {}
        for i, name in enumerate(kernel_families()):
            n, ms, w = ctypes.c_int64(0), ctypes.c_double(0), ctypes.c_double(0)
            _check(lib.paci_stage_kernel_times(self.h, i, ctypes.byref(n), ctypes.byref(ms), ctypes.byref(w)),
                   "paci_stage_kernel_times")
            out[name] = dict(launches=n.value, ms=ms.value, work=w.value)
        return out


# The C ABI's names for the three events and the constructor.
def stage_init(cfg, K=None, delay=None):
    return Stage(cfg, K, delay)


def stage_forward(stage, mb, inp, out, targets=None):
    return stage.forward(mb, inp, out, targets)


def stage_backward(stage, mb, grad_out=None, grad_in=None):
    return stage.backward(mb, grad_out, grad_in)


def stage_step(stage):
    return stage.step()
