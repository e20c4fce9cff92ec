"""ctypes binding of libinfs.so -- argument marshalling only.

Every call maps one-to-one onto the C function of the same name in
``include/infs.h``; device buffers are passed as integers or as objects with a
``data_ptr()`` method (e.g. torch tensors), streams as integers or objects with
a ``cuda_stream`` attribute.  A non-OK status raises ``InfsError``.
The library must have been built (``python -m paper_2506_22950_amd.build``);
there is no fallback.
"""

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# The library to load: libinfs.so next to this file, or the build named by
# INFS_LIBRARY (for instance the host-sanitizer build, see build.py).
LIB_PATH = os.environ.get("INFS_LIBRARY") or os.path.join(HERE, "libinfs.so")

OK, E_ARG, E_STATE, E_CAPACITY, E_DUP, E_NOMEM, E_DEVICE = 0, -1, -2, -3, -4, -5, -6
STATUS_NAMES = {0: "OK", -1: "E_ARG", -2: "E_STATE", -3: "E_CAPACITY", -4: "E_DUP", -5: "E_NOMEM", -6: "E_DEVICE"}
F32, BF16 = 0, 1
NAIVE, FIXED_ROW, FIFO, SJF, FPTAS, FPTAS_SJF, LPT = 0, 1, 2, 3, 4, 5, 6
POLICY = {"naive": NAIVE, "fixed_row": FIXED_ROW, "fifo": FIFO, "sjf": SJF, "fptas": FPTAS, "fptas_sjf": FPTAS_SJF,
          "lpt": LPT}
FPTAS_EPSILON = 0.1
FLAG_DRY_RUN = 1
FLAG_KV_FP8 = 2
STATIC_SCRATCH_BYTES = 16 << 20

# Every symbol include/infs.h declares.
EXPORTS = (
    "infs_abi_version", "infs_create", "infs_destroy", "infs_reset", "infs_prefill_shared",
    "infs_refill_slot", "infs_retire_slot", "infs_decode_step", "infs_end_step", "infs_slot_state",
    "infs_sample_tokens", "infs_sync", "infs_get_stats", "infs_timing_begin", "infs_timing_end",
    "infs_last_error", "infs_sched_create", "infs_sched_next", "infs_sched_done", "infs_sched_pending",
    "infs_sched_destroy", "infs_fptas_assign", "infs_probe_step", "infs_end_probe_step", "infs_probe_batch",
    "infs_probe_state", "infs_release_sample", "infs_read_prefix", "infs_read_response", "infs_set_merge_wait",
    "infs_get_kernel_info", "infs_set_exchange", "infs_exchange_mode", "infs_decode_step_static",
    "infs_sched_optimum", "infs_decode_step_layers", "infs_step_launch_workgroups", "infs_set_step_split",
    "infs_step_split_plan", "infs_probe_step_layers",
)


class InfsError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class Config(ctypes.Structure):
    _fields_ = [
        ("num_layers", ctypes.c_int32), ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("num_prompts", ctypes.c_int32), ("slots_per_prompt", ctypes.c_int32),
        ("samples_per_prompt", ctypes.c_int32), ("max_prompt_len", ctypes.c_int32),
        ("max_suffix_len", ctypes.c_int32), ("page_tokens", ctypes.c_int32), ("num_pages", ctypes.c_int32),
        ("split_tokens", ctypes.c_int32), ("dtype", ctypes.c_int32), ("scale", ctypes.c_float),
        ("flags", ctypes.c_uint32), ("probe_tokens", ctypes.c_int32),
    ]


class KernelInfo(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("bf16", "head_dim", "hpk", "mfma", "prefix_rows", "kv_fp8",
                                             "probe_mfma", "probe_prefix_rows")]


class Stats(ctypes.Structure):
    _fields_ = [("steps", ctypes.c_int64), ("launches", ctypes.c_int64), ("tokens", ctypes.c_int64),
                ("alg_bytes", ctypes.c_double), ("alg_flops", ctypes.c_double)]


_lib = None


def load():
    """Load libinfs.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2506_22950_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, F, U32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_uint32
    sig = {
        "infs_abi_version": (I32, []),
        "infs_create": (I32, [ctypes.POINTER(Config), P, ctypes.POINTER(P)]),
        "infs_destroy": (None, [P]),
        "infs_reset": (I32, [P]),
        "infs_prefill_shared": (I32, [P, I32, I32, I32, P, P]),
        "infs_refill_slot": (I32, [P, I32, I32, I64]),
        "infs_retire_slot": (I32, [P, I32]),
        "infs_decode_step": (I32, [P, I32, P, P, P, P]),
        "infs_decode_step_static": (I32, [P, I32, P, P, P, P]),
        "infs_decode_step_layers": (I32, [P, P, P, P, P, I64, I64, I64]),
        "infs_step_launch_workgroups": (I32, [P]),
        "infs_end_step": (I32, [P]),
        "infs_slot_state": (I32, [P, I32, ctypes.POINTER(I64), ctypes.POINTER(I32)]),
        "infs_sample_tokens": (I32, [P, I32, ctypes.POINTER(I32), I32]),
        "infs_sync": (I32, [P]),
        "infs_get_stats": (I32, [P, ctypes.POINTER(Stats)]),
        "infs_get_kernel_info": (I32, [P, ctypes.POINTER(KernelInfo)]),
        "infs_set_exchange": (I32, [P, I32]),
        "infs_exchange_mode": (I32, [P]),
        "infs_set_step_split": (I32, [P, I32]),
        "infs_step_split_plan": (I32, [I32, I32, I32, I32, ctypes.POINTER(I32), I32, I32, I32, ctypes.POINTER(I32),
                                       ctypes.POINTER(I32)]),
        "infs_timing_begin": (I32, [P]),
        "infs_timing_end": (I32, [P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                  ctypes.POINTER(I64)]),
        "infs_last_error": (ctypes.c_char_p, [P]),
        "infs_sched_create": (I32, [I32, I32, I32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(P)]),
        "infs_sched_next": (I32, [P, I32, ctypes.POINTER(I64)]),
        "infs_sched_done": (I32, [P, I32]),
        "infs_sched_pending": (I32, [P]),
        "infs_sched_destroy": (None, [P]),
        "infs_fptas_assign": (I32, [I32, I32, ctypes.POINTER(ctypes.c_double), ctypes.c_double,
                                    ctypes.POINTER(I32), ctypes.POINTER(I32)]),
        "infs_sched_optimum": (I32, [I32, I32, ctypes.POINTER(I32), I64, ctypes.POINTER(I64), ctypes.POINTER(I64),
                                     ctypes.POINTER(I32)]),
        "infs_probe_step": (I32, [P, I32, I32, I32, I32, ctypes.POINTER(ctypes.c_uint8), P, P, P, P]),
        "infs_probe_step_layers": (I32, [P, I32, I32, I32, ctypes.POINTER(ctypes.c_uint8), P, P, P, P, I64, I64,
                                         I64]),
        "infs_end_probe_step": (I32, [P]),
        "infs_probe_batch": (I32, [P]),
        "infs_probe_state": (I32, [P, I32, I64, ctypes.POINTER(I32)]),
        "infs_release_sample": (I32, [P, I32, I64]),
        "infs_read_prefix": (I32, [P, I32, I32, P, P]),
        "infs_read_response": (I32, [P, I32, I32, P, P]),
        "infs_set_merge_wait": (I32, [P, I32]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def _stream(s):
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return int(s.cuda_stream)


def _check(ctx_handle, st):
    if st != OK:
        msg = load().infs_last_error(ctx_handle)
        raise InfsError(st, msg.decode() if msg else "")


def make_config(**kw) -> Config:
    c = Config()
    for k, v in kw.items():
        setattr(c, k, v)
    return c


class Context:
    """One infs_ctx.  Methods carry the names of the C calls without the prefix."""

    def __init__(self, config: Config, stream=None):
        lib = load()
        h = ctypes.c_void_p()
        _check(None, lib.infs_create(ctypes.byref(config), _stream(stream), ctypes.byref(h)))
        self._h = h
        self.config = config

    def destroy(self):
        if self._h:
            load().infs_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass

    def _call(self, fn, *args):
        _check(self._h, fn(self._h, *args))

    def reset(self):
        self._call(load().infs_reset)

    def prefill_shared(self, prompt, layer, prompt_len, k, v):
        self._call(load().infs_prefill_shared, prompt, layer, prompt_len, _ptr(k), _ptr(v))

    def refill_slot(self, slot, prompt, sample_id):
        self._call(load().infs_refill_slot, slot, prompt, sample_id)

    def retire_slot(self, slot):
        self._call(load().infs_retire_slot, slot)

    def decode_step(self, layer, q, k_new, v_new, o):
        self._call(load().infs_decode_step, layer, _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(o))

    def decode_step_static(self, layer, q, k_new, v_new, o):
        self._call(load().infs_decode_step_static, layer, _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(o))

    def decode_step_layers(self, q, k_new, v_new, o, q_layer_stride=0, kv_layer_stride=0, o_layer_stride=0):
        self._call(load().infs_decode_step_layers, _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(o), q_layer_stride,
                   kv_layer_stride, o_layer_stride)

    @property
    def step_launch_workgroups(self):
        return load().infs_step_launch_workgroups(self._h)

    def end_step(self):
        self._call(load().infs_end_step)

    def slot_state(self, slot):
        sid, ln = ctypes.c_int64(), ctypes.c_int32()
        self._call(load().infs_slot_state, slot, ctypes.byref(sid), ctypes.byref(ln))
        return sid.value, ln.value

    def sample_tokens(self, prompt):
        n = self.config.samples_per_prompt
        buf = (ctypes.c_int32 * n)()
        self._call(load().infs_sample_tokens, prompt, buf, n)
        return np.frombuffer(buf, dtype=np.int32).copy()

    def sync(self):
        self._call(load().infs_sync)

    def set_merge_wait(self, max_polls):
        self._call(load().infs_set_merge_wait, max_polls)

    @property
    def probe_batch(self):
        return load().infs_probe_batch(self._h)

    def probe_step(self, layer, prompt, first_sample, n, live, q, k_new, v_new, o):
        """live: n truthy values, or None for all live."""
        buf = None
        if live is not None:
            buf = (ctypes.c_uint8 * n)(*[1 if x else 0 for x in live])
        self._call(load().infs_probe_step, layer, prompt, first_sample, n, buf, _ptr(q), _ptr(k_new), _ptr(v_new),
                   _ptr(o))

    def probe_step_layers(self, prompt, first_sample, n, live, q, k_new, v_new, o, q_layer_stride=0,
                          kv_layer_stride=0, o_layer_stride=0):
        """Every layer of one probe step in one launch; strides in bytes (0: n rows)."""
        buf = None
        if live is not None:
            buf = (ctypes.c_uint8 * n)(*[1 if x else 0 for x in live])
        self._call(load().infs_probe_step_layers, prompt, first_sample, n, buf, _ptr(q), _ptr(k_new), _ptr(v_new),
                   _ptr(o), q_layer_stride, kv_layer_stride, o_layer_stride)

    def end_probe_step(self):
        self._call(load().infs_end_probe_step)

    def probe_state(self, prompt, sample_id):
        n = ctypes.c_int32()
        self._call(load().infs_probe_state, prompt, sample_id, ctypes.byref(n))
        return n.value

    def release_sample(self, prompt, sample_id):
        self._call(load().infs_release_sample, prompt, sample_id)

    def _kv_dtype(self):
        if self.config.flags & FLAG_KV_FP8:
            return np.uint8
        return np.uint16 if self.config.dtype == BF16 else np.float32

    def read_prefix(self, prompt, layer, prompt_len):
        """(K, V) of a prefilled prompt as stored, numpy [prompt_len, Hkv, d]."""
        c = self.config
        shape = (prompt_len, c.num_kv_heads, c.head_dim)
        k = np.zeros(shape, dtype=self._kv_dtype())
        v = np.zeros(shape, dtype=self._kv_dtype())
        self._call(load().infs_read_prefix, prompt, layer, k.ctypes.data, v.ctypes.data)
        return k, v

    def read_response(self, slot, layer):
        """(K, V) of a live slot's response as stored, numpy [len, Hkv, d]."""
        c = self.config
        _, n = self.slot_state(slot)
        shape = (n, c.num_kv_heads, c.head_dim)
        k = np.zeros(shape, dtype=self._kv_dtype())
        v = np.zeros(shape, dtype=self._kv_dtype())
        self._call(load().infs_read_response, slot, layer, k.ctypes.data, v.ctypes.data)
        return k, v

    def get_stats(self) -> Stats:
        s = Stats()
        self._call(load().infs_get_stats, ctypes.byref(s))
        return s

    def set_exchange(self, mode: int):
        """0: partials through the device coherence point; 1: through the XCD's L2
        (the default where available); 2: as 1 with the XCD check forced to fail."""
        self._call(load().infs_set_exchange, mode)

    def exchange_mode(self) -> int:
        return load().infs_exchange_mode(self._h)

    def set_step_split(self, mode: int):
        """Work split of step launches: 1 near-equal response pieces (default), 0 the
        per-layer launch's chunks."""
        self._call(load().infs_set_step_split, mode)

    def kernel_info(self) -> dict:
        """The decode (and probe) kernel instantiation this context runs."""
        k = KernelInfo()
        self._call(load().infs_get_kernel_info, ctypes.byref(k))
        return {n: getattr(k, n) for n, _ in KernelInfo._fields_}

    def timing_begin(self):
        self._call(load().infs_timing_begin)

    def timing_end(self):
        """(summed kernel ms, region ms from HIP events, launches)."""
        ms, region, n = ctypes.c_double(), ctypes.c_double(), ctypes.c_int64()
        self._call(load().infs_timing_end, ctypes.byref(ms), ctypes.byref(region), ctypes.byref(n))
        return ms.value, region.value, n.value

    @property
    def last_error(self):
        return load().infs_last_error(self._h).decode()


class Sched:
    """One infs_sched (host refill policy for one prompt's m slots)."""

    def __init__(self, G, m, policy, pred_len=None):
        lib = load()
        if isinstance(policy, str):
            policy = POLICY[policy]
        h = ctypes.c_void_p()
        arr = None
        if pred_len is not None:
            self._pred = np.ascontiguousarray(pred_len, dtype=np.float64)
            arr = self._pred.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
        st = lib.infs_sched_create(G, m, policy, arr, ctypes.byref(h))
        if st != OK:
            raise InfsError(st, "infs_sched_create")
        self._h = h

    def next(self, slot):
        out = ctypes.c_int64()
        st = load().infs_sched_next(self._h, slot, ctypes.byref(out))
        if st != OK:
            raise InfsError(st, f"infs_sched_next(slot={slot})")
        return out.value

    def done(self, slot):
        st = load().infs_sched_done(self._h, slot)
        if st != OK:
            raise InfsError(st, f"infs_sched_done(slot={slot})")

    @property
    def pending(self):
        return load().infs_sched_pending(self._h)

    def __del__(self):
        try:
            if self._h:
                load().infs_sched_destroy(self._h)
                self._h = None
        except Exception:
            pass


def fptas_assign(pred_len, N, epsilon=FPTAS_EPSILON):
    """infs_fptas_assign: (group, pos) arrays of Algorithm 2."""
    pred = np.ascontiguousarray(pred_len, dtype=np.float64)
    G = len(pred)
    group = np.zeros(G, dtype=np.int32)
    pos = np.zeros(G, dtype=np.int32)
    I32P = ctypes.POINTER(ctypes.c_int32)
    st = load().infs_fptas_assign(G, N, pred.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), epsilon,
                                  group.ctypes.data_as(I32P), pos.ctypes.data_as(I32P))
    if st != OK:
        raise InfsError(st, "infs_fptas_assign")
    return group, pos


def sched_optimum(lengths, m, max_nodes=20_000_000):
    """infs_sched_optimum: (best, lower, slot array); best == lower when the optimum is proven."""
    L = np.ascontiguousarray(lengths, dtype=np.int32)
    slot = np.zeros(len(L), dtype=np.int32)
    best, lower = ctypes.c_int64(), ctypes.c_int64()
    I32P = ctypes.POINTER(ctypes.c_int32)
    st = load().infs_sched_optimum(len(L), m, L.ctypes.data_as(I32P), max_nodes, ctypes.byref(best),
                                   ctypes.byref(lower), slot.ctypes.data_as(I32P))
    if st != OK:
        raise InfsError(st, "infs_sched_optimum")
    return best.value, lower.value, slot


def step_split_plan(nj, lens, n_prefix_items, prefix_split, split, scmax, mode=1):
    """infs_step_split_plan: (roles, pieces) of one step launch, roles = dict(n_pre, n_suf, n_merge,
    items, cut) and pieces[s] the response items of slot s."""
    L = np.ascontiguousarray(lens, dtype=np.int32)
    pieces = np.zeros(len(L), dtype=np.int32)
    roles = np.zeros(5, dtype=np.int32)
    I32P = ctypes.POINTER(ctypes.c_int32)
    st = load().infs_step_split_plan(nj, len(L), n_prefix_items, prefix_split, L.ctypes.data_as(I32P), split, scmax,
                                     mode, pieces.ctypes.data_as(I32P), roles.ctypes.data_as(I32P))
    if st != OK:
        raise InfsError(st, "infs_step_split_plan")
    return dict(zip(("n_pre", "n_suf", "n_merge", "items", "cut"), (int(x) for x in roles))), pieces
