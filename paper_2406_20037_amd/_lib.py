"""ctypes binding of ``libdroplet.so`` (argument marshalling only).

Every function here forwards to the C ABI declared in ``include/droplet.h``
under the same name.  Tensors may be passed as ``torch.Tensor`` (their
``data_ptr()`` is used) or as raw integer device addresses; streams as
``torch.cuda.Stream``, an integer ``hipStream_t`` or ``None`` (the current
torch stream when torch has a device, else the null stream).

The library must have been built (``paper_2406_20037_amd.build``); importing
this module without it raises, there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os

try:
    # PyTorch ships its own HIP runtime (same soname).  Loading it before the
    # library makes the library bind to that runtime, so device pointers and
    # streams handed over from torch belong to the runtime the kernels use.
    import torch as _torch  # noqa: F401
except ImportError:  # plain C-ABI use without torch
    _torch = None

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdroplet.so")

DS_OK = 0
DS_EINVAL = -1
DS_EUNSUPPORTED = -2
DS_EINVALID_SCHED = -3
DS_EHIP = -4
DS_EPARITY = -5
DS_EBUDGET = -6
DS_EEXHAUSTED = -7
DS_ENOMEM = -8
STATUS_NAMES = {0: "DS_OK", -1: "DS_EINVAL", -2: "DS_EUNSUPPORTED", -3: "DS_EINVALID_SCHED",
                -4: "DS_EHIP", -5: "DS_EPARITY", -6: "DS_EBUDGET", -7: "DS_EEXHAUSTED",
                -8: "DS_ENOMEM"}

DS_OP_CONV2D_NCHW = 1
DS_OP_MATMUL_RM = 2
DS_KERNEL_CONV_VALU, DS_KERNEL_CONV_MFMA, DS_KERNEL_MM_VALU, DS_KERNEL_MM_MFMA, DS_KERNEL_CONV_MFMA2 = 1, 2, 3, 4, 5
DS_MAX_KNOBS = 12
DS_MAX_REPEATS = 64
DS_NOALLOC_MAX_FLOATS = 8388608   # kernel_run_noalloc: split partials capacity


class ds_sched(C.Structure):
    _fields_ = [("op", C.c_int32), ("nknobs", C.c_int32), ("shape", C.c_int64 * 9),
                ("idx", C.c_int32 * DS_MAX_KNOBS)]

    def index(self):
        return tuple(self.idx[a] for a in range(self.nknobs))


class ds_geometry(C.Structure):
    _fields_ = [("valid", C.c_int32), ("threads", C.c_int32), ("grid", C.c_int64),
                ("lds_bytes", C.c_int32), ("acc", C.c_int32), ("unroll_eff", C.c_int32),
                ("t0", C.c_int32), ("t1", C.c_int32), ("red", C.c_int32), ("chunks", C.c_int64)]


class ds_kernel_info(C.Structure):
    _fields_ = [("family", C.c_int32), ("nparams", C.c_int32), ("params", C.c_int32 * 6),
                ("instance", C.c_int32), ("threads", C.c_int32), ("grid", C.c_int64),
                ("lds_bytes", C.c_int32), ("splits", C.c_int32), ("args_hash", C.c_uint64),
                ("num_regs", C.c_int32), ("max_threads_per_block", C.c_int32),
                ("local_bytes", C.c_int64), ("static_lds_bytes", C.c_int64)]

    def as_dict(self):
        return {f: (list(getattr(self, f))[: self.nparams] if f == "params" else getattr(self, f))
                for f, _ in self._fields_}


class ds_measure_cfg(C.Structure):
    _fields_ = [("warmup", C.c_int32), ("repeat", C.c_int32), ("min_repeat_ms", C.c_double),
                ("max_number", C.c_int32), ("slow_cut", C.c_double), ("tol", C.c_double),
                ("check", C.c_int32), ("graph", C.c_int32)]


class ds_measurement(C.Structure):
    _fields_ = [("status", C.c_int32), ("n_repeats", C.c_int32), ("number", C.c_int32),
                ("cut", C.c_int32), ("median_ms", C.c_double), ("mean_ms", C.c_double),
                ("min_ms", C.c_double), ("first_ms", C.c_double), ("max_err", C.c_double),
                ("max_ref", C.c_double), ("nonfinite", C.c_int64),
                ("repeats_ms", C.c_double * DS_MAX_REPEATS)]

    def repeats(self):
        return [self.repeats_ms[i] for i in range(self.n_repeats)]


class ds_tune_io(C.Structure):
    _fields_ = [("x", C.c_void_p), ("w", C.c_void_p), ("y", C.c_void_p), ("ref", C.c_void_p),
                ("stream", C.c_void_p)]


class ds_tune_cfg(C.Structure):
    _fields_ = [("n_explore", C.c_int32), ("budget", C.c_int32), ("alpha", C.c_double),
                ("seed", C.c_uint64), ("frozen_mask", C.c_uint32), ("measure", ds_measure_cfg)]


class ds_tune_result(C.Structure):
    _fields_ = [("best", ds_sched), ("best_ms", C.c_double), ("seed_point", ds_sched),
                ("seed_ms", C.c_double), ("status", C.c_int32), ("n_explore_measured", C.c_int32),
                ("n_droplet_measured", C.c_int32), ("n_failed", C.c_int32), ("n_moves", C.c_int32),
                ("wall_s", C.c_double), ("explore_s", C.c_double), ("droplet_s", C.c_double),
                ("best_meas", ds_measurement)]


class ds_trace_entry(C.Structure):
    _fields_ = [("stage", C.c_int32), ("status", C.c_int32), ("key", C.c_uint64),
                ("median_ms", C.c_double)]


class ds_trace(C.Structure):
    _fields_ = [("entries", C.POINTER(ds_trace_entry)), ("cap", C.c_int32), ("n", C.c_int32)]


ds_measure_fn = C.CFUNCTYPE(C.c_int, C.c_void_p, C.POINTER(ds_sched), C.POINTER(ds_measurement))


class ds_exploit_cfg(C.Structure):
    _fields_ = [("kind", C.c_int32), ("budget", C.c_int32), ("seed", C.c_uint64),
                ("valid_only", C.c_int32), ("pop", C.c_int32), ("elite", C.c_int32),
                ("mutation", C.c_double)]


class ds_task(C.Structure):
    _fields_ = [("space", C.c_void_p), ("io", ds_tune_io), ("fn", ds_measure_fn),
                ("ctx", C.c_void_p), ("weight", C.c_double), ("seed", C.c_uint64)]


class ds_round(C.Structure):
    _fields_ = [("task", C.c_int32), ("trials", C.c_int32)]


DS_EXPLOIT_DROPLET, DS_EXPLOIT_RANDOM, DS_EXPLOIT_GRID, DS_EXPLOIT_GA = 0, 1, 2, 3
DS_EXPLOIT_DROPLET_LINE = 4

# name -> (restype, argtypes); the list is also the set of exported symbols
SIGNATURES = {
    "sched_space_create": (C.c_int, [C.c_int, C.POINTER(C.c_int64), C.c_int, C.POINTER(C.c_void_p)]),
    "sched_space_create_lattice": (C.c_int, [C.c_int, C.POINTER(C.c_int32), C.POINTER(C.c_int32),
                                             C.POINTER(C.c_uint64), C.c_int, C.POINTER(C.c_void_p)]),
    "sched_space_destroy": (None, [C.c_void_p]),
    "sched_space_info": (C.c_int, [C.c_void_p, C.POINTER(C.c_int), C.POINTER(C.c_int),
                                   C.POINTER(C.c_uint64)]),
    "sched_space_axis": (C.c_int, [C.c_void_p, C.c_int, C.POINTER(C.c_char_p), C.POINTER(C.c_int),
                                   C.POINTER(C.POINTER(C.c_int32))]),
    "sched_valid": (C.c_int, [C.c_void_p, C.POINTER(ds_sched)]),
    "sched_key": (C.c_int, [C.c_void_p, C.POINTER(ds_sched), C.POINTER(C.c_uint64)]),
    "sched_from_key": (C.c_int, [C.c_void_p, C.c_uint64, C.POINTER(ds_sched)]),
    "sched_neighbors": (C.c_int, [C.c_void_p, C.POINTER(ds_sched), C.POINTER(ds_sched), C.c_int,
                                  C.POINTER(C.c_int)]),
    "sched_origin": (C.c_int, [C.c_void_p, C.POINTER(ds_sched)]),
    "sched_geometry": (C.c_int, [C.c_void_p, C.POINTER(ds_sched), C.POINTER(ds_geometry)]),
    "ansor_draw": (C.c_int, [C.c_void_p, C.c_uint64, C.c_int, C.POINTER(ds_sched),
                             C.POINTER(C.c_int)]),
    "sched_has_kernel": (C.c_int, [C.c_void_p, C.POINTER(ds_sched)]),
    "sched_space_programs": (C.c_int, [C.c_void_p, C.POINTER(C.c_uint64), C.POINTER(C.c_int32),
                                       C.POINTER(C.c_uint64), C.c_int64, C.POINTER(C.c_int64)]),
    "sched_kernel_info": (C.c_int, [C.c_void_p, C.POINTER(ds_sched), C.c_int,
                                    C.POINTER(ds_kernel_info)]),
    "kernel_run": (C.c_int, [C.c_int, C.POINTER(ds_sched), C.c_void_p, C.c_void_p, C.c_void_p,
                             C.c_void_p]),
    "kernel_run_noalloc": (C.c_int, [C.c_int, C.POINTER(ds_sched), C.c_void_p, C.c_void_p,
                                     C.c_void_p, C.c_void_p]),
    "kernel_run_reference": (C.c_int, [C.c_int, C.POINTER(C.c_int64), C.c_void_p, C.c_void_p,
                                       C.c_void_p, C.c_void_p]),
    "ds_measure_cfg_default": (None, [C.POINTER(ds_measure_cfg)]),
    "ds_measure": (C.c_int, [C.POINTER(ds_sched), C.POINTER(ds_tune_io), C.POINTER(ds_measure_cfg),
                             C.c_double, C.POINTER(ds_measurement)]),
    "ds_empty_kernel_floor": (C.c_int, [C.c_void_p, C.POINTER(ds_measure_cfg),
                                        C.POINTER(ds_measurement)]),
    "ds_mfma_ceiling": (C.c_int, [C.c_void_p, C.c_void_p, C.c_int64, C.c_int,
                                  C.POINTER(ds_measure_cfg), C.POINTER(ds_measurement),
                                  C.POINTER(C.c_double)]),
    "ds_tune_cfg_default": (None, [C.POINTER(ds_tune_cfg)]),
    "ansor_sample": (C.c_int, [C.c_void_p, C.c_uint64, C.c_int, C.POINTER(ds_tune_io),
                               C.POINTER(ds_measure_cfg), C.POINTER(ds_sched),
                               C.POINTER(C.c_double), C.POINTER(ds_trace)]),
    "droplet_tune_ex": (C.c_int, [C.c_void_p, C.POINTER(ds_sched), C.c_int, C.POINTER(ds_tune_cfg),
                                  C.POINTER(ds_tune_io), ds_measure_fn, C.c_void_p,
                                  C.POINTER(ds_tune_result), C.POINTER(ds_trace)]),
    "ds_tune": (C.c_int, [C.c_void_p, C.POINTER(ds_tune_cfg), C.POINTER(ds_tune_io), ds_measure_fn,
                          C.c_void_p, C.POINTER(ds_tune_result), C.POINTER(ds_trace)]),
    "ds_cache_create": (C.c_int, [C.c_void_p, C.POINTER(C.c_void_p)]),
    "ds_cache_destroy": (None, [C.c_void_p]),
    "ds_cache_clone": (C.c_int, [C.c_void_p, C.POINTER(C.c_void_p)]),
    "ds_cache_size": (C.c_int, [C.c_void_p]),
    "ds_cache_get": (C.c_int, [C.c_void_p, C.POINTER(ds_sched), C.POINTER(ds_measurement)]),
    "ds_explore": (C.c_int, [C.c_void_p, C.POINTER(ds_tune_cfg), C.POINTER(ds_tune_io),
                             ds_measure_fn, C.c_void_p, C.c_void_p, C.POINTER(ds_tune_result),
                             C.POINTER(ds_trace)]),
    "ds_exploit_cfg_default": (None, [C.POINTER(ds_exploit_cfg)]),
    "ds_exploit": (C.c_int, [C.c_void_p, C.POINTER(ds_sched), C.POINTER(ds_exploit_cfg),
                             C.POINTER(ds_tune_cfg), C.POINTER(ds_tune_io), ds_measure_fn,
                             C.c_void_p, C.c_void_p, C.POINTER(ds_tune_result),
                             C.POINTER(ds_trace)]),
    "ds_tune_tasks": (C.c_int, [C.POINTER(ds_task), C.c_int, C.c_int, C.POINTER(ds_tune_cfg),
                                C.POINTER(ds_tune_result), C.POINTER(ds_round), C.c_int,
                                C.POINTER(C.c_int), C.POINTER(C.c_double)]),
    "droplet_tune": (C.c_int, [C.c_int, C.POINTER(C.c_int64), C.POINTER(ds_sched), C.c_int,
                               C.POINTER(ds_sched), C.POINTER(C.c_double)]),
    "ds_last_error": (C.c_char_p, []),
    "ds_gen_uniform": (C.c_int, [C.c_uint64, C.c_int64, C.POINTER(C.c_float)]),
    "ds_device_info": (C.c_int, [C.POINTER(C.c_int), C.POINTER(C.c_int), C.c_char_p, C.c_int]),
    "ds_num_instances": (C.c_int, []),
    "ds_shutdown": (None, []),
}

if not os.path.exists(LIB_PATH):
    raise RuntimeError(
        f"{LIB_PATH} is missing: build it with `python -m paper_2406_20037_amd.build` "
        "(there is no CPU fallback for the HIP path)")

lib = C.CDLL(LIB_PATH)
for _name, (_res, _args) in SIGNATURES.items():
    _f = getattr(lib, _name)
    _f.restype = _res
    _f.argtypes = _args


class DsError(RuntimeError):
    def __init__(self, func, rc):
        msg = lib.ds_last_error()
        super().__init__(f"{func} -> {STATUS_NAMES.get(rc, rc)}: {msg.decode() if msg else ''}")
        self.rc = rc


def check(func, rc):
    if rc < 0:
        raise DsError(func, rc)
    return rc


def ptr(t):
    """Device address of a tensor or an integer address."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return int(t.data_ptr())


def stream_handle(stream=None):
    if stream is None:
        try:
            import torch
            if torch.cuda.is_available():
                return int(torch.cuda.current_stream().cuda_stream) or None
        except Exception:
            pass
        return None
    if isinstance(stream, int):
        return stream or None
    return int(stream.cuda_stream) or None


def make_io(x, w, y, ref=None, stream=None):
    return ds_tune_io(ptr(x), ptr(w), ptr(y), ptr(ref), stream_handle(stream))


def measure_cfg(**kw):
    cfg = ds_measure_cfg()
    lib.ds_measure_cfg_default(C.byref(cfg))
    for k, v in kw.items():
        setattr(cfg, k, v)
    return cfg


def tune_cfg(measure=None, **kw):
    cfg = ds_tune_cfg()
    lib.ds_tune_cfg_default(C.byref(cfg))
    for k, v in kw.items():
        setattr(cfg, k, v)
    if measure is not None:
        cfg.measure = measure
    return cfg


class Space:
    """A ``ds_space`` handle (sched_space_create / sched_space_create_lattice)."""

    def __init__(self, op=None, shape=None, *, lattice=None, invalid_keys=()):
        h = C.c_void_p()
        if lattice is not None:
            nv = (C.c_int32 * len(lattice))(*[len(v) for v in lattice])
            flat = [int(x) for v in lattice for x in v]
            vals = (C.c_int32 * len(flat))(*flat)
            inv = (C.c_uint64 * max(1, len(invalid_keys)))(*invalid_keys)
            check("sched_space_create_lattice",
                  lib.sched_space_create_lattice(len(lattice), nv, vals, inv, len(invalid_keys),
                                                 C.byref(h)))
        else:
            sh = (C.c_int64 * len(shape))(*[int(v) for v in shape])
            check("sched_space_create", lib.sched_space_create(op, sh, len(shape), C.byref(h)))
        self.h = h
        op_, nk, size = C.c_int(), C.c_int(), C.c_uint64()
        check("sched_space_info", lib.sched_space_info(h, C.byref(op_), C.byref(nk), C.byref(size)))
        self.op, self.nknobs, self.size = op_.value, nk.value, size.value
        self.shape = tuple(int(v) for v in shape) if shape is not None else ()
        self.names, self.values = [], []
        for a in range(self.nknobs):
            name, n, vals = C.c_char_p(), C.c_int(), C.POINTER(C.c_int32)()
            check("sched_space_axis",
                  lib.sched_space_axis(h, a, C.byref(name), C.byref(n), C.byref(vals)))
            self.names.append(name.value.decode())
            self.values.append([vals[i] for i in range(n.value)])
        self.sizes = [len(v) for v in self.values]

    def __del__(self):
        h = getattr(self, "h", None)
        if h and lib is not None:
            try:
                lib.sched_space_destroy(h)
            except Exception:   # interpreter shutdown
                pass
            self.h = None

    def sched(self, idx):
        s = ds_sched()
        s.op = self.op
        s.nknobs = self.nknobs
        for i, v in enumerate(self.shape):
            s.shape[i] = v
        for a, i in enumerate(idx):
            s.idx[a] = int(i)
        return s

    def sched_of(self, **knobs):
        return self.sched([self.values[a].index(knobs[n]) for a, n in enumerate(self.names)])

    def knobs(self, s):
        idx = s.index() if isinstance(s, ds_sched) else tuple(s)
        return {n: self.values[a][i] for a, (n, i) in enumerate(zip(self.names, idx))}

    def valid(self, idx):
        return bool(check("sched_valid", lib.sched_valid(self.h, C.byref(self.sched(idx)))))

    def key(self, idx):
        k = C.c_uint64()
        check("sched_key", lib.sched_key(self.h, C.byref(self.sched(idx)), C.byref(k)))
        return k.value

    def from_key(self, key):
        s = ds_sched()
        check("sched_from_key", lib.sched_from_key(self.h, key, C.byref(s)))
        return s.index()

    def neighbors(self, idx):
        out = (ds_sched * (2 * DS_MAX_KNOBS))()
        n = C.c_int()
        check("sched_neighbors",
              lib.sched_neighbors(self.h, C.byref(self.sched(idx)), out, len(out), C.byref(n)))
        return [out[i].index() for i in range(n.value)]

    def origin(self):
        s = ds_sched()
        check("sched_origin", lib.sched_origin(self.h, C.byref(s)))
        return s.index()

    def geometry(self, idx):
        g = ds_geometry()
        check("sched_geometry", lib.sched_geometry(self.h, C.byref(self.sched(idx)), C.byref(g)))
        return dict(valid=bool(g.valid), grid=g.grid, threads=g.threads, lds_bytes=g.lds_bytes,
                    acc=g.acc, unroll_eff=g.unroll_eff, t0=g.t0, t1=g.t1, red=g.red,
                    chunks=g.chunks)

    def has_kernel(self, idx):
        return bool(check("sched_has_kernel", lib.sched_has_kernel(self.h, C.byref(self.sched(idx)))))

    def kernel_info(self, idx, with_attrs=False):
        """Compiled instance, launch geometry and argument hash of a valid point."""
        out = ds_kernel_info()
        check("sched_kernel_info", lib.sched_kernel_info(self.h, C.byref(self.sched(idx)),
                                                         int(with_attrs), C.byref(out)))
        return out.as_dict()

    def programs(self):
        """(keys, instances, args_hashes) of every valid point, key order (numpy)."""
        import numpy as np
        n = C.c_int64()
        check("sched_space_programs", lib.sched_space_programs(self.h, None, None, None, 0,
                                                               C.byref(n)))
        keys = np.zeros(max(1, n.value), np.uint64)
        inst = np.zeros(max(1, n.value), np.int32)
        hashes = np.zeros(max(1, n.value), np.uint64)
        check("sched_space_programs", lib.sched_space_programs(
            self.h, keys.ctypes.data_as(C.POINTER(C.c_uint64)),
            inst.ctypes.data_as(C.POINTER(C.c_int32)),
            hashes.ctypes.data_as(C.POINTER(C.c_uint64)), n.value, C.byref(n)))
        return keys[: n.value], inst[: n.value], hashes[: n.value]

    def draw(self, seed, n):
        out = (ds_sched * max(1, n))()
        m = C.c_int()
        rc = lib.ansor_draw(self.h, C.c_uint64(seed), n, out, C.byref(m))
        if rc != DS_EEXHAUSTED:
            check("ansor_draw", rc)
        return [out[i].index() for i in range(m.value)]


def kernel_run(op, sched, x, w, y, stream=None):
    return check("kernel_run", lib.kernel_run(op, C.byref(sched), ptr(x), ptr(w), ptr(y),
                                              stream_handle(stream)))


def kernel_run_noalloc(op, sched, x, w, y, stream=None):
    return check("kernel_run_noalloc",
                 lib.kernel_run_noalloc(op, C.byref(sched), ptr(x), ptr(w), ptr(y),
                                        stream_handle(stream)))


def kernel_run_reference(op, shape, x, w, y, stream=None):
    sh = (C.c_int64 * len(shape))(*[int(v) for v in shape])
    return check("kernel_run_reference",
                 lib.kernel_run_reference(op, sh, ptr(x), ptr(w), ptr(y), stream_handle(stream)))


def ds_measure(sched, io, cfg=None, best_so_far_ms=0.0):
    m = ds_measurement()
    check("ds_measure", lib.ds_measure(C.byref(sched), C.byref(io),
                                       C.byref(cfg) if cfg is not None else None,
                                       best_so_far_ms, C.byref(m)))
    return m


def ds_empty_kernel_floor(stream=None, cfg=None):
    m = ds_measurement()
    check("ds_empty_kernel_floor",
          lib.ds_empty_kernel_floor(stream_handle(stream), C.byref(cfg) if cfg else None,
                                    C.byref(m)))
    return m


DS_MFMA_CEILING_SINK = 262144


def ds_mfma_ceiling(sink, iters=512, stream=None, cfg=None):
    """(measurement, flop per launch) of the library's pure-MFMA calibration
    kernel; sink is a float32 device tensor of >= DS_MFMA_CEILING_SINK elements."""
    m = ds_measurement()
    flop = C.c_double()
    check("ds_mfma_ceiling",
          lib.ds_mfma_ceiling(stream_handle(stream), ptr(sink), sink.numel(), iters,
                              C.byref(cfg) if cfg else None, C.byref(m), C.byref(flop)))
    return m, flop.value


def _trace(cap):
    if not cap:
        return None, None
    arr = (ds_trace_entry * cap)()
    return arr, ds_trace(C.cast(arr, C.POINTER(ds_trace_entry)), cap, 0)


def _trace_list(arr, tr):
    if tr is None:
        return None
    return [(arr[i].stage, arr[i].status, arr[i].key, arr[i].median_ms)
            for i in range(min(tr.n, tr.cap))]


def _callback(fn):
    """Wraps fn(idx) -> float | list[float] | None (failure) as a ds_measure_fn."""
    if fn is None:
        return ds_measure_fn(), None

    def cb(ctx, s, out):
        try:
            v = fn(s.contents.index())
        except Exception:
            return DS_EHIP
        if v is None:
            return DS_EHIP
        reps = list(v) if isinstance(v, (list, tuple)) else [float(v)]
        m = out.contents
        m.status = 0
        m.n_repeats = min(len(reps), DS_MAX_REPEATS)
        for i in range(m.n_repeats):
            m.repeats_ms[i] = reps[i]
        srt = sorted(reps)
        n = len(srt)
        m.median_ms = srt[n // 2] if n % 2 else 0.5 * (srt[n // 2 - 1] + srt[n // 2])
        return DS_OK

    c = ds_measure_fn(cb)
    return c, c


def ansor_sample(space, seed, n_explore, io, cfg=None, trace_cap=0):
    best, ms = ds_sched(), C.c_double()
    arr, tr = _trace(trace_cap)
    check("ansor_sample", lib.ansor_sample(space.h, C.c_uint64(seed), n_explore, C.byref(io),
                                           C.byref(cfg) if cfg else None, C.byref(best),
                                           C.byref(ms), C.byref(tr) if tr else None))
    return best, ms.value, _trace_list(arr, tr)


def droplet_tune_ex(space, start, budget, cfg=None, io=None, cost=None, trace_cap=0):
    res = ds_tune_result()
    arr, tr = _trace(trace_cap)
    cb, keep = _callback(cost)
    st = space.sched(start) if start is not None and not isinstance(start, ds_sched) else start
    check("droplet_tune_ex",
          lib.droplet_tune_ex(space.h, C.byref(st) if st is not None else None, budget,
                              C.byref(cfg) if cfg else None, C.byref(io) if io else None, cb, None,
                              C.byref(res), C.byref(tr) if tr else None))
    del keep
    return res, _trace_list(arr, tr)


def ds_tune(space, cfg=None, io=None, cost=None, trace_cap=0):
    res = ds_tune_result()
    arr, tr = _trace(trace_cap)
    cb, keep = _callback(cost)
    check("ds_tune", lib.ds_tune(space.h, C.byref(cfg) if cfg else None,
                                 C.byref(io) if io else None, cb, None, C.byref(res),
                                 C.byref(tr) if tr else None))
    del keep
    return res, _trace_list(arr, tr)


def exploit_cfg(**kw):
    cfg = ds_exploit_cfg()
    lib.ds_exploit_cfg_default(C.byref(cfg))
    for k, v in kw.items():
        setattr(cfg, k, v)
    return cfg


class Cache:
    """Owns a ds_cache of one space."""

    def __init__(self, space, _handle=None):
        self.space = space
        self.h = C.c_void_p(_handle) if _handle else C.c_void_p()
        if not _handle:
            check("ds_cache_create", lib.ds_cache_create(space.h, C.byref(self.h)))

    def __del__(self):
        try:
            if self.h:
                lib.ds_cache_destroy(self.h)
                self.h = C.c_void_p()
        except Exception:
            pass

    def clone(self):
        h = C.c_void_p()
        check("ds_cache_clone", lib.ds_cache_clone(self.h, C.byref(h)))
        return Cache(self.space, h.value)

    def __len__(self):
        n = lib.ds_cache_size(self.h)
        check("ds_cache_size", min(n, 0))
        return n

    def get(self, idx):
        """The cached ds_measurement of idx, or None."""
        m = ds_measurement()
        s = self.space.sched(idx) if not isinstance(idx, ds_sched) else idx
        rc = lib.ds_cache_get(self.h, C.byref(s), C.byref(m))
        check("ds_cache_get", min(rc, 0))
        return m if rc == 1 else None


def ds_explore(space, cache, cfg=None, io=None, cost=None, trace_cap=0):
    res = ds_tune_result()
    arr, tr = _trace(trace_cap)
    cb, keep = _callback(cost)
    check("ds_explore", lib.ds_explore(space.h, C.byref(cfg) if cfg else None,
                                       C.byref(io) if io else None, cb, None, cache.h,
                                       C.byref(res), C.byref(tr) if tr else None))
    del keep
    return res, _trace_list(arr, tr)


def ds_exploit(space, start, ecfg=None, cfg=None, io=None, cost=None, cache=None, trace_cap=0):
    res = ds_tune_result()
    arr, tr = _trace(trace_cap)
    cb, keep = _callback(cost)
    st = start if isinstance(start, ds_sched) else space.sched(start)
    check("ds_exploit", lib.ds_exploit(space.h, C.byref(st), C.byref(ecfg) if ecfg else None,
                                       C.byref(cfg) if cfg else None, C.byref(io) if io else None,
                                       cb, None, cache.h if cache is not None else None,
                                       C.byref(res), C.byref(tr) if tr else None))
    del keep
    return res, _trace_list(arr, tr)


def ds_tune_tasks(spaces, weights, seeds, total_trials, cfg=None, ios=None, costs=None,
                  rounds_cap=4096):
    """One exploration budget over several tasks, then Droplet per task.
    Returns (results[list of ds_tune_result], rounds[list of (task, n)], network_ms)."""
    n = len(spaces)
    tasks = (ds_task * n)()
    keep = []
    for t in range(n):
        tasks[t].space = spaces[t].h
        if ios is not None:
            tasks[t].io = ios[t]
        cb, k = _callback(costs[t] if costs is not None else None)
        keep.append(k)
        tasks[t].fn = cb
        tasks[t].weight = float(weights[t])
        tasks[t].seed = int(seeds[t])
    results = (ds_tune_result * n)()
    rounds = (ds_round * max(1, rounds_cap))()
    nr, net = C.c_int(), C.c_double()
    check("ds_tune_tasks", lib.ds_tune_tasks(tasks, n, int(total_trials),
                                             C.byref(cfg) if cfg else None, results, rounds,
                                             rounds_cap, C.byref(nr), C.byref(net)))
    del keep
    return (list(results), [(rounds[i].task, rounds[i].trials) for i in range(min(nr.value, rounds_cap))],
            net.value)


def droplet_tune(op, shape, start=None, budget=100):
    sh = (C.c_int64 * len(shape))(*[int(v) for v in shape])
    best, ms = ds_sched(), C.c_double()
    check("droplet_tune", lib.droplet_tune(op, sh, C.byref(start) if start is not None else None,
                                           budget, C.byref(best), C.byref(ms)))
    return best, ms.value


def ds_gen_uniform(seed, n):
    buf = (C.c_float * max(1, n))()
    check("ds_gen_uniform", lib.ds_gen_uniform(C.c_uint64(seed), n, buf))
    return buf


def ds_device_info():
    cus, clk = C.c_int(), C.c_int()
    arch = C.create_string_buffer(64)
    check("ds_device_info", lib.ds_device_info(C.byref(cus), C.byref(clk), arch, 64))
    return dict(cus=cus.value, clock_khz=clk.value, arch=arch.value.decode())


def ds_num_instances():
    return lib.ds_num_instances()


def ds_shutdown():
    lib.ds_shutdown()
