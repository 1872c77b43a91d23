"""ctypes binding of the C-ABI library ``lib/libarplan.so`` (include/ar_plan.h).

Argument marshalling only: every function here forwards to the C function
of the same name and raises ``ArError`` on a non-zero status.  All work,
including plan expansion, happens in the library.  Importing this module
loads the library and raises ImportError if it has not been built: there is
no fallback path.

Buffers may be passed as integers (device addresses) or as objects with a
``data_ptr()`` method (e.g. torch tensors), or as the pointer array
``pointers(bufs)`` returns, which repeated executions on the same buffers can
reuse; streams as integers (hipStream_t handles, 0 = default stream) or
objects with a ``cuda_stream`` attribute.
"""

import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_float, c_int32, c_int64, c_void_p

# One HIP runtime per process: buffers and streams come from torch, so the
# library must bind to the HIP runtime torch loads.  Both runtimes carry the
# SONAME libamdhip64.so.7; loading torch first makes the library's
# dependency resolve to torch's copy instead of a second runtime instance.
try:
    import torch  # noqa: F401
except ImportError:
    torch = None

# The test suite loads this file a second time under another module name,
# bound to the test build of the library (the same code plus its checking
# hooks), by placing _LIB_PATH in the module's namespace before running it;
# ARPLAN_LIB names another build of the same library (the sanitized
# host-test build) to load instead.
LIB_PATH = globals().get("_LIB_PATH") or os.environ.get("ARPLAN_LIB") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "lib", "libarplan.so")
if not os.path.exists(LIB_PATH):
    raise ImportError(
        "libarplan.so is not built (%s); run "
        "`python -m paper_2409_04202_amd.build` first" % LIB_PATH)
_lib = ctypes.CDLL(LIB_PATH)

AR_OK, AR_ERR_INVALID_ARG, AR_ERR_UNSUPPORTED, AR_ERR_OOM, AR_ERR_HIP, \
    AR_ERR_INTERNAL = range(6)
AR_F32, AR_I32, AR_BF16 = range(3)
AR_RING, AR_RHD, AR_CPS, AR_TREE, AR_RB, AR_GENTREE = range(6)
AR_OP_REDUCE, AR_OP_COPY = range(2)
AR_OPT_FUSE, AR_OPT_SLICE, AR_OPT_RESIDENT = 0, 1, 2

DTYPES = {"f32": AR_F32, "i32": AR_I32, "bf16": AR_BF16}
KINDS = {"ring": AR_RING, "rhd": AR_RHD, "cps": AR_CPS, "tree": AR_TREE,
         "rb": AR_RB, "gentree": AR_GENTREE}
ESIZE = {AR_F32: 4, AR_I32: 4, AR_BF16: 2}


class ar_topology(ctypes.Structure):
    _fields_ = [("kind", c_int32), ("num_levels", c_int32),
                ("fanin", POINTER(c_int32))]


class ar_step(ctypes.Structure):
    _fields_ = [("phase", c_int32), ("op", c_int32), ("dst", c_int32),
                ("nsrc", c_int32), ("srcs", POINTER(c_int32)),
                ("begin", c_int64), ("end", c_int64)]


_P = c_void_p
_sig = {
    "ar_plan_create": [c_int32, c_int64, c_int32, POINTER(ar_topology),
                       POINTER(_P)],
    "ar_plan_create_custom": [c_int32, c_int64, c_int32, POINTER(ar_step),
                              c_int64, POINTER(_P)],
    "ar_plan_create_gentree": [c_int64, c_int32, c_int32, POINTER(c_int32),
                               POINTER(_P)],
    "ar_plan_destroy": [_P],
    "ar_plan_execute": [_P, POINTER(c_void_p), c_void_p],
    "ar_plan_execute_strided": [_P, c_void_p, c_int64, c_void_p],
    "ar_plan_execute_noalloc": [_P, POINTER(c_void_p), c_void_p],
    "ar_plan_execute_timed": [_P, POINTER(c_void_p), c_void_p, _P],
    "ar_plan_info": [_P, POINTER(c_int32), POINTER(c_int64), POINTER(c_int32),
                     POINTER(c_int32), POINTER(c_int64)],
    "ar_plan_get_step": [_P, c_int64, POINTER(ar_step)],
    "ar_plan_phase_info": [_P, c_int32, POINTER(c_int32), POINTER(c_int64),
                           POINTER(c_int64), POINTER(c_int64)],
    "ar_plan_owner": [_P, c_int32, POINTER(c_int64), POINTER(c_int64)],
    "ar_plan_bytes": [_P, POINTER(c_int64), POINTER(c_int64)],
    "ar_plan_set_option": [_P, c_int32, c_int64],
    "ar_plan_num_launches": [_P, POINTER(c_int32)],
    "ar_plan_launch_info": [_P, c_int32, POINTER(c_int32), POINTER(c_int32),
                            POINTER(c_int32), POINTER(c_int64), POINTER(c_int64)],
    "ar_plan_launch_kernel": [_P, c_int32, POINTER(c_int32)],
    "ar_genmodel_terms": [_P, c_int64, POINTER(c_double)],
    "ar_genmodel_terms_tiered": [_P, c_int32, POINTER(c_int64), POINTER(c_double)],
    "ar_genmodel_select_tiered": [c_int32, c_int64, c_int32, POINTER(c_double), c_int32,
                                  POINTER(c_int64), c_int32, POINTER(c_int32), POINTER(c_int32),
                                  POINTER(c_int32), POINTER(c_double)],
    "ar_genmodel_select": [c_int32, c_int64, c_int32, POINTER(c_double), c_int64, c_int32,
                           POINTER(c_int32), POINTER(c_int32), POINTER(c_int32),
                           POINTER(c_double)],
    "ar_timer_create": [c_int64, POINTER(_P)],
    "ar_timer_reset": [_P],
    "ar_timer_read": [_P, c_int64, POINTER(c_int64), POINTER(c_int32),
                      POINTER(c_float)],
    "ar_timer_destroy": [_P],
}
for _name, _args in _sig.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = c_int32
_lib.ar_status_string.argtypes = [c_int32]
_lib.ar_status_string.restype = c_char_p
_lib.ar_last_error.argtypes = []
_lib.ar_last_error.restype = c_char_p

EXPORTED = sorted(list(_sig) + ["ar_status_string", "ar_last_error"])


class ArError(RuntimeError):
    def __init__(self, status, detail):
        self.status = status
        super().__init__("%s: %s" % (ar_status_string(status), detail))


def ar_status_string(status):
    return _lib.ar_status_string(int(status)).decode()


def ar_last_error():
    return _lib.ar_last_error().decode()


def _check(status):
    if status != AR_OK:
        raise ArError(status, ar_last_error())


def _ptr(x):
    if x is None:
        return None
    if hasattr(x, "data_ptr"):
        return int(x.data_ptr())
    return int(x)


def pointers(bufs):
    """The C array of device pointers ``ar_plan_execute`` takes, built once
    for a buffer set (reading ``data_ptr()`` of many tensors per call costs
    more host time than launching a short plan)."""
    return (c_void_p * max(1, len(bufs)))(*[_ptr(b) for b in bufs])


def _ptr_array(bufs):
    return bufs if isinstance(bufs, ctypes.Array) else pointers(bufs)


def _stream(s):
    if s is None:
        return None
    if hasattr(s, "cuda_stream"):
        return int(s.cuda_stream) or None
    return int(s) or None


def _dtype(d):
    return DTYPES[d] if isinstance(d, str) else int(d)


def _kind(k):
    return KINDS[k] if isinstance(k, str) else int(k)


# ----------------------------------------------------------------- plans

def ar_plan_create(n, N, dtype, kind, fanin=None):
    """Returns the plan handle (an int)."""
    fan = list(fanin or [])
    arr = (c_int32 * max(1, len(fan)))(*fan)
    topo = ar_topology(_kind(kind), len(fan), arr if fan else None)
    out = _P()
    _check(_lib.ar_plan_create(int(n), int(N), _dtype(dtype),
                               ctypes.byref(topo), ctypes.byref(out)))
    return out.value


def ar_plan_create_gentree(N, dtype, nchild):
    """``nchild``: child counts of the tree's nodes in preorder (0 = server).
    Returns the plan handle."""
    counts = list(nchild)
    arr = (c_int32 * max(1, len(counts)))(*counts)
    out = _P()
    _check(_lib.ar_plan_create_gentree(int(N), _dtype(dtype), len(counts), arr,
                                       ctypes.byref(out)))
    return out.value


def ar_plan_create_custom(n, N, dtype, steps):
    """``steps``: iterable of (phase, op, dst, srcs, begin, end); op is
    "reduce"/"copy" or AR_OP_*."""
    steps = list(steps)
    arr = (ar_step * max(1, len(steps)))()
    keep = []
    for i, (ph, op, dst, srcs, b, e) in enumerate(steps):
        srcs = list(srcs)
        sa = (c_int32 * max(1, len(srcs)))(*srcs)
        keep.append(sa)
        if isinstance(op, str):
            op = AR_OP_REDUCE if op == "reduce" else AR_OP_COPY
        arr[i] = ar_step(int(ph), int(op), int(dst), len(srcs),
                         ctypes.cast(sa, POINTER(c_int32)), int(b), int(e))
    out = _P()
    _check(_lib.ar_plan_create_custom(int(n), int(N), _dtype(dtype), arr,
                                      len(steps), ctypes.byref(out)))
    return out.value


def ar_plan_destroy(plan):
    _check(_lib.ar_plan_destroy(plan))


def ar_plan_execute(plan, bufs, stream=None):
    _check(_lib.ar_plan_execute(plan, _ptr_array(bufs), _stream(stream)))


def ar_plan_execute_noalloc(plan, bufs, stream=None):
    _check(_lib.ar_plan_execute_noalloc(plan, _ptr_array(bufs), _stream(stream)))


AR_NOALLOC_MAX_BYTES = 32 << 20


def ar_plan_execute_strided(plan, base, stride_bytes, stream=None):
    _check(_lib.ar_plan_execute_strided(plan, _ptr(base), int(stride_bytes),
                                        _stream(stream)))


def ar_plan_execute_timed(plan, bufs, stream, timer):
    _check(_lib.ar_plan_execute_timed(plan, _ptr_array(bufs), _stream(stream), timer))


def ar_plan_info(plan):
    """(n, N, dtype, num_phases, num_steps)"""
    n, N, dt, ph, st = c_int32(), c_int64(), c_int32(), c_int32(), c_int64()
    _check(_lib.ar_plan_info(plan, ctypes.byref(n), ctypes.byref(N),
                             ctypes.byref(dt), ctypes.byref(ph),
                             ctypes.byref(st)))
    return n.value, N.value, dt.value, ph.value, st.value


def ar_plan_get_step(plan, i):
    """(phase, op, dst, srcs tuple, begin, end)"""
    s = ar_step()
    _check(_lib.ar_plan_get_step(plan, int(i), ctypes.byref(s)))
    return (s.phase, s.op, s.dst, tuple(s.srcs[j] for j in range(s.nsrc)),
            s.begin, s.end)


def ar_plan_phase_info(plan, phase):
    """(op, first_step, num_steps, bytes)"""
    op, f, c, b = c_int32(), c_int64(), c_int64(), c_int64()
    _check(_lib.ar_plan_phase_info(plan, int(phase), ctypes.byref(op),
                                   ctypes.byref(f), ctypes.byref(c),
                                   ctypes.byref(b)))
    return op.value, f.value, c.value, b.value


def ar_plan_owner(plan, p):
    b, e = c_int64(), c_int64()
    _check(_lib.ar_plan_owner(plan, int(p), ctypes.byref(b), ctypes.byref(e)))
    return b.value, e.value


def ar_plan_bytes(plan):
    """(reduce_bytes, copy_bytes)"""
    r, c = c_int64(), c_int64()
    _check(_lib.ar_plan_bytes(plan, ctypes.byref(r), ctypes.byref(c)))
    return r.value, c.value


def ar_plan_set_option(plan, option, value):
    _check(_lib.ar_plan_set_option(plan, int(option), int(value)))


def ar_plan_num_launches(plan):
    c = c_int32()
    _check(_lib.ar_plan_num_launches(plan, ctypes.byref(c)))
    return c.value


def ar_plan_launch_info(plan, i):
    """(phase, nsrc, max_dst, num_steps, bytes)"""
    ph, k, d, n, b = c_int32(), c_int32(), c_int32(), c_int64(), c_int64()
    _check(_lib.ar_plan_launch_info(plan, int(i), ctypes.byref(ph),
                                    ctypes.byref(k), ctypes.byref(d),
                                    ctypes.byref(n), ctypes.byref(b)))
    return ph.value, k.value, d.value, n.value, b.value


KERNEL_NAMES = {0: "phase_kernel", 1: "split_kernel", 2: "sliced_kernel",
                3: "resident_kernel", 4: "stream_kernel"}


def ar_plan_launch_kernel(plan, i):
    """Name of the kernel launch i runs on 16-byte aligned buffers."""
    k = c_int32()
    _check(_lib.ar_plan_launch_kernel(plan, int(i), ctypes.byref(k)))
    return KERNEL_NAMES[k.value]


# -------------------------------------------------------------- GenModel

AR_GENMODEL_TERMS = 6


def ar_genmodel_terms(plan, cache_bytes):
    """(A, K, Dh, Dc, Bh, Bc) of a plan, as numbers."""
    t = (c_double * AR_GENMODEL_TERMS)()
    _check(_lib.ar_genmodel_terms(plan, int(cache_bytes), t))
    return tuple(t)


def ar_genmodel_terms_tiered(plan, cache_bytes):
    """The tiered terms of a plan (cache_bytes: the tiers' sizes, largest
    first): A, K, reduce bytes from HBM and each tier, copy bytes likewise."""
    tiers = len(cache_bytes)
    sizes = (c_int64 * max(1, tiers))(*[int(x) for x in cache_bytes])
    t = (c_double * (4 + 2 * max(1, tiers)))()
    _check(_lib.ar_genmodel_terms_tiered(plan, tiers, sizes, t))
    return tuple(t)


def ar_genmodel_select_tiered(n, N, dtype, params, cache_bytes, max_levels=3):
    """(kind name, fan-in tuple or None, predicted seconds) under the tiered
    terms (params: one per term)."""
    tiers = len(cache_bytes)
    if len(params) != 4 + 2 * tiers:
        raise ValueError("%d parameters expected" % (4 + 2 * tiers))
    sizes = (c_int64 * max(1, tiers))(*[int(x) for x in cache_bytes])
    pa = (c_double * len(params))(*[float(x) for x in params])
    kind, lv = c_int32(), c_int32()
    fan = (c_int32 * max(1, int(max_levels)))()
    sec = c_double()
    _check(_lib.ar_genmodel_select_tiered(int(n), int(N), _dtype(dtype), pa, tiers, sizes,
                                          int(max_levels), ctypes.byref(kind), ctypes.byref(lv),
                                          fan, ctypes.byref(sec)))
    name = {v: k for k, v in KINDS.items()}[kind.value]
    return name, (tuple(fan[i] for i in range(lv.value)) if lv.value else None), sec.value


def ar_genmodel_select(n, N, dtype, params, cache_bytes, max_levels=3):
    """(kind name, fan-in tuple or None, predicted seconds)."""
    if len(params) != AR_GENMODEL_TERMS:
        raise ValueError("%d parameters expected" % AR_GENMODEL_TERMS)
    pa = (c_double * AR_GENMODEL_TERMS)(*[float(x) for x in params])
    kind, lv = c_int32(), c_int32()
    fan = (c_int32 * max(1, int(max_levels)))()
    sec = c_double()
    _check(_lib.ar_genmodel_select(int(n), int(N), _dtype(dtype), pa, int(cache_bytes),
                                   int(max_levels), ctypes.byref(kind), ctypes.byref(lv),
                                   fan, ctypes.byref(sec)))
    name = {v: k for k, v in KINDS.items()}[kind.value]
    return name, (tuple(fan[i] for i in range(lv.value)) if lv.value else None), sec.value


# ---------------------------------------------------------------- timing

def ar_timer_create(capacity):
    out = _P()
    _check(_lib.ar_timer_create(int(capacity), ctypes.byref(out)))
    return out.value


def ar_timer_reset(timer):
    _check(_lib.ar_timer_reset(timer))


def ar_timer_read(timer, cap):
    """Returns a list of (launch index, ms) for up to ``cap`` records."""
    cnt = c_int64()
    ph = (c_int32 * max(1, cap))()
    ms = (c_float * max(1, cap))()
    _check(_lib.ar_timer_read(timer, int(cap), ctypes.byref(cnt), ph, ms))
    return [(ph[i], ms[i]) for i in range(cnt.value)]


def ar_timer_destroy(timer):
    _check(_lib.ar_timer_destroy(timer))


# ------------------------------------------------------------ convenience

class Plan:
    """Owning wrapper around a plan handle.  ``kind="gentree"`` takes the
    tree as ``fanin`` = child counts in preorder (``n`` is then ignored)."""

    def __init__(self, n, N, dtype, kind, fanin=None):
        if kind == "gentree":
            self.handle = ar_plan_create_gentree(N, dtype, fanin)
        else:
            self.handle = ar_plan_create(n, N, dtype, kind, fanin)
        self.n, self.N, self.dtype, self.num_phases, self.num_steps = \
            ar_plan_info(self.handle)
        self.esize = ESIZE[self.dtype]

    def _bufs(self, bufs):
        if len(bufs) != self.n:
            raise ValueError("plan has %d processors, got %d buffers" % (self.n, len(bufs)))
        return bufs

    def execute(self, bufs, stream=None):
        ar_plan_execute(self.handle, self._bufs(bufs), stream)

    def execute_noalloc(self, bufs, stream=None):
        ar_plan_execute_noalloc(self.handle, self._bufs(bufs), stream)

    def execute_strided(self, base, stride_bytes, stream=None):
        ar_plan_execute_strided(self.handle, base, stride_bytes, stream)

    def execute_timed(self, bufs, stream, timer):
        ar_plan_execute_timed(self.handle, self._bufs(bufs), stream, timer)

    def steps(self):
        return [ar_plan_get_step(self.handle, i) for i in range(self.num_steps)]

    def phases(self):
        """Steps grouped by phase, as (op_name, dst, srcs, begin, end)."""
        out = [[] for _ in range(self.num_phases)]
        for ph, op, dst, srcs, b, e in self.steps():
            out[ph].append(("reduce" if op == AR_OP_REDUCE else "copy", dst,
                            srcs, b, e))
        return out

    def phase_info(self, p):
        return ar_plan_phase_info(self.handle, p)

    def owner(self, p):
        return ar_plan_owner(self.handle, p)

    def bytes(self):
        return ar_plan_bytes(self.handle)

    def set_option(self, option, value):
        ar_plan_set_option(self.handle, option, value)

    def launches(self):
        """[(phase, nsrc, max_dst, num_steps, bytes)] per kernel launch; phase
        is the plan phase of a phase launch, -1 for a sliced launch, -2 for a
        resident one and -3 for a streamed resident one."""
        return [ar_plan_launch_info(self.handle, i)
                for i in range(ar_plan_num_launches(self.handle))]

    def launch_kernels(self):
        """Name of the kernel of each launch (on 16-byte aligned buffers)."""
        return [ar_plan_launch_kernel(self.handle, i)
                for i in range(ar_plan_num_launches(self.handle))]

    def close(self):
        if self.handle:
            ar_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()
