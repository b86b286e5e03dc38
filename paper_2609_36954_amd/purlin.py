"""Thin ctypes binding of libpurlin.so (include/purlin.h).

Argument marshalling only: every step of the datapath runs in the library's
HIP kernels.  PyTorch supplies device memory (``tensor.data_ptr()``) and the
stream (``torch.cuda.current_stream().cuda_stream``, a hipStream_t on ROCm).
There is no CPU fallback: if the library is missing, every call raises.

The functions keep the C names (``purlin_plan``, ``purlin_exec``, ...);
``Plan`` wraps a plan handle.
"""

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpurlin.so")

PURLIN_OK = 0
PURLIN_ERR_INVALID = 1
PURLIN_ERR_UNSUPPORTED = 2
PURLIN_ERR_NOMEM = 3
PURLIN_ERR_DEVICE = 4

OPS = {"allreduce": 0, "reduce_scatter": 1, "allgather": 2, "alltoall": 3,
       "broadcast": 4, "reduce": 5, "scatter": 6, "gather": 7,
       "allgatherv": 8, "reduce_scatterv": 9, "alltoallv": 10}
ROOTED = ("broadcast", "reduce", "scatter", "gather")
VOPS = ("allgatherv", "reduce_scatterv", "alltoallv")
DTYPES = {"fp32": 0, "bf16": 1}
ELEM_BYTES = {"fp32": 4, "bf16": 2}
KIND_COPY = 0
KIND_REDUCE = 1
PLAN_HOST_ONLY = 1
PLAN_COUNTS_TRANSPOSED = 2
PLAN_SHARE_PUSH = 4
MAX_RANKS = 16

# numpy view of purlin_desc (64 bytes, no padding)
DESC_DTYPE = np.dtype(
    [
        ("kind", "<u4"),
        ("phase", "<u4"),
        ("nsrc", "<u4"),
        ("src_buf", "<u4"),
        ("src_step", "<u4"),
        ("ndst", "<u4"),
        ("dst_buf", "<u4"),
        ("dst_step", "<u4"),
        ("src_off", "<u8"),
        ("dst_off", "<u8"),
        ("bytes", "<u8"),
        ("part", "<u4"),
        ("chunk", "<u4"),
    ]
)
assert DESC_DTYPE.itemsize == 64


class PurlinError(RuntimeError):
    def __init__(self, status, what=""):
        self.status = status
        super().__init__(f"{what}: purlin status {status} ({status_string(status)})" if what else status_string(status))


class Policy(ctypes.Structure):
    _fields_ = [
        ("item_bytes", ctypes.c_uint64),
        ("fanout", ctypes.c_uint32),
        ("ar_mode", ctypes.c_uint32),
        ("load_hint", ctypes.c_uint32),  # 0 auto, 1 cached, 2 non-temporal
        ("store_hint", ctypes.c_uint32),
        ("max_workgroups", ctypes.c_uint32),  # 0 = one wavefront per work item
        ("copy_depth", ctypes.c_uint32),  # 16-byte loads in flight per lane for copies (0 = auto)
        ("reserved", ctypes.c_uint32 * 3),
    ]


_lib = None
_c_u64p = ctypes.POINTER(ctypes.c_uint64)
_vp = ctypes.c_void_p


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise PurlinError(PURLIN_ERR_UNSUPPORTED, f"HIP library not built ({LIB_PATH}); run python -m paper_2609_36954_amd.build")
    L = ctypes.CDLL(LIB_PATH)
    i32, u32, u64 = ctypes.c_int, ctypes.c_uint32, ctypes.c_uint64
    L.purlin_plan.argtypes = [i32, i32, u64, i32, u64, ctypes.POINTER(_vp)]
    L.purlin_plan_ex.argtypes = [i32, i32, u64, i32, u64, ctypes.POINTER(Policy), u32, ctypes.POINTER(_vp)]
    L.purlin_plan_rooted.argtypes = [i32, i32, i32, u64, i32, u64, ctypes.POINTER(Policy), u32, ctypes.POINTER(_vp)]
    L.purlin_plan_v.argtypes = [i32, i32, u64, u64, i32, u64, u64, ctypes.POINTER(Policy), u32, ctypes.POINTER(_vp)]
    L.purlin_plan_share.argtypes = [i32, i32, i32, i32, u64, i32, u64, ctypes.POINTER(Policy), u32, ctypes.POINTER(_vp)]
    L.purlin_exec_v.argtypes = [_vp, ctypes.POINTER(_vp), _vp, _vp, _vp]
    L.purlin_plan_info.argtypes = [_vp, _c_u64p, _c_u64p, _c_u64p, _c_u64p]
    L.purlin_plan_descriptors.argtypes = [_vp, ctypes.POINTER(_vp), _c_u64p, _c_u64p]
    L.purlin_plan_items.argtypes = [_vp, ctypes.POINTER(_vp), _c_u64p, _c_u64p]
    L.purlin_exec.argtypes = [_vp, ctypes.POINTER(_vp), _vp]
    L.purlin_plan_device_error.argtypes = [_vp, ctypes.POINTER(ctypes.c_uint32)]
    L.purlin_plan_device_error.restype = ctypes.c_int
    L.purlin_plan_destroy.argtypes = [_vp]
    L.purlin_plan_destroy.restype = None
    L.purlin_pack_workspace_size.argtypes = [i32, i32, i32, _c_u64p]
    L.purlin_pack_single_launch.argtypes = [i32, i32, i32, i32, ctypes.POINTER(ctypes.c_int)]
    L.purlin_pack.argtypes = [i32, i32, i32, i32, i32] + [_vp] * 10 + [u64, _vp]
    L.purlin_pack_static.argtypes = [i32, i32, i32, i32, i32] + [_vp] * 10
    L.purlin_pack_meta.argtypes = [i32, i32, i32, i32] + [_vp] * 7 + [u64, _vp]
    L.purlin_pack_rows.argtypes = [i32, i32, i32, i32] + [_vp] * 5 + [u64, _vp]
    L.purlin_unpack.argtypes = [i32, i32, i32] + [_vp] * 6
    L.purlin_pack_dedup_workspace_size.argtypes = [i32, i32, _c_u64p]
    L.purlin_pack_dedup.argtypes = [i32, i32, i32, i32, i32] + [_vp] * 8 + [u64, _vp]
    L.purlin_unpack_dedup.argtypes = [i32, i32, i32, ctypes.c_int64] + [_vp] * 5
    _pa = ctypes.POINTER(_vp)
    L.purlin_ep_dispatch_workspace_size.argtypes = [i32, i32, i32, i32, _c_u64p]
    L.purlin_ep_dispatch.argtypes = [i32] * 5 + [_pa, _pa, _pa, u64, _vp, _vp, _vp, _vp, u64, _vp]
    L.purlin_ep_combine.argtypes = [i32] * 5 + [_pa, u64, _pa, _vp, _pa, _pa, _vp, _vp]
    L.purlin_ep_dispatch_dedup_workspace_size.argtypes = [i32, i32, _c_u64p]
    L.purlin_ep_dispatch_dedup.argtypes = [i32] * 5 + [_pa, _pa, _pa, u64, _vp, _vp, _vp, _vp, u64, _vp]
    L.purlin_ep_combine_dedup.argtypes = [i32] * 3 + [_pa, u64, _vp, _pa, _vp, _vp]
    L.purlin_stream_copy.argtypes = [_vp, _vp, u64, _vp]
    L.purlin_stream.argtypes = [ctypes.POINTER(_vp), i32, ctypes.POINTER(_vp), i32, u64, _vp, u32, _vp]
    L.purlin_stream_timed.argtypes = [ctypes.POINTER(_vp), i32, ctypes.POINTER(_vp), i32, u64, _vp, u32, _vp, u64,
                                      _c_u64p, _vp]
    L.purlin_pack_timed.argtypes = [i32, i32, i32, i32, i32] + [_vp] * 10 + [u64, _c_u64p, _vp]
    L.purlin_status_string.argtypes = [i32]
    L.purlin_status_string.restype = ctypes.c_char_p
    L.purlin_version.argtypes = []
    L.purlin_version.restype = ctypes.c_char_p
    for name in ("purlin_plan", "purlin_plan_ex", "purlin_plan_rooted", "purlin_plan_v", "purlin_plan_share",
                 "purlin_exec_v",
                 "purlin_plan_info", "purlin_plan_descriptors", "purlin_plan_items",
                 "purlin_exec", "purlin_pack_workspace_size", "purlin_pack_single_launch", "purlin_pack", "purlin_unpack",
                 "purlin_pack_dedup_workspace_size", "purlin_pack_dedup", "purlin_unpack_dedup",
                 "purlin_ep_dispatch_workspace_size", "purlin_ep_dispatch", "purlin_ep_combine",
                 "purlin_ep_dispatch_dedup_workspace_size", "purlin_ep_dispatch_dedup", "purlin_ep_combine_dedup",
                 "purlin_stream_copy", "purlin_stream_timed", "purlin_pack_timed"):
        getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def status_string(status):
    if _lib is None and not os.path.exists(LIB_PATH):
        return f"status {status}"
    return lib().purlin_status_string(int(status)).decode()


purlin_status_string = status_string


def purlin_version():
    return lib().purlin_version().decode()


def _check(status, what):
    if status != PURLIN_OK:
        raise PurlinError(status, what)


def _stream_handle(stream):
    import torch

    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream))


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _require_cuda(t, name, itemsize=None):
    if not t.is_cuda:
        raise PurlinError(PURLIN_ERR_INVALID, f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise PurlinError(PURLIN_ERR_INVALID, f"{name} must be contiguous")
    if itemsize is not None and t.element_size() != itemsize:
        raise PurlinError(PURLIN_ERR_INVALID, f"{name} must have {itemsize}-byte elements")


class Plan:
    """A planned collective (immutable).  ``exec`` runs it on a stream."""

    def __init__(self, op, P, count, dtype, chunk, policy=None, host_only=False, root=None, unit=None,
                 out_capacity=None, counts_transposed=False, share=None, push=False):
        if op not in OPS:
            raise PurlinError(PURLIN_ERR_INVALID, f"unknown op {op!r}")
        if dtype not in DTYPES:
            raise PurlinError(PURLIN_ERR_INVALID, f"unknown dtype {dtype!r}")
        if (op in ROOTED) != (root is not None):
            raise PurlinError(PURLIN_ERR_INVALID, f"{op} {'needs' if op in ROOTED else 'takes no'} root")
        self.op, self.P, self.count, self.dtype, self.chunk = op, int(P), int(count), dtype, int(chunk)
        self.root = root
        self.unit = unit
        self.host_only = bool(host_only)
        self.share = share
        self.push = bool(push)
        self._used = None
        if push and share is None:
            raise PurlinError(PURLIN_ERR_INVALID, "push applies to a rank's share")
        if share is not None and op in VOPS:
            raise PurlinError(PURLIN_ERR_INVALID, f"{op} has no rank shares")
        if (op in VOPS) != (unit is not None):
            raise PurlinError(PURLIN_ERR_INVALID, f"{op} {'needs' if op in VOPS else 'takes no'} unit")
        h = ctypes.c_void_p()
        L = lib()
        if unit is not None:
            pol = None
            if policy is not None:
                pol = policy if isinstance(policy, Policy) else Policy(**policy)
            out_cap = int(count) if out_capacity is None else int(out_capacity)
            flags = (PLAN_HOST_ONLY if host_only else 0) | (PLAN_COUNTS_TRANSPOSED if counts_transposed else 0)
            st = L.purlin_plan_v(OPS[op], int(P), int(count), out_cap, DTYPES[dtype], int(chunk), int(unit),
                                 ctypes.byref(pol) if pol is not None else None, flags, ctypes.byref(h))
        elif share is not None:
            pol = None
            if policy is not None:
                pol = policy if isinstance(policy, Policy) else Policy(**policy)
            flags = (PLAN_HOST_ONLY if host_only else 0) | (PLAN_SHARE_PUSH if push else 0)
            st = L.purlin_plan_share(OPS[op], int(P), -1 if root is None else int(root), int(share), int(count),
                                     DTYPES[dtype], int(chunk), ctypes.byref(pol) if pol is not None else None,
                                     flags, ctypes.byref(h))
        elif root is not None:
            pol = None
            if policy is not None:
                pol = policy if isinstance(policy, Policy) else Policy(**policy)
            st = L.purlin_plan_rooted(OPS[op], int(P), int(root), int(count), DTYPES[dtype], int(chunk),
                                      ctypes.byref(pol) if pol is not None else None,
                                      PLAN_HOST_ONLY if host_only else 0, ctypes.byref(h))
        elif policy is None and not host_only:
            st = L.purlin_plan(OPS[op], int(P), int(count), DTYPES[dtype], int(chunk), ctypes.byref(h))
        else:
            pol = None
            if policy is not None:
                pol = policy if isinstance(policy, Policy) else Policy(**policy)
            st = L.purlin_plan_ex(OPS[op], int(P), int(count), DTYPES[dtype], int(chunk),
                                  ctypes.byref(pol) if pol is not None else None,
                                  PLAN_HOST_ONLY if host_only else 0, ctypes.byref(h))
        _check(st, "purlin_plan")
        self._h = h
        info = self.info()
        self.n_desc = info["n_desc"]
        self.in_bytes = info["in_bytes_per_rank"]
        self.out_bytes = info["out_bytes_per_rank"]
        self.sched_bytes = info["sched_bytes"]

    @property
    def handle(self):
        if self._h is None:
            raise PurlinError(PURLIN_ERR_INVALID, "plan destroyed")
        return self._h

    def info(self):
        vals = [ctypes.c_uint64() for _ in range(4)]
        _check(lib().purlin_plan_info(self.handle, *[ctypes.byref(v) for v in vals]), "purlin_plan_info")
        return dict(zip(("n_desc", "in_bytes_per_rank", "out_bytes_per_rank", "sched_bytes"), (v.value for v in vals)))

    def descriptors(self):
        """Copy of the chunk descriptor table as a structured numpy array."""
        p, n, stride = ctypes.c_void_p(), ctypes.c_uint64(), ctypes.c_uint64()
        _check(lib().purlin_plan_descriptors(self.handle, ctypes.byref(p), ctypes.byref(n), ctypes.byref(stride)),
               "purlin_plan_descriptors")
        assert stride.value == DESC_DTYPE.itemsize
        return self._copy_table(p, n.value)

    def items(self):
        """(work items as a structured array, [phase0_begin, phase1_begin, n])."""
        p, n = ctypes.c_void_p(), ctypes.c_uint64()
        pb = (ctypes.c_uint64 * 3)()
        _check(lib().purlin_plan_items(self.handle, ctypes.byref(p), ctypes.byref(n), pb), "purlin_plan_items")
        return self._copy_table(p, n.value), list(pb)

    @staticmethod
    def _copy_table(p, n):
        if n == 0:
            return np.zeros(0, dtype=DESC_DTYPE)
        buf = (ctypes.c_char * (n * DESC_DTYPE.itemsize)).from_address(p.value)
        return np.frombuffer(bytes(buf), dtype=DESC_DTYPE).copy()

    def device_error(self):
        """Device error word (single-launch AllReduce plans); synchronises."""
        e = ctypes.c_uint32()
        _check(lib().purlin_plan_device_error(self.handle, ctypes.byref(e)), "purlin_plan_device_error")
        return e.value

    def exec(self, ins, outs, stream=None):
        """Run on device tensors ``ins`` (P inputs) and ``outs`` (P outputs)."""
        purlin_exec(self, ins, outs, stream)

    def exec_v(self, ins, outs, counts, dev_status=None, stream=None):
        """Run a variable-size plan; ``counts`` is a device int32 tensor."""
        purlin_exec_v(self, ins, outs, counts, dev_status, stream)

    def bind(self, ins, outs, counts=None, dev_status=None, stream=None):
        """Validate the buffers once and return a callable that enqueues the
        plan on them (on ``stream``, default: the current stream at bind
        time) with no further Python-side work: for serving loops that run
        the same collective on the same buffers."""
        return BoundExec(self, ins, outs, counts, dev_status, stream)

    def destroy(self):
        if getattr(self, "_h", None) is not None and _lib is not None:
            _lib.purlin_plan_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


class BoundExec:
    """A plan bound to fixed buffers and a stream (see ``Plan.bind``).  It
    keeps references to the tensors, so they outlive it."""

    def __init__(self, plan, ins, outs, counts=None, dev_status=None, stream=None):
        self._plan = plan
        self._keep = (list(ins), list(outs), counts, dev_status)
        L = lib()
        if plan.unit is not None:
            if counts is None:
                raise PurlinError(PURLIN_ERR_INVALID, "a variable-size plan needs counts")
            _require_cuda(counts, "counts", 4)
            need = plan.P * plan.P if plan.op == "alltoallv" else plan.P
            if counts.numel() < need:
                raise PurlinError(PURLIN_ERR_INVALID, f"{plan.op} needs {need} counts")
            arr = _buffer_array(plan, ins, outs)
            args = (plan.handle, arr, _ptr(counts), _ptr(dev_status), _stream_handle(stream))
            self._fn, self._args = L.purlin_exec_v, args
        else:
            if counts is not None:
                raise PurlinError(PURLIN_ERR_INVALID, "counts are for variable-size plans")
            if plan.count:
                arr = _buffer_array(plan, ins, outs)
            else:
                arr = (ctypes.c_void_p * (2 * plan.P))()
            self._fn, self._args = L.purlin_exec, (plan.handle, arr, _stream_handle(stream) if plan.count else None)

    def __call__(self):
        st = self._fn(*self._args)
        if st:
            _check(st, "purlin_exec")


def purlin_plan(op, P, count, dtype, chunk, policy=None, host_only=False):
    return Plan(op, P, count, dtype, chunk, policy=policy, host_only=host_only)


def purlin_plan_rooted(op, P, root, count, dtype, chunk, policy=None, host_only=False):
    return Plan(op, P, count, dtype, chunk, policy=policy, host_only=host_only, root=root)


def used_buffers(plan):
    """(inputs used, outputs used) as lists of booleans, rank order."""
    P, op, root = plan.P, plan.op, plan.root
    if getattr(plan, "share", None) is not None:  # the buffers its descriptors name
        if plan._used is None:
            ins, outs = [False] * P, [False] * P
            for d in plan.descriptors():
                for j in range(int(d["nsrc"])):
                    b = int(d["src_buf"]) + j * int(d["src_step"])
                    (ins if b < P else outs)[b % P] = True
                for j in range(int(d["ndst"])):
                    outs[int(d["dst_buf"]) + j * int(d["dst_step"]) - P] = True
            plan._used = (ins, outs)
        return plan._used
    ins = [True] * P
    outs = [True] * P
    if op in ("broadcast", "scatter"):
        ins = [r == root for r in range(P)]
    if op in ("reduce", "gather"):
        outs = [r == root for r in range(P)]
    return ins, outs


def purlin_plan_v(op, P, in_capacity, dtype, chunk, unit=1, out_capacity=None, policy=None, host_only=False,
                  counts_transposed=False):
    """Variable-size plan; ``in_capacity``/``out_capacity`` in elements
    (``out_capacity`` defaults to ``in_capacity``).  ``counts_transposed``
    (alltoallv): the P x P sizes are read column-major."""
    return Plan(op, P, in_capacity, dtype, chunk, policy=policy, host_only=host_only, unit=unit,
                out_capacity=out_capacity, counts_transposed=counts_transposed)


def _buffer_array(plan, ins, outs):
    P = plan.P
    if len(ins) != P or len(outs) != P:
        raise PurlinError(PURLIN_ERR_INVALID, f"need {P} inputs and {P} outputs")
    use_in, use_out = used_buffers(plan)
    s = ELEM_BYTES[plan.dtype]
    for t, u in zip(ins, use_in):
        if u:
            _require_cuda(t, "input", s)
            if t.numel() * s < plan.in_bytes:
                raise PurlinError(PURLIN_ERR_INVALID, "input buffer too small")
    for t, u in zip(outs, use_out):
        if u:
            _require_cuda(t, "output", s)
            if t.numel() * s < plan.out_bytes:
                raise PurlinError(PURLIN_ERR_INVALID, "output buffer too small")
    return (ctypes.c_void_p * (2 * P))(*[(t.data_ptr() if t is not None else 0) for t in list(ins) + list(outs)])


def purlin_exec_v(plan, ins, outs, counts, dev_status=None, stream=None):
    """Variable-size collective; ``counts``: device int32 tensor (P, or P*P
    row-major for alltoallv), in units of the plan's ``unit`` elements."""
    _require_cuda(counts, "counts", 4)
    need = plan.P * plan.P if plan.op == "alltoallv" else plan.P
    if counts.numel() < need:
        raise PurlinError(PURLIN_ERR_INVALID, f"{plan.op} needs {need} counts")
    arr = _buffer_array(plan, ins, outs)
    _check(lib().purlin_exec_v(plan.handle, arr, _ptr(counts), _ptr(dev_status), _stream_handle(stream)),
           "purlin_exec_v")


def purlin_exec(plan, ins, outs, stream=None):
    """``ins``/``outs``: P device tensors each; for a rooted plan, entries of
    buffers it does not use may be None."""
    P = plan.P
    if len(ins) != P or len(outs) != P:
        raise PurlinError(PURLIN_ERR_INVALID, f"need {P} inputs and {P} outputs")
    use_in, use_out = used_buffers(plan)
    if plan.count:
        s = ELEM_BYTES[plan.dtype]
        for t, u in zip(ins, use_in):
            if not u:
                continue
            _require_cuda(t, "input", s)
            if t.numel() * s < plan.in_bytes:
                raise PurlinError(PURLIN_ERR_INVALID, "input buffer too small")
        for t, u in zip(outs, use_out):
            if not u:
                continue
            _require_cuda(t, "output", s)
            if t.numel() * s < plan.out_bytes:
                raise PurlinError(PURLIN_ERR_INVALID, "output buffer too small")
    arr = (ctypes.c_void_p * (2 * P))(*[(t.data_ptr() if t is not None else 0) for t in list(ins) + list(outs)])
    _check(lib().purlin_exec(plan.handle, arr, _stream_handle(stream) if plan.count else None), "purlin_exec")


def _check_sizes(tensors, shapes):
    """Every output the kernels write must be a contiguous device tensor
    with at least as many elements of the right size as its shape holds."""
    for name, (shape, dt) in shapes.items():
        t = tensors[name]
        need = int(np.prod(shape))
        _require_cuda(t, name, 2 if name == "packed" else 4)
        if t.numel() < need:
            raise PurlinError(PURLIN_ERR_INVALID, f"{name} holds {t.numel()} elements, needs {need}")


def purlin_pack_workspace_size(T, K, E):
    b = ctypes.c_uint64()
    _check(lib().purlin_pack_workspace_size(int(T), int(K), int(E), ctypes.byref(b)), "purlin_pack_workspace_size")
    return b.value


def purlin_pack_single_launch(T, H, K, E):
    """True when ``purlin_pack`` runs in one launch for this shape."""
    v = ctypes.c_int(0)
    _check(lib().purlin_pack_single_launch(int(T), int(H), int(K), int(E), ctypes.byref(v)),
           "purlin_pack_single_launch")
    return bool(v.value)


def purlin_pack(x, ids, E, P, out=None, workspace=None, dev_status=None, stream=None):
    """MoE dispatch of ``x`` (bf16 [T, H]) by ``ids`` (int32 [T, K]).

    Returns a dict of device tensors: packed [T*K, H], dest_counts [P],
    dest_offsets [P], expert_counts [E], expert_offsets [E], pos [T, K].
    ``out`` may supply preallocated tensors under the same keys.
    """
    import torch

    T, H = x.shape
    K = ids.shape[1]
    if ids.shape[0] != T:
        raise PurlinError(PURLIN_ERR_INVALID, "x and ids disagree on T")
    _require_cuda(x, "x", 2)
    _require_cuda(ids, "ids", 4)
    dev = x.device
    o = dict(out or {})
    shapes = {"packed": ((T * K, H), x.dtype), "dest_counts": ((P,), torch.int32), "dest_offsets": ((P,), torch.int32),
              "expert_counts": ((E,), torch.int32), "expert_offsets": ((E,), torch.int32),
              "pos": ((T, K), torch.int32)}
    for name, (shape, dt) in shapes.items():
        if name not in o:  # allocate only what the caller did not supply
            o[name] = torch.empty(shape, dtype=dt, device=dev)
    _check_sizes(o, shapes)
    wsb = purlin_pack_workspace_size(T, K, E)
    if workspace is None:
        workspace = torch.empty(max(wsb, 16), dtype=torch.uint8, device=dev)
    st = lib().purlin_pack(int(T), int(H), int(K), int(E), int(P), _ptr(x), _ptr(ids), _ptr(o["packed"]),
                           _ptr(o["dest_counts"]), _ptr(o["dest_offsets"]), _ptr(o["expert_counts"]),
                           _ptr(o["expert_offsets"]), _ptr(o["pos"]), _ptr(dev_status), _ptr(workspace),
                           int(workspace.numel() * workspace.element_size()), _stream_handle(stream))
    _check(st, "purlin_pack")
    return o


def purlin_pack_meta(ids, E, P, out, workspace, dev_status=None, stream=None):
    """The metadata half of ``purlin_pack``: fills ``out``'s dest_counts,
    dest_offsets, expert_counts and expert_offsets (and ``dev_status``) and
    leaves the row positions' inputs in ``workspace``."""
    import torch

    T, K = ids.shape
    if T:
        _require_cuda(ids, "ids", 4)
    shapes = {"dest_counts": ((P,), torch.int32), "dest_offsets": ((P,), torch.int32),
              "expert_counts": ((E,), torch.int32), "expert_offsets": ((E,), torch.int32)}
    _check_sizes(out, shapes)
    st = lib().purlin_pack_meta(int(T), int(K), int(E), int(P), _ptr(ids), _ptr(out["dest_counts"]),
                                _ptr(out["dest_offsets"]), _ptr(out["expert_counts"]), _ptr(out["expert_offsets"]),
                                _ptr(dev_status), _ptr(workspace), int(workspace.numel() * workspace.element_size()),
                                _stream_handle(stream))
    _check(st, "purlin_pack_meta")
    return out


def purlin_pack_rows(x, ids, E, out, workspace, stream=None):
    """The rows half of ``purlin_pack`` (after ``purlin_pack_meta`` on the
    same workspace has finished): fills ``out``'s packed and pos."""
    import torch

    T, H = x.shape
    K = ids.shape[1]
    if ids.shape[0] != T:
        raise PurlinError(PURLIN_ERR_INVALID, "x and ids disagree on T")
    _require_cuda(x, "x", 2)
    _require_cuda(ids, "ids", 4)
    _check_sizes(out, {"packed": ((T * K, H), x.dtype), "pos": ((T, K), torch.int32)})
    st = lib().purlin_pack_rows(int(T), int(H), int(K), int(E), _ptr(x), _ptr(ids), _ptr(out["packed"]),
                                _ptr(out["pos"]), _ptr(workspace), int(workspace.numel() * workspace.element_size()),
                                _stream_handle(stream))
    _check(st, "purlin_pack_rows")
    return out


def purlin_pack_static(x, ids, E, P, out, dev_status=None, stream=None):
    """``purlin_pack`` through the entry point that allocates nothing: its
    workspace is the library's per-GPU array.  ``out`` must supply every
    output tensor (keys as returned by ``purlin_pack``)."""
    T, H = x.shape
    K = ids.shape[1]
    if ids.shape[0] != T:
        raise PurlinError(PURLIN_ERR_INVALID, "x and ids disagree on T")
    _require_cuda(x, "x", 2)
    _require_cuda(ids, "ids", 4)
    import torch

    shapes = {"packed": ((T * K, H), x.dtype), "dest_counts": ((P,), torch.int32), "dest_offsets": ((P,), torch.int32),
              "expert_counts": ((E,), torch.int32), "expert_offsets": ((E,), torch.int32),
              "pos": ((T, K), torch.int32)}
    missing = [name for name in shapes if name not in out]
    if missing:
        raise PurlinError(PURLIN_ERR_INVALID, f"out lacks {', '.join(missing)}")
    _check_sizes(out, shapes)
    st = lib().purlin_pack_static(int(T), int(H), int(K), int(E), int(P), _ptr(x), _ptr(ids), _ptr(out["packed"]),
                                  _ptr(out["dest_counts"]), _ptr(out["dest_offsets"]), _ptr(out["expert_counts"]),
                                  _ptr(out["expert_offsets"]), _ptr(out["pos"]), _ptr(dev_status),
                                  _stream_handle(stream))
    _check(st, "purlin_pack_static")
    return out


def purlin_unpack(y, pos, gates, out=None, dev_status=None, stream=None):
    """MoE combine: bf16 [T, H] = sum_k gates[t, k] * y[pos[t, k]] in slot order."""
    import torch

    T, K = pos.shape
    H = y.shape[1]
    _require_cuda(y, "y", 2)
    _require_cuda(pos, "pos", 4)
    _require_cuda(gates, "gates", 4)
    if gates.dtype != torch.float32:
        raise PurlinError(PURLIN_ERR_INVALID, "gates must be float32")
    if y.shape[0] < T * K or gates.numel() < T * K:
        raise PurlinError(PURLIN_ERR_INVALID, "y needs T*K rows and gates T*K entries")
    if out is None:
        out = torch.empty((T, H), dtype=y.dtype, device=y.device)
    _require_cuda(out, "out", 2)
    if out.numel() < T * H:
        raise PurlinError(PURLIN_ERR_INVALID, "out holds fewer than T*H elements")
    st = lib().purlin_unpack(int(T), int(H), int(K), _ptr(y), _ptr(pos), _ptr(gates), _ptr(out), _ptr(dev_status),
                             _stream_handle(stream))
    _check(st, "purlin_unpack")
    return out


def purlin_pack_dedup_workspace_size(T, P):
    b = ctypes.c_uint64()
    _check(lib().purlin_pack_dedup_workspace_size(int(T), int(P), ctypes.byref(b)),
           "purlin_pack_dedup_workspace_size")
    return b.value


def purlin_pack_dedup(x, ids, E, P, out=None, workspace=None, dev_status=None, stream=None):
    """De-duplicated MoE dispatch of ``x`` (bf16 [T, H]) by ``ids`` (int32
    [T, K]): one row per (token, destination rank).

    Returns a dict of device tensors: packed [T*min(K, P), H] (the first
    sum(dest_counts) rows written), dest_counts [P], dest_offsets [P],
    row_of [T, P].  ``out`` may supply preallocated tensors under the same
    keys.
    """
    import torch

    T, H = x.shape
    K = ids.shape[1]
    if ids.shape[0] != T:
        raise PurlinError(PURLIN_ERR_INVALID, "x and ids disagree on T")
    _require_cuda(x, "x", 2)
    _require_cuda(ids, "ids", 4)
    dev = x.device
    o = dict(out or {})
    shapes = {"packed": ((T * min(K, P), H), x.dtype), "dest_counts": ((P,), torch.int32),
              "dest_offsets": ((P,), torch.int32), "row_of": ((T, P), torch.int32)}
    for name, (shape, dt) in shapes.items():
        if name not in o:  # allocate only what the caller did not supply
            o[name] = torch.empty(shape, dtype=dt, device=dev)
    _check_sizes(o, shapes)
    wsb = purlin_pack_dedup_workspace_size(T, P)
    if workspace is None:
        workspace = torch.empty(max(wsb, 16), dtype=torch.uint8, device=dev)
    st = lib().purlin_pack_dedup(int(T), int(H), int(K), int(E), int(P), _ptr(x), _ptr(ids), _ptr(o["packed"]),
                                 _ptr(o["dest_counts"]), _ptr(o["dest_offsets"]), _ptr(o["row_of"]),
                                 _ptr(dev_status), _ptr(workspace), int(workspace.numel() * workspace.element_size()),
                                 _stream_handle(stream))
    _check(st, "purlin_pack_dedup")
    return o


def purlin_unpack_dedup(y, row_of, out=None, dev_status=None, stream=None):
    """Combine of the de-duplicated dispatch: bf16 [T, H] = sum over ranks r
    (ascending) of y[row_of[t, r]], skipping -1 entries."""
    import torch

    T, P = row_of.shape
    rows, H = y.shape
    _require_cuda(y, "y", 2)
    _require_cuda(row_of, "row_of", 4)
    if out is None:
        out = torch.empty((T, H), dtype=y.dtype, device=y.device)
    _require_cuda(out, "out", 2)
    if out.numel() < T * H:
        raise PurlinError(PURLIN_ERR_INVALID, "out holds fewer than T*H elements")
    st = lib().purlin_unpack_dedup(int(T), int(H), int(P), int(rows), _ptr(y), _ptr(row_of), _ptr(out),
                                   _ptr(dev_status), _stream_handle(stream))
    _check(st, "purlin_unpack_dedup")
    return out


def _ptr_array(tensors):
    return (ctypes.c_void_p * len(tensors))(*[t.data_ptr() for t in tensors])


def _rows_capacity(bufs, H, name):
    for b in bufs:
        _require_cuda(b, name, 2)
    return min(b.numel() for b in bufs) // H


def purlin_ep_dispatch_workspace_size(T, K, E, P):
    b = ctypes.c_uint64()
    _check(lib().purlin_ep_dispatch_workspace_size(int(T), int(K), int(E), int(P), ctypes.byref(b)),
           "purlin_ep_dispatch_workspace_size")
    return b.value


def purlin_ep_dispatch(xs, idss, E, recv, counts=None, recv_pos=None, workspace=None, dev_status=None, stream=None):
    """Expert-parallel dispatch over P = len(xs) ranks in one pass: rank p's
    pack followed by the AllToAllV of the packed rows, written straight into
    the receive buffers ``recv`` (P bf16 tensors of ``capacity`` rows of H).

    Returns a dict with ``counts`` (int32 [P*P], rows rank p sends rank r at
    p*P + r) and ``recv_pos`` (int32 [P, T, K]).
    """
    import torch

    P = len(xs)
    if len(idss) != P or len(recv) != P:
        raise PurlinError(PURLIN_ERR_INVALID, "need P token matrices, P id matrices and P receive buffers")
    T, H = xs[0].shape
    K = idss[0].shape[1]
    for x, ids in zip(xs, idss):
        _require_cuda(x, "x", 2)
        _require_cuda(ids, "ids", 4)
        if tuple(x.shape) != (T, H) or tuple(ids.shape) != (T, K):
            raise PurlinError(PURLIN_ERR_INVALID, "every rank needs x [T, H] and ids [T, K]")
    capacity = _rows_capacity(recv, H, "recv")
    dev = xs[0].device
    if counts is None:
        counts = torch.empty(P * P, dtype=torch.int32, device=dev)
    if recv_pos is None:
        recv_pos = torch.empty((P, T, K), dtype=torch.int32, device=dev)
    _require_cuda(counts, "counts", 4)
    _require_cuda(recv_pos, "recv_pos", 4)
    if counts.numel() < P * P or recv_pos.numel() < P * T * K:
        raise PurlinError(PURLIN_ERR_INVALID, "counts needs P*P entries and recv_pos P*T*K")
    wsb = purlin_ep_dispatch_workspace_size(T, K, E, P)
    if workspace is None:
        workspace = torch.empty(max(wsb, 16), dtype=torch.uint8, device=dev)
    st = lib().purlin_ep_dispatch(int(T), int(H), int(K), int(E), int(P), _ptr_array(xs), _ptr_array(idss),
                                  _ptr_array(recv), int(capacity), _ptr(counts), _ptr(recv_pos), _ptr(dev_status),
                                  _ptr(workspace), int(workspace.numel() * workspace.element_size()),
                                  _stream_handle(stream))
    _check(st, "purlin_ep_dispatch")
    return {"counts": counts, "recv_pos": recv_pos}


def purlin_ep_combine(ys, idss, recv_pos, gatess, E, outs=None, dev_status=None, stream=None):
    """The matching combine: P expert-output tensors ``ys`` in the receive
    layout -> P bf16 [T, H] outputs, each slot's output weighted by its gate
    and summed in slot order (as ``purlin_unpack``)."""
    import torch

    P = len(ys)
    if len(idss) != P or len(gatess) != P:
        raise PurlinError(PURLIN_ERR_INVALID, "need P expert outputs, P id matrices and P gate matrices")
    T, K = idss[0].shape
    H = ys[0].shape[-1]
    capacity = _rows_capacity(ys, H, "y")
    for ids, g in zip(idss, gatess):
        _require_cuda(ids, "ids", 4)
        _require_cuda(g, "gates", 4)
        if g.dtype != torch.float32 or tuple(ids.shape) != (T, K) or g.numel() < T * K:
            raise PurlinError(PURLIN_ERR_INVALID, "every rank needs ids [T, K] and float32 gates [T, K]")
    _require_cuda(recv_pos, "recv_pos", 4)
    if recv_pos.numel() < P * T * K:
        raise PurlinError(PURLIN_ERR_INVALID, "recv_pos needs P*T*K entries")
    if outs is None:
        outs = [torch.empty((T, H), dtype=ys[0].dtype, device=ys[0].device) for _ in range(P)]
    for o in outs:
        _require_cuda(o, "out", 2)
        if o.numel() < T * H:
            raise PurlinError(PURLIN_ERR_INVALID, "every output needs T*H elements")
    st = lib().purlin_ep_combine(int(T), int(H), int(K), int(E), int(P), _ptr_array(ys), int(capacity),
                                 _ptr_array(idss), _ptr(recv_pos), _ptr_array(gatess), _ptr_array(outs),
                                 _ptr(dev_status), _stream_handle(stream))
    _check(st, "purlin_ep_combine")
    return outs


def purlin_ep_dispatch_dedup_workspace_size(T, P):
    b = ctypes.c_uint64()
    _check(lib().purlin_ep_dispatch_dedup_workspace_size(int(T), int(P), ctypes.byref(b)),
           "purlin_ep_dispatch_dedup_workspace_size")
    return b.value


def purlin_ep_dispatch_dedup(xs, idss, E, recv, counts=None, recv_row=None, workspace=None, dev_status=None,
                             stream=None):
    """De-duplicated dispatch over P = len(xs) ranks in one pass: one row per
    token and owning rank, written straight into the receive buffers.

    Returns a dict with ``counts`` (int32 [P*P]) and ``recv_row`` (int32
    [P, T, P], -1 where a token has no expert on a rank)."""
    import torch

    P = len(xs)
    if len(idss) != P or len(recv) != P:
        raise PurlinError(PURLIN_ERR_INVALID, "need P token matrices, P id matrices and P receive buffers")
    T, H = xs[0].shape
    K = idss[0].shape[1]
    for x, ids in zip(xs, idss):
        _require_cuda(x, "x", 2)
        _require_cuda(ids, "ids", 4)
        if tuple(x.shape) != (T, H) or tuple(ids.shape) != (T, K):
            raise PurlinError(PURLIN_ERR_INVALID, "every rank needs x [T, H] and ids [T, K]")
    capacity = _rows_capacity(recv, H, "recv")
    dev = xs[0].device
    if counts is None:
        counts = torch.empty(P * P, dtype=torch.int32, device=dev)
    if recv_row is None:
        recv_row = torch.empty((P, T, P), dtype=torch.int32, device=dev)
    _require_cuda(counts, "counts", 4)
    _require_cuda(recv_row, "recv_row", 4)
    if counts.numel() < P * P or recv_row.numel() < P * T * P:
        raise PurlinError(PURLIN_ERR_INVALID, "counts needs P*P entries and recv_row P*T*P")
    wsb = purlin_ep_dispatch_dedup_workspace_size(T, P)
    if workspace is None:
        workspace = torch.empty(max(wsb, 16), dtype=torch.uint8, device=dev)
    st = lib().purlin_ep_dispatch_dedup(int(T), int(H), int(K), int(E), int(P), _ptr_array(xs), _ptr_array(idss),
                                        _ptr_array(recv), int(capacity), _ptr(counts), _ptr(recv_row),
                                        _ptr(dev_status), _ptr(workspace),
                                        int(workspace.numel() * workspace.element_size()), _stream_handle(stream))
    _check(st, "purlin_ep_dispatch_dedup")
    return {"counts": counts, "recv_row": recv_row}


def purlin_ep_combine_dedup(ys, recv_row, outs=None, dev_status=None, stream=None):
    """Its combine: rank-order sum of every rank's partial output row."""
    import torch

    P = len(ys)
    T = recv_row.shape[1]
    H = ys[0].shape[-1]
    capacity = _rows_capacity(ys, H, "y")
    _require_cuda(recv_row, "recv_row", 4)
    if recv_row.numel() < P * T * P:
        raise PurlinError(PURLIN_ERR_INVALID, "recv_row needs P*T*P entries")
    if outs is None:
        outs = [torch.empty((T, H), dtype=ys[0].dtype, device=ys[0].device) for _ in range(P)]
    for o in outs:
        _require_cuda(o, "out", 2)
        if o.numel() < T * H:
            raise PurlinError(PURLIN_ERR_INVALID, "every output needs T*H elements")
    st = lib().purlin_ep_combine_dedup(int(T), int(H), int(P), _ptr_array(ys), int(capacity), _ptr(recv_row),
                                       _ptr_array(outs), _ptr(dev_status), _stream_handle(stream))
    _check(st, "purlin_ep_combine_dedup")
    return outs


def purlin_stream_copy(dst, src, stream=None):
    """Plain copy of ``src``'s bytes into ``dst`` (the reference stream the
    executor's copies are measured against; not a step of the method)."""
    _require_cuda(src, "src")
    _require_cuda(dst, "dst")
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() < nbytes:
        raise PurlinError(PURLIN_ERR_INVALID, "dst is smaller than src")
    st = lib().purlin_stream_copy(_ptr(dst), _ptr(src), int(nbytes), _stream_handle(stream))
    _check(st, "purlin_stream_copy")
    return dst


def purlin_stream(dsts, srcs, nbytes=None, sink=None, nt_load=False, nt_store=False, stream=None):
    """Reference stream: every destination receives the XOR of the sources,
    16 bytes at a time (no sources: a counting pattern; no destinations:
    read only, ``sink`` a 16-byte device tensor; ``nt_load`` / ``nt_store``:
    non-temporal loads / stores).  Not a step of the method:
    the access mixes the executor's kernels are measured against."""
    for t in list(dsts) + list(srcs) + ([sink] if sink is not None else []):
        _require_cuda(t, "stream buffer")
    if nbytes is None:
        nbytes = min(t.numel() * t.element_size() for t in list(dsts) + list(srcs))
    for t in list(dsts) + list(srcs):
        if t.numel() * t.element_size() < nbytes:
            raise PurlinError(PURLIN_ERR_INVALID, "a stream buffer is smaller than nbytes")
    d = (_vp * max(1, len(dsts)))(*[t.data_ptr() for t in dsts])
    s = (_vp * max(1, len(srcs)))(*[t.data_ptr() for t in srcs])
    hints = (1 if nt_load else 0) | (2 if nt_store else 0)
    st = lib().purlin_stream(d, len(dsts), s, len(srcs), int(nbytes), _ptr(sink), hints, _stream_handle(stream))
    _check(st, "purlin_stream")


def _timed_records(rec, groups):
    """Host copy of a timing record: (rate_khz, per-workgroup int64 array
    [groups, 4] of XCD id, entry, metadata done, end in wall-clock ticks)."""
    import numpy as np

    a = rec[: 4 * (groups + 1)].cpu().numpy().astype(np.int64)
    return int(a[0]), a[4:].reshape(groups, 4)


def xcd_finish_times(rate_khz, per_group):
    """Per-XCD summary of a timing record: microseconds from the first
    workgroup's entry to the last completion of each XCD, and the same for
    the metadata phase (the last workgroup of the XCD to finish it)."""
    import numpy as np

    t0 = per_group[:, 1].min()
    us = 1e3 / rate_khz
    out = {}
    for k in sorted(set(per_group[:, 0].tolist())):
        sel = per_group[:, 0] == k
        out[int(k)] = {"groups": int(sel.sum()), "end_us": float((per_group[sel, 3].max() - t0) * us),
                       "meta_us": float((per_group[sel, 2].max() - t0) * us)}
    return out


def purlin_stream_timed(dsts, srcs, nbytes=None, sink=None, nt_load=False, nt_store=False, stream=None):
    """``purlin_stream`` with a timing record per workgroup; returns
    (rate_khz, records [groups, 4]) after the stream's device work has
    finished (the call synchronises its stream)."""
    import torch

    for t in list(dsts) + list(srcs) + ([sink] if sink is not None else []):
        _require_cuda(t, "stream buffer")
    if nbytes is None:
        nbytes = min(t.numel() * t.element_size() for t in list(dsts) + list(srcs))
    for t in list(dsts) + list(srcs):
        if t.numel() * t.element_size() < nbytes:
            raise PurlinError(PURLIN_ERR_INVALID, "a stream buffer is smaller than nbytes")
    d = (_vp * max(1, len(dsts)))(*[t.data_ptr() for t in dsts])
    s = (_vp * max(1, len(srcs)))(*[t.data_ptr() for t in srcs])
    hints = (1 if nt_load else 0) | (2 if nt_store else 0)
    g = ctypes.c_uint64(0)
    _check(lib().purlin_stream_timed(d, len(dsts), s, len(srcs), int(nbytes), _ptr(sink), hints, None, 0,
                                     ctypes.byref(g), None), "purlin_stream_timed")
    dev = (list(dsts) + list(srcs))[0].device
    rec = torch.zeros(4 * (g.value + 1), dtype=torch.int64, device=dev)
    _check(lib().purlin_stream_timed(d, len(dsts), s, len(srcs), int(nbytes), _ptr(sink), hints, _ptr(rec),
                                     rec.numel(), None, _stream_handle(stream)), "purlin_stream_timed")
    torch.cuda.synchronize(dev)
    return _timed_records(rec, g.value)


def purlin_pack_timed(x, ids, E, P, out, dev_status=None, rec=None, stream=None):
    """The one-launch ``purlin_pack`` with a timing record per workgroup, into
    ``rec`` (a device int64 tensor of at least 4 * (groups + 1) entries, or
    None to allocate one).  Returns (rec, groups); read it with
    ``_timed_records(rec, groups)`` once the stream has finished."""
    import torch

    T, H = x.shape
    K = ids.shape[1]
    _require_cuda(x, "x", 2)
    _require_cuda(ids, "ids", 4)
    shapes = {"packed": ((T * K, H), x.dtype), "dest_counts": ((P,), torch.int32), "dest_offsets": ((P,), torch.int32),
              "expert_counts": ((E,), torch.int32), "expert_offsets": ((E,), torch.int32),
              "pos": ((T, K), torch.int32)}
    _check_sizes(out, shapes)
    g = ctypes.c_uint64(0)
    args = [int(T), int(H), int(K), int(E), int(P), _ptr(x), _ptr(ids), _ptr(out["packed"]), _ptr(out["dest_counts"]),
            _ptr(out["dest_offsets"]), _ptr(out["expert_counts"]), _ptr(out["expert_offsets"]), _ptr(out["pos"]),
            _ptr(dev_status)]
    _check(lib().purlin_pack_timed(*args, None, 0, ctypes.byref(g), None), "purlin_pack_timed")
    if rec is None:
        rec = torch.zeros(4 * (g.value + 1), dtype=torch.int64, device=x.device)
    _check(lib().purlin_pack_timed(*args, _ptr(rec), rec.numel(), None, _stream_handle(stream)), "purlin_pack_timed")
    return rec, g.value


# Short names: plan(...) -> Plan; pack(...) -> (packed, dest_counts,
# dest_offsets, expert_counts, pos); unpack(...) -> out.
def plan(op, P, count, dtype, chunk, **kw):
    return Plan(op, P, count, dtype, chunk, **kw)


def pack(x, ids, E, P, **kw):
    r = purlin_pack(x, ids, E, P, **kw)
    return r["packed"], r["dest_counts"], r["dest_offsets"], r["expert_counts"], r["pos"]


def unpack(y, pos, gates, **kw):
    return purlin_unpack(y, pos, gates, **kw)
