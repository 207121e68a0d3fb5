"""Python binding of libcsg, the chunk-scheduled GEMM library for MI355X (gfx950).

Argument marshalling only: every function here converts Python values (ints,
numpy arrays, torch tensors and streams) to the C ABI of ``include/csg.h`` and
calls the function of the same name in ``libcsg.so``; every step of the GEMM
runs in the library's HIP kernels and copy-engine driver. There is no fallback:
if ``libcsg.so`` has not been built (``python -m paper_2601_20595_amd.build``),
the first call raises ``CsgLibraryMissing``.

A non-OK status raises ``CsgError`` carrying the status and the library's
message. Thin ``Schedule`` and ``Plan`` classes own the C objects.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcsg.so")

# csg_status
CSG_OK, CSG_ERR_INVALID, CSG_ERR_UNSUPPORTED, CSG_ERR_HIP, CSG_ERR_NOMEM, CSG_ERR_TIMEOUT, CSG_ERR_STATE = range(7)
# csg_dtype
CSG_BF16, CSG_F32 = 0, 1
# csg_op
CSG_AG_GEMM, CSG_GEMM_RS, CSG_GROUPED_GEMM, CSG_GEMM_AR = 0, 1, 2, 3
# csg_order
CSG_ORDER_RING, CSG_ORDER_SWIZZLE1D, CSG_ORDER_PERMUTATION, CSG_ORDER_RS_RING = 0, 1, 2, 3
# csg_mode
CSG_MODE_OVERLAP, CSG_MODE_COMPUTE_ONLY, CSG_MODE_COPY_ONLY = 0, 1, 2
# csg_copy_backend
CSG_COPY_SDMA, CSG_COPY_KERNEL = 0, 1

ORDERS = {"ring": CSG_ORDER_RING, "swizzle1d": CSG_ORDER_SWIZZLE1D, "permutation": CSG_ORDER_PERMUTATION,
          "rs_ring": CSG_ORDER_RS_RING}
MODES = {"overlap": CSG_MODE_OVERLAP, "compute_only": CSG_MODE_COMPUTE_ONLY, "copy_only": CSG_MODE_COPY_ONLY}
DTYPES = {"bf16": CSG_BF16, "f32": CSG_F32}
OPS = {"ag": CSG_AG_GEMM, "rs": CSG_GEMM_RS, "grouped": CSG_GROUPED_GEMM, "ar": CSG_GEMM_AR}
COPY_BACKENDS = {"sdma": CSG_COPY_SDMA, "kernel": CSG_COPY_KERNEL}

# every symbol include/csg.h declares
ABI_FUNCTIONS = (
    "csg_version", "csg_status_str", "csg_last_error", "csg_device_check",
    "csg_schedule_create", "csg_schedule_uniform", "csg_schedule_grouped", "csg_schedule_info",
    "csg_schedule_get", "csg_schedule_destroy",
    "csg_plan_create", "csg_plan_info_get", "csg_plan_get_map", "csg_plan_set_copy_delays",
    "csg_ag_gemm", "csg_gemm_rs", "csg_gemm_ar", "csg_grouped_gemm", "csg_plan_check", "csg_plan_kernel_times",
    "csg_plan_trace", "csg_plan_destroy", "csg_attn_plan_create", "csg_ring_attn", "csg_plan_join",
    "csg_measure_mfma_peak", "csg_ag_gemm_noalloc",
)


class CsgLibraryMissing(RuntimeError):
    pass


class CsgError(RuntimeError):
    def __init__(self, status: int, where: str, message: str):
        self.status = status
        super().__init__("%s failed with %s: %s" % (where, _status_name(status), message))


class csg_chunk(ctypes.Structure):
    _fields_ = [("row_begin", ctypes.c_int64), ("row_end", ctypes.c_int64), ("src_rank", ctypes.c_int32),
                ("group", ctypes.c_int32), ("is_local", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class csg_plan_cfg(ctypes.Structure):
    _fields_ = [("bm", ctypes.c_int32), ("bn", ctypes.c_int32), ("bk", ctypes.c_int32),
                ("intra_order", ctypes.c_int32), ("tile_dispatch", ctypes.c_int32),
                ("num_workgroups", ctypes.c_int32), ("copy_engines", ctypes.c_int32), ("timeout_ms", ctypes.c_int32),
                ("split_k", ctypes.c_int32), ("tail_split", ctypes.c_int32), ("tail_chunks", ctypes.c_int32),
                ("trace", ctypes.c_int32), ("warm_rows", ctypes.c_int32), ("copy_backend", ctypes.c_int32),
                ("copy_workgroups", ctypes.c_int32), ("group_m", ctypes.c_int32), ("tail_wave", ctypes.c_int32),
                ("copy_split", ctypes.c_int32), ("tail_taper", ctypes.c_int32)]


class csg_plan_info(ctypes.Structure):
    _fields_ = [("n_tiles", ctypes.c_int32), ("n_chunks", ctypes.c_int32), ("nnz", ctypes.c_int32),
                ("n_tiles_n", ctypes.c_int32), ("num_workgroups", ctypes.c_int32), ("bm", ctypes.c_int32),
                ("bn", ctypes.c_int32), ("bk", ctypes.c_int32), ("n_units", ctypes.c_int32)]


class csg_trace_unit(ctypes.Structure):
    _fields_ = [("raster", ctypes.c_int32), ("slice", ctypes.c_int32), ("n_slices", ctypes.c_int32),
                ("xcd", ctypes.c_int32), ("workgroup", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("t_take", ctypes.c_uint64), ("t_start", ctypes.c_uint64), ("t_end", ctypes.c_uint64),
                ("cycles", ctypes.c_uint64)]


class csg_diag(ctypes.Structure):
    _fields_ = [("timed_out", ctypes.c_int32), ("chunk", ctypes.c_int32), ("tile", ctypes.c_int32),
                ("observed", ctypes.c_uint32), ("epoch", ctypes.c_uint32), ("reserved", ctypes.c_int32)]


_lib_handle = None


def _lib():
    global _lib_handle
    if _lib_handle is not None:
        return _lib_handle
    if not os.path.exists(LIB_PATH):
        raise CsgLibraryMissing("libcsg.so is not built at %s; run `python -m paper_2601_20595_amd.build`"
                                % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    i32, i64, u64, vp, st = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_int
    P = ctypes.POINTER
    sig = {
        "csg_version": ([], ctypes.c_char_p),
        "csg_status_str": ([st], ctypes.c_char_p),
        "csg_last_error": ([], ctypes.c_char_p),
        "csg_device_check": ([ctypes.c_int, ctypes.c_char_p, ctypes.c_size_t], st),
        "csg_schedule_create": ([P(csg_chunk), i32, P(i32), P(vp)], st),
        "csg_schedule_uniform": ([i32, i32, i64, i32, st, P(i32), P(vp)], st),
        "csg_schedule_grouped": ([i32, i32, i32, P(i64), P(vp)], st),
        "csg_schedule_info": ([vp, P(i32), P(i64)], st),
        "csg_schedule_get": ([vp, P(csg_chunk), P(i32)], st),
        "csg_schedule_destroy": ([vp], None),
        "csg_plan_create": ([st, i64, i64, i64, st, st, vp, P(i64), i32, P(csg_plan_cfg), ctypes.c_int, P(vp)], st),
        "csg_plan_info_get": ([vp, P(csg_plan_info)], st),
        "csg_plan_get_map": ([vp, P(i32), P(i32), P(i32), P(i32), P(i32)], st),
        "csg_plan_set_copy_delays": ([vp, P(ctypes.c_float), i32], st),
        "csg_ag_gemm": ([vp, vp, vp, vp, vp, st, vp, vp], st),
        "csg_gemm_rs": ([vp, vp, vp, vp, vp, st, vp, vp], st),
        "csg_gemm_ar": ([vp, vp, vp, vp, vp, vp, vp, vp, st, vp, vp], st),
        "csg_attn_plan_create": ([i32, i32, i32, i64, vp, P(csg_plan_cfg), ctypes.c_int, P(vp)], st),
        "csg_ring_attn": ([vp, vp, vp, vp, vp, vp, vp, vp, st, vp, vp], st),
        "csg_grouped_gemm": ([vp, vp, vp, vp, vp, st, vp, vp], st),
        "csg_plan_check": ([vp, P(csg_diag)], st),
        "csg_plan_kernel_times": ([vp, P(ctypes.c_float), i32, P(i32)], st),
        "csg_plan_trace": ([vp, P(csg_trace_unit), i32, P(i32)], st),
        "csg_plan_destroy": ([vp], None),
        "csg_plan_join": ([vp, vp], st),
        "csg_ag_gemm_noalloc": ([vp, i64, i64, i64, st, st, vp, vp, vp, vp, st, i32, ctypes.c_int, vp], st),
        "csg_measure_mfma_peak": ([ctypes.c_int, i32, P(ctypes.c_double), P(ctypes.c_double), P(ctypes.c_double)],
                                  st),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    _lib_handle = lib
    return lib


def _status_name(s: int) -> str:
    try:
        return _lib().csg_status_str(s).decode()
    except Exception:
        return "status %d" % s


def _check(status: int, where: str) -> None:
    if status != CSG_OK:
        raise CsgError(status, where, _lib().csg_last_error().decode())


def _i32_array(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


def _ptr(t) -> int:
    """Device pointer of a torch tensor (or an int / None)."""
    if t is None:
        return 0
    if isinstance(t, int):
        return t
    return int(t.data_ptr())


def _elem_bytes(dtype) -> int:
    d = DTYPES[dtype] if isinstance(dtype, str) else int(dtype)
    return 2 if d == CSG_BF16 else 4


def _buf(t, need: int, what: str) -> None:
    """Checks a tensor argument before its pointer reaches the library, which reads and
    writes dense row-major buffers of the plan's shape: it must be contiguous, hold at
    least ``need`` bytes and live on a GPU. Raw integer pointers and None pass
    unchecked (the C calls reject a NULL where one is required)."""
    if t is None or isinstance(t, int):
        return
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % what)
    have = t.numel() * t.element_size()
    if have < need:
        raise ValueError("%s holds %d bytes; the plan needs %d" % (what, have, need))
    if t.device.type != "cuda":
        raise ValueError("%s must be a GPU tensor" % what)


def _stream(s) -> int:
    if s is None:
        return 0
    if isinstance(s, int):
        return s
    return int(s.cuda_stream)


# ---------------------------------------------------------------------------------
# Functions with the C names
# ---------------------------------------------------------------------------------
def csg_version() -> str:
    return _lib().csg_version().decode()


def csg_status_str(status: int) -> str:
    return _lib().csg_status_str(status).decode()


def csg_last_error() -> str:
    return _lib().csg_last_error().decode()


def csg_device_check(device: int = 0) -> str:
    buf = ctypes.create_string_buffer(64)
    _check(_lib().csg_device_check(device, buf, 64), "csg_device_check")
    return buf.value.decode()


def csg_schedule_create(chunks: Sequence[Sequence[int]], order: Sequence[int]) -> int:
    """chunks: rows of (row_begin, row_end, src_rank, group, is_local)."""
    n = len(chunks)
    arr = (csg_chunk * max(n, 1))()
    for i, c in enumerate(chunks):
        arr[i] = csg_chunk(int(c[0]), int(c[1]), int(c[2]), int(c[3]), int(c[4]), 0)
    o = _i32_array(order)
    out = ctypes.c_void_p()
    _check(_lib().csg_schedule_create(arr, n, o.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), ctypes.byref(out)),
           "csg_schedule_create")
    return out.value


def csg_schedule_uniform(world: int, rank: int, shard_rows: int, chunks_per_shard: int, order,
                         remote_perm: Optional[Sequence[int]] = None) -> int:
    kind = ORDERS[order] if isinstance(order, str) else int(order)
    perm = None if remote_perm is None else _i32_array(remote_perm)
    pp = None if perm is None else perm.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    out = ctypes.c_void_p()
    _check(_lib().csg_schedule_uniform(world, rank, shard_rows, chunks_per_shard, kind, pp, ctypes.byref(out)),
           "csg_schedule_uniform")
    return out.value


def csg_schedule_grouped(world: int, rank: int, counts) -> int:
    c = np.ascontiguousarray(np.asarray(counts, dtype=np.int64))
    assert c.ndim == 2 and c.shape[0] == world
    out = ctypes.c_void_p()
    _check(_lib().csg_schedule_grouped(world, rank, c.shape[1], c.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                       ctypes.byref(out)), "csg_schedule_grouped")
    return out.value


def csg_schedule_info(sched: int):
    n = ctypes.c_int32()
    rows = ctypes.c_int64()
    _check(_lib().csg_schedule_info(sched, ctypes.byref(n), ctypes.byref(rows)), "csg_schedule_info")
    return n.value, rows.value


def csg_schedule_get(sched: int):
    n, _ = csg_schedule_info(sched)
    arr = (csg_chunk * n)()
    order = np.zeros(n, dtype=np.int32)
    _check(_lib().csg_schedule_get(sched, arr, order.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))),
           "csg_schedule_get")
    chunks = [(c.row_begin, c.row_end, c.src_rank, c.group, c.is_local) for c in arr]
    return chunks, order.tolist()


def csg_schedule_destroy(sched: int) -> None:
    _lib().csg_schedule_destroy(sched)


def csg_plan_create(op, M: int, N: int, K: int, in_dtype, out_dtype, sched: int, group_rows=None,
                    cfg: Optional[dict] = None, device: int = 0) -> int:
    op = OPS[op] if isinstance(op, str) else int(op)
    ind = DTYPES[in_dtype] if isinstance(in_dtype, str) else int(in_dtype)
    outd = DTYPES[out_dtype] if isinstance(out_dtype, str) else int(out_dtype)
    cfg = dict(cfg or {})
    if isinstance(cfg.get("copy_backend"), str):
        cfg["copy_backend"] = COPY_BACKENDS[cfg["copy_backend"]]
    c = csg_plan_cfg(**cfg)
    if group_rows is not None:
        g = np.ascontiguousarray(np.asarray(group_rows, dtype=np.int64))
        gp, ng = g.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), g.size
    else:
        g, gp, ng = None, None, 0
    out = ctypes.c_void_p()
    _check(_lib().csg_plan_create(op, M, N, K, ind, outd, sched, gp, ng, ctypes.byref(c), device,
                                  ctypes.byref(out)), "csg_plan_create")
    return out.value


def csg_plan_info_get(plan: int) -> csg_plan_info:
    info = csg_plan_info()
    _check(_lib().csg_plan_info_get(plan, ctypes.byref(info)), "csg_plan_info_get")
    return info


def csg_plan_get_map(plan: int) -> dict:
    info = csg_plan_info_get(plan)
    tp = np.zeros(info.n_tiles + 1, dtype=np.int32)
    tc = np.zeros(max(info.nnz, 1), dtype=np.int32)
    cp = np.zeros(info.n_chunks + 1, dtype=np.int32)
    ct = np.zeros(max(info.nnz, 1), dtype=np.int32)
    od = np.zeros(info.n_tiles, dtype=np.int32)
    P = ctypes.POINTER(ctypes.c_int32)
    _check(_lib().csg_plan_get_map(plan, tp.ctypes.data_as(P), tc.ctypes.data_as(P), cp.ctypes.data_as(P),
                                   ct.ctypes.data_as(P), od.ctypes.data_as(P)), "csg_plan_get_map")
    return {"tile_ptr": tp, "tile_chunks": tc[:info.nnz], "chunk_ptr": cp, "chunk_tiles": ct[:info.nnz],
            "tile_order": od}


def csg_plan_set_copy_delays(plan: int, delays_us=None) -> None:
    if delays_us is None:
        _check(_lib().csg_plan_set_copy_delays(plan, None, 0), "csg_plan_set_copy_delays")
        return
    d = np.ascontiguousarray(np.asarray(delays_us, dtype=np.float32))
    _check(_lib().csg_plan_set_copy_delays(plan, d.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), d.size),
           "csg_plan_set_copy_delays")


def _mode(mode) -> int:
    return MODES[mode] if isinstance(mode, str) else int(mode)


def csg_ag_gemm(plan: int, a_landing, a_staging, b_nk, c, mode="overlap", compute_stream=None,
                copy_stream=None) -> None:
    _check(_lib().csg_ag_gemm(plan, _ptr(a_landing), _ptr(a_staging), _ptr(b_nk), _ptr(c), _mode(mode),
                              _stream(compute_stream), _stream(copy_stream)), "csg_ag_gemm")


def csg_gemm_rs(plan: int, a, b_nk, c, c_outgoing, mode="overlap", compute_stream=None, copy_stream=None) -> None:
    _check(_lib().csg_gemm_rs(plan, _ptr(a), _ptr(b_nk), _ptr(c), _ptr(c_outgoing), _mode(mode),
                              _stream(compute_stream), _stream(copy_stream)), "csg_gemm_rs")


def csg_attn_plan_create(n_heads: int, n_kv_heads: int, head_dim: int, q_rows: int, sched: int,
                         cfg: Optional[dict] = None, device: int = 0) -> int:
    c = csg_plan_cfg(**(cfg or {}))
    out = ctypes.c_void_p()
    _check(_lib().csg_attn_plan_create(n_heads, n_kv_heads, head_dim, q_rows, sched, ctypes.byref(c), device,
                                       ctypes.byref(out)), "csg_attn_plan_create")
    return out.value


def csg_ring_attn(plan: int, q, k_landing, v_landing, k_staging, v_staging, o, lse, mode="overlap",
                  compute_stream=None, copy_stream=None) -> None:
    _check(_lib().csg_ring_attn(plan, _ptr(q), _ptr(k_landing), _ptr(v_landing), _ptr(k_staging), _ptr(v_staging),
                                _ptr(o), _ptr(lse), _mode(mode), _stream(compute_stream), _stream(copy_stream)),
           "csg_ring_attn")


def csg_gemm_ar(plan: int, a, b_nk, c, c_outgoing, partials_staging, partials_landing, reduced_staging,
                mode="overlap", compute_stream=None, copy_stream=None) -> None:
    _check(_lib().csg_gemm_ar(plan, _ptr(a), _ptr(b_nk), _ptr(c), _ptr(c_outgoing), _ptr(partials_staging),
                              _ptr(partials_landing), _ptr(reduced_staging), _mode(mode), _stream(compute_stream),
                              _stream(copy_stream)), "csg_gemm_ar")


def csg_grouped_gemm(plan: int, x_landing, x_staging, b_enk, c, mode="overlap", compute_stream=None,
                     copy_stream=None) -> None:
    _check(_lib().csg_grouped_gemm(plan, _ptr(x_landing), _ptr(x_staging), _ptr(b_enk), _ptr(c), _mode(mode),
                                   _stream(compute_stream), _stream(copy_stream)), "csg_grouped_gemm")


def csg_plan_check(plan: int) -> csg_diag:
    """Waits for the plan's last call; raises CsgError(CSG_ERR_TIMEOUT) if a wait expired."""
    d = csg_diag()
    st = _lib().csg_plan_check(plan, ctypes.byref(d))
    if st == CSG_ERR_TIMEOUT:
        err = CsgError(st, "csg_plan_check", _lib().csg_last_error().decode())
        err.diag = d
        raise err
    _check(st, "csg_plan_check")
    return d


def csg_ag_gemm_noalloc(schedule, M, N, K, in_dtype, out_dtype, a_landing, a_staging, b_nk, c, mode="overlap",
                        copy_workgroups=0, device=0, stream=None) -> None:
    """The all-gather GEMM without a plan, on the library's static device scratch
    (allocates nothing). `schedule` is a Schedule or a csg_schedule handle."""
    h = schedule.handle if isinstance(schedule, Schedule) else schedule
    ib = _elem_bytes(in_dtype)
    for t, n, what in ((a_landing, M * K * ib, "a_landing"), (a_staging, M * K * ib, "a_staging"),
                       (b_nk, N * K * ib, "b_nk"), (c, M * N * _elem_bytes(out_dtype), "c")):
        _buf(t, n, what)
    _check(_lib().csg_ag_gemm_noalloc(h, M, N, K, DTYPES[in_dtype] if isinstance(in_dtype, str) else in_dtype,
                                      DTYPES[out_dtype] if isinstance(out_dtype, str) else out_dtype,
                                      _ptr(a_landing), _ptr(a_staging), _ptr(b_nk), _ptr(c), _mode(mode),
                                      copy_workgroups, device, _stream(stream)), "csg_ag_gemm_noalloc")


def csg_plan_join(plan: int, stream) -> None:
    """Queues on `stream` a wait, on the device, for every copy of the plan's last call."""
    _check(_lib().csg_plan_join(plan, _stream(stream)), "csg_plan_join")


def csg_measure_mfma_peak(device: int = 0, iters: int = 4096):
    """(TFLOP/s, ms, GHz) of the MFMA microbenchmark: dense bf16 rate on every SIMD."""
    tf, ms, ghz = ctypes.c_double(0), ctypes.c_double(0), ctypes.c_double(0)
    _check(_lib().csg_measure_mfma_peak(device, iters, ctypes.byref(tf), ctypes.byref(ms), ctypes.byref(ghz)),
           "csg_measure_mfma_peak")
    return tf.value, ms.value, ghz.value


def csg_plan_kernel_times(plan: int, n: int = 256) -> np.ndarray:
    """Durations (ms) of the plan's last n kernel launches, oldest first."""
    buf = np.zeros(max(n, 1), dtype=np.float32)
    got = ctypes.c_int32(0)
    _check(_lib().csg_plan_kernel_times(plan, buf.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), n,
                                        ctypes.byref(got)), "csg_plan_kernel_times")
    return buf[:got.value].copy()


def csg_plan_trace(plan: int, n: int) -> np.ndarray:
    """Trace of the plan's last kernel run: a structured array with fields raster,
    slice, n_slices, xcd, workgroup, t_take, t_start, t_end (100 MHz ticks) and cycles
    (shader clock, t_start to t_end)."""
    buf = (csg_trace_unit * max(n, 1))()
    got = ctypes.c_int32(0)
    _check(_lib().csg_plan_trace(plan, buf, n, ctypes.byref(got)), "csg_plan_trace")
    dt = np.dtype([("raster", np.int32), ("slice", np.int32), ("n_slices", np.int32), ("xcd", np.int32),
                   ("workgroup", np.int32), ("reserved", np.int32), ("t_take", np.uint64), ("t_start", np.uint64),
                   ("t_end", np.uint64), ("cycles", np.uint64)])
    return np.frombuffer(bytes(buf), dtype=dt, count=got.value).copy()


def csg_plan_destroy(plan: int) -> None:
    _lib().csg_plan_destroy(plan)


# ---------------------------------------------------------------------------------
# Owning wrappers
# ---------------------------------------------------------------------------------
class Schedule:
    """Owns a csg_schedule."""

    def __init__(self, handle: int):
        self.handle = handle

    @classmethod
    def uniform(cls, world, rank, shard_rows, chunks_per_shard, order, remote_perm=None):
        return cls(csg_schedule_uniform(world, rank, shard_rows, chunks_per_shard, order, remote_perm))

    @classmethod
    def grouped(cls, world, rank, counts):
        return cls(csg_schedule_grouped(world, rank, counts))

    @classmethod
    def create(cls, chunks, order):
        return cls(csg_schedule_create(chunks, order))

    def get(self):
        return csg_schedule_get(self.handle)

    def close(self):
        if self.handle:
            csg_schedule_destroy(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Plan:
    """Owns a csg_plan; methods forward to the C calls."""

    def __init__(self, op, M, N, K, in_dtype, out_dtype, schedule: Schedule, group_rows=None, cfg=None,
                 device: int = 0):
        self.op = op
        self.handle = csg_plan_create(op, M, N, K, in_dtype, out_dtype, schedule.handle, group_rows, cfg, device)
        # buffer sizes the calls check tensor arguments against
        ib, ob = _elem_bytes(in_dtype), _elem_bytes(out_dtype)
        groups = len(group_rows) if group_rows is not None else 1
        self._bytes = {"a": M * K * ib, "b": groups * N * K * ib, "c": M * N * ob}
        if op == "ar":
            chunks, _ = schedule.get()
            own = sum(c[1] - c[0] for c in chunks if c[4])
            self._bytes["partials"] = (M // own - 1) * own * N * ob

    @property
    def info(self) -> csg_plan_info:
        return csg_plan_info_get(self.handle)

    def get_map(self) -> dict:
        return csg_plan_get_map(self.handle)

    def set_copy_delays(self, delays_us=None):
        csg_plan_set_copy_delays(self.handle, delays_us)

    def ag_gemm(self, a_landing, a_staging, b_nk, c, mode="overlap", compute_stream=None, copy_stream=None):
        z = self._bytes
        for t, n, what in ((a_landing, z.get("a", 0), "a_landing"), (a_staging, z.get("a", 0), "a_staging"), (b_nk, z.get("b", 0), "b_nk"),
                           (c, z.get("c", 0), "c")):
            _buf(t, n, what)
        csg_ag_gemm(self.handle, a_landing, a_staging, b_nk, c, mode, compute_stream, copy_stream)

    def gemm_rs(self, a, b_nk, c, c_outgoing, mode="overlap", compute_stream=None, copy_stream=None):
        z = self._bytes
        for t, n, what in ((a, z.get("a", 0), "a"), (b_nk, z.get("b", 0), "b_nk"), (c, z.get("c", 0), "c"), (c_outgoing, z.get("c", 0), "c_outgoing")):
            _buf(t, n, what)
        csg_gemm_rs(self.handle, a, b_nk, c, c_outgoing, mode, compute_stream, copy_stream)

    def gemm_ar(self, a, b_nk, c, c_outgoing, partials_staging, partials_landing, reduced_staging, mode="overlap",
                compute_stream=None, copy_stream=None):
        z = self._bytes
        for t, n, what in ((a, z.get("a", 0), "a"), (b_nk, z.get("b", 0), "b_nk"), (c, z.get("c", 0), "c"), (c_outgoing, z.get("c", 0), "c_outgoing"),
                           (partials_staging, z.get("partials", 0), "partials_staging"),
                           (partials_landing, z.get("partials", 0), "partials_landing"),
                           (reduced_staging, z.get("c", 0), "reduced_staging")):
            _buf(t, n, what)
        csg_gemm_ar(self.handle, a, b_nk, c, c_outgoing, partials_staging, partials_landing, reduced_staging, mode,
                    compute_stream, copy_stream)

    def grouped_gemm(self, x_landing, x_staging, b_enk, c, mode="overlap", compute_stream=None, copy_stream=None):
        z = self._bytes
        for t, n, what in ((x_landing, z.get("a", 0), "x_landing"), (x_staging, z.get("a", 0), "x_staging"), (b_enk, z.get("b", 0), "b_enk"),
                           (c, z.get("c", 0), "c")):
            _buf(t, n, what)
        csg_grouped_gemm(self.handle, x_landing, x_staging, b_enk, c, mode, compute_stream, copy_stream)

    def check(self) -> csg_diag:
        return csg_plan_check(self.handle)

    def kernel_times(self, n: int = 256) -> np.ndarray:
        return csg_plan_kernel_times(self.handle, n)

    def join(self, stream) -> None:
        csg_plan_join(self.handle, stream)

    def trace(self) -> np.ndarray:
        return csg_plan_trace(self.handle, self.info.n_units)

    def close(self):
        if self.handle:
            csg_plan_destroy(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class AttnPlan(Plan):
    """Owns a ring-attention csg_plan (csg_attn_plan_create)."""

    def __init__(self, n_heads, n_kv_heads, head_dim, q_rows, schedule: Schedule, cfg=None, device: int = 0):
        self.op = "attn"
        self.handle = csg_attn_plan_create(n_heads, n_kv_heads, head_dim, q_rows, schedule.handle, cfg, device)
        chunks, _ = schedule.get()
        keys = chunks[-1][1] if chunks else 0
        self._bytes = {"q": q_rows * n_heads * head_dim * 2, "kv": keys * n_kv_heads * head_dim * 2,
                       "lse": n_heads * q_rows * 4}

    def ring_attn(self, q, k_landing, v_landing, k_staging, v_staging, o, lse, mode="overlap", compute_stream=None,
                  copy_stream=None):
        z = self._bytes
        for t, n, what in ((q, z.get("q", 0), "q"), (k_landing, z.get("kv", 0), "k_landing"), (v_landing, z.get("kv", 0), "v_landing"),
                           (k_staging, z.get("kv", 0), "k_staging"), (v_staging, z.get("kv", 0), "v_staging"), (o, z.get("q", 0), "o"),
                           (lse, z.get("lse", 0), "lse")):
            _buf(t, n, what)
        csg_ring_attn(self.handle, q, k_landing, v_landing, k_staging, v_staging, o, lse, mode, compute_stream,
                      copy_stream)
