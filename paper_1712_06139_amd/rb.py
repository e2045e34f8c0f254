"""ctypes binding of librbatch.so (declared in include/rb.h).

Argument marshalling only: every step of the batching path runs in the C++
runtime and the HIP kernels. torch is used for device memory (tensors whose
data_ptr() is handed over) and nothing else. Names follow the C ABI.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librbatch.so")

RB_OK, RB_EINVAL, RB_EBUSY, RB_EAGAIN, RB_EEMPTY = 0, -1, -2, -3, -4
RB_ESIZE, RB_ENOENT, RB_EDEVICE, RB_ENOMEM, RB_ERANGE = -5, -6, -7, -8, -9
RB_MODEL_MLP, RB_MODEL_RANKING, RB_MODEL_SEQPOOL = 0, 1, 2
RB_DT_F32, RB_DT_BF16 = 0, 1
RB_ACT_NONE, RB_ACT_RELU, RB_ACT_SIGMOID, RB_ACT_SOFTMAX = 0, 1, 2, 3
RB_MODE_DEVICE, RB_MODE_NO_DEVICE = 0, 1
INT64_MAX = 2 ** 63 - 1

ACT = {"none": RB_ACT_NONE, "relu": RB_ACT_RELU, "sigmoid": RB_ACT_SIGMOID, "softmax": RB_ACT_SOFTMAX}
KIND = {"mlp": RB_MODEL_MLP, "ranking": RB_MODEL_RANKING, "seqpool": RB_MODEL_SEQPOOL}
DTYPE = {"f32": RB_DT_F32, "bf16": RB_DT_BF16}

p_f32 = C.POINTER(C.c_float)
p_i32 = C.POINTER(C.c_int32)
p_i64 = C.POINTER(C.c_int64)


class RBError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {_lib().rb_status_str(status).decode()} ({status})")


class rb_layer_desc(C.Structure):
    _fields_ = [("fan_in", C.c_int32), ("fan_out", C.c_int32), ("act", C.c_int32), ("w", p_f32), ("b", p_f32)]


class rb_model_desc(C.Structure):
    _fields_ = [("kind", C.c_int32), ("dtype", C.c_int32), ("n_layers", C.c_int32),
                ("layers", C.POINTER(rb_layer_desc)), ("n_tables", C.c_int32), ("table_rows", C.c_int64),
                ("emb_dim", C.c_int32), ("n_dense", C.c_int32), ("tables", C.POINTER(p_f32)),
                ("head", rb_layer_desc)]


class rb_sched_opts(C.Structure):
    _fields_ = [("mode", C.c_int32), ("window_batches", C.c_int32), ("pad_value", C.c_float),
                ("profile", C.c_int32), ("n_streams", C.c_int32), ("seq_pack", C.c_int32),
                ("clocked_windows", C.c_int32), ("emb_dedup", C.c_int32), ("fuse_mlp_tail", C.c_int32)]


class rb_queue_opts(C.Structure):
    _fields_ = [("max_batch_size", C.c_int32), ("allowed_batch_sizes", p_i32), ("n_allowed", C.c_int32),
                ("batch_timeout_ns", C.c_int64), ("bucket_len", C.c_int32), ("service_ns", p_i64),
                ("n_service", C.c_int32), ("window_ns", C.c_int64), ("window_tail_ns", C.c_int64)]


class rb_request(C.Structure):
    _fields_ = [("n_rows", C.c_int32), ("dense", p_f32), ("n_dense", C.c_int64), ("lens", p_i32),
                ("n_lens", C.c_int64), ("ids", p_i32), ("n_ids", C.c_int64)]


class rb_batch_info(C.Structure):
    _fields_ = [("batch_id", C.c_uint64), ("queue", C.c_int32), ("real_rows", C.c_int32),
                ("padded_rows", C.c_int32), ("n_req", C.c_int32), ("close_ns", C.c_int64),
                ("dispatch_ns", C.c_int64), ("done_ns", C.c_int64), ("req_ids", C.POINTER(C.c_uint64))]


class rb_window_info(C.Structure):
    _fields_ = [("n_batches", C.c_int32), ("batches", C.POINTER(rb_batch_info))]


class rb_servable(C.Structure):
    _fields_ = [("n_queues", C.c_int32), ("queues", C.POINTER(C.c_void_p))]


class rb_trace(C.Structure):
    _fields_ = [("n_requests", C.c_int32), ("servable", p_i32), ("arrival_ns", p_i64), ("n_rows", p_i32),
                ("max_len", p_i32), ("dense", C.c_void_p), ("dense_off", p_i64), ("lens", C.c_void_p),
                ("lens_off", p_i64), ("ids", C.c_void_p), ("ids_off", p_i64), ("out", C.c_void_p),
                ("out_off", p_i64)]


class rb_log(C.Structure):
    _fields_ = [("req_done_ns", p_i64), ("req_queue", p_i32), ("max_batches", C.c_int64),
                ("n_batches", C.c_int64), ("b_queue", p_i32), ("b_real", p_i32), ("b_padded", p_i32),
                ("b_close_ns", p_i64), ("b_dispatch_ns", p_i64), ("b_done_ns", p_i64),
                ("b_req_begin", p_i64), ("b_reqs", p_i32)]


class rb_k_req(C.Structure):
    _fields_ = [("dense_off", C.c_int64), ("dense_end", C.c_int64), ("lens_off", C.c_int64),
                ("ids_off", C.c_int64), ("ids_end", C.c_int64), ("out_off", C.c_int64),
                ("n_rows", C.c_int32), ("tok_off", C.c_int32)]


class rb_k_batch(C.Structure):
    _fields_ = [("req_begin", C.c_int32), ("n_req", C.c_int32), ("row_base", C.c_int32),
                ("padded", C.c_int32), ("real", C.c_int32), ("seq_T", C.c_int32)]


class rb_k_row(C.Structure):
    _fields_ = [("src", C.c_int64), ("aux", C.c_int64), ("lens", C.c_int64), ("out", C.c_int64)]


# numpy views of the device-side descriptor records
K_REQ_DTYPE = np.dtype([("dense_off", "<i8"), ("dense_end", "<i8"), ("lens_off", "<i8"), ("ids_off", "<i8"),
                        ("ids_end", "<i8"), ("out_off", "<i8"), ("n_rows", "<i4"), ("tok_off", "<i4")])
K_BATCH_DTYPE = np.dtype([("req_begin", "<i4"), ("n_req", "<i4"), ("row_base", "<i4"), ("padded", "<i4"),
                          ("real", "<i4"), ("seq_T", "<i4")])
K_ROW_DTYPE = np.dtype([("src", "<i8"), ("aux", "<i8"), ("lens", "<i8"), ("out", "<i8")])

_LIB: Optional[C.CDLL] = None

_SIGS = {
    "rb_status_str": (C.c_char_p, [C.c_int32]),
    "rb_ctx_create": (C.c_int32, [C.c_int32, C.POINTER(C.c_void_p)]),
    "rb_ctx_destroy": (C.c_int32, [C.c_void_p]),
    "rb_model_create": (C.c_int32, [C.c_void_p, C.POINTER(rb_model_desc), C.POINTER(C.c_void_p)]),
    "rb_model_info": (C.c_int32, [C.c_void_p, p_i32, p_i32]),
    "rb_model_destroy": (C.c_int32, [C.c_void_p]),
    "rb_sched_create": (C.c_int32, [C.c_void_p, C.POINTER(rb_sched_opts), C.POINTER(C.c_void_p)]),
    "rb_sched_destroy": (C.c_int32, [C.c_void_p]),
    "rb_sync": (C.c_int32, [C.c_void_p]),
    "rb_sched_kernel_stats": (C.c_int32, [C.c_void_p, C.c_char_p, p_i64, C.POINTER(C.c_double)]),
    "rb_sched_stream": (C.c_int32, [C.c_void_p, C.POINTER(C.c_void_p)]),
    "rb_queue_create": (C.c_int32, [C.c_void_p, C.c_void_p, C.POINTER(rb_queue_opts), C.POINTER(C.c_void_p)]),
    "rb_queue_destroy": (C.c_int32, [C.c_void_p]),
    "rb_queue_id": (C.c_int32, [C.c_void_p, p_i32]),
    "rb_queue_set_model": (C.c_int32, [C.c_void_p, C.c_void_p]),
    "rb_submit": (C.c_int32, [C.c_void_p, C.POINTER(rb_request), C.c_int64, C.POINTER(C.c_uint64)]),
    "rb_advance": (C.c_int32, [C.c_void_p, C.c_int64]),
    "rb_flush": (C.c_int32, [C.c_void_p]),
    "rb_run_next": (C.c_int32, [C.c_void_p, C.POINTER(rb_batch_info)]),
    "rb_run_window": (C.c_int32, [C.c_void_p, C.POINTER(rb_window_info)]),
    "rb_collect": (C.c_int32, [C.c_void_p, C.c_uint64, p_f32, C.c_size_t, p_i32]),
    "rb_sim_run": (C.c_int32, [C.c_void_p, C.POINTER(rb_servable), C.c_int32, C.POINTER(rb_trace),
                               C.POINTER(rb_log)]),
    "rb_run_group": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_int64,
                                 C.c_int64, C.c_void_p, C.c_int64, C.c_void_p, C.c_int64, C.c_void_p, C.c_int64,
                                 C.c_void_p, C.c_int64]),
    "rb_run_group_static": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32,
                                        C.c_int64, C.c_int64, C.c_void_p, C.c_int64, C.c_void_p, C.c_int64,
                                        C.c_void_p, C.c_int64, C.c_void_p, C.c_int64]),
    "rb_k_route": (C.c_int32, [C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_void_p,
                               C.c_int64, C.c_int32, C.c_int32, C.c_int32, C.c_void_p, C.c_int32, C.c_int64,
                               C.c_void_p]),
    "rb_k_assemble": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_int32, C.c_void_p, C.c_int64,
                                  C.c_int32, C.c_void_p, C.c_int32, C.c_int32, C.c_float, C.c_void_p]),
    "rb_k_embbag": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p,
                                C.c_int32, C.c_int64, C.c_int32, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32,
                                C.c_float, C.c_void_p]),
    "rb_k_embbag_dedup": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_int64,
                                      C.c_void_p, C.c_int32, C.c_int64, C.c_int32, C.c_void_p, C.c_int32,
                                      C.c_void_p, C.c_int32, C.c_float, C.c_void_p]),
    "rb_k_gemm_bf16": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_void_p,
                                   C.c_void_p, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32]),
    "rb_k_gemm_f32": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_void_p,
                                  C.c_void_p, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                  C.c_void_p, C.c_int32]),
    "rb_k_head": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_void_p, C.c_float,
                              C.c_int32, C.c_int32, C.c_void_p]),
    "rb_k_gemm_bf16_rows": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_void_p,
                                        C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_void_p, C.c_int32,
                                        C.c_void_p]),
    "rb_k_gemm_f32_rows": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_void_p,
                                       C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_void_p, C.c_int32,
                                       C.c_void_p]),
    "rb_k_gemm_head": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32,
                                   C.c_int32, C.c_int32, C.c_void_p, C.c_void_p, C.c_float, C.c_int32, C.c_void_p]),
    "rb_k_mlp_tail": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_int32, C.c_void_p,
                                  C.c_int32, C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_float,
                                  C.c_int32, C.c_void_p]),
    "rb_k_seqpool": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_int64, C.c_void_p, C.c_int32,
                                 C.c_int32, C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_void_p]),
    "rb_k_split": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_int32,
                               C.c_void_p]),
}

EXPORTS = tuple(_SIGS)


def _lib() -> C.CDLL:
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build() first")
        lib = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        _LIB = lib
    return _LIB


def lib() -> C.CDLL:
    return _lib()


def check(status: int, what: str) -> int:
    if status != RB_OK:
        raise RBError(status, what)
    return status


def _ptr(a: Optional[np.ndarray], t):
    if a is None:
        return C.cast(None, t)
    return a.ctypes.data_as(t)


def dptr(t) -> Optional[int]:
    """Device address of a torch tensor (None for None)."""
    return None if t is None else int(t.data_ptr())


def torch_stream_ptr(stream=None) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def _batch_dict(info: rb_batch_info) -> dict:
    return {"batch_id": info.batch_id, "queue": info.queue, "real": info.real_rows, "padded": info.padded_rows,
            "reqs": [info.req_ids[i] for i in range(info.n_req)], "close_ns": info.close_ns,
            "dispatch_ns": info.dispatch_ns, "done_ns": info.done_ns}


# ---------------------------------------------------------------- objects

class Ctx:
    def __init__(self, device: int = 0):
        h = C.c_void_p()
        check(_lib().rb_ctx_create(device, C.byref(h)), "rb_ctx_create")
        self.h = h
        self.device = device

    def destroy(self):
        if self.h:
            check(_lib().rb_ctx_destroy(self.h), "rb_ctx_destroy")
            self.h = None


class Model:
    """A model whose host parameters are copied into the library.

    layers: [(W [fan_out, fan_in] f32, b [fan_out] f32, act name)]
    tables: ranking tables ([rows, 64] f32 each); head: seqpool (W, b, act).
    W / b may be None in a host-only context (shapes only).
    """

    def __init__(self, ctx: Ctx, kind: str, dtype: str, layers, tables=None, n_dense: int = 0,
                 head=None, shapes: Optional[List[Tuple[int, int]]] = None, table_rows: int = 0):
        keep = []

        def f32(a):
            if a is None:
                return None
            a = np.ascontiguousarray(a, dtype=np.float32)
            keep.append(a)
            return a

        L = (rb_layer_desc * len(layers))()
        for i, (W, b, act) in enumerate(layers):
            W, b = f32(W), f32(b)
            fo, fi = (W.shape if W is not None else shapes[i])
            L[i] = rb_layer_desc(fi, fo, ACT[act], _ptr(W, p_f32), _ptr(b, p_f32))
        d = rb_model_desc()
        d.kind, d.dtype, d.n_layers, d.layers = KIND[kind], DTYPE[dtype], len(layers), L
        if kind == "ranking":
            ts = [f32(t) for t in (tables or [])]
            d.n_tables = len(ts) if ts else int(shapes[-1][0])
            d.table_rows = ts[0].shape[0] if ts else table_rows
            d.emb_dim = 64
            d.n_dense = n_dense
            if ts:
                arr = (p_f32 * len(ts))(*[_ptr(t, p_f32) for t in ts])
                keep.append(arr)
                d.tables = arr
        if head is not None:
            W, b, act = head
            W, b = f32(W), f32(b)
            fo, fi = W.shape
            d.head = rb_layer_desc(fi, fo, ACT[act], _ptr(W, p_f32), _ptr(b, p_f32))
        h = C.c_void_p()
        check(_lib().rb_model_create(ctx.h, C.byref(d), C.byref(h)), "rb_model_create")
        self.h = h
        self.kind = kind
        di, do = C.c_int32(), C.c_int32()
        check(_lib().rb_model_info(h, C.byref(di), C.byref(do)), "rb_model_info")
        self.d_in, self.d_out = di.value, do.value

    def destroy(self):
        if self.h:
            check(_lib().rb_model_destroy(self.h), "rb_model_destroy")
            self.h = None


class Queue:
    def __init__(self, sched: "Sched", model: Model, max_batch_size: int, allowed: Sequence[int] = (),
                 timeout_ns: Optional[int] = None, bucket_len: int = 0,
                 service_ns: Optional[Sequence[int]] = None, window_ns: int = 0, window_tail_ns: int = 0):
        al = np.ascontiguousarray(allowed, dtype=np.int32)
        sv = None if service_ns is None else np.ascontiguousarray(service_ns, dtype=np.int64)
        o = rb_queue_opts(max_batch_size, _ptr(al, p_i32) if al.size else C.cast(None, p_i32), int(al.size),
                          INT64_MAX if timeout_ns is None else int(timeout_ns), bucket_len,
                          _ptr(sv, p_i64), 0 if sv is None else int(sv.size), int(window_ns),
                          int(window_tail_ns))
        h = C.c_void_p()
        check(_lib().rb_queue_create(sched.h, model.h, C.byref(o), C.byref(h)), "rb_queue_create")
        self.h = h
        self.model = model
        self.bucket_len = bucket_len
        qid = C.c_int32()
        check(_lib().rb_queue_id(h, C.byref(qid)), "rb_queue_id")
        self.id = qid.value

    def run_group(self, stream: int, batches, n_batches: int, reqs, n_reqs: int, slots: int, tokens: int,
                  dense, dense_len: int, lens, lens_len: int, ids, ids_len: int, out, out_len: int,
                  entry: str = "rb_run_group"):
        """One launch group on device-resident descriptors and arenas
        (torch tensors; `stream` a hipStream_t address, 0 for the
        scheduler's)."""
        check(getattr(_lib(), entry)(self.h, stream or None, dptr(batches), n_batches, dptr(reqs), n_reqs, slots,
                                     tokens, dptr(dense), dense_len, dptr(lens), lens_len, dptr(ids), ids_len,
                                     dptr(out), out_len), entry)

    def set_model(self, model: Optional[Model]):
        """Version transition: batches dispatched from now on run `model`;
        None holds the queue (no version bound, nothing dispatched)."""
        check(_lib().rb_queue_set_model(self.h, None if model is None else model.h), "rb_queue_set_model")
        self.model = model

    def destroy(self):
        if self.h:
            check(_lib().rb_queue_destroy(self.h), "rb_queue_destroy")
            self.h = None


class Sched:
    def __init__(self, ctx: Ctx, device: bool = True, window_batches: int = 1, pad_value: float = 0.0,
                 profile: int = 0, n_streams: int = 1, seq_pack: bool = False, clocked_windows: bool = False,
                 emb_dedup: bool = False, fused_tail: bool = False):
        o = rb_sched_opts(RB_MODE_DEVICE if device else RB_MODE_NO_DEVICE, window_batches, pad_value,
                          int(profile), n_streams, int(seq_pack), int(clocked_windows), int(emb_dedup),
                          int(fused_tail))
        h = C.c_void_p()
        check(_lib().rb_sched_create(ctx.h, C.byref(o), C.byref(h)), "rb_sched_create")
        self.h = h

    def destroy(self):
        if self.h:
            check(_lib().rb_sched_destroy(self.h), "rb_sched_destroy")
            self.h = None

    def sync(self):
        check(_lib().rb_sync(self.h), "rb_sync")

    def stream(self) -> int:
        p = C.c_void_p()
        check(_lib().rb_sched_stream(self.h, C.byref(p)), "rb_sched_stream")
        return p.value or 0

    def kernel_stats(self, kernel: str) -> Tuple[int, float]:
        n, ms = C.c_int64(), C.c_double()
        check(_lib().rb_sched_kernel_stats(self.h, kernel.encode(), C.byref(n), C.byref(ms)),
              "rb_sched_kernel_stats")
        return n.value, ms.value

    # serving API
    def submit(self, q: Queue, n_rows: int, dense: np.ndarray, lens: Optional[np.ndarray] = None,
               ids: Optional[np.ndarray] = None, arrival_ns: int = 0) -> int:
        d = np.ascontiguousarray(dense, dtype=np.float32).ravel()
        ln = None if lens is None else np.ascontiguousarray(lens, dtype=np.int32).ravel()
        ii = None if ids is None else np.ascontiguousarray(ids, dtype=np.int32).ravel()
        r = rb_request(n_rows, _ptr(d, p_f32), d.size, _ptr(ln, p_i32), 0 if ln is None else ln.size,
                       _ptr(ii, p_i32), 0 if ii is None else ii.size)
        out = C.c_uint64()
        check(_lib().rb_submit(q.h, C.byref(r), arrival_ns, C.byref(out)), "rb_submit")
        return out.value

    def advance(self, now_ns: int):
        check(_lib().rb_advance(self.h, now_ns), "rb_advance")

    def run_next(self) -> Optional[dict]:
        info = rb_batch_info()
        st = _lib().rb_run_next(self.h, C.byref(info))
        if st == RB_EEMPTY:
            return None
        check(st, "rb_run_next")
        return _batch_dict(info)

    def run_window(self) -> Optional[List[dict]]:
        info = rb_window_info()
        st = _lib().rb_run_window(self.h, C.byref(info))
        if st == RB_EEMPTY:
            return None
        check(st, "rb_run_window")
        return [_batch_dict(info.batches[i]) for i in range(info.n_batches)]

    def collect(self, req_id: int, n_rows: int, d_out: int) -> np.ndarray:
        out = np.empty(n_rows * d_out, dtype=np.float32)
        rows = C.c_int32()
        check(_lib().rb_collect(self.h, req_id, _ptr(out, p_f32), out.nbytes, C.byref(rows)), "rb_collect")
        return out.reshape(rows.value, d_out)

    def sim_run(self, servables: Sequence[Sequence[Queue]], servable: np.ndarray, arrival_ns: np.ndarray,
                n_rows: np.ndarray, max_len: Optional[np.ndarray] = None, dense=None, dense_off=None,
                lens=None, lens_off=None, ids=None, ids_off=None, out=None, out_off=None) -> dict:
        """Replay a trace. Host arrays are numpy; dense/lens/ids/out are device
        tensors (or None in no-device mode). Returns the batch log."""
        return self.prepare_sim_run(servables, servable, arrival_ns, n_rows, max_len, dense, dense_off, lens,
                                    lens_off, ids, ids_off, out, out_off)()

    def prepare_sim_run(self, servables: Sequence[Sequence[Queue]], servable: np.ndarray, arrival_ns: np.ndarray,
                        n_rows: np.ndarray, max_len: Optional[np.ndarray] = None, dense=None, dense_off=None,
                        lens=None, lens_off=None, ids=None, ids_off=None, out=None, out_off=None):
        """The arguments of sim_run marshalled once; returns a function that
        makes the rb_sim_run call with them (again on every call) and returns
        the batch log, so that a caller can time the library call alone."""
        n = int(len(n_rows))
        keep = []

        def arr(a, dt):
            if a is None:
                return None
            a = np.ascontiguousarray(a, dtype=dt)
            keep.append(a)
            return a

        sv = (rb_servable * len(servables))()
        for i, qs in enumerate(servables):
            qa = (C.c_void_p * len(qs))(*[q.h.value for q in qs])
            keep.append(qa)
            sv[i] = rb_servable(len(qs), C.cast(qa, C.POINTER(C.c_void_p)))
        t = rb_trace()
        t.n_requests = n
        t.servable = _ptr(arr(servable, np.int32), p_i32)
        t.arrival_ns = _ptr(arr(arrival_ns, np.int64), p_i64)
        t.n_rows = _ptr(arr(n_rows, np.int32), p_i32)
        t.max_len = _ptr(arr(max_len, np.int32), p_i32)
        t.dense, t.lens, t.ids, t.out = dptr(dense), dptr(lens), dptr(ids), dptr(out)
        t.dense_off = _ptr(arr(dense_off, np.int64), p_i64)
        t.lens_off = _ptr(arr(lens_off, np.int64), p_i64)
        t.ids_off = _ptr(arr(ids_off, np.int64), p_i64)
        t.out_off = _ptr(arr(out_off, np.int64), p_i64)
        lg = {
            "req_done_ns": np.zeros(n, np.int64), "req_queue": np.zeros(n, np.int32),
            "b_queue": np.zeros(n, np.int32), "b_real": np.zeros(n, np.int32), "b_padded": np.zeros(n, np.int32),
            "b_close_ns": np.zeros(n, np.int64), "b_dispatch_ns": np.zeros(n, np.int64),
            "b_done_ns": np.zeros(n, np.int64), "b_req_begin": np.zeros(n + 1, np.int64),
            "b_reqs": np.zeros(n, np.int32),
        }
        L = rb_log()
        L.max_batches = n
        for k, v in lg.items():
            setattr(L, k, _ptr(v, p_i64 if v.dtype == np.int64 else p_i32))
        f = _lib().rb_sim_run
        ns = len(servables)

        def call() -> dict:
            check(f(self.h, sv, ns, C.byref(t), C.byref(L)), "rb_sim_run")
            nb = int(L.n_batches)
            res = {k: (v[:nb] if k.startswith("b_") and k != "b_req_begin" and k != "b_reqs" else v)
                   for k, v in lg.items()}
            res["b_req_begin"] = lg["b_req_begin"][:nb + 1]
            res["n_batches"] = nb
            return res
        call.keep = keep
        return call
