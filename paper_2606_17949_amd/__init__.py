"""Python binding of ``librouteb.so``, the gfx950 RouteBalance routing path.

Thin ctypes marshalling over the C ABI in ``include/routebalance.h``: each
``rb_*`` function here has the same name and meaning as the C entry point,
takes torch tensors that already live on the GPU, passes their device pointers
and the current HIP stream, and raises :class:`RbError` on a non-OK status.
All computation happens in the HIP kernels; torch only provides device memory
and streams. There is no CPU fallback: importing this package fails if the
library has not been built (``python -m paper_2606_17949_amd.build``).
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librouteb.so")

RB_OK, RB_ERR_NULL, RB_ERR_DIMS, RB_ERR_DTYPE, RB_ERR_WEIGHTS = 0, -1, -2, -3, -4
RB_ERR_WORKSPACE, RB_ERR_UNSUPPORTED, RB_ERR_HIP, RB_ERR_ALIGN, RB_ERR_SCRATCH = -5, -6, -7, -8, -9
RB_F32, RB_BF16 = 0, 1
RB_KNN_UNIFORM, RB_KNN_INV_DIST = 0, 1
RB_ORDER_ARRIVAL, RB_ORDER_LPT = 0, 1
RB_FLAG_OVERLAP, RB_FLAG_LISTS_ONLY, RB_FLAG_FROM_LISTS = 1, 2, 4
RB_MAX_K, RB_MAX_D, RB_MAX_I, RB_MAX_M = 64, 2048, 1024, 1024
RB_SCRATCH_BYTES = 64 << 20

# every symbol include/routebalance.h declares
EXPORTS = ("rb_status_string", "rb_workspace_size", "rb_bank_norms", "rb_knn_topk", "rb_predict",
           "rb_score", "rb_assign", "rb_assign_ex", "rb_knn_predict", "rb_route_batch",
           "rb_route_batch_ex", "rb_advance_state", "rb_profile_scan_events",
           "rb_route_batch_noalloc")


class RbError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {rb_status_string(status)} ({status})")


class rb_weights(ctypes.Structure):
    _fields_ = [("w_qual", ctypes.c_float), ("w_lat", ctypes.c_float), ("w_cost", ctypes.c_float)]


class rb_instances(ctypes.Structure):
    _fields_ = [("model", ctypes.c_void_p), ("prefill_q", ctypes.c_void_p),
                ("decode_q", ctypes.c_void_p), ("prefill_rate", ctypes.c_void_p),
                ("decode_rate", ctypes.c_void_p), ("price_in", ctypes.c_void_p),
                ("price_out", ctypes.c_void_p)]


class rb_options(ctypes.Structure):
    _fields_ = [("order", ctypes.c_int), ("weighting", ctypes.c_int), ("budget", ctypes.c_void_p),
                ("instance_mask", ctypes.c_void_p), ("order_out", ctypes.c_void_p),
                ("flags", ctypes.c_uint32)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2606_17949_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, i, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    st = ctypes.c_int
    sig = {
        "rb_status_string": ([st], ctypes.c_char_p),
        "rb_workspace_size": ([i, i, i, i, i, i, ctypes.POINTER(sz)], st),
        "rb_bank_norms": ([P, i, i, i, P, P], st),
        "rb_knn_topk": ([P, P, P, i, i, i, i, i, P, P, P, sz, P], st),
        "rb_predict": ([P, P, i, i, i, P, P, i, i, P, P, P], st),
        "rb_score": ([P, P, P, i, i, ctypes.POINTER(rb_instances), i, rb_weights, P, P], st),
        "rb_assign": ([P, P, P, i, i, ctypes.POINTER(rb_instances), i, rb_weights, P, P, P, P],
                      st),
        "rb_assign_ex": ([P, P, P, i, i, ctypes.POINTER(rb_instances), i, rb_weights,
                          ctypes.POINTER(rb_options), P, P, P, P], st),
        "rb_knn_predict": ([P, P, P, i, i, i, i, i, P, P, i, ctypes.POINTER(rb_options), P, P, P,
                            P, P, sz, P], st),
        "rb_route_batch": ([P, P, P, i, i, i, i, i, P, P, i, P, ctypes.POINTER(rb_instances), i,
                            rb_weights, P, P, P, P, P, P, P, P, sz, P], st),
        "rb_route_batch_ex": ([P, P, P, i, i, i, i, i, P, P, i, P, ctypes.POINTER(rb_instances),
                               i, rb_weights, ctypes.POINTER(rb_options), P, P, P, P, P, P, P, P,
                               sz, P], st),
        "rb_route_batch_noalloc": ([P, P, P, i, i, i, i, i, P, P, i, P,
                                    ctypes.POINTER(rb_instances), i, rb_weights, P, P, P, P, P,
                                    P, P, P], st),
        "rb_advance_state": ([ctypes.POINTER(rb_instances), i, ctypes.c_float, P], st),
        "rb_profile_scan_events": ([P, P], st),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    return lib


_lib = _load()


def rb_status_string(status: int) -> str:
    return _lib.rb_status_string(int(status)).decode()


def _check(status: int, where: str):
    if status != RB_OK:
        raise RbError(status, where)


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return ctypes.c_void_p(t.data_ptr()) if t.numel() else None


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return RB_F32
    if t.dtype == torch.bfloat16:
        return RB_BF16
    raise ValueError(f"unsupported embedding dtype {t.dtype}")


def _expect(t: torch.Tensor, dtype, shape, name):
    """dtype and shape of a tensor argument, checked before anything reaches
    the library (a short or mistyped buffer would be read or written out of
    bounds on the GPU)."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name}: expected a torch tensor, got {type(t).__name__}")
    if t.dtype != dtype:
        raise ValueError(f"{name}: expected {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")


def _expect_opt(t: Optional[torch.Tensor], dtype, shape, name):
    if t is not None:
        _expect(t, dtype, shape, name)


def _embeddings(queries, bank):
    """(B, N, d) of a query batch and a bank of the same dtype and width."""
    for t, name in ((queries, "queries"), (bank, "bank")):
        if not isinstance(t, torch.Tensor) or t.dim() != 2:
            raise ValueError(f"{name}: expected a 2-d tensor")
        if t.dtype not in (torch.float32, torch.bfloat16):
            raise ValueError(f"{name}: unsupported embedding dtype {t.dtype}")
    if queries.dtype != bank.dtype:
        raise ValueError(f"queries ({queries.dtype}) and bank ({bank.dtype}) must share a dtype")
    if queries.shape[1] != bank.shape[1]:
        raise ValueError(f"queries (d={queries.shape[1]}) and bank (d={bank.shape[1]}) must "
                         "share the embedding width")
    return int(queries.shape[0]), int(bank.shape[0]), int(bank.shape[1])


def _labels(bank_qual, bank_len, N):
    """M of the per-model label tables [N][M] fp32."""
    if not isinstance(bank_qual, torch.Tensor) or bank_qual.dim() != 2:
        raise ValueError("bank_qual: expected a 2-d tensor")
    M = int(bank_qual.shape[1])
    _expect(bank_qual, torch.float32, (N, M), "bank_qual")
    _expect(bank_len, torch.float32, (N, M), "bank_len")
    return M


def _predictions(q_hat, l_hat):
    """(B, M) of the prediction tables [B][M] fp32."""
    if not isinstance(q_hat, torch.Tensor) or q_hat.dim() != 2:
        raise ValueError("q_hat: expected a 2-d tensor")
    B, M = (int(x) for x in q_hat.shape)
    _expect(q_hat, torch.float32, (B, M), "q_hat")
    _expect(l_hat, torch.float32, (B, M), "l_hat")
    return B, M


@dataclasses.dataclass
class DeviceInstances:
    """Instance table on the GPU (struct of arrays, each of length I).

    ``prefill_q`` and ``decode_q`` are the dead-reckoned state that
    :func:`rb_assign`, :func:`rb_route_batch` and :func:`rb_advance_state`
    update in place.
    """
    model: torch.Tensor         # int32
    prefill_q: torch.Tensor     # fp32
    decode_q: torch.Tensor      # fp32
    prefill_rate: torch.Tensor  # fp32
    decode_rate: torch.Tensor   # fp32
    price_in: torch.Tensor      # fp32
    price_out: torch.Tensor     # fp32

    FIELDS = ("model", "prefill_q", "decode_q", "prefill_rate", "decode_rate", "price_in",
              "price_out")

    @property
    def I(self) -> int:
        return int(self.model.shape[0])

    @classmethod
    def from_host(cls, inst, device="cuda") -> "DeviceInstances":
        """From any object with numpy/torch fields named as in ``FIELDS``."""
        vals = {}
        for f in cls.FIELDS:
            dt = torch.int32 if f == "model" else torch.float32
            vals[f] = torch.as_tensor(getattr(inst, f)).to(device=device, dtype=dt).contiguous()
        return cls(**vals)

    def clone(self) -> "DeviceInstances":
        return DeviceInstances(*[getattr(self, f).clone() for f in self.FIELDS])

    def struct(self) -> rb_instances:
        I = self.I
        for f in self.FIELDS:
            t = getattr(self, f)
            _expect(t, torch.int32 if f == "model" else torch.float32, (I,), f)
        return rb_instances(*[_ptr(getattr(self, f)) for f in self.FIELDS])


def rb_workspace_size(B: int, N: int, d: int, dtype: int, k: int, M: int) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib.rb_workspace_size(B, N, d, dtype, k, M, ctypes.byref(n)), "rb_workspace_size")
    return int(n.value)


def workspace(B: int, N: int, d: int, dtype: int, k: int, M: int, device="cuda") -> torch.Tensor:
    """A device workspace of the size rb_workspace_size asks for."""
    n = rb_workspace_size(B, N, d, dtype, k, M)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=device)


def rb_bank_norms(bank: torch.Tensor, norms: Optional[torch.Tensor] = None, stream=None):
    if not isinstance(bank, torch.Tensor) or bank.dim() != 2 or \
            bank.dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("bank: expected a 2-d fp32 or bf16 tensor")
    N, d = bank.shape
    if norms is None:
        norms = torch.empty(N, dtype=torch.float32, device=bank.device)
    _expect(norms, torch.float32, (N,), "norms")
    _check(_lib.rb_bank_norms(_ptr(bank), _dtype_code(bank), N, d, _ptr(norms), _stream(stream)),
           "rb_bank_norms")
    return norms


def rb_knn_topk(queries: torch.Tensor, bank: torch.Tensor, bank_norms: torch.Tensor, k: int,
                nbr_idx: Optional[torch.Tensor] = None, nbr_dist: Optional[torch.Tensor] = None,
                ws: Optional[torch.Tensor] = None, stream=None, want_dist: bool = True):
    B, N, d = _embeddings(queries, bank)
    _expect(bank_norms, torch.float32, (N,), "bank_norms")
    _expect_opt(nbr_idx, torch.int32, (B, k), "nbr_idx")
    _expect_opt(nbr_dist, torch.float32, (B, k), "nbr_dist")
    _expect_opt(ws, torch.uint8, (ws.numel(),) if ws is not None else (), "ws")
    dev = queries.device
    if nbr_idx is None:
        nbr_idx = torch.empty(B, k, dtype=torch.int32, device=dev)
    if nbr_dist is None and want_dist:
        nbr_dist = torch.empty(B, k, dtype=torch.float32, device=dev)
    if ws is None:
        ws = workspace(B, N, d, _dtype_code(bank), k, 1, dev)
    _check(_lib.rb_knn_topk(_ptr(queries), _ptr(bank), _ptr(bank_norms), _dtype_code(bank), B, N,
                            d, k, _ptr(nbr_idx), _ptr(nbr_dist), _ptr(ws), ws.numel(),
                            _stream(stream)), "rb_knn_topk")
    return nbr_idx, nbr_dist


def rb_predict(nbr_idx: torch.Tensor, bank_qual: torch.Tensor, bank_len: torch.Tensor,
               nbr_dist: Optional[torch.Tensor] = None, weighting: int = RB_KNN_UNIFORM,
               q_hat: Optional[torch.Tensor] = None, l_hat: Optional[torch.Tensor] = None,
               stream=None):
    if not isinstance(nbr_idx, torch.Tensor) or nbr_idx.dim() != 2:
        raise ValueError("nbr_idx: expected a 2-d tensor")
    B, k = (int(x) for x in nbr_idx.shape)
    _expect(nbr_idx, torch.int32, (B, k), "nbr_idx")
    if not isinstance(bank_qual, torch.Tensor) or bank_qual.dim() != 2:
        raise ValueError("bank_qual: expected a 2-d tensor")
    N = int(bank_qual.shape[0])
    M = _labels(bank_qual, bank_len, N)
    _expect_opt(nbr_dist, torch.float32, (B, k), "nbr_dist")
    _expect_opt(q_hat, torch.float32, (B, M), "q_hat")
    _expect_opt(l_hat, torch.float32, (B, M), "l_hat")
    dev = nbr_idx.device
    if q_hat is None:
        q_hat = torch.empty(B, M, dtype=torch.float32, device=dev)
    if l_hat is None:
        l_hat = torch.empty(B, M, dtype=torch.float32, device=dev)
    _check(_lib.rb_predict(_ptr(nbr_idx), _ptr(nbr_dist), B, k, int(weighting), _ptr(bank_qual),
                           _ptr(bank_len), N, M, _ptr(q_hat), _ptr(l_hat), _stream(stream)),
           "rb_predict")
    return q_hat, l_hat


def _w(weights) -> rb_weights:
    return rb_weights(*[float(x) for x in weights])


def _request_args(q_hat, l_hat, prompt_len):
    B, M = _predictions(q_hat, l_hat)
    _expect(prompt_len, torch.int32, (B,), "prompt_len")
    return B, M


def rb_score(q_hat, l_hat, prompt_len, inst: DeviceInstances, weights,
             score0: Optional[torch.Tensor] = None, stream=None):
    B, M = _request_args(q_hat, l_hat, prompt_len)
    I = inst.I
    _expect_opt(score0, torch.float32, (B, I), "score0")
    if score0 is None:
        score0 = torch.empty(B, I, dtype=torch.float32, device=q_hat.device)
    s = inst.struct()
    _check(_lib.rb_score(_ptr(q_hat), _ptr(l_hat), _ptr(prompt_len), B, M, ctypes.byref(s), I,
                         _w(weights), _ptr(score0), _stream(stream)), "rb_score")
    return score0


def _assign_outputs(B, I, dev, assign, chosen, decided, want_chosen):
    _expect_opt(assign, torch.int32, (B,), "assign")
    _expect_opt(chosen, torch.float32, (B,), "chosen")
    _expect_opt(decided, torch.float32, (B, I), "decided")
    if assign is None:
        assign = torch.empty(B, dtype=torch.int32, device=dev)
    if chosen is None and want_chosen:
        chosen = torch.empty(B, dtype=torch.float32, device=dev)
    return assign, chosen


def rb_assign(q_hat, l_hat, prompt_len, inst: DeviceInstances, weights,
              assign: Optional[torch.Tensor] = None, chosen: Optional[torch.Tensor] = None,
              stream=None, want_chosen: bool = True, decided: Optional[torch.Tensor] = None):
    """Greedy assignment; ``decided`` [B][I] fp32, when given, receives the
    Eq. 1 row each request was decided on."""
    B, M = _request_args(q_hat, l_hat, prompt_len)
    assign, chosen = _assign_outputs(B, inst.I, q_hat.device, assign, chosen, decided,
                                     want_chosen)
    s = inst.struct()
    _check(_lib.rb_assign(_ptr(q_hat), _ptr(l_hat), _ptr(prompt_len), B, M, ctypes.byref(s),
                          inst.I, _w(weights), _ptr(assign), _ptr(chosen), _ptr(decided),
                          _stream(stream)), "rb_assign")
    return assign, chosen


def _route_args(queries, bank, bank_norms, k, bank_qual, bank_len, prompt_len, inst, ws,
                nbr_idx, nbr_dist, q_hat, l_hat, score0, chosen, assign):
    B, N, d = _embeddings(queries, bank)
    _expect(bank_norms, torch.float32, (N,), "bank_norms")
    M = _labels(bank_qual, bank_len, N)
    _expect(prompt_len, torch.int32, (B,), "prompt_len")
    _expect_opt(nbr_idx, torch.int32, (B, k), "nbr_idx")
    _expect_opt(nbr_dist, torch.float32, (B, k), "nbr_dist")
    _expect_opt(q_hat, torch.float32, (B, M), "q_hat")
    _expect_opt(l_hat, torch.float32, (B, M), "l_hat")
    _expect_opt(score0, torch.float32, (B, inst.I), "score0")
    _expect_opt(chosen, torch.float32, (B,), "chosen")
    _expect_opt(assign, torch.int32, (B,), "assign")
    _expect_opt(ws, torch.uint8, (ws.numel(),) if ws is not None else (), "ws")
    return B, N, d, M


def rb_route_batch(queries, bank, bank_norms, k: int, bank_qual, bank_len, prompt_len,
                   inst: DeviceInstances, weights, ws: Optional[torch.Tensor] = None,
                   assign: Optional[torch.Tensor] = None, chosen: Optional[torch.Tensor] = None,
                   nbr_idx: Optional[torch.Tensor] = None, nbr_dist: Optional[torch.Tensor] = None,
                   q_hat: Optional[torch.Tensor] = None, l_hat: Optional[torch.Tensor] = None,
                   stream=None, score0: Optional[torch.Tensor] = None):
    """The fused path; intermediates are returned only if the caller passes buffers."""
    B, N, d, M = _route_args(queries, bank, bank_norms, k, bank_qual, bank_len, prompt_len, inst,
                             ws, nbr_idx, nbr_dist, q_hat, l_hat, score0, chosen, assign)
    dev = queries.device
    if assign is None:
        assign = torch.empty(B, dtype=torch.int32, device=dev)
    if ws is None:
        ws = workspace(B, N, d, _dtype_code(bank), k, M, dev)
    s = inst.struct()
    _check(_lib.rb_route_batch(_ptr(queries), _ptr(bank), _ptr(bank_norms), _dtype_code(bank), B,
                               N, d, k, _ptr(bank_qual), _ptr(bank_len), M, _ptr(prompt_len),
                               ctypes.byref(s), inst.I, _w(weights), _ptr(assign), _ptr(chosen),
                               _ptr(nbr_idx), _ptr(nbr_dist), _ptr(q_hat), _ptr(l_hat),
                               _ptr(score0), _ptr(ws), ws.numel(), _stream(stream)),
           "rb_route_batch")
    return assign


def rb_route_batch_noalloc(queries, bank, bank_norms, k: int, bank_qual, bank_len, prompt_len,
                           inst: DeviceInstances, weights, assign: Optional[torch.Tensor] = None,
                           chosen: Optional[torch.Tensor] = None,
                           nbr_idx: Optional[torch.Tensor] = None,
                           nbr_dist: Optional[torch.Tensor] = None,
                           q_hat: Optional[torch.Tensor] = None,
                           l_hat: Optional[torch.Tensor] = None, stream=None,
                           score0: Optional[torch.Tensor] = None):
    """rb_route_batch on the library's static per-GPU workspace (no device
    allocation by the library; ``assign`` should be passed in by callers that
    cannot allocate, since otherwise this wrapper allocates it)."""
    B, N, d, M = _route_args(queries, bank, bank_norms, k, bank_qual, bank_len, prompt_len, inst,
                             None, nbr_idx, nbr_dist, q_hat, l_hat, score0, chosen, assign)
    if assign is None:
        assign = torch.empty(B, dtype=torch.int32, device=queries.device)
    s = inst.struct()
    _check(_lib.rb_route_batch_noalloc(_ptr(queries), _ptr(bank), _ptr(bank_norms),
                                       _dtype_code(bank), B, N, d, k, _ptr(bank_qual),
                                       _ptr(bank_len), M, _ptr(prompt_len), ctypes.byref(s),
                                       inst.I, _w(weights), _ptr(assign), _ptr(chosen),
                                       _ptr(nbr_idx), _ptr(nbr_dist), _ptr(q_hat), _ptr(l_hat),
                                       _ptr(score0), _stream(stream)), "rb_route_batch_noalloc")
    return assign


def options(order: int = RB_ORDER_ARRIVAL, weighting: int = RB_KNN_UNIFORM,
            budget: Optional[torch.Tensor] = None, instance_mask: Optional[torch.Tensor] = None,
            order_out: Optional[torch.Tensor] = None, flags: int = 0) -> rb_options:
    """An rb_options struct; budget fp32 [B], instance_mask uint8 [I], order_out int32 [B].

    The struct holds references to the tensors, so their memory stays
    allocated for as long as the struct lives."""
    for t, dt, name in ((budget, torch.float32, "budget"), (instance_mask, torch.uint8,
                                                          "instance_mask"),
                        (order_out, torch.int32, "order_out")):
        if t is not None and t.dtype != dt:
            raise ValueError(f"{name}: expected {dt}, got {t.dtype}")
        if t is not None and not t.is_cuda:
            raise ValueError(f"{name}: must live on the GPU")
    o = rb_options(int(order), int(weighting), _ptr(budget), _ptr(instance_mask),
                   _ptr(order_out), int(flags))
    o._tensors = (budget, instance_mask, order_out)
    return o


def _check_opts(opts: rb_options, B: int, I: int):
    """The option arrays must cover the batch and the instance table."""
    budget, mask, order_out = getattr(opts, "_tensors", (None, None, None))
    for t, n, name in ((budget, B, "budget"), (mask, I, "instance_mask"),
                       (order_out, B, "order_out")):
        if t is not None and t.numel() != n:
            raise ValueError(f"{name}: expected {n} elements, got {t.numel()}")


def rb_assign_ex(q_hat, l_hat, prompt_len, inst: DeviceInstances, weights, opts: rb_options,
                 assign: Optional[torch.Tensor] = None, chosen: Optional[torch.Tensor] = None,
                 stream=None, want_chosen: bool = True, decided: Optional[torch.Tensor] = None):
    B, M = _request_args(q_hat, l_hat, prompt_len)
    assign, chosen = _assign_outputs(B, inst.I, q_hat.device, assign, chosen, decided,
                                     want_chosen)
    _check_opts(opts, B, inst.I)
    s = inst.struct()
    _check(_lib.rb_assign_ex(_ptr(q_hat), _ptr(l_hat), _ptr(prompt_len), B, M, ctypes.byref(s),
                             inst.I, _w(weights), ctypes.byref(opts), _ptr(assign), _ptr(chosen),
                             _ptr(decided), _stream(stream)), "rb_assign_ex")
    return assign, chosen


def rb_knn_predict(queries, bank, bank_norms, k: int, bank_qual, bank_len,
                   opts: Optional[rb_options] = None, ws: Optional[torch.Tensor] = None,
                   q_hat: Optional[torch.Tensor] = None, l_hat: Optional[torch.Tensor] = None,
                   nbr_idx: Optional[torch.Tensor] = None, nbr_dist: Optional[torch.Tensor] = None,
                   stream=None):
    """KNN lookup and label average in one call: returns (q_hat, l_hat).

    With RB_FLAG_LISTS_ONLY in ``opts.flags`` only the seed and the bank scan
    run (their lists stay in ``ws``; returns (None, None) unless buffers are
    given); with RB_FLAG_FROM_LISTS only the merge and average of the lists a
    LISTS_ONLY call left in ``ws`` (the same shapes and overlap flag)."""
    B, N, d = _embeddings(queries, bank)
    _expect(bank_norms, torch.float32, (N,), "bank_norms")
    M = _labels(bank_qual, bank_len, N)
    _expect_opt(q_hat, torch.float32, (B, M), "q_hat")
    _expect_opt(l_hat, torch.float32, (B, M), "l_hat")
    _expect_opt(nbr_idx, torch.int32, (B, k), "nbr_idx")
    _expect_opt(nbr_dist, torch.float32, (B, k), "nbr_dist")
    _expect_opt(ws, torch.uint8, (ws.numel(),) if ws is not None else (), "ws")
    dev = queries.device
    lists_only = opts is not None and (opts.flags & RB_FLAG_LISTS_ONLY)
    if q_hat is None and not lists_only:
        q_hat = torch.empty(B, M, dtype=torch.float32, device=dev)
    if l_hat is None and not lists_only:
        l_hat = torch.empty(B, M, dtype=torch.float32, device=dev)
    if ws is None:
        ws = workspace(B, N, d, _dtype_code(bank), k, M, dev)
    _check(_lib.rb_knn_predict(_ptr(queries), _ptr(bank), _ptr(bank_norms), _dtype_code(bank), B,
                               N, d, k, _ptr(bank_qual), _ptr(bank_len), M,
                               ctypes.byref(opts) if opts is not None else None, _ptr(nbr_idx),
                               _ptr(nbr_dist), _ptr(q_hat), _ptr(l_hat), _ptr(ws), ws.numel(),
                               _stream(stream)), "rb_knn_predict")
    return q_hat, l_hat


def rb_route_batch_ex(queries, bank, bank_norms, k: int, bank_qual, bank_len, prompt_len,
                      inst: DeviceInstances, weights, opts: rb_options,
                      ws: Optional[torch.Tensor] = None, assign: Optional[torch.Tensor] = None,
                      chosen: Optional[torch.Tensor] = None,
                      nbr_idx: Optional[torch.Tensor] = None,
                      nbr_dist: Optional[torch.Tensor] = None,
                      q_hat: Optional[torch.Tensor] = None, l_hat: Optional[torch.Tensor] = None,
                      stream=None, score0: Optional[torch.Tensor] = None):
    """rb_route_batch with options (order, weighting, budgets, availability)."""
    B, N, d, M = _route_args(queries, bank, bank_norms, k, bank_qual, bank_len, prompt_len, inst,
                             ws, nbr_idx, nbr_dist, q_hat, l_hat, score0, chosen, assign)
    dev = queries.device
    if assign is None:
        assign = torch.empty(B, dtype=torch.int32, device=dev)
    if ws is None:
        ws = workspace(B, N, d, _dtype_code(bank), k, M, dev)
    _check_opts(opts, B, inst.I)
    s = inst.struct()
    _check(_lib.rb_route_batch_ex(_ptr(queries), _ptr(bank), _ptr(bank_norms), _dtype_code(bank),
                                  B, N, d, k, _ptr(bank_qual), _ptr(bank_len), M,
                                  _ptr(prompt_len), ctypes.byref(s), inst.I, _w(weights),
                                  ctypes.byref(opts), _ptr(assign), _ptr(chosen), _ptr(nbr_idx),
                                  _ptr(nbr_dist), _ptr(q_hat), _ptr(l_hat), _ptr(score0),
                                  _ptr(ws), ws.numel(), _stream(stream)), "rb_route_batch_ex")
    return assign


def rb_advance_state(inst: DeviceInstances, dt_seconds: float, stream=None):
    s = inst.struct()
    _check(_lib.rb_advance_state(ctypes.byref(s), inst.I, float(dt_seconds), _stream(stream)),
           "rb_advance_state")


def rb_profile_scan_events(begin=None, end=None):
    """Record torch.cuda.Event ``begin``/``end`` around every later bank-scan
    kernel launched from this thread; ``None, None`` stops."""
    b = ctypes.c_void_p(begin.cuda_event) if begin is not None else None
    e = ctypes.c_void_p(end.cuda_event) if end is not None else None
    _check(_lib.rb_profile_scan_events(b, e), "rb_profile_scan_events")
