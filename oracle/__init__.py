"""CPU oracle for the RouteBalance routing path (arXiv 2606.17949).

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg may import this package; the product path never
does. It shares no code with the GPU library ``paper_2606_17949_amd`` and does
not import it.

The arithmetic lives in ``rb_oracle.c`` (plain C, fp64, scalar loops); this
module compiles it with gcc on first use and marshals numpy arrays to it.
Every function follows the passage named in the C source:
  knn      -- exact k nearest neighbours (Sec. 4.2, KNN lookup of Alg. 1)
  predict  -- uniform KNN mean of per-model quality and length labels (Sec. 4.2)
  score    -- dense score matrix at the batch-start state (Eq. 1, Eq. 2)
  score_row-- one request's scores, latencies and costs at a given state
  assign   -- greedy arrival-order assignment with dead reckoning (Alg. 1, Sec. 4.1-4.2)
  advance  -- drain the state over an inter-batch gap (clamped linear drain)
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "rb_oracle.c")
_LIB = os.path.join(_HERE, "librb_oracle.so")
# A mutant build of the oracle, used only by the mutation test that checks the
# pins fail when a mistake is planted in the oracle.
_LIB_OVERRIDE = os.environ.get("RB_ORACLE_LIB")
_lock = threading.Lock()
_lib = None

F32, BF16 = 0, 1


def build(force: bool = False) -> str:
    """Compile the oracle shared library with gcc (no GPU code involved)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread",
                               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if _LIB_OVERRIDE:
                lib = ctypes.CDLL(_LIB_OVERRIDE)
            else:
                build()
                lib = ctypes.CDLL(_LIB)
            P = ctypes.c_void_p
            i = ctypes.c_int
            dbl = ctypes.c_double
            lib.oracle_knn.argtypes = [P, P, i, i, i, i, i, P, P, i]
            lib.oracle_predict.argtypes = [P, i, i, P, P, i, i, P, P]
            lib.oracle_score_row.argtypes = [P, P, i, dbl, P, P, P, P, P, P, P, i, dbl, dbl, dbl,
                                             P, P, P]
            lib.oracle_score.argtypes = [P, P, P, i, i, P, P, P, P, P, P, P, i, dbl, dbl, dbl, P]
            lib.oracle_assign.argtypes = [P, P, P, i, i, P, P, P, P, P, P, P, i, dbl, dbl, dbl,
                                          P, P, P, P]
            lib.oracle_advance.argtypes = [P, P, P, P, i, dbl]
            for f in ("oracle_knn", "oracle_predict", "oracle_score_row", "oracle_score",
                      "oracle_assign", "oracle_advance"):
                getattr(lib, f).restype = ctypes.c_int
            _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _check(rc, name):
    if rc != 0:
        raise ValueError(f"{name}: invalid arguments (rc={rc})")


def _as_storage(x):
    """Accept a numpy array or a CPU torch tensor; bf16 is passed as its raw bits."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            x = x.detach().cpu().contiguous()
            if x.dtype == torch.bfloat16:
                return x.view(torch.int16).numpy().view(np.uint16), BF16
            return _c(x.numpy(), np.float32), F32
    except ImportError:  # pragma: no cover
        pass
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return np.ascontiguousarray(x), BF16
    return _c(x, np.float32), F32


def knn(queries, bank, k: int, nthreads: int = 1):
    """Exact k-NN under (squared L2 ascending, bank index ascending).

    ``queries`` [B][d] and ``bank`` [N][d], both fp32 or both bf16 (torch bf16
    tensors or uint16 bit arrays). Returns (idx int32 [B][k], dist fp64 [B][k]).
    """
    q, dq = _as_storage(queries)
    x, dx = _as_storage(bank)
    if dq != dx:
        raise ValueError("queries and bank must share a dtype")
    B, d = q.shape
    N, d2 = x.shape
    if d != d2:
        raise ValueError("dimension mismatch")
    idx = np.zeros((B, k), dtype=np.int32)
    dist = np.zeros((B, k), dtype=np.float64)
    _check(_load().oracle_knn(_ptr(q), _ptr(x), dq, B, N, d, k, _ptr(idx), _ptr(dist),
                              int(nthreads)), "oracle_knn")
    return idx, dist


def predict(nbr, qual, length):
    """Uniform mean of the neighbours' labels: (q_hat, l_hat), fp64 [B][M]."""
    nbr = _c(nbr, np.int32)
    qual = _c(qual, np.float32)
    length = _c(length, np.float32)
    B, k = nbr.shape
    N, M = qual.shape
    qh = np.zeros((B, M))
    lh = np.zeros((B, M))
    _check(_load().oracle_predict(_ptr(nbr), B, k, _ptr(qual), _ptr(length), N, M, _ptr(qh),
                                  _ptr(lh)), "oracle_predict")
    return qh, lh


def _inst_arrays(inst):
    return (_c(inst.model, np.int32), _c(inst.prefill_q, np.float64), _c(inst.decode_q, np.float64),
            _c(inst.prefill_rate, np.float64), _c(inst.decode_rate, np.float64),
            _c(inst.price_in, np.float64), _c(inst.price_out, np.float64))


def score_row(q_hat_r, l_hat_r, plen, inst, p, a, weights):
    """Scores, latencies and costs of one request at state (p, a): (S, T, C) fp64 [I]."""
    model, _, _, P, D, cin, cout = _inst_arrays(inst)
    q = _c(q_hat_r, np.float64)
    l = _c(l_hat_r, np.float64)
    p = _c(p, np.float64)
    a = _c(a, np.float64)
    I = model.shape[0]
    S, T, C = np.zeros(I), np.zeros(I), np.zeros(I)
    _check(_load().oracle_score_row(_ptr(q), _ptr(l), q.shape[0], float(plen), _ptr(model),
                                    _ptr(p), _ptr(a), _ptr(P), _ptr(D), _ptr(cin), _ptr(cout), I,
                                    *map(float, weights), _ptr(S), _ptr(T), _ptr(C)),
           "oracle_score_row")
    return S, T, C


def score(q_hat, l_hat, plen, inst, weights):
    """Dense score matrix S0 [B][I] (fp64) at the instances' current state."""
    model, p, a, P, D, cin, cout = _inst_arrays(inst)
    qh = _c(q_hat, np.float64)
    lh = _c(l_hat, np.float64)
    pl = _c(plen, np.int32)
    B, M = qh.shape
    I = model.shape[0]
    S0 = np.zeros((B, I))
    _check(_load().oracle_score(_ptr(qh), _ptr(lh), _ptr(pl), B, M, _ptr(model), _ptr(p), _ptr(a),
                                _ptr(P), _ptr(D), _ptr(cin), _ptr(cout), I, *map(float, weights),
                                _ptr(S0)), "oracle_score")
    return S0


def assign(q_hat, l_hat, plen, inst, weights, p=None, a=None, trace=False):
    """Greedy arrival-order assignment.

    Starts from (p, a) if given (fp64), else from the instances' fp32 state.
    Returns dict(assign int32 [B], chosen fp64 [B], p, a final fp64 [I]) and,
    with ``trace``, trace_p / trace_a fp64 [B+1][I] (state before each step).
    """
    model, p0, a0, P, D, cin, cout = _inst_arrays(inst)
    p = _c(p0 if p is None else p, np.float64).copy()
    a = _c(a0 if a is None else a, np.float64).copy()
    qh = _c(q_hat, np.float64)
    lh = _c(l_hat, np.float64)
    pl = _c(plen, np.int32)
    B, M = qh.shape
    I = model.shape[0]
    out = np.zeros(B, dtype=np.int32)
    chosen = np.zeros(B)
    tp = np.zeros((B + 1, I)) if trace else None
    ta = np.zeros((B + 1, I)) if trace else None
    _check(_load().oracle_assign(_ptr(qh), _ptr(lh), _ptr(pl), B, M, _ptr(model), _ptr(p), _ptr(a),
                                 _ptr(P), _ptr(D), _ptr(cin), _ptr(cout), I, *map(float, weights),
                                 _ptr(out), _ptr(chosen), _ptr(tp) if trace else None,
                                 _ptr(ta) if trace else None), "oracle_assign")
    res = {"assign": out, "chosen": chosen, "p": p, "a": a}
    if trace:
        res["trace_p"], res["trace_a"] = tp, ta
    return res


def advance(p, a, prefill_rate, decode_rate, dt):
    """State after a gap of ``dt`` seconds: (p, a) fp64 [I]."""
    p = _c(p, np.float64).copy()
    a = _c(a, np.float64).copy()
    P = _c(prefill_rate, np.float64)
    D = _c(decode_rate, np.float64)
    _check(_load().oracle_advance(_ptr(p), _ptr(a), _ptr(P), _ptr(D), p.shape[0], float(dt)),
           "oracle_advance")
    return p, a
