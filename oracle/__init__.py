"""CPU oracle for the RouteBalance routing path (arXiv 2606.17949).

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg may import this package; the product path never
does. It shares no code with the GPU library ``paper_2606_17949_amd`` and does
not import it.

The arithmetic lives in ``rb_oracle.c`` (plain C, fp64, scalar loops); this
module compiles it with gcc on first use and marshals numpy arrays to it.
Every function follows the passage named in the C source:
  knn      -- exact k nearest neighbours (Sec. 4.2, KNN lookup of Alg. 1)
  predict  -- KNN mean of per-model quality and length labels, plain or
              inverse-distance weighted (Sec. 4.2)
  score    -- dense score matrix at the batch-start state (Eq. 1, Eq. 2)
  score_row-- one request's scores, latencies, costs and candidate set at a
              given state (Eq. 1, Eq. 2, the budget filter of Alg. 1)
  lpt_order-- longest-predicted-first processing order (Alg. 1, Sec. 4.1)
  assign   -- greedy assignment with dead reckoning, in arrival or LPT order,
              over each request's candidate set (Alg. 1, Sec. 4.1-4.2)
  advance  -- drain the state over an inter-batch gap (clamped linear drain)
  batch_matching -- the exact batch-level matching on a logged score matrix
              that Sec. 4.1 compares the greedy with (Hungarian method)
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
                               "-ffp-contract=off", "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"])
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
            lib.oracle_predict_ex.argtypes = [P, P, i, i, P, P, i, i, i, P, P]
            lib.oracle_score_row.argtypes = [P, P, i, dbl, P, P, P, P, P, P, P, i, dbl, dbl, dbl,
                                             P, P, P]
            lib.oracle_score_row_ex.argtypes = [P, P, i, dbl, P, P, P, P, P, P, P, i, dbl, dbl,
                                                dbl, P, P, P, P, P, P]
            lib.oracle_score.argtypes = [P, P, P, i, i, P, P, P, P, P, P, P, i, dbl, dbl, dbl, P]
            lib.oracle_lpt_order.argtypes = [P, i, i, P]
            lib.oracle_assign.argtypes = [P, P, P, i, i, P, P, P, P, P, P, P, i, dbl, dbl, dbl,
                                          P, P, P, P]
            lib.oracle_assign_ex.argtypes = [P, P, P, i, i, P, P, P, P, P, P, P, i, dbl, dbl, dbl,
                                             i, P, P, P, P, P, P, P]
            lib.oracle_advance.argtypes = [P, P, P, P, i, dbl]
            for f in ("oracle_knn", "oracle_predict", "oracle_predict_ex", "oracle_score_row",
                      "oracle_score_row_ex", "oracle_score", "oracle_lpt_order", "oracle_assign",
                      "oracle_assign_ex", "oracle_advance"):
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


WEIGHTINGS = {"uniform": 0, "inv_dist": 1}
ORDERS = ("arrival", "lpt")


def predict(nbr, qual, length, dist=None, weighting: str = "uniform"):
    """KNN-averaged predictions (q_hat, l_hat), fp64 [B][M].

    ``weighting`` "uniform": the plain mean; "inv_dist": weights
    1/(sqrt(max(dist, 0)) + 1e-6) from the squared distances ``dist`` [B][k],
    normalised to sum 1.
    """
    nbr = _c(nbr, np.int32)
    qual = _c(qual, np.float32)
    length = _c(length, np.float32)
    B, k = nbr.shape
    N, M = qual.shape
    wmode = WEIGHTINGS[weighting]
    dd = None
    if wmode:
        dd = _c(dist, np.float64)
        if dd.shape != nbr.shape:
            raise ValueError("dist must have the shape of nbr")
    qh = np.zeros((B, M))
    lh = np.zeros((B, M))
    _check(_load().oracle_predict_ex(_ptr(nbr), _ptr(dd) if wmode else None, B, k, _ptr(qual),
                                     _ptr(length), N, M, wmode, _ptr(qh), _ptr(lh)),
           "oracle_predict_ex")
    return qh, lh


def _inst_arrays(inst):
    return (_c(inst.model, np.int32), _c(inst.prefill_q, np.float64), _c(inst.decode_q, np.float64),
            _c(inst.prefill_rate, np.float64), _c(inst.decode_rate, np.float64),
            _c(inst.price_in, np.float64), _c(inst.price_out, np.float64))


def score_row(q_hat_r, l_hat_r, plen, inst, p, a, weights, budget_r=None, mask=None,
              with_candidates=False):
    """Scores, latencies and costs of one request at state (p, a): (S, T, C) fp64 [I].

    ``budget_r`` (a scalar) and ``mask`` [I] restrict the candidate set; the
    maxima run over the candidates and the others score NaN. With
    ``with_candidates`` the candidate flags (bool [I]) are returned too.
    """
    model, _, _, P, D, cin, cout = _inst_arrays(inst)
    q = _c(q_hat_r, np.float64)
    l = _c(l_hat_r, np.float64)
    p = _c(p, np.float64)
    a = _c(a, np.float64)
    I = model.shape[0]
    S, T, C = np.zeros(I), np.zeros(I), np.zeros(I)
    cand = np.zeros(I, dtype=np.uint8)
    b = None if budget_r is None else np.array([budget_r], dtype=np.float32)
    mk = None if mask is None else _c(mask, np.uint8)
    _check(_load().oracle_score_row_ex(_ptr(q), _ptr(l), q.shape[0], float(plen), _ptr(model),
                                       _ptr(p), _ptr(a), _ptr(P), _ptr(D), _ptr(cin), _ptr(cout),
                                       I, *map(float, weights), _ptr(b) if b is not None else None,
                                       _ptr(mk) if mk is not None else None, _ptr(S), _ptr(T),
                                       _ptr(C), _ptr(cand)), "oracle_score_row_ex")
    if with_candidates:
        return S, T, C, cand.astype(bool)
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


def lpt_order(l_hat):
    """Longest-predicted-first order of the batch: int32 [B] request indices."""
    lh = _c(l_hat, np.float64)
    B, M = lh.shape
    order = np.zeros(B, dtype=np.int32)
    _check(_load().oracle_lpt_order(_ptr(lh), B, M, _ptr(order)), "oracle_lpt_order")
    return order


def assign(q_hat, l_hat, plen, inst, weights, p=None, a=None, trace=False, order="arrival",
           budget=None, mask=None):
    """Greedy assignment with dead reckoning.

    Starts from (p, a) if given (fp64), else from the instances' fp32 state.
    ``order`` is "arrival" or "lpt"; ``budget`` [B] (fp32 per-request cost
    budgets) and ``mask`` [I] (nonzero = available) restrict each request's
    candidate set, and a request without candidates gets -1.
    Returns dict(assign int32 [B], chosen fp64 [B], order int32 [B], p, a final
    fp64 [I]) and, with ``trace``, trace_p / trace_a fp64 [B+1][I] (state
    before each step, in processing order).
    """
    if order not in ORDERS:
        raise ValueError(f"order must be one of {ORDERS}")
    model, p0, a0, P, D, cin, cout = _inst_arrays(inst)
    p = _c(p0 if p is None else p, np.float64).copy()
    a = _c(a0 if a is None else a, np.float64).copy()
    qh = _c(q_hat, np.float64)
    lh = _c(l_hat, np.float64)
    pl = _c(plen, np.int32)
    B, M = qh.shape
    I = model.shape[0]
    bud = None if budget is None else _c(budget, np.float32)
    mk = None if mask is None else _c(mask, np.uint8)
    if bud is not None and bud.shape != (B,):
        raise ValueError("budget must have shape [B]")
    if mk is not None and mk.shape != (I,):
        raise ValueError("mask must have shape [I]")
    out = np.zeros(B, dtype=np.int32)
    chosen = np.zeros(B)
    ordr = np.zeros(B, dtype=np.int32)
    tp = np.zeros((B + 1, I)) if trace else None
    ta = np.zeros((B + 1, I)) if trace else None
    _check(_load().oracle_assign_ex(_ptr(qh), _ptr(lh), _ptr(pl), B, M, _ptr(model), _ptr(p),
                                    _ptr(a), _ptr(P), _ptr(D), _ptr(cin), _ptr(cout), I,
                                    *map(float, weights), int(order == "lpt"),
                                    _ptr(bud) if bud is not None else None,
                                    _ptr(mk) if mk is not None else None, _ptr(out),
                                    _ptr(chosen), _ptr(ordr), _ptr(tp) if trace else None,
                                    _ptr(ta) if trace else None), "oracle_assign_ex")
    res = {"assign": out, "chosen": chosen, "order": ordr, "p": p, "a": a}
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


def batch_matching(S0, capacity):
    """Exact batch-level matching on a logged batch-start score matrix.

    Sec. 4.1 compares the greedy pass with a batch-level matching (e.g. the
    Hungarian method) over the logged score matrices: each request goes to
    one instance, scored at the batch-start state (no within-batch updates),
    maximising the total score. The paper gives no instance capacity; here
    instance i offers ``capacity`` slots (an int, or an int array [I]), and
    the matching is the linear assignment of the B requests to the slots.
    With capacity >= B it reduces to the row-wise argmax of S0 (lowest
    instance on ties). Non-finite entries of S0 (non-candidates) are never
    matched while a finite choice remains.

    Returns int32 [B] instance per request. The assignment step is scipy's
    linear_sum_assignment (a library primitive for the Hungarian problem).
    """
    from scipy.optimize import linear_sum_assignment

    S0 = np.asarray(S0, np.float64)
    B, I = S0.shape
    cap = np.broadcast_to(np.asarray(capacity, np.int64), (I,))
    if np.any(cap < 0) or cap.sum() < B:
        raise ValueError("the slots must cover the batch")
    if B == 0:
        return np.zeros(0, np.int32)
    if np.all(cap >= B):
        # every request takes its best instance
        V = np.where(np.isfinite(S0), S0, -np.inf)
        return np.argmax(V, axis=1).astype(np.int32)
    cols = np.repeat(np.arange(I), np.minimum(cap, B))
    finite = np.isfinite(S0)
    span = (np.abs(S0[finite]).max() if finite.any() else 1.0) + 1.0
    # a non-candidate costs more than any total of finite scores can regain
    V = np.where(finite, S0, -(2.0 * span * (B + 1)))
    rows, c = linear_sum_assignment(-V[:, cols])
    out = np.empty(B, np.int32)
    out[rows] = cols[c]
    return out
