"""fp64 CPU oracle for HeadWiseKV's grouped-cache runtime (ctypes over oracle.c).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, the smoke check and the
benchmark's CPU-baseline leg may import this package.  It shares no code with
the HIP library: it loads its own ``liboracle.so`` built from ``oracle.c``.

What it computes, and the passage each part follows (all definitions are
restated in ``oracle.c``):

* residency ``R(n) = {p < S} U {p >= n - w}`` -- window semantics J_t(w)
  (Method, sequential calibration) with the additive sink prefix of the
  sink+recent control (Appendix, baseline controls);
* capacity and accounting -- r_C(w), Eq. nominal-storage, Eq. normalized-rate
  (Method, structured residency model);
* the slot table after prefill materialisation and appends (canonical ring
  slot rule, a reading of an unspecified arrangement);
* attention outputs -- Eqs. conditional-attention-weight and
  conditional-attention, fp64, over the retained set;
* the calibration replay -- candidate outputs o^(w) for every codebook
  window (the same attention with window w), the stabilised cosine score
  (Eq. stabilized-cosine), the per-head mean score (Eq.
  conditional-similarity), the threshold selection (Eq.
  threshold-selection) and the finite-grid budget selector (Eq.
  budget-selector).
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# HWKV_ORACLE_LIBRARY may name the sanitizer build of the same source.
_LIB_PATH = os.environ.get("HWKV_ORACLE_LIBRARY") or os.path.join(_HERE, "liboracle.so")
_lib = None

_i64 = ctypes.c_int64
_dbl = ctypes.c_double
_vp = ctypes.c_void_p


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.orc_bf16_to_f64.argtypes = [ctypes.c_uint16]
    lib.orc_bf16_to_f64.restype = _dbl
    lib.orc_is_resident.argtypes = [_i64, _i64, _i64, _i64]
    lib.orc_is_resident.restype = ctypes.c_int
    lib.orc_resident_count.argtypes = [_i64, _i64, _i64]
    lib.orc_resident_count.restype = _i64
    lib.orc_capacity.argtypes = [_i64, _i64, _i64]
    lib.orc_capacity.restype = _i64
    lib.orc_slot.argtypes = [_i64, _i64, _i64]
    lib.orc_slot.restype = _i64
    lib.orc_retained_tokens.argtypes = [_i64, _i64, _i64]
    lib.orc_retained_tokens.restype = _i64
    lib.orc_unit_bytes.argtypes = [_i64, _i64, _i64, _i64, _i64, _dbl, _dbl]
    lib.orc_unit_bytes.restype = _dbl
    lib.orc_policy_bytes.argtypes = [_i64, _i64, _i64, _vp, _i64, _i64, _dbl, _dbl]
    lib.orc_policy_bytes.restype = _dbl
    lib.orc_rate.argtypes = [_i64, _i64, _i64, _vp, _i64, _i64, _dbl, _dbl]
    lib.orc_rate.restype = _dbl
    lib.orc_table_init.argtypes = [_vp, _i64]
    lib.orc_table_init.restype = None
    lib.orc_table_prefill.argtypes = [_vp, _i64, _i64, _i64, _i64, _i64]
    lib.orc_table_prefill.restype = ctypes.c_int
    lib.orc_table_append.argtypes = [_vp, _i64, _i64, _i64, _i64]
    lib.orc_table_append.restype = ctypes.c_int
    lib.orc_attend_row.argtypes = [_vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _dbl, _vp]
    lib.orc_attend_row.restype = None
    lib.orc_attend_slots.argtypes = [_vp, _vp, _vp, _i64, _vp, _i64, _dbl, _vp]
    lib.orc_attend_slots.restype = ctypes.c_int
    lib.orc_decode_layer.argtypes = [ctypes.c_int, _i64, _i64, _i64, _i64, _i64,
                                     _vp, _vp, _vp, _vp, _vp, _dbl, _vp]
    lib.orc_decode_layer.restype = ctypes.c_int
    lib.orc_cos_eval.argtypes = [_vp, _vp, _i64]
    lib.orc_cos_eval.restype = _dbl
    _lib = lib
    return lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _u16(a):
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError("bf16 arrays are passed as uint16 bit patterns")
    return a


# --------------------------------------------------------------------------
# bf16 and residency
# --------------------------------------------------------------------------
def bf16_to_f64(bits):
    """Exact widening of bf16 bit patterns (uint16 array or int) to fp64."""
    lib = _load()
    if np.isscalar(bits):
        return lib.orc_bf16_to_f64(int(bits))
    b = np.asarray(bits, dtype=np.uint16)
    return np.array([lib.orc_bf16_to_f64(int(x)) for x in b.ravel()]).reshape(b.shape)


def is_resident(p, n, n_sinks, window):
    return bool(_load().orc_is_resident(p, n, n_sinks, window))


def resident_count(n, n_sinks, window):
    return int(_load().orc_resident_count(n, n_sinks, window))


def capacity(n_sinks, window, max_ctx):
    return int(_load().orc_capacity(n_sinks, window, max_ctx))


def slot(p, n_sinks, window):
    return int(_load().orc_slot(p, n_sinks, window))


def retained_tokens(ctx, n_sinks, window):
    return int(_load().orc_retained_tokens(ctx, n_sinks, window))


# --------------------------------------------------------------------------
# accounting
# --------------------------------------------------------------------------
def unit_bytes(ctx, n_sinks, window, d_k, d_v, b_k, b_v):
    return _load().orc_unit_bytes(ctx, n_sinks, window, d_k, d_v, b_k, b_v)


def policy_bytes(ctx, n_sinks, windows, d_k, d_v, b_k=2.0, b_v=2.0):
    w = np.ascontiguousarray(windows, dtype=np.int64)
    return _load().orc_policy_bytes(ctx, n_sinks, w.size, _ptr(w), d_k, d_v, b_k, b_v)


def rate(ctx, n_sinks, windows, d_k=1, d_v=1, b_k=2.0, b_v=2.0):
    w = np.ascontiguousarray(windows, dtype=np.int64)
    return _load().orc_rate(ctx, n_sinks, w.size, _ptr(w), d_k, d_v, b_k, b_v)


# --------------------------------------------------------------------------
# slot-table simulation of one (unit, sequence)
# --------------------------------------------------------------------------
class UnitTable:
    """Which position each physical slot holds, for one unit and sequence.

    ``table[j]`` is the position stored in slot ``j`` (``-1`` = empty) and
    ``n`` the sequence length seen so far."""

    def __init__(self, n_sinks, window, max_ctx):
        self.n_sinks = int(n_sinks)
        self.window = int(window)
        self.cap = capacity(n_sinks, window, max_ctx)
        self.table = np.empty(self.cap, dtype=np.int64)
        _load().orc_table_init(_ptr(self.table), self.cap)
        self.n = 0

    def prefill(self, p0, p1):
        if p0 != self.n:
            raise ValueError("prefill must start at the current length")
        rc = _load().orc_table_prefill(_ptr(self.table), self.cap,
                                       self.n_sinks, self.window, p0, p1)
        if rc != 0:
            raise ValueError("capacity exceeded")
        self.n = p1

    def append(self):
        rc = _load().orc_table_append(_ptr(self.table), self.cap,
                                      self.n_sinks, self.window, self.n)
        if rc != 0:
            raise ValueError("capacity exceeded")
        self.n += 1

    @property
    def n_valid(self):
        return int(np.count_nonzero(self.table >= 0))


# --------------------------------------------------------------------------
# attention
# --------------------------------------------------------------------------
def attend_row(q, k_hist, v_hist, t, n_sinks, window, scale):
    """One query head at position ``t`` over the masked full history.

    ``q`` is ``[d]`` bf16 bits; ``k_hist``/``v_hist`` are ``[>= t+1, d]`` bf16
    bits for this KV head (rows are positions).  Returns fp64 ``[d]``."""
    q = _u16(q)
    k = _u16(k_hist)
    v = _u16(v_hist)
    d = q.shape[-1]
    if k.shape[0] < t + 1 or v.shape[0] < t + 1:
        raise ValueError("history shorter than t + 1")
    out = np.empty(d, dtype=np.float64)
    _load().orc_attend_row(_ptr(q), _ptr(k), _ptr(v), d, d, t, n_sinks,
                           window, scale, _ptr(out))
    return out


def attend_slots(q, cache_k, cache_v, slot_pos, scale):
    """Same output from a compacted unit (rows per slot + slot->position)."""
    q = _u16(q)
    ck = _u16(cache_k)
    cv = _u16(cache_v)
    sp = np.ascontiguousarray(slot_pos, dtype=np.int64)
    d = q.shape[-1]
    out = np.empty(d, dtype=np.float64)
    n = _load().orc_attend_slots(_ptr(q), _ptr(ck), _ptr(cv), d, _ptr(sp),
                                 sp.size, scale, _ptr(out))
    if n < 0:
        raise MemoryError
    return out


def decode_layer(q, k_hist, v_hist, t, n_sinks, windows, scale, n_threads=1):
    """One decode step of one layer for every sequence and query head.

    ``q`` ``[B, Hq, d]`` bf16 bits; ``k_hist[b]``/``v_hist[b]``
    ``[>= t[b]+1, Hkv, d]`` bf16 bits; ``windows`` ``[Hkv]`` (0 = full);
    ``t[b]`` the query position.  Returns fp64 ``[B, Hq, d]``."""
    q = _u16(q)
    B, Hq, d = q.shape
    ks = [_u16(x) for x in k_hist]
    vs = [_u16(x) for x in v_hist]
    Hkv = ks[0].shape[1]
    t = np.ascontiguousarray(t, dtype=np.int64)
    w = np.ascontiguousarray(windows, dtype=np.int64)
    for b in range(B):
        if ks[b].shape[0] < t[b] + 1 or vs[b].shape[0] < t[b] + 1:
            raise ValueError("history shorter than t + 1")
    kp = (ctypes.c_void_p * B)(*[x.ctypes.data for x in ks])
    vp = (ctypes.c_void_p * B)(*[x.ctypes.data for x in vs])
    out = np.empty((B, Hq, d), dtype=np.float64)
    rc = _load().orc_decode_layer(int(n_threads), B, Hq, Hkv, d, n_sinks,
                                  _ptr(w), _ptr(t), _ptr(q), kp, vp,
                                  float(scale), _ptr(out))
    if rc != 0:
        raise ValueError("invalid decode_layer arguments")
    return out


# --------------------------------------------------------------------------
# calibration replay and selection
# --------------------------------------------------------------------------
def cos_eval(u, v):
    """Stabilised cosine of two vectors (Eq. stabilized-cosine), fp64."""
    u = np.ascontiguousarray(u, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    if u.shape != v.shape or u.ndim != 1:
        raise ValueError("u and v must be vectors of one length")
    return float(_load().orc_cos_eval(_ptr(u), _ptr(v), u.size))


def replay_outputs(q_rows, k_hist, v_hist, rows, n_sinks, windows, scale, n_threads=8):
    """Candidate outputs o^(w) of every sampled row for every window of
    ``windows`` (0 = full), Eq. conditional-attention with window w.
    ``q_rows`` ``[R, Hq, d]``, ``k_hist``/``v_hist`` ``[N, Hkv, d]`` bf16 bits,
    ``rows`` the query positions.  Returns fp64 ``[len(windows), R, Hq, d]``."""
    rows = np.asarray(rows, dtype=np.int64)
    Hkv = np.asarray(k_hist).shape[1]
    out = []
    for w in windows:
        out.append(decode_layer(q_rows, [k_hist] * len(rows), [v_hist] * len(rows), rows,
                                n_sinks, [int(w)] * Hkv, scale, n_threads=n_threads))
    return np.stack(out)


def replay_scores(outs):
    """cos_eval of every finite candidate against the full one: ``outs`` is
    ``[K + 1, R, Hq, d]`` with the full candidate last; returns ``[K, R, Hq]``."""
    K = outs.shape[0] - 1
    sc = np.empty((K,) + outs.shape[1:3], dtype=np.float64)
    for k in range(K):
        for r in range(outs.shape[1]):
            for q in range(outs.shape[2]):
                sc[k, r, q] = cos_eval(outs[k, r, q], outs[K, r, q])
    return sc


def head_means(scores, group):
    """Eq. conditional-similarity: the mean of the scores of KV head h over
    its index set (every sampled row and every query head q with
    q // group == h).  ``scores`` ``[K, R, Hq]``; returns ``[K, Hkv]``."""
    scores = np.asarray(scores, dtype=np.float64)
    K, R, Hq = scores.shape
    Hkv = Hq // group
    out = np.empty((K, Hkv), dtype=np.float64)
    for k in range(K):
        for h in range(Hkv):
            out[k, h] = scores[k, :, h * group:(h + 1) * group].mean()
    return out


def select_windows(means, windows, n_sinks, ctx, tau):
    """Eq. threshold-selection for one layer: per KV head, the candidate of
    lowest cost min(S + w, ctx) whose mean score is at least ``tau``; equal
    costs go to the earlier codebook entry.  ``means`` ``[K, Hkv]`` for the
    finite ``windows`` (in codebook order); the full candidate (score one,
    cost ctx) is always feasible and is returned as index K."""
    means = np.asarray(means, dtype=np.float64)
    K, Hkv = means.shape
    choice = []
    for h in range(Hkv):
        best, best_cost = None, None
        # candidates in codebook order, full (index K, score 1, cost ctx) last
        for k in range(K + 1):
            score = means[k, h] if k < K else 1.0
            cost = min(n_sinks + int(windows[k]), ctx) if k < K else ctx
            if score >= tau and (best is None or cost < best_cost):
                best, best_cost = k, cost
        choice.append(best)
    return choice


def budget_select(rates, floors, budget):
    """Eq. budget-selector over a recorded grid: among runs g (in grid order)
    with rate <= budget, maximise the floor, then minimise the rate, then the
    grid index.  Returns the 0-based grid index, or None if no run fits."""
    feas = [g for g in range(len(rates)) if rates[g] <= budget]
    if not feas:
        return None
    phi = max(floors[g] for g in feas)
    beta = min(rates[g] for g in feas if floors[g] == phi)
    return min(g for g in feas if floors[g] == phi and rates[g] == beta)
