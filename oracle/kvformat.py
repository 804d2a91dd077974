"""Cache formats p_KV for the oracle (numpy, fp64).  TEST INFRASTRUCTURE ONLY.

The paper's storage accounting carries a cache format p_KV through the
effective bytes per element b^K, b^V (Method, Eq. nominal-storage), and when
the format changes numerical execution every consumer of the cache (the full
reference, the compressed policy, calibration) uses it.  The formats and how
an element is stored:

* ``bf16``: stored as given (the input format);
* ``f16``: IEEE binary16 of the element, round to nearest even, overflow to
  infinity -- numpy's float16 conversion, a library primitive;
* ``fp8``: OCP FP8 E4M3 ("E4M3FN") code of ``x / s`` for the fp32 scale
  ``s`` of the (layer, KV head) and tensor (K or V).  The quotient is the
  correctly rounded fp32 division; the code is the finite E4M3 value nearest
  to it, ties to the code with an even last bit, magnitudes beyond 448
  (infinity included) giving 448, NaN giving S.1111.111, and the sign bit
  copied from the quotient.  Encoding looks the quotient up in the sorted
  table of all finite codes, built from the definition of the format (sign,
  4 exponent bits of bias 7, 3 mantissa bits; exponent field 0 holds the
  subnormals m * 2^-9).

The value of a stored element is its decoded value, times ``s`` for fp8.
``attend_values`` is decode attention (Eqs. conditional-attention-weight and
conditional-attention) over such values, with the residency of the sink +
window rule: a plain fp64 softmax over the retained positions.
"""
import numpy as np

FORMATS = {"bf16": 0, "f16": 1, "fp8": 2}
BYTES = {"bf16": 2, "f16": 2, "fp8": 1}


def _e4m3_value(code):
    sign = -1.0 if code & 0x80 else 1.0
    e = (code >> 3) & 0xF
    m = code & 0x7
    if e == 0xF and m == 0x7:
        return np.nan
    if e == 0:
        return sign * (m / 8.0) * 2.0 ** -6
    return sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)


E4M3_TABLE = np.array([_e4m3_value(c) for c in range(256)], dtype=np.float64)
E4M3_MAX = 448.0


def bf16_values(bits):
    """Exact fp64 values of bf16 bit patterns (uint16 array)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    with np.errstate(invalid="ignore"):
        return b.view(np.float32).astype(np.float64)


def e4m3_encode(x, scale, chunk=1 << 22):
    """E4M3 codes (uint8) of ``x`` (values exactly representable in fp32,
    e.g. bf16 values) divided by the fp32 ``scale``: nearest finite code,
    ties to even, saturating, NaN to 0x7F | sign.  The nearest code is found
    in the sorted table of the 127 finite magnitudes: of the two table
    entries around |y|, the closer one, or the one with the even code on a
    tie."""
    y = np.asarray(x, dtype=np.float64).astype(np.float32)
    with np.errstate(over="ignore", invalid="ignore", divide="ignore"):
        y = (y / np.float32(scale)).astype(np.float32).ravel()
    out = np.empty(y.size, dtype=np.uint8)
    mags = E4M3_TABLE[:127]           # codes 0x00 .. 0x7E, increasing
    for i0 in range(0, y.size, chunk):
        yy = y[i0:i0 + chunk].astype(np.float64)
        a = np.abs(yy)
        fin = np.isfinite(a)
        # beyond 448 the nearest finite code is 448 whatever the magnitude
        af = np.minimum(np.where(fin, a, 0.0), 448.0)
        hi = np.clip(np.searchsorted(mags, af, side="left"), 1, 126)   # mags[hi-1] < af <= mags[hi]
        lo = hi - 1
        dlo = af - mags[lo]            # exact: neighbours of af within a binade or two
        dhi = mags[hi] - af
        c = np.where(dlo < dhi, lo, np.where(dhi < dlo, hi, np.where(lo % 2 == 0, lo, hi)))
        c = np.where(af == 0.0, 0, c).astype(np.uint8)
        c = np.where(np.isinf(a), np.uint8(0x7E), c)
        c = np.where(np.isnan(a), np.uint8(0x7F), c)
        c = c | np.where(np.signbit(yy), np.uint8(0x80), np.uint8(0))
        out[i0:i0 + chunk] = c
    return out.reshape(np.shape(x))


def e4m3_values(codes, scale=1.0):
    """fp64 values of E4M3 codes, times ``scale`` (exact in fp64)."""
    return E4M3_TABLE[np.asarray(codes, dtype=np.uint8)] * float(np.float32(scale))


def f16_encode(x):
    """IEEE binary16 bit patterns (uint16) of fp64 values ``x``."""
    with np.errstate(over="ignore"):
        return np.asarray(x, dtype=np.float64).astype(np.float16).view(np.uint16)


def f16_values(bits):
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


_ALL_BF16 = np.arange(65536, dtype=np.uint32).astype(np.uint16)
_TABLES = {}


def _pattern_table(fmt, scale):
    """The stored element of every bf16 bit pattern (the encoding is a
    function of the pattern and the scale), computed once per scale."""
    key = (fmt, float(np.float32(scale)))
    if key not in _TABLES:
        x = bf16_values(_ALL_BF16)
        _TABLES[key] = f16_encode(x) if fmt == "f16" else e4m3_encode(x, scale)
    return _TABLES[key]


def store(bits_bf16, fmt, scale=1.0):
    """Stored elements of bf16 inputs in format ``fmt``: uint16 bf16 bits,
    uint16 binary16 bits or uint8 E4M3 codes."""
    bits_bf16 = np.asarray(bits_bf16, dtype=np.uint16)
    if fmt == "bf16":
        return bits_bf16.copy()
    if fmt in ("f16", "fp8"):
        return _pattern_table(fmt, scale if fmt == "fp8" else 1.0)[bits_bf16]
    raise ValueError(f"unknown format {fmt!r}")


def values(stored, fmt, scale=1.0):
    """fp64 values of stored elements."""
    if fmt == "bf16":
        return bf16_values(stored)
    if fmt == "f16":
        return f16_values(stored)
    if fmt == "fp8":
        return e4m3_values(stored, scale)
    raise ValueError(f"unknown format {fmt!r}")


def retained_positions(t, n_sinks, window):
    """Positions s <= t retained for a query at t: R(t + 1) within [0, t]
    (every s for window 0 = full; else s < S or s >= t + 1 - w)."""
    s = np.arange(t + 1)
    if window == 0:
        return s
    return s[(s < n_sinks) | (s >= t + 1 - window)]


def attend_values(q, k_vals, v_vals, t, n_sinks, windows, scale):
    """Decode attention over fp64 K/V values.

    ``q`` ``[B, Hq, d]`` fp64; ``k_vals[b]``, ``v_vals[b]`` ``[>= t[b] + 1,
    Hkv, d]`` fp64; ``windows[h]`` (0 = full); ``t[b]`` the query position.
    out[b, qh] = sum_s softmax_s(scale * q . k_s) v_s over the retained
    positions of KV head qh // G.  Returns fp64 ``[B, Hq, d]``."""
    q = np.asarray(q, dtype=np.float64)
    B, Hq, d = q.shape
    Hkv = np.asarray(k_vals[0]).shape[1]
    G = Hq // Hkv
    out = np.empty((B, Hq, d), dtype=np.float64)
    for b in range(B):
        for h in range(Hkv):
            pos = retained_positions(int(t[b]), n_sinks, int(windows[h]))
            K = np.asarray(k_vals[b], dtype=np.float64)[pos, h]
            V = np.asarray(v_vals[b], dtype=np.float64)[pos, h]
            z = scale * (q[b, h * G:(h + 1) * G] @ K.T)          # [G, n]
            p = np.exp(z - z.max(axis=1, keepdims=True))
            out[b, h * G:(h + 1) * G] = (p @ V) / p.sum(axis=1, keepdims=True)
    return out


def replay_outputs_values(q_rows, k_vals, v_vals, rows, n_sinks, windows, scale):
    """Calibration candidate outputs o^(w) over fp64 K/V values (a traced
    layer as a cache of some format stores it): for every window of
    ``windows`` (0 = full), the attention of each row at its own position.
    ``q_rows`` [R, Hq, d], ``k_vals``/``v_vals`` [N, Hkv, d] fp64.  Returns
    [len(windows), R, Hq, d]."""
    rows = np.asarray(rows, dtype=np.int64)
    Hkv = np.asarray(k_vals).shape[1]
    return np.stack([attend_values(q_rows, [k_vals] * len(rows), [v_vals] * len(rows), rows,
                                   n_sinks, [int(w)] * Hkv, scale) for w in windows])
