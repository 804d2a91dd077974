"""ctypes binding of ``libhwkv.so`` (the C ABI in ``include/hwkv.h``).

Argument marshalling only: every step of the data path runs in the HIP
kernels behind the C ABI.  Functions keep the C names without the ``hwkv_``
prefix.  Device arguments are torch tensors on the GPU (bf16 inputs, fp32
outputs, contiguous); ``stream`` defaults to torch's current stream.  There is
no fallback: if the library is missing, importing this module raises.
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# HWKV_LIBRARY may name another build of the same library (the CPU tests'
# host-sanitizer build); by default the in-tree one is loaded.
LIB_PATH = os.environ.get("HWKV_LIBRARY") or os.path.join(_HERE, "_lib", "libhwkv.so")

OK, EINVAL, ENOMEM, ECAPACITY, ESTATE, EDEVICE = 0, 1, 2, 3, 4, 5
# cache formats (HWKV_KV_*): name -> (code, bytes per element)
KV_FORMATS = {"bf16": (0, 2), "f16": (1, 2), "fp8": (2, 1)}
PAGE_TOKENS = 256   # rows per page of a paged cache's full units
_NAMES = {EINVAL: "EINVAL", ENOMEM: "ENOMEM", ECAPACITY: "ECAPACITY",
          ESTATE: "ESTATE", EDEVICE: "EDEVICE"}

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build it with paper_2609_02029_amd.build.build() "
        "(or __graft_entry__.build()) first")

# torch owns device memory and streams: load it (and the HIP runtime it
# initialises) before the library, so both use that one runtime whatever the
# caller's import order.
import torch  # noqa: E402,F401

_lib = ctypes.CDLL(LIB_PATH)

_i32, _i64, _dbl, _flt, _vp, _sz = (ctypes.c_int32, ctypes.c_int64, ctypes.c_double,
                                     ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t)
_P = ctypes.POINTER

SYMBOLS = {
    "hwkv_last_error": ([], ctypes.c_char_p),
    "hwkv_policy_set": ([_P(_vp), _i32, _i32, _i32, _i32, _i32, _i32, _P(_i64), _P(_i32)], ctypes.c_int),
    "hwkv_policy_free": ([_vp], ctypes.c_int),
    "hwkv_policy_bytes": ([_vp, _i64, _P(_dbl)], ctypes.c_int),
    "hwkv_policy_rate": ([_vp, _i64, _P(_dbl)], ctypes.c_int),
    "hwkv_policy_bytes_format": ([_vp, _i64, _i32, _P(_dbl)], ctypes.c_int),
    "hwkv_cache_bytes_format": ([_vp, _i32, _i64, _i32, _P(_sz)], ctypes.c_int),
    "hwkv_cache_alloc_format": ([_P(_vp), _vp, _i32, _i64, _i32, _vp, _vp, _vp, _sz],
                                ctypes.c_int),
    "hwkv_cache_format": ([_vp, _P(_i32), _vp, _vp], ctypes.c_int),
    "hwkv_cache_bytes_paged": ([_vp, _i32, _i64, _i32, _i64, _P(_sz)], ctypes.c_int),
    "hwkv_cache_alloc_paged": ([_P(_vp), _vp, _i32, _i64, _i32, _vp, _vp, _i64, _vp, _sz],
                               ctypes.c_int),
    "hwkv_cache_pages": ([_vp, _P(_i64), _P(_i64)], ctypes.c_int),
    "hwkv_cache_reset_seq": ([_vp, _i32], ctypes.c_int),
    "hwkv_cache_bytes": ([_vp, _i32, _i64, _P(_sz)], ctypes.c_int),
    "hwkv_cache_alloc": ([_P(_vp), _vp, _i32, _i64, _vp, _sz], ctypes.c_int),
    "hwkv_cache_free": ([_vp], ctypes.c_int),
    "hwkv_cache_seq_len": ([_vp, _i32, _i32, _P(_i64)], ctypes.c_int),
    "hwkv_cache_unit_info": ([_vp, _i32, _i32, _P(_i64), _P(_i64)], ctypes.c_int),
    "hwkv_prefill_write": ([_vp, _i32, _i32, _i64, _i64, _vp, _vp, _vp], ctypes.c_int),
    "hwkv_prefill_attn": ([_vp, _i32, _i32, _i64, _i64, _vp, _vp, _vp, ctypes.c_float, _vp,
                           _vp], ctypes.c_int),
    "hwkv_prefill_attn_workspace_bytes": ([_vp, _i64, _P(_sz)], ctypes.c_int),
    "hwkv_prefill_attn_ws": ([_vp, _i32, _i32, _i64, _i64, _vp, _vp, _vp, ctypes.c_float, _vp,
                              _vp, _sz, _vp], ctypes.c_int),
    "hwkv_append": ([_vp, _i32, _vp, _vp, _vp], ctypes.c_int),
    "hwkv_decode_workspace_bytes": ([_vp, _P(_sz)], ctypes.c_int),
    "hwkv_decode_attn": ([_vp, _i32, _vp, _flt, _vp, _vp, _sz, _vp], ctypes.c_int),
    "hwkv_append_decode_attn": ([_vp, _i32, _vp, _vp, _vp, _flt, _vp, _vp, _sz, _vp], ctypes.c_int),
    "hwkv_append_decode_attn_noalloc": ([_vp, _i32, _vp, _vp, _vp, _flt, _vp, _vp], ctypes.c_int),
    "hwkv_cache_read_unit": ([_vp, _i32, _i32, _i32, _vp, _vp, _P(_i64)], ctypes.c_int),
    "hwkv_decode_timing": ([_vp, _i32], ctypes.c_int),
    "hwkv_decode_timing_read": ([_vp, _P(_dbl), _P(_dbl), _P(_i64)], ctypes.c_int),
    "hwkv_calib_workspace_bytes": ([_i32, _i32, _i32, _i64, _i64, _P(_sz)], ctypes.c_int),
    "hwkv_calib_replay": ([_i32, _i32, _i32, _i32, _i32, _vp, _i64, _vp, _vp, _i64, _vp, _vp,
                           _flt, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp], ctypes.c_int),
    "hwkv_calib_workspace_bytes_format": ([_i32, _i32, _i32, _i32, _i64, _i64, _i32, _P(_sz)],
                                          ctypes.c_int),
    "hwkv_calib_replay_format": ([_i32, _i32, _i32, _i32, _i32, _vp, _i64, _vp, _vp, _i64, _vp, _vp,
                                  _flt, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _vp, _vp, _sz, _vp],
                                 ctypes.c_int),
    "hwkv_calib_select": ([_i32, _i32, _vp, _i32, _i64, _vp, _dbl, _vp, _P(_dbl)], ctypes.c_int),
    "hwkv_budget_select": ([_i32, _vp, _vp, _dbl, _P(_i32)], ctypes.c_int),
    "hwkv_policy_shape": ([_vp, _P(_i32), _P(_i32), _P(_i32), _P(_i32), _P(_i32), _P(_i32)],
                          ctypes.c_int),
    "hwkv_policy_serialize": ([_vp, ctypes.c_char_p, ctypes.c_uint64, _i32, _dbl, _dbl, _dbl,
                               _vp, _sz, _P(_sz)], ctypes.c_int),
    "hwkv_policy_deserialize": ([ctypes.c_char_p, _sz, _P(_vp), _vp, _sz,
                                 _P(ctypes.c_uint64), _P(_i32), _P(_dbl), _P(_dbl), _P(_dbl)],
                                ctypes.c_int),
}
for _name, (_args, _res) in SYMBOLS.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = _res


class HwkvError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{_NAMES.get(code, code)}: {msg}")
        self.code = code


def last_error():
    return _lib.hwkv_last_error().decode()


def _check(rc):
    if rc != OK:
        raise HwkvError(rc, last_error())


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _dev(t, dtype_name, what):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{what} must be a device tensor")
    if str(t.dtype) != f"torch.{dtype_name}":
        raise ValueError(f"{what} must be {dtype_name}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    return t.data_ptr()


class Policy:
    """Owns an ``hwkv_policy*``."""

    _free = _lib.hwkv_policy_free  # kept alive until interpreter shutdown

    def __init__(self, handle):
        self.handle = handle

    def __del__(self):
        if getattr(self, "handle", None):
            self._free(self.handle)
            self.handle = None


class Cache:
    """Owns an ``hwkv_cache*``."""

    _free = _lib.hwkv_cache_free

    def __init__(self, handle, n_layers, n_kv_heads, n_q_heads, head_dim, batch):
        self.handle = handle
        self.n_layers, self.n_kv_heads, self.n_q_heads = n_layers, n_kv_heads, n_q_heads
        self.head_dim, self.batch = head_dim, batch

    def free(self):
        if getattr(self, "handle", None):
            h, self.handle = self.handle, None
            _check(_lib.hwkv_cache_free(h))

    def __del__(self):
        if getattr(self, "handle", None):
            self._free(self.handle)
            self.handle = None


# ---------------------------------------------------------------------------
# policy
# ---------------------------------------------------------------------------
def policy_set(n_layers, n_kv_heads, n_q_heads, head_dim, n_sinks, level_window,
               level_of_unit):
    lw = (_i64 * len(level_window))(*[int(x) for x in level_window])
    flat = [int(x) for row in level_of_unit for x in (row if hasattr(row, "__len__") else [row])]
    lu = (_i32 * max(1, len(flat)))(*flat)
    h = _vp()
    _check(_lib.hwkv_policy_set(ctypes.byref(h), n_layers, n_kv_heads, n_q_heads, head_dim,
                                n_sinks, len(level_window), lw, lu))
    p = Policy(h)
    p.n_layers, p.n_kv_heads, p.n_q_heads, p.head_dim = n_layers, n_kv_heads, n_q_heads, head_dim
    return p


def policy_free(policy):
    if policy.handle:
        _check(_lib.hwkv_policy_free(policy.handle))
        policy.handle = None


def _fmt_code(kv_format):
    if kv_format not in KV_FORMATS:
        raise ValueError(f"kv_format must be one of {sorted(KV_FORMATS)}")
    return KV_FORMATS[kv_format][0]


def policy_bytes(policy, ctx, kv_format="bf16"):
    r = _dbl()
    _check(_lib.hwkv_policy_bytes_format(policy.handle, ctx, _fmt_code(kv_format),
                                         ctypes.byref(r)))
    return r.value


def policy_rate(policy, ctx):
    r = _dbl()
    _check(_lib.hwkv_policy_rate(policy.handle, ctx, ctypes.byref(r)))
    return r.value


# ---------------------------------------------------------------------------
# cache
# ---------------------------------------------------------------------------
def cache_bytes(policy, batch, max_ctx, kv_format="bf16", n_pages=None):
    """Device bytes of a cache; ``n_pages`` (not None): a paged cache with a
    pool of that many pages."""
    r = _sz()
    if n_pages is None:
        _check(_lib.hwkv_cache_bytes_format(policy.handle, batch, max_ctx,
                                            _fmt_code(kv_format), ctypes.byref(r)))
    else:
        _check(_lib.hwkv_cache_bytes_paged(policy.handle, batch, max_ctx,
                                           _fmt_code(kv_format), n_pages, ctypes.byref(r)))
    return r.value


def _scales(policy, x):
    """Host fp32 [n_layers][n_kv_heads] scales (array-like or scalar) or None."""
    if x is None:
        return None
    import numpy as np
    a = np.ascontiguousarray(np.broadcast_to(np.asarray(x, dtype=np.float32),
                                             (policy.n_layers, policy.n_kv_heads)))
    return a


def cache_alloc(policy, batch, max_ctx, dev_buf=None, kv_format="bf16", k_scale=None,
                v_scale=None, n_pages=None):
    """``dev_buf``: optional uint8 device tensor to adopt (kept alive).
    ``kv_format``: "bf16", "f16" or "fp8"; ``k_scale``/``v_scale``: fp8 scales,
    a scalar or ``[n_layers, n_kv_heads]`` (None = 1.0).  ``n_pages`` (not
    None): full units are paged from a pool of that many pages."""
    h = _vp()
    ptr = None
    nbytes = 0
    if dev_buf is not None:
        ptr = _dev(dev_buf, "uint8", "dev_buf")
        nbytes = dev_buf.numel()
    ks = _scales(policy, k_scale)
    vs = _scales(policy, v_scale)
    kp = None if ks is None else ks.ctypes.data_as(_vp)
    vp = None if vs is None else vs.ctypes.data_as(_vp)
    if n_pages is None:
        _check(_lib.hwkv_cache_alloc_format(ctypes.byref(h), policy.handle, batch, max_ctx,
                                            _fmt_code(kv_format), kp, vp, ptr, nbytes))
    else:
        _check(_lib.hwkv_cache_alloc_paged(ctypes.byref(h), policy.handle, batch, max_ctx,
                                           _fmt_code(kv_format), kp, vp, n_pages, ptr, nbytes))
    c = Cache(h, policy.n_layers, policy.n_kv_heads, policy.n_q_heads, policy.head_dim, batch)
    c.dev_buf = dev_buf
    c.kv_format = kv_format
    return c


def cache_pages(cache):
    """(pool pages, free pages) of a paged cache; (0, 0) otherwise."""
    t, f = _i64(), _i64()
    _check(_lib.hwkv_cache_pages(cache.handle, ctypes.byref(t), ctypes.byref(f)))
    return t.value, f.value


def cache_reset_seq(cache, seq):
    _check(_lib.hwkv_cache_reset_seq(cache.handle, seq))


def cache_format(cache):
    """Returns (kv_format name, k_scale, v_scale): scales as numpy fp32
    ``[n_layers, n_kv_heads]``."""
    import numpy as np
    code = _i32()
    ks = np.empty((cache.n_layers, cache.n_kv_heads), dtype=np.float32)
    vs = np.empty_like(ks)
    _check(_lib.hwkv_cache_format(cache.handle, ctypes.byref(code), ks.ctypes.data_as(_vp),
                                  vs.ctypes.data_as(_vp)))
    name = [k for k, (c, _) in KV_FORMATS.items() if c == code.value][0]
    return name, ks, vs


def cache_free(cache):
    cache.free()


def cache_seq_len(cache, layer, seq):
    r = _i64()
    _check(_lib.hwkv_cache_seq_len(cache.handle, layer, seq, ctypes.byref(r)))
    return r.value


def cache_unit_info(cache, layer, kv_head):
    cap, win = _i64(), _i64()
    _check(_lib.hwkv_cache_unit_info(cache.handle, layer, kv_head, ctypes.byref(cap),
                                     ctypes.byref(win)))
    return cap.value, win.value


def cache_read_unit(cache, layer, kv_head, seq):
    """Returns (k, v, n_valid): numpy [capacity, head_dim] stored elements --
    uint16 bit patterns (bf16, f16) or uint8 E4M3 codes (fp8)."""
    import numpy as np
    cap, _ = cache_unit_info(cache, layer, kv_head)
    dt = np.uint8 if getattr(cache, "kv_format", "bf16") == "fp8" else np.uint16
    k = np.empty((cap, cache.head_dim), dtype=dt)
    v = np.empty((cap, cache.head_dim), dtype=dt)
    nv = _i64()
    _check(_lib.hwkv_cache_read_unit(cache.handle, layer, kv_head, seq,
                                     k.ctypes.data_as(_vp), v.ctypes.data_as(_vp),
                                     ctypes.byref(nv)))
    return k, v, nv.value


# ---------------------------------------------------------------------------
# data path
# ---------------------------------------------------------------------------
def prefill_write(cache, layer, seq, pos0, k, v, stream=None):
    """``k``, ``v``: bf16 [n_tokens, n_kv_heads, head_dim] device tensors."""
    n = k.shape[0]
    if tuple(k.shape) != (n, cache.n_kv_heads, cache.head_dim) or tuple(v.shape) != tuple(k.shape):
        raise ValueError("k and v must be [n_tokens, n_kv_heads, head_dim]")
    _check(_lib.hwkv_prefill_write(cache.handle, layer, seq, pos0, n,
                                   _dev(k, "bfloat16", "k"), _dev(v, "bfloat16", "v"),
                                   _stream(stream)))


def prefill_attn_workspace_bytes(cache, n_tokens):
    r = _sz()
    _check(_lib.hwkv_prefill_attn_workspace_bytes(cache.handle, n_tokens, ctypes.byref(r)))
    return r.value


def prefill_attn(cache, layer, seq, pos0, q, k, v, scale, out, ws=None, stream=None):
    """``q``: bf16 [n_tokens, n_q_heads, head_dim]; ``k``, ``v``: bf16
    [n_tokens, n_kv_heads, head_dim]; ``out``: fp32 like ``q`` (device).
    ``ws``: uint8 device workspace (hwkv_prefill_attn_ws; needed by fp8
    caches, see prefill_attn_workspace_bytes)."""
    n = q.shape[0]
    if tuple(q.shape) != (n, cache.n_q_heads, cache.head_dim):
        raise ValueError("q must be [n_tokens, n_q_heads, head_dim]")
    if tuple(k.shape) != (n, cache.n_kv_heads, cache.head_dim) or tuple(v.shape) != tuple(k.shape):
        raise ValueError("k and v must be [n_tokens, n_kv_heads, head_dim]")
    if tuple(out.shape) != tuple(q.shape):
        raise ValueError("out must be [n_tokens, n_q_heads, head_dim]")
    if ws is None:
        _check(_lib.hwkv_prefill_attn(cache.handle, layer, seq, pos0, n,
                                      _dev(q, "bfloat16", "q"), _dev(k, "bfloat16", "k"),
                                      _dev(v, "bfloat16", "v"), float(scale),
                                      _dev(out, "float32", "out"), _stream(stream)))
    else:
        _check(_lib.hwkv_prefill_attn_ws(cache.handle, layer, seq, pos0, n,
                                         _dev(q, "bfloat16", "q"), _dev(k, "bfloat16", "k"),
                                         _dev(v, "bfloat16", "v"), float(scale),
                                         _dev(out, "float32", "out"), _dev(ws, "uint8", "ws"),
                                         ws.numel(), _stream(stream)))


def append(cache, layer, k_new, v_new, stream=None):
    shp = (cache.batch, cache.n_kv_heads, cache.head_dim)
    if tuple(k_new.shape) != shp or tuple(v_new.shape) != shp:
        raise ValueError("k_new and v_new must be [batch, n_kv_heads, head_dim]")
    _check(_lib.hwkv_append(cache.handle, layer, _dev(k_new, "bfloat16", "k_new"),
                            _dev(v_new, "bfloat16", "v_new"), _stream(stream)))


def decode_workspace_bytes(cache):
    r = _sz()
    _check(_lib.hwkv_decode_workspace_bytes(cache.handle, ctypes.byref(r)))
    return r.value


def _decode_shapes(cache, q, out, ws):
    shp = (cache.batch, cache.n_q_heads, cache.head_dim)
    if tuple(q.shape) != shp or tuple(out.shape) != shp:
        raise ValueError("q and out must be [batch, n_q_heads, head_dim]")
    return _dev(ws, "uint8", "ws"), ws.numel()


def decode_attn(cache, layer, q, scale, out, ws, stream=None):
    """``q`` bf16 and ``out`` fp32 [batch, n_q_heads, head_dim]; ``ws`` uint8."""
    wp, wn = _decode_shapes(cache, q, out, ws)
    _check(_lib.hwkv_decode_attn(cache.handle, layer, _dev(q, "bfloat16", "q"), float(scale),
                                 _dev(out, "float32", "out"), wp, wn, _stream(stream)))


def append_decode_attn(cache, layer, k_new, v_new, q, scale, out, ws, stream=None):
    shp = (cache.batch, cache.n_kv_heads, cache.head_dim)
    if tuple(k_new.shape) != shp or tuple(v_new.shape) != shp:
        raise ValueError("k_new and v_new must be [batch, n_kv_heads, head_dim]")
    wp, wn = _decode_shapes(cache, q, out, ws)
    _check(_lib.hwkv_append_decode_attn(
        cache.handle, layer, _dev(k_new, "bfloat16", "k_new"), _dev(v_new, "bfloat16", "v_new"),
        _dev(q, "bfloat16", "q"), float(scale), _dev(out, "float32", "out"), wp, wn,
        _stream(stream)))


def append_decode_attn_noalloc(cache, layer, k_new, v_new, q, scale, out, stream=None):
    """``append_decode_attn`` without a workspace: the split partials go to
    the library's static scratch (``hwkv_append_decode_attn_noalloc``)."""
    shp = (cache.batch, cache.n_kv_heads, cache.head_dim)
    if tuple(k_new.shape) != shp or tuple(v_new.shape) != shp:
        raise ValueError("k_new and v_new must be [batch, n_kv_heads, head_dim]")
    qshp = (cache.batch, cache.n_q_heads, cache.head_dim)
    if tuple(q.shape) != qshp or tuple(out.shape) != qshp:
        raise ValueError("q and out must be [batch, n_q_heads, head_dim]")
    _check(_lib.hwkv_append_decode_attn_noalloc(
        cache.handle, layer, _dev(k_new, "bfloat16", "k_new"), _dev(v_new, "bfloat16", "v_new"),
        _dev(q, "bfloat16", "q"), float(scale), _dev(out, "float32", "out"), _stream(stream)))


def append_decode_attn_ptr(cache, layer, k_new, v_new, q, scale, out, ws, ws_bytes, stream):
    """``append_decode_attn`` on raw device addresses (ints) and a raw stream
    handle: no Python-side checks (the library still validates what it can),
    for callers that issue many calls on tensors they have already checked."""
    _check(_lib.hwkv_append_decode_attn(cache.handle, layer, k_new, v_new, q, scale, out, ws,
                                        ws_bytes, stream))


def decode_timing(cache, enable):
    _check(_lib.hwkv_decode_timing(cache.handle, 1 if enable else 0))


def decode_timing_read(cache):
    """Returns (split_ms, merge_ms, launches) summed since the last read."""
    sp, mg, n = _dbl(), _dbl(), _i64()
    _check(_lib.hwkv_decode_timing_read(cache.handle, ctypes.byref(sp), ctypes.byref(mg),
                                        ctypes.byref(n)))
    return sp.value, mg.value, n.value


def calib_workspace_bytes(n_q_heads, head_dim, n_sinks, n_hist, n_rows, n_kv_heads=None,
                          kv_format="bf16"):
    """Workspace of the replay; an fp8 ``kv_format`` also needs ``n_kv_heads``
    (the staged trace)."""
    n = _sz()
    if kv_format == "bf16":
        _check(_lib.hwkv_calib_workspace_bytes(int(n_q_heads), int(head_dim), int(n_sinks),
                                               int(n_hist), int(n_rows), ctypes.byref(n)))
    else:
        _check(_lib.hwkv_calib_workspace_bytes_format(
            int(n_kv_heads), int(n_q_heads), int(head_dim), int(n_sinks), int(n_hist),
            int(n_rows), _fmt_code(kv_format), ctypes.byref(n)))
    return n.value


def _i64_array(x):
    import numpy as np
    return np.ascontiguousarray(x, dtype=np.int64)


def calib_replay(k, v, rows, q, windows, n_sinks, scale, outs, scores, means, ws,
                 ref_full=None, check=None, stream=None, kv_format="bf16", k_scale=None,
                 v_scale=None):
    """Candidate replay of one traced layer (see ``hwkv_calib_replay``).

    ``k``, ``v``: bf16 [n_hist, Hkv, D]; ``q``: bf16 [R, Hq, D]; ``rows``:
    R increasing positions (host); ``windows``: the finite codebook in
    order; ``outs``: fp32 [K + 1, R, Hq, D]; ``scores``: fp32 [K, R, Hq];
    ``means``: fp32 [K, Hkv]; ``ws``: device workspace tensor.  ``kv_format``
    "fp8": attend over the trace as an fp8 cache stores it, with per-KV-head
    ``k_scale``, ``v_scale`` (host arrays or scalars; None = 1.0)."""
    n_hist, hkv, d = k.shape
    R, hq, _ = q.shape
    w = _i64_array(windows)
    r = _i64_array(rows)
    if r.shape != (R,):
        raise ValueError("rows must hold one position per query row")
    K = w.size
    if tuple(outs.shape) != (K + 1, R, hq, d):
        raise ValueError("outs must be [n_windows + 1, n_rows, n_q_heads, head_dim]")
    if K and (tuple(scores.shape) != (K, R, hq) or tuple(means.shape) != (K, hkv)):
        raise ValueError("scores must be [n_windows, n_rows, n_q_heads], means [n_windows, n_kv_heads]")
    import numpy as np
    sc = lambda x: None if x is None else np.ascontiguousarray(
        np.broadcast_to(np.asarray(x, dtype=np.float32), (hkv,)))
    ks, vs = sc(k_scale), sc(v_scale)
    _check(_lib.hwkv_calib_replay_format(
        hkv, hq, d, int(n_sinks), K, w.ctypes.data if K else None, n_hist,
        _dev(k, "bfloat16", "k"), _dev(v, "bfloat16", "v"), R, r.ctypes.data,
        _dev(q, "bfloat16", "q"), float(scale), _dev(outs, "float32", "outs"),
        _dev(scores, "float32", "scores") if K else None,
        _dev(means, "float32", "means") if K else None,
        _dev(ref_full, "float32", "ref_full"), _dev(check, "float32", "check"),
        _fmt_code(kv_format), None if ks is None else ks.ctypes.data_as(_vp),
        None if vs is None else vs.ctypes.data_as(_vp),
        _dev(ws, "uint8", "ws"), ws.numel(), _stream(stream)))


def calib_select(means, windows, n_sinks, ctx, tau):
    """Eq. threshold-selection on host ``means`` [K, Hkv]; returns
    (choice per KV head with K = full, floor)."""
    import numpy as np
    m = np.ascontiguousarray(means, dtype=np.float64)
    w = _i64_array(windows)
    K, hkv = m.shape
    choice = np.zeros(hkv, dtype=np.int32)
    fl = _dbl()
    _check(_lib.hwkv_calib_select(hkv, K, w.ctypes.data if K else None, int(n_sinks), int(ctx),
                                  m.ctypes.data if K else None, float(tau), choice.ctypes.data,
                                  ctypes.byref(fl)))
    return [int(x) for x in choice], fl.value


def budget_select(rates, floors, budget):
    """Eq. budget-selector; returns the grid index or None."""
    import numpy as np
    r = np.ascontiguousarray(rates, dtype=np.float64)
    f = np.ascontiguousarray(floors, dtype=np.float64)
    g = _i32()
    _check(_lib.hwkv_budget_select(r.size, r.ctypes.data, f.ctypes.data, float(budget),
                                   ctypes.byref(g)))
    return None if g.value < 0 else g.value


def policy_serialize(policy, artifact, seed, grid_index, tau, rate, floor):
    """The calibration artifact of ``policy`` as text (the keyword names match
    the record ``policy_deserialize`` returns)."""
    n = _sz()
    aid = artifact.encode("ascii")
    _check(_lib.hwkv_policy_serialize(policy.handle, aid, int(seed), int(grid_index), float(tau),
                                      float(rate), float(floor), None, 0, ctypes.byref(n)))
    buf = ctypes.create_string_buffer(n.value + 1)
    _check(_lib.hwkv_policy_serialize(policy.handle, aid, int(seed), int(grid_index), float(tau),
                                      float(rate), float(floor), buf, n.value + 1,
                                      ctypes.byref(n)))
    return buf.value.decode("ascii")


def policy_deserialize(text):
    """Parses an artifact: returns (Policy, dict of the recorded fields)."""
    raw = text.encode("ascii") if isinstance(text, str) else bytes(text)
    h = _vp()
    aid = ctypes.create_string_buffer(256)
    seed, gi = ctypes.c_uint64(), _i32()
    tau, rate, fl = _dbl(), _dbl(), _dbl()
    _check(_lib.hwkv_policy_deserialize(raw, len(raw), ctypes.byref(h), aid, 256,
                                        ctypes.byref(seed), ctypes.byref(gi), ctypes.byref(tau),
                                        ctypes.byref(rate), ctypes.byref(fl)))
    p = Policy(h.value)
    L, H, Q, D = _i32(), _i32(), _i32(), _i32()
    _check(_lib.hwkv_policy_shape(p.handle, ctypes.byref(L), ctypes.byref(H), ctypes.byref(Q),
                                  ctypes.byref(D), None, None))
    p.n_layers, p.n_kv_heads, p.n_q_heads, p.head_dim = L.value, H.value, Q.value, D.value
    return p, dict(artifact=aid.value.decode("ascii"), seed=seed.value, grid_index=gi.value,
                   tau=tau.value, rate=rate.value, floor=fl.value)
