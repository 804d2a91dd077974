"""CPU tests of libhwkv's host side: exports, policy validation, accounting,
layout sizes, and the error paths that return before any device work.

No kernel is launched here.  Caches are created over a never-dereferenced
fake device pointer (the adopt-a-buffer path makes no HIP call), which is
enough to reach every host-side validation."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hwkv.h")


@pytest.fixture(scope="module")
def hw():
    from paper_2609_02029_amd import hwkv
    return hwkv


def header_symbols():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(hwkv_[a-z_]+)\s*\(", txt)))


def test_library_exports_every_declared_symbol(hw):
    syms = header_symbols()
    assert len(syms) >= 15
    out = subprocess.run(["nm", "-D", "--defined-only", hw.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r" T (hwkv_[a-z_]+)$", out, flags=re.M))
    missing = [s for s in syms if s not in exported]
    assert not missing, missing
    # the binding declares every one of them
    assert set(syms) <= set(hw.SYMBOLS)


def test_error_codes_match_header(hw):
    txt = open(HEADER).read()
    for name in ("OK", "EINVAL", "ENOMEM", "ECAPACITY", "ESTATE", "EDEVICE"):
        v = int(re.search(rf"#define HWKV_{name} (\d+)", txt).group(1))
        assert getattr(hw, name) == v


def _pol(hw, **kw):
    a = dict(n_layers=2, n_kv_heads=2, n_q_heads=8, head_dim=64, n_sinks=4,
             level_window=[256, 0], level_of_unit=[[0, 1], [1, 0]])
    a.update(kw)
    return hw.policy_set(**a)


@pytest.mark.parametrize("kw", [
    dict(n_q_heads=6),                  # not a multiple of n_kv_heads
    dict(n_q_heads=6, n_kv_heads=2),    # group 3 unsupported
    dict(head_dim=96),
    dict(n_sinks=-1),
    dict(level_window=[-5, 0]),
    dict(level_of_unit=[[0, 2], [1, 0]]),
    dict(level_of_unit=[[0, -1], [1, 0]]),
    dict(n_layers=0),
    dict(n_kv_heads=65, n_q_heads=65, level_of_unit=[[0] * 65] * 2),
])
def test_policy_validation(hw, kw):
    with pytest.raises(hw.HwkvError) as e:
        _pol(hw, **kw)
    assert e.value.code == hw.EINVAL
    assert hw.last_error()


def test_policy_rate_matches_oracle_and_paper(hw, golden):
    g = golden("accounting.json")["sink_recent_control"]
    p = hw.policy_set(1, 1, 1, 64, g["n_sinks"], [g["window"]], [[0]])
    assert hw.policy_rate(p, g["ctx"]) == g["cache_tokens"] / g["ctx"]
    q = golden("accounting.json")["quarter_example"]
    p = hw.policy_set(1, 1, 1, 128, 0, [q["window"]], [[0]])
    assert hw.policy_rate(p, q["ctx"]) == q["rate"]
    r = np.random.default_rng(0)
    for _ in range(50):
        L, H = int(r.integers(1, 5)), int(r.choice([1, 2, 4]))
        lw = [int(x) for x in r.integers(1, 3000, size=3)] + [0]
        lv = r.integers(0, 4, size=(L, H))
        S = int(r.integers(0, 8))
        ctx = int(r.integers(1, 5000))
        p = hw.policy_set(L, H, H * 2, 64, S, lw, lv.tolist())
        wins = np.array(lw)[lv].ravel()
        assert hw.policy_rate(p, ctx) == pytest.approx(oracle.rate(ctx, S, wins), rel=1e-14)
        assert hw.policy_bytes(p, ctx) == pytest.approx(
            oracle.policy_bytes(ctx, S, wins, 64, 64, 2.0, 2.0), rel=1e-14)


def test_cache_bytes_exact(hw):
    r = np.random.default_rng(1)
    for _ in range(50):
        L, H, D = int(r.integers(1, 4)), int(r.choice([1, 2, 4])), int(r.choice([64, 128, 256]))
        lw = [int(x) for x in r.integers(1, 3000, size=3)] + [0]
        lv = r.integers(0, 4, size=(L, H))
        S = int(r.integers(0, 8))
        B = int(r.integers(1, 5))
        max_ctx = int(r.integers(1, 6000))
        p = hw.policy_set(L, H, H, D, S, lw, lv.tolist())
        exp = 0
        for w in np.array(lw)[lv].ravel():
            cap = oracle.capacity(S, int(w), max_ctx)
            exp += B * ((cap + 63) // 64 * 64) * D * 4
        assert hw.cache_bytes(p, B, max_ctx) == exp


def test_cache_bytes_errors(hw):
    p = _pol(hw)
    for B, ctx in ((0, 10), (1, 0), (1, 1 << 31), (1, (1 << 24) + 1)):
        with pytest.raises(hw.HwkvError) as e:
            hw.cache_bytes(p, B, ctx)
        assert e.value.code == hw.EINVAL


FAKE = 0x7F0000000000  # adopted, never dereferenced by host code


def _fake_cache(hw, p, B, max_ctx):
    h = ctypes.c_void_p()
    nbytes = hw.cache_bytes(p, B, max_ctx)
    rc = hw._lib.hwkv_cache_alloc(ctypes.byref(h), p.handle, B, max_ctx, FAKE, nbytes)
    assert rc == hw.OK, hw.last_error()
    return h


def test_adopted_buffer_too_small(hw):
    p = _pol(hw)
    nbytes = hw.cache_bytes(p, 2, 1000)
    h = ctypes.c_void_p()
    assert hw._lib.hwkv_cache_alloc(ctypes.byref(h), p.handle, 2, 1000, FAKE, nbytes - 1) == hw.ENOMEM
    assert not h.value


def test_canonicalisation_and_capacity(hw):
    # S + w >= max_ctx is full; capacity S + w otherwise
    p = hw.policy_set(1, 4, 4, 64, 4, [96, 100, 200, 0], [[0, 1, 2, 3]])
    h = _fake_cache(hw, p, 1, 104)
    cap, win = ctypes.c_int64(), ctypes.c_int64()
    exp = [(100, 96), (104, 0), (104, 0), (104, 0)]
    for kv in range(4):
        assert hw._lib.hwkv_cache_unit_info(h, 0, kv, ctypes.byref(cap), ctypes.byref(win)) == 0
        assert (cap.value, win.value) == exp[kv]
        assert cap.value == oracle.capacity(4, [96, 100, 200, 0][kv], 104)
    hw._lib.hwkv_cache_free(h)


def test_host_error_paths_change_no_state(hw):
    p = _pol(hw)
    h = _fake_cache(hw, p, 2, 300)
    L = hw._lib
    n = ctypes.c_int64()
    # prefill must start at the current length
    assert L.hwkv_prefill_write(h, 0, 0, 5, 10, FAKE, FAKE, None) == hw.ESTATE
    # a full unit cannot pass max_ctx
    assert L.hwkv_prefill_write(h, 0, 0, 0, 301, FAKE, FAKE, None) == hw.ECAPACITY
    # bad indices and null inputs
    assert L.hwkv_prefill_write(h, 2, 0, 0, 1, FAKE, FAKE, None) == hw.EINVAL
    assert L.hwkv_prefill_write(h, 0, 2, 0, 1, FAKE, FAKE, None) == hw.EINVAL
    assert L.hwkv_prefill_write(h, 0, 0, 0, 1, None, FAKE, None) == hw.EINVAL
    assert L.hwkv_prefill_write(h, 0, 0, 0, -1, FAKE, FAKE, None) == hw.EINVAL
    # empty chunk: no-op
    assert L.hwkv_prefill_write(h, 0, 0, 0, 0, None, None, None) == hw.OK
    # decode on empty sequences, short workspace, bad scale
    ws = ctypes.c_size_t()
    assert L.hwkv_decode_workspace_bytes(h, ctypes.byref(ws)) == hw.OK
    assert ws.value > 0
    assert L.hwkv_decode_attn(h, 0, FAKE, ctypes.c_float(0.125), FAKE, FAKE, ws.value, None) == hw.EINVAL
    assert L.hwkv_decode_attn(h, 0, FAKE, ctypes.c_float(float("nan")), FAKE, FAKE, ws.value, None) == hw.EINVAL
    assert L.hwkv_append_decode_attn(h, 0, FAKE, FAKE, FAKE, ctypes.c_float(0.125), FAKE, FAKE, 0,
                                     None) == hw.EINVAL
    assert L.hwkv_append_decode_attn(h, 0, None, FAKE, FAKE, ctypes.c_float(0.125), FAKE, FAKE,
                                     ws.value, None) == hw.EINVAL
    assert L.hwkv_append(h, 0, None, FAKE, None) == hw.EINVAL
    assert L.hwkv_append(h, 3, FAKE, FAKE, None) == hw.EINVAL
    for layer in range(2):
        for seq in range(2):
            assert L.hwkv_cache_seq_len(h, layer, seq, ctypes.byref(n)) == hw.OK
            assert n.value == 0
    assert L.hwkv_cache_seq_len(h, 2, 0, ctypes.byref(n)) == hw.EINVAL
    L.hwkv_cache_free(h)


def test_prefill_attn_host_errors(hw):
    p = _pol(hw)
    h = _fake_cache(hw, p, 2, 300)
    L = hw._lib
    sc = ctypes.c_float(0.125)
    args = lambda layer=0, seq=0, pos0=0, n=10, q=FAKE, scale=sc: (
        h, layer, seq, pos0, n, q, FAKE, FAKE, scale, FAKE, None)
    assert L.hwkv_prefill_attn(None, 0, 0, 0, 1, FAKE, FAKE, FAKE, sc, FAKE, None) == hw.EINVAL
    assert L.hwkv_prefill_attn(*args(layer=2)) == hw.EINVAL
    assert L.hwkv_prefill_attn(*args(seq=2)) == hw.EINVAL
    assert L.hwkv_prefill_attn(*args(seq=-1)) == hw.EINVAL
    assert L.hwkv_prefill_attn(*args(n=-1)) == hw.EINVAL
    for bad in (float("nan"), float("inf"), 0.0, -0.5):
        assert L.hwkv_prefill_attn(*args(scale=ctypes.c_float(bad))) == hw.EINVAL
    assert L.hwkv_prefill_attn(*args(pos0=3)) == hw.ESTATE
    assert L.hwkv_prefill_attn(*args(n=301)) == hw.ECAPACITY
    assert L.hwkv_prefill_attn(*args(q=None)) == hw.EINVAL
    # an empty chunk is a no-op, null pointers allowed
    assert L.hwkv_prefill_attn(h, 0, 0, 0, 0, None, None, None, sc, None, None) == hw.OK
    n = ctypes.c_int64()
    for layer in range(2):
        for seq in range(2):
            assert L.hwkv_cache_seq_len(h, layer, seq, ctypes.byref(n)) == hw.OK
            assert n.value == 0
    L.hwkv_cache_free(h)


def test_prefill_sample_rows_rule():
    cfg = W.CONFIGS["prefill128k"]
    rows = W.prefill_sample_rows(cfg)
    assert len(rows) == 512 and len(set(rows)) == 512 and rows == sorted(rows)
    assert 0 <= rows[0] and rows[-1] < cfg["prompt"][0]
    N, C, S = cfg["prompt"][0], cfg["chunk"], cfg["n_sinks"]
    must = {x for p0 in range(0, N, C) for x in (p0, p0 + C - 1)}
    must |= {S + w + d for w in (2048, 8192, 32768) for d in (-1, 0, 1)} | {S - 1, S}
    assert must <= set(rows)
    assert rows == W.prefill_sample_rows(cfg)


def test_workspace_bytes_cover_full_capacity(hw):
    p = hw.policy_set(2, 4, 24, 256, 4, [2048, 8192, 32768, 0], [[0, 1, 2, 3], [3, 3, 3, 3]])
    h = _fake_cache(hw, p, 1, 114688)
    ws = ctypes.c_size_t()
    hw._lib.hwkv_decode_workspace_bytes(h, ctypes.byref(ws))
    # at least one partial (6 heads x (256 + 2) fp32) per 64 tokens of the
    # longest layer, at most one per 64 tokens plus one per unit
    rows = 4 * 114688
    part = 6 * 258 * 4
    assert ws.value <= (rows // 64 + 4) * part
    assert ws.value >= part * 4
    hw._lib.hwkv_cache_free(h)


def test_decode_timing_without_calls(hw):
    p = _pol(hw)
    h = _fake_cache(hw, p, 1, 100)
    L = hw._lib
    assert L.hwkv_decode_timing(h, 1) == hw.OK
    sp, mg, n = ctypes.c_double(), ctypes.c_double(), ctypes.c_int64()
    assert L.hwkv_decode_timing_read(h, ctypes.byref(sp), ctypes.byref(mg), ctypes.byref(n)) == hw.OK
    assert (sp.value, mg.value, n.value) == (0.0, 0.0, 0)
    assert L.hwkv_decode_timing(None, 1) == hw.EINVAL
    L.hwkv_cache_free(h)


def test_calib_selection_matches_golden_and_oracle(hw, golden):
    g = golden("calibration.json")
    for case in g["threshold"]:
        got, fl = hw.calib_select(np.array(case["means"]), case["windows"], case["n_sinks"],
                                  case["ctx"], case["tau"])
        assert got == case["choice"], case["derivation"]
        sel = [case["means"][c][h] if c < len(case["windows"]) else 1.0
               for h, c in enumerate(got)]
        assert fl == min(sel)
    for case in g["budget"]:
        assert hw.budget_select(case["rates"], case["floors"], case["budget"]) == case["chosen"]
    r = np.random.default_rng(3)
    for _ in range(300):
        K, H = int(r.integers(0, 5)), int(r.integers(1, 9))
        wins = sorted(set(int(x) for x in r.integers(1, 400, size=K)))
        K = len(wins)
        means = r.choice([0.9, 0.99, 0.995, 0.999, 1.0], size=(K, H))
        S, ctx, tau = int(r.integers(0, 5)), int(r.integers(50, 500)), float(r.choice([0.99, 0.995]))
        got, _ = hw.calib_select(means, wins, S, ctx, tau)
        assert got == oracle.select_windows(means, wins, S, ctx, tau)
        n = int(r.integers(1, 8))
        rates = r.choice([0.3, 0.45, 0.5, 0.7], size=n).tolist()
        floors = r.choice([0.99, 0.995, 0.999], size=n).tolist()
        assert hw.budget_select(rates, floors, 0.5) == oracle.budget_select(rates, floors, 0.5)


def test_calib_workspace_formula(hw):
    """The replay workspace: the row positions (256-byte aligned) and
    ceil(n_hist / 4096) + 3 partial sets of rows x q heads x (d + 4) fp32,
    whatever the number of windows."""
    for hq, d, S, n_hist, nr in [(8, 64, 4, 50, 3), (24, 256, 4, 131072, 256),
                                 (8, 128, 0, 4096, 7), (8, 128, 40, 4097, 7)]:
        rows_b = -(-nr * 4 // 256) * 256
        sets = -(-(-(-n_hist // 32)) // 128) + 3
        assert hw.calib_workspace_bytes(hq, d, S, n_hist, nr) == \
            rows_b + sets * nr * hq * (d + 4) * 4, (hq, d, S, n_hist, nr)


def test_calib_host_errors(hw):
    L = hw._lib
    sc = ctypes.c_float(0.125)
    wins = np.array([16, 64], dtype=np.int64)
    rows = np.array([3, 9, 40], dtype=np.int64)
    ws_ok = hw.calib_workspace_bytes(8, 64, 4, 50, 3)

    def call(hkv=2, hq=8, d=64, S=4, K=2, w=wins, n_hist=50, nr=3, r=rows, scale=sc,
             ws=FAKE, wsb=ws_ok, ref=None, chk=None, scores=FAKE):
        return L.hwkv_calib_replay(hkv, hq, d, S, K, w.ctypes.data, n_hist, FAKE, FAKE, nr,
                                   r.ctypes.data, FAKE, scale, FAKE, scores, FAKE, ref, chk,
                                   ws, wsb, None)
    assert call(d=96) == hw.EINVAL
    assert call(hq=6) == hw.EINVAL                  # G = 3
    assert call(S=-1) == hw.EINVAL
    assert call(w=np.array([64, 16], dtype=np.int64)) == hw.EINVAL
    assert call(w=np.array([0, 16], dtype=np.int64)) == hw.EINVAL
    assert call(r=np.array([9, 3, 40], dtype=np.int64)) == hw.EINVAL
    assert call(r=np.array([3, 3, 40], dtype=np.int64)) == hw.EINVAL
    assert call(r=np.array([3, 9, 50], dtype=np.int64)) == hw.EINVAL   # >= n_hist
    assert call(scale=ctypes.c_float(float("nan"))) == hw.EINVAL
    assert call(ws=None) == hw.EINVAL
    assert call(wsb=ws_ok - 1) == hw.EINVAL
    assert call(ref=FAKE) == hw.EINVAL               # check missing
    assert call(scores=None) == hw.EINVAL
    assert call(n_hist=0) == hw.EINVAL
    n = ctypes.c_size_t()
    assert L.hwkv_calib_workspace_bytes(8, 64, 4, 50, 0, ctypes.byref(n)) == hw.EINVAL
    assert L.hwkv_calib_workspace_bytes(8, 96, 4, 50, 3, ctypes.byref(n)) == hw.EINVAL
    ch = np.zeros(2, dtype=np.int32)
    assert L.hwkv_calib_select(2, 2, wins.ctypes.data, 4, 100, None, ctypes.c_double(0.99),
                               ch.ctypes.data, None) == hw.EINVAL
    m = np.ones((2, 2))
    assert L.hwkv_calib_select(2, 2, wins.ctypes.data, 4, 100, m.ctypes.data,
                               ctypes.c_double(1.5), ch.ctypes.data, None) == hw.EINVAL
    g = ctypes.c_int32()
    assert L.hwkv_budget_select(0, None, None, ctypes.c_double(0.5), ctypes.byref(g)) == hw.EINVAL


def test_policy_artifact_format(hw, golden):
    g = golden("policy_artifact.json")
    a = g["inputs"]
    p = hw.policy_set(a["n_layers"], a["n_kv_heads"], a["n_q_heads"], a["head_dim"],
                      a["n_sinks"], a["level_window"], a["level_of_unit"])
    text = hw.policy_serialize(p, a["artifact"], a["seed"], a["grid_index"], a["tau"], a["rate"],
                               a["floor"])
    assert text == g["text"]
    q, meta = hw.policy_deserialize(g["text"])
    assert meta == {k: a[k] for k in ("artifact", "seed", "grid_index", "tau", "rate", "floor")}
    assert (q.n_layers, q.n_kv_heads, q.n_q_heads, q.head_dim) == (2, 2, 8, 64)


def test_policy_artifact_round_trip(hw):
    r = np.random.default_rng(9)
    for _ in range(100):
        L, H = int(r.integers(1, 6)), int(r.choice([1, 2, 4]))
        lw = [int(x) for x in r.integers(1, 100000, size=int(r.integers(1, 5)))] + [0]
        lv = r.integers(0, len(lw), size=(L, H)).tolist()
        S = int(r.integers(0, 9))
        p = hw.policy_set(L, H, H * int(r.choice([1, 2, 4, 6, 8])), int(r.choice([64, 128, 256])),
                          S, lw, lv)
        meta = dict(artifact=f"r{int(r.integers(1 << 30))}", seed=int(r.integers(0, 1 << 63)),
                    grid_index=int(r.integers(0, 50)), tau=float(r.random()),
                    rate=float(r.random()), floor=float(r.random()))
        text = hw.policy_serialize(p, **meta)
        q, back = hw.policy_deserialize(text)
        assert back == meta                                   # doubles bit for bit
        assert hw.policy_serialize(q, **meta) == text
        for ctx in (1, 1000, 123457):
            assert hw.policy_rate(q, ctx) == hw.policy_rate(p, ctx)
            assert hw.policy_bytes(q, ctx) == hw.policy_bytes(p, ctx)


def test_policy_artifact_rejects_malformed_text(hw, golden):
    good = golden("policy_artifact.json")["text"]
    bad = [
        good.replace('"format": "hwkv-policy/1"', '"format": "hwkv-policy/2"'),
        good.replace('  "seed": 42,\n', ''),                             # missing key
        good.replace('"seed": 42,', '"seed": 42,\n  "seed": 43,'),        # repeated key
        good.replace('"seed": 42,', '"seed": 42,\n  "colour": 1,'),       # unknown key
        good + "x",                                                       # trailing text
        good[:-10],                                                       # truncated
        good.replace('[1, 1]\n', '[1, 1.5]\n'),                           # non-integer level
        good.replace('[1, 1]\n', '[1]\n'),                                # ragged rows
        good.replace('[1, 1]\n', '[1, 2]\n'),                             # level out of range
        good.replace('"n_layers": 2', '"n_layers": 3'),                   # shape mismatch
        good.replace('"seed": 42', '"seed": -42'),
        good.replace('"tau": 0.5', '"tau": "0.5"'),
        good.replace('"run-1"', '"run\\"1"'),
    ]
    for text in bad:
        with pytest.raises(hw.HwkvError) as e:
            hw.policy_deserialize(text)
        assert e.value.code == hw.EINVAL, text
    p = hw.policy_set(1, 1, 1, 64, 0, [0], [[0]])
    for aid in ('a"b', "a\\b", "tab\there", "é"):
        with pytest.raises((hw.HwkvError, UnicodeEncodeError)):
            hw.policy_serialize(p, aid, 1, 0, 0.5, 0.5, 1.0)
    n = ctypes.c_size_t()
    assert hw._lib.hwkv_policy_serialize(p.handle, b"x", 1, 0, ctypes.c_double(0.5),
                                         ctypes.c_double(0.5), ctypes.c_double(1.0), None, 0,
                                         ctypes.byref(n)) == hw.OK
    small = ctypes.create_string_buffer(n.value)                          # no room for the NUL
    assert hw._lib.hwkv_policy_serialize(p.handle, b"x", 1, 0, ctypes.c_double(0.5),
                                         ctypes.c_double(0.5), ctypes.c_double(1.0), small,
                                         n.value, ctypes.byref(n)) == hw.ENOMEM


def _deserialize_exact(hw, raw):
    """hwkv_policy_deserialize over a malloc'd block of exactly len(raw)
    bytes with no NUL after it: a read past the stated length is then a heap
    overflow that the address-sanitizer build of the library reports.
    Returns (status, policy handle or None)."""
    libc = ctypes.CDLL(None)
    libc.malloc.restype = ctypes.c_void_p
    libc.malloc.argtypes = [ctypes.c_size_t]
    libc.free.argtypes = [ctypes.c_void_p]
    buf = libc.malloc(max(1, len(raw)))
    try:
        ctypes.memmove(buf, raw, len(raw))
        h = ctypes.c_void_p()
        aid = ctypes.create_string_buffer(256)
        seed, gi = ctypes.c_uint64(), ctypes.c_int32()
        tau, rate, fl = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
        rc = hw._lib.hwkv_policy_deserialize(ctypes.cast(buf, ctypes.c_char_p), len(raw),
                                             ctypes.byref(h), aid, 256, ctypes.byref(seed),
                                             ctypes.byref(gi), ctypes.byref(tau),
                                             ctypes.byref(rate), ctypes.byref(fl))
    finally:
        libc.free(buf)
    return rc, h.value


def test_policy_artifact_every_prefix_and_seeded_mutations(hw, golden):
    """Every prefix of a valid artifact that cuts into its text is refused;
    seeded one-byte
    mutations are refused with EINVAL or, where the text stays well formed,
    parse to a policy whose artifact parses back to itself.  Run under the
    sanitizer tier, this is where an unchecked read or length shows."""
    good = golden("policy_artifact.json")["text"].encode("ascii")
    rc, h = _deserialize_exact(hw, good)
    assert rc == hw.OK and h
    hw._lib.hwkv_policy_free(ctypes.c_void_p(h))
    body = len(good.rstrip())          # trailing white space is optional
    for n in range(len(good)):
        rc, h = _deserialize_exact(hw, good[:n])
        if n >= body:
            assert rc == hw.OK, n
            hw._lib.hwkv_policy_free(ctypes.c_void_p(h))
        else:
            assert (rc, h) == (hw.EINVAL, None), n
    r = np.random.default_rng(17)
    alphabet = b'"{}[],:-+.eE0129 \\\n\x00\xff'
    accepted = 0
    for _ in range(600):
        raw = bytearray(good)
        for _k in range(int(r.integers(1, 4))):
            i = int(r.integers(0, len(raw)))
            raw[i] = alphabet[int(r.integers(0, len(alphabet)))]
        rc, h = _deserialize_exact(hw, bytes(raw))
        assert rc in (hw.OK, hw.EINVAL)
        if rc == hw.OK:
            accepted += 1
            hw._lib.hwkv_policy_free(ctypes.c_void_p(h))
            q, meta = hw.policy_deserialize(bytes(raw))
            text = hw.policy_serialize(q, **meta)
            q2, meta2 = hw.policy_deserialize(text)
            assert meta2 == meta and hw.policy_serialize(q2, **meta2) == text
        else:
            assert h is None
    assert accepted < 600


# --------------------------------------------------------------------------
# cache formats
# --------------------------------------------------------------------------
def test_format_accounting_matches_oracle(hw):
    r = np.random.default_rng(3)
    for _ in range(30):
        L, H, D = int(r.integers(1, 4)), int(r.choice([1, 2, 4])), int(r.choice([64, 128, 256]))
        lw = [int(x) for x in r.integers(1, 3000, size=3)] + [0]
        lv = r.integers(0, 4, size=(L, H))
        S = int(r.integers(0, 8))
        ctx = int(r.integers(1, 5000))
        B = int(r.integers(1, 4))
        p = hw.policy_set(L, H, H, D, S, lw, lv.tolist())
        wins = np.array(lw)[lv].ravel()
        for fmt, b in (("bf16", 2.0), ("f16", 2.0), ("fp8", 1.0)):
            assert hw.policy_bytes(p, ctx, fmt) == pytest.approx(
                oracle.policy_bytes(ctx, S, wins, D, D, b, b), rel=1e-14)
        # fp8 elements are one byte: exactly half the 16-bit layouts
        b16 = hw.cache_bytes(p, B, ctx)
        assert hw.cache_bytes(p, B, ctx, "f16") == b16
        assert 2 * hw.cache_bytes(p, B, ctx, "fp8") == b16


def test_format_context_limit(hw):
    # one unit's K or V must stay below 2^31 bytes: twice the tokens at 1 byte
    p = _pol(hw)
    n = (1 << 24) + 1                     # head_dim 64: over the limit at 2 bytes
    with pytest.raises(hw.HwkvError):
        hw.cache_bytes(p, 1, n, "bf16")
    assert hw.cache_bytes(p, 1, n, "fp8") > 0
    with pytest.raises(hw.HwkvError):
        hw.cache_bytes(p, 1, (1 << 25) + 1, "fp8")


def _alloc_fmt(hw, p, fmt, ks=None, vs=None, B=1, max_ctx=300):
    h = ctypes.c_void_p()
    nbytes = hw.cache_bytes(p, B, max_ctx, "bf16")
    arr = lambda x: None if x is None else np.ascontiguousarray(x, dtype=np.float32)
    ka, va = arr(ks), arr(vs)
    rc = hw._lib.hwkv_cache_alloc_format(
        ctypes.byref(h), p.handle, B, max_ctx, fmt,
        None if ka is None else ka.ctypes.data_as(ctypes.c_void_p),
        None if va is None else va.ctypes.data_as(ctypes.c_void_p), FAKE, nbytes)
    return rc, h


def test_format_alloc_validation(hw):
    p = _pol(hw)                          # 2 layers x 2 kv heads
    good = np.full((2, 2), 0.05)
    # unknown formats
    for fmt in (-1, 3, 99):
        rc, h = _alloc_fmt(hw, p, fmt)
        assert rc == hw.EINVAL and not h.value
        b = ctypes.c_size_t()
        assert hw._lib.hwkv_cache_bytes_format(p.handle, 1, 300, fmt, ctypes.byref(b)) == hw.EINVAL
        d = ctypes.c_double()
        assert hw._lib.hwkv_policy_bytes_format(p.handle, 300, fmt, ctypes.byref(d)) == hw.EINVAL
    with pytest.raises(ValueError):       # the binding names the formats
        hw.cache_bytes(p, 1, 300, "fp4")
    # scales belong to fp8 only
    for fmt in (0, 1):
        rc, h = _alloc_fmt(hw, p, fmt, ks=good)
        assert rc == hw.EINVAL and not h.value
    # each scale positive, finite, normal
    for bad in (0.0, -1.0, float("inf"), float("nan"), 1e-40):
        ks = good.copy()
        ks[1, 0] = bad
        rc, h = _alloc_fmt(hw, p, 2, ks=ks)
        assert rc == hw.EINVAL and not h.value, bad
        rc, h = _alloc_fmt(hw, p, 2, vs=ks)
        assert rc == hw.EINVAL and not h.value, bad
    # accepted, and reported back
    ks = np.arange(1, 5, dtype=np.float32).reshape(2, 2) / 8
    rc, h = _alloc_fmt(hw, p, 2, ks=ks)
    assert rc == hw.OK, hw.last_error()
    code = ctypes.c_int32()
    k_out = np.zeros((2, 2), dtype=np.float32)
    v_out = np.zeros((2, 2), dtype=np.float32)
    assert hw._lib.hwkv_cache_format(h, ctypes.byref(code), k_out.ctypes.data_as(ctypes.c_void_p),
                                     v_out.ctypes.data_as(ctypes.c_void_p)) == hw.OK
    assert code.value == 2 and np.array_equal(k_out, ks) and np.all(v_out == 1.0)
    # prefill attention reads bf16 caches only: rejected before any device work
    rc = hw._lib.hwkv_prefill_attn(h, 0, 0, 0, 4, FAKE, FAKE, FAKE, 0.1, FAKE, None)
    assert rc == hw.EINVAL and "bf16" in hw.last_error()
    hw._lib.hwkv_cache_free(h)


# --------------------------------------------------------------------------
# paged full units
# --------------------------------------------------------------------------
def _r256(x):
    return (x + 255) // 256 * 256


def test_paged_cache_bytes(hw):
    r = np.random.default_rng(5)
    for _ in range(40):
        L, H, D = int(r.integers(1, 4)), int(r.choice([1, 2, 4])), int(r.choice([64, 128, 256]))
        lw = [int(x) for x in r.integers(1, 3000, size=3)] + [0]
        lv = r.integers(0, 4, size=(L, H))
        S = int(r.integers(0, 8))
        B = int(r.integers(1, 5))
        ctx = int(r.integers(1, 6000))
        n_pages = int(r.integers(0, 50))
        fmt, b = [("bf16", 2), ("f16", 2), ("fp8", 1)][int(r.integers(0, 3))]
        p = hw.policy_set(L, H, H, D, S, lw, lv.tolist())
        finite, n_full = 0, 0
        for w in np.array(lw)[lv].ravel():
            if w == 0 or S + w >= ctx:
                n_full += 1
            else:
                finite += B * ((S + int(w) + 63) // 64 * 64) * D * 2 * b
        exp = _r256(_r256(finite) + n_pages * 2 * 256 * D * b) + n_full * B * ((ctx + 255) // 256) * 4
        assert hw.cache_bytes(p, B, ctx, fmt, n_pages=n_pages) == exp
        # with no full unit and no pool, only the 256-byte rounding remains
        if n_full == 0 and n_pages == 0:
            assert hw.cache_bytes(p, B, ctx, fmt, n_pages=0) == _r256(hw.cache_bytes(p, B, ctx, fmt))
    p = _pol(hw)
    for bad in (-1, 1 << 31):
        with pytest.raises(hw.HwkvError):
            hw.cache_bytes(p, 1, 300, n_pages=bad)


def _fake_paged(hw, p, B, max_ctx, n_pages):
    h = ctypes.c_void_p()
    nbytes = hw.cache_bytes(p, B, max_ctx, n_pages=n_pages)
    rc = hw._lib.hwkv_cache_alloc_paged(ctypes.byref(h), p.handle, B, max_ctx, 0, None, None,
                                        n_pages, FAKE, nbytes)
    assert rc == hw.OK, hw.last_error()
    return h


def test_paged_pool_checks_before_device_work(hw):
    p = _pol(hw)                        # 2 layers x 2 kv heads: one full unit per layer
    L = hw._lib
    h = _fake_paged(hw, p, 2, 1000, 1)
    t, f = ctypes.c_int64(), ctypes.c_int64()
    assert L.hwkv_cache_pages(h, ctypes.byref(t), ctypes.byref(f)) == hw.OK
    assert (t.value, f.value) == (1, 1)
    # 300 rows of the full unit need 2 pages: ENOMEM before any launch
    assert L.hwkv_prefill_write(h, 0, 0, 0, 300, FAKE, FAKE, None) == hw.ENOMEM
    assert "page" in hw.last_error()
    n = ctypes.c_int64()
    assert L.hwkv_cache_seq_len(h, 0, 0, ctypes.byref(n)) == hw.OK and n.value == 0
    assert L.hwkv_cache_pages(h, ctypes.byref(t), ctypes.byref(f)) == hw.OK and f.value == 1
    assert L.hwkv_cache_reset_seq(h, 1) == hw.OK
    assert L.hwkv_cache_reset_seq(h, 2) == hw.EINVAL
    assert L.hwkv_cache_reset_seq(h, -1) == hw.EINVAL
    L.hwkv_cache_free(h)
    # an unpaged cache reports no pool
    h = _fake_cache(hw, p, 1, 300)
    assert L.hwkv_cache_pages(h, ctypes.byref(t), ctypes.byref(f)) == hw.OK
    assert (t.value, f.value) == (0, 0)
    L.hwkv_cache_free(h)


def test_read_probe_argument_errors():
    """The read probe (its own library, measurement tooling beside the
    runtime) validates everything before touching the device, and the
    runtime's library does not export it."""
    from paper_2609_02029_amd import build
    L = ctypes.CDLL(build.PROBE_LIB)
    L.hwkv_read_probe.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                  ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    f = ctypes.c_void_p(FAKE)
    assert L.hwkv_read_probe(None, 65536, 0, 2, f, None) == 1
    assert L.hwkv_read_probe(f, 65536, 0, 2, None, None) == 1
    for bytes_ in (0, -65536, 65535, 65536 + 1024, 1 << 31):
        assert L.hwkv_read_probe(f, bytes_, 0, 2, f, None) == 1, bytes_
    assert L.hwkv_read_probe(f, 65536, 2, 2, f, None) == 1
    for pattern in (0, 1):
        for wps in (0, 1, 3, 16):
            assert L.hwkv_read_probe(f, 65536, pattern, wps, f, None) == 1, wps
    runtime = ctypes.CDLL(build.LIB)
    assert not hasattr(runtime, "hwkv_read_probe")

