"""Pins for the fp64 oracle, checked against things other than itself.

Each test ties part of the oracle to a value the paper prints, a hand
derivation, a closed form, an independent brute-force simulation, or a
library routine (torch fp64 scaled-dot-product attention).  A plausible
mistake anywhere in the oracle (an off-by-one window edge, a dropped sink, a
wrong softmax shift sign, a swapped GQA mapping, a transposed operand) fails
at least one of them.
"""
import collections
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W


def f64(bits):
    """Independent bf16 widening (numpy bit view) used by the tests."""
    return W.bf16_bits_to_f32(bits).astype(np.float64)


def bf16(x):
    return W.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


# --------------------------------------------------------------------------
# an independent residency simulation: sinks + a bounded deque of the most
# recent tokens (no slot arithmetic, no window comparisons)
# --------------------------------------------------------------------------
class DequeUnit:
    def __init__(self, n_sinks, window):
        self.n_sinks = n_sinks
        self.window = window
        self.sinks = []
        self.recent = collections.deque(maxlen=window if window else None)
        self.n = 0

    def push(self):
        p = self.n
        if len(self.sinks) < self.n_sinks:
            self.sinks.append(p)
        else:
            self.recent.append(p)
        self.n += 1

    def resident(self):
        return set(self.sinks) | set(self.recent)


# --------------------------------------------------------------------------
# bf16 widening
# --------------------------------------------------------------------------
def test_bf16_widening_exact():
    r = np.random.default_rng(0)
    bits = r.integers(0, 1 << 16, size=2000, dtype=np.uint16)
    bits = bits[~np.isnan(W.bf16_bits_to_f32(bits))]
    a = oracle.bf16_to_f64(bits)
    b = f64(bits)
    assert np.array_equal(a, b)


# --------------------------------------------------------------------------
# accounting: printed values
# --------------------------------------------------------------------------
def test_paper_sink_recent_control(golden):
    g = golden("accounting.json")["sink_recent_control"]
    S, w, C = g["n_sinks"], g["window"], g["ctx"]
    assert oracle.retained_tokens(C, S, w) == g["cache_tokens"]
    assert oracle.capacity(S, w, C) == g["cache_tokens"]
    r = oracle.rate(C, S, [w])
    assert round(100 * r, 2) == g["rate_percent_2dp"]
    assert r == g["cache_tokens"] / C
    # eviction begins above 90,368 tokens
    n0 = g["last_length_without_eviction"]
    assert oracle.resident_count(n0, S, w) == n0
    assert oracle.resident_count(n0 + 1, S, w) == n0
    assert not oracle.is_resident(S, n0 + 1, S, w)      # first non-sink token gone
    assert oracle.is_resident(S - 1, n0 + 1, S, w)      # sinks stay
    assert oracle.is_resident(S + 1, n0 + 1, S, w)


def test_paper_quarter_and_half(golden):
    g = golden("accounting.json")
    q = g["quarter_example"]
    assert oracle.rate(q["ctx"], q["n_sinks"], [q["window"]]) == q["rate"]
    h = g["half_example"]
    assert oracle.rate(h["ctx"], h["n_sinks"], h["windows"]) == h["rate"]


def test_nominal_storage_is_linear_sum():
    # Eq. nominal-storage: r_C(w) (d^K b^K + d^V b^V) summed over units
    C, S = 4096, 3
    ws = [0, 16, 4093, 5000, 100]
    got = oracle.policy_bytes(C, S, ws, 256, 128, 2.0, 1.0)
    exp = C * 640 + 19 * 640 + C * 640 + C * 640 + 103 * 640
    assert got == exp
    assert oracle.rate(C, S, [0] * 7) == 1.0


# --------------------------------------------------------------------------
# residency: closed form and brute force
# --------------------------------------------------------------------------
def test_retained_count_closed_form():
    for S in range(0, 4):
        for w in range(1, 9):
            for n in range(0, 41):
                assert oracle.resident_count(n, S, w) == min(n, S + w), (S, w, n)
            for n in range(0, 41):
                assert oracle.resident_count(n, S, 0) == n


def test_window_at_least_context_is_full():
    # "any w >= C is equivalent to full"
    for S in range(0, 4):
        for n in range(1, 30):
            for w in range(n, n + 4):
                for p in range(n):
                    assert oracle.is_resident(p, n, S, w)
                    assert oracle.slot(p, S, w) == p
    assert oracle.capacity(4, 100, 104) == 104
    assert oracle.capacity(4, 100, 105) == 104
    assert oracle.capacity(4, 0, 105) == 105


def _run_ops(unit, deque_unit, ops):
    for op in ops:
        if op[0] == "prefill":
            unit.prefill(op[1], op[2])
            for _ in range(op[2] - op[1]):
                deque_unit.push()
        else:
            unit.append()
            deque_unit.push()


def test_slot_table_matches_deque_simulation():
    r = np.random.default_rng(1)
    for trial in range(300):
        S = int(r.integers(0, 4))
        full = r.random() < 0.2
        w = 0 if full else int(r.integers(1, 9))
        max_ctx = 60
        unit = oracle.UnitTable(S, w, max_ctx)
        dq = DequeUnit(S, w)
        n = 0
        ops = []
        while n < 45:
            if r.random() < 0.5:
                c = int(r.integers(1, 12))
                ops.append(("prefill", n, n + c))
                n += c
            else:
                ops.append(("append",))
                n += 1
        for op in ops:
            _run_ops(unit, dq, [op])
            occ = unit.table[unit.table >= 0]
            # the set of stored positions is the deque's resident set
            assert set(occ.tolist()) == dq.resident(), (S, w, ops)
            # occupied slots are exactly [0, n_valid), no duplicates
            nv = len(dq.resident())
            assert np.all(unit.table[:nv] >= 0) and np.all(unit.table[nv:] < 0)
            assert len(set(occ.tolist())) == occ.size
            # sinks sit in slots 0..S-1
            for p in range(min(S, unit.n)):
                assert unit.table[p] == p


def test_worked_slot_tables(golden):
    g = golden("worked_slots.json")
    for seq in g["sequences"]:
        u = oracle.UnitTable(g["n_sinks"], g["window"], g["max_ctx"])
        for op in seq["ops"]:
            if op[0] == "prefill":
                u.prefill(op[1], op[2])
            else:
                u.append()
        assert u.table.tolist() == seq["table"], seq["why"]


def test_prefill_then_appends_equals_longer_prefill():
    for S in range(0, 3):
        for w in (1, 2, 5, 0):
            for P in range(0, 20):
                for k in range(0, 8):
                    a = oracle.UnitTable(S, w, 64)
                    a.prefill(0, P)
                    for _ in range(k):
                        a.append()
                    b = oracle.UnitTable(S, w, 64)
                    b.prefill(0, P + k)
                    assert np.array_equal(a.table, b.table)


def test_chunked_prefill_equals_one_shot():
    r = np.random.default_rng(2)
    for trial in range(200):
        S = int(r.integers(0, 4))
        w = int(r.integers(0, 10))
        P = int(r.integers(1, 50))
        cuts = sorted(set(r.integers(1, P, size=int(r.integers(0, 5))).tolist())) if P > 1 else []
        a = oracle.UnitTable(S, w, 64)
        prev = 0
        for c in cuts + [P]:
            a.prefill(prev, c)
            prev = c
        b = oracle.UnitTable(S, w, 64)
        b.prefill(0, P)
        assert np.array_equal(a.table, b.table)


def test_capacity_error_on_full_unit_overflow():
    u = oracle.UnitTable(4, 0, 8)
    u.prefill(0, 8)
    with pytest.raises(ValueError):
        u.append()
    # a finite unit never overflows
    v = oracle.UnitTable(1, 3, 8)
    v.prefill(0, 8)
    for _ in range(20):
        v.append()


# --------------------------------------------------------------------------
# attention
# --------------------------------------------------------------------------
def test_worked_attention(golden):
    g = golden("worked_attention.json")
    q = bf16(g["q"])
    k = bf16(g["k"])
    v = bf16(g["v"])
    for c in g["cases"]:
        o = oracle.attend_row(q, k, v, c["t"], c["n_sinks"], c["window"], math.log(2.0))
        assert np.allclose(o, c["out"], rtol=0, atol=1e-12), c["why"]


def _rand_bf16(r, shape, scale=1.0):
    return bf16(r.standard_normal(shape).astype(np.float32) * scale)


def test_all_full_matches_torch_causal_sdpa():
    r = np.random.default_rng(3)
    for n, d in ((1, 8), (7, 16), (33, 64)):
        q = _rand_bf16(r, (n, d))
        k = _rand_bf16(r, (n, d))
        v = _rand_bf16(r, (n, d))
        scale = 1.0 / math.sqrt(d)
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(f64(q))[None, None], torch.from_numpy(f64(k))[None, None],
            torch.from_numpy(f64(v))[None, None], is_causal=True, scale=scale)[0, 0].numpy()
        for t in range(n):
            o = oracle.attend_row(q[t], k, v, t, 4, 0, scale)
            assert np.allclose(o, ref[t], rtol=1e-12, atol=1e-12)


def test_windowed_matches_sdpa_with_deque_mask():
    # the mask comes from the independent deque simulation, the arithmetic
    # from torch's fp64 attention
    r = np.random.default_rng(4)
    n, d = 40, 32
    for S, w in ((0, 1), (0, 5), (2, 3), (3, 1), (1, 39), (4, 8)):
        q = _rand_bf16(r, (n, d))
        k = _rand_bf16(r, (n, d), 2.0)
        v = _rand_bf16(r, (n, d))
        dq = DequeUnit(S, w)
        mask = np.zeros((n, n), dtype=bool)
        for t in range(n):
            dq.push()
            for s in dq.resident():
                mask[t, s] = True
        scale = 1.0 / math.sqrt(d)
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(f64(q))[None, None], torch.from_numpy(f64(k))[None, None],
            torch.from_numpy(f64(v))[None, None], attn_mask=torch.from_numpy(mask)[None, None],
            scale=scale)[0, 0].numpy()
        for t in range(n):
            o = oracle.attend_row(q[t], k, v, t, S, w, scale)
            assert np.allclose(o, ref[t], rtol=1e-12, atol=1e-12), (S, w, t)


def test_gqa_mapping_matches_torch_enable_gqa():
    # contiguous GQA groups: query head qh reads kv head qh // G
    r = np.random.default_rng(5)
    B, Hq, Hkv, d, n = 2, 6, 2, 16, 12
    q = _rand_bf16(r, (B, Hq, d))
    kh = [_rand_bf16(r, (n, Hkv, d)) for _ in range(B)]
    vh = [_rand_bf16(r, (n, Hkv, d)) for _ in range(B)]
    t = np.array([n - 1, n - 4])
    out = oracle.decode_layer(q, kh, vh, t, 0, [0, 0], 0.25, n_threads=3)
    for b in range(B):
        T = t[b] + 1
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(f64(q[b]))[None, :, None, :],
            torch.from_numpy(f64(kh[b][:T])).permute(1, 0, 2)[None],
            torch.from_numpy(f64(vh[b][:T])).permute(1, 0, 2)[None],
            scale=0.25, enable_gqa=True)[0, :, 0, :].numpy()
        assert np.allclose(out[b], ref, rtol=1e-12, atol=1e-12)


def test_decode_layer_threads_are_bitwise_stable():
    r = np.random.default_rng(6)
    B, Hq, Hkv, d, n = 3, 8, 2, 32, 50
    q = _rand_bf16(r, (B, Hq, d))
    kh = [_rand_bf16(r, (n, Hkv, d)) for _ in range(B)]
    vh = [_rand_bf16(r, (n, Hkv, d)) for _ in range(B)]
    t = np.array([49, 10, 30])
    a = oracle.decode_layer(q, kh, vh, t, 2, [5, 0], 0.2, n_threads=1)
    b = oracle.decode_layer(q, kh, vh, t, 2, [5, 0], 0.2, n_threads=5)
    assert np.array_equal(a, b)
    for bb in range(B):
        for qh in range(Hq):
            h = qh // (Hq // Hkv)
            o = oracle.attend_row(q[bb, qh], kh[bb][:, h], vh[bb][:, h], t[bb], 2,
                                  [5, 0][h], 0.2)
            assert np.array_equal(o, a[bb, qh])


def test_local_truncation_identity():
    # Eq. local-attention-bound: o_F - o_w = m_w (mu_wbar - mu_w), norm <= m_w Delta_V
    r = np.random.default_rng(7)
    n, d = 30, 16
    for S, w in ((0, 4), (2, 6), (1, 1), (3, 20)):
        q = _rand_bf16(r, (d,), 3.0)
        k = _rand_bf16(r, (n, d))
        v = _rand_bf16(r, (n, d))
        t = n - 1
        scale = 0.5
        oF = oracle.attend_row(q, k, v, t, S, 0, scale)
        ow = oracle.attend_row(q, k, v, t, S, w, scale)
        z = torch.from_numpy(f64(k)) @ torch.from_numpy(f64(q)) * scale
        alpha = torch.softmax(z, dim=0).numpy()
        dq = DequeUnit(S, w)
        for _ in range(n):
            dq.push()
        keep = sorted(dq.resident())
        omit = [s for s in range(n) if s not in dq.resident()]
        vv = f64(v)
        mw = alpha[omit].sum()
        mu_keep = (alpha[keep, None] * vv[keep]).sum(0) / (1 - mw)
        mu_omit = (alpha[omit, None] * vv[omit]).sum(0) / mw
        assert np.allclose(ow, mu_keep, rtol=1e-11, atol=1e-12)
        assert np.allclose(oF - ow, mw * (mu_omit - mu_keep), rtol=1e-10, atol=1e-12)
        dv = max(np.linalg.norm(vv[a] - vv[b]) for a in keep for b in omit)
        assert np.linalg.norm(oF - ow) <= mw * dv * (1 + 1e-12)


def test_single_token_and_zero_keys():
    r = np.random.default_rng(8)
    d = 64
    q = _rand_bf16(r, (d,))
    k = _rand_bf16(r, (10, d))
    v = _rand_bf16(r, (10, d))
    o = oracle.attend_row(q, k, v, 0, 4, 3, 0.125)
    assert np.array_equal(o, f64(v[0]))
    kz = np.zeros_like(k)
    for S, w, t in ((0, 3, 9), (2, 3, 9), (0, 0, 6)):
        o = oracle.attend_row(q, kz, v, t, S, w, 0.125)
        dq = DequeUnit(S, w)
        for _ in range(t + 1):
            dq.push()
        mean = f64(v)[sorted(dq.resident())].mean(0)
        assert np.allclose(o, mean, rtol=1e-14, atol=1e-15)


def test_compacted_equals_masked_full_bitwise():
    r = np.random.default_rng(9)
    d = 32
    for S, w, P, k in ((4, 8, 50, 5), (0, 3, 10, 9), (2, 0, 20, 3), (1, 100, 30, 2)):
        n_total = P + k
        kh = _rand_bf16(r, (n_total, d))
        vh = _rand_bf16(r, (n_total, d))
        q = _rand_bf16(r, (d,))
        u = oracle.UnitTable(S, w, 200)
        u.prefill(0, P)
        for _ in range(k):
            u.append()
        ck = np.zeros((u.cap, d), dtype=np.uint16)
        cv = np.zeros((u.cap, d), dtype=np.uint16)
        occ = u.table >= 0
        ck[occ] = kh[u.table[occ]]
        cv[occ] = vh[u.table[occ]]
        a = oracle.attend_slots(q, ck, cv, u.table, 0.3)
        b = oracle.attend_row(q, kh, vh, n_total - 1, S, w, 0.3)
        assert np.array_equal(a, b)
        perm = r.permutation(u.cap)
        c = oracle.attend_slots(q, ck[perm], cv[perm], u.table[perm], 0.3)
        assert np.array_equal(a, c)


# ---------------------------------------------------------------------------
# calibration score and selection rules
# ---------------------------------------------------------------------------
def test_cos_eval_special_cases():
    r = np.random.default_rng(7)
    u = r.standard_normal(64)
    v = r.standard_normal(64)
    assert oracle.cos_eval(u, u) == pytest.approx(1.0, abs=1e-15)
    assert oracle.cos_eval(u, -u) == pytest.approx(-1.0, abs=1e-15)
    e0, e1 = np.eye(64)[0], np.eye(64)[1]
    assert oracle.cos_eval(e0, e1) == 0.0
    # scale invariance for positive factors
    assert oracle.cos_eval(3.0 * u, 0.25 * v) == pytest.approx(oracle.cos_eval(u, v), abs=1e-15)
    # the library routine on ordinary vectors
    for _ in range(20):
        a, b = r.standard_normal(256), r.standard_normal(256)
        ref = float(np.dot(a, b) / (np.linalg.norm(a) * np.linalg.norm(b)))
        assert oracle.cos_eval(a, b) == pytest.approx(ref, abs=1e-14)
    # stabilisation: norms <= 1e-12 count as zero
    z = np.zeros(64)
    tiny = e0 * 1e-13
    small = e0 * 1e-11
    assert oracle.cos_eval(z, z) == 1.0
    assert oracle.cos_eval(z, u) == 0.0 and oracle.cos_eval(u, z) == 0.0
    assert oracle.cos_eval(tiny, z) == 1.0 and oracle.cos_eval(tiny, e1 * 1e-13) == 1.0
    assert oracle.cos_eval(tiny, u) == 0.0
    assert oracle.cos_eval(small, e0) == pytest.approx(1.0, abs=1e-15)
    assert oracle.cos_eval(e0 * 1e-12, e0) == 0.0          # the bound is inclusive


def test_replay_window_covering_the_history_is_full():
    """A window that reaches back to position 0 retains the whole history, so
    its candidate output is the full one bit for bit and scores one."""
    r = np.random.default_rng(8)
    N, Hkv, G, d = 40, 2, 3, 16
    k = W.f32_to_bf16_bits(r.standard_normal((N, Hkv, d)).astype(np.float32))
    v = W.f32_to_bf16_bits(r.standard_normal((N, Hkv, d)).astype(np.float32))
    rows = [5, 17, 39]
    q = W.f32_to_bf16_bits(r.standard_normal((3, Hkv * G, d)).astype(np.float32))
    outs = oracle.replay_outputs(q, k, v, rows, 2, [40, 37, 7, 0], 0.25)
    assert np.array_equal(outs[0], outs[3])          # 40 >= t + 1 for every row
    assert np.array_equal(outs[1, :2], outs[3, :2])  # 2 + 37 covers rows 5 and 17
    assert not np.array_equal(outs[1, 2], outs[3, 2])  # ... but leaves out position 2 of row 39
    sc = oracle.replay_scores(outs)
    assert np.all(np.abs(sc[0] - 1.0) <= 1e-15)
    assert np.all(np.abs(sc[2, 0] - 1.0) <= 1e-15)   # 2 + 7 >= 6 covers row 5
    assert np.all(sc[2, 1:] < 1.0 - 1e-6)            # rows 17 and 39 lose keys


def test_head_means_average_each_group():
    K, R, Hq, G = 2, 3, 6, 3
    scores = np.zeros((K, R, Hq))
    for k in range(K):
        for r_ in range(R):
            for q in range(Hq):
                scores[k, r_, q] = 100 * k + 10 * r_ + q
    m = oracle.head_means(scores, G)
    # head h averages q in {3h, 3h+1, 3h+2} and r in {0, 1, 2}: 100k + 10 + 3h + 1
    for k in range(K):
        for h in range(2):
            assert m[k, h] == pytest.approx(100 * k + 10 + 3 * h + 1)


def test_selection_rules_on_worked_examples(golden):
    g = golden("calibration.json")
    for case in g["threshold"]:
        means = np.array(case["means"])
        got = oracle.select_windows(means, case["windows"], case["n_sinks"], case["ctx"],
                                    case["tau"])
        assert got == case["choice"], case["derivation"]
    for case in g["budget"]:
        got = oracle.budget_select(case["rates"], case["floors"], case["budget"])
        assert got == case["chosen"], case["derivation"]


# --------------------------------------------------------------------------
# cache formats p_KV (Eq. nominal-storage carries b^K, b^V; the stored value
# of an element is what attention sees)
# --------------------------------------------------------------------------
from oracle import kvformat as KF  # noqa: E402


def test_e4m3_table_follows_the_format_definition():
    T = KF.E4M3_TABLE
    assert T[0x00] == 0.0 and T[0x80] == 0.0 and np.signbit(T[0x80])
    assert T[0x01] == 2.0 ** -9             # smallest subnormal
    assert T[0x07] == 7 * 2.0 ** -9         # largest subnormal
    assert T[0x08] == 2.0 ** -6             # smallest normal
    assert T[0x38] == 1.0 and T[0x39] == 1.125 and T[0x40] == 2.0
    assert T[0x7D] == 416.0 and T[0x7E] == 448.0 and T[0xFE] == -448.0
    assert np.isnan(T[0x7F]) and np.isnan(T[0xFF])
    assert np.all(np.diff(T[:0x7F]) > 0)    # magnitudes strictly increase
    assert np.array_equal(T[0x80:0xFF], -T[0x00:0x7F])
    # an independent decoder: torch's float8_e4m3fn, all 256 codes
    t = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    nan = np.isnan(T)
    assert np.array_equal(np.isnan(t), nan)
    assert np.array_equal(t[~nan], T[~nan])


@pytest.mark.parametrize("x,s,code", [
    (1.0, 1.0, 0x38),
    (1.0625, 1.0, 0x38),          # tie 1.0 / 1.125: even code
    (1.1875, 1.0, 0x3A),          # tie 1.125 / 1.25: even code
    (2.0 ** -10, 1.0, 0x00),      # tie 0 / 2^-9: even code (zero)
    (3 * 2.0 ** -10, 1.0, 0x02),  # tie 2^-9 / 2^-8: even code
    (5 * 2.0 ** -10, 1.0, 0x02),  # tie 2 / 3 x 2^-9
    (2.0 ** -6 * (1 - 2.0 ** -20), 1.0, 0x08),   # rounds up to the smallest normal
    (240.0, 1.0, 0x77),
    (432.0, 1.0, 0x7E),           # tie 416 (odd) / 448 (even)
    (448.0, 1.0, 0x7E),
    (460.0, 1.0, 0x7E),           # saturates
    (1e30, 1.0, 0x7E),
    (float("inf"), 1.0, 0x7E),
    (float("-inf"), 1.0, 0xFE),
    (float("nan"), 1.0, 0x7F),
    (0.0, 1.0, 0x00),
    (-0.0, 1.0, 0x80),
    (-1e-30, 1.0, 0x80),          # rounds to zero, keeps the sign
    (1.0, 0.5, 0x40),             # 1 / 0.5 = 2
    (1.0, 3.0, 0x2B),             # fp32(1/3) = 1.333 x 2^-2 -> m = 3 (0.375 nearer than 0.25)
    (-300.0, 0.25, 0xFE),         # -1200 saturates
])
def test_e4m3_encode_worked_cases(x, s, code):
    assert int(KF.e4m3_encode(np.array([x]), s)[0]) == code


@pytest.mark.parametrize("s", [1.0, 0.0123, 3.7e-3, 17.5])
def test_e4m3_encode_matches_torch_on_every_bf16(s):
    """Below the overflow threshold the encoder is the IEEE-style conversion
    torch implements (round to nearest even); above it, it saturates."""
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    x = KF.bf16_values(bits)
    got = KF.e4m3_encode(x, s)
    with np.errstate(all="ignore"):
        y = (x.astype(np.float32) / np.float32(s)).astype(np.float32)
    sel = np.isfinite(y) & (np.abs(y) < 464)
    t = torch.from_numpy(y[sel]).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(got[sel], t)
    big = np.isfinite(y) & (np.abs(y) >= 464) | np.isinf(y)
    assert np.all((got[big] & 0x7F) == 0x7E)
    assert np.all((got[np.isnan(y)] & 0x7F) == 0x7F)
    # and every code decodes to within half a step of its input
    fin = np.isfinite(y) & (np.abs(y) <= 448)
    v = KF.e4m3_values(got[fin])
    a = np.abs(y[fin].astype(np.float64))
    step = np.where(a < 2.0 ** -6, 2.0 ** -9, 2.0 ** (np.floor(np.log2(np.maximum(a, 2.0 ** -6))) - 3))
    assert np.all(np.abs(v - y[fin]) <= step / 2)


@pytest.mark.parametrize("x,bits", [
    (1.0, 0x3C00), (1.0078125, 0x3C08), (65504.0, 0x7BFF), (65519.0, 0x7BFF),
    (65520.0, 0x7C00),            # tie 65504 (odd) / overflow: to infinity
    (2.0 ** -24, 0x0001), (2.0 ** -25, 0x0000), (3 * 2.0 ** -25, 0x0002),
    (-(2.0 ** -25), 0x8000), (2.0 ** -14, 0x0400),
])
def test_f16_encode_worked_cases(x, bits):
    assert int(KF.f16_encode(np.array([x]))[0]) == bits


def test_f16_is_exact_on_bf16_values_in_its_normal_range():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    x = KF.bf16_values(bits)
    sel = np.isfinite(x) & (np.abs(x) >= 2.0 ** -14) & (np.abs(x) <= 65504)
    assert np.array_equal(KF.values(KF.store(bits[sel], "f16"), "f16"), x[sel])


def test_attend_values_matches_the_c_oracle_on_bf16_values():
    r = np.random.default_rng(21)
    B, Hq, Hkv, d = 2, 6, 2, 32
    n = 90
    q = bf16(r.standard_normal((B, Hq, d)))
    k = [bf16(r.standard_normal((n, Hkv, d))) for _ in range(B)]
    v = [bf16(r.standard_normal((n, Hkv, d))) for _ in range(B)]
    t = np.array([89, 40])
    for S, wins in ((0, [0, 0]), (3, [7, 0]), (2, [1, 50])):
        ref = oracle.decode_layer(q, k, v, t, S, wins, 0.3)
        got = KF.attend_values(f64(q), [f64(x) for x in k], [f64(x) for x in v], t, S, wins, 0.3)
        assert np.max(np.abs(got - ref)) <= 1e-13 * np.max(np.abs(ref))


def test_attend_values_closed_forms():
    r = np.random.default_rng(22)
    d, n = 16, 40
    q = r.standard_normal((1, 2, d))
    kk = np.tile(r.standard_normal(d), (n, 1, 1))          # identical keys
    vv = r.standard_normal((n, 1, d))
    out = KF.attend_values(q, [kk], [vv], [n - 1], 3, [10], 0.7)
    pos = list(range(3)) + list(range(n - 10, n))
    assert np.allclose(out[0, 0], vv[pos, 0].mean(axis=0), rtol=0, atol=1e-14)
    assert np.allclose(out[0, 1], vv[pos, 0].mean(axis=0), rtol=0, atol=1e-14)
    one = KF.attend_values(q, [kk], [vv], [0], 0, [5], 0.7)  # a single retained token
    assert np.array_equal(one[0, 0], vv[0, 0])


def test_storage_accounting_per_format():
    """Eq. nominal-storage with b^K = b^V = 1 (fp8) is exactly half of the
    16-bit formats, unit by unit."""
    wins = np.array([2048, 0, 512])
    for ctx in (100, 4096, 131072):
        b16 = oracle.policy_bytes(ctx, 4, wins, 256, 256, 2.0, 2.0)
        b8 = oracle.policy_bytes(ctx, 4, wins, 256, 256, 1.0, 1.0)
        assert b8 * 2 == b16
        exp = sum(min(4 + w, ctx) if w else ctx for w in wins) * 256 * 2
        assert b8 == exp
