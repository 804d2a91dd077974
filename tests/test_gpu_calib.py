"""GPU parity of the calibration replay (hwkv_calib_replay) and the
selection rules against the fp64 oracle.

* candidate outputs o^(w): the windowed attention of every sampled row, per
  channel within the bf16 weight-rounding bound (2^-8 + 2e-5) max |v| over
  the retained keys, as for prefill attention (same kernel);
* scores: the score kernel must return the stabilised cosine of the outputs
  it was given, to fp32 dot-product accuracy ((2 D + 8) 2^-24); against the
  oracle's own scores, within the bound the measured output deviations
  imply, 2 (|du| / |u| + |dv| / |v|) plus that accuracy;
* means: the group averages of the GPU scores within n 2^-24 (n = rows x G);
* selection: on the same means, the library's choice equals the oracle's.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from hwkv_harness import log, retained_absmax, up
from paper_2609_02029_amd import hwkv

pytestmark = pytest.mark.gpu

P_ROUND = 2.0 ** -8 + 2e-5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def replay(k, v, q, rows, windows, S, scale, ref_full=None, dev="cuda:0", kv_format="bf16",
           k_scale=None, v_scale=None):
    """Runs hwkv_calib_replay (hwkv_calib_replay_format for another format)
    on device tensors; returns host arrays."""
    R, Hq, D = q.shape
    Hkv = k.shape[1]
    K = len(windows)
    outs = torch.full((K + 1, R, Hq, D), float("nan"), dtype=torch.float32, device=dev)
    scores = torch.full((max(K, 1), R, Hq), float("nan"), dtype=torch.float32, device=dev)[:K]
    means = torch.full((max(K, 1), Hkv), float("nan"), dtype=torch.float32, device=dev)[:K]
    ws = torch.zeros(hwkv.calib_workspace_bytes(Hq, D, S, k.shape[0], R, n_kv_heads=Hkv,
                                                kv_format=kv_format),
                     dtype=torch.uint8, device=dev)
    check = None
    if ref_full is not None:
        check = torch.full((R, Hq), float("nan"), dtype=torch.float32, device=dev)
    hwkv.calib_replay(k, v, rows, q, windows, S, scale, outs, scores.contiguous(),
                      means.contiguous(), ws, ref_full=ref_full, check=check,
                      kv_format=kv_format, k_scale=k_scale, v_scale=v_scale)
    torch.cuda.synchronize()
    res = dict(outs=outs.cpu().numpy().astype(np.float64),
               scores=scores.cpu().numpy().astype(np.float64),
               means=means.cpu().numpy().astype(np.float64))
    if check is not None:
        res["check"] = check.cpu().numpy().astype(np.float64)
    return res


def vmax_retained(vh, rows, windows, S):
    """[K + 1, R, Hkv, D]: max |v| per channel over each row's retained keys,
    for every candidate window and the full window last."""
    av = np.abs(W.bf16_bits_to_f32(vh))
    out = np.empty((len(windows) + 1, len(rows), av.shape[1], av.shape[2]))
    for ki, w in enumerate(list(windows) + [0]):
        for i, t in enumerate(rows):
            out[ki, i] = retained_absmax(av, int(t), w, S)
    return out


def check_all(res, ref_outs, kh, vh, rows, windows, S, G, what, vmax=None):
    K = len(windows)
    outs = res["outs"]
    assert np.all(np.isfinite(outs)), f"{what}: non-finite output"
    # candidate outputs
    if vmax is None:
        vmax = vmax_retained(vh, rows, windows, S)
    vb = np.repeat(vmax, G, axis=2)
    ratio = float((np.abs(outs - ref_outs) / (P_ROUND * vb)).max())
    assert ratio <= 1.0, f"{what}: outputs {ratio:.3f} x the rounding bound"
    D = outs.shape[-1]
    tol = (2 * D + 8) * 2.0 ** -24
    # scores: the cosine of the given outputs
    for k in range(K):
        for r in range(outs.shape[1]):
            for q in range(outs.shape[2]):
                c = oracle.cos_eval(outs[k, r, q], outs[K, r, q])
                assert abs(res["scores"][k, r, q] - c) <= tol, (what, k, r, q)
    # scores against the oracle's, within the deviation-implied bound
    ref_sc = oracle.replay_scores(ref_outs)
    du = np.linalg.norm(outs - ref_outs, axis=-1) / np.maximum(
        np.linalg.norm(ref_outs, axis=-1), 1e-30)
    bound = 2.0 * (du[:K] + du[K][None]) + tol
    err = np.abs(res["scores"] - ref_sc)
    assert np.all(err <= bound), f"{what}: score error {float(err.max())}"
    # means of the GPU scores
    n = outs.shape[1] * G
    m_ref = oracle.head_means(res["scores"], G)
    assert np.all(np.abs(res["means"] - m_ref) <= n * 2.0 ** -24), what
    # selection on identical means
    for tau in (0.9, 0.99, 0.995, 0.999):
        got, _ = hwkv.calib_select(res["means"], windows, S, int(kh.shape[0]), tau)
        assert got == oracle.select_windows(res["means"], windows, S, int(kh.shape[0]), tau)
    return ratio, float(err.max())


def small_case(seed, N, Hkv, G, D, windows, S, extra_rows=32):
    r = np.random.default_rng(seed)
    kh = W.normal_bf16((N, Hkv, D), seed, 0, W.K, 0)
    vh = W.normal_bf16((N, Hkv, D), seed, 0, W.V, 0)
    edge = {0, 1, S - 1, S, N - 1}
    for w in windows:
        edge |= {S + w - 1, S + w, S + w + 1, w - 1, w}
    edge = {x for x in edge if 0 <= x < N}
    rest = np.setdiff1d(np.arange(N), sorted(edge))
    rows = sorted(edge | {int(x) for x in r.choice(rest, size=extra_rows, replace=False)})
    qh = W.normal_bf16((len(rows), Hkv * G, D), seed, 0, W.Q_PROMPT, 7)
    return kh, vh, qh, rows


@pytest.mark.parametrize("D,G", [(64, 4), (128, 1), (128, 8), (256, 6)])
def test_replay_small(D, G):
    S, windows = 4, [16, 64, 200]
    kh, vh, qh, rows = small_case(31, 600, 2, G, D, windows, S)
    scale = 1.0 / math.sqrt(D)
    res = replay(up(kh, "cuda:0"), up(vh, "cuda:0"), up(qh, "cuda:0"), rows, windows, S, scale)
    ref = oracle.replay_outputs(qh, kh, vh, rows, S, list(windows) + [0], scale)
    ratio, serr = check_all(res, ref, kh, vh, rows, windows, S, G, f"D={D} G={G}")
    log(f"replay D={D} G={G}: {len(rows)} rows, outputs {ratio:.3f} of the bound, "
        f"max score error {serr:.2e}")


@pytest.mark.parametrize("D,G", [(128, 4), (256, 6)])
def test_replay_split_keys(D, G):
    """A history long enough that its keys are split over several workgroups
    and the candidates merged from the splits' and the edges' partials."""
    S, windows = 4, [100, 5000]
    kh, vh, qh, rows = small_case(34, 9000, 2, G, D, windows, S, extra_rows=24)
    scale = 1.0 / math.sqrt(D)
    res = replay(up(kh, "cuda:0"), up(vh, "cuda:0"), up(qh, "cuda:0"), rows, windows, S, scale)
    ref = oracle.replay_outputs(qh, kh, vh, rows, S, list(windows) + [0], scale, n_threads=16)
    ratio, serr = check_all(res, ref, kh, vh, rows, windows, S, G, f"split D={D} G={G}")
    log(f"replay split D={D} G={G}: outputs {ratio:.3f} of the bound, score error {serr:.2e}")


def test_replay_edges_and_full_check():
    """Sinks 0 and 3, a window of 1, windows beyond the history, a row at
    position 0; the full-window check against the oracle's full output."""
    for S, windows in ((0, [1, 33, 5000]), (3, [2, 31, 32, 100])):
        kh, vh, qh, rows = small_case(32, 300, 2, 4, 128, windows, S, extra_rows=16)
        rows = sorted(set(rows) | {0})
        qh = W.normal_bf16((len(rows), 8, 128), 32, 0, W.Q_PROMPT, 8)
        scale = 1.0 / math.sqrt(128)
        ref = oracle.replay_outputs(qh, kh, vh, rows, S, list(windows) + [0], scale)
        ref_full = torch.from_numpy(ref[-1].astype(np.float32)).to("cuda:0")
        res = replay(up(kh, "cuda:0"), up(vh, "cuda:0"), up(qh, "cuda:0"), rows, windows, S,
                     scale, ref_full=ref_full)
        check_all(res, ref, kh, vh, rows, windows, S, 4, f"S={S}")
        assert np.all(res["check"] >= 0.99)
        # the row at position 0 sees one key under every candidate: score one
        assert np.all(np.abs(res["scores"][:, 0] - 1.0) <= 1e-6)
        # windows reaching back past the history equal the full candidate
        for k, w in enumerate(windows):
            covered = [i for i, t in enumerate(rows) if S + w >= t + 1]
            assert np.array_equal(res["outs"][k, covered], res["outs"][-1, covered])


def _split_keys(N, R, G, Hkv):
    """Keys per split of the one-pass replay for this shape, by the library's
    rule: about one workgroup per CU over the column blocks, at most the
    workspace's split count (128 tiles each), at least 8 tiles per split."""
    n_cus = torch.cuda.get_device_properties(0).multi_processor_count
    nb = -(-R * G // 256)
    tiles = -(-N // 32)
    ws_splits = -(-tiles // 128)
    want = min(ws_splits, max(1, n_cus // (nb * Hkv)))
    max_tiles = (N - 1) // 32 + 1
    tps = max(8, -(-max_tiles // want), -(-max_tiles // ws_splits))
    return 32 * tps, -(-max_tiles // tps)


def test_replay_one_pass_boundaries():
    """The one-pass replay's edges: window edges exactly on, just below and
    just above split boundaries and tile boundaries, several edges in one
    tile, 40 sinks over two tiles, windows at and past the history."""
    N, Hkv, G, D, S = 20000, 1, 4, 64, 40
    windows = [1, 2, 31, 32, 33, 100, 4095, 19999, 25000]
    R = 192
    T, n_splits = _split_keys(N, R, G, Hkv)
    assert n_splits >= 3, (T, n_splits)
    want = {0, 1, S - 1, S, S + 1, 63, 64, N - 1}
    for w in (1, 33, 100, 4095):
        for j in range(1, n_splits):
            for d in (-33, -1, 0, 1, 31, 32):
                want.add(j * T + d + w - 1)          # edge t + 1 - w = j T + d
        want |= {S + w - 2, S + w - 1, S + w}      # edges around the sinks
    want = sorted(x for x in want if 0 <= x < N)
    r = np.random.default_rng(41)
    rest = np.setdiff1d(np.arange(N), want)
    assert len(want) <= R
    rows = sorted(set(want) | {int(x) for x in r.choice(rest, size=R - len(want), replace=False)})
    kh = W.normal_bf16((N, Hkv, D), 41, 0, W.K, 0)
    vh = W.normal_bf16((N, Hkv, D), 41, 0, W.V, 0)
    qh = W.normal_bf16((R, Hkv * G, D), 41, 0, W.Q_PROMPT, 7)
    scale = 1.0 / math.sqrt(D)
    res = replay(up(kh, "cuda:0"), up(vh, "cuda:0"), up(qh, "cuda:0"), rows, windows, S, scale)
    ref = oracle.replay_outputs(qh, kh, vh, rows, S, list(windows) + [0], scale, n_threads=16)
    ratio, serr = check_all(res, ref, kh, vh, rows, windows, S, G, "one-pass boundaries")
    # windows reaching back past the history equal the full candidate
    for k, w in enumerate(windows):
        covered = [i for i, t in enumerate(rows) if S + w >= t + 1]
        assert np.array_equal(res["outs"][k, covered], res["outs"][-1, covered])
    log(f"one-pass boundaries: {n_splits} splits of {T} keys, {R} rows, outputs "
        f"{ratio:.3f} of the bound, score error {serr:.2e}")


def test_replay_64_windows():
    """The most candidate windows the replay takes (64), at head_dim 64,
    without sinks, over a split history."""
    N, Hkv, G, D, S = 9000, 2, 2, 64, 0
    windows = list(range(1, 33)) + [40 + 37 * i for i in range(24)] + [5000, 8998, 8999, 9000,
                                                                       9001, 12000, 20000, 40000]
    assert len(windows) == 64 and all(b > a for a, b in zip(windows, windows[1:]))
    kh, vh, qh, rows = small_case(43, N, Hkv, G, D, [1, 32, 100, 5000], S, extra_rows=24)
    scale = 1.0 / math.sqrt(D)
    res = replay(up(kh, "cuda:0"), up(vh, "cuda:0"), up(qh, "cuda:0"), rows, windows, S, scale)
    ref = oracle.replay_outputs(qh, kh, vh, rows, S, list(windows) + [0], scale, n_threads=16)
    ratio, serr = check_all(res, ref, kh, vh, rows, windows, S, G, "64 windows")
    log(f"64 windows: {len(rows)} rows, outputs {ratio:.3f} of the bound, score error {serr:.2e}")


def test_replay_full_only_and_single_rows():
    """No finite window (the full candidate alone), and one sampled row at
    the first, a middle and the last position, with and without sinks."""
    N, Hkv, G, D = 5000, 2, 4, 128
    kh = W.normal_bf16((N, Hkv, D), 45, 0, W.K, 0)
    vh = W.normal_bf16((N, Hkv, D), 45, 0, W.V, 0)
    scale = 1.0 / math.sqrt(D)
    for S in (0, 4):
        rows = [3, 777, 2048, 4999]
        qh = W.normal_bf16((len(rows), Hkv * G, D), 45, S, W.Q_PROMPT, 0)
        res = replay(up(kh, "cuda:0"), up(vh, "cuda:0"), up(qh, "cuda:0"), rows, [], S, scale)
        ref = oracle.replay_outputs(qh, kh, vh, rows, S, [0], scale, n_threads=16)
        vb = np.repeat(vmax_retained(vh, rows, [], S), G, axis=2)
        ratio = float((np.abs(res["outs"] - ref) / (P_ROUND * vb)).max())
        assert np.all(np.isfinite(res["outs"])) and ratio <= 1.0, (S, ratio)
        for t in (0, 2500, N - 1):
            q1 = W.normal_bf16((1, Hkv * G, D), 46, t, W.Q_PROMPT, 0)
            res = replay(up(kh, "cuda:0"), up(vh, "cuda:0"), up(q1, "cuda:0"), [t], [1, 64, 3000],
                         S, scale)
            ref = oracle.replay_outputs(q1, kh, vh, [t], S, [1, 64, 3000, 0], scale)
            check_all(res, ref, kh, vh, [t], [1, 64, 3000], S, G, f"one row at {t}, S={S}")


def test_replay_zero_values_score_one():
    """V = 0 makes every output the zero vector: stabilised cosine 1."""
    kh = W.normal_bf16((100, 1, 64), 33, 0, W.K, 0)
    vh = np.zeros((100, 1, 64), dtype=np.uint16)
    qh = W.normal_bf16((5, 2, 64), 33, 0, W.Q_PROMPT, 0)
    res = replay(up(kh, "cuda:0"), up(vh, "cuda:0"), up(qh, "cuda:0"), [3, 10, 50, 60, 99],
                 [8, 32], 2, 0.125)
    assert np.all(res["outs"] == 0.0)
    assert np.all(res["scores"] == 1.0) and np.all(res["means"] == 1.0)


def test_calib128k_workload():
    """The calibration workload in full: a 128K trace, 256 rows from the final
    quarter; outputs checked on 24 of the rows, scores, means and selection
    on all of them."""
    cfg = W.CONFIGS["calib128k"]
    N, Hq, Hkv, D, S = cfg["prompt"][0], cfg["n_q_heads"], cfg["n_kv_heads"], cfg["head_dim"], \
        cfg["n_sinks"]
    G = Hq // Hkv
    windows = [w for w in cfg["level_windows"] if w]
    rows = W.calib_rows(cfg)
    dev = "cuda:0"
    k = W.normal_bf16_device((N, Hkv, D), cfg["seed"], 0, W.K, 0, device=dev)
    v = W.normal_bf16_device((N, Hkv, D), cfg["seed"], 0, W.V, 0, device=dev)
    q = W.normal_bf16_device((len(rows), Hq, D), cfg["seed"], 0, W.Q_PROMPT, 0, device=dev)
    scale = 1.0 / math.sqrt(D)
    res = replay(k, v, q, rows, windows, S, scale)
    bits = lambda t: t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    kh, vh, qh = bits(k), bits(v), bits(q)
    pick = list(range(0, len(rows), len(rows) // 24))[:24]
    sub_rows = [rows[i] for i in pick]
    ref = oracle.replay_outputs(qh[pick], kh, vh, sub_rows, S, list(windows) + [0], scale,
                                n_threads=16)
    outs = res["outs"][:, pick]
    vb = np.repeat(vmax_retained(vh, sub_rows, windows, S), G, axis=2)
    ratio = float((np.abs(outs - ref) / (P_ROUND * vb)).max())
    assert ratio <= 1.0
    tol = (2 * D + 8) * 2.0 ** -24
    for kk in range(len(windows)):
        for r in range(0, len(rows), 7):
            for qq in range(Hq):
                c = oracle.cos_eval(res["outs"][kk, r, qq], res["outs"][-1, r, qq])
                assert abs(res["scores"][kk, r, qq] - c) <= tol
    m_ref = oracle.head_means(res["scores"], G)
    assert np.all(np.abs(res["means"] - m_ref) <= len(rows) * G * 2.0 ** -24)
    for tau in (0.99, 0.995, 0.999):
        got, _ = hwkv.calib_select(res["means"], windows, S, N, tau)
        assert got == oracle.select_windows(res["means"], windows, S, N, tau)
    log(f"calib128k: outputs {ratio:.3f} of the (retained-max) bound; means {res['means'].round(4)}")


# ---------------------------------------------------------------------------
# the replay under an fp8 cache format: every candidate, the full one
# included, over the trace as an fp8 cache stores it
# ---------------------------------------------------------------------------
def _fp8_values(x_bits, scales):
    from oracle import kvformat as KF
    return np.stack([KF.values(KF.store(x_bits[:, h], "fp8", scales[h]), "fp8", scales[h])
                     for h in range(x_bits.shape[1])], axis=1)


def _vmax_values(vals, rows, windows, S):
    av = np.abs(vals)
    pos = np.arange(av.shape[0])
    out = np.empty((len(windows) + 1, len(rows), av.shape[1], av.shape[2]))
    for ki, w in enumerate(list(windows) + [0]):
        for i, t in enumerate(rows):
            keep = pos <= t
            if w:
                keep &= (pos < S) | (pos >= t + 1 - w)
            out[ki, i] = av[keep].max(axis=0)
    return out


@pytest.mark.parametrize("N,windows,D,G", [(600, [16, 64, 200], 64, 4),
                                           (600, [16, 64, 200], 256, 6),
                                           (9000, [100, 5000], 128, 4)])
def test_replay_fp8(N, windows, D, G):
    from oracle import kvformat as KF
    S = 4
    kh, vh, qh, rows = small_case(37, N, 2, G, D, windows, S, extra_rows=24)
    ks = np.array([0.013, 0.021], dtype=np.float32)
    vs = np.array([0.009, 0.017], dtype=np.float32)
    scale = 1.0 / math.sqrt(D)
    res = replay(up(kh, "cuda:0"), up(vh, "cuda:0"), up(qh, "cuda:0"), rows, windows, S, scale,
                 kv_format="fp8", k_scale=ks, v_scale=vs)
    kv, vv = _fp8_values(kh, ks), _fp8_values(vh, vs)
    ref = KF.replay_outputs_values(KF.bf16_values(qh), kv, vv, rows, S, list(windows) + [0],
                                   scale)
    ratio, serr = check_all(res, ref, kh, vh, rows, windows, S, G, f"fp8 N={N} D={D} G={G}",
                            vmax=_vmax_values(vv, rows, windows, S))
    log(f"replay fp8 N={N} D={D} G={G}: outputs {ratio:.3f} of the bound, score error {serr:.2e}")


def test_replay_format_errors():
    dev = "cuda:0"
    kh = up(W.normal_bf16((64, 1, 64), 38, 0, W.K, 0), dev)
    qh = up(W.normal_bf16((2, 2, 64), 38, 0, W.Q_PROMPT, 0), dev)
    outs = torch.zeros((2, 2, 2, 64), dtype=torch.float32, device=dev)
    sc = torch.zeros((1, 2, 2), dtype=torch.float32, device=dev)
    mn = torch.zeros((1, 1), dtype=torch.float32, device=dev)
    ws = torch.zeros(1 << 22, dtype=torch.uint8, device=dev)
    for kw in (dict(kv_format="f16"), dict(kv_format="bf16", k_scale=0.5),
               dict(kv_format="fp8", k_scale=0.0), dict(kv_format="fp8", v_scale=float("inf"))):
        with pytest.raises(hwkv.HwkvError) as e:
            hwkv.calib_replay(kh, kh, [10, 20], qh, [8], 0, 0.125, outs, sc, mn, ws, **kw)
        assert e.value.code == hwkv.EINVAL, kw
    need = hwkv.calib_workspace_bytes(2, 64, 0, 64, 2, n_kv_heads=1, kv_format="fp8")
    assert need > hwkv.calib_workspace_bytes(2, 64, 0, 64, 2)
    with pytest.raises(hwkv.HwkvError):
        hwkv.calib_replay(kh, kh, [10, 20], qh, [8], 0, 0.125, outs, sc, mn, ws[: need - 1],
                          kv_format="fp8")


def test_replay_back_to_back_row_staging():
    """Two replays enqueued on one stream without a wait between them, the
    second with more rows than the library's initial row staging buffer (so
    the buffer grows while the first call's copy may still be queued): each
    equals the same replay run on its own."""
    S, windows, D, G, Hkv, N = 4, [16, 64, 200], 64, 2, 1, 1500
    kh = W.normal_bf16((N, Hkv, D), 41, 0, W.K, 0)
    vh = W.normal_bf16((N, Hkv, D), 41, 0, W.V, 0)
    rows_a = sorted({int(x) for x in np.random.default_rng(5).choice(N, size=40, replace=False)})
    rows_b = list(range(N - 1100, N))
    qa = W.normal_bf16((len(rows_a), Hkv * G, D), 41, 0, W.Q_PROMPT, 3)
    qb = W.normal_bf16((len(rows_b), Hkv * G, D), 41, 0, W.Q_PROMPT, 4)
    scale = 1.0 / math.sqrt(D)
    k, v = up(kh, "cuda:0"), up(vh, "cuda:0")
    alone_a = replay(k, v, up(qa, "cuda:0"), rows_a, windows, S, scale)
    alone_b = replay(k, v, up(qb, "cuda:0"), rows_b, windows, S, scale)
    K = len(windows)
    bufs = []
    for rows, q in ((rows_a, qa), (rows_b, qb)):
        R = len(rows)
        outs = torch.full((K + 1, R, G * Hkv, D), float("nan"), dtype=torch.float32, device="cuda:0")
        scores = torch.full((K, R, G * Hkv), float("nan"), dtype=torch.float32, device="cuda:0")
        means = torch.full((K, Hkv), float("nan"), dtype=torch.float32, device="cuda:0")
        ws = torch.zeros(hwkv.calib_workspace_bytes(G * Hkv, D, S, N, R, n_kv_heads=Hkv),
                         dtype=torch.uint8, device="cuda:0")
        bufs.append((rows, up(q, "cuda:0"), outs, scores, means, ws))
    torch.cuda.synchronize()
    for rows, q, outs, scores, means, ws in bufs:        # no wait between the two
        hwkv.calib_replay(k, v, rows, q, windows, S, scale, outs, scores, means, ws)
    torch.cuda.synchronize()
    for (rows, q, outs, scores, means, ws), alone in zip(bufs, (alone_a, alone_b)):
        assert np.array_equal(outs.cpu().numpy().astype(np.float64), alone["outs"])
        assert np.array_equal(scores.cpu().numpy().astype(np.float64), alone["scores"])
        assert np.array_equal(means.cpu().numpy().astype(np.float64), alone["means"])
    log(f"back-to-back replays of {len(rows_a)} and {len(rows_b)} rows equal the lone ones")
