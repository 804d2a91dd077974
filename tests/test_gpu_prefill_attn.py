"""GPU parity of prefill attention (hwkv_prefill_attn) against the fp64
masked-full-cache oracle.

Each chunk's queries attend over the cache as it stands before the chunk is
materialised plus the chunk's own K/V; the oracle evaluates every checked
query token over its retained set inside the full host history.  Outputs
must be within max relative error 1e-2 per row (|o - ref|_inf / |ref|_inf);
the cache must be left untouched by the attention call and, after the
chunk-by-chunk writes, hold bit-exactly the oracle's residency.

A tighter bound follows from the arithmetic.  Products q.k and the sums are
fp32 on exact bf16 inputs; the only coarse rounding is that of each softmax
weight p_s (at most 2^8 after the running shift) to bf16 before the value
product, a relative error of at most 2^-8 (8 significant bits), while the
normaliser sums the unrounded weights.  Hence, per channel i,
    |o_i - ref_i| = |sum_s (p~_s - p_s) v_si| / sum_s p_s <= 2^-8 max_s |v_si|
over the row's retained keys s, plus fp32 slack (taken as 2e-5 max |v_si|).
"""
import numpy as np
import pytest
import torch

import workloads as W
from hwkv_harness import REL_TOL, Run, log, rel_err, retained_absmax, timed
from paper_2609_02029_amd import hwkv

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def mini(**kw):
    c = dict(name="mini-prefill", seed=21, n_layers=1, batch=1, n_q_heads=8, n_kv_heads=2,
             head_dim=64, n_sinks=4, level_windows=[100, 0], levels=[[0, 1]],
             prompt=[700], steps=0, max_ctx=800)
    c.update(kw)
    return c


P_ROUND = 2.0 ** -8 + 2e-5   # bf16 rounding of the weights, plus fp32 slack


def vmax_bound(r, layer, b, rows):
    """[rows, Hkv, D]: max |v| per channel over each row's retained keys
    (its head's window), at every size."""
    av = np.abs(W.bf16_bits_to_f32(r.vh[layer][b][: int(rows[-1]) + 1]))   # [n, Hkv, D]
    out = np.empty((len(rows), r.Hkv, r.D), dtype=np.float64)
    for i, t in enumerate(rows):
        for h in range(r.Hkv):
            out[i, h] = retained_absmax(av[:, h], int(t), r.windows[layer][h], r.S)
    return out


def check_rows(r, layer, b, rows, q_rows, out, what):
    """Compares out[rows] with the oracle (``q_rows``: the queries of those
    rows, bf16 bits): the relative-error bar and the weight-rounding bound.
    Returns (max relative error, max error / bound)."""
    torch.cuda.synchronize()
    rows = np.asarray(rows, dtype=np.int64)
    assert np.all(np.diff(rows) > 0)
    ref = r.oracle_rows(layer, b, rows, q_rows)
    got = out[torch.from_numpy(rows).to(out.device)].cpu().numpy()
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    e = rel_err(got.reshape(-1, r.D), ref.reshape(-1, r.D))
    assert e <= REL_TOL, f"{what}: max rel err {e} > {REL_TOL}"
    vb = np.repeat(vmax_bound(r, layer, b, rows), r.G, axis=1)     # [rows, Hq, D]
    ratio = float((np.abs(got - ref) / (P_ROUND * vb)).max())
    assert ratio <= 1.0, f"{what}: error {ratio:.3f} x the weight-rounding bound"
    return e, ratio


@pytest.mark.parametrize("D", [64, 128, 256])
@pytest.mark.parametrize("G", [1, 2, 4, 6, 8])
def test_dims_and_groups_all_rows(D, G):
    log(f"prefill attn D={D} G={G}")
    cfg = mini(head_dim=D, n_q_heads=2 * G, level_windows=[150, 0], seed=22)
    r = Run(cfg)
    q, qh, out = r.prefill_with_attn(0, 0, chunks=[1, 100, 333])
    rows = np.arange(700)
    e, ratio = check_rows(r, 0, 0, rows, qh[rows], out, f"D={D} G={G}")
    r.check_layer(0)
    log(f"D={D} G={G}: max rel err {e:.3e}, {ratio:.3f} of the rounding bound")
    r.free()


# sinks, windows (below, at and above the 32-key tile, w = 1), prompt and
# chunk cuts (single tokens, ragged, a chunk ending at S + w)
EDGES = [
    (0, 1, 90, [1, 2, 50]),
    (3, 1, 90, [5]),
    (4, 5, 200, [1, 9, 10, 11, 77]),
    (4, 31, 300, [35, 36, 64]),
    (4, 32, 300, [36, 37, 100]),
    (4, 33, 300, [20, 37, 38, 199]),
    (2, 64, 500, [66, 67, 130, 131]),
    (4, 200, 700, [203, 204, 205, 600]),
    (4, 650, 700, [3, 4, 654, 655]),
    (0, 100, 700, [100, 101, 640]),
    (4, 96, 100, []),
]


@pytest.mark.parametrize("S,w,P,cuts", EDGES)
def test_window_edges_all_rows(S, w, P, cuts):
    log(f"prefill attn edge S={S} w={w} P={P} cuts={cuts}")
    cfg = mini(n_sinks=S, level_windows=[w, 0], prompt=[P], max_ctx=P + 8, seed=23)
    r = Run(cfg)
    q, qh, out = r.prefill_with_attn(0, 0, chunks=cuts, check_untouched=True)
    rows = np.arange(P)
    e, ratio = check_rows(r, 0, 0, rows, qh[rows], out, f"S={S} w={w} P={P}")
    r.check_layer(0)
    log(f"edge S={S} w={w} P={P}: max rel err {e:.3e}, {ratio:.3f} of the rounding bound")
    r.free()


def test_first_token_is_its_value_exactly():
    """Token 0 attends only to itself: out = v_0 (exact after widening)."""
    cfg = mini(head_dim=128, n_q_heads=12, n_kv_heads=2, level_windows=[16, 0], prompt=[40],
               max_ctx=64, seed=24)
    r = Run(cfg)
    q, qh, out = r.prefill_with_attn(0, 0, chunks=[1, 2])
    torch.cuda.synchronize()
    v0 = W.bf16_bits_to_f32(r.vh[0][0][0])   # [Hkv, D]
    got = out[0].cpu().numpy()                 # [Hq, D]
    for qh_i in range(r.Hq):
        assert np.array_equal(got[qh_i], v0[qh_i // r.G]), qh_i
    r.free()


def test_batched_layers_and_chunkings():
    """Several sequences and layers (region offsets), prefilled with
    different chunkings; every row checked."""
    cfg = mini(batch=3, n_layers=2, head_dim=256, n_kv_heads=4, n_q_heads=24,
               level_windows=[40, 300, 1000, 0], levels=[[0, 1, 2, 3], [3, 0, 2, 1]],
               prompt=[257, 1200, 900], max_ctx=1300, seed=25)
    r = Run(cfg)
    chunkings = {0: [64], 1: [1, 300, 301, 999], 2: []}
    for layer in range(2):
        for b in range(3):
            q, qh, out = r.prefill_with_attn(layer, b, chunks=chunkings[b])
            rows = np.arange(r.prompts[b])
            e, ratio = check_rows(r, layer, b, rows, qh[rows], out, f"layer {layer} seq {b}")
            log(f"layer {layer} seq {b}: max rel err {e:.3e}, {ratio:.3f} of the bound")
        r.check_layer(layer)
    r.free()


def test_every_chunking_meets_the_bound():
    """Chunk boundaries move the key tiles (and so the fp32 summation
    order) but every chunking stays within the same bounds of the oracle."""
    cfg = mini(head_dim=128, n_kv_heads=2, n_q_heads=12, level_windows=[333, 0],
               prompt=[1500], max_ctx=1600, seed=26)
    for cuts in ([], [700], list(range(97, 1500, 97))):
        r = Run(cfg)
        q, qh, out = r.prefill_with_attn(0, 0, chunks=cuts)
        rows = np.arange(1500)
        e, ratio = check_rows(r, 0, 0, rows, qh[rows], out, f"cuts {cuts[:3]}")
        log(f"cuts {cuts[:3]}: max rel err {e:.3e}, {ratio:.3f} of the bound")
        r.free()


def test_prefill128k_workload_sampled_rows():
    """The long-prefill workload in full: 128K tokens in 8K chunks, windows
    {2048, 8192, 32768, full} on kv heads 0..3, attention then write per
    chunk; 512 sampled rows against the oracle, final residency bit-exact."""
    cfg = W.CONFIGS["prefill128k"]
    N, C = cfg["prompt"][0], cfg["chunk"]
    r = Run(cfg, device_gen=True)
    with timed("prefill128k attn+write"):
        q, _, out = r.prefill_with_attn(0, 0, chunks=list(range(C, N, C)))
        torch.cuda.synchronize()
    rows = W.prefill_sample_rows(cfg)
    assert len(rows) == 512
    q_rows = q[torch.tensor(rows, device=q.device)].contiguous().view(torch.int16).cpu() \
        .numpy().view(np.uint16)
    with timed("oracle 512 rows"):
        e, ratio = check_rows(r, 0, 0, rows, q_rows, out, "prefill128k")
    log(f"prefill128k: max rel err {e:.3e} over {len(rows)} rows, {ratio:.3f} of the bound")
    with timed("residency"):
        r.check_layer(0)
    r.free()
