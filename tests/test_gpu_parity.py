"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Residency (which position each slot holds, and its bytes) must match
bit-exactly; attention outputs within max relative error 1e-2 per output row
(|o - ref|_inf / |ref|_inf), and additionally within 2e-4, which fp32
accumulation over bf16 inputs meets with a wide margin.
"""
import numpy as np
import pytest
import torch

import workloads as W
from hwkv_harness import Run, log, timed, up
from paper_2609_02029_amd import hwkv

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def mini(**kw):
    c = dict(name="mini", seed=11, n_layers=1, batch=1, n_q_heads=8, n_kv_heads=2,
             head_dim=64, n_sinks=4, level_windows=[256, 0], levels=[[0, 1]],
             prompt=[300], steps=4, max_ctx=400)
    c.update(kw)
    return c


# ---------------------------------------------------------------------------
# the 2048-token, d=64, GQA-4 workload in full: residency after prefill and
# after every append, every output of every step
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("fused", [False, True])
def test_pr1_workload(fused):
    cfg = W.CONFIGS["pr1"]
    log(f"pr1 fused={fused}")
    r = Run(cfg, fused=fused)
    r.prefill(0, 0)
    r.check_layer(0)
    worst = 0.0
    for st in range(cfg["steps"]):
        qa, out = r.step(0)
        worst = max(worst, r.check_out(0, qa, out, f"step {st}"))
        r.check_layer(0)
    log(f"pr1 fused={fused}: max rel err {worst:.3e}")
    r.free()


# ---------------------------------------------------------------------------
# lengths around every boundary: n < S, n = S + w, n = S + w + 1, one tile,
# one split (512 tokens), w >= n, S = 0, w = 1
# ---------------------------------------------------------------------------
EDGES = [
    (0, 1, 1), (0, 1, 5), (3, 5, 2), (3, 5, 7), (3, 5, 8), (3, 5, 9),
    (4, 60, 63), (4, 60, 64), (4, 60, 65), (4, 508, 511), (4, 508, 512),
    (4, 508, 513), (0, 600, 1025), (4, 3000, 100), (2, 1, 700), (4, 2000, 2500),
]


@pytest.mark.parametrize("S,w,P", EDGES)
def test_edge_lengths(S, w, P):
    log(f"edge S={S} w={w} P={P}")
    cfg = mini(n_sinks=S, level_windows=[w, 0], prompt=[P], max_ctx=P + 8)
    r = Run(cfg)
    r.prefill(0, 0)
    r.check_layer(0)
    for st in range(4):
        qa, out = r.step(0, fused=bool(st % 2))
        r.check_out(0, qa, out, f"S={S} w={w} P={P} step {st}")
        r.check_layer(0)
    r.free()


@pytest.mark.parametrize("D", [64, 128, 256])
@pytest.mark.parametrize("G", [1, 2, 4, 6, 8])
def test_head_dims_and_groups(D, G):
    log(f"dims D={D} G={G}")
    cfg = mini(head_dim=D, n_kv_heads=2, n_q_heads=2 * G, level_windows=[700, 0],
               prompt=[1500], max_ctx=1600, seed=12)
    r = Run(cfg)
    r.prefill(0, 0)
    for st in range(2):
        qa, out = r.step(0, fused=bool(st))
        r.check_out(0, qa, out, f"D={D} G={G} step {st}")
    r.check_layer(0)
    r.free()


def test_chunked_prefill_bit_exact():
    cfg = mini(head_dim=128, n_kv_heads=4, n_q_heads=8, n_sinks=3,
               level_windows=[5, 64, 300, 0], levels=[[0, 1, 2, 3]], prompt=[2000],
               max_ctx=2100, seed=13)
    for chunks in ([1, 7, 64, 65, 200, 513, 900], [3], list(range(1, 2000, 37)), [1999]):
        log(f"chunked {chunks[:5]}...")
        a = Run(cfg)
        a.prefill(0, 0, chunks=chunks)
        b = Run(cfg)
        b.prefill(0, 0)
        for h in range(4):
            ka, va, na = hwkv.cache_read_unit(a.cache, 0, h, 0)
            kb, vb, nb = hwkv.cache_read_unit(b.cache, 0, h, 0)
            assert na == nb
            assert np.array_equal(ka[:na], kb[:nb]) and np.array_equal(va[:na], vb[:nb])
        a.check_layer(0)
        a.free()
        b.free()


def test_batched_ragged():
    cfg = mini(batch=5, head_dim=256, n_kv_heads=4, n_q_heads=24,
               level_windows=[100, 600, 2000, 0], levels=[[0, 1, 2, 3], [3, 2, 0, 0]],
               n_layers=2, prompt=[1, 63, 700, 1500, 2049], max_ctx=2100, seed=14)
    r = Run(cfg)
    for l in range(2):
        for b in range(5):
            r.prefill(l, b)
        r.check_layer(l)
    for st in range(3):
        for l in range(2):
            qa, out = r.step(l, fused=bool((st + l) % 2))
            r.check_out(l, qa, out, f"layer {l} step {st}")
    for l in range(2):
        r.check_layer(l)
    r.free()


def test_more_items_than_one_launch():
    # 17 sequences x 4 kv heads = 68 items: two launches per call
    cfg = mini(batch=17, n_kv_heads=4, n_q_heads=16, level_windows=[30, 0],
               levels=[[0, 1, 1, 0]], prompt=[int(x) for x in range(40, 40 + 17 * 23, 23)],
               max_ctx=600, seed=15)
    r = Run(cfg)
    for b in range(17):
        r.prefill(0, b)
    for st in range(2):
        qa, out = r.step(0, fused=bool(st))
        r.check_out(0, qa, out, f"step {st}")
    r.check_layer(0)
    r.free()


def test_single_token_is_v0_exactly():
    cfg = mini(prompt=[1], max_ctx=16)
    for fused in (False, True):
        r = Run(cfg)
        qa = W.normal_bf16((1, 8, 64), 1, 0, W.Q, 0)
        kv = W.normal_bf16((1, 2, 64), 1, 0, W.K, 0)
        vv = W.normal_bf16((1, 2, 64), 1, 0, W.V, 0)
        out = torch.empty((1, 8, 64), dtype=torch.float32, device="cuda")
        if fused:
            hwkv.append_decode_attn(r.cache, 0, up(kv, "cuda"), up(vv, "cuda"), up(qa, "cuda"),
                                    0.125, out, r.ws)
        else:
            hwkv.prefill_write(r.cache, 0, 0, 0, up(kv, "cuda"), up(vv, "cuda"))
            hwkv.decode_attn(r.cache, 0, up(qa, "cuda"), 0.125, out, r.ws)
        torch.cuda.synchronize()
        v0 = W.bf16_bits_to_f32(vv[0])  # [2, 64]
        got = out.cpu().numpy()
        for qh in range(8):
            assert np.array_equal(got[0, qh], v0[qh // 4]), (fused, qh)
        r.free()


def test_deterministic():
    cfg = mini(prompt=[3000], max_ctx=3100, level_windows=[1000, 0], head_dim=256,
               n_q_heads=12, seed=16)
    outs = []
    for _ in range(2):
        r = Run(cfg, track=[])
        r.prefill(0, 0)
        o = []
        for _ in range(3):
            _, out = r.step(0)
            o.append(out.cpu().numpy())
        outs.append(np.stack(o))
        r.free()
    assert np.array_equal(outs[0], outs[1])


def test_capacity_errors_leave_state():
    cfg = mini(prompt=[64], max_ctx=64)
    r = Run(cfg)
    r.prefill(0, 0)
    kn = torch.zeros((1, 2, 64), dtype=torch.bfloat16, device="cuda")
    q = torch.zeros((1, 8, 64), dtype=torch.bfloat16, device="cuda")
    out = torch.zeros((1, 8, 64), dtype=torch.float32, device="cuda")
    with pytest.raises(hwkv.HwkvError) as e:
        hwkv.append(r.cache, 0, kn, kn)
    assert e.value.code == hwkv.ECAPACITY
    with pytest.raises(hwkv.HwkvError) as e:
        hwkv.append_decode_attn(r.cache, 0, kn, kn, q, 0.125, out, r.ws)
    assert e.value.code == hwkv.ECAPACITY
    with pytest.raises(hwkv.HwkvError) as e:
        hwkv.prefill_write(r.cache, 0, 0, 64, kn[0:1, :, :].reshape(1, 2, 64), kn[0:1].reshape(1, 2, 64))
    assert e.value.code == hwkv.ECAPACITY
    assert hwkv.cache_seq_len(r.cache, 0, 0) == 64
    r.check_layer(0)
    # a windowed-only layer keeps going past max_ctx
    r2 = Run(mini(prompt=[64], max_ctx=64, level_windows=[20, 20]))
    r2.prefill(0, 0)
    for st in range(3):
        qa, o = r2.step(0)
        r2.check_out(0, qa, o, f"stream step {st}")
    r2.check_layer(0)
    r.free()
    r2.free()


# ---------------------------------------------------------------------------
# the 32K workload (d=256, GQA 6, outlier channels), all 256 steps run,
# outputs checked at 32 seeded steps, residency after prefill and at the end
# ---------------------------------------------------------------------------
@pytest.mark.timeout(900)
def test_ctx32k_workload():
    """Residency of every unit after prefill and after every one of the 256
    steps; outputs at 34 seeded steps (the first and the last among them)."""
    cfg = W.CONFIGS["ctx32k"]
    r = Run(cfg)
    with timed("ctx32k prefill"):
        r.prefill(0, 0)
        r.check_layer(0)
    check = set(W.rng(cfg["seed"], 0, W.SAMPLE, 0).choice(cfg["steps"], size=32, replace=False).tolist())
    check |= {0, cfg["steps"] - 1}
    worst = 0.0
    with timed("ctx32k steps, residency of every unit after each"):
        for st in range(cfg["steps"]):
            qa, out = r.step(0)
            if st in check:
                worst = max(worst, r.check_out(0, qa, out, f"ctx32k step {st}"))
            r.check_layer(0)
    log(f"ctx32k: levels {r.levels} max rel err {worst:.3e}")
    r.free()


# ---------------------------------------------------------------------------
# the 112K, 16-layer workload at full size, in the launch configuration the
# benchmark times (fused append + decode per layer)
# ---------------------------------------------------------------------------
@pytest.mark.timeout(1200)
def test_ctx112k_workload_full_size():
    """Residency of all 64 units after prefill and after the last step;
    outputs of every layer and query head at steps 0, 1, 63, 126 and 127."""
    cfg = W.CONFIGS["ctx112k"]
    r = Run(cfg, device_gen=True)
    with timed("ctx112k prefill + residency of all 64 units"):
        for l in range(cfg["n_layers"]):
            r.prefill(l, 0)
            r.check_layer(l)
    sample = {0, 1, 63, 126, 127}
    worst = 0.0
    with timed("ctx112k 128 steps x 16 layers"):
        for st in range(cfg["steps"]):
            for l in range(cfg["n_layers"]):
                qa, out = r.step(l)
                if st in sample:
                    worst = max(worst, r.check_out(l, qa, out, f"ctx112k layer {l} step {st}"))
    with timed("ctx112k final residency"):
        for l in range(cfg["n_layers"]):
            r.check_layer(l)
    log(f"ctx112k: max rel err {worst:.3e}")
    r.free()


# ---------------------------------------------------------------------------
# batched serving: 16 ragged sequences (16K..64K), 8 layers, 64 steps
# ---------------------------------------------------------------------------
@pytest.mark.timeout(1200)
def test_batch16_workload_full_size():
    """Residency of every (sequence, unit) after prefill and at the end;
    outputs of every layer and sequence at the first and the last step."""
    cfg = W.CONFIGS["batch16"]
    r = Run(cfg, device_gen=True)
    log(f"batch16 prompts {r.prompts}")
    with timed("batch16 prefill"):
        for l in range(cfg["n_layers"]):
            for b in range(cfg["batch"]):
                r.prefill(l, b)
            r.check_layer(l)
    worst = 0.0
    with timed("batch16 64 steps x 8 layers"):
        for st in range(cfg["steps"]):
            for l in range(cfg["n_layers"]):
                qa, out = r.step(l)
                if st in (0, cfg["steps"] - 1):
                    worst = max(worst, r.check_out(l, qa, out, f"batch16 layer {l} step {st}"))
    with timed("batch16 final residency"):
        for l in range(cfg["n_layers"]):
            r.check_layer(l)
    log(f"batch16: max rel err {worst:.3e}")
    r.free()


# ---------------------------------------------------------------------------
# the largest documented capacity: one full unit of 4,194,240 rows at
# head_dim 256 (2,147,450,880 bytes of K or V, just under the 2^31 byte
# offsets the kernels use), filled to its last row
# ---------------------------------------------------------------------------
@pytest.mark.timeout(1200)
def test_largest_capacity():
    cap = 4194240
    assert (cap + 63) // 64 * 64 * 256 * 2 < 2 ** 31
    cfg = dict(name="maxcap", seed=19, n_layers=1, batch=1, n_q_heads=2, n_kv_heads=1,
               head_dim=256, n_sinks=0, level_windows=[0], levels=[[0]],
               prompt=[cap - 24], steps=24, max_ctx=cap)
    r = Run(cfg, device_gen=True)
    with timed("max capacity prefill"):
        r.prefill(0, 0, chunks=[1 << 20, 2 << 20, 3 << 20])
    worst = 0.0
    with timed("max capacity 24 steps"):
        for st in range(24):
            qa, out = r.step(0, fused=bool(st % 2))
            if st in (0, 23):
                worst = max(worst, r.check_out(0, qa, out, f"max capacity step {st}"))
    assert hwkv.cache_seq_len(r.cache, 0, 0) == cap
    with timed("max capacity residency"):
        r.check_layer(0)
    dev = torch.device("cuda:0")
    kn = torch.zeros((1, 1, 256), dtype=torch.bfloat16, device=dev)
    with pytest.raises(hwkv.HwkvError) as e:
        hwkv.append(r.cache, 0, kn, kn)
    assert e.value.code == hwkv.ECAPACITY
    log(f"max capacity: max rel err {worst:.3e}")
    r.free()
    # one row more does not fit the 32-bit offsets
    pol = hwkv.policy_set(1, 1, 2, 256, 0, [0], [[0]])
    with pytest.raises(hwkv.HwkvError):
        hwkv.cache_bytes(pol, 1, cap + 64)


# ---------------------------------------------------------------------------
# the read probe of the decode roofline: every pattern runs over a buffer of
# equal words (every fold is zero), and leaves the sink untouched
# ---------------------------------------------------------------------------
def test_read_probe_runs():
    import ctypes

    from paper_2609_02029_amd import build
    lib = ctypes.CDLL(build.PROBE_LIB)
    lib.hwkv_read_probe.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                    ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    dev = torch.device("cuda:0")
    buf = torch.full((64 << 20,), 7, dtype=torch.uint8, device=dev)
    sink = torch.zeros(1, dtype=torch.float32, device=dev)
    s = torch.cuda.current_stream().cuda_stream
    for pattern, wps in [(0, 2), (0, 4), (0, 8), (1, 2), (1, 4), (1, 8)]:
        assert lib.hwkv_read_probe(buf.data_ptr(), buf.numel(), pattern, wps, sink.data_ptr(), s) == 0
        # fewer tiles than workgroups
        assert lib.hwkv_read_probe(buf.data_ptr(), 3 << 16, pattern, wps, sink.data_ptr(), s) == 0
    torch.cuda.synchronize()
    assert float(sink.cpu()[0]) == 0.0

