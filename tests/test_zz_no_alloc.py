"""The allocation-free decode entry point against the workspace one.

hwkv_append_decode_attn_noalloc runs the kernels of hwkv_append_decode_attn
with the split partials in the library's static scratch instead of a caller
workspace.  On identical caches and inputs the two calls must give the same
outputs and leave the same residency, bit for bit; two calls in a row, the
second on a smaller problem (fewer partials than the first left behind).
"""
import math

import numpy as np
import pytest
import torch

from paper_2609_02029_amd import hwkv

pytestmark = pytest.mark.gpu


def _pair(L, B, Hq, Hkv, D, S, windows, levels, prompt, max_ctx, seed, dev):
    """Two caches of one policy holding the same seeded prompt."""
    pol = hwkv.policy_set(L, Hkv, Hq, D, S, windows, levels)
    caches = [hwkv.cache_alloc(pol, B, max_ctx) for _ in range(2)]
    g = torch.Generator(device="cpu").manual_seed(seed)
    for l in range(L):
        for b in range(B):
            k = torch.randn((prompt, Hkv, D), generator=g).to(torch.bfloat16).to(dev)
            v = torch.randn((prompt, Hkv, D), generator=g).to(torch.bfloat16).to(dev)
            for c in caches:
                hwkv.prefill_write(c, l, b, 0, k, v)
    return pol, caches, g


def _check_case(L, B, Hq, Hkv, D, S, windows, levels, prompt, max_ctx, seed, steps):
    dev = torch.device("cuda:0")
    pol, (ca, cb), g = _pair(L, B, Hq, Hkv, D, S, windows, levels, prompt, max_ctx, seed, dev)
    ws = torch.zeros(hwkv.decode_workspace_bytes(ca), dtype=torch.uint8, device=dev)
    scale = 1.0 / math.sqrt(D)
    for step in range(steps):
        for l in range(L):
            q = torch.randn((B, Hq, D), generator=g).to(torch.bfloat16).to(dev)
            kn = torch.randn((B, Hkv, D), generator=g).to(torch.bfloat16).to(dev)
            vn = torch.randn((B, Hkv, D), generator=g).to(torch.bfloat16).to(dev)
            oa = torch.full((B, Hq, D), float("nan"), dtype=torch.float32, device=dev)
            ob = torch.full((B, Hq, D), float("nan"), dtype=torch.float32, device=dev)
            hwkv.append_decode_attn(ca, l, kn, vn, q, scale, oa, ws)
            hwkv.append_decode_attn_noalloc(cb, l, kn, vn, q, scale, ob)
            torch.cuda.synchronize()
            assert torch.isfinite(oa).all(), (step, l)
            assert torch.equal(oa, ob), (step, l, float((oa - ob).abs().max()))
    for l in range(L):
        for h in range(Hkv):
            for b in range(B):
                ka, va, na = hwkv.cache_read_unit(ca, l, h, b)
                kb, vb, nb = hwkv.cache_read_unit(cb, l, h, b)
                assert na == nb
                assert np.array_equal(ka[:na], kb[:nb]) and np.array_equal(va[:na], vb[:nb])
    ca.free()
    cb.free()


def test_no_alloc_matches_workspace_call_then_smaller():
    # a problem with many split workgroups per item (ring and full units,
    # two sequences), then a smaller one on the same static scratch
    _check_case(L=2, B=2, Hq=12, Hkv=2, D=256, S=4, windows=[256, 0], levels=[[0, 1], [1, 0]],
                prompt=3000, max_ctx=4096, seed=11, steps=2)
    _check_case(L=1, B=1, Hq=4, Hkv=1, D=128, S=2, windows=[64, 0], levels=[[1]],
                prompt=300, max_ctx=512, seed=12, steps=3)


def test_no_alloc_refuses_more_than_its_scratch():
    # 384 (sequence, kv head) items of 2,560 rows at head_dim 256 and 8 q
    # heads per kv head: six launches of about 512 split workgroups need
    # about 25 MB of partials, more than the 16 MiB scratch; the call is
    # refused before any launch and changes nothing
    dev = torch.device("cuda:0")
    B, Hkv, Hq, D, rows = 96, 4, 32, 256, 2560
    pol = hwkv.policy_set(1, Hkv, Hq, D, 0, [0], [[0] * Hkv])
    c = hwkv.cache_alloc(pol, B, rows + 64)
    try:
        k = torch.zeros((rows, Hkv, D), dtype=torch.bfloat16, device=dev)
        for b in range(B):
            hwkv.prefill_write(c, 0, b, 0, k, k)
        q = torch.zeros((B, Hq, D), dtype=torch.bfloat16, device=dev)
        kn = torch.zeros((B, Hkv, D), dtype=torch.bfloat16, device=dev)
        out = torch.zeros((B, Hq, D), dtype=torch.float32, device=dev)
        with pytest.raises(hwkv.HwkvError) as e:
            hwkv.append_decode_attn_noalloc(c, 0, kn, kn, q, 0.0625, out)
        assert e.value.code == hwkv.EINVAL
        assert "static scratch" in str(e.value)
        assert hwkv.cache_seq_len(c, 0, 0) == rows
        # the same call with a workspace runs
        ws = torch.zeros(hwkv.decode_workspace_bytes(c), dtype=torch.uint8, device=dev)
        hwkv.append_decode_attn(c, 0, kn, kn, q, 0.0625, out, ws)
        torch.cuda.synchronize()
        assert hwkv.cache_seq_len(c, 0, 0) == rows + 1
    finally:
        c.free()
