"""Shared driver for the GPU parity tests: runs a workload through the C ABI
(via the ctypes binding) and checks it against the fp64 oracle.

Inputs come from ``workloads`` (seeded, bf16).  Every comparison is made on
the same bf16 bit patterns: residency bit-exact (slot j of a unit must hold
the K and V rows of the position the oracle's slot table names), outputs
within the stated tolerance.
"""
import math
import sys
import time

import numpy as np
import torch

import oracle
import workloads as W
from oracle import kvformat as KF
from paper_2609_02029_amd import hwkv

REL_TOL = 1e-2     # the bar: max over rows of |o - ref|_inf / |ref|_inf
TIGHT_TOL = 2e-4   # fp32 accumulation over bf16 inputs stays far below it


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def up(a, dev):
    """Host bf16 bits (uint16) -> device torch.bfloat16."""
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)


def down(t):
    """Device torch.bfloat16 -> host uint16 bits."""
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def retained_absmax(av, t, w, S):
    """Max over the keys row t retains with window w (w = 0: every key up to
    t) of ``av`` [n, ..., D] (absolute values): the sinks [0, S) and the
    recent keys [t + 1 - w, t], each taken as a slice."""
    lo = max(0, t + 1 - w) if w else 0
    m = av[lo:t + 1].max(axis=0)
    s = min(S, lo)
    if s > 0:
        m = np.maximum(m, av[:s].max(axis=0))
    return m


def rel_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    num = np.abs(got - ref).max(axis=-1)
    den = np.abs(ref).max(axis=-1)
    return float((num / den).max())


class Run:
    """One workload on one GPU: policy, cache, seeded inputs, host histories.

    ``track``: layers whose full K/V history is kept on the host for the
    oracle (``None`` = all).  ``device_gen``: draw prompts on the device
    (large workloads) instead of on the host."""

    def __init__(self, cfg, dev="cuda:0", fused=True, track=None, device_gen=False,
                 levels=None, prompts=None, kv_format="bf16", k_scale=None, v_scale=None,
                 n_pages=None):
        self.cfg = cfg
        self.kv_format = kv_format
        self.dev = torch.device(dev)
        self.fused = fused
        self.device_gen = device_gen
        c = cfg
        self.L, self.B = c["n_layers"], c["batch"]
        self.Hq, self.Hkv, self.D, self.S = c["n_q_heads"], c["n_kv_heads"], c["head_dim"], c["n_sinks"]
        self.G = self.Hq // self.Hkv
        self.levels = levels if levels is not None else W.levels(c)
        self.windows = [[int(c["level_windows"][k]) for k in row] for row in self.levels]
        self.prompts = prompts if prompts is not None else W.prompts(c)
        self.max_ctx = c["max_ctx"]
        self.hist_len = max(self.max_ctx, max(self.prompts)) + 256
        self.scale = 1.0 / math.sqrt(self.D)
        self.outliers = W.outlier_channels(c)
        self.track = set(range(self.L)) if track is None else set(track)
        self.pol = hwkv.policy_set(self.L, self.Hkv, self.Hq, self.D, self.S,
                                   c["level_windows"], self.levels)
        self.cache = hwkv.cache_alloc(self.pol, self.B, self.max_ctx, kv_format=kv_format,
                                      k_scale=k_scale, v_scale=v_scale, n_pages=n_pages)
        self.gen = [0] * self.B      # refills of each sequence (seeds its new data)
        # per-unit fp8 scales as the library holds them (1.0 otherwise)
        _, self.k_scale, self.v_scale = hwkv.cache_format(self.cache)
        self.ws = torch.zeros(hwkv.decode_workspace_bytes(self.cache), dtype=torch.uint8,
                              device=self.dev)
        # host histories [layer][b] -> uint16 [max_ctx, Hkv, D]
        self.kh = {l: [None] * self.B for l in self.track}
        self.vh = {l: [None] * self.B for l in self.track}
        self.n = np.zeros((self.L, self.B), dtype=np.int64)
        self.step_no = np.zeros(self.L, dtype=np.int64)

    # ---------------- inputs
    def _kv(self, shape, layer, kind, idx):
        seed = self.cfg["seed"]
        if self.device_gen:
            t = W.normal_bf16_device(shape, seed, layer, kind, idx, device=self.dev,
                                     scale_channels=self.outliers, scale=self.cfg.get("outlier_scale", 1.0))
            return t, None
        a = W.normal_bf16(shape, seed, layer, kind, idx, scale_channels=self.outliers,
                          scale=self.cfg.get("outlier_scale", 1.0))
        return up(a, self.dev), a

    def prompt_kv(self, layer, b, P):
        idx = b + 1000 * self.gen[b]
        k, kh = self._kv((P, self.Hkv, self.D), layer, W.K, idx)
        v, vh = self._kv((P, self.Hkv, self.D), layer, W.V, idx)
        return k, v, kh, vh

    def reset(self, b):
        """Release sequence b (hwkv_cache_reset_seq); its next prompt is drawn
        from new seeds."""
        hwkv.cache_reset_seq(self.cache, b)
        self.n[:, b] = 0
        self.gen[b] += 1
        for l in self.track:
            if self.kh[l][b] is not None:
                self.kh[l][b][:] = 0
                self.vh[l][b][:] = 0

    def prompt_q(self, layer, b, P):
        """Queries of the prompt tokens, [P, Hq, D] (device, host or None)."""
        seed = self.cfg["seed"]
        if self.device_gen:
            return W.normal_bf16_device((P, self.Hq, self.D), seed, layer, W.Q_PROMPT, b,
                                        device=self.dev), None
        a = W.normal_bf16((P, self.Hq, self.D), seed, layer, W.Q_PROMPT, b)
        return up(a, self.dev), a

    def _hist(self, layer, b):
        if self.kh[layer][b] is None:
            self.kh[layer][b] = np.zeros((self.hist_len, self.Hkv, self.D), dtype=np.uint16)
            self.vh[layer][b] = np.zeros((self.hist_len, self.Hkv, self.D), dtype=np.uint16)
        return self.kh[layer][b], self.vh[layer][b]

    # ---------------- operations
    def prefill(self, layer, b, P=None, chunks=None):
        P = self.prompts[b] if P is None else P
        k, v, kh, vh = self.prompt_kv(layer, b, P)
        cuts = [0] + sorted(chunks or []) + [P]
        for p0, p1 in zip(cuts[:-1], cuts[1:]):
            if p1 > p0:
                hwkv.prefill_write(self.cache, layer, b, p0, k[p0:p1], v[p0:p1])
        if layer in self.track:
            hk, hv = self._hist(layer, b)
            hk[:P] = kh if kh is not None else down(k)
            hv[:P] = vh if vh is not None else down(v)
        self.n[layer, b] = P
        del k, v

    def prefill_with_attn(self, layer, b, P=None, chunks=None, check_untouched=False):
        """Chunked prefill with attention: per chunk [p0, p1), prefill_attn
        of its queries over the cache as it stands plus the chunk, then
        prefill_write of the chunk.  Returns (q device, q host or None,
        out fp32 device [P, Hq, D])."""
        P = self.prompts[b] if P is None else P
        k, v, kh, vh = self.prompt_kv(layer, b, P)
        q, qh = self.prompt_q(layer, b, P)
        out = torch.full((P, self.Hq, self.D), float("nan"), dtype=torch.float32, device=self.dev)
        cuts = [0] + sorted(chunks or []) + [P]
        for p0, p1 in zip(cuts[:-1], cuts[1:]):
            if p1 <= p0:
                continue
            before = self._snapshot(layer, b) if check_untouched else None
            hwkv.prefill_attn(self.cache, layer, b, p0, q[p0:p1], k[p0:p1], v[p0:p1],
                              self.scale, out[p0:p1], ws=self.prefill_ws(P))
            if check_untouched:
                after = self._snapshot(layer, b)
                for x, y in zip(before, after):
                    assert np.array_equal(x, y), "prefill_attn changed the cache"
            hwkv.prefill_write(self.cache, layer, b, p0, k[p0:p1], v[p0:p1])
        if layer in self.track:
            hk, hv = self._hist(layer, b)
            hk[:P] = kh if kh is not None else down(k)
            hv[:P] = vh if vh is not None else down(v)
        self.n[layer, b] = P
        del k, v
        return q, qh, out

    def prefill_ws(self, n_tokens):
        """Workspace of hwkv_prefill_attn_ws for chunks of up to n_tokens
        (None for a bf16 cache)."""
        if self.kv_format == "bf16":
            return None
        need = hwkv.prefill_attn_workspace_bytes(self.cache, n_tokens)
        if getattr(self, "_pws", None) is None or self._pws.numel() < need:
            self._pws = torch.zeros(max(need, 1), dtype=torch.uint8, device=self.dev)
        return self._pws

    def _snapshot(self, layer, b):
        res = []
        for h in range(self.Hkv):
            k, v, nv = hwkv.cache_read_unit(self.cache, layer, h, b)
            res += [k[:nv], v[:nv]]
        return res

    def oracle_rows(self, layer, b, rows, q_rows, n_threads=16):
        """Masked-full-cache oracle for query tokens ``rows`` of sequence b:
        each row attends over the retained set at its own position within
        the full host history.  ``q_rows`` [len(rows), Hq, D] bf16 bits."""
        rows = np.asarray(rows, dtype=np.int64)
        hk, hv = self.kh[layer][b], self.vh[layer][b]
        if self.kv_format != "bf16":   # attention over the stored values
            n = int(rows[-1]) + 1
            kv, vv = self.stored_values(layer, hk[:n], hv[:n])
            return KF.attend_values(KF.bf16_values(q_rows), [kv] * len(rows), [vv] * len(rows),
                                    rows, self.S, self.windows[layer], self.scale)
        return oracle.decode_layer(q_rows, [hk] * len(rows), [hv] * len(rows), rows, self.S,
                                   self.windows[layer], self.scale, n_threads=n_threads)

    def step(self, layer, fused=None):
        """Append one token to every sequence of ``layer`` and attend."""
        fused = self.fused if fused is None else fused
        st = int(self.step_no[layer])
        seed = self.cfg["seed"]
        qa = W.normal_bf16((self.B, self.Hq, self.D), seed, layer, W.Q, st)
        ka = W.normal_bf16((self.B, self.Hkv, self.D), seed, layer, W.K_NEW, st,
                           scale_channels=self.outliers, scale=self.cfg.get("outlier_scale", 1.0))
        va = W.normal_bf16((self.B, self.Hkv, self.D), seed, layer, W.V_NEW, st,
                           scale_channels=self.outliers, scale=self.cfg.get("outlier_scale", 1.0))
        q, kn, vn = up(qa, self.dev), up(ka, self.dev), up(va, self.dev)
        out = torch.empty((self.B, self.Hq, self.D), dtype=torch.float32, device=self.dev)
        if fused:
            hwkv.append_decode_attn(self.cache, layer, kn, vn, q, self.scale, out, self.ws)
        else:
            hwkv.append(self.cache, layer, kn, vn)
            hwkv.decode_attn(self.cache, layer, q, self.scale, out, self.ws)
        if layer in self.track:
            for b in range(self.B):
                hk, hv = self._hist(layer, b)
                hk[self.n[layer, b]] = ka[b]
                hv[self.n[layer, b]] = va[b]
        self.n[layer] += 1
        self.step_no[layer] += 1
        return qa, out

    # ---------------- checks
    def history(self, layer, b):
        """Regenerate the full K/V history of (layer, b) from the seeds:
        the prompt plus every token appended so far."""
        P = self.prompts[b]
        k, v, kh, vh = self.prompt_kv(layer, b, P)
        hk = np.zeros((self.hist_len, self.Hkv, self.D), dtype=np.uint16)
        hv = np.zeros_like(hk)
        hk[:P] = kh if kh is not None else down(k)
        hv[:P] = vh if vh is not None else down(v)
        del k, v
        seed = self.cfg["seed"]
        sc, s = self.outliers, self.cfg.get("outlier_scale", 1.0)
        for st in range(int(self.step_no[layer])):
            hk[P + st] = W.normal_bf16((self.B, self.Hkv, self.D), seed, layer, W.K_NEW, st,
                                       scale_channels=sc, scale=s)[b]
            hv[P + st] = W.normal_bf16((self.B, self.Hkv, self.D), seed, layer, W.V_NEW, st,
                                       scale_channels=sc, scale=s)[b]
        return hk, hv

    def stored(self, layer, hk, hv):
        """Stored elements (the oracle's encoding) of host histories [n, Hkv, D]
        in the cache format, with each KV head's scales."""
        if self.kv_format == "bf16":
            return hk, hv
        sk = np.stack([KF.store(hk[:, h], self.kv_format, self.k_scale[layer, h])
                       for h in range(self.Hkv)], axis=1)
        sv = np.stack([KF.store(hv[:, h], self.kv_format, self.v_scale[layer, h])
                       for h in range(self.Hkv)], axis=1)
        return sk, sv

    def stored_values(self, layer, hk, hv):
        """fp64 values of the stored elements of host histories."""
        sk, sv = self.stored(layer, hk, hv)
        kv = np.stack([KF.values(sk[:, h], self.kv_format, self.k_scale[layer, h])
                       for h in range(self.Hkv)], axis=1)
        vv = np.stack([KF.values(sv[:, h], self.kv_format, self.v_scale[layer, h])
                       for h in range(self.Hkv)], axis=1)
        return kv, vv

    def retained_values(self, layer, b, h, t):
        """(positions, K values, V values) of the positions query t of
        sequence b retains in unit (layer, h): the stored elements of those
        rows only, fp64 [n, D] each."""
        pos = KF.retained_positions(int(t), self.S, self.windows[layer][h])
        fmt = self.kv_format
        kv = KF.values(KF.store(self.kh[layer][b][pos, h], fmt, self.k_scale[layer, h]), fmt,
                       self.k_scale[layer, h])
        vv = KF.values(KF.store(self.vh[layer][b][pos, h], fmt, self.v_scale[layer, h]), fmt,
                       self.v_scale[layer, h])
        return pos, kv, vv

    def _stored_oracle(self, layer, qa):
        """Oracle outputs over the stored values, and max |v| per (sequence,
        kv head, channel) over the retained rows.  Per (sequence, kv head):
        the oracle's attention over that head's retained rows alone (gathered
        before decoding; as a one-head problem whose every row is retained,
        the same sums in the same order as over the whole history)."""
        t = self.n[layer] - 1
        qv = KF.bf16_values(qa)
        G = self.G
        out = np.empty(qv.shape, dtype=np.float64)
        vmax = np.zeros((self.B, self.Hkv, self.D))
        for b in range(self.B):
            for h in range(self.Hkv):
                pos, kv, vv = self.retained_values(layer, b, h, t[b])
                out[b, h * G:(h + 1) * G] = KF.attend_values(
                    qv[b:b + 1, h * G:(h + 1) * G], [kv[:, None]], [vv[:, None]],
                    [len(pos) - 1], 0, [0], self.scale)[0]
                vmax[b, h] = np.abs(vv).max(axis=0)
        return out, vmax

    def oracle_out(self, layer, qa, n_threads=8):
        t = self.n[layer] - 1
        if self.kv_format != "bf16":
            return self._stored_oracle(layer, qa)[0]
        return oracle.decode_layer(qa, [self.kh[layer][b][: t[b] + 1] for b in range(self.B)],
                                   [self.vh[layer][b][: t[b] + 1] for b in range(self.B)], t,
                                   self.S, self.windows[layer], self.scale, n_threads=n_threads)

    def value_bound(self, layer):
        """max_s |v_s[c]| over the retained positions of each (sequence, KV
        head, channel) at the current lengths: [B, Hkv, D]."""
        t = self.n[layer] - 1
        out = np.zeros((self.B, self.Hkv, self.D))
        for b in range(self.B):
            for h in range(self.Hkv):
                _, _, vv = self.retained_values(layer, b, h, t[b])
                out[b, h] = np.abs(vv).max(axis=0)
        return out

    def check_out(self, layer, qa, out, what=""):
        torch.cuda.synchronize()
        if self.kv_format != "bf16":
            ref, vbound = self._stored_oracle(layer, qa)
        else:
            ref = self.oracle_out(layer, qa)
        got = out.cpu().numpy()
        e = rel_err(got.reshape(-1, self.D), ref.reshape(-1, self.D))
        assert np.all(np.isfinite(got)), f"{what}: non-finite output"
        assert e <= REL_TOL, f"{what}: max rel err {e} > {REL_TOL}"
        if self.kv_format == "fp8":
            # the softmax weights enter the value product as two bf16 terms
            # (hi = round(p), lo = round(p - hi)), which leave at most
            # 2^-18 p of each weight behind; with margin, per channel
            # |o - ref| <= (2^-16 + 2e-5) max_s |v_s| (fp32 accumulation and
            # the exp2 rounding take the 2e-5)
            vmax = np.repeat(vbound, self.G, axis=1)
            err = np.abs(got - ref)
            lim = (2.0 ** -16 + 2e-5) * vmax
            assert np.all(err <= lim), (f"{what}: weight-rounding bound exceeded by "
                                        f"{float((err / np.maximum(lim, 1e-300)).max()):.3f}x")
        else:
            assert e <= TIGHT_TOL, f"{what}: max rel err {e} > {TIGHT_TOL} (fp32 accumulation bound)"
        return e

    def check_unit(self, layer, h, b, hist=None):
        """Bit-exact residency of one (unit, sequence) against the oracle."""
        tab = oracle.UnitTable(self.S, self.windows[layer][h], self.max_ctx)
        if self.n[layer, b] > 0:
            tab.prefill(0, int(self.n[layer, b]))
        k, v, nv = hwkv.cache_read_unit(self.cache, layer, h, b)
        assert nv == tab.n_valid, (layer, h, b, nv, tab.n_valid)
        assert k.shape[0] == tab.cap
        occ = tab.table[:nv]
        assert np.all(occ >= 0)
        hk, hv = (self.kh[layer][b], self.vh[layer][b]) if hist is None else hist
        ek = KF.store(hk[occ, h], self.kv_format, self.k_scale[layer, h])
        ev = KF.store(hv[occ, h], self.kv_format, self.v_scale[layer, h])
        assert np.array_equal(k[:nv], ek), f"K residency differs: layer {layer} head {h} seq {b}"
        assert np.array_equal(v[:nv], ev), f"V residency differs: layer {layer} head {h} seq {b}"

    def check_layer(self, layer, hist=None):
        for b in range(self.B):
            for h in range(self.Hkv):
                self.check_unit(layer, h, b, hist=None if hist is None else hist[b])

    def free(self):
        self.cache.free()


def timed(label):
    class _T:
        def __enter__(self):
            self.t = time.time()
            log(f"[{label}] start")
            return self

        def __exit__(self, *a):
            log(f"[{label}] done in {time.time() - self.t:.1f}s")
    return _T()
