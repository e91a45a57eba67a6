"""Seeded synthetic streams shaped like the paper's video-LLM workloads.

This module only draws inputs: keys, values, queries and PQ codebooks.  It
holds none of the method's arithmetic (no assignment, aggregation, decoding
or attention), so both the HIP path and the CPU oracle can be fed from it.

The paper's datasets (RVS-Ego/Movie, OVO-Bench, StreamingBench) and model
weights are not available; these streams stand in for them with the shapes
of a 7B video LLM (head_dim 128, 196 visual tokens per frame on a 14x14 grid,
GQA) and a key distribution with object-like structure: keys are drawn from a
Gaussian mixture whose cluster identity persists across frames, values are
standard normal.

Two generators share one recipe:

* ``HostStream`` (numpy, PCG64) produces exact bytes; parity tests feed the
  same bytes to the oracle and to the GPU.
* ``DeviceStream`` (torch, on the GPU) draws the same distribution directly
  in device memory for throughput runs.  Its bytes differ from the host
  generator's.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence

import numpy as np

# --------------------------------------------------------------------------
# Workload descriptions
# --------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    num_layers: int
    num_kv_heads: int
    num_q_heads: int
    head_dim: int
    grid_h: int
    grid_w: int
    frames: int
    window_frames: int
    capacity: int
    query_tokens: int
    kv_dtype: str            # "bf16" or "fp32"
    clusters: int
    structure: str           # "iid" | "persistent" | "cue" | "spatial"
    streams: int = 1
    seed_base: int = 20260
    sigma: float = 0.1       # per-dimension key noise around the cluster mean
    persist_redraw: float = 0.02
    drift: float = 0.02
    query_every: int = 0     # multi-stream: one query per stream every N frames

    @property
    def tokens_per_frame(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def units(self) -> int:
        """(layer, kv head) pairs of one stream."""
        return self.num_layers * self.num_kv_heads

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    # 1 layer x 1 KV head, fp32, 8x8 grid, 32 frames, window 4 frames, K=64.
    "tiny": Workload("tiny-1x1-d128-fp32-k64", 1, 1, 1, 128, 8, 8, 32, 4, 64,
                     16, "fp32", 8, "iid", seed_base=21260),
    # 7B-class video LLM: 28 layers x 4 KV heads (28 query heads), bf16,
    # 196 tokens/frame (14x14), 256 frames, window 8 frames, K=256.
    "7b": Workload("7b-28x4-d128-bf16-t196-w8-k256", 28, 4, 28, 128, 14, 14,
                   256, 8, 256, 32, "bf16", 64, "persistent", seed_base=22260),
    # Long delay: same model, 4096 frames, window 16 frames, K=1024, rare cue
    # cluster in frames 100-102 only.
    "long": Workload("long-delay-28x4-d128-bf16-t196-w16-k1024", 28, 4, 28, 128,
                     14, 14, 4096, 16, 1024, 64, "bf16", 256, "cue",
                     seed_base=23260),
    # High resolution: 32 layers x 8 KV heads (32 query heads), 576 tokens per
    # frame (24x24), 1024 frames, window 8 frames, K=2048.
    "hires": Workload("hires-32x8-d128-bf16-t576-w8-k2048", 32, 8, 32, 128, 24,
                      24, 1024, 8, 2048, 32, "bf16", 64, "spatial",
                      seed_base=24260),
    # 64 concurrent streams of the 7B shape, K=512, one 32-token query per
    # stream every 128 frames.
    "multi": Workload("multistream-64x28x4-d128-bf16-t196-w8-k512", 28, 4, 28,
                      128, 14, 14, 1024, 8, 512, 32, "bf16", 64, "persistent",
                      streams=64, seed_base=25260, query_every=128),
}

CUE_FRAMES = (100, 101, 102)
CUE_PATCH = 4
SPATIAL_BANDWIDTH = 0.15


def frame_coordinates(grid_h: int, grid_w: int) -> np.ndarray:
    """Cell-centre coordinates (x, y) in [0,1]^2 in raster order (float64).

    Used by the generator for the per-position spatial bias only."""
    rows, cols = np.divmod(np.arange(grid_h * grid_w), grid_w)
    return np.stack([(cols + 0.5) / grid_w, (rows + 0.5) / grid_h], axis=1)


# --------------------------------------------------------------------------
# bf16 helpers (generator side)
# --------------------------------------------------------------------------


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round to bfloat16 (round-to-nearest-even via float32) -> uint16 bits."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def quantize(x: np.ndarray, kv_dtype: str) -> np.ndarray:
    """Values as stored in the KV cache, returned as float32."""
    if kv_dtype == "bf16":
        return bf16_bits_to_f32(to_bf16_bits(x))
    return np.asarray(x, dtype=np.float32)


# --------------------------------------------------------------------------
# Host (numpy) generator: exact bytes for parity
# --------------------------------------------------------------------------


class _HeadProcess:
    """Label process and cluster means of one (stream, layer, kv head)."""

    def __init__(self, wl: Workload, rng: np.random.Generator):
        self.wl = wl
        self.rng = rng
        D, C, T = wl.head_dim, wl.clusters, wl.tokens_per_frame
        z = rng.standard_normal((C, D))
        self.means = z / np.linalg.norm(z, axis=1, keepdims=True)
        if wl.structure == "iid":
            self.labels = None
        elif wl.structure == "persistent":
            coarse = rng.integers(0, C, size=(8, 8))
            r = (np.arange(wl.grid_h) * 8) // wl.grid_h
            c = (np.arange(wl.grid_w) * 8) // wl.grid_w
            self.labels = coarse[r[:, None], c[None, :]].reshape(T)
        elif wl.structure == "cue":
            self.labels = rng.integers(1, C, size=T)
            pr = int(rng.integers(0, wl.grid_h - CUE_PATCH + 1))
            pc = int(rng.integers(0, wl.grid_w - CUE_PATCH + 1))
            rows, cols = np.divmod(np.arange(T), wl.grid_w)
            self.cue_mask = ((rows >= pr) & (rows < pr + CUE_PATCH)
                             & (cols >= pc) & (cols < pc + CUE_PATCH))
        elif wl.structure == "spatial":
            self.labels = None
            anchors = rng.random((C, 2))
            s = frame_coordinates(wl.grid_h, wl.grid_w)
            d2 = ((s[:, None, :] - anchors[None, :, :]) ** 2).sum(-1)
            w = np.exp(-d2 / (2 * SPATIAL_BANDWIDTH ** 2))
            self.cdf = np.cumsum(w / w.sum(axis=1, keepdims=True), axis=1)
        else:
            raise ValueError(wl.structure)
        self.frame = 0

    def _frame_labels(self) -> np.ndarray:
        wl, rng, T, C = self.wl, self.rng, self.wl.tokens_per_frame, self.wl.clusters
        if wl.structure == "iid":
            return rng.integers(0, C, size=T)
        if wl.structure == "spatial":
            u = rng.random(T)
            lab = (self.cdf < u[:, None]).sum(axis=1)
            return np.minimum(lab, C - 1)
        if self.frame > 0:
            redraw = rng.random(T) < wl.persist_redraw
            lo = 1 if wl.structure == "cue" else 0
            self.labels[redraw] = rng.integers(lo, C, size=int(redraw.sum()))
            xi = rng.standard_normal(self.means.shape)
            m = self.means + wl.drift * xi / math.sqrt(wl.head_dim)
            self.means = m / np.linalg.norm(m, axis=1, keepdims=True)
        lab = self.labels.copy()
        if wl.structure == "cue" and self.frame in CUE_FRAMES:
            lab[self.cue_mask] = 0
        return lab

    def next(self):
        lab = self._frame_labels()
        T, D = self.wl.tokens_per_frame, self.wl.head_dim
        k = self.means[lab] + self.wl.sigma * self.rng.standard_normal((T, D))
        v = self.rng.standard_normal((T, D))
        self.frame += 1
        return lab, k, v


class HostStream:
    """Seeded frames of one stream for a chosen subset of (layer, kv head) units.

    Each unit has its own PCG64 generator, so the bytes of a unit do not
    depend on which other units are generated.  Frames come out as float32
    arrays holding values exactly representable in the workload's KV dtype.
    """

    def __init__(self, wl: Workload, stream: int = 0,
                 units: Optional[Sequence[int]] = None):
        self.wl = wl
        self.stream = stream
        self.units = list(range(wl.units)) if units is None else list(units)
        ss = np.random.SeedSequence(wl.seed_base + stream).spawn(wl.units)
        self._heads = {u: _HeadProcess(wl, np.random.Generator(np.random.PCG64(ss[u])))
                       for u in self.units}
        self.frame = 0

    def next_frame(self):
        """-> (K, V) float32 [len(units)][T][D] in the KV dtype's values."""
        ks, vs = [], []
        for u in self.units:
            _, k, v = self._heads[u].next()
            ks.append(k)
            vs.append(v)
        self.frame += 1
        return (quantize(np.stack(ks), self.wl.kv_dtype),
                quantize(np.stack(vs), self.wl.kv_dtype))

    def query(self, seed_offset: int = 0) -> np.ndarray:
        """Query Q float32 [L][Tq][Hq][D] for the current stream state.

        Needs every unit of the stream (all query heads are drawn).  The first
        half of the tokens are N(0, I); the second half are aligned with one
        cluster of the owning KV head (the cue cluster for the long-delay
        stream): q = 4 sqrt(D) mu + N(0, I), i.e. logit ~4 on that cluster.
        """
        wl = self.wl
        assert len(self.units) == wl.units, "query needs all units of the stream"
        rng = np.random.Generator(np.random.PCG64(
            np.random.SeedSequence([wl.seed_base + self.stream, 7, self.frame, seed_offset])))
        L, Tq, Hq, Hkv, D = wl.num_layers, wl.query_tokens, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
        grp = Hq // Hkv
        q = rng.standard_normal((L, Tq, Hq, D))
        half = Tq // 2
        for l in range(L):
            for h in range(Hq):
                u = l * Hkv + h // grp
                means = self._heads[u].means
                for t in range(half, Tq):
                    c = 0 if wl.structure == "cue" else int(rng.integers(0, wl.clusters))
                    q[l, t, h] += 4.0 * math.sqrt(D) * means[c]
        return quantize(q, wl.kv_dtype)


def make_codebooks(wl: Workload, stream: int = 0, units: Optional[Sequence[int]] = None,
                   samples: int = 2048, iters: int = 12, G: int = 8, C: int = 16) -> np.ndarray:
    """Per-unit PQ codebooks float32 [len(units)][2][G][C][D/G] (keys, values).

    Lloyd k-means per subspace on a seeded warm-up sample of residuals
    (key residuals sigma*N(0,I) around the cluster mean, values N(0,I)),
    standing in for the paper's warm-up reservoir.  Initial centres are
    the first C samples; ties go to the lowest index.
    """
    D = wl.head_dim
    Dp = D // G
    units = list(range(wl.units)) if units is None else list(units)
    out = np.zeros((len(units), 2, G, C, Dp), dtype=np.float32)
    for i, u in enumerate(units):
        rng = np.random.Generator(np.random.PCG64(
            np.random.SeedSequence([wl.seed_base + stream, 11, u])))
        for kv in range(2):
            scale = wl.sigma if kv == 0 else 1.0
            x = scale * rng.standard_normal((samples, G, Dp))
            for g in range(G):
                pts = x[:, g, :]
                cen = pts[:C].copy()
                for _ in range(iters):
                    d2 = ((pts[:, None, :] - cen[None, :, :]) ** 2).sum(-1)
                    lab = np.argmin(d2, axis=1)
                    for c in range(C):
                        sel = pts[lab == c]
                        if len(sel):
                            cen[c] = sel.mean(axis=0)
                out[i, kv, g] = cen.astype(np.float32)
    return out


# --------------------------------------------------------------------------
# Device (torch) generator: same recipe, device-resident, for throughput runs
# --------------------------------------------------------------------------


class DeviceStream:
    """Frames for all units of ``n_streams`` streams, drawn on the GPU.

    Same distribution as ``HostStream`` (different bytes).  Output layout is
    [n_streams][L][Hkv][T][D] in the workload's KV dtype (torch tensors).
    """

    def __init__(self, wl: Workload, n_streams: int = 1, device="cuda", seed: int = 0):
        import torch
        self.torch = torch
        self.wl = wl
        self.device = device
        self.gen = torch.Generator(device=device)
        self.gen.manual_seed(wl.seed_base * 1000 + seed)
        U = n_streams * wl.units
        D, C, T = wl.head_dim, wl.clusters, wl.tokens_per_frame
        self.shape = (n_streams, wl.num_layers, wl.num_kv_heads, T, D)
        z = torch.randn(U, C, D, generator=self.gen, device=device, dtype=torch.float32)
        self.means = z / z.norm(dim=-1, keepdim=True)
        if wl.structure in ("persistent", "cue"):
            lo = 1 if wl.structure == "cue" else 0
            if wl.structure == "persistent":
                coarse = torch.randint(0, C, (U, 8, 8), generator=self.gen, device=device)
                r = (torch.arange(wl.grid_h, device=device) * 8) // wl.grid_h
                c = (torch.arange(wl.grid_w, device=device) * 8) // wl.grid_w
                self.labels = coarse[:, r[:, None], c[None, :]].reshape(U, T)
            else:
                self.labels = torch.randint(lo, C, (U, T), generator=self.gen, device=device)
                # one seeded CUE_PATCH x CUE_PATCH patch per unit shows cluster 0 in CUE_FRAMES
                pr = torch.randint(0, wl.grid_h - CUE_PATCH + 1, (U, 1), generator=self.gen, device=device)
                pc = torch.randint(0, wl.grid_w - CUE_PATCH + 1, (U, 1), generator=self.gen, device=device)
                pos = torch.arange(T, device=device)[None, :]
                rows, cols = pos // wl.grid_w, pos % wl.grid_w
                self.cue_mask = ((rows >= pr) & (rows < pr + CUE_PATCH)
                                 & (cols >= pc) & (cols < pc + CUE_PATCH))
        else:
            self.labels = None
        if wl.structure == "spatial":
            anchors = torch.rand(U, C, 2, generator=self.gen, device=device)
            s = torch.tensor(frame_coordinates(wl.grid_h, wl.grid_w), device=device,
                             dtype=torch.float32)
            d2 = ((s[None, :, None, :] - anchors[:, None, :, :]) ** 2).sum(-1)
            w = torch.exp(-d2 / (2 * SPATIAL_BANDWIDTH ** 2))
            self.cdf = torch.cumsum(w / w.sum(-1, keepdim=True), dim=-1)
        self.frame = 0
        self.U = U

    def next_frame(self):
        torch, wl = self.torch, self.wl
        C, T, D = wl.clusters, wl.tokens_per_frame, wl.head_dim
        if wl.structure == "iid":
            lab = torch.randint(0, C, (self.U, T), generator=self.gen, device=self.device)
        elif wl.structure == "spatial":
            u = torch.rand(self.U, T, 1, generator=self.gen, device=self.device)
            lab = (self.cdf < u).sum(-1).clamp_max(C - 1)
        else:
            if self.frame > 0:
                lo = 1 if wl.structure == "cue" else 0
                redraw = torch.rand(self.U, T, generator=self.gen, device=self.device) < wl.persist_redraw
                fresh = torch.randint(lo, C, (self.U, T), generator=self.gen, device=self.device)
                self.labels = torch.where(redraw, fresh, self.labels)
                xi = torch.randn(self.means.shape, generator=self.gen, device=self.device)
                m = self.means + wl.drift * xi / math.sqrt(D)
                self.means = m / m.norm(dim=-1, keepdim=True)
            lab = self.labels
            if wl.structure == "cue" and self.frame in CUE_FRAMES:
                lab = torch.where(self.cue_mask, torch.zeros_like(lab), lab)
        k = torch.gather(self.means, 1, lab[..., None].expand(self.U, T, D))
        k = k + wl.sigma * torch.randn(self.U, T, D, generator=self.gen, device=self.device)
        v = torch.randn(self.U, T, D, generator=self.gen, device=self.device)
        dt = torch.bfloat16 if wl.kv_dtype == "bf16" else torch.float32
        self.frame += 1
        return k.to(dt).reshape(self.shape).contiguous(), v.to(dt).reshape(self.shape).contiguous()

    def query(self):
        torch, wl = self.torch, self.wl
        L, Tq, Hq, Hkv, D = wl.num_layers, wl.query_tokens, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
        grp = Hq // Hkv
        q = torch.randn(L, Tq, Hq, D, generator=self.gen, device=self.device)
        half = Tq // 2
        # cluster-aligned half, using stream 0's unit means
        c = torch.randint(0, wl.clusters, (L, Tq - half, Hq), generator=self.gen, device=self.device)
        if wl.structure == "cue":
            c.zero_()
        unit = (torch.arange(L, device=self.device)[:, None] * Hkv
                + torch.arange(Hq, device=self.device)[None, :] // grp)      # [L][Hq]
        mu = self.means[unit[:, None, :].expand(L, Tq - half, Hq), c]       # [L][Tq-half][Hq][D]
        q[:, half:] += 4.0 * math.sqrt(D) * mu
        dt = torch.bfloat16 if wl.kv_dtype == "bf16" else torch.float32
        return q.to(dt).contiguous()


def make_codebooks_device(wl: Workload, n_streams: int = 1, samples: int = 2048, iters: int = 12,
                          G: int = 8, C: int = 16, device="cuda", seed: int = 0):
    """Same recipe as ``make_codebooks`` (Lloyd k-means per subspace on seeded
    warm-up residuals), batched over every unit on the GPU.  Returns a numpy
    float32 array [n_streams][units][2][G][C][D/G]."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(wl.seed_base * 7919 + seed)
    U = n_streams * wl.units
    Dp = wl.head_dim // G
    scale = torch.tensor([wl.sigma, 1.0], device=device).view(1, 2, 1, 1, 1)
    x = torch.randn(U, 2, G, samples, Dp, generator=gen, device=device) * scale
    x = x.reshape(U * 2 * G, samples, Dp)
    cen = x[:, :C].clone()
    for _ in range(iters):
        lab = torch.cdist(x, cen).argmin(dim=-1)                       # [B][samples]
        onehot = torch.nn.functional.one_hot(lab, C).to(x.dtype)       # [B][samples][C]
        cnt = onehot.sum(1)                                            # [B][C]
        tot = torch.einsum("bsc,bsd->bcd", onehot, x)
        cen = torch.where(cnt[..., None] > 0, tot / cnt.clamp_min(1)[..., None], cen)
    return cen.reshape(n_streams, wl.units, 2, G, C, Dp).float().cpu().numpy()
