"""Seeded synthetic attention inputs.

The only module shared by the HIP path's callers and the oracle side: it
draws random numbers and rounds them to bf16 bit patterns, and holds none of
the method's arithmetic.  Every tensor is drawn on the CPU with numpy's
PCG64 so that both sides see identical bits.

The five workloads stand in for the paper's evaluation models (Sec. 4: the
long-context LLM runs at 32K-96K tokens, the Wan-2.2 text-to-video model),
whose weights and activations are not available: LLM-shaped prefill with
outlier channels, batched GQA decode over a KV cache with log-normal key
norms, a ViT/multimodal-shaped encoder, and a long-context prefill with an
attention-sink prefix.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    Hq: int
    Hkv: int
    Sq: int
    Sk: int
    D: int
    causal: bool
    block: int
    outliers: bool = False     # ceil(1% of D) shared channels of Q and K scaled x20
    sink: int = 0              # first `sink` key rows scaled x8
    lognormal_k: bool = False  # per-token key norm drawn LogNormal(0, 0.5)

    @property
    def flops(self) -> float:
        """Algorithmic FLOPs: 4*D per unmasked (query, key) pair."""
        return 4.0 * self.D * self.pairs * self.B * self.Hq

    @property
    def pairs(self) -> int:
        """Unmasked (query, key) pairs of one head (bottom-right causal)."""
        if not self.causal:
            return self.Sq * self.Sk
        r = np.arange(self.Sq, dtype=np.int64)
        return int(np.clip(r + (self.Sk - self.Sq) + 1, 0, self.Sk).sum())

    @property
    def bytes_qkvo(self) -> int:
        """Bytes of Q, K, V (bf16) read and O (fp32) + lse (fp32) written."""
        q = self.B * self.Hq * self.Sq * self.D * 2
        kv = 2 * self.B * self.Hkv * self.Sk * self.D * 2
        o = self.B * self.Hq * self.Sq * self.D * 4
        lse = self.B * self.Hq * self.Sq * 4
        return q + kv + o + lse


WORKLOADS = {
    1: Workload("tiny 1x1x256x256 d64", 1, 1, 1, 256, 256, 64, False, 64),
    2: Workload("llama3-8b prefill 4096 gqa32/8 d128 causal", 1, 32, 8, 4096, 4096, 128, True, 128,
                outliers=True),
    3: Workload("batched decode b64 sk8192 gqa32/8 d128", 64, 32, 8, 1, 8192, 128, False, 128,
                lognormal_k=True),
    4: Workload("vit encoder b8 h16 4096 d64", 8, 16, 16, 4096, 4096, 64, False, 64),
    5: Workload("long prefill 32768 gqa32/8 d128 causal sink4", 1, 32, 8, 32768, 32768, 128, True, 128,
                outliers=True, sink=4),
}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (to nearest, ties to even) and return the
    16-bit patterns.  Inputs are finite."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _normal(seed: int, shape) -> np.ndarray:
    return np.random.Generator(np.random.PCG64(seed)).standard_normal(shape, dtype=np.float32)


def make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=0, outliers=False, sink=0, lognormal_k=False,
             q_scale=1.0, k_scale=1.0):
    """bf16 bit patterns q [B,Hq,Sq,D], k, v [B,Hkv,Sk,D].

    Seeds: seed+1000 for Q, seed+2000 for K, seed+3000 for V, seed+4000 for
    the outlier channels and the key norms."""
    q = _normal(seed + 1000, (B, Hq, Sq, D)) * np.float32(q_scale)
    k = _normal(seed + 2000, (B, Hkv, Sk, D)) * np.float32(k_scale)
    v = _normal(seed + 3000, (B, Hkv, Sk, D))
    aux = np.random.Generator(np.random.PCG64(seed + 4000))
    if outliers:
        nch = max(1, math.ceil(0.01 * D))
        ch = aux.choice(D, size=nch, replace=False)
        q[..., ch] *= np.float32(20.0)
        k[..., ch] *= np.float32(20.0)
    if lognormal_k:
        g = aux.lognormal(0.0, 0.5, size=(B, Hkv, Sk, 1)).astype(np.float32)
        k *= g
    if sink:
        k[:, :, :sink, :] *= np.float32(8.0)
    return f32_to_bf16_bits(q), f32_to_bf16_bits(k), f32_to_bf16_bits(v)


def make_slow_climb(B, Hq, Hkv, Sq, Sk, D, delta, block, seed=0):
    """bf16 q [B,Hq,Sq,D], k, v [B,Hkv,Sk,D] whose scores climb slowly along
    the keys: every query is close to the all-ones vector and key t carries
    the offset t * delta / (block * sqrt(D) * log2(e)) in every channel, so
    the score in log2 units (scale 1/sqrt(D)) rises by about `delta` per key
    block.  The running maximum then moves by a small non-integer step at
    nearly every block while the early blocks keep their weight: the case
    where the rescale factors of the online softmax compound.  Small noise
    (seed+1000 for Q, seed+2000 for K, seed+3000 for V) keeps rows distinct."""
    q = np.float32(1.0) + np.float32(0.01) * _normal(seed + 1000, (B, Hq, Sq, D))
    ramp = (np.arange(Sk, dtype=np.float64) * delta / (block * math.sqrt(D) * math.log2(math.e))).astype(np.float32)
    k = ramp[None, None, :, None] + np.float32(0.01) * _normal(seed + 2000, (B, Hkv, Sk, D))
    v = _normal(seed + 3000, (B, Hkv, Sk, D))
    return f32_to_bf16_bits(q), f32_to_bf16_bits(k), f32_to_bf16_bits(v)


def quantize_e4m3(x: np.ndarray, scale: float) -> np.ndarray:
    """OCP FP8 E4M3 codes of x / scale: round to nearest, ties to even,
    saturating at +-448 (the inputs of the FP8 Q/K path)."""
    y = np.asarray(x, dtype=np.float64) / float(np.float32(scale))
    a = np.minimum(np.abs(y), 448.0)
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -9)))
    e = np.maximum(e, -6.0)                           # subnormals share the step 2^-9
    step = 2.0 ** (e - 3)
    q = np.round(a / step) * step                     # numpy rounds ties to even
    q = np.minimum(q, 448.0)
    e2 = np.floor(np.log2(np.maximum(q, 2.0 ** -9)))
    norm = q >= 2.0 ** -6
    m_norm = np.round(q / 2.0 ** e2 * 8.0 - 8.0)
    code = np.where(norm, ((e2 + 7).astype(np.int64) << 3) | m_norm.astype(np.int64),
                    np.round(q / 2.0 ** -9).astype(np.int64))
    code = np.where(q == 0, 0, code)
    return (code | np.where(np.signbit(y) & (q > 0), 0x80, 0)).astype(np.uint8)


def make_qk_fp8(q_bits: np.ndarray, k_bits: np.ndarray):
    """FP8 E4M3 codes of bf16 Q and K with per-tensor power-of-two scales
    that put each tensor's largest magnitude near the top of the format."""
    out = []
    for bits in (q_bits, k_bits):
        amax = float(np.abs(bf16_bits_to_f32(bits)).max()) or 1.0
        scale = 2.0 ** np.ceil(np.log2(amax / 448.0))
        out += [quantize_e4m3(bf16_bits_to_f32(bits), scale), scale]
    return out[0], out[2], out[1], out[3]


def make_workload(cfg: int):
    """(Workload, q, k, v) of one of the five configurations, seed = cfg."""
    w = WORKLOADS[cfg]
    q, k, v = make_qkv(w.B, w.Hq, w.Hkv, w.Sq, w.Sk, w.D, seed=cfg, outliers=w.outliers,
                       sink=w.sink, lognormal_k=w.lognormal_k)
    return w, q, k, v


def sample_rows(w: Workload, every: int = 64, tile: int = 128, heads=None) -> np.ndarray:
    """Deterministic query-row subset for checks at full size: every
    `every`-th row of every (batch, head), plus the last row of each
    `tile`-row query tile (where the causal diagonal ends)."""
    rows = []
    hs = range(w.Hq) if heads is None else heads
    rr = sorted(set(range(0, w.Sq, every)) | set(range(tile - 1, w.Sq, tile)) | {w.Sq - 1})
    rr = np.array(rr, dtype=np.int64)
    for b in range(w.B):
        for h in hs:
            rows.append((b * w.Hq + h) * w.Sq + rr)
    return np.concatenate(rows) if rows else np.zeros(0, np.int64)


def random_scores(rows, cols, seed=0, std=4.0, masked_frac=0.0):
    """fp32 score rows in log2 units for the standalone softmax-block step."""
    g = np.random.Generator(np.random.PCG64(seed + 5000))
    s = (g.standard_normal((rows, cols), dtype=np.float32) * np.float32(std))
    if masked_frac > 0:
        s[g.random((rows, cols)) < masked_frac] = -np.inf
    return s
