"""Seeded synthetic inputs for packed variable-length video-latent attention.

This module holds no attention arithmetic. It only draws inputs: per-clip token
counts from latent grids (frames x height x width patches, one clip = one
sequence, Section III Observation 2), the pack order, and q/k/v/dout values.
Both the HIP path and the float64 oracle consume what it returns.

Value recipe: every tensor is float32 N(0, 1), rounded to bfloat16 with
round-to-nearest-even. Shapes come from ``numpy.random.default_rng(seed)``:
(1) clip lengths, (2) pack-order permutation. Tensor values come from
``numpy.random.SeedSequence(seed)``: child i of four is q, k, v, dout in that
order, and each tensor's flattened elements are cut into fixed chunks of
2^22 values, chunk c drawn from child c of that tensor's sequence. The result
does not depend on how many threads draw the chunks.
The paper's datasets (WebVid, Koala, internal Lynx) are not available; these
shapes stand in for them.
"""
from __future__ import annotations

import concurrent.futures as cf
import dataclasses
import math
import os

import numpy as np

# Latent grids (frames, height, width) -> tokens, named after what they are.
GRID_5x16x16 = 5 * 16 * 16        # 1,280
GRID_9x24x32 = 9 * 24 * 32        # 6,912
GRID_13x30x52 = 13 * 30 * 52      # 20,280


@dataclasses.dataclass
class Pack:
    """A packed batch: tensors are bf16 bit patterns (uint16) laid out [T, H, D]."""
    name: str
    cu_seqlens: np.ndarray          # int32 [nseq + 1], cu[0] = 0
    heads: int
    head_dim: int
    scale: float
    q: np.ndarray | None = None     # uint16 [T, H, D]
    k: np.ndarray | None = None     # uint16 [Tk, H, D] (Tk = T unless cu_seqlens_k is set)
    v: np.ndarray | None = None
    dout: np.ndarray | None = None
    cu_seqlens_k: np.ndarray | None = None  # key offsets for cross-attention; None: self-attention

    @property
    def nseq(self) -> int:
        return int(self.cu_seqlens.shape[0] - 1)

    @property
    def total_tokens(self) -> int:
        return int(self.cu_seqlens[-1])

    @property
    def lengths(self) -> np.ndarray:
        return np.diff(self.cu_seqlens).astype(np.int64)

    @property
    def sum_sq_len(self) -> int:
        return int(np.sum(self.lengths ** 2))

    @property
    def lengths_k(self) -> np.ndarray:
        cu = self.cu_seqlens if self.cu_seqlens_k is None else self.cu_seqlens_k
        return np.diff(cu).astype(np.int64)

    @property
    def total_tokens_k(self) -> int:
        cu = self.cu_seqlens if self.cu_seqlens_k is None else self.cu_seqlens_k
        return int(cu[-1])

    @property
    def sum_qk(self) -> int:
        """sum over sequences of Lq * Lk: the score-matrix entries per head (sum L^2 for self-attention)."""
        return int(np.sum(self.lengths * self.lengths_k))

    def f32(self, name: str) -> np.ndarray:
        """The bf16 values of tensor ``name`` widened exactly to float32."""
        return bf16_bits_to_f32(getattr(self, name))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round-to-nearest-even), returning uint16 bits.

    Inputs are finite, so the 32-bit sum below cannot overflow.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def cu_from_lengths(lengths) -> np.ndarray:
    lengths = np.asarray(lengths, dtype=np.int64)
    cu = np.zeros(lengths.shape[0] + 1, dtype=np.int64)
    np.cumsum(lengths, out=cu[1:])
    if cu[-1] >= 2 ** 31:
        raise ValueError("total tokens exceed int32")
    return cu.astype(np.int32)


CHUNK = 1 << 22
_THREADS = min(16, os.cpu_count() or 1)


def _draw_tensor(ss: np.random.SeedSequence, shape) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16)
    nchunks = (n + CHUNK - 1) // CHUNK
    children = ss.spawn(nchunks)

    def fill(c):
        a, b = c * CHUNK, min(n, (c + 1) * CHUNK)
        x = np.random.default_rng(children[c]).standard_normal(b - a, dtype=np.float32)
        out[a:b] = f32_to_bf16_bits(x)

    if nchunks <= 1:
        for c in range(nchunks):
            fill(c)
    else:
        with cf.ThreadPoolExecutor(_THREADS) as ex:
            list(ex.map(fill, range(nchunks)))
    return out.reshape(shape)


def _draw_tensors(seed: int, shape):
    """q, k, v, dout for ``shape``: four independent streams of the seed."""
    return [_draw_tensor(ss, shape) for ss in np.random.SeedSequence(seed).spawn(4)]


WORKLOADS = ("tiny", "uniform", "hetero", "long", "skew", "cross")

DESCRIPTIONS = {
    "tiny": "2 clips (4x8x8=256, 6x8x8=384 tokens), 2 heads x 64",
    "uniform": "8 clips x 4,096 tokens (16x16x16), 24 heads x 128",
    "hetero": "16 clips drawn from {5x16x16=1,280 p.5; 9x24x32=6,912 p.35; 13x30x52=20,280 p.15}, shuffled, 24 heads x 128",
    "long": "1 clip of 75,600 tokens (21x45x80), 24 heads x 128",
    "skew": "1 clip of 100,800 tokens (28x60x60) + 64 images of 1,024 tokens (1x32x32), shuffled, 40 heads x 128",
    "cross": "cross-attention: the 16 video clips of the heterogeneous mix as queries, each against 32-256 text "
             "tokens as keys, 12 heads x 128 (Wan2.1 1.3B)",
}


def workload_shape(name: str, seed: int = 0):
    """Lengths, heads and head_dim of a named workload, consuming the rng like make_workload."""
    rng = np.random.default_rng(seed)
    if name == "tiny":
        lengths, H, D = [4 * 8 * 8, 6 * 8 * 8], 2, 64
    elif name == "uniform":
        lengths, H, D = [16 * 16 * 16] * 8, 24, 128
    elif name == "hetero":
        grid = np.array([GRID_5x16x16, GRID_9x24x32, GRID_13x30x52])
        idx = rng.choice(3, size=16, p=[0.5, 0.35, 0.15])
        lengths = grid[idx][rng.permutation(16)].tolist()
        H, D = 24, 128
    elif name == "long":
        lengths, H, D = [21 * 45 * 80], 24, 128
    elif name == "skew":
        base = np.array([28 * 60 * 60] + [1 * 32 * 32] * 64)
        lengths = base[rng.permutation(base.shape[0])].tolist()
        H, D = 40, 128
    elif name == "cross":
        # Query (video) lengths: the heterogeneous mix's draws; the returned rng then draws the
        # key (text) lengths (cross_text_lengths).
        rng, lengths, _, _ = workload_shape("hetero", seed)
        H, D = 12, 128
    else:
        raise KeyError(f"unknown workload {name!r}; known: {WORKLOADS}")
    return rng, lengths, H, D


def cross_text_lengths(rng, nseq: int) -> list:
    """Text token counts of a cross-attention pack: uniform in [32, 256] (text sequences are
    short, typically under 256 tokens: Section IV-B footnote)."""
    return rng.integers(32, 257, size=nseq).tolist()


def make_workload(name: str, seed: int = 0, tensors: bool = True) -> Pack:
    """One of the named workloads, drawn from ``seed``."""
    rng, lengths, H, D = workload_shape(name, seed)
    if name == "cross":
        return make_pack_qk(lengths, cross_text_lengths(rng, len(lengths)), H, D, seed=seed, name=name,
                            tensors=tensors)
    cu = cu_from_lengths(lengths)
    pack = Pack(name=name, cu_seqlens=cu, heads=H, head_dim=D, scale=1.0 / math.sqrt(D))
    if tensors:
        pack.q, pack.k, pack.v, pack.dout = _draw_tensors(seed, (int(cu[-1]), H, D))
    return pack


def make_pack(lengths, heads: int, head_dim: int, seed: int = 0, scale: float | None = None,
              name: str = "custom") -> Pack:
    """A pack with explicit clip lengths (zero-length clips allowed), drawn from ``seed``."""
    cu = cu_from_lengths(lengths)
    sc = 1.0 / math.sqrt(head_dim) if scale is None else float(scale)
    pack = Pack(name=name, cu_seqlens=cu, heads=heads, head_dim=head_dim, scale=sc)
    pack.q, pack.k, pack.v, pack.dout = _draw_tensors(seed, (int(cu[-1]), heads, head_dim))
    return pack


def make_pack_qk(lengths_q, lengths_k, heads: int, head_dim: int, seed: int = 0, scale: float | None = None,
                 name: str = "cross", tensors: bool = True) -> Pack:
    """A cross-attention pack: sequence s has lengths_q[s] queries and lengths_k[s] keys.
    q and dout have Tq rows, k and v Tk rows; the four tensors come from the same four
    streams of the seed as in make_pack (q, k, v, dout)."""
    cuq, cuk = cu_from_lengths(lengths_q), cu_from_lengths(lengths_k)
    sc = 1.0 / math.sqrt(head_dim) if scale is None else float(scale)
    pack = Pack(name=name, cu_seqlens=cuq, heads=heads, head_dim=head_dim, scale=sc, cu_seqlens_k=cuk)
    if tensors:
        ss = np.random.SeedSequence(seed).spawn(4)
        tq, tk = int(cuq[-1]), int(cuk[-1])
        pack.q = _draw_tensor(ss[0], (tq, heads, head_dim))
        pack.k = _draw_tensor(ss[1], (tk, heads, head_dim))
        pack.v = _draw_tensor(ss[2], (tk, heads, head_dim))
        pack.dout = _draw_tensor(ss[3], (tq, heads, head_dim))
    return pack


def attention_flops(pack: Pack) -> dict:
    """FLOP conventions for bidirectional attention over the pack (per sequence Lq * Lk work;
    L^2 for self-attention)."""
    base = pack.heads * pack.head_dim * pack.sum_qk
    return {"fwd": 4 * base, "bwd": 10 * base, "fwd_bwd": 14 * base,
            "no_recompute": 12 * base, "executed": 18 * base}
