"""Seeded synthetic workloads shared by the GPU prover's tests/benchmark and the
CPU oracle.

This module holds no arithmetic of the proof system: it draws quantised
integer matrices, lays out layer chains (identity links for MLPs, im2col links
for convolutions), zero-pads dimensions to powers of two, and produces the
verifier's random challenges as a stream of uniform field elements.

Challenge stream: xorshift64 with shifts (13, 7, 17) (Marsaglia, "Xorshift
RNGs", J. Stat. Softw. 8(14), 2003) from a nonzero seed; each challenge is
the next 64-bit output reduced mod p = 2^61 - 1 (values below 8 are twice as
likely as the rest, a bias of about 2^-61).  This is the Python side's own
implementation of the published generator; the prover library has its own
(a context created from a seed), and tests compare the two.

Workloads (fixed-point layers of the shapes the paper's experiments use --
a 64x64 matrix product with rounding, an MNIST-sized MLP -- plus larger
shapes; see the module docstring of each builder):
  1  one 64x64x64 layer, entries uniform in [-2^10, 2^10), s = 8, ReLU
  2  MLP 784-256-128-10 at batch 64, N(0, 0.5^2) values quantised with s = 8,
     ReLU on hidden layers
  3  one 1024x1024x1024 layer, uniform int16 entries, s = 12, ReLU
  4  CNN as im2col products, batch 32, 32x32x3 input: conv3x3 3->32,
     2x2 stride-2 conv 32->32, conv3x3 32->64, 2x2 stride-2 conv 64->64,
     FC 4096->10; input U[0,1) and weights N(0, 0.5^2), s = 10, ReLU per layer
  5  X 512x4096 . W1 4096x4096, ReLU, . W2 4096x4096; N(0, 0.5^2), s = 12
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, List, Optional

import numpy as np

FIELD_BITS = 61
MASK61 = (1 << FIELD_BITS) - 1
CHALLENGE_SEED_BASE = 0x9E3779B97F4A7C15
DATA_SEED_BASE = 1000
CHALLENGES_PER_LAYER = 256


def xorshift64_stream(seed: int, count: int) -> np.ndarray:
    """The first `count` challenges of the stream of `seed`: xorshift64(13, 7, 17)
    outputs reduced mod 2^61 - 1."""
    x = seed & 0xFFFFFFFFFFFFFFFF
    if x == 0:
        raise ValueError("xorshift64 seed must be nonzero")
    out = np.empty(count, dtype=np.uint64)
    for i in range(count):
        x ^= (x << 13) & 0xFFFFFFFFFFFFFFFF
        x ^= x >> 7
        x ^= (x << 17) & 0xFFFFFFFFFFFFFFFF
        out[i] = x % MASK61
    return out


def next_pow2(v: int) -> int:
    return 1 if v <= 1 else 1 << (int(v) - 1).bit_length()


def pad2(M: np.ndarray, rows: Optional[int] = None, cols: Optional[int] = None) -> np.ndarray:
    r, c = M.shape
    R = next_pow2(r) if rows is None else rows
    Cc = next_pow2(c) if cols is None else cols
    out = np.zeros((R, Cc), dtype=M.dtype)
    out[:r, :c] = M
    return out


def quantise(x: np.ndarray, f: int) -> np.ndarray:
    """Fixed point with f fractional bits: rint(x 2^f), clipped to int16."""
    return np.clip(np.rint(x * (1 << f)), -32768, 32767).astype(np.int16)


@dataclass
class Layer:
    B: np.ndarray          # int16, (m x k) padded to powers of two
    s: int                 # fractional bits removed by the rescale
    relu: bool
    name: str = ""
    k_real: int = 0        # unpadded output width


@dataclass
class Workload:
    name: str
    X: np.ndarray                              # int16 layer-0 A (padded)
    layers: List[Layer]
    links: List[Optional[Callable]] = field(default_factory=list)  # links[i]: Z_{i-1} -> A_i
    mode: int = 0                              # 0 nearest (Sec. II-A operator), 1 floor
    challenges: np.ndarray = None              # the first draws of the stream of challenge_seed
    challenge_seed: int = 0
    description: str = ""

    def layer_input(self, li: int, Z_prev):
        """A of layer li as a host array: X for the first layer, else the
        link applied to the previous layer's output (host array)."""
        if li == 0:
            return self.X
        link = self.links[li]
        return np.asarray(Z_prev) if link is None else link(np.asarray(Z_prev))

    def link_map(self, li: int) -> np.ndarray:
        """The gather map of layer li's input link (layer li - 1's output Z,
        n' x k', to layer li's A, n x m): an int64 array of n * m source
        indices (row-major into Z) with -1 where A is zero padding."""
        link = self.links[li]
        zr, zc = self.shapes()[li - 1][0], self.layers[li - 1].B.shape[1]
        idx = (np.arange(zr * zc, dtype=np.int64) + 1).reshape(zr, zc)
        return link(idx).reshape(-1) - 1

    def fs_inputs(self):
        """The caller inputs of a non-interactive proof of this workload: the
        transcript's 32-byte domain and one 32-byte public digest per layer
        (synthetic labels; a deployment would bind its model and input)."""
        import hashlib
        domain = hashlib.sha256(("range-arithmetic workload " + self.name).encode()).digest()
        pubs = [hashlib.sha256(f"{self.name} / layer {li}".encode()).digest() for li in range(len(self.layers))]
        return domain, pubs

    def shapes(self):
        out = []
        n = self.X.shape[0]
        for li, L in enumerate(self.layers):
            m, k = L.B.shape
            if li == 0:
                n = self.X.shape[0]
            elif self.links[li] is not None:
                n = self.links[li].rows
            out.append((n, m, k))
        return out


class Im2col:
    """Zero-padded 'same' (pad = kh//2) or strided patch extraction of an
    activation stored as (batch*H*W) x C rows, columns ordered (dy, dx, c),
    then padded to `cols` columns."""

    def __init__(self, batch, H, W, C, kh, kw, stride, pad, cols):
        self.batch, self.H, self.W, self.C = batch, H, W, C
        self.kh, self.kw, self.stride, self.pad, self.cols = kh, kw, stride, pad, cols
        self.Ho = (H + 2 * pad - kh) // stride + 1
        self.Wo = (W + 2 * pad - kw) // stride + 1
        self.rows = batch * self.Ho * self.Wo

    def __call__(self, Z):
        Cz = Z.shape[1]
        act = Z.reshape(self.batch, self.H, self.W, Cz)[..., :self.C]
        p = self.pad
        act = np.pad(act, ((0, 0), (p, p), (p, p), (0, 0)))
        cols = []
        for dy in range(self.kh):
            for dx in range(self.kw):
                cols.append(act[:, dy:dy + self.stride * self.Ho:self.stride,
                                dx:dx + self.stride * self.Wo:self.stride, :])
        patches = np.stack(cols, axis=3).reshape(self.rows, self.kh * self.kw * self.C)
        out = np.zeros((self.rows, self.cols), dtype=Z.dtype)
        out[:, :patches.shape[1]] = patches
        return out


class Flatten:
    """(batch*H*W) x C activation -> batch x (H*W*C) rows, padded columns."""

    def __init__(self, batch, HW, C, cols):
        self.batch, self.HW, self.C, self.cols = batch, HW, C, cols
        self.rows = batch

    def __call__(self, Z):
        a = Z[:, :self.C].reshape(self.batch, self.HW * self.C)
        out = np.zeros((self.batch, self.cols), dtype=Z.dtype)
        out[:, :a.shape[1]] = a
        return out


def _challenges(cfg: int, n_layers: int):
    """(challenges, challenge_seed) of workload cfg: seed CHALLENGE_SEED_BASE + cfg."""
    seed = CHALLENGE_SEED_BASE + cfg
    return xorshift64_stream(seed, CHALLENGES_PER_LAYER * n_layers), seed


def cfg1(seed_off: int = 0, n: int = 64, m: int = 64, k: int = 64) -> Workload:
    """One fixed-point layer, A (n x m), B (m x k) int16 uniform in
    [-2^10, 2^10), s = 8, rescale then ReLU."""
    rng = np.random.default_rng(DATA_SEED_BASE + 1 + seed_off)
    X = rng.integers(-2 ** 10, 2 ** 10, size=(n, m)).astype(np.int16)
    B = rng.integers(-2 ** 10, 2 ** 10, size=(m, k)).astype(np.int16)
    return Workload(f"single-layer {n}x{m}x{k} int16 s=8 relu", pad2(X), [Layer(pad2(B), 8, True, "L1", k)],
                    [None], 0, *_challenges(1 + seed_off, 1))


def mlp(batch: int, widths, f: int, relu_last: bool, cfg: int, std: float = 0.5,
        name: str = "mlp") -> Workload:
    """Dense chain widths[0] -> widths[1] -> ... with N(0, std^2) inputs and
    weights quantised to f fractional bits; ReLU on hidden layers (and on the
    last one if relu_last)."""
    rng = np.random.default_rng(DATA_SEED_BASE + cfg)
    X = pad2(quantise(rng.normal(0.0, std, size=(batch, widths[0])), f))
    layers = []
    for i in range(len(widths) - 1):
        W = quantise(rng.normal(0.0, std, size=(widths[i], widths[i + 1])), f)
        last = i == len(widths) - 2
        layers.append(Layer(pad2(W), f, (not last) or relu_last, f"L{i + 1}", widths[i + 1]))
    return Workload(name, X, layers, [None] * len(layers), 0, *_challenges(cfg, len(layers)))


def cfg2(batch: int = 64) -> Workload:
    """MNIST-shaped MLP 784-256-128-10 at batch 64, f = 8."""
    return mlp(batch, [784, 256, 128, 10], 8, False, 2, name=f"mlp 784-256-128-10 batch {batch} s=8")


def cfg3(n: int = 1024) -> Workload:
    """One n x n x n layer, int16 entries uniform over the full int16 range,
    s = 12, rescale then ReLU."""
    rng = np.random.default_rng(DATA_SEED_BASE + 3)
    X = rng.integers(-2 ** 15, 2 ** 15, size=(n, n)).astype(np.int16)
    B = rng.integers(-2 ** 15, 2 ** 15, size=(n, n)).astype(np.int16)
    return Workload(f"single-layer {n}x{n}x{n} int16 s=12 relu", X, [Layer(B, 12, True, "L1", n)], [None], 0,
                    *_challenges(3, 1))


def cfg4(batch: int = 32, H: int = 32) -> Workload:
    """Small CNN as im2col matrix products: conv3x3 3->32, 2x2/2 conv 32->32,
    conv3x3 32->64, 2x2/2 conv 64->64, FC (H/4)^2*64 -> 10; f = 10; input
    U[0,1), weights N(0, 0.5^2); rescale + ReLU after every layer."""
    f = 10
    rng = np.random.default_rng(DATA_SEED_BASE + 4)
    img = quantise(rng.random(size=(batch * H * H, 3)), f)            # rows (b, y, x), cols c
    first = Im2col(batch, H, H, 3, 3, 3, 1, 1, 32)
    X = first(img.astype(np.int16))

    def w(rows, cols, kpad=None):
        Wm = quantise(rng.normal(0.0, 0.5, size=(rows, cols)), f)
        return pad2(Wm, next_pow2(rows), kpad or next_pow2(cols))

    H2, H4 = H // 2, H // 4
    layers = [Layer(w(27, 32), f, True, "conv1", 32),
              Layer(w(128, 32), f, True, "pool1", 32),
              Layer(w(288, 64), f, True, "conv2", 64),
              Layer(w(256, 64), f, True, "pool2", 64),
              Layer(w(H4 * H4 * 64, 10), f, True, "fc", 10)]
    links = [None,
             Im2col(batch, H, H, 32, 2, 2, 2, 0, 128),
             Im2col(batch, H2, H2, 32, 3, 3, 1, 1, 512),
             Im2col(batch, H2, H2, 64, 2, 2, 2, 0, 256),
             Flatten(batch, H4 * H4, 64, next_pow2(H4 * H4 * 64))]
    return Workload(f"cnn batch {batch} {H}x{H}x3 s=10", X, layers, links, 0, *_challenges(4, len(layers)))


def cfg5(batch: int = 512, d: int = 4096) -> Workload:
    """Transformer-block-shaped MLP: X (batch x d) . W1 (d x d), ReLU, . W2
    (d x d); N(0, 0.5^2) values, f = 12."""
    return mlp(batch, [d, d, d], 12, False, 5, name=f"mlp {d}-{d}-{d} batch {batch} s=12")


FULL = {1: cfg1, 2: cfg2, 3: cfg3, 4: cfg4, 5: cfg5}


def small(cfg: int) -> Workload:
    """Reduced shapes of each workload with the same value distributions,
    sized for the oracle to finish in seconds while spanning several GPU
    tiles and ragged (padded) dimensions."""
    if cfg == 1:
        return cfg1()
    if cfg == 2:
        return cfg2(batch=8)
    if cfg == 3:
        return cfg3(n=128)
    if cfg == 4:
        return cfg4(batch=2, H=8)
    if cfg == 5:
        return cfg5(batch=32, d=256)
    raise ValueError(cfg)


def workload(cfg: int, size: str = "full") -> Workload:
    return FULL[cfg]() if size == "full" else small(cfg)
