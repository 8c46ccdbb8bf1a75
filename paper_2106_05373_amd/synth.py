"""Seeded synthetic inputs for the BCPNN layer (shapes of the paper's MNIST and STL-10 runs).

This module is shared by the tests, the benchmark and the CPU oracle's driver.  It holds only
input generation: images, their (x, 1-x) unit encoding, receptive-field masks, per-epoch
shuffles, one-hot labels and the preset layer/workload descriptions.  It contains none of the
method's arithmetic (no support, softmax, trace, weight or plasticity computation).

The paper trains on MNIST (28x28 grey) and STL-10 (96x96x3 colour) (Sec. 4, results); neither
dataset is available here, so these generators reproduce the image shapes, value range [0, 1]
and coarse statistics (sparse strokes on a dark background; smooth colour fields with oriented
class textures) from fixed seeds.  Every array is float32, C-contiguous.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

__all__ = [
    "LayerShape", "Workload", "WORKLOADS", "rng", "encode_pixels", "blob_images",
    "stroke_images", "texture_images", "random_mask", "full_mask", "active_count",
    "epoch_permutation", "one_hot", "dataset",
]


def rng(seed: int) -> np.random.Generator:
    """NumPy PCG64 stream for a seed."""
    return np.random.Generator(np.random.PCG64(int(seed)))


# ----------------------------------------------------------------------------------------
# Layer and workload presets
# ----------------------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class LayerShape:
    in_hcu: int
    in_mcu: int
    out_hcu: int
    out_mcu: int

    @property
    def n_in(self) -> int:
        return self.in_hcu * self.in_mcu

    @property
    def n_out(self) -> int:
        return self.out_hcu * self.out_mcu


@dataclasses.dataclass(frozen=True)
class Workload:
    """A training workload: data generator, hidden layer, schedule and seeds."""
    name: str
    data: str                 # "blobs8" | "strokes28" | "textures96"
    n_train: int
    layer: LayerShape
    batch: int
    alpha: float
    epochs: int
    mask_frac: float          # fraction of input HCUs active per hidden HCU (1.0 = full)
    period: int               # structural-plasticity period in batches (0 = never)
    gain: float = 1.0
    bias_gain: float = 1.0    # k_B of the hidden layer
    seed_data: int = 0
    seed_test: int = 1
    seed_mask: int = 2
    seed_shuffle: int = 3
    seed_noise: int = 4
    init_noise: float = 0.1
    n_test: int = 0
    readout_mcu: int = 0      # classes of a supervised readout layer (0 = none)
    readout_epochs: int = 0
    storage: str = "f32"      # storage format of Pij and W: "f32", "bf16", "m10"
    # the inputs are pixels encoded as complementary pairs (x, 1 - x) (encode_pixels), which a
    # layer may exploit in its joint-trace contraction (bcpnn_config.complement_pairs)
    complement_pairs: bool = True


def _mnist_like(name: str, **kw) -> Workload:
    base = dict(name=name, data="strokes28", n_train=60000,
                layer=LayerShape(784, 2, 30, 100), batch=128, alpha=1e-3, epochs=5,
                mask_frac=0.10, period=100)
    base.update(kw)
    return Workload(**base)


WORKLOADS = {
    # 8x8 blobs, 64 input HCUs of 2 MCUs -> 4 HCUs x 16 MCUs, full mask, no plasticity.
    "tiny": Workload(name="tiny", data="blobs8", n_train=1024, layer=LayerShape(64, 2, 4, 16),
                     batch=32, alpha=0.01, epochs=2, mask_frac=1.0, period=0,
                     seed_data=0, seed_test=0, seed_mask=0, seed_shuffle=0, seed_noise=0),
    # 28x28 strokes -> 30 x 100, 10% receptive fields, plasticity every 100 batches.
    "mnist": _mnist_like("mnist"),
    # the same hidden layer trained for 3 epochs plus a 1 x 10 supervised readout.  Learning
    # settings under which 3 epochs form a hidden code (alpha 1e-3 with k_B = 1 collapses every
    # hidden HCU onto one winning MCU in that time).
    "mnist_pipeline": _mnist_like("mnist_pipeline", epochs=3, n_test=10000, readout_mcu=10,
                                  readout_epochs=1, alpha=1e-2, gain=4.0, bias_gain=0.0),
    # 96x96x3 textures -> 100 x 100, 5% receptive fields, plasticity every 20 batches.
    "stl": Workload(name="stl", data="textures96", n_train=5000,
                    layer=LayerShape(27648, 2, 100, 100), batch=256, alpha=1e-3, epochs=1,
                    mask_frac=0.05, period=20),
    # One GPU's share of the STL-shaped layer sharded by hidden HCU over eight GPUs: 13 of the
    # 100 hidden HCUs against the whole input (the per-shard kernels at their real shape).
    "stl_shard8": Workload(name="stl_shard8", data="textures96", n_train=5000,
                           layer=LayerShape(27648, 2, 13, 100), batch=256, alpha=1e-3, epochs=1,
                           mask_frac=0.05, period=20),
    # MNIST-shaped layer with Pij and W stored in bf16, or with a 10-bit mantissa.
    "mnist_bf16": _mnist_like("mnist_bf16", storage="bf16"),
    "mnist_m10": _mnist_like("mnist_m10", storage="m10"),
}


# ----------------------------------------------------------------------------------------
# Input encoding
# ----------------------------------------------------------------------------------------
def encode_pixels(pixels: np.ndarray) -> np.ndarray:
    """Each pixel value x in [0, 1] becomes an input HCU of two MCUs: unit 2p = x, 2p+1 = 1 - x.

    The paper leaves the input encoding open (it only names N_F input features, Sec. 2); this
    complementary pair makes every input HCU a two-valued discrete variable whose activities sum
    to one, the same normalisation the hidden HCUs get from their softmax.
    """
    x = np.ascontiguousarray(pixels, dtype=np.float32)
    out = np.empty(x.shape[:-1] + (2 * x.shape[-1],), dtype=np.float32)
    out[..., 0::2] = x
    out[..., 1::2] = np.float32(1.0) - x
    return out


# ----------------------------------------------------------------------------------------
# Image generators
# ----------------------------------------------------------------------------------------
def _gauss_kernel1d(sigma: float) -> np.ndarray:
    r = int(np.ceil(3.0 * sigma))
    t = np.arange(-r, r + 1, dtype=np.float64)
    k = np.exp(-0.5 * (t / sigma) ** 2)
    return k / k.sum()


def _blur2d(img: np.ndarray, sigma: float) -> np.ndarray:
    """Separable Gaussian blur with zero padding over the last two axes."""
    k = _gauss_kernel1d(sigma)
    r = len(k) // 2
    pad = [(0, 0)] * (img.ndim - 2) + [(r, r), (r, r)]
    p = np.pad(img.astype(np.float64), pad)
    h, w = img.shape[-2:]
    rows = sum(k[t] * p[..., t:t + h, :] for t in range(len(k)))
    return sum(k[t] * rows[..., :, t:t + w] for t in range(len(k)))


def blob_images(n: int, seed: int = 0, side: int = 8, n_proto: int = 4):
    """8x8 images: 4 Gaussian-blob prototypes (centres U[1,7]^2, sigma U[1,2]) plus U(-0.2, 0.2)
    pixel noise, clipped to [0, 1].  Returns (pixels [n, side*side] float32, labels [n] int64)."""
    g = rng(seed)
    cy, cx = g.uniform(1.0, side - 1.0, size=(2, n_proto))
    sig = g.uniform(1.0, 2.0, size=n_proto)
    yy, xx = np.mgrid[0:side, 0:side].astype(np.float64)
    protos = np.exp(-((yy[None] - cy[:, None, None]) ** 2 + (xx[None] - cx[:, None, None]) ** 2)
                    / (2.0 * sig[:, None, None] ** 2))
    labels = g.integers(0, n_proto, size=n)
    noise = g.uniform(-0.2, 0.2, size=(n, side, side))
    img = np.clip(protos[labels] + noise, 0.0, 1.0)
    return img.reshape(n, side * side).astype(np.float32), labels.astype(np.int64)


def _stroke_prototypes(g: np.random.Generator, n_proto: int = 10, side: int = 28,
                       steps: int = 60) -> np.ndarray:
    disk = np.array([[0.0, 1.0, 0.0], [1.0, 1.0, 1.0], [0.0, 1.0, 0.0]])
    protos = np.zeros((n_proto, side, side))
    for k in range(n_proto):
        img = np.zeros((side + 2, side + 2))
        pos = g.uniform(10.0, 18.0, size=2)
        ang = g.uniform(0.0, 2.0 * np.pi)
        vel = np.array([np.cos(ang), np.sin(ang)])
        for _ in range(steps):
            ang = g.uniform(0.0, 2.0 * np.pi)
            vel = 0.8 * vel + 0.45 * np.array([np.cos(ang), np.sin(ang)])
            vel /= max(np.linalg.norm(vel), 1e-9)
            pos = pos + 0.75 * vel
            for d in range(2):                       # reflect at a 4-pixel border
                if pos[d] < 4.0:
                    pos[d], vel[d] = 8.0 - pos[d], -vel[d]
                if pos[d] > side - 5.0:
                    pos[d], vel[d] = 2.0 * (side - 5.0) - pos[d], -vel[d]
            y, x = int(round(pos[0])) + 1, int(round(pos[1])) + 1
            img[y - 1:y + 2, x - 1:x + 2] = np.maximum(img[y - 1:y + 2, x - 1:x + 2], disk)
        img = _blur2d(img[1:-1, 1:-1], 1.0)
        protos[k] = img / img.max()
    return protos


def stroke_images(n: int, seed: int = 0, proto_seed: int = 0):
    """28x28 MNIST-shaped images.  10 stroke prototypes (a 60-step momentum random walk of
    0.75 px steps from the centre region, stamped with a plus-shaped 3x3 disk, blurred with
    sigma 1, normalised to max 1; about 75% of pixels end up below 0.1, mean 0.13; drawn from
    `proto_seed`, so train and held-out sets share classes).  A sample picks a class, shifts it by
    an integer offset in [-2, 2]^2, scales it by U(0.7, 1.0), adds N(0, 0.05) noise and clips to
    [0, 1].  Returns (pixels [n, 784] float32, labels [n] int64)."""
    protos = _stroke_prototypes(rng(1000 + proto_seed))
    g = rng(seed)
    labels = g.integers(0, 10, size=n)
    shift = g.integers(-2, 3, size=(n, 2))
    scale = g.uniform(0.7, 1.0, size=n)
    noise = g.normal(0.0, 0.05, size=(n, 28, 28))
    img = np.empty((n, 28, 28))
    padded = np.pad(protos, ((0, 0), (2, 2), (2, 2)))
    for dy in range(-2, 3):
        for dx in range(-2, 3):
            sel = np.nonzero((shift[:, 0] == dy) & (shift[:, 1] == dx))[0]
            img[sel] = padded[labels[sel], 2 - dy:30 - dy, 2 - dx:30 - dx]
    img = np.clip(img * scale[:, None, None] + noise, 0.0, 1.0)
    return img.reshape(n, 784).astype(np.float32), labels.astype(np.int64)


def texture_images(n: int, seed: int = 0, proto_seed: int = 0, side: int = 96, chunk: int = 250):
    """96x96x3 STL-10-shaped images (channel-major, pixel p = c*side*side + y*side + x).
    Each image mixes 50/50 a smooth random colour field (white noise blurred with sigma 8 px per
    channel, rescaled to [0.2, 0.8]) with the texture of its class (an oriented grating,
    theta_k = k*pi/10, 2-12 cycles per image, random phase, class tint), adds N(0, 0.02) and
    clips to [0, 1].  Returns (pixels [n, 3*side*side] float32, labels [n] int64)."""
    gp = rng(2000 + proto_seed)
    theta = np.arange(10) * np.pi / 10.0
    cycles = np.linspace(2.0, 12.0, 10)
    tint = gp.uniform(0.5, 1.0, size=(10, 3))
    g = rng(seed)
    labels = g.integers(0, 10, size=n)
    out = np.empty((n, 3, side, side), dtype=np.float32)
    yy, xx = np.mgrid[0:side, 0:side].astype(np.float64) / side
    fy = np.fft.fftfreq(side)[:, None]
    fx = np.fft.rfftfreq(side)[None, :]
    sigma = 8.0
    transfer = np.exp(-2.0 * (np.pi * sigma) ** 2 * (fy ** 2 + fx ** 2))   # periodic blur
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        m = e - s
        white = g.normal(0.0, 1.0, size=(m, 3, side, side))
        field = np.fft.irfft2(np.fft.rfft2(white) * transfer, s=(side, side))
        lo = field.min(axis=(2, 3), keepdims=True)
        hi = field.max(axis=(2, 3), keepdims=True)
        field = 0.2 + 0.6 * (field - lo) / np.maximum(hi - lo, 1e-12)
        lab = labels[s:e]
        phase = g.uniform(0.0, 2.0 * np.pi, size=m)
        arg = (np.cos(theta[lab])[:, None, None] * xx[None] + np.sin(theta[lab])[:, None, None]
               * yy[None]) * cycles[lab][:, None, None] * 2.0 * np.pi + phase[:, None, None]
        grating = 0.5 + 0.5 * np.sin(arg)
        tex = grating[:, None] * tint[lab][:, :, None, None]
        img = 0.5 * field + 0.5 * tex + g.normal(0.0, 0.02, size=(m, 3, side, side))
        out[s:e] = np.clip(img, 0.0, 1.0)
    return out.reshape(n, 3 * side * side), labels.astype(np.int64)


def dataset(w: Workload, split: str = "train", n: Optional[int] = None):
    """Pixels and labels of a workload's train or held-out split (n overrides the size)."""
    seed = w.seed_data if split == "train" else w.seed_test
    if n is None:
        n = w.n_train if split == "train" else w.n_test
    if w.data == "blobs8":
        return blob_images(n, seed=seed)
    if w.data == "strokes28":
        return stroke_images(n, seed=seed, proto_seed=w.seed_data)
    if w.data == "textures96":
        return texture_images(n, seed=seed, proto_seed=w.seed_data)
    raise ValueError(f"unknown data kind {w.data!r}")


# ----------------------------------------------------------------------------------------
# Masks, shuffles, labels
# ----------------------------------------------------------------------------------------
def active_count(in_hcu: int, frac: float) -> int:
    """Active input HCUs per hidden HCU: frac * H_in rounded half up, at least 1."""
    return max(1, min(in_hcu, int(np.floor(frac * in_hcu + 0.5))))


def full_mask(in_hcu: int, out_hcu: int) -> np.ndarray:
    return np.ones((in_hcu, out_hcu), dtype=np.uint8)


def random_mask(in_hcu: int, out_hcu: int, k: int, seed: int) -> np.ndarray:
    """Random initial receptive fields: for each hidden HCU, a partial Fisher-Yates shuffle over
    the H_in input HCUs picks k of them.  Layout [H_in, H_out] uint8 (1 = active)."""
    g = rng(seed)
    mask = np.zeros((in_hcu, out_hcu), dtype=np.uint8)
    for hj in range(out_hcu):
        idx = np.arange(in_hcu)
        for t in range(k):
            r = t + int(g.integers(0, in_hcu - t))
            idx[t], idx[r] = idx[r], idx[t]
        mask[idx[:k], hj] = 1
    return mask


def epoch_permutation(n: int, seed_shuffle: int, epoch: int) -> np.ndarray:
    """Sample order of epoch `epoch` (0-based): a permutation from PCG64(seed_shuffle + epoch)."""
    return rng(seed_shuffle + epoch).permutation(n)


def one_hot(labels: np.ndarray, n_classes: int) -> np.ndarray:
    out = np.zeros((len(labels), n_classes), dtype=np.float32)
    out[np.arange(len(labels)), labels] = 1.0
    return out
