"""Seeded synthetic workloads shared by the HIP path, its tests and the oracle.

This module holds inputs only: layer lists of the evaluated nets, images,
labels and initial weights.  It contains none of the method's arithmetic
(no forward pass, no gradient); both the oracle and the GPU library receive
the bytes produced here.

Net layer lists (kind, maps, kernel), kinds CONV=1, MAXPOOL=2, FC=3:
  small, medium  Table I (Section IV-A) small and medium architectures.
  large          conv20 k4 -> max2 -> conv60 k3 -> conv100 k6 -> max2 ->
                 FC150 -> FC10; the large net used for the throughput figure
                 (363,960 parameters).
  large_table1   Table I large architecture.  Its last pooling row prints
                 "map 2x2, kernel 3x3" while the following FC layer has
                 150*(900+1) weights; 900 = 100*3*3 so the map is 3x3 and the
                 kernel 2x2 (6/2 = 3).  The 1x1 max-pool row is kept.

Images stand in for MNIST (60,000 train / 10,000 test images padded to 29x29,
Section IV-A): every pixel is U[0,1) and is independently set to zero with
probability 0.8 (MNIST digits are mostly background).
"""
from __future__ import annotations

import numpy as np

CONV, MAXPOOL, FC = 1, 2, 3
IN_H = IN_W = 29
N_CLASSES = 10

NETS = {
    "small": [(CONV, 5, 4), (MAXPOOL, 0, 2), (CONV, 10, 5), (MAXPOOL, 0, 3),
              (FC, 50, 0), (FC, 10, 0)],
    "medium": [(CONV, 20, 4), (MAXPOOL, 0, 2), (CONV, 40, 5), (MAXPOOL, 0, 3),
               (FC, 150, 0), (FC, 10, 0)],
    "large": [(CONV, 20, 4), (MAXPOOL, 0, 2), (CONV, 60, 3), (CONV, 100, 6),
              (MAXPOOL, 0, 2), (FC, 150, 0), (FC, 10, 0)],
    "large_table1": [(CONV, 20, 4), (MAXPOOL, 0, 1), (CONV, 60, 5), (MAXPOOL, 0, 2),
                     (CONV, 100, 6), (MAXPOOL, 0, 2), (FC, 150, 0), (FC, 10, 0)],
}

# Seeds of the standard workloads.
SEED_TINY = 0        # 1,000-sample correctness run, uniform labels
SEED_TRAIN = 1       # 60,000-sample training set
SEED_PROJ = 2        # random projection that defines the learnable labels
SEED_TEST = 3        # 10,000-sample test set
SEED_BATCH = 4       # 16,384-sample frozen-weight gradient batch
SEED_INIT = 5        # initial weights


def layer_fan_in(layers, in_h: int = IN_H, in_w: int = IN_W):
    """Per layer: (fan_in, n_weights, n_bias) for weighted layers, None for pools.

    Bookkeeping for the initial-weight draw only: conv(M, k) on C input maps
    has fan-in C*k*k, FC(N) on a flattened input of size S has fan-in S.
    """
    c, h, w = 1, in_h, in_w
    out = []
    for kind, maps, k in layers:
        if kind == CONV:
            out.append((c * k * k, maps * c * k * k, maps))
            c, h, w = maps, h - k + 1, w - k + 1
        elif kind == MAXPOOL:
            out.append(None)
            h, w = h // k, w // k
        elif kind == FC:
            s = c * h * w
            out.append((s, maps * s, maps))
            c, h, w = maps, 1, 1
        else:
            raise ValueError(f"unknown layer kind {kind}")
    return out


def init_params(layers, seed: int = SEED_INIT, in_h: int = IN_H, in_w: int = IN_W) -> np.ndarray:
    """Initial weights in the canonical layout, fp32.

    Layers are concatenated in order; conv: W[o][i][u][v] then b[o]; FC:
    W[j][i] then b[j].  Every weight and bias is U(-1/sqrt(fan_in),
    +1/sqrt(fan_in)), drawn layer by layer from one PCG64 stream.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    parts = []
    for entry in layer_fan_in(layers, in_h, in_w):
        if entry is None:
            continue
        fan_in, nw, nb = entry
        bound = 1.0 / np.sqrt(fan_in)
        parts.append(rng.uniform(-bound, bound, size=nw + nb))
    return np.concatenate(parts).astype(np.float32)


def images(n: int, seed: int, hw: int = IN_H * IN_W) -> np.ndarray:
    """n images of hw pixels, fp32: U[0,1) with each pixel zeroed with p=0.8."""
    rng = np.random.Generator(np.random.PCG64(seed))
    x = rng.random((n, hw), dtype=np.float32)
    keep = rng.random((n, hw), dtype=np.float32) >= 0.8
    return np.where(keep, x, np.float32(0.0)).astype(np.float32)


def uniform_labels(n: int, seed: int) -> np.ndarray:
    """Labels uniform over 0..9 (independent of the pixels), int32."""
    rng = np.random.Generator(np.random.PCG64(seed + 1000))
    return rng.integers(0, N_CLASSES, size=n).astype(np.int32)


def projection_matrix(seed: int = SEED_PROJ, grid: int = 4, hw: int = IN_H) -> np.ndarray:
    """Seeded random linear projection P [10 x hw*hw] that is constant over a
    grid x grid partition of the image into cells of about 7x7 pixels.

    P[k] takes one N(0,1) value per cell.  A spatially smooth projection keeps
    the task learnable by pooled CNN features; a projection with an independent
    weight per pixel is barely learnable by these nets.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    coarse = rng.standard_normal((N_CLASSES, grid, grid))
    cell = (np.arange(hw) * grid) // hw
    return coarse[:, cell[:, None], cell[None, :]].reshape(N_CLASSES, hw * hw)


def projection_labels(x: np.ndarray, seed: int = SEED_PROJ) -> np.ndarray:
    """Learnable labels: argmax_k (P (x - 0.1))_k for the projection above.

    Centering by the pixel mean 0.1 keeps the classes roughly balanced.
    Ties (probability zero) go to the lowest index.
    """
    p = projection_matrix(seed, hw=int(round(np.sqrt(x.shape[1]))))
    scores = (x.astype(np.float64) - 0.1) @ p.T
    return np.argmax(scores, axis=1).astype(np.int32)


def tiny_set(n: int = 1000):
    """The 1,000-sample sequential correctness run (uniform labels)."""
    return images(n, SEED_TINY), uniform_labels(n, SEED_TINY)


def train_set(n: int = 60000):
    x = images(n, SEED_TRAIN)
    return x, projection_labels(x)


def test_set(n: int = 10000):
    x = images(n, SEED_TEST)
    return x, projection_labels(x)


def batch_set(n: int = 16384):
    x = images(n, SEED_BATCH)
    return x, projection_labels(x)
