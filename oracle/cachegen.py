"""CPU oracle of SqueezeNeRF cache generation -- TEST INFRASTRUCTURE.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this module.  Plain numpy in binary64, written from the paper:

  * Sec. 3.2 / Sec. 3.4: three position networks F_pos^j, j in (xy, yz, zx),
    each an MLP of 6 layers of 256 hidden units on the positional encoding of
    the plane's two coordinates; one direction network F_dir, 4 layers of 128
    units on the encoding of the viewing direction.  The encoding and the
    ReLU hidden activations follow NeRF, as Sec. 3.4 says.
  * Eq. 3: F_pos^j emits (sigma_0, w_sigma, w_u, u_0, w_v, v_0, w_w, w_0), in
    that order (the order of the Sec. 3.2 listing); the cached values are
    sigma^j = sigma_0 w_sigma and k^j = w_k * k_0 (point-wise) for
    k in (u, v, w).
  * Sec. 3.3: the networks are evaluated on the cache grids: n_p vertex-
    aligned nodes per axis over the scene box for each plane (plane j indexed
    [first axis][second axis]), and n_theta x n_phi direction nodes (theta
    from +z over [0, pi], phi = -pi + b 2 pi / n_phi), the layout the
    renderer reads.

Weights are taken as given (binary16 matrices and binary32 biases in the
tests); all arithmetic here is binary64.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple

import numpy as np

# plane j -> (first axis, second axis)
PLANE_AXES = ((0, 1), (1, 2), (2, 0))


def encode(p: np.ndarray, n_freq: int) -> np.ndarray:
    """NeRF positional encoding of the last axis of p (c components):
    [p, sin(2^0 pi p), cos(2^0 pi p), ..., sin(2^(L-1) pi p),
    cos(2^(L-1) pi p)], c (1 + 2L) values."""
    p = np.asarray(p, dtype=np.float64)
    parts = [p]
    for k in range(n_freq):
        a = (2.0 ** k) * math.pi * p
        parts.append(np.sin(a))
        parts.append(np.cos(a))
    return np.concatenate(parts, axis=-1)


def mlp(x: np.ndarray, layers: Sequence[Tuple[np.ndarray, np.ndarray]]) -> np.ndarray:
    """layers = [(W, b), ...] with W [out][in]; ReLU after every layer but
    the last, which is linear."""
    h = np.asarray(x, dtype=np.float64)
    for n, (W, b) in enumerate(layers):
        h = h @ np.asarray(W, dtype=np.float64).T + np.asarray(b, dtype=np.float64)
        if n + 1 < len(layers):
            h = np.maximum(h, 0.0)
    return h


def grid_nodes(n: int, lo: float, hi: float) -> np.ndarray:
    """n vertex-aligned nodes over [lo, hi] (both ends included), computed
    as lo + i (hi - lo) / (n - 1)."""
    return lo + np.arange(n, dtype=np.float64) * ((float(hi) - float(lo)) / (n - 1))


def position_outputs(layers, n_p: int, plane: int, bmin, bmax, n_freq: int = 10) -> np.ndarray:
    """Raw F_pos^j outputs on the plane's grid: [n_p][n_p][2 + 6D]."""
    ra, rb = PLANE_AXES[plane]
    a = grid_nodes(n_p, bmin[ra], bmax[ra])
    b = grid_nodes(n_p, bmin[rb], bmax[rb])
    pts = np.stack(np.meshgrid(a, b, indexing="ij"), axis=-1)      # [n_p][n_p][2]
    return mlp(encode(pts, n_freq), layers)


def position_cache(layers, n_p: int, plane: int, bmin, bmax, D: int,
                   n_freq: int = 10) -> Tuple[np.ndarray, np.ndarray]:
    """Eq. 3 on the F_pos^j outputs: (sigma^j [n_p][n_p], uvw^j
    [n_p][n_p][3D] = u^j, v^j, w^j)."""
    o = position_outputs(layers, n_p, plane, bmin, bmax, n_freq)
    assert o.shape[-1] == 2 + 6 * D
    sigma = o[..., 0] * o[..., 1]
    uvw = []
    for c in range(3):
        w = o[..., 2 + 2 * c * D: 2 + (2 * c + 1) * D]
        k0 = o[..., 2 + (2 * c + 1) * D: 2 + (2 * c + 2) * D]
        uvw.append(w * k0)
    return sigma, np.concatenate(uvw, axis=-1)


def direction_nodes(n_theta: int, n_phi: int) -> np.ndarray:
    """Unit directions of the direction-cache nodes: theta_a = a pi /
    (n_theta - 1) from +z, phi_b = -pi + b 2 pi / n_phi; [n_theta][n_phi][3]."""
    th = np.arange(n_theta, dtype=np.float64) * (math.pi / (n_theta - 1))
    ph = -math.pi + np.arange(n_phi, dtype=np.float64) * (2.0 * math.pi / n_phi)
    T, P = np.meshgrid(th, ph, indexing="ij")
    return np.stack([np.sin(T) * np.cos(P), np.sin(T) * np.sin(P), np.cos(T)], axis=-1)


def direction_cache(layers, n_theta: int, n_phi: int, n_freq: int = 4) -> np.ndarray:
    """beta = F_dir(encoding of the node direction): [n_theta][n_phi][D]."""
    return mlp(encode(direction_nodes(n_theta, n_phi), n_freq), layers)


def caches(pos_layers: List, dir_layers, n_p: int, n_theta: int, n_phi: int, bmin, bmax,
           D: int, pos_freq: int = 10, dir_freq: int = 4):
    """All cache arrays: ([sigma^xy, sigma^yz, sigma^zx], [uvw^xy, ...], beta)."""
    sig, uvw = [], []
    for j in range(3):
        s, u = position_cache(pos_layers[j], n_p, j, bmin, bmax, D, pos_freq)
        sig.append(s)
        uvw.append(u)
    return sig, uvw, direction_cache(dir_layers, n_theta, n_phi, dir_freq)


def position_cache_points(layers, n_p: int, plane: int, bmin, bmax, D: int, ia, ib,
                          n_freq: int = 10) -> Tuple[np.ndarray, np.ndarray]:
    """position_cache at the grid points (ia[n], ib[n]) only: (sigma^j [n],
    uvw^j [n][3D])."""
    ra, rb = PLANE_AXES[plane]
    a = grid_nodes(n_p, bmin[ra], bmax[ra])[np.asarray(ia)]
    b = grid_nodes(n_p, bmin[rb], bmax[rb])[np.asarray(ib)]
    o = mlp(encode(np.stack([a, b], axis=-1), n_freq), layers)
    sigma = o[..., 0] * o[..., 1]
    uvw = [o[..., 2 + 2 * c * D: 2 + (2 * c + 1) * D] * o[..., 2 + (2 * c + 1) * D: 2 + (2 * c + 2) * D]
           for c in range(3)]
    return sigma, np.concatenate(uvw, axis=-1)
