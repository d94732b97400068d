"""Single-type block-scaled formats the paper compares IF4 against in
Table 1 (MXFP4, NVINT4, NVFP4 with 4/6).  Test infrastructure: they are used
only to pin the oracle to Table 1's MSE column and never run on the GPU.

Vectorised numpy, fp64 values rounded through the same rules the paper
states: E2M1 elements (Sec. 1), E4M3 group scales with an FP32 tensor scale
(Sec. 3, Eq. 1-2), a UE8M0 power-of-two scale per 32 values for MXFP4
(Sec. 1 / Table 1), and for 4/6 the two scalings to a group maximum of 6 or
4 with the tensor scale max|X|/(6*256) (Sec. 3, list item 2).
"""
from __future__ import annotations

import numpy as np

E2M1 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def _nearest_on_grid(x: np.ndarray, grid: np.ndarray) -> np.ndarray:
    """Nearest grid magnitude to |x| (ties to the even grid index), signed."""
    m = np.abs(x)
    d = np.abs(m[..., None] - grid)
    best = np.argmin(d, axis=-1)
    # ties: argmin returns the lower index; move to the even one if tied
    lower_tied = (best + 1 < len(grid))
    nxt = np.minimum(best + 1, len(grid) - 1)
    tie = lower_tied & (np.take_along_axis(d, nxt[..., None], -1)[..., 0] ==
                        np.take_along_axis(d, best[..., None], -1)[..., 0])
    best = np.where(tie & (best % 2 == 1), nxt, best)
    return np.copysign(grid[best], x)


def _e4m3_values() -> np.ndarray:
    vals = []
    for code in range(127):
        E, M = code >> 3, code & 7
        vals.append(M * 2.0 ** -9 if E == 0 else (1 + M / 8) * 2.0 ** (E - 7))
    return np.array(vals)


E4M3 = _e4m3_values()


def _e4m3_round(x: np.ndarray) -> np.ndarray:
    return np.abs(_nearest_on_grid(np.abs(x), E4M3))


def nvint4_dequant(x: np.ndarray) -> np.ndarray:
    """NVINT4: INT4 (+-7) per group of 16 with an E4M3 scale; max 7*448."""
    g = x.reshape(-1, 16).astype(np.float64)
    alpha = np.float32(np.abs(g).max() / (7 * 448))
    amax_g = np.abs(g).max(axis=1, keepdims=True)
    delta = _e4m3_round(amax_g / (float(alpha) * 7))
    s = float(alpha) * delta
    with np.errstate(divide="ignore", invalid="ignore"):
        q = np.where(s > 0, np.clip(np.rint(g / s), -7, 7), 0)
    return (q * s).reshape(x.shape)


def nvfp4_46_dequant(x: np.ndarray) -> np.ndarray:
    """NVFP4 with Four Over Six: each group scaled to a maximum of 6 or 4,
    whichever gives less squared error; tensor scale max|X|/(6*256)."""
    g = x.reshape(-1, 16).astype(np.float64)
    alpha = float(np.float32(np.abs(g).max() / (6 * 256)))
    amax_g = np.abs(g).max(axis=1, keepdims=True)
    best = None
    best_err = None
    for target in (6.0, 4.0):
        delta = _e4m3_round(amax_g / (alpha * target))
        s = alpha * delta
        with np.errstate(divide="ignore", invalid="ignore"):
            q = np.where(s > 0, _nearest_on_grid(np.where(s > 0, g / s, 0), E2M1), 0)
        deq = q * s
        err = ((deq - g) ** 2).sum(axis=1, keepdims=True)
        if best is None:
            best, best_err = deq, err
        else:
            take = err < best_err
            best = np.where(take, deq, best)
            best_err = np.where(take, err, best_err)
    return best.reshape(x.shape)


def mxfp4_dequant(x: np.ndarray) -> np.ndarray:
    """MXFP4: E2M1 per group of 32 with a power-of-two (UE8M0) scale equal to
    2^(floor(log2 max|X_g|) - 2), 2 being the largest E2M1 exponent."""
    g = x.reshape(-1, 32).astype(np.float64)
    amax_g = np.abs(g).max(axis=1, keepdims=True)
    with np.errstate(divide="ignore"):
        e = np.where(amax_g > 0, np.floor(np.log2(np.where(amax_g > 0, amax_g, 1))) - 2, 0)
    s = 2.0 ** e
    q = _nearest_on_grid(g / s, E2M1)
    return (q * s).reshape(x.shape)
