"""Seeded synthetic inputs for the SLA library's tests and benchmark.

This module only draws inputs: window geometry (per-voxel window ids or CSR
offsets) and i.i.d. normal values rounded to the storage type.  It holds none of
the attention arithmetic, and both the CPU oracle side and the HIP side of the
tests read the same arrays from it.

The paper evaluates on the Waymo Open Dataset and nuScenes, neither of which is
available here; the generators stand in for them with LiDAR-shaped synthetic
scenes: 0.32 m pillars on a 468 x 468 grid cut into 12 x 12 windows (the Waymo
voxel and window sizes of Sec. 4.2), 4 heads over 128 channels (Sec. 4.2), and
occupancy that falls off as 1/range from the sensor.

Storage types: "f32" -> numpy float32, "f16" -> numpy float16, "bf16" -> numpy
uint16 holding bfloat16 bit patterns (round-to-nearest-even from float32).
"""
from __future__ import annotations

import math

import numpy as np

GRID = 468          # pillar grid side (cells)
WIN = 12            # window side (cells)
WIN_PER_SIDE = GRID // WIN   # 39
FRAME_WINDOWS = WIN_PER_SIDE * WIN_PER_SIDE   # 1,521 window slots per frame
FRAME_TARGET_N = 60_000

CONFIG_NAMES = {
    1: "tiny: 64 windows, lengths U{1..60}, CSR input, H=2 d=32, f32",
    2: "waymo-like frame: 468x468 grid, 12x12 windows, ~60k pillars, H=4 d=32, f16",
    3: "large sparse frame: 4,096 log-normal windows (median 20, 1..1024), ~200k, H=8 d=16, bf16",
    4: "4 waymo-like frames as one sequence, ~240k, H=8 d=32, bf16",
    5: "training step on waymo-like frame shapes (build+fwd+bwd), ~60k, H=4 d=32, f16",
}


# ----------------------------------------------------------------- value rounding
def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns, round-to-nearest-even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + rounding) >> np.uint32(16)).astype(np.uint16)


def cast_values(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float32 values to the storage type (round-to-nearest-even)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "f32":
        return x
    if dtype == "f16":
        return x.astype(np.float16)
    if dtype == "bf16":
        return to_bf16_bits(x)
    raise ValueError(f"unknown dtype {dtype!r}")


def normal_values(rng: np.random.Generator, n: int, heads: int, head_dim: int, dtype: str):
    """i.i.d. N(0, 1) values [n, heads, head_dim], drawn in float32 then rounded."""
    return cast_values(rng.standard_normal((n, heads, head_dim), dtype=np.float32), dtype)


# ---------------------------------------------------------------------- geometry
def _occupancy_prob(c: float, r: np.ndarray) -> np.ndarray:
    return np.where(r <= GRID / 2, np.minimum(1.0, c / r), 0.0)


def _cell_ranges() -> np.ndarray:
    ys, xs = np.mgrid[0:GRID, 0:GRID]
    cx = xs + 0.5 - GRID / 2
    cy = ys + 0.5 - GRID / 2
    return np.sqrt(cx * cx + cy * cy)


def _solve_density(target: float, r: np.ndarray) -> float:
    lo, hi = 0.0, float(GRID)
    for _ in range(100):
        mid = 0.5 * (lo + hi)
        if _occupancy_prob(mid, r).sum() < target:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


_R = None
_C = None


def waymo_like_pillars(rng: np.random.Generator):
    """(x, y) cell coordinates of the occupied pillars of one synthetic frame, in
    raster order (y major).

    A cell at range r (cells) from the grid centre is occupied with probability
    min(1, c / r) inside the sensor range (r <= 234 cells), 0 beyond; c is set so
    that the expected number of pillars is 60,000.
    """
    global _R, _C
    if _R is None:
        _R = _cell_ranges()
        _C = _solve_density(FRAME_TARGET_N, _R)
    occ = rng.random((GRID, GRID)) < _occupancy_prob(_C, _R)
    y, x = np.nonzero(occ)
    return x.astype(np.int32), y.astype(np.int32)


def window_ids(x: np.ndarray, y: np.ndarray) -> np.ndarray:
    """Window id of a cell: (y // 12) * 39 + x // 12."""
    return ((y // WIN) * WIN_PER_SIDE + x // WIN).astype(np.int32)


def waymo_like_ids(rng: np.random.Generator) -> np.ndarray:
    """Window id of each occupied pillar of one synthetic frame, in raster order
    (not window-sorted)."""
    x, y = waymo_like_pillars(rng)
    return window_ids(x, y)


def make_cwi_frame(seed=0, channels: int = 128, taps: int = 13, dtype: str = "f16") -> dict:
    """One Waymo-like pillar frame for the cross-window interaction: coordinates
    (x, y, 0) on the 468 x 468 grid, window ids, features x [n, channels] ~ N(0, 1),
    and depthwise weights for the two axis branches (taps x channels / 4) and the
    3 x 3 x 3 branch (27 x channels / 4), ~ N(0, 1 / taps).  Geometry seed
    [6, 0, seed], values [6, 1, seed]."""
    geo = np.random.default_rng([6, 0, seed])
    val = np.random.default_rng([6, 1, seed])
    x, y = waymo_like_pillars(geo)
    n, c = x.size, channels // 4
    coords = np.stack([x, y, np.zeros_like(x)], axis=1).astype(np.int32)
    feats = cast_values(val.standard_normal((n, channels), dtype=np.float32), dtype)
    w = lambda k: cast_values((val.standard_normal((k, c)) / np.sqrt(k)).astype(np.float32), dtype)  # noqa: E731
    return {"name": f"waymo-like pillar frame for CWI: 468x468 grid, ~60k pillars, C={channels}, "
                    f"{taps}-tap axis kernels, {dtype}",
            "n": n, "grid": (GRID, GRID, 1), "coords": coords, "ids": window_ids(x, y),
            "num_windows": FRAME_WINDOWS, "channels": channels, "taps": taps, "dtype": dtype,
            "x": feats, "w_x": w(taps), "w_y": w(taps), "w_3": w(27)}


def _lognormal_round_clip_mean(mu: float, sigma: float, lo: int, hi: int) -> float:
    def cdf(x):
        return 0.5 * (1.0 + math.erf((math.log(x) - mu) / (sigma * math.sqrt(2.0))))

    mean = 0.0
    prev = 0.0
    for m in range(lo, hi):
        c = cdf(m + 0.5)
        mean += m * (c - prev)
        prev = c
    mean += hi * (1.0 - prev)
    return mean


def lognormal_lengths(rng: np.random.Generator, windows: int = 4096, target_n: int = 200_000,
                      median: float = 20.0, max_len: int = 1024, singleton_frac: float = 0.05):
    """Window lengths: 5% forced to 1, the rest round(LogNormal(ln median, sigma))
    clipped to [1, max_len], sigma chosen so that the expected total is target_n."""
    n1 = int(round(singleton_frac * windows))
    rest = windows - n1
    mu = math.log(median)
    need = (target_n - n1) / rest
    lo, hi = 0.05, 4.0
    for _ in range(80):
        mid = 0.5 * (lo + hi)
        if _lognormal_round_clip_mean(mu, mid, 1, max_len) < need:
            lo = mid
        else:
            hi = mid
    sigma = 0.5 * (lo + hi)
    lengths = np.clip(np.rint(rng.lognormal(mu, sigma, size=windows)), 1, max_len).astype(np.int64)
    ones = rng.choice(windows, size=n1, replace=False)
    lengths[ones] = 1
    return lengths, sigma


def ids_from_lengths(lengths: np.ndarray, rng: np.random.Generator | None = None) -> np.ndarray:
    """Per-row window ids for the given window lengths; rows shuffled if rng given."""
    ids = np.repeat(np.arange(len(lengths), dtype=np.int32), np.asarray(lengths, dtype=np.int64))
    if rng is not None:
        ids = ids[rng.permutation(ids.size)]
    return ids.astype(np.int32)


def offsets_from_lengths(lengths: np.ndarray) -> np.ndarray:
    off = np.zeros(len(lengths) + 1, dtype=np.int64)
    off[1:] = np.cumsum(lengths)
    return off.astype(np.int32)


# ----------------------------------------------------------------------- configs
def make_config(cfg: int, with_grad: bool | None = None) -> dict:
    """The five synthetic workloads.  Seeds: geometry default_rng([cfg, 0]),
    values default_rng([cfg, 1]); config 4 draws frame f's geometry from
    default_rng([4, 0, f])."""
    geo = np.random.default_rng([cfg, 0])
    val = np.random.default_rng([cfg, 1])
    out = {"cfg": cfg, "name": CONFIG_NAMES[cfg], "ids": None, "offsets": None}
    if cfg == 1:
        lengths = geo.integers(1, 61, size=64)
        out.update(heads=2, head_dim=32, dtype="f32", num_windows=64,
                   offsets=offsets_from_lengths(lengths))
        n = int(lengths.sum())
    elif cfg in (2, 5):
        ids = waymo_like_ids(geo)
        out.update(heads=4, head_dim=32, dtype="f16", num_windows=FRAME_WINDOWS, ids=ids)
        n = ids.size
    elif cfg == 3:
        lengths, _ = lognormal_lengths(geo)
        ids = ids_from_lengths(lengths, geo)
        out.update(heads=8, head_dim=16, dtype="bf16", num_windows=lengths.size, ids=ids)
        n = ids.size
    elif cfg == 4:
        frames = [waymo_like_ids(np.random.default_rng([4, 0, f])) + f * FRAME_WINDOWS
                  for f in range(4)]
        ids = np.concatenate(frames).astype(np.int32)
        out.update(heads=8, head_dim=32, dtype="bf16", num_windows=4 * FRAME_WINDOWS, ids=ids,
                   frames=4)
        n = ids.size
    else:
        raise ValueError(f"unknown config {cfg}")
    H, d, dt = out["heads"], out["head_dim"], out["dtype"]
    out["n"] = n
    out["q"] = normal_values(val, n, H, d, dt)
    out["k"] = normal_values(val, n, H, d, dt)
    out["v"] = normal_values(val, n, H, d, dt)
    if with_grad is None:
        with_grad = cfg == 5
    out["dout"] = normal_values(val, n, H, d, dt) if with_grad else None
    out.setdefault("frames", 1)
    return out


def shuffled(wl: dict, seed) -> dict:
    """Same workload with its rows in a fresh random order (config 5 re-shuffles
    every iteration with default_rng([5, 2, iteration]))."""
    rng = np.random.default_rng(seed)
    p = rng.permutation(wl["n"])
    out = dict(wl)
    out["ids"] = np.ascontiguousarray(wl["ids"][p])
    for key in ("q", "k", "v", "dout"):
        if wl.get(key) is not None:
            out[key] = np.ascontiguousarray(wl[key][p])
    return out
