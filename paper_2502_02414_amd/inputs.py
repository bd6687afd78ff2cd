"""Seeded synthetic inputs for one Physics-Attention layer.

This module only draws numbers: point clouds, features, weights, Gumbel
samples and upstream gradients.  It holds none of the layer's arithmetic, so
the HIP path and the CPU oracle can both be fed from it without sharing any
of the method.  The paper's datasets (standard PDE benchmarks, DrivAerNet++,
AirCraft; Section 5 and Table 1) are not available, so each workload is a
synthetic stand-in with the same point count, channel count, slice count and
a value distribution of the same kind (grid coordinates, or random Fourier
features of surface points and normals).

Randomness is counter-based: draw k of stream s under seed q is
``mix(key(q, s) + (k + 1) * GAMMA)`` with ``mix`` the SplitMix64 finaliser
(Steele, Lea, Flood, "Fast splittable pseudorandom number generators",
OOPSLA 2014), so any slice of any array can be regenerated on its own.
Streams: 0 geometry and x, 1 weights, 2 Gumbel uniforms, 3 upstream gradient,
4 random-Fourier-feature matrix.  Configuration k uses seed 20250204 + k.

All floating outputs are float32 arrays.  For bf16 workloads the point-side
tensors (x, G, dY) and the slice projection (A, a) are rounded once, to
nearest even, to bf16-representable values, so the float32 arrays hold
exactly what a bf16 device buffer holds.
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional

import numpy as np

GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

STREAM_GEOM, STREAM_WEIGHTS, STREAM_GUMBEL, STREAM_GRAD, STREAM_RFF = range(5)
BASE_SEED = 20250204
CHUNK = 1 << 22  # draws per vectorised block (bounds host memory)


def _mix(z: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def _key(seed: int, stream: int) -> np.uint64:
    s = np.array([(seed * 0x100000001B3 + stream * 0x9E37) & 0xFFFFFFFFFFFFFFFF],
                 dtype=np.uint64)
    return _mix(s + GAMMA)[0]


def raw64(seed: int, stream: int, start: int, count: int) -> np.ndarray:
    """Draws start .. start+count-1 of a stream as uint64."""
    k = _key(seed, stream)
    idx = np.arange(start + 1, start + count + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        return _mix(k + idx * GAMMA)


def uniform(seed: int, stream: int, start: int, count: int) -> np.ndarray:
    """float64 in (0, 1): (24-bit draw + 1/2) / 2^24, never 0 or 1."""
    r = raw64(seed, stream, start, count)
    return ((r >> np.uint64(40)).astype(np.float64) + 0.5) * (1.0 / (1 << 24))


def _blocks(count: int, fn, chunk: int = CHUNK) -> None:
    """Run fn(s, n) over [0, count) in blocks of ``chunk`` on a few threads
    (numpy releases the GIL); the values do not depend on the thread count."""
    spans = [(s, min(chunk, count - s)) for s in range(0, count, chunk)]
    if len(spans) <= 1:
        for s, n in spans:
            fn(s, n)
        return
    workers = max(1, min(16, os.cpu_count() or 1, len(spans)))
    with ThreadPoolExecutor(workers) as ex:
        list(ex.map(lambda sn: fn(*sn), spans))


def normal(seed: int, stream: int, start: int, count: int,
           dtype=np.float64) -> np.ndarray:
    """N(0,1) (computed in float64), Box-Muller on the two 24-bit halves of each draw."""
    out = np.empty(count, dtype=dtype)

    def blk(s, n):
        r = raw64(seed, stream, start + s, n)
        u1 = ((r >> np.uint64(40)).astype(np.float64) + 0.5) * (1.0 / (1 << 24))
        u2 = (((r >> np.uint64(8)) & np.uint64(0xFFFFFF)).astype(np.float64) + 0.5) * (
            1.0 / (1 << 24))
        out[s:s + n] = np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * math.pi * u2)

    _blocks(count, blk)
    return out


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); float32 result."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    flat = a.reshape(-1)
    out = np.empty_like(flat)
    ou = out.view(np.uint32)

    def blk(s, n):
        u = flat[s:s + n].view(np.uint32)
        with np.errstate(over="ignore"):
            r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(
                0xFFFF0000)
        nan = np.isnan(flat[s:s + n])
        ou[s:s + n] = np.where(nan, np.uint32(0x7FC00000), r)

    _blocks(flat.size, blk)
    return out.reshape(a.shape)


def gumbel(seed: int, N: int, M: int, start_point: int = 0) -> np.ndarray:
    """Gumbel(0,1) samples g = -log(-log U), U ~ Uniform(1e-6, 1), shape [N,M] float64."""
    out = np.empty(N * M, dtype=np.float64)

    def blk(s, n):
        u = uniform(seed, STREAM_GUMBEL, start_point * M + s, n)
        U = 1e-6 + (1.0 - 1e-6) * u
        out[s:s + n] = -np.log(-np.log(U))

    _blocks(N * M, blk)
    return out.reshape(N, M)


def xavier_uniform(seed: int, start: int, fan_in: int, fan_out: int,
                   shape) -> np.ndarray:
    bound = math.sqrt(6.0 / (fan_in + fan_out))
    n = int(np.prod(shape))
    u = uniform(seed, STREAM_WEIGHTS, start, n)
    return ((2.0 * u - 1.0) * bound).reshape(shape)


# --------------------------------------------------------------------------
# Point clouds
# --------------------------------------------------------------------------

def _unit_dirs(seed: int, start: int, n: int) -> np.ndarray:
    g = normal(seed, STREAM_GEOM, start, 3 * n).reshape(n, 3)
    return g / np.linalg.norm(g, axis=1, keepdims=True)


def ellipsoid_points(seed: int, N: int, axes=(4.0, 1.8, 1.4), radial_noise=0.02):
    """Area-uniform points on an ellipsoid with the given semi-axes (metres).

    Directions uniform on the unit sphere are mapped by diag(axes) and kept
    with probability proportional to the area element of that map; each kept
    point is scaled radially by (1 + radial_noise * xi), xi ~ N(0,1).
    """
    a, b, c = axes
    gmax = max(b * c, a * c, a * b)
    pts, start = [], 0
    have = 0
    while have < N:
        n = 2 * (N - have) + 1024
        d = _unit_dirs(seed, start, n)
        acc = uniform(seed, STREAM_GEOM, (1 << 40) + start, n)
        gel = np.sqrt((b * c * d[:, 0]) ** 2 + (a * c * d[:, 1]) ** 2 + (a * b * d[:, 2]) ** 2)
        keep = acc * gmax < gel
        p = d[keep] * np.array(axes)
        pts.append(p)
        have += len(p)
        start += n
    p = np.concatenate(pts)[:N]
    xi = normal(seed, STREAM_GEOM, 1 << 41, N)
    return p * (1.0 + radial_noise * xi)[:, None]


# Car-like closed surface: body, cabin and underbody superellipsoids
# |x/a|^3 + |y/b|^3 + |z/c|^3 = 1 with these centres and semi-axes (metres).
CAR_PARTS = (
    ((0.0, 0.0, 0.55), (2.30, 0.95, 0.40)),   # body
    ((-0.25, 0.0, 1.05), (1.20, 0.80, 0.35)),  # cabin
    ((0.0, 0.0, 0.25), (2.00, 0.85, 0.18)),   # underbody
)


def _superellipsoid_F(p, axes, e=3.0):
    return np.sum(np.abs(p / np.asarray(axes)) ** e, axis=1)


def car_surface(seed: int, N: int, jitter=0.01):
    """Points and unit normals on the union of the CAR_PARTS superellipsoids.

    Random directions from each part's centre are projected radially onto its
    surface (F is homogeneous of degree 3, so r = F(d)^(-1/3)); points inside
    another part are dropped; a 1 % radial jitter is applied; normals are the
    normalised gradient of F.  Parts get candidates in proportion to a rough
    surface-area estimate; the result is truncated to exactly N points.
    Returns float64 [N, 6] = (xyz, normal).
    """
    areas = []
    for _, ax in CAR_PARTS:
        a, b, c = ax
        # Knud Thomsen's approximation of an ellipsoid's surface area
        areas.append(4 * math.pi * (((a * b) ** 1.6 + (a * c) ** 1.6 + (b * c) ** 1.6) / 3)
                     ** (1 / 1.6))
    areas = np.array(areas) / sum(areas)
    out, have, start, rnd = [], 0, 0, 0
    while have < N:
        need = N - have
        batch = []
        for k, (cen, ax) in enumerate(CAR_PARTS):
            n = int(need * areas[k] * 1.6) + 256
            d = _unit_dirs(seed, start, n)
            start += n
            r = _superellipsoid_F(d, ax) ** (-1.0 / 3.0)
            xi = normal(seed, STREAM_GEOM, (1 << 42) + start, n)
            p = d * (r * (1.0 + jitter * xi))[:, None] + np.asarray(cen)
            inside = np.zeros(n, dtype=bool)
            for k2, (cen2, ax2) in enumerate(CAR_PARTS):
                if k2 != k:
                    inside |= _superellipsoid_F(p - np.asarray(cen2), ax2) < 1.0
            q = (p - np.asarray(cen)) / np.asarray(ax)
            nrm = 3.0 * np.sign(q) * q * q / np.asarray(ax)
            nrm /= np.linalg.norm(nrm, axis=1, keepdims=True)
            keep = ~inside
            batch.append(np.concatenate([p[keep], nrm[keep]], axis=1))
        # interleave parts deterministically so truncation keeps all of them
        cat = np.concatenate(batch)
        perm = np.argsort(raw64(seed, STREAM_GEOM, (1 << 43) + rnd * (1 << 30), len(cat)),
                          kind="stable")
        out.append(cat[perm])
        have += len(cat)
        rnd += 1
    return np.concatenate(out)[:N]


def aircraft_surface(seed: int, N: int, jitter=0.01):
    """Points and normals on a cylinder fuselage (radius 2, length 40, flat
    caps) plus two thin wing slabs (18 x 5 x 0.4 m); float64 [N, 6]."""
    R, L = 2.0, 40.0
    wing = (18.0, 5.0, 0.4)
    a_cyl = 2 * math.pi * R * L + 2 * math.pi * R * R
    a_wing = 2 * (2 * (wing[0] * wing[1] + wing[0] * wing[2] + wing[1] * wing[2]))
    n_cyl = int(N * a_cyl / (a_cyl + a_wing))
    u = uniform(seed, STREAM_GEOM, 0, 4 * N).reshape(N, 4)
    pts = np.empty((N, 3))
    nrm = np.empty((N, 3))
    # fuselage: side or caps by area
    i = np.arange(n_cyl)
    side = u[i, 0] < (2 * math.pi * R * L) / a_cyl
    th = 2 * math.pi * u[i, 1]
    xs = L * (u[i, 2] - 0.5)
    cap_r = R * np.sqrt(u[i, 2])
    cap_x = np.where(u[i, 3] < 0.5, -L / 2, L / 2)
    pts[i, 0] = np.where(side, xs, cap_x)
    rr = np.where(side, R, cap_r)
    pts[i, 1] = rr * np.cos(th)
    pts[i, 2] = rr * np.sin(th)
    nrm[i, 0] = np.where(side, 0.0, np.sign(cap_x))
    nrm[i, 1] = np.where(side, np.cos(th), 0.0)
    nrm[i, 2] = np.where(side, np.sin(th), 0.0)
    # wings: two slabs at y = +-(R + wing_span/2), top/bottom faces dominate
    j = np.arange(n_cyl, N)
    sgn = np.where(u[j, 0] < 0.5, -1.0, 1.0)
    top = np.where(u[j, 3] < 0.5, 1.0, -1.0)
    pts[j, 0] = wing[1] * (u[j, 1] - 0.5)
    pts[j, 1] = sgn * (R + wing[0] * u[j, 2])
    pts[j, 2] = top * wing[2] / 2
    nrm[j] = 0.0
    nrm[j, 2] = top
    xi = normal(seed, STREAM_GEOM, 1 << 41, N)
    pts = pts * (1.0 + jitter * xi)[:, None]
    return np.concatenate([pts, nrm], axis=1)


def fourier_features(seed: int, p: np.ndarray, C: int, sigma: float = 1.0) -> np.ndarray:
    """phi(p) = [cos(2 pi B p), sin(2 pi B p)], B [C/2, d] ~ N(0, sigma^2) (float32)."""
    d = p.shape[1]
    B = sigma * normal(seed, STREAM_RFF, 0, (C // 2) * d).reshape(C // 2, d)
    out = np.empty((p.shape[0], C), dtype=np.float32)

    def blk(s, n):
        proj = 2.0 * math.pi * (p[s:s + n] @ B.T)
        out[s:s + n, :C // 2] = np.cos(proj)
        out[s:s + n, C // 2:] = np.sin(proj)

    _blocks(p.shape[0], blk, chunk=max(1, CHUNK // C))
    return out


# --------------------------------------------------------------------------
# Workloads
# --------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    N: int
    C: int
    H: int
    M: int
    dtype: str          # "f32" or "bf16": storage of x, G, A, a, y, dY, dx
    backward: bool
    geometry: str       # "normal", "grid2d", "ellipsoid", "car", "aircraft", "uniform"
    seed: int
    tau0: float = 0.5
    tau_min: float = 0.01
    eps: float = 1e-5


WORKLOADS = {
    "ns2d_fwd_f32": Workload("ns2d_fwd_f32", 4096, 64, 4, 16, "f32", False, "normal",
                             BASE_SEED + 1),
    "grid2d_16k_f32": Workload("grid2d_16k_f32", 16384, 128, 8, 64, "f32", True, "grid2d",
                               BASE_SEED + 2),
    "ellipsoid_32k_bf16": Workload("ellipsoid_32k_bf16", 32768, 256, 8, 32, "bf16", True,
                                   "ellipsoid", BASE_SEED + 3),
    "car_1m_bf16": Workload("car_1m_bf16", 1_000_000, 256, 8, 32, "bf16", True, "car",
                            BASE_SEED + 4),
    "aircraft_2p5m_bf16": Workload("aircraft_2p5m_bf16", 2_500_000, 256, 8, 64, "bf16", True,
                                   "aircraft", BASE_SEED + 5),
}


def make_x(w: Workload, N: Optional[int] = None) -> np.ndarray:
    """Point features x [N,C] float32 for a workload (first N points)."""
    N = w.N if N is None else N
    if w.geometry == "normal":
        x = normal(w.seed, STREAM_GEOM, 0, N * w.C).reshape(N, w.C)
    elif w.geometry == "uniform":
        x = 2.0 * uniform(w.seed, STREAM_GEOM, 0, N * w.C).reshape(N, w.C) - 1.0
    elif w.geometry == "grid2d":
        side = int(round(math.sqrt(w.N)))
        k = np.arange(N)
        uv = np.stack([(k // side + 0.5) / side, (k % side + 0.5) / side], axis=1)
        L = normal(w.seed, STREAM_RFF, 0, 2 * w.C).reshape(2, w.C)
        x = uv @ L + 0.1 * normal(w.seed, STREAM_GEOM, 0, N * w.C).reshape(N, w.C)
    elif w.geometry == "ellipsoid":
        x = fourier_features(w.seed, ellipsoid_points(w.seed, N), w.C)
    elif w.geometry == "car":
        x = fourier_features(w.seed, car_surface(w.seed, N), w.C)
    elif w.geometry == "aircraft":
        x = fourier_features(w.seed, aircraft_surface(w.seed, N), w.C)
    else:
        raise ValueError(w.geometry)
    x = np.ascontiguousarray(x, dtype=np.float32)
    return round_bf16(x) if w.dtype == "bf16" else x


def make_gumbel(w: Workload, N: Optional[int] = None) -> np.ndarray:
    N = w.N if N is None else N
    G = gumbel(w.seed, N, w.M).astype(np.float32)
    return round_bf16(G) if w.dtype == "bf16" else G


def make_grad(w: Workload, N: Optional[int] = None) -> np.ndarray:
    """Upstream gradient dY [N,C] ~ N(0,1)."""
    N = w.N if N is None else N
    g = normal(w.seed, STREAM_GRAD, 0, N * w.C, dtype=np.float32).reshape(N, w.C)
    return round_bf16(g) if w.dtype == "bf16" else g


def make_params(w: Workload, biases: bool = False, out_proj: bool = False) -> dict:
    """Xavier-uniform weights for the slice projection A [C,M], the Ada-Temp
    projection a [C] (fan-out 1) and the token attention W_q, W_k, W_v [C,C]
    (plus W_o with ``out_proj``).  Biases are 0 unless ``biases`` is set, in
    which case they are small nonzero values (tests use them).  A and a are
    rounded to bf16 for bf16 workloads; everything else is float32."""
    C, M = w.C, w.M
    off = 0
    p = {}
    A = xavier_uniform(w.seed, off, C, M, (C, M)).astype(np.float32); off += C * M
    a = xavier_uniform(w.seed, off, C, 1, (C,)).astype(np.float32); off += C
    if w.dtype == "bf16":
        A, a = round_bf16(A), round_bf16(a)
    p["A"], p["a"] = A, a
    names = ["Wq", "Wk", "Wv"] + (["Wo"] if out_proj else [])
    for n in names:
        p[n] = xavier_uniform(w.seed, off, C, C, (C, C)).astype(np.float32)
        off += C * C
    if biases:
        u = lambda n: (0.2 * (2 * uniform(w.seed, STREAM_WEIGHTS, (1 << 40) + n * 4096, 4096)
                              - 1)).astype(np.float32)
        p["b"] = u(0)[:M].copy()
        p["b_t"] = float(u(1)[0])
        for k, n in enumerate(["bq", "bk", "bv"] + (["bo"] if out_proj else [])):
            p[n] = u(2 + k)[:C].copy()
    else:
        p["b"] = np.zeros(M, dtype=np.float32)
        p["b_t"] = 0.0
        for n in ["bq", "bk", "bv"] + (["bo"] if out_proj else []):
            p[n] = np.zeros(C, dtype=np.float32)
    return p


def layer_workload(w: Workload, layer: int) -> Workload:
    """The workload of block `layer` of a stack: the same shapes, its own
    seed (its own parameters and Gumbel noise)."""
    return dataclasses.replace(w, seed=w.seed + 100003 * (layer + 1))


def make_block_params(w: Workload, layer: int) -> dict:
    """Parameters of block `layer` of a Transolver++ block stack: the layer's
    (make_params of the layer's workload, with small nonzero biases and an
    output projection Wo, bo) plus Algorithm 1's Project Wp [C,C], bp [C],
    the two LayerNorms' gains (1 + small) and biases (small), and the MLP
    W1 [C,4C], b1, W2 [4C,C], b2 (Xavier-uniform; W1, W2 rounded to bf16 for
    bf16 workloads, as they feed bf16 GEMMs).  All float32."""
    wl = layer_workload(w, layer)
    C = w.C
    p = make_params(wl, biases=True, out_proj=True)
    off = 1 << 44                     # past make_params' draws in the weights stream
    p["Wp"] = xavier_uniform(wl.seed, off, C, C, (C, C)).astype(np.float32); off += C * C
    p["W1"] = xavier_uniform(wl.seed, off, C, 4 * C, (C, 4 * C)).astype(np.float32)
    off += 4 * C * C
    p["W2"] = xavier_uniform(wl.seed, off, 4 * C, C, (4 * C, C)).astype(np.float32)
    off += 4 * C * C
    if w.dtype == "bf16":
        p["W1"], p["W2"] = round_bf16(p["W1"]), round_bf16(p["W2"])
    small_u = lambda n, k: (0.2 * (2 * uniform(wl.seed, STREAM_WEIGHTS, off + k * 8192, n) - 1)
                            ).astype(np.float32)
    p["bp"] = small_u(C, 0)
    p["ln1_g"] = 1.0 + small_u(C, 1)
    p["ln1_b"] = small_u(C, 2)
    p["ln2_g"] = 1.0 + small_u(C, 3)
    p["ln2_b"] = small_u(C, 4)
    p["b1"] = small_u(4 * C, 5)
    p["b2"] = small_u(C, 6)
    return p


def make_layer_gumbel(w: Workload, layer: int, N: Optional[int] = None) -> np.ndarray:
    """The Gumbel noise of block `layer` [N,M] (storage dtype values)."""
    return make_gumbel(layer_workload(w, layer), N)


def small(name: str, N: int, C: int, H: int, M: int, dtype: str = "f32",
          geometry: str = "normal", seed: int = 7, **kw) -> Workload:
    """An ad-hoc workload (tests, sweeps)."""
    return Workload(name, N, C, H, M, dtype, True, geometry, seed, **kw)


def head_workload(w: Workload, head: int) -> Workload:
    """The workload of head `head` of a per-head sliced layer: D = C/H
    channels, one head, its own seed (its own slice parameters and noise)."""
    return dataclasses.replace(w, C=w.C // w.H, H=1, seed=w.seed + 7919 * (head + 1))


def make_head_params(w: Workload, shared: bool = False, biases: bool = True,
                     out_proj: bool = False) -> dict:
    """Parameters of a per-head sliced layer: the slice parameters of every
    head stacked on a leading axis of H (A [H,D,M], b [H,M], a [H,D], b_t
    [H]; each head's from make_params of its head workload), or one set for
    all heads with ``shared`` (head 0's: A [D,M], b [M], a [D], b_t float),
    and the token projections Wq, Wk, Wv (Wo) [D,D] with biases [D], shared
    by the heads (head 0's).  float32, A and a rounded to bf16 for bf16
    workloads."""
    hp = [make_params(head_workload(w, h), biases=biases, out_proj=out_proj)
          for h in range(1 if shared else w.H)]
    p = {k: v for k, v in hp[0].items() if k not in ("A", "b", "a", "b_t")}
    if shared:
        p.update({k: hp[0][k] for k in ("A", "b", "a", "b_t")})
    else:
        for k in ("A", "b", "a"):
            p[k] = np.ascontiguousarray(np.stack([q[k] for q in hp]))
        p["b_t"] = np.array([q["b_t"] for q in hp], dtype=np.float32)
    return p


def make_head_gumbel(w: Workload, N: Optional[int] = None) -> np.ndarray:
    """Gumbel noise of every head [H,N,M] (storage dtype values)."""
    return np.ascontiguousarray(np.stack([make_gumbel(head_workload(w, h), N)
                                          for h in range(w.H)]))
