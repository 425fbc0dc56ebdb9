"""Seeded synthetic inputs for the grid-octree workloads.

This module holds no part of the method's arithmetic: it only draws voxel
occupancy grids, dense colour channels, per-leaf features and weights.  Both
the GPU path and the CPU oracle consume what it returns.

Randomness: numpy PCG64 seeded with SeedSequence([161105009, config, sample,
stream]); stream 0 = geometry, 1 = features, 2 + k = weights of layer k.

The shapes stand in for the paper's workloads: voxelised object surfaces
(ModelNet10/40 at 8^3..256^3, batch 32) and facade scenes with colour
(RueMonge2014 at 256^3).  Neither dataset is available; nothing here
reproduces their items.

Workloads (name -> parameters):
  c1  32^3,  N=1,  one sphere surface, conv 1->8
  c2  64^3,  N=32, 1-3 primitive surfaces (sizes 8-40), conv 8->16, ReLU, pool
  c3  128^3, N=32, sizes 16-100, conv 16->32, ReLU, conv 32->32, ReLU, pool
  c4  256^3, N=16, sizes 32-220 with occupancy in [1%, 3%], conv 32->32, unpool
  c5  256^3, N=4,  facades + 2% noise, 4 channels, conv 4->16, ReLU, pool,
      conv 16->32, ReLU, guided unpool, conv 32->8
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

ROOT_SEED = 161105009


def rng_for(config: int, sample: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([ROOT_SEED, config, sample, stream])))


# ----------------------------------------------------------------------------
# Geometry: solid primitives and their 1-voxel-thick surfaces
# ----------------------------------------------------------------------------


def _random_rotation(rng: np.random.Generator) -> np.ndarray:
    q = rng.standard_normal(4)
    q /= np.linalg.norm(q)
    a, b, c, d = q
    return np.array([
        [a * a + b * b - c * c - d * d, 2 * (b * c - a * d), 2 * (b * d + a * c)],
        [2 * (b * c + a * d), a * a - b * b + c * c - d * d, 2 * (c * d - a * b)],
        [2 * (b * d - a * c), 2 * (c * d + a * b), a * a - b * b - c * c + d * d],
    ])


@dataclass
class Primitive:
    kind: str                 # "sphere" | "box" | "ellipsoid"
    centre: np.ndarray        # (3,) voxel units, (d, h, w)
    size: np.ndarray          # (3,) diameter / edge / axis length per axis
    rot: np.ndarray = field(default_factory=lambda: np.eye(3))

    def half_extent(self) -> np.ndarray:
        if self.kind == "ellipsoid":
            return np.full(3, self.size.max() / 2.0)
        return self.size / 2.0


def sample_primitive(rng: np.random.Generator, res: int, smin: float, smax: float) -> Primitive:
    kind = ("sphere", "box", "ellipsoid")[int(rng.integers(0, 3))]
    if kind == "sphere":
        size = np.full(3, rng.uniform(smin, smax))
        rot = np.eye(3)
    elif kind == "box":
        size = rng.uniform(smin, smax, size=3)
        rot = np.eye(3)
    else:
        size = rng.uniform(smin, smax, size=3)
        rot = _random_rotation(rng)
    prim = Primitive(kind, np.zeros(3), size, rot)
    ext = prim.half_extent()
    lo = np.minimum(ext, res / 2.0)
    prim.centre = np.array([rng.uniform(lo[a], res - lo[a]) for a in range(3)])
    return prim


def _solid_block(prim: Primitive, lo: np.ndarray, hi: np.ndarray) -> np.ndarray:
    """Solid indicator over voxels [lo, hi) (voxel centres at index + 0.5)."""
    axes = [np.arange(lo[a], hi[a], dtype=np.float64) + 0.5 - prim.centre[a] for a in range(3)]
    d, h, w = np.meshgrid(*axes, indexing="ij", sparse=True)
    if prim.kind == "sphere":
        r = prim.size[0] / 2.0
        return d * d + h * h + w * w <= r * r
    if prim.kind == "box":
        e = prim.size / 2.0
        return (np.abs(d) <= e[0]) & (np.abs(h) <= e[1]) & (np.abs(w) <= e[2])
    R = prim.rot  # body coordinates q = R^T (p - c)
    inv = 2.0 / prim.size
    acc = np.zeros(np.broadcast_shapes(d.shape, h.shape, w.shape), dtype=np.float64)
    for k in range(3):
        q = R[0, k] * d + R[1, k] * h + R[2, k] * w
        acc += (q * inv[k]) ** 2
    return acc <= 1.0


def add_surface(occ: np.ndarray, prim: Primitive) -> None:
    """OR the 1-voxel-thick surface of prim into occ (uint8 cube).  A surface
    voxel is solid with at least one 6-neighbour outside the solid; voxels
    outside the grid count as outside."""
    res = np.array(occ.shape)
    ext = prim.half_extent()
    lo = np.maximum(np.floor(prim.centre - ext).astype(int) - 1, 0)
    hi = np.minimum(np.ceil(prim.centre + ext).astype(int) + 2, res)
    if np.any(hi <= lo):
        return
    # Solid over the block grown by one voxel; cells beyond the grid are empty.
    glo, ghi = lo - 1, hi + 1
    solid = np.zeros(tuple(ghi - glo), dtype=bool)
    clo, chi = np.maximum(glo, 0), np.minimum(ghi, res)
    sl = tuple(slice(clo[a] - glo[a], chi[a] - glo[a]) for a in range(3))
    solid[sl] = _solid_block(prim, clo, chi)
    core = solid[1:-1, 1:-1, 1:-1]
    interior = core.copy()
    interior &= solid[:-2, 1:-1, 1:-1]
    interior &= solid[2:, 1:-1, 1:-1]
    interior &= solid[1:-1, :-2, 1:-1]
    interior &= solid[1:-1, 2:, 1:-1]
    interior &= solid[1:-1, 1:-1, :-2]
    interior &= solid[1:-1, 1:-1, 2:]
    surf = core & ~interior
    view = occ[lo[0]:hi[0], lo[1]:hi[1], lo[2]:hi[2]]
    view |= surf.astype(np.uint8)


def surface_sample(rng: np.random.Generator, res: int, smin: float, smax: float) -> np.ndarray:
    occ = np.zeros((res, res, res), dtype=np.uint8)
    k = int(rng.integers(1, 4))
    for _ in range(k):
        add_surface(occ, sample_primitive(rng, res, smin, smax))
    return occ


def sphere_sample(rng: np.random.Generator) -> np.ndarray:
    """One sphere surface in a 32^3 grid: centre U[12,20]^3, radius U[6,12]."""
    occ = np.zeros((32, 32, 32), dtype=np.uint8)
    centre = rng.uniform(12.0, 20.0, size=3)
    radius = rng.uniform(6.0, 12.0)
    add_surface(occ, Primitive("sphere", centre, np.full(3, 2.0 * radius)))
    return occ


# ----------------------------------------------------------------------------
# Facade scenes
# ----------------------------------------------------------------------------


def facade_sample(rng: np.random.Generator, res: int = 256, noise: float = 0.02):
    """3-6 axis-aligned facades (d is up) of thickness 1-2 with a grid of
    rectangular holes, plus Bernoulli(noise) scattered points.
    Returns (occupancy uint8 [res]^3, colour float32 [res]^3 x 3)."""
    occ = np.zeros((res, res, res), dtype=np.uint8)
    n_fac = int(rng.integers(3, 7))
    for _ in range(n_fac):
        normal = 1 + int(rng.integers(0, 2))          # 1: h, 2: w
        other = 3 - normal
        thick = 1 + int(rng.integers(0, 2))
        ext_d = int(rng.integers(64, res))
        ext_o = int(rng.integers(64, res))
        pos_n = int(rng.integers(0, res - thick + 1))
        org_d = int(rng.integers(0, res - ext_d + 1))
        org_o = int(rng.integers(0, res - ext_o + 1))
        slab = np.ones((ext_d, ext_o), dtype=bool)
        rows, cols = int(rng.integers(2, 7)), int(rng.integers(2, 7))
        hole_d, hole_o = int(rng.integers(4, 17)), int(rng.integers(4, 17))
        cell_d, cell_o = ext_d / rows, ext_o / cols
        hd = min(hole_d, max(int(cell_d) - 2, 0))
        ho = min(hole_o, max(int(cell_o) - 2, 0))
        for r in range(rows):
            for c in range(cols):
                cd = int((r + 0.5) * cell_d) - hd // 2
                co = int((c + 0.5) * cell_o) - ho // 2
                slab[cd:cd + hd, co:co + ho] = False
        idx = [slice(None)] * 3
        idx[0] = slice(org_d, org_d + ext_d)
        idx[normal] = slice(pos_n, pos_n + thick)
        idx[other] = slice(org_o, org_o + ext_o)
        view = occ[tuple(idx)]
        # broadcast the (d, other) slab over the thickness axis
        shape = [ext_d, 1, 1]
        shape[other] = ext_o
        view |= slab.reshape(shape).astype(np.uint8)
    occ |= (rng.random((res, res, res), dtype=np.float32) < noise).astype(np.uint8)
    colour = rng.random((res, res, res, 3), dtype=np.float32)
    colour *= occ[..., None]
    return occ, colour


def facade_points(rng: np.random.Generator, res: int = 256, noise: float = 0.002):
    """A coloured facade point cloud: 1 + Poisson(0.5) points per occupied
    voxel of a facade scene (uniform within the voxel).  Returns
    (points float32 [P, 3] in voxels along (d, h, w), features float32
    [P, 7] = RGB, a unit normal, height d / res, labels int32 [P] in 0..6,
    constant over 32^3 blocks of the scene)."""
    occ, colour = facade_sample(rng, res, noise)
    vox = np.argwhere(occ > 0)
    k = 1 + rng.poisson(0.5, size=len(vox))
    vox = np.repeat(vox, k, axis=0)
    pts = (vox + rng.random((len(vox), 3), dtype=np.float32)).astype(np.float32)
    rgb = colour[vox[:, 0], vox[:, 1], vox[:, 2]] + 0.05 * rng.standard_normal((len(vox), 3), dtype=np.float32)
    nrm = rng.standard_normal((len(vox), 3), dtype=np.float32)
    nrm /= np.maximum(np.linalg.norm(nrm, axis=1, keepdims=True), 1e-6)
    height = (pts[:, :1] / res).astype(np.float32)
    feat = np.concatenate([rgb, nrm, height], axis=1).astype(np.float32)
    labels = ((vox[:, 0] // 32) * 3 + (vox[:, 1] // 32) + 2 * (vox[:, 2] // 32)) % 7
    return pts, feat, labels.astype(np.int32)


# ----------------------------------------------------------------------------
# Workloads
# ----------------------------------------------------------------------------


@dataclass
class Layer:
    op: str              # "conv" | "relu" | "pool" | "unpool" | "unpool_guided" | "save" | "concat"
    cin: int = 0
    cout: int = 0


@dataclass
class Workload:
    key: str
    index: int
    res: int
    batch: int
    cin: int
    layers: list
    dense_features: bool  # True: leaf features = ten2oc(avg) of a dense input
    description: str
    points: bool = False  # True: the input is a point cloud (occupancy + mean features per leaf)

    @property
    def grid(self) -> int:
        return self.res // 8


WORKLOADS = {
    "c1": Workload("c1", 1, 32, 1, 1, [Layer("conv", 1, 8)], True,
                   "32^3 grid, batch 1, one sphere surface; conv3x3x3 1->8"),
    "c2": Workload("c2", 2, 64, 32, 8, [Layer("conv", 8, 16), Layer("relu"), Layer("pool")], False,
                   "64^3 grid, batch 32, primitive surfaces; conv3x3x3 8->16, ReLU, max-pool 2^3"),
    "c3": Workload("c3", 3, 128, 32, 16,
                   [Layer("conv", 16, 32), Layer("relu"), Layer("conv", 32, 32), Layer("relu"),
                    Layer("pool")], False,
                   "128^3 grid, batch 32; conv 16->32, ReLU, conv 32->32, ReLU, max-pool 2^3"),
    "c4": Workload("c4", 4, 256, 16, 32, [Layer("conv", 32, 32), Layer("unpool")], False,
                   "256^3 grid, batch 16, 1-3% occupied surfaces; conv3x3x3 32->32, unpool 2^3"),
    "c5": Workload("c5", 5, 256, 4, 4,
                   [Layer("conv", 4, 16), Layer("relu"), Layer("pool"), Layer("conv", 16, 32),
                    Layer("relu"), Layer("unpool_guided"), Layer("conv", 32, 8)], True,
                   "256^3 facade scenes, batch 4, 4 channels; conv 4->16, ReLU, pool, conv 16->32,"
                   " ReLU, guided unpool, conv 32->8"),
}

def _unet_layers():
    """The segmentation encoder-decoder of the paper's architecture table:
    four (conv, conv, max-pool) encoder levels, three convs at the coarsest
    level, and four (guided unpool, concat with the encoder output of that
    level, conv, conv) decoder levels; ReLU after every conv but the last.
    "save" keeps an encoder output for the matching "concat"."""
    L = []
    enc = [(8, 8, 16), (16, 16, 32), (32, 32, 64), (64, 64, 128)]
    for a, b, c in enc:
        L += [Layer("conv", a, b), Layer("relu"), Layer("conv", b, c), Layer("relu"), Layer("save"),
              Layer("pool")]
    for _ in range(3):
        L += [Layer("conv", 128, 128), Layer("relu")]
    dec = [(256, 128, 64), (128, 64, 32), (64, 32, 16), (32, 32, 8)]
    for i, (a, b, c) in enumerate(dec):
        L += [Layer("unpool_guided"), Layer("concat"), Layer("conv", a, b), Layer("relu"),
              Layer("conv", b, c)]
        if i < 3:
            L += [Layer("relu")]
    return L


WORKLOADS["unet"] = Workload(
    "unet", 6, 256, 1, 8, _unet_layers(), False,
    "256^3 facade point cloud, batch 1, 8 input channels (occupancy, RGB, normal, height averaged per"
    " leaf); the segmentation U-Net (4 levels, skip concats, guided unpooling)", points=True)


def point_cloud(wl: Workload, batch: int | None = None):
    """(points [P, 3], batch index [P], features [P, 7], labels [P]) of the
    workload's samples, concatenated."""
    n = wl.batch if batch is None else batch
    P, B, F, L = [], [], [], []
    for s in range(n):
        p, f, l = facade_points(rng_for(wl.index, s, 0), wl.res)
        P.append(p)
        F.append(f)
        L.append(l)
        B.append(np.full(len(p), s, dtype=np.int32))
    return np.concatenate(P), np.concatenate(B), np.concatenate(F), np.concatenate(L)

SIZE_RANGE = {2: (8.0, 40.0), 3: (16.0, 100.0), 4: (32.0, 220.0)}


def occupancy(wl: Workload, batch: int | None = None, samples=None) -> np.ndarray:
    """uint8 [N, res, res, res] occupancy for the workload (c1-c4, the U-Net's facades)."""
    idx = list(range(wl.batch if batch is None else batch)) if samples is None else list(samples)
    out = np.zeros((len(idx), wl.res, wl.res, wl.res), dtype=np.uint8)
    for j, s in enumerate(idx):
        rng = rng_for(wl.index, s, 0)
        if wl.index == 1:
            out[j] = sphere_sample(rng)
        elif wl.index in (2, 3):
            smin, smax = SIZE_RANGE[wl.index]
            out[j] = surface_sample(rng, wl.res, smin, smax)
        elif wl.index == 4:
            smin, smax = SIZE_RANGE[4]
            for _ in range(100):
                occ = surface_sample(rng, wl.res, smin, smax)
                frac = occ.mean(dtype=np.float64)
                if 0.01 <= frac <= 0.03:
                    break
            out[j] = occ
        elif wl.index == 6:
            out[j] = facade_sample(rng, wl.res)[0]
        else:
            raise ValueError("workload %s has a dense colour input; use facade_input" % wl.key)
    return out


def facade_input(wl: Workload, batch: int | None = None):
    """(occupancy uint8 [N,res^3], dense NDHWC float32 [N,res^3,4]) for c5."""
    n = wl.batch if batch is None else batch
    occ = np.zeros((n, wl.res, wl.res, wl.res), dtype=np.uint8)
    dense = np.zeros((n, wl.res, wl.res, wl.res, 4), dtype=np.float32)
    for s in range(n):
        o, col = facade_sample(rng_for(wl.index, s, 0), wl.res)
        occ[s] = o
        dense[s, ..., 0] = o
        dense[s, ..., 1:] = col
    return occ, dense


def leaf_features(wl: Workload, n_leaves: int, channels: int) -> np.ndarray:
    """float32 [n_leaves, channels] ~ N(0,1) (stream 1)."""
    return rng_for(wl.index, 0, 1).standard_normal((n_leaves, channels), dtype=np.float32)


def conv_weights(wl: Workload, layer: int, cin: int, cout: int, bias_std: float = 0.0):
    """(w float32 [cout, cin, 3, 3, 3], b float32 [cout]) for conv layer k.
    c1: N(0, 0.1^2); otherwise He-normal std sqrt(2 / (27 cin))."""
    rng = rng_for(wl.index, 0, 2 + layer)
    std = 0.1 if wl.index == 1 else float(np.sqrt(2.0 / (27.0 * cin)))
    w = (rng.standard_normal((cout, cin, 3, 3, 3)) * std).astype(np.float32)
    b = (rng.standard_normal(cout) * bias_std).astype(np.float32)
    return w, b


# ----------------------------------------------------------------------------
# Small random structures for unit tests
# ----------------------------------------------------------------------------


def random_occupancy(rng: np.random.Generator, n: int, gd: int, gh: int, gw: int,
                     density: float = 0.05, blobs: int = 3) -> np.ndarray:
    """A mix of sparse random voxels and solid boxes, so that every leaf size
    (1, 2, 4, 8) and every neighbour pattern shows up on tiny grids."""
    D, H, W = 8 * gd, 8 * gh, 8 * gw
    occ = (rng.random((n, D, H, W)) < density).astype(np.uint8)
    for s in range(n):
        for _ in range(blobs):
            lo = [int(rng.integers(0, x)) for x in (D, H, W)]
            ext = [int(rng.integers(1, max(2, x // 2))) for x in (D, H, W)]
            occ[s, lo[0]:lo[0] + ext[0], lo[1]:lo[1] + ext[1], lo[2]:lo[2] + ext[2]] = 1
        # clear a random box so that large empty leaves appear too
        lo = [int(rng.integers(0, x)) for x in (D, H, W)]
        ext = [int(rng.integers(1, x)) for x in (D, H, W)]
        occ[s, lo[0]:lo[0] + ext[0], lo[1]:lo[1] + ext[1], lo[2]:lo[2] + ext[2]] = 0
    return occ


def random_trees(rng: np.random.Generator, n: int, gd: int, gh: int, gw: int,
                 p_root: float = 0.5, p_d1: float = 0.5, p_d2: float = 0.5) -> np.ndarray:
    """uint32 [n*gd*gh*gw, 4]: canonical split strings drawn node by node (a
    root splits with p_root, a depth-1 node of a split root with p_d1, a
    depth-2 node of a split depth-1 node with p_d2), bit j at word j >> 5,
    position j & 31.  Gives every cell size next to every kind of neighbour
    on small grids."""
    nt = n * gd * gh * gw
    bits = np.zeros((nt, 73), dtype=bool)
    bits[:, 0] = rng.random(nt) < p_root
    for i in range(1, 9):
        bits[:, i] = bits[:, 0] & (rng.random(nt) < p_d1)
    for i in range(9, 73):
        bits[:, i] = bits[:, (i - 1) // 8] & (rng.random(nt) < p_d2)
    words = np.zeros((nt, 4), dtype=np.uint32)
    for j in range(73):
        words[:, j >> 5] |= bits[:, j].astype(np.uint32) << np.uint32(j & 31)
    return words
