"""Seeded synthetic inputs for the CG convolution.

This module is shared by the tests, ``bench.py`` and ``__graft_entry__`` and
feeds the same arrays to the GPU library and to the CPU oracle.  It holds no
Clebsch-Gordan or convolution arithmetic: only geometry sampling, real
spherical harmonics of sample directions (to give features the structure of
the paper's workloads), and dtype conversion.

Workloads (shapes of the paper's experiments, §5; none of its datasets are
available, so these synthetic sets stand in for them):

  tiny        B=1,  N=64,    L=2, C=4   i.i.d. N(0,1)
  nbody       B=16, N=256,   L=3, C=16  particles uniform in the unit ball;
              Y_lm(x/|x|) * exp(-|x|^2) in every channel, plus N(0, 0.1^2)
              noise drawn separately for q and k
  molecule    B=32, N=32,    L=4, C=32  9..29 real atoms (rest zero padding),
              Gaussian cloud sigma=1.5; Y_lm of the direction from the
              centroid times a per-channel linear map of a one-hot atom type
              (5 types), separate maps for q and k
  pointcloud  B=8,  N=16384, L=6, C=32  points uniform on the surfaces of
              1..4 random ellipsoids (semi-axes U[0.2,1]); Y_lm of the surface
              normal times per-channel N(0,1) weights (separate for q and k)
  large       B=2,  N=65536, L=8, C=64  i.i.d. N(0, 1/(2l+1)) per degree
  graph       B=4,  N=4096,  L=6, C=32  the point-cloud recipe with surface
              positions kept; features as for pointcloud, plus per sample the
              eigenbasis U of the normalised Laplacian of the symmetrised
              16-nearest-neighbour graph of the positions (for the graph
              Fourier variant of the convolution)

Seeds: workload s uses numpy SeedSequence(s).spawn(3) -> (geometry, q, k)
streams, s = 1001..1005 in the order above.  Values are generated in float64
and rounded once to float32, except the i.i.d. workloads (tiny, large), which
are drawn directly in float32.
"""

from __future__ import annotations

from math import factorial, pi, sqrt

import numpy as np

WORKLOADS = {
    "tiny": dict(B=1, N=64, L=2, C=4, seed=1001),
    "nbody": dict(B=16, N=256, L=3, C=16, seed=1002),
    "molecule": dict(B=32, N=32, L=4, C=32, seed=1003),
    "pointcloud": dict(B=8, N=16384, L=6, C=32, seed=1004),
    "large": dict(B=2, N=65536, L=8, C=64, seed=1005),
    "graph": dict(B=4, N=4096, L=6, C=32, seed=1006),
}


def _streams(seed: int):
    return [np.random.default_rng(s) for s in np.random.SeedSequence(seed).spawn(3)]


def real_ylm(L: int, xyz: np.ndarray) -> np.ndarray:
    """Real spherical harmonics (no Condon-Shortley phase in the real form)
    of the directions of ``xyz`` (n, 3): Y_l0 = N_l0 P_l, Y_{l,+m} =
    sqrt2 N_lm P_l^m cos(m phi), Y_{l,-m} = sqrt2 N_lm P_l^m sin(m phi), stacked
    at index l^2+l+m.  Degree 1 is sqrt(3/4pi) * (y, z, x)/r.  Own associated-
    Legendre recurrence; returns (n, (L+1)^2) float64."""
    xyz = np.asarray(xyz, dtype=np.float64)
    r = np.linalg.norm(xyz, axis=1)
    r = np.where(r == 0.0, 1.0, r)
    ct = xyz[:, 2] / r
    st = np.sqrt(np.maximum(0.0, 1.0 - ct * ct))
    phi = np.arctan2(xyz[:, 1], xyz[:, 0])
    n = xyz.shape[0]
    P = {}
    for m in range(L + 1):
        pmm = np.ones(n)
        for i in range(1, m + 1):
            pmm = pmm * (2 * i - 1) * st
        P[(m, m)] = pmm
        if m + 1 <= L:
            P[(m + 1, m)] = ct * (2 * m + 1) * pmm
        for l in range(m + 2, L + 1):
            P[(l, m)] = ((2 * l - 1) * ct * P[(l - 1, m)] - (l + m - 1) * P[(l - 2, m)]) / (l - m)
    out = np.empty((n, (L + 1) ** 2))
    for l in range(L + 1):
        for m in range(0, l + 1):
            nlm = sqrt((2 * l + 1) / (4 * pi) * factorial(l - m) / factorial(l + m))
            if m == 0:
                out[:, l * l + l] = nlm * P[(l, 0)]
            else:
                out[:, l * l + l + m] = sqrt(2.0) * nlm * P[(l, m)] * np.cos(m * phi)
                out[:, l * l + l - m] = sqrt(2.0) * nlm * P[(l, m)] * np.sin(m * phi)
    return out


def _unit(rng, n):
    v = rng.standard_normal((n, 3))
    return v / np.linalg.norm(v, axis=1, keepdims=True)


def _rotation(rng):
    A = rng.standard_normal((3, 3))
    Q, Rr = np.linalg.qr(A)
    Q = Q * np.sign(np.diag(Rr))
    if np.linalg.det(Q) < 0:
        Q[:, 0] = -Q[:, 0]
    return Q


def iid(B, N, L, C, seed, per_degree_variance=False):
    """i.i.d. Gaussian q, k of shape (B, N, (L+1)^2, C), float32.  With
    ``per_degree_variance`` the variance of degree l is 1/(2l+1)."""
    _, rq, rk = _streams(seed)
    K = (L + 1) ** 2
    scale = np.ones(K)
    if per_degree_variance:
        for l in range(L + 1):
            scale[l * l:(l + 1) ** 2] = 1.0 / sqrt(2 * l + 1)
    out = []
    for r in (rq, rk):
        a = np.empty((B, N, K, C), dtype=np.float32)
        for b in range(B):
            # drawn directly in float32 (numpy's float32 ziggurat): the large
            # workload has 1.4e9 values and float64 temporaries cost minutes
            r.standard_normal(dtype=np.float32, out=a[b])
            if per_degree_variance:
                a[b] *= scale.astype(np.float32)[None, :, None]
        out.append(a)
    return out[0], out[1]


def nbody(B, N, L, C, seed):
    rg, rq, rk = _streams(seed)
    K = (L + 1) ** 2
    q = np.empty((B, N, K, C), dtype=np.float32)
    k = np.empty_like(q)
    for b in range(B):
        d = _unit(rg, N)
        rad = rg.uniform(0.0, 1.0, N) ** (1.0 / 3.0)
        x = d * rad[:, None]
        base = real_ylm(L, x) * np.exp(-rad * rad)[:, None]
        q[b] = (base[:, :, None] + 0.1 * rq.standard_normal((N, K, C))).astype(np.float32)
        k[b] = (base[:, :, None] + 0.1 * rk.standard_normal((N, K, C))).astype(np.float32)
    return q, k


def molecule(B, N, L, C, seed, n_types=5, n_min=9, n_max=29):
    rg, rq, rk = _streams(seed)
    K = (L + 1) ** 2
    Wq = rq.standard_normal((n_types, C))
    Wk = rk.standard_normal((n_types, C))
    q = np.zeros((B, N, K, C), dtype=np.float32)
    k = np.zeros_like(q)
    n_real = rg.integers(n_min, min(n_max, N) + 1, size=B)
    for b in range(B):
        n = int(n_real[b])
        pos = 1.5 * rg.standard_normal((n, 3))
        rel = pos - pos.mean(axis=0, keepdims=True)
        nrm = np.linalg.norm(rel, axis=1)
        rel[nrm < 1e-12] = np.array([0.0, 0.0, 1.0])
        Y = real_ylm(L, rel)
        types = rg.integers(0, n_types, size=n)
        q[b, :n] = (Y[:, :, None] * Wq[types][:, None, :]).astype(np.float32)
        k[b, :n] = (Y[:, :, None] * Wk[types][:, None, :]).astype(np.float32)
    return q, k, n_real


def _ellipsoid_normals(rg, n, axes, rot):
    """n points uniform (by area) on an ellipsoid surface; returns unit normals."""
    a = np.asarray(axes)
    gmax = 1.0 / a.min()
    out = []
    have = 0
    while have < n:
        u = _unit(rg, max(2 * (n - have), 64))
        g = np.sqrt((u[:, 0] / a[0]) ** 2 + (u[:, 1] / a[1]) ** 2 + (u[:, 2] / a[2]) ** 2)
        keep = rg.uniform(0.0, gmax, u.shape[0]) < g
        nr = u[keep] / a[None, :]
        nr /= np.linalg.norm(nr, axis=1, keepdims=True)
        out.append(nr)
        have += nr.shape[0]
    return (np.concatenate(out)[:n]) @ rot.T


def pointcloud(B, N, L, C, seed):
    rg, rq, rk = _streams(seed)
    K = (L + 1) ** 2
    q = np.empty((B, N, K, C), dtype=np.float32)
    k = np.empty_like(q)
    for b in range(B):
        n_ell = int(rg.integers(1, 5))
        axes = rg.uniform(0.2, 1.0, size=(n_ell, 3))
        rots = [_rotation(rg) for _ in range(n_ell)]
        _centres = rg.uniform(-0.5, 0.5, size=(n_ell, 3))  # positions do not enter the features
        # surface areas by Monte Carlo: area = 4 pi abc E_u[g(u)]
        u = _unit(rg, 4096)
        areas = np.array([4 * pi * np.prod(ax) * np.mean(np.sqrt(((u / ax) ** 2).sum(1)))
                          for ax in axes])
        counts = np.floor(N * areas / areas.sum()).astype(int)
        counts[0] += N - counts.sum()
        normals = np.concatenate([_ellipsoid_normals(rg, int(cnt), axes[e], rots[e])
                                  for e, cnt in enumerate(counts) if cnt > 0])
        normals = normals[rg.permutation(N)]
        Y = real_ylm(L, normals)
        wq = rq.standard_normal(C)
        wk = rk.standard_normal(C)
        _outer_into(q[b], Y, wq)
        _outer_into(k[b], Y, wk)
    return q, k


def _outer_into(dst, Y, w, rows=1024):
    """dst[n, k, c] = float32(Y[n, k] * w[c]), product taken in float64."""
    for n0 in range(0, Y.shape[0], rows):
        dst[n0:n0 + rows] = Y[n0:n0 + rows, :, None] * w[None, None, :]


def _ellipsoid_points(rg, n, axes, rot, centre):
    """n points uniform (by area) on an ellipsoid surface; returns (positions,
    unit normals).  Same rejection rule as _ellipsoid_normals: u uniform on
    the sphere, accepted with probability proportional to the area element;
    the point is axes * u, its normal is proportional to u / axes."""
    a = np.asarray(axes)
    gmax = 1.0 / a.min()
    pos, nrm = [], []
    have = 0
    while have < n:
        u = _unit(rg, max(2 * (n - have), 64))
        g = np.sqrt((u[:, 0] / a[0]) ** 2 + (u[:, 1] / a[1]) ** 2 + (u[:, 2] / a[2]) ** 2)
        keep = rg.uniform(0.0, gmax, u.shape[0]) < g
        uk = u[keep]
        nr = uk / a[None, :]
        nr /= np.linalg.norm(nr, axis=1, keepdims=True)
        pos.append(uk * a[None, :])
        nrm.append(nr)
        have += uk.shape[0]
    P = np.concatenate(pos)[:n] @ rot.T + centre
    Nr = np.concatenate(nrm)[:n] @ rot.T
    return P, Nr


def laplacian_eigenbasis(points, knn: int):
    """(U, eigenvalues) of the normalised Laplacian I - D^-1/2 A D^-1/2 of the
    symmetrised knn-nearest-neighbour graph of the points (A_ij = 1 if j is
    among the knn nearest neighbours of i or i among those of j).  U holds
    the eigenvectors as columns, eigenvalues ascending (float64)."""
    P = np.asarray(points, dtype=np.float64)
    n = P.shape[0]
    d2 = ((P[:, None, :] - P[None, :, :]) ** 2).sum(-1)
    np.fill_diagonal(d2, np.inf)
    nbr = np.argpartition(d2, min(knn, n - 1) - 1, axis=1)[:, :min(knn, n - 1)]
    A = np.zeros((n, n))
    A[np.repeat(np.arange(n), nbr.shape[1]), nbr.ravel()] = 1.0
    A = np.maximum(A, A.T)
    dinv = 1.0 / np.sqrt(A.sum(1))
    Lap = np.eye(n) - dinv[:, None] * A * dinv[None, :]
    lam, U = np.linalg.eigh(Lap)
    return U, lam


def graph_pointcloud(B, N, L, C, seed, knn=16):
    """Point-cloud features with positions kept and the graph basis: returns
    q, k (B, N, K, C) float32 and U (B, N, N) float32."""
    rg, rq, rk = _streams(seed)
    K = (L + 1) ** 2
    q = np.empty((B, N, K, C), dtype=np.float32)
    k = np.empty_like(q)
    U = np.empty((B, N, N), dtype=np.float32)
    for b in range(B):
        n_ell = int(rg.integers(1, 5))
        axes = rg.uniform(0.2, 1.0, size=(n_ell, 3))
        rots = [_rotation(rg) for _ in range(n_ell)]
        centres = rg.uniform(-0.5, 0.5, size=(n_ell, 3))
        u = _unit(rg, 4096)
        areas = np.array([4 * pi * np.prod(ax) * np.mean(np.sqrt(((u / ax) ** 2).sum(1)))
                          for ax in axes])
        counts = np.floor(N * areas / areas.sum()).astype(int)
        counts[0] += N - counts.sum()
        parts = [_ellipsoid_points(rg, int(cnt), axes[e], rots[e], centres[e])
                 for e, cnt in enumerate(counts) if cnt > 0]
        order = rg.permutation(N)
        pos = np.concatenate([p for p, _ in parts])[order]
        normals = np.concatenate([nr for _, nr in parts])[order]
        Y = real_ylm(L, normals)
        _outer_into(q[b], Y, rq.standard_normal(C))
        _outer_into(k[b], Y, rk.standard_normal(C))
        U[b] = laplacian_eigenbasis(pos, knn)[0]
    return q, k, U


def make(name: str):
    """Inputs (q, k) float32 of the named workload (for "graph", use
    graph_pointcloud, which also returns the bases)."""
    w = WORKLOADS[name]
    B, N, L, C, s = w["B"], w["N"], w["L"], w["C"], w["seed"]
    if name == "tiny":
        return iid(B, N, L, C, s)
    if name == "nbody":
        return nbody(B, N, L, C, s)
    if name == "molecule":
        q, k, _ = molecule(B, N, L, C, s)
        return q, k
    if name == "pointcloud":
        return pointcloud(B, N, L, C, s)
    if name == "large":
        return iid(B, N, L, C, s, per_degree_variance=True)
    if name == "graph":
        q, k, _ = graph_pointcloud(B, N, L, C, s)
        return q, k
    raise KeyError(name)


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round to nearest, ties to even); returns
    the raw 16-bit patterns as uint16.  NaN is not expected in inputs."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + rounding) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
