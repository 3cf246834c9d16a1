"""Brute-force constructions straight from the lattice definition, used to pin
the oracle.  Nothing here follows the oracle's rounding / ranking procedure:
simplices are found by exhaustive search with a linear solve, neighbours by
exhaustive pairwise comparison, convolutions by dictionaries of keys.

Lattice (Permutohedral Lattice section, d = 3): the points of H_d (coordinates
summing to zero) that are integer with all coordinates congruent to one
remainder k mod d+1.  Its Delaunay simplices are x + k*1 - (d+1)*[last k
coordinates of a permutation], k = 0..d, for a remainder-0 point x.
"""
from __future__ import annotations

import itertools

import numpy as np

D1 = 4


def neighbour_vectors() -> np.ndarray:
    """n_j = (d+1) e_j - 1 and their negatives, in tap order 1..2d+2."""
    n = np.full((D1, D1), -1, dtype=np.int64) + D1 * np.eye(D1, dtype=np.int64)
    return np.concatenate([n, -n], axis=0)


def tap_offsets() -> np.ndarray:
    return np.concatenate([np.zeros((1, D1), np.int64), neighbour_vectors()], axis=0)


def lattice_points_in_box(radius: int) -> np.ndarray:
    """All lattice points with every coordinate in [-radius, radius]."""
    r = np.arange(-radius, radius + 1)
    g = np.stack(np.meshgrid(r, r, r, indexing="ij"), -1).reshape(-1, 3)
    last = -g.sum(axis=1, keepdims=True)
    pts = np.concatenate([g, last], axis=1)
    rem = np.mod(pts, D1)
    ok = (rem == rem[:, :1]).all(axis=1) & (np.abs(last[:, 0]) <= radius)
    return pts[ok]


def candidate_simplices(y: np.ndarray):
    """All (vertices 4x4, barycentric 4) of Delaunay simplices near y whose
    barycentric coordinates of y are all >= -1e-9."""
    y = np.asarray(y, dtype=np.float64)
    y = y - y.mean()        # float32 input may miss H_d by rounding
    out = []
    choices = [4 * np.floor(yi / 4) + 4 * np.arange(-1, 3) for yi in y[:3]]
    for x3 in itertools.product(*choices):
        x = np.array(list(x3) + [-sum(x3)], dtype=np.float64)
        if abs(x[3] - y[3]) > 12:
            continue
        for perm in itertools.permutations(range(D1)):
            V = np.empty((D1, D1))
            for k in range(D1):
                v = x + k
                for i in perm[D1 - k:]:
                    v[i] -= D1
                V[k] = v
            A = np.vstack([V.T, np.ones((1, D1))])
            rhs = np.concatenate([y, [1.0]])
            lam, *_ = np.linalg.lstsq(A, rhs, rcond=None)
            if np.abs(A @ lam - rhs).max() > 1e-9 * (1.0 + np.abs(y).max()):
                continue
            if lam.min() >= -1e-9:
                out.append((V.astype(np.int64), lam))
    return out


def brute_lattice(Y: np.ndarray):
    """Vertex set (lexicographic order), per-point vertex index and weights
    from the exhaustive simplex search.  Requires points strictly inside a
    simplex (a unique candidate)."""
    simplices = []
    for y in Y.astype(np.float64):
        cands = candidate_simplices(y)
        if len(cands) != 1:
            raise ValueError("point not strictly inside one simplex")
        V, lam = cands[0]
        order = np.argsort(np.mod(V[:, 0], D1))   # vertex k has remainder k
        simplices.append((V[order], lam[order]))
    keyset = sorted({tuple(v) for V, _ in simplices for v in V})
    index = {k: i for i, k in enumerate(keyset)}
    idx = np.array([[index[tuple(v)] for v in V] for V, _ in simplices], dtype=np.int64)
    w = np.array([lam for _, lam in simplices])
    return np.array(keyset, dtype=np.int64), index, idx, w


def brute_neighbours(keys: np.ndarray) -> np.ndarray:
    """O(n^2) scan: nbr[v][t] = u when keys[u] - keys[v] equals tap offset t."""
    n = keys.shape[0]
    offs = tap_offsets()
    diff = keys[None, :, :] - keys[:, None, :]              # [v, u, :]
    nb = np.full((n, 9), -1, dtype=np.int64)
    for t in range(9):
        hit = (diff == offs[t]).all(axis=2)
        v, u = np.nonzero(hit)
        nb[v, t] = u
    return nb


def brute_conv(keys_dst, keys_src_index, X, W, dst_scale=1, relu=False):
    """Y[v] = sum_t X[key(dst_scale * c_v + o_t)] W[t] by dictionary lookup."""
    offs = tap_offsets()
    Y = np.zeros((keys_dst.shape[0], W.shape[2]))
    for v, c in enumerate(keys_dst):
        for t in range(9):
            u = keys_src_index.get(tuple(dst_scale * c + offs[t]))
            if u is not None:
                Y[v] += X[u] @ W[t]
    return np.maximum(Y, 0) if relu else Y
