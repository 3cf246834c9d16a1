"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test ties one part of the oracle to something other than itself: a
hand-derived case, a closed form, an invariant stated in the paper, or a
brute-force construction from the lattice definition (tests/bruteforce.py).
"""
from __future__ import annotations

import json
import os

import numpy as np
import pytest

from tests import bruteforce as bf
from workloads import configs, generators as gen
from workloads.rng import Stream

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _tiny_cloud(seed, m=150, extent=1.0):
    st = Stream(seed, "tiny")
    return (extent * st.uniform(3 * m).reshape(m, 3)).astype(np.float32)


# ----------------------------------------------------------------------------
# embedding: hand-derived cases, closed forms, invariants
# ----------------------------------------------------------------------------
def test_golden_simplex_cases(oracle_mod):
    """Hand-derived simplices (tie rules, faces, vertices of each class)."""
    cases = json.load(open(os.path.join(GOLDEN, "simplex_cases.json")))["cases"]
    Y = np.array([c["y"] for c in cases], np.float32)
    keys, w = oracle_mod.simplex(Y)
    for i, c in enumerate(cases):
        assert keys[i].tolist() == c["keys"], c["derivation"]
        assert w[i].tolist() == c["w"], c["derivation"]


def test_keys_are_lattice_points_of_each_remainder(oracle_mod):
    """Every key sums to zero and vertex k has all coordinates = k mod d+1
    (Permutohedral Lattice section)."""
    wl = configs.make(1)
    y = oracle_mod.elevate(wl.positions, wl.sigma)
    keys, w = oracle_mod.simplex(y)
    assert (keys.sum(axis=2) == 0).all()
    for k in range(4):
        assert (np.mod(keys[:, k, :], 4) == k).all()


def test_barycentric_weights_and_reconstruction(oracle_mod):
    """b >= 0, sum b = 1 up to rounding, and sum_k b_k c_k = y."""
    for cfg in (1, 2, 4):
        wl = configs.make(cfg)
        y = oracle_mod.elevate(wl.positions, wl.sigma)
        keys, w = oracle_mod.simplex(y)
        assert (w >= 0).all()
        assert np.abs(w.astype(np.float64).sum(axis=1) - 1.0).max() <= 4 * np.finfo(np.float32).eps
        rec = np.einsum("pk,pki->pi", w.astype(np.float64), keys.astype(np.float64))
        scale = np.abs(y).max(axis=1, keepdims=True) + 1.0
        assert (np.abs(rec - y) / scale).max() < 2e-6


def test_point_on_a_vertex_gets_weight_one(oracle_mod):
    """A point exactly on a lattice vertex of remainder k: b_k = 1 and
    vertex k is that point."""
    pts = bf.lattice_points_in_box(12)
    keys, w = oracle_mod.simplex(pts.astype(np.float32))
    rem = np.mod(pts[:, 0], 4)
    for p in range(pts.shape[0]):
        k = rem[p]
        assert w[p, k] == 1.0
        assert (keys[p, k] == pts[p]).all()


def test_simplex_matches_exhaustive_search(oracle_mod):
    """The rounding construction's simplex is the one an exhaustive search
    over all Delaunay simplices finds, with the same barycentric weights."""
    st = Stream(7, "bf-simplex")
    g = st.uniform_range(3 * 60, -3.0, 3.0).reshape(60, 3).astype(np.float32)
    y = oracle_mod.elevate(g, np.array([0.7, 0.9, 1.3], np.float32))
    keys, w = oracle_mod.simplex(y)
    for p in range(y.shape[0]):
        cands = bf.candidate_simplices(y[p])
        assert cands, "no simplex contains the point"
        ok = False
        for V, lam in cands:
            order = np.argsort(np.mod(V[:, 0], 4))
            if (V[order] == keys[p]).all():
                assert np.abs(lam[order] - w[p]).max() < 1e-5
                ok = True
        assert ok


def test_elevation_is_scaled_isometry_onto_hyperplane(oracle_mod):
    """Elevation maps R^3 isometrically (times s = (d+1) sqrt(2/3)) onto H_d:
    coordinates sum to 0 and pairwise distances scale by s/sigma."""
    st = Stream(3, "iso")
    g = st.uniform_range(3 * 200, -5, 5).reshape(200, 3).astype(np.float32)
    sigma = np.array([0.5, 0.25, 2.0], np.float32)
    y = oracle_mod.elevate(g, sigma).astype(np.float64)
    assert np.abs(y.sum(axis=1)).max() < 1e-4
    s = 4.0 * np.sqrt(2.0 / 3.0)
    gs = g.astype(np.float64) / sigma.astype(np.float64)
    dg = np.linalg.norm(gs[:, None] - gs[None], axis=2) * s
    dy = np.linalg.norm(y[:, None] - y[None], axis=2)
    assert np.abs(dg - dy).max() / dg.max() < 1e-6


def test_neighbour_shell_of_the_lattice():
    """The nearest lattice points of the origin are exactly the 2(d+1) vectors
    +-[-1..d..-1] (Permutohedral Lattice section), at squared norm d(d+1)."""
    pts = bf.lattice_points_in_box(8)
    sq = (pts ** 2).sum(axis=1)
    nonzero = sq > 0
    nearest = pts[nonzero & (sq == sq[nonzero].min())]
    assert sq[nonzero].min() == 12
    assert sorted(map(tuple, nearest)) == sorted(map(tuple, bf.neighbour_vectors()))


def test_error_codes(oracle_mod):
    with pytest.raises(oracle_mod.OracleError) as e:
        oracle_mod.Lattice.create(np.array([[0, np.nan, 0]], np.float32), np.ones(3, np.float32))
    assert e.value.code == -6
    with pytest.raises(oracle_mod.OracleError) as e:
        oracle_mod.Lattice.create(np.array([[1e7, 0, 0]], np.float32), np.full(3, 0.1, np.float32))
    assert e.value.code == -5
    L = oracle_mod.Lattice.create(np.zeros((0, 3), np.float32), np.ones(3, np.float32))
    assert L.n == 0 and L.m == 0


# ----------------------------------------------------------------------------
# lattice structure
# ----------------------------------------------------------------------------
def test_lattice_matches_bruteforce_construction(oracle_mod):
    """Vertex set, numbering and per-point simplices equal those built from
    the exhaustive simplex search (points strictly inside simplices)."""
    pos = _tiny_cloud(11, 120, extent=0.6)
    sigma = np.full(3, 0.1, np.float32)
    L = oracle_mod.Lattice.create(pos, sigma)
    y = L.elevated()
    keys_b, _, idx_b, w_b = bf.brute_lattice(y)
    assert (L.keys() == keys_b).all()
    idx, w = L.simplices()
    assert (idx == idx_b).all()
    assert np.abs(w - w_b).max() < 1e-5


def test_neighbours_match_pairwise_scan(oracle_mod):
    for seed in (1, 2):
        L = oracle_mod.Lattice.create(_tiny_cloud(seed, 200), np.full(3, 0.15, np.float32))
        assert (L.neighbors() == bf.brute_neighbours(L.keys().astype(np.int64))).all()


def test_coarse_level_equals_doubled_sigma(oracle_mod):
    """Halving positions (Downsample) equals creating with 2*sigma, bitwise."""
    wl = configs.make(2)
    L0 = oracle_mod.Lattice.create(wl.positions, wl.sigma)
    L1 = L0.coarsen()
    L1b = oracle_mod.Lattice.create(wl.positions, 2 * wl.sigma)
    assert (L1.keys() == L1b.keys()).all()
    i1, w1 = L1.simplices()
    i2, w2 = L1b.simplices()
    assert (i1 == i2).all() and (w1 == w2).all()
    assert L1.level == 1 and L1.n < L0.n


def test_down_table_by_embedding(oracle_mod):
    """Coarse vertex c reads the fine vertex at 2c + o_t (pairwise search)."""
    L0 = oracle_mod.Lattice.create(_tiny_cloud(5, 200), np.full(3, 0.12, np.float32))
    L1 = L0.coarsen()
    kf, kc = L0.keys().astype(np.int64), L1.keys().astype(np.int64)
    offs = bf.tap_offsets()
    tab = L1.down_table()
    for v in range(L1.n):
        for t in range(9):
            hit = np.nonzero((kf == 2 * kc[v] + offs[t]).all(axis=1))[0]
            assert tab[v, t] == (hit[0] if hit.size else -1)


# ----------------------------------------------------------------------------
# operators
# ----------------------------------------------------------------------------
def test_splat_mass_and_constant(oracle_mod):
    """Raw splat conserves sum_p f_p (weights sum to 1); the normalised splat
    of a constant, sliced back, returns the constant."""
    wl = configs.make(1)
    L = oracle_mod.Lattice.create(wl.positions, wl.sigma)
    F = wl.features.astype(np.float64)
    X, W = L.splat(F, normalize=False)
    assert np.allclose(X.sum(axis=0), F.sum(axis=0), rtol=1e-6, atol=1e-6)
    assert abs(W.sum() - wl.m) < 1e-3
    const = np.full((wl.m, 3), 2.5)
    Xc, _ = L.splat(const, normalize=True)
    assert np.abs(L.slice(Xc) - 2.5).max() < 1e-5


def test_splat_matches_definition(oracle_mod):
    pos = _tiny_cloud(12, 100, 0.5)
    L = oracle_mod.Lattice.create(pos, np.full(3, 0.1, np.float32))
    keys_b, index, idx_b, w_b = bf.brute_lattice(L.elevated())
    F = np.random.default_rng(0).normal(size=(100, 5))
    X = np.zeros((len(keys_b), 5))
    Wb = np.zeros(len(keys_b))
    for p in range(100):
        for k in range(4):
            X[idx_b[p, k]] += w_b[p, k] * F[p]
            Wb[idx_b[p, k]] += w_b[p, k]
    Xo, Wo = L.splat(F, normalize=False)
    assert np.abs(Xo - X).max() < 1e-5 and np.abs(Wo - Wb).max() < 1e-5
    Xn, _ = L.splat(F, normalize=True)
    ref = np.where(Wb[:, None] > 0, X / np.where(Wb > 0, Wb, 1)[:, None], 0)
    assert np.abs(Xn - ref).max() < 1e-4


def test_slice_reproduces_affine_functions(oracle_mod):
    """With x_v = c_v, slicing returns the elevated position (barycentric
    interpolation reproduces affine functions)."""
    wl = configs.make(1)
    L = oracle_mod.Lattice.create(wl.positions, wl.sigma)
    out = L.slice(L.keys().astype(np.float64))
    assert np.abs(out - L.elevated()).max() < 2e-5


def test_conv_identity_shift_and_definition(oracle_mod):
    L = oracle_mod.Lattice.create(_tiny_cloud(21, 200), np.full(3, 0.12, np.float32))
    keys = L.keys().astype(np.int64)
    index = {tuple(k): i for i, k in enumerate(keys)}
    rng = np.random.default_rng(1)
    X = rng.normal(size=(L.n, 6))
    W = np.zeros((9, 6, 6))
    W[0] = np.eye(6)
    assert np.abs(L.conv(L, X, W) - X).max() == 0
    offs = bf.tap_offsets()
    for t in range(1, 9):
        W = np.zeros((9, 6, 6))
        W[t] = np.eye(6)
        Y = L.conv(L, X, W)
        for v in range(L.n):
            u = index.get(tuple(keys[v] + offs[t]))
            assert np.array_equal(Y[v], X[u] if u is not None else np.zeros(6))
    W = rng.normal(size=(9, 6, 4))
    b = rng.normal(size=4)
    ref = bf.brute_conv(keys, index, X, W) + b
    assert np.abs(L.conv(L, X, W, bias=b) - ref).max() < 1e-12
    assert np.abs(L.conv(L, X, W, bias=b, relu=True) - np.maximum(ref, 0)).max() < 1e-12
    rows = np.array([3, 0, L.n - 1])
    assert np.abs(L.conv(L, X, W, bias=b, rows=rows) - ref[rows]).max() < 1e-12


def test_strided_conv_matches_definition(oracle_mod):
    L0 = oracle_mod.Lattice.create(_tiny_cloud(22, 200), np.full(3, 0.12, np.float32))
    L1 = L0.coarsen()
    kf = L0.keys().astype(np.int64)
    index_f = {tuple(k): i for i, k in enumerate(kf)}
    rng = np.random.default_rng(2)
    X = rng.normal(size=(L0.n, 5))
    W = rng.normal(size=(9, 5, 3))
    ref = bf.brute_conv(L1.keys().astype(np.int64), index_f, X, W, dst_scale=2)
    assert np.abs(L1.conv(L0, X, W) - ref).max() < 1e-12


def _mirror(t):
    return 0 if t == 0 else (t + 4 if t <= 4 else t - 4)


def test_refine_is_adjoint_of_coarsen(oracle_mod):
    """Upsample is the transposed convolution of Downsample:
    <coarsen_W(X), Z> = <X, refine_W'(Z)>, W'[t] = W[mirror t]^T."""
    for seed, cfg_sigma in ((31, 0.12), (32, 0.07)):
        L0 = oracle_mod.Lattice.create(_tiny_cloud(seed, 300), np.full(3, cfg_sigma, np.float32))
        L1 = L0.coarsen()
        rng = np.random.default_rng(seed)
        X = rng.normal(size=(L0.n, 4))
        Z = rng.normal(size=(L1.n, 3))
        W = rng.normal(size=(9, 4, 3))
        Wt = np.stack([W[_mirror(t)].T for t in range(9)])
        lhs = np.sum(L1.conv(L0, X, W) * Z)
        rhs = np.sum(X * L0.refine_into(L1, Z, Wt))
        assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs)), (lhs, rhs)


def test_refine_support_of_one_coarse_vertex(oracle_mod):
    """A one-hot coarse vertex c reaches exactly the existing fine vertices
    2c + o_t, through tap mirror(t)."""
    L0 = oracle_mod.Lattice.create(_tiny_cloud(33, 300), np.full(3, 0.1, np.float32))
    L1 = L0.coarsen()
    kf, kc = L0.keys().astype(np.int64), L1.keys().astype(np.int64)
    index_f = {tuple(k): i for i, k in enumerate(kf)}
    offs = bf.tap_offsets()
    for c in range(0, L1.n, max(1, L1.n // 15)):
        Z = np.zeros((L1.n, 1))
        Z[c] = 1.0
        for t in range(9):
            W = np.zeros((9, 1, 1))
            W[_mirror(t)] = 1.0
            Y = L0.refine_into(L1, Z, W)[:, 0]
            expect = np.zeros(L0.n)
            f = index_f.get(tuple(2 * kc[c] + offs[t]))
            if f is not None:
                expect[f] = 1.0
            assert np.array_equal(Y, expect)


def test_deform_slice_special_cases_and_equivariance(oracle_mod):
    wl = configs.make(1)
    L = oracle_mod.Lattice.create(wl.positions, wl.sigma)
    rng = np.random.default_rng(3)
    X = rng.normal(size=(L.n, 8))
    zero = np.zeros(8)
    out, delta = L.deform_slice(X, zero, 0.0)
    assert np.array_equal(out, L.slice(X)) and not delta.any()
    idx, w = L.simplices()
    out, delta = L.deform_slice(X, zero, 0.3)
    ref = L.slice(X) + np.tanh(0.3) * X[idx].sum(axis=1)
    assert np.abs(out - ref).max() < 1e-12
    wv = rng.normal(size=8)
    o1, d1 = oracle_mod.deform_slice_raw(X, idx, w, wv, 0.1)
    perm = np.array([2, 0, 3, 1])
    o2, d2 = oracle_mod.deform_slice_raw(X, idx[:, perm], w[:, perm], wv, 0.1)
    assert np.abs(o1 - o2).max() < 1e-12
    assert np.abs(d1[:, perm] - d2).max() < 1e-15


def test_deform_slice_golden(oracle_mod):
    """Hand-worked DeformSlice of two points with explicit weights and vertex
    values (tests/golden/deform_slice_cases.json): the maximum per channel
    over b_k x_k of all d+1 vertices, the vertex itself included, subtracted
    before the linear map and tanh."""
    doc = json.load(open(os.path.join(GOLDEN, "deform_slice_cases.json")))
    X = np.array(doc["X"], np.float64)
    idx = np.array([c["idx"] for c in doc["points"]], np.int64)
    w = np.array([c["b"] for c in doc["points"]], np.float32)
    out, delta = oracle_mod.deform_slice_raw(X, idx, w, np.array(doc["wv"]), doc["beta"])
    for p, c in enumerate(doc["points"]):
        np.testing.assert_allclose(delta[p], c["delta"], rtol=0, atol=1e-14)
        np.testing.assert_allclose(out[p], c["out"], rtol=0, atol=1e-13)


def test_end_to_end_bruteforce(oracle_mod):
    """splat -> conv -> slice on a tiny cloud from brute-force definitions."""
    pos = _tiny_cloud(41, 150, 0.8)
    L = oracle_mod.Lattice.create(pos, np.full(3, 0.13, np.float32))
    keys_b, index, idx_b, w_b = bf.brute_lattice(L.elevated())
    rng = np.random.default_rng(4)
    F = rng.normal(size=(150, 4))
    W = rng.normal(size=(9, 4, 5))
    X = np.zeros((len(keys_b), 4))
    Ws = np.zeros(len(keys_b))
    for p in range(150):
        for k in range(4):
            X[idx_b[p, k]] += w_b[p, k] * F[p]
            Ws[idx_b[p, k]] += w_b[p, k]
    X = np.where(Ws[:, None] > 0, X / np.where(Ws > 0, Ws, 1)[:, None], 0)
    Y = bf.brute_conv(keys_b, index, X, W)
    out = np.einsum("pk,pkc->pc", w_b, Y[idx_b])
    Xo, _ = L.splat(F)
    got = L.slice(L.conv(L, Xo, W))
    assert np.abs(got - out).max() < 1e-4 * (1 + np.abs(out).max())


def test_bf16_rounding(oracle_mod):
    """Round to nearest even at 8 significant bits."""
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -3.14159, 0.0, 1e-3])
    r = oracle_mod.round_bf16(x)
    assert r[0] == 1.0 and r[1] == 1.0 and r[2] == 1.0 + 2 ** -6 and r[3] == 1.0
    bits = gen.to_bf16_bits(x.astype(np.float32))
    assert np.array_equal(gen.bf16_bits_to_f32(bits).astype(np.float64)[4:], r[4:])


# ---------------------------------------------------------------------------
# Distribute + PointNet (Proposed Operations, Eq. (distribute))
# ---------------------------------------------------------------------------
def _point_sets(ol):
    """J_v from the exported simplices: the points whose simplex holds v."""
    idx, _ = ol.simplices()
    J = [[] for _ in range(ol.n)]
    for p in range(idx.shape[0]):
        for k in range(4):
            J[idx[p, k]].append(p)
    return J


def _selector(rows, cols, pick, sign=1.0):
    W = np.zeros((rows, cols))
    for o, i in enumerate(pick):
        W[o, i] = sign
    return W


def _pointnet_layers(st, cin, widths=(16, 32, 64)):
    layers, k = [], cin
    for c in widths:
        layers.append((st.normal(c * k).reshape(c, k), st.normal(c)))
        k = c
    return layers


def test_distribute_invariances(oracle_mod):
    """Translating the cloud leaves g_p - mu_v unchanged; the operator does
    not depend on the order of the points."""
    O = oracle_mod
    G = _tiny_cloud(91, m=300)
    st = Stream(91, "dist-f")
    F = st.normal(300 * 5).reshape(300, 5)
    layers = _pointnet_layers(st, 8)
    gn = (1.0 + 0.1 * st.normal(8 + 16 + 32), 0.1 * st.normal(8 + 16 + 32))
    ol = O.Lattice.create(G, np.full(3, 0.15, np.float32))
    X = ol.distribute_pointnet(G.astype(np.float64), F, layers, gn)
    shift = np.array([0.25, -0.5, 0.125])
    # same lattice (built from G), shifted coordinates: mu shifts with them
    Xs = ol.distribute_pointnet(G.astype(np.float64) + shift, F, layers, gn)
    np.testing.assert_allclose(Xs, X, rtol=1e-9, atol=1e-9)
    perm = st.permutation(300)
    olp = O.Lattice.create(G[perm], np.full(3, 0.15, np.float32))
    assert np.array_equal(olp.keys(), ol.keys())    # vertices numbered by key: same rows
    Xp = olp.distribute_pointnet(G[perm].astype(np.float64), F[perm], layers, gn)
    np.testing.assert_allclose(Xp, X, rtol=1e-9, atol=1e-9)


def _pointnet_golden_case(c):
    def dense(rows, cols, nz):
        W = np.zeros((rows, cols))
        for o, i, v in nz:
            W[o, i] = v
        return W
    c1, c2, c3 = c["widths"]
    layers = [(dense(c1, 4, c["W1_nonzero"]), np.array(c["b1"])), (dense(c2, c1, c["W2_nonzero"]), np.array(c["b2"])),
              (dense(c3, c2, c["W3_nonzero"]), np.array(c["b3"]))]
    return layers, (np.array(c["gamma"]), np.array(c["beta"]))


def test_distribute_golden(oracle_mod):
    """Hand-worked Distribute + PointNet of two points sharing one simplex
    (tests/golden/distribute_cases.json): positions in units of sigma, mean
    subtracted, three [GroupNorm, ReLU, 1x1] blocks with statistics over all
    distributed rows (one channel per group up to 32 channels, 32 groups of
    two for a 64-wide layer), MaxPool over J_v."""
    doc = json.load(open(os.path.join(GOLDEN, "distribute_cases.json")))
    for c in doc["cases"]:
        G = np.array(c["positions"], np.float32)
        ol = oracle_mod.Lattice.create(G, np.full(3, c["sigma"], np.float32))
        idx, _ = ol.simplices()
        assert ol.n == 4 and sorted(idx[0]) == sorted(idx[1]) == [0, 1, 2, 3], "both points in one simplex"
        layers, gn = _pointnet_golden_case(c)
        X = ol.distribute_pointnet(G.astype(np.float64), np.array(c["features"]), layers, gn, eps=c["eps"])
        for v in range(4):
            np.testing.assert_allclose(X[v], c["expected"], rtol=0, atol=1e-12, err_msg=c["name"])


def test_distribute_positions_in_units_of_sigma(oracle_mod):
    """The coordinates enter as g / sigma: scaling the cloud and sigma by 8
    (exact in float32: the same lattice bit for bit) changes nothing, while
    with eps > 0 a raw-position reading would (the normalisation's eps acts
    on a variance 64 times larger)."""
    O = oracle_mod
    G = _tiny_cloud(95, m=300)
    st = Stream(95, "dist-sigma")
    F = st.normal(300 * 2).reshape(300, 2)
    layers = _pointnet_layers(st, 5)
    ol = O.Lattice.create(G, np.full(3, 0.15, np.float32))
    ol8 = O.Lattice.create(G * 8, np.full(3, 1.2, np.float32))
    assert np.array_equal(ol.keys(), ol8.keys())
    X = ol.distribute_pointnet(G.astype(np.float64), F, layers, eps=0.1)
    X8 = ol8.distribute_pointnet(G.astype(np.float64) * 8, F, layers, eps=0.1)
    np.testing.assert_allclose(X8, X, rtol=1e-10, atol=1e-10)
    # the same raw positions against a lattice of sigma/2 (positions halved
    # relative to sigma): no longer equal, so sigma is not ignored
    Xh = O.Lattice.create(G * 2, np.full(3, 0.3, np.float32)).distribute_pointnet(G.astype(np.float64), F, layers,
                                                                                  eps=0.1)
    assert np.abs(Xh - X).max() > 1e-3


def test_distribute_normalises_each_raw_channel(oracle_mod):
    """With eps = 0 the first normalisation makes the result invariant to a
    positive affine map of every raw feature channel and to a positive
    scale of every coordinate axis (one channel per group, statistics over
    all distributed rows)."""
    O = oracle_mod
    G = _tiny_cloud(96, m=300)
    st = Stream(96, "dist-affine")
    F = st.normal(300 * 3).reshape(300, 3)
    layers = _pointnet_layers(st, 6)
    ol = O.Lattice.create(G, np.full(3, 0.15, np.float32))
    X = ol.distribute_pointnet(G.astype(np.float64), F, layers, eps=0.0)
    a = np.array([3.0, 0.25, 7.0])
    b = np.array([-2.0, 5.0, 0.5])
    Xa = ol.distribute_pointnet(G.astype(np.float64) * np.array([2.0, 0.5, 4.0]), F * a + b, layers, eps=0.0)
    np.testing.assert_allclose(Xa, X, rtol=1e-9, atol=1e-9)


def test_distribute_selectors_reduce_to_zscores(oracle_mod):
    """Selector weights (each output copies one input) with eps = 0 and the
    identity affine: every block is a per-column z-score (scipy.stats.zscore,
    population variance) over the distributed rows followed by a ReLU, so
    x_v = max over J_v of relu(z(relu(z(relu(z(r)))))) column by column,
    with the rows r_p = [g_p / sigma - mean over J_v ; f_p] built here from
    the exported simplices."""
    from scipy.stats import zscore
    O = oracle_mod
    G = _tiny_cloud(97, m=250).astype(np.float64)
    st = Stream(97, "dist-z")
    F = st.normal(250 * 2).reshape(250, 2)
    sigma = 0.15
    ol = O.Lattice.create(G.astype(np.float32), np.full(3, sigma, np.float32))
    J = _point_sets(ol)
    rows, owner = [], []
    for v in range(ol.n):
        pts = G[J[v]] / sigma
        for p, g in zip(J[v], pts):
            rows.append(np.concatenate([g - pts.mean(axis=0), F[p]]))
            owner.append(v)
    R = np.array(rows)
    owner = np.array(owner)
    cin = R.shape[1]
    dup = lambda rows_, cols: _selector(rows_, cols, [o % cols for o in range(rows_)])
    layers = [(dup(16, cin), None), (dup(32, 16), None), (dup(16, 32), None)]
    X = ol.distribute_pointnet(G, F, layers, eps=0.0)
    relu = lambda x: np.maximum(x, 0.0)
    A = relu(zscore(R, axis=0))
    H1 = A[:, [o % cin for o in range(16)]]
    A = relu(zscore(H1, axis=0))
    H2 = A[:, [o % 16 for o in range(32)]]
    A = relu(zscore(H2, axis=0))
    H3 = A[:, [o % 32 for o in range(16)]]
    want = np.full((ol.n, 16), -np.inf)
    for q, v in enumerate(owner):
        want[v] = np.maximum(want[v], H3[q])
    np.testing.assert_allclose(X, want, rtol=1e-9, atol=1e-9)


def test_distribute_nan_propagates(oracle_mod):
    """A NaN feature poisons the statistics of its channel and, through the
    first layer, every output value."""
    O = oracle_mod
    G = _tiny_cloud(98, m=100)
    st = Stream(98, "dist-nan")
    F = st.normal(100 * 2).reshape(100, 2)
    F[7, 1] = np.nan
    ol = O.Lattice.create(G, np.full(3, 0.15, np.float32))
    X = ol.distribute_pointnet(G.astype(np.float64), F, _pointnet_layers(st, 5))
    assert np.isnan(X).all()


# ----------------------------------------------------------------------------
# backward passes: adjoint identities against the forward operators, and
# central finite differences where the forward is not linear
# ----------------------------------------------------------------------------
def _dot(a, b):
    return float(np.sum(np.asarray(a, np.float64) * np.asarray(b, np.float64)))


def test_splat_and_slice_backward_are_adjoints(oracle_mod):
    """<splat(F), G> = <F, splat^T(G)> for the raw and the normalised splat,
    and <slice(X), H> = <X, slice^T(H)>."""
    for seed in (41, 42):
        L = oracle_mod.Lattice.create(_tiny_cloud(seed, 250), np.full(3, 0.1, np.float32))
        rng = np.random.default_rng(seed)
        F = rng.normal(size=(L.m, 5))
        G = rng.normal(size=(L.n, 5))
        for norm in (False, True):
            X, _ = L.splat(F, normalize=norm)
            lhs, rhs = _dot(X, G), _dot(F, L.splat_backward(G, normalize=norm))
            assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs)), (norm, lhs, rhs)
        X = rng.normal(size=(L.n, 3))
        H = rng.normal(size=(L.m, 3))
        lhs, rhs = _dot(L.slice(X), H), _dot(X, L.slice_backward(H))
        assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs)), (lhs, rhs)


def _conv_forms(oracle_mod, seed):
    L0 = oracle_mod.Lattice.create(_tiny_cloud(seed, 300), np.full(3, 0.11, np.float32))
    L1 = L0.coarsen()
    return [("same", L0, L0, lambda X, W, b, r: L0.conv(L0, X, W, bias=b, relu=r)),
            ("strided", L1, L0, lambda X, W, b, r: L1.conv(L0, X, W, bias=b, relu=r)),
            ("upsample", L0, L1, lambda X, W, b, r: L0.refine_into(L1, X, W, bias=b, relu=r))]


def test_conv_backward_linear_part(oracle_mod):
    """Without the ReLU: dX is the adjoint, <conv(X), G> = <X, dX>; the
    forward is linear in W and in the bias, so <dW, E> = <G, conv_E(X)> and
    <dbias, e> = <G, 1 e^T> hold exactly, for the 1-hop, strided and Upsample
    forms."""
    for seed in (43, 44):
        rng = np.random.default_rng(seed)
        for name, dst, src, fwd in _conv_forms(oracle_mod, seed):
            X = rng.normal(size=(src.n, 4))
            W = rng.normal(size=(9, 4, 3))
            G = rng.normal(size=(dst.n, 3))
            dX, dW, db = dst.conv_backward(src, X, W, G)
            Y = fwd(X, W, None, False)
            assert abs(_dot(Y, G) - _dot(X, dX)) <= 1e-12 * max(1.0, abs(_dot(Y, G))), name
            E = rng.normal(size=W.shape)
            lhs, rhs = _dot(dW, E), _dot(G, fwd(X, E, None, False))
            assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs)), name
            e = rng.normal(size=3)
            lhs, rhs = _dot(db, e), _dot(G, np.ones((dst.n, 1)) * e)
            assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs)), name


def test_conv_backward_relu_finite_differences(oracle_mod):
    """With the ReLU, L = <relu(conv(X) + b), G> is piecewise linear; central
    differences in random directions of X, W and b match the gradients."""
    h = 1e-6
    rng = np.random.default_rng(45)
    for name, dst, src, fwd in _conv_forms(oracle_mod, 45):
        X = rng.normal(size=(src.n, 4))
        W = rng.normal(size=(9, 4, 5))
        b = rng.normal(size=5) * 0.5
        G = rng.normal(size=(dst.n, 5))
        Y = fwd(X, W, b, True)
        assert (Y == 0).mean() > 0.2, "the ReLU should clip a good share"
        dX, dW, db = dst.conv_backward(src, X, W, G, relu=True, Y=Y)
        loss = lambda X_, W_, b_: _dot(fwd(X_, W_, b_, True), G)
        for _ in range(2):
            D = rng.normal(size=X.shape)
            fd = (loss(X + h * D, W, b) - loss(X - h * D, W, b)) / (2 * h)
            assert abs(fd - _dot(dX, D)) <= 1e-6 * max(1.0, abs(fd)), (name, fd, _dot(dX, D))
            E = rng.normal(size=W.shape)
            fd = (loss(X, W + h * E, b) - loss(X, W - h * E, b)) / (2 * h)
            assert abs(fd - _dot(dW, E)) <= 1e-6 * max(1.0, abs(fd)), name
            e = rng.normal(size=5)
            fd = (loss(X, W, b + h * e) - loss(X, W, b - h * e)) / (2 * h)
            assert abs(fd - _dot(db, e)) <= 1e-6 * max(1.0, abs(fd)), name


def test_deform_slice_backward_finite_differences(oracle_mod):
    """L = <deform_slice(X, w, beta), G>: central differences in random
    directions of X and w, and in beta, match the gradients, and so do
    single coordinates of dX at the vertex holding a channel's maximum."""
    h = 1e-6
    for seed, C in ((46, 6), (47, 16)):
        L = oracle_mod.Lattice.create(_tiny_cloud(seed, 200, 0.6), np.full(3, 0.1, np.float32))
        rng = np.random.default_rng(seed)
        X = rng.normal(size=(L.n, C))
        wv = rng.normal(size=C) * 0.5
        beta = 0.2
        G = rng.normal(size=(L.m, C))
        dX, dwv, dbeta = L.deform_slice_backward(X, wv, beta, G)
        loss = lambda X_, w_, b_: _dot(L.deform_slice(X_, w_, b_)[0], G)
        for _ in range(3):
            D = rng.normal(size=X.shape)
            fd = (loss(X + h * D, wv, beta) - loss(X - h * D, wv, beta)) / (2 * h)
            assert abs(fd - _dot(dX, D)) <= 1e-6 * max(1.0, abs(fd)), (fd, _dot(dX, D))
            d = rng.normal(size=C)
            fd = (loss(X, wv + h * d, beta) - loss(X, wv - h * d, beta)) / (2 * h)
            assert abs(fd - _dot(dwv, d)) <= 1e-6 * max(1.0, abs(fd)), (fd, _dot(dwv, d))
        fd = (loss(X, wv, beta + h) - loss(X, wv, beta - h)) / (2 * h)
        assert abs(fd - dbeta) <= 1e-6 * max(1.0, abs(fd)), (fd, dbeta)
        # single coordinates of dX, among them the vertex holding a maximum
        idx, w = L.simplices()
        for p in (0, 5, L.m - 1):
            q = w[p, :, None].astype(np.float64) * X[idx[p]]
            k = int(np.argmax(q[:, 0]))
            v = idx[p, k]
            D = np.zeros_like(X)
            D[v, 0] = 1.0
            fd = (loss(X + h * D, wv, beta) - loss(X - h * D, wv, beta)) / (2 * h)
            assert abs(fd - dX[v, 0]) <= 1e-6 * max(1.0, abs(fd)), (p, fd, dX[v, 0])


# ----------------------------------------------------------------------------
# Group Normalization (pre-activation of the convolutions)
# ----------------------------------------------------------------------------
def test_groupnorm_worked_cases(oracle_mod):
    cases = json.load(open(os.path.join(GOLDEN, "groupnorm_cases.json")))["cases"]
    for c in cases:
        Y = oracle_mod.groupnorm(np.array(c["X"], np.float64), c["groups"], c.get("gamma"), c.get("beta"),
                                 c["eps"], c["relu"])
        assert np.abs(Y - np.array(c["Y"])).max() < 1e-12, c["derivation"]


def test_groupnorm_invariants(oracle_mod):
    """Each group of the normalised output has mean 0 and variance
    var / (var + eps); the output does not change when a group is scaled by
    a positive factor and shifted (eps -> 0); gamma and beta act per channel
    after the normalisation; groups = C normalises every channel alone."""
    rng = np.random.default_rng(7)
    X = rng.normal(size=(500, 64)) * rng.uniform(0.5, 3.0, size=64) + rng.normal(size=64) * 4
    for G in (32, 8, 1, 64):
        Y = oracle_mod.groupnorm(X, G, eps=1e-5)
        per = 64 // G
        for g in range(G):
            blk, yb = X[:, g * per:(g + 1) * per], Y[:, g * per:(g + 1) * per]
            assert abs(yb.mean()) < 1e-12
            v = blk.var()
            assert abs(yb.var() - v / (v + 1e-5)) < 1e-12
    Y0 = oracle_mod.groupnorm(X, 32, eps=1e-12)
    a = np.repeat(rng.uniform(0.2, 5.0, size=32), 2)
    b = np.repeat(rng.normal(size=32) * 10, 2)
    assert np.abs(oracle_mod.groupnorm(X * a + b, 32, eps=1e-12) - Y0).max() < 1e-8
    gam, bet = rng.normal(size=64), rng.normal(size=64)
    Yab = oracle_mod.groupnorm(X, 32, gam, bet, eps=1e-5)
    assert np.abs(Yab - (oracle_mod.groupnorm(X, 32, eps=1e-5) * gam + bet)).max() < 1e-12
    Yr = oracle_mod.groupnorm(X, 32, gam, bet, eps=1e-5, relu=True)
    assert np.array_equal(Yr, np.maximum(Yab, 0.0))


def test_deform_slice_classify_special_cases(oracle_mod):
    """The fused classifier reduces to DeformSlice with Wc = I and no bias,
    picks channel c with the one-hot row e_c, returns the bias with Wc = 0,
    and is linear in Wc."""
    L = oracle_mod.Lattice.create(_tiny_cloud(61, 300), np.full(3, 0.1, np.float32))
    rng = np.random.default_rng(61)
    C = 12
    X = rng.normal(size=(L.n, C))
    wv = rng.normal(size=C) * 0.3
    ds, _ = L.deform_slice(X, wv, 0.2)
    assert np.abs(L.deform_slice_classify(X, wv, 0.2, np.eye(C)) - ds).max() < 1e-12
    for c in (0, 5, C - 1):
        e = np.zeros((1, C))
        e[0, c] = 1.0
        assert np.abs(L.deform_slice_classify(X, wv, 0.2, e)[:, 0] - ds[:, c]).max() < 1e-12
    bc = rng.normal(size=7)
    assert np.abs(L.deform_slice_classify(X, wv, 0.2, np.zeros((7, C)), bc) - bc).max() == 0
    W1, W2 = rng.normal(size=(7, C)), rng.normal(size=(7, C))
    lhs = L.deform_slice_classify(X, wv, 0.2, W1 + W2)
    rhs = L.deform_slice_classify(X, wv, 0.2, W1) + L.deform_slice_classify(X, wv, 0.2, W2)
    assert np.abs(lhs - rhs).max() < 1e-12


# ----------------------------------------------------------------------------
# Backward of GroupNorm (+ ReLU), of the pre-activated convolution and of the
# fused classifier: finite differences of the oracle's forwards, invariances
# ----------------------------------------------------------------------------
def test_groupnorm_backward_finite_differences(oracle_mod):
    """L = <GN(X), G> (with and without the ReLU, with gamma and beta):
    central differences in random directions of X, gamma and beta match the
    gradients."""
    h = 1e-6
    rng = np.random.default_rng(71)
    for n, C, groups, relu in ((40, 8, 2, False), (40, 8, 8, True), (25, 12, 1, True), (30, 16, 4, False)):
        X = rng.normal(size=(n, C)) * rng.uniform(0.5, 2.0, size=C) + rng.normal(size=C)
        gam, bet = rng.normal(size=C), rng.normal(size=C) * 0.5
        G = rng.normal(size=(n, C))
        dX, dg, db = oracle_mod.groupnorm_backward(X, G, groups, gam, bet, 1e-3, relu)
        loss = lambda X_, g_, b_: _dot(oracle_mod.groupnorm(X_, groups, g_, b_, 1e-3, relu), G)
        for _ in range(3):
            D = rng.normal(size=X.shape)
            fd = (loss(X + h * D, gam, bet) - loss(X - h * D, gam, bet)) / (2 * h)
            assert abs(fd - _dot(dX, D)) <= 1e-6 * max(1.0, abs(fd)), (n, C, groups, relu, fd, _dot(dX, D))
            e = rng.normal(size=C)
            fd = (loss(X, gam + h * e, bet) - loss(X, gam - h * e, bet)) / (2 * h)
            assert abs(fd - _dot(dg, e)) <= 1e-6 * max(1.0, abs(fd)), (n, C, groups, relu)
            fd = (loss(X, gam, bet + h * e) - loss(X, gam, bet - h * e)) / (2 * h)
            assert abs(fd - _dot(db, e)) <= 1e-6 * max(1.0, abs(fd)), (n, C, groups, relu)


def test_groupnorm_backward_invariances(oracle_mod):
    """GN's output does not change when one group's inputs are shifted by a
    constant, so each group's input gradient sums to zero (any loss, ReLU or
    not); with eps = 0 it does not change when a group is scaled either, so
    sum (x - mean_g) dX = 0 per group.  Two values of a group normalise to
    -1 and +1 whatever they are: their gradient is zero."""
    rng = np.random.default_rng(72)
    X = rng.normal(size=(60, 16)) * 2 + 3
    G = rng.normal(size=(60, 16))
    gam, bet = rng.normal(size=16), rng.normal(size=16)
    for groups, relu in ((4, False), (4, True), (16, True), (1, False)):
        per = 16 // groups
        for eps in (1e-5, 0.0):
            dX, _, _ = oracle_mod.groupnorm_backward(X, G, groups, gam, bet, eps, relu)
            for g in range(groups):
                blk = slice(g * per, (g + 1) * per)
                scale = np.abs(dX[:, blk]).sum()
                assert abs(dX[:, blk].sum()) <= 1e-12 * scale
                if eps == 0.0:
                    xc = X[:, blk] - X[:, blk].mean()
                    assert abs((xc * dX[:, blk]).sum()) <= 1e-12 * np.abs(xc * dX[:, blk]).sum()
    dX, dg, db = oracle_mod.groupnorm_backward(np.array([[0.0], [2.0]]), np.array([[1.0], [0.0]]), 1, eps=0.0)
    assert np.abs(dX).max() < 1e-15
    assert dg[0] == -1.0 and db[0] == 1.0       # sum dY xhat with xhat = (-1, +1); sum dY


def test_preact_conv_backward_composite(oracle_mod):
    """L = <conv(relu(GN(X)), W) + b, G> over the three forms (1-hop,
    strided, Upsample): the chain conv backward (on relu(GN(X))) then GN
    backward (with the ReLU) matches central differences of the forward in
    X, W, b, gamma and beta."""
    h = 1e-6
    rng = np.random.default_rng(73)
    for name, dst, src, fwd in _conv_forms(oracle_mod, 73):
        C, Co, groups = 8, 5, 4
        X = rng.normal(size=(src.n, C)) * 1.5 + 0.5
        W = rng.normal(size=(9, C, Co))
        b = rng.normal(size=Co) * 0.5
        gam, bet = rng.normal(size=C), rng.normal(size=C) * 0.3
        G = rng.normal(size=(dst.n, Co))
        A = oracle_mod.groupnorm(X, groups, gam, bet, 1e-5, relu=True)
        dA, dW, db = dst.conv_backward(src, A, W, G)
        dX, dg, dbe = oracle_mod.groupnorm_backward(X, dA, groups, gam, bet, 1e-5, relu=True)

        def loss(X_, W_, b_, g_, be_):
            return _dot(fwd(oracle_mod.groupnorm(X_, groups, g_, be_, 1e-5, relu=True), W_, b_, False), G)

        base = (X, W, b, gam, bet)
        for i, grad in enumerate((dX, dW, db, dg, dbe)):
            D = rng.normal(size=base[i].shape)
            up = list(base)
            dn = list(base)
            up[i] = base[i] + h * D
            dn[i] = base[i] - h * D
            fd = (loss(*up) - loss(*dn)) / (2 * h)
            assert abs(fd - _dot(grad, D)) <= 1e-6 * max(1.0, abs(fd)), (name, i, fd, _dot(grad, D))


def test_deform_slice_classify_backward_finite_differences(oracle_mod):
    """L = <classify(X, wv, beta, Wc, bc), Z>: central differences in random
    directions of X, wv, Wc and bc, and in beta, match the gradients."""
    h = 1e-6
    L = oracle_mod.Lattice.create(_tiny_cloud(74, 250, 0.6), np.full(3, 0.1, np.float32))
    rng = np.random.default_rng(74)
    C, K = 8, 5
    X = rng.normal(size=(L.n, C))
    wv = rng.normal(size=C) * 0.5
    Wc, bc = rng.normal(size=(K, C)), rng.normal(size=K)
    Z = rng.normal(size=(L.m, K))
    dX, dwv, dbeta, dWc, dbc = L.deform_slice_classify_backward(X, wv, 0.15, Wc, Z)
    loss = lambda X_, w_, be_, Wc_, bc_: _dot(L.deform_slice_classify(X_, w_, be_, Wc_, bc_), Z)
    base = (X, wv, 0.15, Wc, bc)
    for i, grad in enumerate((dX, dwv, dbeta, dWc, dbc)):
        D = rng.normal(size=np.shape(base[i])) if i != 2 else 1.0
        up = list(base)
        dn = list(base)
        up[i] = base[i] + h * D
        dn[i] = base[i] - h * D
        fd = (loss(*up) - loss(*dn)) / (2 * h)
        an = _dot(grad, D) if i != 2 else grad
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(fd)), (i, fd, an)


def test_distribute_backward_finite_differences(oracle_mod):
    """L = <Distribute+PointNet(G, F), D>: central differences in random
    directions of F, of each layer's weights and bias and of the three
    normalisations' gamma and beta match the gradients (tiny cloud, widths
    8/16/16, with and without features)."""
    h = 1e-6
    O = oracle_mod
    for seed, cf in ((93, 3), (94, 0)):
        G = _tiny_cloud(seed, m=120)
        st = Stream(seed, "dist-bwd")
        F = st.normal(120 * cf).reshape(120, cf) if cf else None
        cin = 3 + cf
        layers = _pointnet_layers(st, cin, (8, 16, 16))
        ng = cin + 8 + 16
        gam, bet = 1.0 + 0.2 * st.normal(ng), 0.2 * st.normal(ng)
        ol = O.Lattice.create(G, np.full(3, 0.2, np.float32))
        Gd = G.astype(np.float64)
        D = st.normal(ol.n * 16).reshape(ol.n, 16)
        gr = ol.distribute_pointnet_backward(Gd, F, layers, D, (gam, bet))

        def loss(F_, layers_, gam_, bet_):
            return _dot(ol.distribute_pointnet(Gd, F_, layers_, (gam_, bet_)), D)

        rng = np.random.default_rng(seed)
        checks = []
        if cf:
            E = rng.normal(size=F.shape)
            checks.append((lambda t, E=E: loss(F + t * E, layers, gam, bet), _dot(gr["dF"], E), "dF"))
        for li in range(3):
            for j, name in ((0, f"dW{li + 1}"), (1, f"db{li + 1}")):
                E = rng.normal(size=layers[li][j].shape)

                def f(t, li=li, j=j, E=E):
                    ls = [list(x) for x in layers]
                    ls[li][j] = ls[li][j] + t * E
                    return loss(F, [tuple(x) for x in ls], gam, bet)
                checks.append((f, _dot(gr[name], E), name))
        E = rng.normal(size=ng)
        checks.append((lambda t, E=E: loss(F, layers, gam + t * E, bet), _dot(gr["dgamma"], E), "dgamma"))
        checks.append((lambda t, E=E: loss(F, layers, gam, bet + t * E), _dot(gr["dbeta"], E), "dbeta"))
        for f, an, name in checks:
            fd = (f(h) - f(-h)) / (2 * h)
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(fd)), (seed, name, fd, an)
        m = gr["margin"]
        assert (m >= 0).all()
        single = np.bincount(ol.simplices()[0].reshape(-1), minlength=ol.n) == 1
        assert np.isinf(m[single]).all() and np.isfinite(m[~single]).all()


def test_distribute_backward_routes_to_the_maximum(oracle_mod):
    """Only the row holding a channel's maximum receives that channel's
    gradient: with dX one-hot at (v, c), dW3 is the outer product e_c a_2^T
    of that single row, so db3 = e_c exactly."""
    O = oracle_mod
    G = _tiny_cloud(95, m=80)
    st = Stream(95, "dist-bwd2")
    layers = _pointnet_layers(st, 3, (8, 16, 16))
    ol = O.Lattice.create(G, np.full(3, 0.2, np.float32))
    D = np.zeros((ol.n, 16))
    v = int(np.argmax(np.bincount(ol.simplices()[0].reshape(-1), minlength=ol.n)))   # the vertex with most points
    D[v, 5] = 1.0
    gr = O.Lattice.distribute_pointnet_backward(ol, G.astype(np.float64), None, layers, D)
    e5 = np.zeros(16)
    e5[5] = 1.0
    assert np.array_equal(gr["db3"], e5)
    assert np.abs(gr["dW3"][np.arange(16) != 5]).max() == 0.0
