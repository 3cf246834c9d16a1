"""GPU parity: liblattice (HIP, gfx950) against the CPU oracle.

Structure (vertex keys, per-point simplices and weights, neighbour tables)
must match bit for bit after ordering vertices by key; features within
1e-4 (fp32) / 2e-2 (bf16) in the per-tensor relative-plus-RMS bound.
Every call goes through the C ABI via the ctypes binding.
"""
from __future__ import annotations

import ctypes
import json
import os

import numpy as np
import pytest

from tests import parity as P
from tests.oracle_pipeline import OraclePipeline
from workloads import configs
from workloads.rng import Stream

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1912_05905_amd import lattice
    lattice.lib()
    return lattice


@pytest.fixture(scope="module")
def O():
    from oracle import oracle
    oracle.lib()
    return oracle


def _cloud(seed, m, extent=1.0):
    st = Stream(seed, "gpu-cloud")
    return (extent * st.uniform(3 * m).reshape(m, 3)).astype(np.float32)


def _dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t if dtype is None else t.to(dtype)


def _host(t):
    torch.cuda.synchronize()
    return t.float().cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy()


def _check_structure(gl, ol):
    """Keys, simplices and neighbour table bit-exact; returns gpu2orc."""
    assert gl.n == ol.n and gl.m == ol.m
    g2o = P.key_permutation(_host(gl.keys()), ol.keys())
    gidx, gw = gl.simplices()
    oidx, ow = ol.simplices()
    assert np.array_equal(P.remap_index(_host(gidx), g2o), oidx), "simplex vertices differ"
    assert np.array_equal(_host(gw), ow), "barycentric weights differ"
    gnb = P.rows_in_oracle_order(P.remap_index(_host(gl.neighbors()), g2o), g2o)
    assert np.array_equal(gnb, ol.neighbors()), "neighbour tables differ"
    return g2o


# ----------------------------------------------------------------------------
# structure
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("seed,m,sigma", [(0, 1, 0.1), (1, 37, 0.1), (2, 1000, 0.05),
                                          (3, 4097, 0.1), (4, 20_000, 0.03)])
def test_create_structure_random(L, O, seed, m, sigma):
    pos = _cloud(seed, m)
    gl = L.Lattice.create(_dev(pos), [sigma] * 3)
    ol = O.Lattice.create(pos, np.full(3, sigma, np.float32))
    _check_structure(gl, ol)


def test_create_structure_adversarial(L, O):
    """Points on lattice vertices, faces and ties; duplicates; one simplex
    shared by thousands of points (insert contention)."""
    a = O.axis_factors(np.ones(3, np.float32)).astype(np.float64)
    grid = np.stack(np.meshgrid(*[np.arange(-3, 4)] * 3, indexing="ij"), -1).reshape(-1, 3) / a
    half = grid * 0.5
    same = np.tile(np.array([[0.123, 0.456, 0.789]]), (5000, 1))
    pos = np.concatenate([grid, half, same, grid[:50]], 0).astype(np.float32)
    gl = L.Lattice.create(_dev(pos), [1.0] * 3)
    ol = O.Lattice.create(pos, np.ones(3, np.float32))
    _check_structure(gl, ol)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_create_structure_configs(L, O, cfg):
    wl = configs.make(cfg)
    gl = L.Lattice.create(_dev(wl.positions), wl.sigma)
    ol = O.Lattice.create(wl.positions, wl.sigma)
    _check_structure(gl, ol)


@pytest.mark.parametrize("cfg,on_stream", [(2, False), (4, False), (4, True)])
def test_coarsen_structure(L, O, cfg, on_stream):
    wl = configs.make(cfg)
    gl = L.Lattice.create(_dev(wl.positions), wl.sigma)
    ol = O.Lattice.create(wl.positions, wl.sigma)
    glv, olv = [gl], [ol]
    for lvl in range(1, 4):
        glv.append(glv[-1].coarsen(on_stream=on_stream))
        olv.append(olv[-1].coarsen())
        assert glv[-1].level == lvl
        lv_c, m_c = ctypes.c_int(), ctypes.c_int64()
        assert L.lib().lattice_level(glv[-1].handle, ctypes.byref(lv_c)) == 0 and lv_c.value == lvl
        assert L.lib().lattice_num_points(glv[-1].handle, ctypes.byref(m_c)) == 0 and m_c.value == gl.m
        _check_structure(glv[-1], olv[-1])


@pytest.mark.parametrize("on_stream", [False, True])
def test_structure_of_large_inserts(L, O, on_stream):
    """A 300k-point cloud at a fine scale (about a thousand insert
    workgroups contending for the vertex counter, most vertices met by a
    single point): the level and its coarsening are bit-exact against the
    oracle, on the library's side stream and on the caller's."""
    pos = _cloud(1900 + int(on_stream), 300_000, 1.0)
    gl = L.Lattice.create(_dev(pos), [0.01] * 3)
    ol = O.Lattice.create(pos, np.full(3, 0.01, np.float32))
    _check_structure(gl, ol)
    g1 = gl.coarsen(on_stream=on_stream)
    o1 = ol.coarsen()
    _check_structure(g1, o1)
    g1.destroy()
    gl.destroy()


def test_empty_cloud(L):
    gl = L.Lattice.create(torch.zeros((0, 3), device="cuda"), [0.1] * 3)
    assert gl.n == 0 and gl.m == 0
    x = gl.splat(torch.zeros((0, 8), device="cuda"))
    assert x.shape == (0, 8)
    y = gl.conv(gl, x, torch.zeros((9, 16, 8), device="cuda"))
    assert y.shape == (0, 16)
    assert gl.slice(y).shape == (0, 16)
    c = gl.coarsen()
    assert c.n == 0


# ----------------------------------------------------------------------------
# errors found on the device
# ----------------------------------------------------------------------------
def test_device_errors(L):
    pos = _cloud(5, 1000)
    bad = pos.copy()
    bad[17, 1] = np.nan
    # creation does not wait: the error comes with the first read of n
    gl = L.Lattice.create(_dev(bad), [0.1] * 3)
    with pytest.raises(L.LatticeError) as e:
        gl.n
    assert e.value.status == -6
    far = pos.copy()
    far[3] = [1e6, 0, 0]
    with pytest.raises(L.LatticeError) as e:
        L.Lattice.create(_dev(far), [0.1] * 3).n
    assert e.value.status == -5
    # a coarse level enqueued from a failed one reports the parent's error,
    # and so does every later call on the parent
    gl = L.Lattice.create(_dev(_cloud(6, 5000)), [0.01] * 3, capacity_hint=16)
    gc = gl.coarsen()
    with pytest.raises(L.LatticeError) as e:
        gc.n
    assert e.value.status == -4
    with pytest.raises(L.LatticeError) as e:
        gl.keys()
    assert e.value.status == -4
    # the library stays usable after device-side errors
    ok = L.Lattice.create(_dev(pos), [0.1] * 3)
    assert ok.n > 0


def test_overflow_rebuild_of_a_hierarchy(L, O):
    """Points far apart on the lattice's scale: nearly 4 vertices per point
    overflow the table sized from the point count.  The coarse levels are
    enqueued before the fine level's count is read back, so each is built
    from a table that overflowed; the first read rebuilds the fine level,
    then each coarse level from the rebuilt one.  Structure and the
    strided / transposed convolutions must match the oracle."""
    pos = _cloud(71, 3000, 1.0)
    sigma = 0.002
    g0 = L.Lattice.create(_dev(pos), [sigma] * 3)
    g1 = g0.coarsen()
    g2 = g1.coarsen()
    o0 = O.Lattice.create(pos, np.full(3, sigma, np.float32))
    o1 = o0.coarsen()
    o2 = o1.coarsen()
    assert o0.n > 2 * 3000 * 1.3          # beyond the first table's reach
    g2o = [_check_structure(g, o) for g, o in ((g2, o2), (g1, o1), (g0, o0))][::-1]
    rng = np.random.default_rng(12)
    for (gf, of, pf), (gc, oc, pc) in (((g0, o0, g2o[0]), (g1, o1, g2o[1])), ((g1, o1, g2o[1]), (g2, o2, g2o[2]))):
        Xf = rng.normal(size=(of.n, 16))
        Wd = _rand_w(rng, 16, 32, 1.0 / 12)
        gy = gc.conv(gf, _dev(Xf[pf].astype(np.float32)), _gpu_w(Wd.astype(np.float32), torch.float32))
        P.assert_close(P.rows_in_oracle_order(_host(gy), pc), oc.conv(of, Xf, Wd), P.TOL_F32, "strided conv")
        Xc = rng.normal(size=(oc.n, 32))
        Wu = _rand_w(rng, 32, 16, 1.0 / 12)
        gz = gf.refine(gc, _dev(Xc[pc].astype(np.float32)), _gpu_w(Wu.astype(np.float32), torch.float32))
        P.assert_close(P.rows_in_oracle_order(_host(gz), pf), of.refine_into(oc, Xc, Wu), P.TOL_F32,
                       "transposed conv")


def _check_down_up(rng, g2o, levels_g, levels_o):
    """Strided and transposed convolutions between consecutive levels (the
    Downsample and Upsample tables) against the oracle."""
    for (gf, of, pf), (gc, oc, pc) in zip(list(zip(levels_g, levels_o, g2o))[:-1],
                                          list(zip(levels_g, levels_o, g2o))[1:]):
        Xf = rng.normal(size=(of.n, 16))
        Wd = _rand_w(rng, 16, 32, 1.0 / 12)
        gy = gc.conv(gf, _dev(Xf[pf].astype(np.float32)), _gpu_w(Wd.astype(np.float32), torch.float32))
        P.assert_close(P.rows_in_oracle_order(_host(gy), pc), oc.conv(of, Xf, Wd), P.TOL_F32, "strided conv")
        Xc = rng.normal(size=(oc.n, 32))
        Wu = _rand_w(rng, 32, 16, 1.0 / 12)
        gz = gf.refine(gc, _dev(Xc[pc].astype(np.float32)), _gpu_w(Wu.astype(np.float32), torch.float32))
        P.assert_close(P.rows_in_oracle_order(_host(gz), pf), of.refine_into(oc, Xc, Wu), P.TOL_F32,
                       "transposed conv")


@pytest.mark.parametrize("cfg,levels", [(2, 3), (4, 3), (4, 1)])
def test_create_hierarchy(L, O, cfg, levels):
    """lattice_create_hierarchy (one call, tables cleared together, inserts
    of all levels in one launch, tables in one launch, row orders batched)
    gives the lattices of create +
    coarsen: every level bit-exact, the Downsample / Upsample tables through
    the strided and transposed convolutions, and a splat on the coarsest
    level (whose lists are built on first use)."""
    wl = configs.make(cfg)
    gls = L.Lattice.create_hierarchy(_dev(wl.positions), wl.sigma, levels)
    ols = [O.Lattice.create(wl.positions, wl.sigma)]
    for _ in range(levels - 1):
        ols.append(ols[-1].coarsen())
    g2o = [_check_structure(g, o) for g, o in zip(gls, ols)]
    _check_down_up(np.random.default_rng(31 + cfg), g2o, gls, ols)
    F = np.random.default_rng(5).normal(size=(wl.m, 8)).astype(np.float32)
    gv = gls[-1].splat(_dev(F))
    P.assert_close(P.rows_in_oracle_order(_host(gv), g2o[-1]), ols[-1].splat(F)[0], P.TOL_F32, "splat")
    for g in reversed(gls):
        g.destroy()


@pytest.mark.parametrize("hints", ["counts", "small", "negative"])
def test_create_hierarchy_capacity_hints(L, O, hints):
    """Hash tables sized from capacity hints: the vertex counts of the same
    cloud (compact tables), hints far too small, whose tables overflow and
    are rebuilt, or negative hints, which count as 0 (automatic); every
    level is bit-exact with the oracle."""
    wl = configs.make(4)
    ols = [O.Lattice.create(wl.positions, wl.sigma)]
    for _ in range(2):
        ols.append(ols[-1].coarsen())
    h = {"counts": [o.n for o in ols], "small": [5, 5, 5], "negative": [-7, 0, -1]}[hints]
    gls = L.Lattice.create_hierarchy(_dev(wl.positions), wl.sigma, 3, capacity_hints=h)
    g2o = [_check_structure(g, o) for g, o in zip(gls, ols)]
    _check_down_up(np.random.default_rng(41), g2o, gls, ols)
    for g in reversed(gls):
        g.destroy()
    with pytest.raises(ValueError):
        L.Lattice.create_hierarchy(_dev(wl.positions), wl.sigma, 3, capacity_hints=[0, 0])


def test_coarsen_after_hierarchy(L, O):
    """A level coarsened from the coarsest level of a hierarchy starts from
    the elevated positions that the one-launch insert stored for it (the
    finest level's, halved once per level): bit-exact with the oracle's
    third level."""
    wl = configs.make(4)
    gls = L.Lattice.create_hierarchy(_dev(wl.positions), wl.sigma, 2)
    g2 = gls[1].coarsen()
    ols = [O.Lattice.create(wl.positions, wl.sigma)]
    for _ in range(2):
        ols.append(ols[-1].coarsen())
    _check_structure(g2, ols[2])
    g2.destroy()
    for g in reversed(gls):
        g.destroy()


def test_create_hierarchy_overflow_rebuild(L, O):
    """A hierarchy built in one call from points far apart on the lattice's
    scale: every level's first table overflows (nearly 4 vertices per
    point), the first read rebuilds the fine level and then each coarse
    level from the rebuilt one, as for create + coarsen."""
    pos = _cloud(72, 3000, 1.0)
    sigma = 0.002
    gls = L.Lattice.create_hierarchy(_dev(pos), [sigma] * 3, 3)
    ols = [O.Lattice.create(pos, np.full(3, sigma, np.float32))]
    for _ in range(2):
        ols.append(ols[-1].coarsen())
    assert ols[0].n > 2 * 3000 * 1.3
    g2o = [_check_structure(g, o) for g, o in zip(gls[::-1], ols[::-1])][::-1]
    _check_down_up(np.random.default_rng(13), g2o, gls, ols)


def test_rebuild_ordered_for_another_stream(L, O):
    """A lattice built on one stream whose table overflows is rebuilt there
    by the first call that needs its vertex count; an operator called on
    another stream (here with other work still queued on the first) is
    ordered after that rebuild, without host synchronisation."""
    pos = _cloud(73, 3000, 1.0)
    sigma = 0.002
    F = np.random.default_rng(74).normal(size=(3000, 8)).astype(np.float32)
    pd, Fd = _dev(pos), _dev(F)
    big = torch.randn((2048, 2048), device="cuda")
    torch.cuda.synchronize()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(sa):
        gl = L.Lattice.create(pd, [sigma] * 3)
        for _ in range(8):
            big = big @ big * 1e-3            # keeps the build stream busy
    with torch.cuda.stream(sb):
        got = gl.splat(Fd)
    torch.cuda.synchronize()
    ol = O.Lattice.create(pos, np.full(3, sigma, np.float32))
    assert ol.n > 2 * 3000 * 1.3              # beyond the first table's reach
    g2o = _check_structure(gl, ol)
    P.assert_close(P.rows_in_oracle_order(_host(got), g2o), ol.splat(F)[0], P.TOL_F32, "splat")
    gl.destroy()


def test_create_hierarchy_rejections(L):
    """Bad arguments return an error and create no handle; an empty cloud
    gives empty levels."""
    pos = torch.zeros((10, 3), device="cuda")
    for levels in (0, 9):
        with pytest.raises(L.LatticeError) as e:
            L.Lattice.create_hierarchy(pos, [0.1] * 3, levels)
        assert e.value.status == -1   # LAT_EINVAL
    with pytest.raises(L.LatticeError) as e:
        L.Lattice.create_hierarchy(pos, [0.1, 0.0, 0.1], 2)
    assert e.value.status == -1   # LAT_EINVAL
    for hints in (None, [10, 10, 10]):
        empty = L.Lattice.create_hierarchy(torch.zeros((0, 3), device="cuda"), [0.1] * 3, 3, capacity_hints=hints)
        assert [g.n for g in empty] == [0, 0, 0] and [g.level for g in empty] == [0, 1, 2]
        for g in reversed(empty):
            g.destroy()


def test_host_validation_on_gpu(L):
    gl = L.Lattice.create(_dev(_cloud(7, 500)), [0.1] * 3)
    x = torch.zeros((gl.n, 6), device="cuda")
    with pytest.raises(L.LatticeError) as e:
        gl.conv(gl, x, torch.zeros((9, 8, 6), device="cuda"))     # Cin % 4 != 0
    assert e.value.status == -2
    x = torch.zeros((gl.n, 8), device="cuda")
    with pytest.raises(L.LatticeError) as e:
        gl.conv(gl, x, torch.zeros((9, 8, 8), device="cuda"), out=x)   # in == out
    assert e.value.status == -1
    other = L.Lattice.create(_dev(_cloud(8, 500)), [0.1] * 3)
    with pytest.raises(L.LatticeError) as e:
        gl.conv(other, x, torch.zeros((9, 8, 8), device="cuda"))
    assert e.value.status == -8
    c = gl.coarsen()
    with pytest.raises(L.LatticeError) as e:
        gl.destroy()                                               # child alive
    assert e.value.status == -8
    c.destroy()
    gl.destroy()


# ----------------------------------------------------------------------------
# operators, one at a time, on the oracle's own inputs
# ----------------------------------------------------------------------------
def _pair(L, O, pos, sigma):
    gl = L.Lattice.create(_dev(pos), [sigma] * 3)
    ol = O.Lattice.create(pos, np.full(3, sigma, np.float32))
    g2o = P.key_permutation(_host(gl.keys()), ol.keys())
    return gl, ol, g2o


@pytest.mark.parametrize("C,normalize", [(4, True), (8, True), (36, False), (64, True), (256, True), (320, False),
                                         (512, True)])
def test_splat(L, O, C, normalize):
    pos = _cloud(10 + C, 9000, 0.7)
    gl, ol, g2o = _pair(L, O, pos, 0.06)
    F = np.random.default_rng(C).normal(size=(pos.shape[0], C)).astype(np.float32)
    ws = torch.empty(gl.n, device="cuda")
    gx = gl.splat(_dev(F), normalize=normalize, wsum=ws)
    ox, ow = ol.splat(F.astype(np.float64), normalize=normalize)
    P.assert_close(P.rows_in_oracle_order(_host(gx), g2o), ox, P.TOL_F32, "splat")
    P.assert_close(P.rows_in_oracle_order(_host(ws), g2o), ow, P.TOL_F32, "wsum")


@pytest.mark.parametrize("C,dtype", [(4, "f32"), (36, "f32"), (64, "f32"), (256, "f32"), (512, "f32"), (64, "bf16"),
                                     (512, "bf16"), (1024, "bf16")])
def test_splat_skewed(L, O, C, dtype):
    """Vertex lists far longer than a workgroup span (a 6000-point clump
    inside one simplex), next to short ones and a ragged end."""
    rng = np.random.default_rng(C)
    clump = (np.array([0.31, 0.42, 0.53]) + 1e-4 * rng.random((6000, 3))).astype(np.float32)
    spread = rng.random((3001, 3)).astype(np.float32)
    pos = np.concatenate([spread[:1500], clump, spread[1500:]]).astype(np.float32)
    gl, ol, g2o = _pair(L, O, pos, 0.05)
    F = rng.normal(size=(pos.shape[0], C)).astype(np.float32)
    if dtype == "bf16":
        F = O.round_bf16(F).astype(np.float32)
        gx = gl.splat(_dev(F, torch.bfloat16))
        ox, _ = ol.splat(F.astype(np.float64))
        P.assert_close(P.rows_in_oracle_order(_host(gx), g2o), O.round_bf16(ox), P.TOL_BF16, "skewed splat bf16")
    else:
        ws = torch.empty(gl.n, device="cuda")
        gx = gl.splat(_dev(F), wsum=ws)
        ox, ow = ol.splat(F.astype(np.float64))
        P.assert_close(P.rows_in_oracle_order(_host(gx), g2o), ox, P.TOL_F32, "skewed splat")
        P.assert_close(P.rows_in_oracle_order(_host(ws), g2o), ow, P.TOL_F32, "skewed wsum")


@pytest.mark.parametrize("m,C,dtype", [(300_000, 64, "f32"), (600_000, 64, "f32"), (600_000, 36, "f32"),
                                       (600_000, 64, "bf16"), (300_000, 128, "bf16")])
def test_splat_long_chunks(L, O, m, C, dtype):
    """Clouds with over a million list entries, where a lane group takes 32
    or 64 entries per chunk instead of 16, with a 20,000-point clump in one
    simplex (a list that runs through many chunks and workgroup spans)."""
    rng0 = np.random.default_rng(m)
    clump = (np.array([0.31, 0.42, 0.53]) + 1e-5 * rng0.random((20_000, 3))).astype(np.float32)
    spread = _cloud(700 + C, m, 0.9)
    pos = np.concatenate([spread[: m // 3], clump, spread[m // 3:]]).astype(np.float32)
    gl, ol, g2o = _pair(L, O, pos, 0.02)
    rng = np.random.default_rng(m + C)
    F = rng.normal(size=(pos.shape[0], C)).astype(np.float32)
    if dtype == "bf16":
        F = O.round_bf16(F).astype(np.float32)
        gx = gl.splat(_dev(F, torch.bfloat16))
        ox, _ = ol.splat(F.astype(np.float64))
        P.assert_close(P.rows_in_oracle_order(_host(gx), g2o), O.round_bf16(ox), P.TOL_BF16, "splat bf16")
    else:
        ws = torch.empty(gl.n, device="cuda")
        gx = gl.splat(_dev(F), wsum=ws)
        ox, ow = ol.splat(F.astype(np.float64))
        P.assert_close(P.rows_in_oracle_order(_host(gx), g2o), ox, P.TOL_F32, "splat")
        P.assert_close(P.rows_in_oracle_order(_host(ws), g2o), ow, P.TOL_F32, "wsum")


def test_splat_bf16(L, O):
    pos = _cloud(31, 9000, 0.7)
    gl, ol, g2o = _pair(L, O, pos, 0.06)
    F = np.random.default_rng(3).normal(size=(pos.shape[0], 64)).astype(np.float32)
    Fb = O.round_bf16(F)
    gx = gl.splat(_dev(Fb.astype(np.float32), torch.bfloat16))
    ox, _ = ol.splat(Fb)
    P.assert_close(P.rows_in_oracle_order(_host(gx), g2o), O.round_bf16(ox), P.TOL_BF16, "splat bf16")


def _rand_w(rng, cin, cout, std):
    return (std * rng.normal(size=(9, cin, cout))).astype(np.float32)


def _gpu_w(W, dtype=torch.float32):
    return _dev(np.ascontiguousarray(np.transpose(W, (0, 2, 1))), dtype).contiguous()


@pytest.mark.parametrize("cin,cout", [(8, 16), (4, 4), (12, 20), (64, 64), (32, 96), (128, 128),
                                      (256, 64)])
def test_conv_fp32(L, O, cin, cout):
    pos = _cloud(40 + cin, 6000, 0.8)
    gl, ol, g2o = _pair(L, O, pos, 0.07)
    rng = np.random.default_rng(cin * 1000 + cout)
    X = rng.normal(size=(ol.n, cin)).astype(np.float32)
    W = _rand_w(rng, cin, cout, 1.0 / np.sqrt(9 * cin))
    b = rng.normal(size=cout).astype(np.float32)
    Xg = np.empty_like(X)
    Xg[np.arange(ol.n)] = X[g2o]          # GPU row v holds oracle row g2o[v]
    for relu in (False, True):
        gy = gl.conv(gl, _dev(Xg), _gpu_w(W), bias=_dev(b), relu=relu)
        oy = ol.conv(ol, X.astype(np.float64), W.astype(np.float64), bias=b.astype(np.float64), relu=relu)
        P.assert_close(P.rows_in_oracle_order(_host(gy), g2o), oy, P.TOL_F32, f"conv {cin}->{cout}")


def test_conv_input_beyond_buffer_reach(L, O):
    """An input whose rows span more than 2 GiB (a wide row stride) takes the
    convolution path without buffer resources."""
    pos = _cloud(77, 3000, 0.8)
    gl, ol, g2o = _pair(L, O, pos, 0.07)
    cin = cout = 64
    ld = ((2**31 // (4 * max(ol.n - 1, 1)) + 64) // 8) * 8
    assert (ol.n - 1) * ld * 4 > 2**31
    rng = np.random.default_rng(77)
    X = rng.normal(size=(ol.n, cin)).astype(np.float32)
    W = _rand_w(rng, cin, cout, 1.0 / np.sqrt(9 * cin))
    big = torch.empty((ol.n, ld), dtype=torch.float32, device="cuda")
    big[:, :cin] = _dev(X[g2o])
    gy = gl.conv(gl, big[:, :cin], _gpu_w(W), relu=True)
    del big
    oy = ol.conv(ol, X.astype(np.float64), W.astype(np.float64), relu=True)
    P.assert_close(P.rows_in_oracle_order(_host(gy), g2o), oy, P.TOL_F32, "conv, 2 GiB input")


@pytest.mark.parametrize("cin,cout", [(64, 64), (8, 24), (128, 192), (384, 192), (256, 256)])
def test_conv_bf16(L, O, cin, cout):
    pos = _cloud(50 + cin, 6000, 0.8)
    gl, ol, g2o = _pair(L, O, pos, 0.07)
    rng = np.random.default_rng(cin + 7 * cout)
    X = O.round_bf16(rng.normal(size=(ol.n, cin)))
    W = O.round_bf16(_rand_w(rng, cin, cout, 1.0 / np.sqrt(9 * cin)))
    Xg = X[g2o].astype(np.float32)
    gy = gl.conv(gl, _dev(Xg, torch.bfloat16), _gpu_w(W.astype(np.float32), torch.bfloat16), relu=True)
    oy = O.round_bf16(ol.conv(ol, X, W, relu=True))
    P.assert_close(P.rows_in_oracle_order(_host(gy), g2o), oy, P.TOL_BF16, f"bf16 conv {cin}->{cout}")


def test_conv_column_slices(L, O):
    """Input and output as column ranges of wider buffers (concatenation)."""
    pos = _cloud(60, 5000, 0.8)
    gl, ol, g2o = _pair(L, O, pos, 0.07)
    rng = np.random.default_rng(9)
    X = rng.normal(size=(ol.n, 32)).astype(np.float32)
    W = _rand_w(rng, 32, 16, 0.1)
    big_in = torch.zeros((gl.n, 96), device="cuda")
    big_in[:, 32:64] = _dev(X[g2o])
    big_out = torch.full((gl.n, 48), 7.0, device="cuda")
    gl.conv(gl, big_in[:, 32:64], _gpu_w(W), out=big_out[:, 16:32])
    oy = ol.conv(ol, X.astype(np.float64), W.astype(np.float64))
    h = _host(big_out)
    P.assert_close(P.rows_in_oracle_order(h[:, 16:32], g2o), oy, P.TOL_F32, "sliced conv")
    assert (h[:, :16] == 7.0).all() and (h[:, 32:] == 7.0).all()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_strided_and_transposed_conv(L, O, dtype):
    pos = _cloud(70, 8000, 0.8)
    sigma = 0.05
    gl = L.Lattice.create(_dev(pos), [sigma] * 3)
    ol = O.Lattice.create(pos, np.full(3, sigma, np.float32))
    gc, oc = gl.coarsen(), ol.coarsen()
    g2o_f = P.key_permutation(_host(gl.keys()), ol.keys())
    g2o_c = P.key_permutation(_host(gc.keys()), oc.keys())
    rng = np.random.default_rng(11)
    bf = dtype == "bf16"
    tdt = torch.bfloat16 if bf else torch.float32
    rnd = O.round_bf16 if bf else (lambda a: np.asarray(a, np.float64))
    tol = P.TOL_BF16 if bf else P.TOL_F32
    Xf = rnd(rng.normal(size=(ol.n, 64)))
    Wd = rnd(_rand_w(rng, 64, 128, 1.0 / 24))
    gy = gc.conv(gl, _dev(Xf[g2o_f].astype(np.float32), tdt), _gpu_w(Wd.astype(np.float32), tdt))
    oy = rnd(oc.conv(ol, Xf, Wd))
    P.assert_close(P.rows_in_oracle_order(_host(gy), g2o_c), oy, tol, "strided conv")
    Xc = rnd(rng.normal(size=(oc.n, 128)))
    Wu = rnd(_rand_w(rng, 128, 64, 1.0 / 24))
    gz = gl.refine(gc, _dev(Xc[g2o_c].astype(np.float32), tdt), _gpu_w(Wu.astype(np.float32), tdt), relu=True)
    oz = rnd(ol.refine_into(oc, Xc, Wu, relu=True))
    P.assert_close(P.rows_in_oracle_order(_host(gz), g2o_f), oz, tol, "transposed conv")


def test_coarse_levels_used_on_another_stream(L, O):
    """Coarse levels are built on the library's own stream.  A second caller
    stream that is ordered only after the coarsen calls were issued (not
    after the builds themselves) must still see finished tables, and their
    point lists built on first use there."""
    pos = _cloud(72, 9000, 0.8)
    sigma = 0.05
    o0 = O.Lattice.create(pos, np.full(3, sigma, np.float32))
    o1 = o0.coarsen()
    o2 = o1.coarsen()
    rng = np.random.default_rng(13)
    Xf = rng.normal(size=(o0.n, 32))
    Wd = _rand_w(rng, 32, 64, 1.0 / 16)
    W2 = _rand_w(rng, 64, 32, 1.0 / 24)
    Wdev, W2dev, posdev = _gpu_w(Wd), _gpu_w(W2), _dev(pos)
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(s1):
        g0 = L.Lattice.create(posdev, [sigma] * 3)
        g1 = g0.coarsen()
        g2 = g1.coarsen()
    s2.wait_stream(s1)
    with torch.cuda.stream(s2):
        g2o0 = P.key_permutation(_host(g0.keys()), o0.keys())
        x = _dev(Xf[g2o0].astype(np.float32))
        y1 = g1.conv(g0, x, Wdev)
        y2 = g2.conv(g1, y1, W2dev)
        vals = g2.slice(y2)
    torch.cuda.synchronize()
    g2o1 = P.key_permutation(_host(g1.keys()), o1.keys())
    g2o2 = P.key_permutation(_host(g2.keys()), o2.keys())
    oy1 = o1.conv(o0, Xf, Wd)
    P.assert_close(P.rows_in_oracle_order(_host(y1), g2o1), oy1, P.TOL_F32, "strided conv, level 1")
    oy2 = o2.conv(o1, oy1, W2)
    P.assert_close(P.rows_in_oracle_order(_host(y2), g2o2), oy2, P.TOL_F32, "strided conv, level 2")
    P.assert_close(_host(vals), o2.slice(oy2), P.TOL_F32, "slice on level 2")
    for g in (g2, g1, g0):
        g.destroy()


@pytest.mark.parametrize("C,dtype", [(4, "f32"), (16, "f32"), (64, "f32"), (128, "f32"),
                                     (512, "f32"), (64, "bf16"), (256, "bf16")])
def test_slice_and_deform_slice(L, O, C, dtype):
    pos = _cloud(80 + C, 7000, 0.8)
    gl, ol, g2o = _pair(L, O, pos, 0.06)
    rng = np.random.default_rng(C)
    bf = dtype == "bf16"
    tdt = torch.bfloat16 if bf else torch.float32
    X = rng.normal(size=(ol.n, C))
    if bf:
        X = O.round_bf16(X)
    Xg = _dev(X[g2o].astype(np.float32), tdt)
    P.assert_close(_host(gl.slice(Xg)), ol.slice(X), P.TOL_F32, "slice")
    if C <= 256:
        wv = (rng.normal(size=C) / np.sqrt(C)).astype(np.float32)
        delta = torch.empty((gl.m, 4), device="cuda")
        out = gl.deform_slice(Xg, _dev(wv), 0.1, delta=delta)
        oo, od = ol.deform_slice(X, wv.astype(np.float64), 0.1)
        P.assert_close(_host(out), oo, P.TOL_F32, "deform slice")
        P.assert_close(_host(delta), od, P.TOL_F32, "deform offsets")
        # both from one pass: the oracle's values, and the separate calls' bits
        s2, d2 = gl.slice_and_deform(Xg, _dev(wv), 0.1)
        P.assert_close(_host(s2), ol.slice(X), P.TOL_F32, "fused slice")
        P.assert_close(_host(d2), oo, P.TOL_F32, "fused deform slice")
        assert np.array_equal(_host(d2), _host(out)), "fused DeformSlice differs from the separate call"
        assert np.array_equal(_host(s2), _host(gl.slice(Xg))), "fused slice differs from the separate call"


# ----------------------------------------------------------------------------
# whole pipelines
# ----------------------------------------------------------------------------
def _step_checked(L, O, wl, olv=None, rng=None, rows_per_op=None, points=None):
    """One GPU step with every operator compared with the oracle as it runs,
    on the inputs the GPU stored for it (its source columns as the GPU wrote
    them, kept on the host as each operator finishes, so buffers reused
    later in the step do not matter): every comparison is one operator deep.
    Lattice structure bit-exact on every level.  Operators: splat and
    Distribute + PointNet on every vertex; convolutions (1-hop, strided,
    Upsample; pre-activated ones with GroupNorm over the whole stored input
    and the residual added) on all rows or on a seeded sample of
    rows_per_op; slice, DeformSlice and DeformSlice + classifier on all
    points or a sample of `points`.  Returns (levels, buffers, outputs,
    oracle levels, number of operators checked)."""
    from paper_1912_05905_amd.pipeline import GpuPipeline
    bf = wl.dtype == "bf16"
    rnd = O.round_bf16 if bf else (lambda a: a)
    tol = P.TOL_BF16 if bf else P.TOL_F32
    if olv is None:
        olv = {}
        for op in wl.ops:
            if op["op"] == "create":
                olv[0] = O.Lattice.create(wl.positions, wl.sigma)
            elif op["op"] == "coarsen":
                olv[op["level"]] = olv[op["level"] - 1].coarsen()
    state = {"g2o": None, "checked": 0}
    mirror = {}

    def cols(spec):
        name, c0, cc = spec
        return np.ascontiguousarray(mirror[name][:, c0:c0 + cc], dtype=np.float64)

    def sample_rows(n):
        if rows_per_op is None or n <= rows_per_op:
            return None
        return np.sort(rng.choice(n, size=rows_per_op, replace=False))

    def sample_points():
        if points is None or wl.m <= points:
            return None
        return np.sort(rng.choice(wl.m, size=points, replace=False))

    def after(i, op, levels, bufs, outs):
        torch.cuda.synchronize()
        if state["g2o"] is None:
            state["g2o"] = {lv: _check_structure(levels[lv], olv[lv]) for lv in sorted(levels)}
        g2o = state["g2o"]
        kind = op["op"]

        def gpu_cols(spec):
            name, c0, cc = spec
            return P.rows_in_oracle_order(_host(bufs[name][:, c0:c0 + cc]), g2o[wl.buffers[name][0]])

        what = f"op {i} {kind} -> {op.get('dst', op.get('out'))}"
        if kind == "splat":
            X, _ = olv[0].splat(wl.features.astype(np.float64), normalize=bool(op["normalize"]))
            P.assert_close(gpu_cols(op["dst"]), rnd(X), tol, what)
        elif kind == "distribute":
            layers = [tuple(a.astype(np.float64) for a in wl.mlp[n]) for n in op["layers"]]
            gn = tuple(a.astype(np.float64) for a in wl.norms[op["norm"]])
            X = olv[op["level"]].distribute_pointnet(wl.positions.astype(np.float64), wl.features.astype(np.float64),
                                                     layers, gn)
            P.assert_close(gpu_cols(op["dst"]), rnd(X), tol, what)
        elif kind in ("conv", "conv_down", "refine"):
            lv = op["level"]
            x = cols(op["src"])
            if "pre" in op:
                gam, bet = wl.norms[op["pre"]["norm"]]
                x = rnd(O.groupnorm(x, op["pre"]["groups"], gam.astype(np.float64), bet.astype(np.float64),
                                    eps=1e-5, relu=True))
            W = wl.weights[op["w"]].astype(np.float64)
            rows = sample_rows(olv[lv].n)
            if kind == "conv":
                y = olv[lv].conv(olv[lv], x, W, relu=op["relu"], rows=rows)
            elif kind == "conv_down":
                y = olv[lv].conv(olv[lv - 1], x, W, relu=op["relu"], rows=rows)
            else:
                y = olv[lv].refine_into(olv[lv + 1], x, W, relu=op["relu"], rows=rows)
            if "res" in op:
                r = cols(op["res"])
                y = y + (r if rows is None else r[rows])
            got = gpu_cols(op["dst"])
            P.assert_close(got if rows is None else got[rows], rnd(y), tol, what)
        elif kind in ("slice", "deform_slice", "deform_classify"):
            pts = sample_points()
            lat = olv[op["level"]]
            if kind == "slice":
                ref = lat.slice(cols(op["src"]), pts=pts)
            elif kind == "deform_slice":
                wv, beta = wl.vectors[op["wv"]]
                ref, _ = lat.deform_slice(cols(op["src"]), wv.astype(np.float64), beta, pts=pts)
            else:
                wv, beta = wl.vectors[op["wv"]]
                Wc, bc = wl.classifiers[op["cls"]]
                if pts is None:
                    ref = lat.deform_slice_classify(cols(op["src"]), wv.astype(np.float64), beta,
                                                    Wc.astype(np.float64), bc.astype(np.float64))
                else:
                    f, _ = lat.deform_slice(cols(op["src"]), wv.astype(np.float64), beta, pts=pts)
                    ref = f @ Wc.astype(np.float64).T + bc.astype(np.float64)
            got = _host(outs[op["out"]])
            P.assert_close(got if pts is None else got[pts], ref, P.TOL_F32, what)
        else:
            raise AssertionError(f"no stored-input check for operator {kind}")
        if "dst" in op:
            name, c0, cc = op["dst"]
            if name not in mirror:
                lv, total = wl.buffers[name]
                mirror[name] = np.zeros((olv[lv].n, total), np.float32)
            mirror[name][:, c0:c0 + cc] = gpu_cols(op["dst"])
        state["checked"] += 1

    levels, bufs, outs = GpuPipeline(wl).step(keep=True, after_op=after)
    return levels, bufs, outs, olv, state["checked"]


def _run_both(L, O, wl):
    """Whole pipeline on the GPU and in the oracle, structure bit-exact on
    every level.  fp32: every written column range and point output
    elementwise.  bf16: every operator elementwise on its stored inputs
    (_step_checked), and every tensor normwise end to end."""
    from paper_1912_05905_amd.pipeline import GpuPipeline
    bf = wl.dtype == "bf16"
    if bf:
        levels, bufs, outs, _, _ = _step_checked(L, O, wl)
    else:
        levels, bufs, outs = GpuPipeline(wl).step()
    olv, obufs, oouts = OraclePipeline(wl).run()
    tol = P.TOL_BF16 if bf else P.TOL_F32
    check = P.assert_normwise if bf else P.assert_close
    g2o = {}
    for lv in sorted(levels):
        g2o[lv] = _check_structure(levels[lv], olv[lv])
    written = []
    for op in wl.ops:
        if "dst" in op and op["dst"] not in written:
            written.append(op["dst"])
    for name, c0, cc in written:
        lv = wl.buffers[name][0]
        got = P.rows_in_oracle_order(_host(bufs[name]), g2o[lv])[:, c0:c0 + cc]
        check(got, obufs[name][:, c0:c0 + cc], tol, f"{name}[{c0}:{c0 + cc}]")
    for name in outs:
        check(_host(outs[name]), oouts[name], tol, name)
    return levels


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 6])
def test_pipeline_full_size(L, O, cfg):
    _run_both(L, O, configs.make(cfg))


def test_pipeline_config5_full_size_sampled(L, O):
    """The 1M-point bf16 U-Net at full size, operator by operator on the
    GPU's own inputs (the oracle would need minutes for the whole network):
    the four-level hierarchy bit-exact, splat on every vertex, each of the
    thirteen convolutions on a seeded sample of 4,000 output rows (1-hop,
    strided and Upsample, concatenated column ranges included), DeformSlice
    on 50,000 points."""
    from paper_1912_05905_amd.pipeline import GpuPipeline
    levels, _, _, _, checked = _step_checked(L, O, configs.make(5), rng=np.random.default_rng(55),
                                             rows_per_op=4000, points=50_000)
    assert checked == 15
    GpuPipeline.release(levels)


@pytest.mark.parametrize("cfg,K", [(5, 2), (10, 2), (6, 3), (8, 3), (9, 3)])
def test_pipeline_bench_layout(L, O, cfg, K):
    """Workloads as the bench runs them (K pipelines whose builds share one
    stream, steps on K compute streams with no host synchronisation between
    them): every step's point outputs match those of a step issued alone
    (whose operators the other tests check against the oracle); bf16
    normwise at the bf16 tolerance, fp32 elementwise (the steps build their
    own lattices, so sums are taken in other orders)."""
    from paper_1912_05905_amd.pipeline import GpuPipeline
    wl = configs.make(cfg)
    lv, _, ref = GpuPipeline(wl).step(keep=True)
    ref = {k: _host(v) for k, v in ref.items()}
    GpuPipeline.release(lv)
    assert ref
    bs = torch.cuda.Stream()
    pipes = [GpuPipeline(wl, overlap=True, build_stream=bs) for _ in range(K)]
    streams = [torch.cuda.current_stream()] + [torch.cuda.Stream() for _ in range(K - 1)]
    bf = wl.dtype == "bf16"
    kept = []
    for i in range(2 * K):
        k = i % K
        with torch.cuda.stream(streams[k]):
            levels, _, outs = pipes[k].step()
            kept.append({n: outs[n].clone() for n in outs})
            pipes[k].finish_step(levels)
        if bf:
            torch.cuda.synchronize()   # bound the clones of 1M-point outputs held at once
            got = kept.pop()
            assert set(got) == set(ref)
            for n, t in got.items():
                P.assert_normwise(_host(t), ref[n], P.TOL_BF16, n)
    torch.cuda.synchronize()
    for got in kept:
        assert set(got) == set(ref)
        for n, t in got.items():
            P.assert_close(_host(t), ref[n], P.TOL_F32, n)
    for p in pipes:
        p.flush()


def test_latticenet_bf16_full_size_sampled(L, O):
    """The LatticeNet forward on the 1M-point room in bf16 (workload 10) at
    full size, operator by operator on the GPU's own inputs: the three-level
    hierarchy bit-exact, Distribute + PointNet on every vertex, each of the
    twenty pre-activated convolutions (GroupNorm over the whole stored input)
    on 4,000 sampled rows with its residual, the fused DeformSlice +
    classifier on 50,000 points."""
    from paper_1912_05905_amd.pipeline import GpuPipeline
    print("latticenet bf16, 1M points, stored-input checks", flush=True)
    levels, _, _, _, checked = _step_checked(L, O, configs.make(10), rng=np.random.default_rng(56),
                                             rows_per_op=4000, points=50_000)
    assert checked == 22
    GpuPipeline.release(levels)


def test_latticenet_bf16_reduced(L, O):
    """The bf16 LatticeNet forward on a reduced room of the same generator:
    every operator on its stored inputs and every tensor normwise against
    the whole oracle network."""
    from paper_1912_05905_amd.pipeline import GpuPipeline
    levels = _run_both(L, O, configs.config10(m=12_000, size=(2.0, 2.0, 2.0), nboxes=3))
    GpuPipeline.release(levels)


def test_pipeline_overlapped_steps(L, O):
    """Steps whose lattice builds overlap the previous step's operators (the
    bench's mode): every step's point outputs match the oracle."""
    from paper_1912_05905_amd.pipeline import GpuPipeline
    wl = configs.make(4)
    _, _, oouts = OraclePipeline(wl).run()
    pipe = GpuPipeline(wl, overlap=True)
    for _ in range(4):
        levels, _, outs = pipe.step()
        for name in ("slice", "deform"):
            P.assert_close(_host(outs[name]), oouts[name], P.TOL_F32, name)
        pipe.finish_step(levels)
    pipe.flush()


@pytest.mark.parametrize("K,shared", [(2, False), (3, True)])
def test_pipeline_steps_on_two_streams(L, O, K, shared):
    """K pipelines, each with its own build stream or all sharing one, take
    steps in turn on K compute streams (the current one and others) with no
    host synchronisation between steps, as the bench runs them: consecutive
    clouds' builds and operators run side by side.  Every step's point
    outputs, copied on its own stream, match the oracle."""
    from paper_1912_05905_amd.pipeline import GpuPipeline
    wl = configs.make(4)
    _, _, oouts = OraclePipeline(wl).run()
    bs = torch.cuda.Stream() if shared else None
    pipes = [GpuPipeline(wl, overlap=True, build_stream=bs) for _ in range(K)]
    streams = [torch.cuda.current_stream()] + [torch.cuda.Stream() for _ in range(K - 1)]
    kept = []
    for i in range(2 * K + 2):
        k = i % K
        with torch.cuda.stream(streams[k]):
            levels, _, outs = pipes[k].step()
            kept.append({name: outs[name].clone() for name in ("slice", "deform")})
            pipes[k].finish_step(levels)
    torch.cuda.synchronize()
    for got in kept:
        for name, t in got.items():
            P.assert_close(_host(t), oouts[name], P.TOL_F32, name)
    for p in pipes:
        p.flush()


def test_latticenet_reduced(L, O):
    """The whole LatticeNet forward (Distribute + PointNet, eight ResNet
    blocks of pre-activated convolutions, two Downsamples, two Upsamples with
    concatenated skips, DeformSlice fused with the classifier) on reduced
    clouds of the LiDAR and room generators: the oracle takes seconds there,
    minutes at full size."""
    for wl in (configs.config8(m=6000), configs.config9(m=12_000, size=(2.0, 2.0, 2.0), nboxes=3)):
        levels = _run_both(L, O, wl)
        from paper_1912_05905_amd.pipeline import GpuPipeline
        GpuPipeline.release(levels)


@pytest.mark.parametrize("seed", [100, 101])
def test_pipeline_other_seeds(L, O, seed):
    for cfg in (1, 2):
        _run_both(L, O, configs.make(cfg, seed=seed))


def test_pipeline_config5_reduced(L, O):
    """The bf16 4-level U-Net on a 30k-point room of the same generator."""
    _run_both(L, O, configs.config5(m=30_000, size=(4.0, 4.0, 3.0), nboxes=20))


# ----------------------------------------------------------------------------
# Distribute + PointNet
# ----------------------------------------------------------------------------
def _pointnet_layers(rng, cin, widths):
    layers, k = [], cin
    for w in widths:
        layers.append(((rng.normal(size=(w, k)) / np.sqrt(k)).astype(np.float32),
                       (0.1 * rng.normal(size=w)).astype(np.float32)))
        k = w
    return layers


def _distribute_pair(L, O, gl, ol, g2o, pos, F, widths, seed, affine=True, eps=1e-5):
    rng = np.random.default_rng(seed)
    cf = 0 if F is None else F.shape[1]
    layers = _pointnet_layers(rng, 3 + cf, widths)
    dev_layers = [(_dev(W), _dev(b)) for W, b in layers]
    tot = 3 + cf + widths[0] + widths[1]
    gn = ((1.0 + 0.1 * rng.normal(size=tot)).astype(np.float32), (0.1 * rng.normal(size=tot)).astype(np.float32)) \
        if affine else None
    gy = gl.distribute_pointnet(_dev(pos), None if F is None else _dev(F), dev_layers,
                                None if gn is None else (_dev(gn[0]), _dev(gn[1])), eps=eps)
    oy = ol.distribute_pointnet(pos.astype(np.float64), None if F is None else F.astype(np.float64),
                                [(W.astype(np.float64), b.astype(np.float64)) for W, b in layers],
                                None if gn is None else tuple(a.astype(np.float64) for a in gn), eps=eps)
    return P.rows_in_oracle_order(_host(gy), g2o), oy


@pytest.mark.parametrize("cf,widths,affine", [(4, (16, 32, 64), True), (0, (16, 32, 64), True),
                                               (13, (32, 32, 48), True), (29, (64, 64, 64), True),
                                               (3, (16, 16, 16), False), (1, (64, 32, 64), True)])
def test_distribute_pointnet(L, O, cf, widths, affine):
    pos = _cloud(200 + cf, 9000, 0.7)
    gl, ol, g2o = _pair(L, O, pos, 0.06)
    F = None if cf == 0 else np.random.default_rng(cf).normal(size=(pos.shape[0], cf)).astype(np.float32)
    g, o = _distribute_pair(L, O, gl, ol, g2o, pos, F, widths, cf, affine)
    P.assert_close(g, o, P.TOL_F32, f"distribute cf={cf} {widths}")


def test_distribute_pointnet_golden_cases(L, O):
    """The hand-worked two-point cases of the oracle's pins, on the GPU."""
    doc = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "distribute_cases.json")))
    for c in doc["cases"]:
        pos = np.array(c["positions"], np.float32)
        gl = L.Lattice.create(_dev(pos), [c["sigma"]] * 3)
        layers = []
        k = 4
        for i, w in enumerate(c["widths"]):
            W = np.zeros((w, k), np.float32)
            for o, j, v in c[f"W{i + 1}_nonzero"]:
                W[o, j] = v
            layers.append((_dev(W), _dev(np.array(c[f"b{i + 1}"], np.float32))))
            k = w
        got = _host(gl.distribute_pointnet(_dev(pos), _dev(np.array(c["features"], np.float32)), layers,
                                           (_dev(np.array(c["gamma"], np.float32)),
                                            _dev(np.array(c["beta"], np.float32))), eps=c["eps"]))
        want = np.array(c["expected"])
        assert got.shape == (4, len(want))
        assert np.abs(got - want[None]).max() <= 1e-5 * (1 + np.abs(want).max()), c["name"]
        gl.destroy()


def test_distribute_pointnet_nonfinite_feature(L, O):
    """A NaN or infinite feature reaches the statistics of its channel; the
    whole output is then NaN, as in the oracle."""
    pos = _cloud(231, 3000, 0.6)
    gl, ol, g2o = _pair(L, O, pos, 0.08)
    for bad in (np.nan, np.inf):
        F = np.random.default_rng(3).normal(size=(pos.shape[0], 2)).astype(np.float32)
        F[1234, 1] = bad
        g, o = _distribute_pair(L, O, gl, ol, g2o, pos, F, (16, 32, 64), 4)
        assert np.isnan(o).all() and np.isnan(g).all()


def test_distribute_pointnet_skewed_and_far(L, O):
    """Lists far longer than the spans of both passes (a 6000-point clump in
    one simplex), and a cloud 40 m from the origin, where g - mu is a small
    difference of large coordinates."""
    rng = np.random.default_rng(5)
    clump = (np.array([0.31, 0.42, 0.53]) + 1e-4 * rng.random((6000, 3))).astype(np.float32)
    spread = rng.random((3001, 3)).astype(np.float32)
    for shift, sigma in ((0.0, 0.05), (40.0, 0.3)):
        pos = (np.concatenate([spread[:1500], clump, spread[1500:]]) * (8.0 if shift else 1.0) + shift).astype(np.float32)
        gl, ol, g2o = _pair(L, O, pos, sigma)
        F = rng.normal(size=(pos.shape[0], 4)).astype(np.float32)
        g, o = _distribute_pair(L, O, gl, ol, g2o, pos, F, (16, 32, 64), 11)
        P.assert_close(g, o, P.TOL_F32, f"distribute shift={shift}")


def test_distribute_pointnet_coarse_and_tiny(L, O):
    pos = _cloud(207, 5000, 0.8)
    gl = L.Lattice.create(_dev(pos), [0.05] * 3)
    ol = O.Lattice.create(pos, np.full(3, 0.05, np.float32))
    gc, oc = gl.coarsen(), ol.coarsen()
    g2o = P.key_permutation(_host(gc.keys()), oc.keys())
    F = np.random.default_rng(2).normal(size=(pos.shape[0], 4)).astype(np.float32)
    g, o = _distribute_pair(L, O, gc, oc, g2o, pos, F, (16, 32, 64), 3)
    P.assert_close(g, o, P.TOL_F32, "distribute on a coarse level")
    gc.destroy()
    gl.destroy()
    for m in (1, 37):
        pos = _cloud(300 + m, m, 0.5)
        gl, ol, g2o = _pair(L, O, pos, 0.1)
        F = np.random.default_rng(m).normal(size=(m, 4)).astype(np.float32)
        g, o = _distribute_pair(L, O, gl, ol, g2o, pos, F, (16, 32, 64), m)
        P.assert_close(g, o, P.TOL_F32, f"distribute m={m}")
    gl = L.Lattice.create(torch.zeros((0, 3), device="cuda"), [0.1] * 3)
    assert gl.distribute_pointnet(torch.zeros((0, 3), device="cuda"), None,
                                  [(torch.zeros((16, 3), device="cuda"), None),
                                   (torch.zeros((32, 16), device="cuda"), None),
                                   (torch.zeros((64, 32), device="cuda"), None)]).shape == (0, 64)


# ----------------------------------------------------------------------------
# backward passes, against the oracle's gradients
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("C,normalize", [(4, True), (36, False), (64, True), (256, False)])
def test_splat_and_slice_backward(L, O, C, normalize):
    pos = _cloud(500 + C, 9000, 0.7)
    gl, ol, g2o = _pair(L, O, pos, 0.06)
    rng = np.random.default_rng(C)
    dX = rng.normal(size=(ol.n, C)).astype(np.float32)
    gf = gl.splat_backward(_dev(dX[g2o]), normalize=normalize)
    of = ol.splat_backward(dX.astype(np.float64), normalize=normalize)
    P.assert_close(_host(gf), of, P.TOL_F32, f"splat backward C={C}")
    if normalize:
        # with the forward's weight sums instead of a pass over the lists
        ws = torch.empty(gl.n, device="cuda")
        gl.splat(_dev(np.zeros((pos.shape[0], 4), np.float32)), wsum=ws)
        gf = gl.splat_backward(_dev(dX[g2o]), normalize=True, wsum=ws)
        P.assert_close(_host(gf), of, P.TOL_F32, f"splat backward with wsum C={C}")
    dO = rng.normal(size=(pos.shape[0], C)).astype(np.float32)
    gx = gl.slice_backward(_dev(dO))
    ox = ol.slice_backward(dO.astype(np.float64))
    P.assert_close(P.rows_in_oracle_order(_host(gx), g2o), ox, P.TOL_F32, f"slice backward C={C}")


def test_slice_backward_skewed(L, O):
    """A 6000-point clump: vertex lists far longer than a workgroup span."""
    rng = np.random.default_rng(9)
    clump = (np.array([0.31, 0.42, 0.53]) + 1e-4 * rng.random((6000, 3))).astype(np.float32)
    spread = rng.random((3001, 3)).astype(np.float32)
    pos = np.concatenate([spread[:1500], clump, spread[1500:]]).astype(np.float32)
    gl, ol, g2o = _pair(L, O, pos, 0.05)
    dO = rng.normal(size=(pos.shape[0], 64)).astype(np.float32)
    gx = gl.slice_backward(_dev(dO))
    ox = ol.slice_backward(dO.astype(np.float64))
    P.assert_close(P.rows_in_oracle_order(_host(gx), g2o), ox, P.TOL_F32, "skewed slice backward")
    dX = rng.normal(size=(ol.n, 64)).astype(np.float32)
    gf = gl.splat_backward(_dev(dX[g2o]), normalize=True)
    P.assert_close(_host(gf), ol.splat_backward(dX.astype(np.float64), normalize=True), P.TOL_F32,
                   "skewed splat backward")


def _conv_backward_pair(L, O, form, seed, m, sigma, cin, cout, relu):
    pos = _cloud(seed, m, 0.8)
    gl = L.Lattice.create(_dev(pos), [sigma] * 3)
    ol = O.Lattice.create(pos, np.full(3, sigma, np.float32))
    g2o_f = P.key_permutation(_host(gl.keys()), ol.keys())
    if form == "same":
        (gd, gs, od, os_, g2o_d, g2o_s) = (gl, gl, ol, ol, g2o_f, g2o_f)
        keep = ()
    else:
        gc, oc = gl.coarsen(), ol.coarsen()
        g2o_c = P.key_permutation(_host(gc.keys()), oc.keys())
        keep = (gc,)
        if form == "strided":
            (gd, gs, od, os_, g2o_d, g2o_s) = (gc, gl, oc, ol, g2o_c, g2o_f)
        else:
            (gd, gs, od, os_, g2o_d, g2o_s) = (gl, gc, ol, oc, g2o_f, g2o_c)
    rng = np.random.default_rng(seed)
    X = rng.normal(size=(os_.n, cin)).astype(np.float32)
    W = _rand_w(rng, cin, cout, 1.0 / np.sqrt(9 * cin))
    b = (0.3 * rng.normal(size=cout)).astype(np.float32)
    dY = rng.normal(size=(od.n, cout)).astype(np.float32)
    if form == "upsample":
        Y = od.refine_into(os_, X.astype(np.float64), W.astype(np.float64), bias=b.astype(np.float64), relu=relu)
    else:
        Y = od.conv(os_, X.astype(np.float64), W.astype(np.float64), bias=b.astype(np.float64), relu=relu)
    odx, odw, odb = od.conv_backward(os_, X.astype(np.float64), W.astype(np.float64), dY.astype(np.float64),
                                     relu=relu, Y=Y if relu else None)
    gdx, gdw, gdb = gd.conv_backward(gs, _dev(X[g2o_s]), _gpu_w(W), _dev(dY[g2o_d]), relu=relu,
                                     y=_dev(Y[g2o_d].astype(np.float32)) if relu else None)
    what = f"{form} {cin}->{cout} relu={relu}"
    P.assert_close(P.rows_in_oracle_order(_host(gdx), g2o_s), odx, P.TOL_F32, "dX " + what)
    P.assert_close(np.transpose(_host(gdw), (0, 2, 1)), odw, P.TOL_F32, "dW " + what)
    P.assert_close(_host(gdb), odb, P.TOL_F32, "dbias " + what)
    del keep


@pytest.mark.parametrize("cin,cout", [(8, 16), (12, 20), (64, 64), (32, 96), (128, 128), (256, 64)])
def test_conv_backward_same_level(L, O, cin, cout):
    for relu in (False, True):
        _conv_backward_pair(L, O, "same", 600 + cin, 6000, 0.07, cin, cout, relu)


@pytest.mark.parametrize("form", ["strided", "upsample"])
def test_conv_backward_across_levels(L, O, form):
    for cin, cout, relu in ((64, 128, True), (128, 64, False), (20, 36, True)):
        _conv_backward_pair(L, O, form, 700 + cin, 8000, 0.05, cin, cout, relu)


def test_conv_backward_partial_outputs_and_tiny(L, O):
    """Only some gradients asked for; a one-point cloud."""
    pos = _cloud(801, 3000, 0.8)
    gl, ol, g2o = _pair(L, O, pos, 0.08)
    rng = np.random.default_rng(801)
    X = rng.normal(size=(ol.n, 16)).astype(np.float32)
    W = _rand_w(rng, 16, 8, 0.1)
    dY = rng.normal(size=(ol.n, 8)).astype(np.float32)
    odx, odw, odb = ol.conv_backward(ol, X.astype(np.float64), W.astype(np.float64), dY.astype(np.float64))
    gdx, gdw, gdb = gl.conv_backward(gl, None, _gpu_w(W), _dev(dY[g2o]), want_dw=False, want_dbias=False)
    assert gdw is None and gdb is None
    P.assert_close(P.rows_in_oracle_order(_host(gdx), g2o), odx, P.TOL_F32, "dX only")
    gdx, gdw, gdb = gl.conv_backward(gl, _dev(X[g2o]), None, _dev(dY[g2o]), want_dx=False)
    P.assert_close(np.transpose(_host(gdw), (0, 2, 1)), odw, P.TOL_F32, "dW only")
    P.assert_close(_host(gdb), odb, P.TOL_F32, "dbias only")
    pos1 = _cloud(802, 1, 0.5)
    g1, o1, g2o1 = _pair(L, O, pos1, 0.1)
    X1 = rng.normal(size=(o1.n, 8)).astype(np.float32)
    W1 = _rand_w(rng, 8, 8, 0.3)
    dY1 = rng.normal(size=(o1.n, 8)).astype(np.float32)
    odx, odw, odb = o1.conv_backward(o1, X1.astype(np.float64), W1.astype(np.float64), dY1.astype(np.float64))
    gdx, gdw, gdb = g1.conv_backward(g1, _dev(X1[g2o1]), _gpu_w(W1), _dev(dY1[g2o1]))
    P.assert_close(P.rows_in_oracle_order(_host(gdx), g2o1), odx, P.TOL_F32, "tiny dX")
    P.assert_close(np.transpose(_host(gdw), (0, 2, 1)), odw, P.TOL_F32, "tiny dW")


def _deform_backward_pair(L, O, gl, ol, g2o, C, seed):
    rng = np.random.default_rng(seed)
    X = rng.normal(size=(ol.n, C)).astype(np.float32)
    wv = (rng.normal(size=C) / np.sqrt(C)).astype(np.float32)
    beta = 0.15
    dO = rng.normal(size=(ol.m, C)).astype(np.float32)
    odx, odw, odb = ol.deform_slice_backward(X.astype(np.float64), wv.astype(np.float64), beta, dO.astype(np.float64))
    gdx, gdw, gdb = gl.deform_slice_backward(_dev(X[g2o]), _dev(wv), beta, _dev(dO))
    P.assert_close(P.rows_in_oracle_order(_host(gdx), g2o), odx, P.TOL_F32, f"DeformSlice dX C={C}")
    P.assert_close(_host(gdw), odw, P.TOL_F32, f"DeformSlice dwv C={C}")
    P.assert_close(_host(gdb), np.array([odb]), P.TOL_F32, f"DeformSlice dbeta C={C}")


@pytest.mark.parametrize("C", [4, 16, 64, 128, 512])
def test_deform_slice_backward(L, O, C):
    pos = _cloud(900 + C, 7000, 0.8)
    gl, ol, g2o = _pair(L, O, pos, 0.06)
    _deform_backward_pair(L, O, gl, ol, g2o, C, C)


def test_deform_slice_backward_skewed_tiny_empty(L, O):
    rng = np.random.default_rng(5)
    clump = (np.array([0.31, 0.42, 0.53]) + 1e-4 * rng.random((6000, 3))).astype(np.float32)
    spread = rng.random((3001, 3)).astype(np.float32)
    pos = np.concatenate([spread[:1500], clump, spread[1500:]]).astype(np.float32)
    gl, ol, g2o = _pair(L, O, pos, 0.05)
    _deform_backward_pair(L, O, gl, ol, g2o, 64, 6)
    for m in (1, 37):
        gl, ol, g2o = _pair(L, O, _cloud(950 + m, m, 0.5), 0.1)
        _deform_backward_pair(L, O, gl, ol, g2o, 32, m)
    ge = L.Lattice.create(torch.zeros((0, 3), device="cuda"), [0.1] * 3)
    dx, dwv, dbeta = ge.deform_slice_backward(torch.zeros((0, 8), device="cuda"), torch.ones(8, device="cuda"), 0.1,
                                              torch.zeros((0, 8), device="cuda"))
    assert dx.shape == (0, 8) and not _host(dwv).any() and _host(dbeta)[0] == 0.0


# ----------------------------------------------------------------------------
# the training step of the LiDAR scan (forward + backward), at full size
# ----------------------------------------------------------------------------
def test_train_step_full_size(L, O):
    """Config 7 at full size.  The backward pass takes discrete decisions from
    the forward activations (ReLU masks Y > 0, DeformSlice's maximal vertex),
    and the GPU's and the oracle's forward activations differ by rounding, so
    at near-ties the two runs may legitimately decide differently and move a
    gradient term.  Hence: (1) every backward operator is replayed on the
    GPU with the oracle's own inputs (its forward activations and upstream
    gradients, rounded to float32) and compared elementwise with the oracle
    on the same inputs; (2) the GPU's end-to-end step is compared elementwise
    on the forward buffers and normwise (1e-3) on the gradients."""
    from paper_1912_05905_amd.pipeline import GpuPipeline
    wl = configs.make(7)
    levels, bufs, outs = GpuPipeline(wl).step()
    olv, obufs, oouts = OraclePipeline(wl).run()
    g2o = {lv: _check_structure(levels[lv], olv[lv]) for lv in sorted(levels)}
    grad_bufs = {name for name in wl.buffers if name.startswith("g")}
    for name, (lv, _) in wl.buffers.items():
        got = P.rows_in_oracle_order(_host(bufs[name]), g2o[lv])
        if name in grad_bufs:
            rel = np.linalg.norm(got - obufs[name]) / np.linalg.norm(obufs[name])
            assert rel <= 1e-3, (name, rel)
        else:
            P.assert_close(got, obufs[name], P.TOL_F32, name)
    for name in oouts:
        if name == "deform":
            P.assert_close(_host(outs[name]), oouts[name], P.TOL_F32, name)
        else:
            rel = np.linalg.norm(_host(outs[name]) - oouts[name]) / max(np.linalg.norm(oouts[name]), 1e-30)
            assert rel <= 1e-3, (name, rel)

    f32 = lambda a: np.asarray(a, np.float64).astype(np.float32)
    gpu_rows = lambda a, lv: _dev(f32(a)[g2o[lv]])
    for op in wl.ops:
        if op["op"] == "deform_slice_bwd":
            lv = op["level"]
            X = f32(obufs[op["x"][0]][:, op["x"][1]:op["x"][1] + op["x"][2]])
            wv, beta = wl.vectors[op["wv"]]
            dO = wl.grads[op["grad"]]
            gdx, gdw, gdb = levels[lv].deform_slice_backward(gpu_rows(X, lv), _dev(wv), beta, _dev(dO))
            odx, odw, odb = olv[lv].deform_slice_backward(X.astype(np.float64), wv.astype(np.float64), beta,
                                                         dO.astype(np.float64))
            P.assert_close(P.rows_in_oracle_order(_host(gdx), g2o[lv]), odx, P.TOL_F32, "replay DeformSlice dX")
            P.assert_close(_host(gdw), odw, P.TOL_F32, "replay DeformSlice dwv")
            P.assert_close(_host(gdb), np.array([odb]), P.TOL_F32, "replay DeformSlice dbeta")
        elif op["op"] == "conv_bwd":
            lv = op["level"]
            slv = {"conv": lv, "conv_down": lv - 1, "refine": lv + 1}[op["kind"]]
            cut = lambda spec: f32(obufs[spec[0]][:, spec[1]:spec[1] + spec[2]])
            X, Y, dY = cut(op["x"]), cut(op["y"]), cut(op["src"])
            W = wl.weights[op["w"]]
            gdx, gdw, gdb = levels[lv].conv_backward(levels[slv], gpu_rows(X, slv), _gpu_w(W), gpu_rows(dY, lv),
                                                     relu=op["relu"], y=gpu_rows(Y, lv) if op["relu"] else None)
            odx, odw, odb = olv[lv].conv_backward(olv[slv], X.astype(np.float64), W.astype(np.float64),
                                                  dY.astype(np.float64), relu=op["relu"],
                                                  Y=Y.astype(np.float64) if op["relu"] else None)
            what = f"replay {op['kind']} level {lv}"
            P.assert_close(P.rows_in_oracle_order(_host(gdx), g2o[slv]), odx, P.TOL_F32, "dX " + what)
            P.assert_close(np.transpose(_host(gdw), (0, 2, 1)), odw, P.TOL_F32, "dW " + what)
            P.assert_close(_host(gdb), odb, P.TOL_F32, "dbias " + what)
        elif op["op"] == "splat_bwd":
            G = f32(obufs[op["src"][0]])
            gf = levels[0].splat_backward(gpu_rows(G, 0), normalize=bool(op["normalize"]))
            of = olv[0].splat_backward(G.astype(np.float64), normalize=bool(op["normalize"]))
            P.assert_close(_host(gf), of, P.TOL_F32, "replay splat backward")
    GpuPipeline.release(levels)


# ----------------------------------------------------------------------------
# pre-activated convolutions: conv(relu(GroupNorm(x)))
# ----------------------------------------------------------------------------
def _preact_case(L, O, gd, gs, od, os_, g2o_d, g2o_s, form, cin, cout, groups, seed, dtype="f32", affine=True,
                 offset=0.0):
    rng = np.random.default_rng(seed)
    bf = dtype == "bf16"
    tdt = torch.bfloat16 if bf else torch.float32
    rnd = O.round_bf16 if bf else (lambda a: np.asarray(a, np.float64))
    X = rnd(offset + rng.normal(size=(os_.n, cin)) * rng.uniform(0.5, 2.0, size=cin))
    W = rnd(_rand_w(rng, cin, cout, 1.0 / np.sqrt(9 * cin)))
    gam = rng.uniform(0.5, 1.5, size=cin).astype(np.float32) if affine else None
    bet = (0.2 * rng.normal(size=cin)).astype(np.float32) if affine else None
    b = rng.normal(size=cout).astype(np.float32)
    A = O.groupnorm(X, groups, gam, bet, eps=1e-5, relu=True)
    if bf:
        A = O.round_bf16(A)
    if form == "upsample":
        oy = od.refine_into(os_, A, W, bias=b.astype(np.float64))
    else:
        oy = od.conv(os_, A, W, bias=b.astype(np.float64))
    gy = gd.conv_preact(gs, _dev(X[g2o_s].astype(np.float32), tdt), _gpu_w(W.astype(np.float32), tdt), groups=groups,
                        gamma=None if gam is None else _dev(gam), beta=None if bet is None else _dev(bet), eps=1e-5,
                        bias=_dev(b), refine=form == "upsample")
    tol = P.TOL_BF16 if bf else P.TOL_F32
    P.assert_close(P.rows_in_oracle_order(_host(gy), g2o_d), rnd(oy), tol,
                   f"preact {form} {cin}->{cout} G={groups} {dtype}")


@pytest.mark.parametrize("cin,cout,groups", [(64, 64, 32), (12, 20, 4), (128, 128, 32), (32, 96, 1), (64, 16, 64),
                                             (256, 64, 32)])
def test_conv_preact_same_level(L, O, cin, cout, groups):
    pos = _cloud(1000 + cin, 6000, 0.8)
    gl, ol, g2o = _pair(L, O, pos, 0.07)
    _preact_case(L, O, gl, gl, ol, ol, g2o, g2o, "same", cin, cout, groups, cin + cout)
    _preact_case(L, O, gl, gl, ol, ol, g2o, g2o, "same", cin, cout, groups, cin + cout + 1, affine=False,
                 offset=300.0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_conv_preact_across_levels(L, O, dtype):
    pos = _cloud(1100, 8000, 0.8)
    gl = L.Lattice.create(_dev(pos), [0.05] * 3)
    ol = O.Lattice.create(pos, np.full(3, 0.05, np.float32))
    gc, oc = gl.coarsen(), ol.coarsen()
    g2o_f = P.key_permutation(_host(gl.keys()), ol.keys())
    g2o_c = P.key_permutation(_host(gc.keys()), oc.keys())
    _preact_case(L, O, gc, gl, oc, ol, g2o_c, g2o_f, "strided", 64, 128, 32, 5, dtype)
    _preact_case(L, O, gl, gc, ol, oc, g2o_f, g2o_c, "upsample", 128, 64, 32, 6, dtype)
    if dtype == "bf16":
        _preact_case(L, O, gl, gl, ol, ol, g2o_f, g2o_f, "same", 64, 64, 32, 7, dtype)


@pytest.mark.parametrize("C,K,dtype", [(4, 7, "f32"), (16, 20, "f32"), (64, 20, "f32"), (64, 64, "f32"),
                                       (128, 33, "f32"), (256, 20, "f32"), (512, 32, "f32"), (64, 20, "bf16"),
                                       (256, 1, "bf16")])
def test_deform_slice_classify(L, O, C, K, dtype):
    pos = _cloud(1200 + C + K, 7000, 0.8)
    gl, ol, g2o = _pair(L, O, pos, 0.06)
    rng = np.random.default_rng(C * 100 + K)
    bf = dtype == "bf16"
    X = rng.normal(size=(ol.n, C))
    if bf:
        X = O.round_bf16(X)
    wv = (rng.normal(size=C) / np.sqrt(C)).astype(np.float32)
    Wc = (rng.normal(size=(K, C)) / np.sqrt(C)).astype(np.float32)
    bc = rng.normal(size=K).astype(np.float32) if K != 64 else None
    gy = gl.deform_slice_classify(_dev(X[g2o].astype(np.float32), torch.bfloat16 if bf else None), _dev(wv), 0.1,
                                  _dev(Wc), None if bc is None else _dev(bc))
    oy = ol.deform_slice_classify(X, wv.astype(np.float64), 0.1, Wc.astype(np.float64),
                                  None if bc is None else bc.astype(np.float64))
    P.assert_close(_host(gy), oy, P.TOL_F32, f"DeformSlice+classifier C={C} K={K} {dtype}")


def test_conv_taps_count_existing_neighbours(L, O):
    """lattice_conv_taps: the (vertex, tap) pairs with an existing neighbour
    of the 1-hop, strided and Upsample tables, against the oracle's tables."""
    pos = _cloud(61, 20_000, 1.0)
    g0 = L.Lattice.create(_dev(pos), [0.05] * 3)
    g1 = g0.coarsen()
    o0 = O.Lattice.create(pos, np.full(3, 0.05, np.float32))
    o1 = o0.coarsen()
    assert g0.conv_taps(g0) == int((o0.neighbors() >= 0).sum())
    assert g1.conv_taps(g1) == int((o1.neighbors() >= 0).sum())
    assert g1.conv_taps(g0) == int((o1.down_table() >= 0).sum())
    assert g0.conv_taps(g1) == int((o1.up_table() >= 0).sum())
    g1.destroy()
    g0.destroy()


# ----------------------------------------------------------------------------
# backward of the pre-activated convolution: GroupNorm + ReLU + conv
# ----------------------------------------------------------------------------
def _preact_backward_case(L, O, gd, gs, od, os_, g2o_d, g2o_s, form, cin, cout, groups, seed, relu, affine=True,
                          offset=0.0):
    rng = np.random.default_rng(seed)
    X = (offset + rng.normal(size=(os_.n, cin)) * rng.uniform(0.5, 2.0, size=cin)).astype(np.float32)
    W = _rand_w(rng, cin, cout, 1.0 / np.sqrt(9 * cin))
    gam = rng.uniform(0.5, 1.5, size=cin).astype(np.float32) if affine else None
    bet = (0.2 * rng.normal(size=cin)).astype(np.float32) if affine else None
    b = rng.normal(size=cout).astype(np.float32)
    dY = rng.normal(size=(od.n, cout)).astype(np.float32)
    X64 = X.astype(np.float64)
    A = O.groupnorm(X64, groups, gam, bet, eps=1e-5, relu=True)
    if form == "upsample":
        Y = od.refine_into(os_, A, W.astype(np.float64), bias=b.astype(np.float64), relu=relu)
    else:
        Y = od.conv(os_, A, W.astype(np.float64), bias=b.astype(np.float64), relu=relu)
    odA, odW, odb = od.conv_backward(os_, A, W.astype(np.float64), dY.astype(np.float64), relu=relu,
                                     Y=Y if relu else None)
    odX, odg, odbe = O.groupnorm_backward(X64, odA, groups, gam, bet, eps=1e-5, relu=True)
    gdX, gdW, gdb, gdg, gdbe = gd.conv_preact_backward(
        gs, _dev(X[g2o_s]), _gpu_w(W), _dev(dY[g2o_d]), groups=groups, gamma=None if gam is None else _dev(gam),
        beta=None if bet is None else _dev(bet), eps=1e-5, relu=relu,
        y=_dev(Y[g2o_d].astype(np.float32)) if relu else None)
    what = f"preact backward {form} {cin}->{cout} G={groups} relu={relu}"
    P.assert_close(P.rows_in_oracle_order(_host(gdX), g2o_s), odX, P.TOL_F32, "dX " + what)
    P.assert_close(np.transpose(_host(gdW), (0, 2, 1)), odW, P.TOL_F32, "dW " + what)
    P.assert_close(_host(gdb), odb, P.TOL_F32, "dbias " + what)
    P.assert_close(_host(gdg), odg, P.TOL_F32, "dgamma " + what)
    P.assert_close(_host(gdbe), odbe, P.TOL_F32, "dbeta " + what)


@pytest.mark.parametrize("cin,cout,groups,relu,affine,offset", [
    (64, 64, 32, False, True, 0.0), (12, 20, 4, True, True, 0.0), (128, 128, 32, True, False, 300.0),
    (32, 96, 1, False, True, 0.0), (64, 16, 64, True, True, 0.0), (256, 64, 32, False, True, 0.0)])
def test_conv_preact_backward_same_level(L, O, cin, cout, groups, relu, affine, offset):
    pos = _cloud(1300 + cin + groups, 6000, 0.8)
    gl, ol, g2o = _pair(L, O, pos, 0.07)
    _preact_backward_case(L, O, gl, gl, ol, ol, g2o, g2o, "same", cin, cout, groups, cin + cout + groups, relu,
                          affine, offset)


def test_conv_preact_backward_across_levels(L, O):
    pos = _cloud(1400, 8000, 0.8)
    gl = L.Lattice.create(_dev(pos), [0.05] * 3)
    ol = O.Lattice.create(pos, np.full(3, 0.05, np.float32))
    gc, oc = gl.coarsen(), ol.coarsen()
    g2o_f = P.key_permutation(_host(gl.keys()), ol.keys())
    g2o_c = P.key_permutation(_host(gc.keys()), oc.keys())
    _preact_backward_case(L, O, gc, gl, oc, ol, g2o_c, g2o_f, "strided", 64, 128, 32, 11, True)
    _preact_backward_case(L, O, gl, gc, ol, oc, g2o_f, g2o_c, "upsample", 128, 64, 32, 12, False)
    _preact_backward_case(L, O, gl, gc, ol, oc, g2o_f, g2o_c, "upsample", 32, 32, 8, 13, True)


def test_conv_preact_backward_partial_outputs_and_tiny(L, O):
    """Only the weight gradients (no GroupNorm backward), only dX, and a
    one-point cloud."""
    pos = _cloud(1450, 3000, 0.8)
    gl, ol, g2o = _pair(L, O, pos, 0.08)
    rng = np.random.default_rng(1450)
    X = rng.normal(size=(ol.n, 16)).astype(np.float32)
    W = _rand_w(rng, 16, 8, 0.1)
    dY = rng.normal(size=(ol.n, 8)).astype(np.float32)
    A = O.groupnorm(X.astype(np.float64), 4, eps=1e-5, relu=True)
    odA, odW, odb = ol.conv_backward(ol, A, W.astype(np.float64), dY.astype(np.float64))
    odX, odg, odbe = O.groupnorm_backward(X.astype(np.float64), odA, 4, eps=1e-5, relu=True)
    gdX, gdW, gdb, gdg, gdbe = gl.conv_preact_backward(gl, _dev(X[g2o]), _gpu_w(W), _dev(dY[g2o]), groups=4,
                                                       want_dx=False, want_dgn=False)
    assert gdX is None and gdg is None and gdbe is None
    P.assert_close(np.transpose(_host(gdW), (0, 2, 1)), odW, P.TOL_F32, "preact dW only")
    P.assert_close(_host(gdb), odb, P.TOL_F32, "preact dbias only")
    gdX, gdW, gdb, gdg, gdbe = gl.conv_preact_backward(gl, _dev(X[g2o]), _gpu_w(W), _dev(dY[g2o]), groups=4,
                                                       want_dw=False, want_dbias=False, want_dgn=False)
    P.assert_close(P.rows_in_oracle_order(_host(gdX), g2o), odX, P.TOL_F32, "preact dX only")
    g1, o1, g2o1 = _pair(L, O, _cloud(1451, 1, 0.5), 0.1)
    X1 = rng.normal(size=(o1.n, 8)).astype(np.float32)
    W1 = _rand_w(rng, 8, 8, 0.3)
    dY1 = rng.normal(size=(o1.n, 8)).astype(np.float32)
    A1 = O.groupnorm(X1.astype(np.float64), 2, eps=1e-5, relu=True)
    odA, odW, odb = o1.conv_backward(o1, A1, W1.astype(np.float64), dY1.astype(np.float64))
    odX, odg, odbe = O.groupnorm_backward(X1.astype(np.float64), odA, 2, eps=1e-5, relu=True)
    gdX, gdW, gdb, gdg, gdbe = g1.conv_preact_backward(g1, _dev(X1[g2o1]), _gpu_w(W1), _dev(dY1[g2o1]), groups=2)
    P.assert_close(P.rows_in_oracle_order(_host(gdX), g2o1), odX, P.TOL_F32, "tiny preact dX")
    P.assert_close(_host(gdg), odg, P.TOL_F32, "tiny preact dgamma")


# ----------------------------------------------------------------------------
# backward of DeformSlice fused with the linear classifier
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("C,K", [(4, 7), (16, 20), (64, 20), (64, 64), (128, 33), (512, 32)])
def test_deform_slice_classify_backward(L, O, C, K):
    pos = _cloud(1500 + C + K, 7000, 0.8)
    gl, ol, g2o = _pair(L, O, pos, 0.06)
    rng = np.random.default_rng(C * 10 + K)
    X = rng.normal(size=(ol.n, C)).astype(np.float32)
    wv = (rng.normal(size=C) / np.sqrt(C)).astype(np.float32)
    Wc = (rng.normal(size=(K, C)) / np.sqrt(C)).astype(np.float32)
    Z = rng.normal(size=(ol.m, K)).astype(np.float32)
    odx, odw, odb, odWc, odbc = ol.deform_slice_classify_backward(X.astype(np.float64), wv.astype(np.float64), 0.1,
                                                                  Wc.astype(np.float64), Z.astype(np.float64))
    gdx, gdw, gdb, gdWc, gdbc = gl.deform_slice_classify_backward(_dev(X[g2o]), _dev(wv), 0.1, _dev(Wc), _dev(Z))
    what = f"classifier backward C={C} K={K}"
    P.assert_close(P.rows_in_oracle_order(_host(gdx), g2o), odx, P.TOL_F32, "dX " + what)
    P.assert_close(_host(gdw), odw, P.TOL_F32, "dwv " + what)
    P.assert_close(_host(gdb), np.array([odb]), P.TOL_F32, "dbeta " + what)
    P.assert_close(_host(gdWc), odWc, P.TOL_F32, "dWc " + what)
    P.assert_close(_host(gdbc), odbc, P.TOL_F32, "dbc " + what)


def test_deform_slice_classify_backward_tiny_and_strided_logits(L, O):
    """A one-point cloud, and dlogits as a column slice of a wider matrix."""
    for m in (1, 2000):
        gl, ol, g2o = _pair(L, O, _cloud(1600 + m, m, 0.6), 0.08)
        rng = np.random.default_rng(m)
        C, K = 32, 5
        X = rng.normal(size=(ol.n, C)).astype(np.float32)
        wv = (rng.normal(size=C) / np.sqrt(C)).astype(np.float32)
        Wc = (rng.normal(size=(K, C)) / np.sqrt(C)).astype(np.float32)
        Zw = rng.normal(size=(ol.m, K + 3)).astype(np.float32)
        odx, odw, odb, odWc, odbc = ol.deform_slice_classify_backward(X.astype(np.float64), wv.astype(np.float64),
                                                                      -0.2, Wc.astype(np.float64),
                                                                      Zw[:, 1:1 + K].astype(np.float64))
        gdx, gdw, gdb, gdWc, gdbc = gl.deform_slice_classify_backward(_dev(X[g2o]), _dev(wv), -0.2, _dev(Wc),
                                                                      _dev(Zw)[:, 1:1 + K])
        P.assert_close(P.rows_in_oracle_order(_host(gdx), g2o), odx, P.TOL_F32, f"classifier backward dX m={m}")
        P.assert_close(_host(gdWc), odWc, P.TOL_F32, f"classifier backward dWc m={m}")
        P.assert_close(_host(gdbc), odbc, P.TOL_F32, f"classifier backward dbc m={m}")


# ----------------------------------------------------------------------------
# backward of Distribute + PointNet
# ----------------------------------------------------------------------------
def _distribute_backward_case(L, O, gl, ol, g2o, pos, F, widths, seed, affine=True):
    rng = np.random.default_rng(seed)
    cf = 0 if F is None else F.shape[1]
    layers = _pointnet_layers(rng, 3 + cf, widths)
    tot = 3 + cf + widths[0] + widths[1]
    gn = ((1.0 + 0.1 * rng.normal(size=tot)).astype(np.float32), (0.1 * rng.normal(size=tot)).astype(np.float32)) \
        if affine else None
    lay64 = [(W.astype(np.float64), b.astype(np.float64)) for W, b in layers]
    gn64 = None if gn is None else tuple(a.astype(np.float64) for a in gn)
    F64 = None if F is None else F.astype(np.float64)
    D = rng.normal(size=(ol.n, widths[2])).astype(np.float32)
    # Where a vertex's two largest rows of a channel lie within 1e-6 of its
    # output's scale, either is a correct choice for the maximum: the
    # upstream gradient is zero there, so the gradients are unique.
    X = ol.distribute_pointnet(pos.astype(np.float64), F64, lay64, gn64)
    margin = ol.distribute_pointnet_backward(pos.astype(np.float64), F64, lay64, D, gn64)["margin"]
    near = margin < 1e-6 * np.sqrt(np.mean(X ** 2))
    D[near] = 0.0
    ref = ol.distribute_pointnet_backward(pos.astype(np.float64), F64, lay64, D.astype(np.float64), gn64)
    got = gl.distribute_pointnet_backward(_dev(pos), None if F is None else _dev(F),
                                          [(_dev(W), _dev(b)) for W, b in layers], _dev(D[g2o]),
                                          None if gn is None else (_dev(gn[0]), _dev(gn[1])))
    what = f"Distribute backward cf={cf} widths={widths}"
    for k in ("dW1", "dW2", "dW3", "db3", "dgamma"):
        P.assert_close(_host(got[k]), ref[k], P.TOL_F32, f"{k} {what}")
    # Without the affine parameters (beta = 0) the coordinate channels of a
    # vertex with a single point sit exactly on the ReLU's kink (g - mu_v = 0
    # and the rows' mean is 0 in exact arithmetic, so the sign of the
    # normalised value is rounding noise): their dbeta is not unique.
    lo = 0 if affine else 3
    P.assert_close(_host(got["dbeta"])[lo:], ref["dbeta"][lo:], P.TOL_F32, f"dbeta {what}")
    for i in (1, 2):
        db, dW = _host(got[f"db{i}"]), ref[f"dW{i}"]
        if widths[i - 1] <= 32:
            # the next normalisation has one channel per group and removes
            # any per-channel shift, so this bias gradient is exactly zero: a
            # sum that cancels, whose float32 error scales with its terms
            # (measured by the layer's weight gradient)
            scale = float(np.sqrt(np.mean(dW ** 2)))
            assert np.abs(ref[f"db{i}"]).max() <= 1e-9 * scale, what
            assert np.abs(db).max() <= P.TOL_F32 * scale, (f"db{i} {what}", np.abs(db).max(), scale)
        else:
            P.assert_close(db, ref[f"db{i}"], P.TOL_F32, f"db{i} {what}")
    if cf:
        P.assert_close(_host(got["dF"]), ref["dF"], P.TOL_F32, f"dF {what}")
    return int(near.sum())


@pytest.mark.parametrize("cf,widths,affine", [(4, (16, 32, 64), True), (0, (16, 32, 64), True),
                                               (13, (32, 32, 48), False), (29, (64, 64, 64), True),
                                               (1, (64, 32, 16), True)])
def test_distribute_pointnet_backward(L, O, cf, widths, affine):
    pos = _cloud(1700 + cf, 6000, 0.7)
    gl, ol, g2o = _pair(L, O, pos, 0.06)
    rng = np.random.default_rng(cf)
    F = rng.normal(size=(pos.shape[0], cf)).astype(np.float32) if cf else None
    _distribute_backward_case(L, O, gl, ol, g2o, pos, F, widths, 17 + cf, affine)


def test_distribute_pointnet_backward_skewed_and_tiny(L, O):
    """A clump of 3000 points in one simplex beside a spread cloud (lists of
    very different lengths), a coarse level, and a one-point cloud."""
    rng = np.random.default_rng(7)
    clump = (np.array([0.31, 0.42, 0.53]) + 1e-4 * rng.random((3000, 3))).astype(np.float32)
    spread = rng.random((2001, 3)).astype(np.float32)
    pos = np.concatenate([spread[:1000], clump, spread[1000:]]).astype(np.float32)
    F = rng.normal(size=(pos.shape[0], 4)).astype(np.float32)
    gl, ol, g2o = _pair(L, O, pos, 0.05)
    _distribute_backward_case(L, O, gl, ol, g2o, pos, F, (16, 32, 64), 21)
    gc, oc = gl.coarsen(), ol.coarsen()
    g2o_c = P.key_permutation(_host(gc.keys()), oc.keys())
    _distribute_backward_case(L, O, gc, oc, g2o_c, pos, F, (16, 32, 64), 22)
    pos5 = _cloud(1751, 5, 0.5)
    g5, o5, g2o5 = _pair(L, O, pos5, 0.1)
    _distribute_backward_case(L, O, g5, o5, g2o5, pos5, rng.normal(size=(5, 2)).astype(np.float32), (16, 16, 16), 24)
    # one point: its d+1 rows share the features and every coordinate row
    # is 0, so each normalisation sees identical rows and every gradient
    # before the last layer cancels exactly; the last layer's are unique
    pos1 = _cloud(1750, 1, 0.5)
    g1, o1, g2o1 = _pair(L, O, pos1, 0.1)
    lay = _pointnet_layers(np.random.default_rng(25), 5, (16, 16, 16))
    F1 = rng.normal(size=(1, 2)).astype(np.float32)
    D = np.random.default_rng(26).normal(size=(o1.n, 16))
    ref = o1.distribute_pointnet_backward(pos1.astype(np.float64), F1.astype(np.float64),
                                          [(W.astype(np.float64), b.astype(np.float64)) for W, b in lay], D)
    got = g1.distribute_pointnet_backward(_dev(pos1), _dev(F1), [(_dev(W), _dev(b)) for W, b in lay],
                                          _dev(D[g2o1].astype(np.float32)))
    for k in ("dW3", "db3"):
        P.assert_close(_host(got[k]), ref[k], P.TOL_F32, f"one-point Distribute backward {k}")
    for k in ("dF", "dW1", "db1", "dW2", "db2", "dgamma", "dbeta"):
        assert np.isfinite(_host(got[k])).all(), k


# ----------------------------------------------------------------------------
# convolution backward of a bfloat16 network
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("form,cin,cout,relu", [("same", 64, 64, True), ("same", 16, 128, False),
                                                 ("strided", 64, 128, True), ("upsample", 128, 64, False),
                                                 ("upsample", 32, 32, True)])
def test_conv_backward_bf16(L, O, form, cin, cout, relu):
    """bf16 X, W, Y and dY (the values a bf16 forward stores): dX in bf16
    against the oracle's float64 gradient rounded once; dW and dbias in
    float32 (bf16 values widen exactly, the error is float32 summation)."""
    seed = 1800 + cin + cout
    pos = _cloud(seed, 8000, 0.8)
    gl = L.Lattice.create(_dev(pos), [0.05] * 3)
    ol = O.Lattice.create(pos, np.full(3, 0.05, np.float32))
    g2o_f = P.key_permutation(_host(gl.keys()), ol.keys())
    keep = ()
    if form == "same":
        gd, gs, od, os_, g2o_d, g2o_s = gl, gl, ol, ol, g2o_f, g2o_f
    else:
        gc, oc = gl.coarsen(), ol.coarsen()
        keep = (gc,)
        g2o_c = P.key_permutation(_host(gc.keys()), oc.keys())
        if form == "strided":
            gd, gs, od, os_, g2o_d, g2o_s = gc, gl, oc, ol, g2o_c, g2o_f
        else:
            gd, gs, od, os_, g2o_d, g2o_s = gl, gc, ol, oc, g2o_f, g2o_c
    rng = np.random.default_rng(seed)
    X = O.round_bf16(rng.normal(size=(os_.n, cin)))
    W = O.round_bf16(rng.normal(size=(9, cin, cout)) / np.sqrt(9 * cin))
    b = O.round_bf16(0.3 * rng.normal(size=cout))
    dY = O.round_bf16(rng.normal(size=(od.n, cout)))
    if form == "upsample":
        Y = od.refine_into(os_, X, W, bias=b, relu=relu)
    else:
        Y = od.conv(os_, X, W, bias=b, relu=relu)
    Yb = O.round_bf16(Y)
    odx, odw, odb = od.conv_backward(os_, X, W, dY, relu=relu, Y=Yb if relu else None)
    bf = torch.bfloat16
    gdx, gdw, gdb = gd.conv_backward_bf16(gs, _dev(X[g2o_s].astype(np.float32), bf), _gpu_w(W.astype(np.float32), bf),
                                          _dev(dY[g2o_d].astype(np.float32), bf), relu=relu,
                                          y=_dev(Yb[g2o_d].astype(np.float32), bf) if relu else None)
    what = f"bf16 backward {form} {cin}->{cout} relu={relu}"
    assert gdx.dtype == bf
    P.assert_close(P.rows_in_oracle_order(_host(gdx.float()), g2o_s), O.round_bf16(odx), P.TOL_BF16, "dX " + what)
    P.assert_close(np.transpose(_host(gdw), (0, 2, 1)), odw, P.TOL_F32, "dW " + what)
    P.assert_close(_host(gdb), odb, P.TOL_F32, "dbias " + what)
    del keep


def test_backward_entry_points_reject_bad_arguments(L):
    """Host-side rejections of the backward calls added for the
    pre-activated convolution, the classifier and Distribute + PointNet:
    nothing is enqueued and the status names the problem."""
    gl = L.Lattice.create(_dev(_cloud(9, 800)), [0.1] * 3)
    dev = dict(dtype=torch.float32, device="cuda")
    x = torch.randn((gl.n, 12), **dev)
    W = torch.randn((9, 8, 12), **dev)
    dy = torch.randn((gl.n, 8), **dev)
    with pytest.raises(L.LatticeError) as e:
        gl.conv_preact_backward(gl, x, W, dy, groups=5)                 # 5 does not divide 12
    assert e.value.status == -1
    with pytest.raises(L.LatticeError) as e:
        gl.conv_preact_backward(gl, x, W, dy, groups=4, eps=0.0)        # eps must be positive
    assert e.value.status == -1
    other = L.Lattice.create(_dev(_cloud(10, 800)), [0.1] * 3)
    with pytest.raises(L.LatticeError) as e:
        gl.conv_preact_backward(other, x, W, dy, groups=4)             # unrelated lattices
    assert e.value.status == -8
    xv = torch.randn((gl.n, 16), **dev)
    with pytest.raises(L.LatticeError) as e:                            # 65 classes
        gl.deform_slice_classify_backward(xv, torch.randn(16, **dev), 0.1, torch.randn((65, 16), **dev),
                                          torch.randn((gl.m, 65), **dev))
    assert e.value.status == -2
    with pytest.raises(L.LatticeError) as e:                            # beta not finite
        gl.deform_slice_classify_backward(xv, torch.randn(16, **dev), float("nan"), torch.randn((4, 16), **dev),
                                          torch.randn((gl.m, 4), **dev))
    assert e.value.status == -1
    pos = _dev(_cloud(9, 800))
    lay = [(torch.randn((16, 5), **dev), None), (torch.randn((48, 16), **dev), None), (torch.randn((16, 48), **dev), None)]
    with pytest.raises(L.LatticeError) as e:                            # a 48-wide normalised layer input
        gl.distribute_pointnet_backward(pos, torch.randn((800, 2), **dev), lay, torch.randn((gl.n, 16), **dev))
    assert e.value.status == -2
    lay = [(torch.randn((16, 5), **dev), None), (torch.randn((32, 16), **dev), None), (torch.randn((16, 32), **dev), None)]
    with pytest.raises(L.LatticeError) as e:                            # Cf = 30 > 29
        gl.distribute_pointnet_backward(pos, torch.randn((800, 30), **dev),
                                        [(torch.randn((16, 33), **dev), None)] + lay[1:],
                                        torch.randn((gl.n, 16), **dev))
    assert e.value.status == -2
    xb = torch.randn((gl.n, 12), **dev).to(torch.bfloat16)
    with pytest.raises(L.LatticeError) as e:                            # bf16 channels not a multiple of 8
        gl.conv_backward_bf16(gl, xb, W.to(torch.bfloat16), dy.to(torch.bfloat16))
    assert e.value.status == -2
    other.destroy()
    gl.destroy()
