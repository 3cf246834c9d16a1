"""lattice_splat_noalloc (the splat whose partials sit in the library's fixed
device scratch) against lattice_splat, through the C ABI: bit-identical
values and weight sums on two calls in a row, the second with a smaller
input; a coarse level whose point lists the call itself builds; the host-side
rejections (count not read yet, partials larger than the scratch)."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1912_05905_amd import lattice
    lattice.lib()
    return lattice


def _cloud(seed, m, extent):
    rng = np.random.default_rng(seed)
    return torch.from_numpy((extent * rng.random((m, 3))).astype(np.float32)).cuda()


def _both(lat, feat, normalize):
    n, C = lat.n, feat.shape[1]
    ref = torch.empty((n, C), dtype=feat.dtype, device="cuda")
    ws_ref = torch.empty(n, device="cuda")
    lat.splat(feat, normalize, out=ref, wsum=ws_ref)
    got = torch.full((n, C), float("nan"), dtype=feat.dtype, device="cuda")
    ws = torch.full((n,), float("nan"), device="cuda")
    lat.splat_noalloc(feat, normalize, out=got, wsum=ws)
    torch.cuda.synchronize()
    assert torch.equal(got.view(torch.int16 if feat.dtype == torch.bfloat16 else torch.int32),
                       ref.view(torch.int16 if feat.dtype == torch.bfloat16 else torch.int32))
    assert torch.equal(ws.view(torch.int32), ws_ref.view(torch.int32))


def test_noalloc_splat_matches_splat(L):
    print("noalloc: 200k points, 64 fp32 channels, then 5k points, 32 bf16 channels", flush=True)
    big = L.Lattice.create(_cloud(1, 200_000, 4.0), [0.05] * 3)
    feat = torch.from_numpy(np.random.default_rng(2).normal(size=(200_000, 64)).astype(np.float32)).cuda()
    _both(big, feat, True)
    small = L.Lattice.create(_cloud(3, 5_000, 1.0), [0.08] * 3)
    fs = torch.from_numpy(np.random.default_rng(4).normal(size=(5_000, 32)).astype(np.float32)).cuda()
    _both(small, fs.to(torch.bfloat16), False)
    # the larger call again after the smaller one (the scratch keeps the
    # smaller call's partials)
    _both(big, feat, False)
    small.destroy()
    big.destroy()


def test_noalloc_splat_on_a_coarse_level(L):
    print("noalloc: coarse level built lazily", flush=True)
    fine = L.Lattice.create(_cloud(5, 50_000, 2.0), [0.05] * 3)
    coarse = fine.coarsen()
    feat = torch.from_numpy(np.random.default_rng(6).normal(size=(50_000, 16)).astype(np.float32)).cuda()
    n = coarse.n
    got = torch.empty((n, 16), device="cuda")
    coarse.splat_noalloc(feat, True, out=got)     # builds the coarse level's lists first
    ref = coarse.splat(feat, True)
    torch.cuda.synchronize()
    assert torch.equal(got.view(torch.int32), ref.view(torch.int32))
    coarse.destroy()
    fine.destroy()


def test_noalloc_splat_rejections(L):
    lib = L.lib()
    pos = _cloud(7, 200_000, 4.0)
    lat = L.Lattice.create(pos, [0.05] * 3)
    feat = torch.zeros((200_000, 1024), device="cuda")
    out = torch.zeros((16, 1024), device="cuda")
    # the vertex count has not been read yet
    st = lib.lattice_splat_noalloc(lat._h, ctypes.c_void_p(feat.data_ptr()), 0, 1024, 0, 1,
                                   ctypes.c_void_p(out.data_ptr()), 0, None, None)
    assert st == -1
    n = lat.n
    vals = torch.zeros((n, 1024), device="cuda")
    # partials of 1024 channels over 800k list entries exceed the scratch
    st = lib.lattice_splat_noalloc(lat._h, ctypes.c_void_p(feat.data_ptr()), 0, 1024, 0, 1,
                                   ctypes.c_void_p(vals.data_ptr()), 0, None, None)
    assert st == -2
    assert b"scratch" in lib.lattice_last_error()
    torch.cuda.synchronize()
    lat.destroy()
