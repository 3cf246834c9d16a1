"""Comparison helpers for GPU-vs-oracle parity tests.

Lattice structure is compared bit for bit after ordering the GPU's vertices
by key (the oracle numbers vertices in lexicographic key order).  Features
are compared with the elementwise bound
    |g - r| <= tol * |r| + tol * rms(r)
per tensor (relative, with an absolute floor at the tensor's RMS so that
entries near zero do not demand more than the arithmetic can give), and
with the normwise relative error ||g - r|| / ||r|| <= tol.

The elementwise bound holds for one operator at a time.  In a bf16 network
both sides round every stored activation, but from accumulators of
different precision (fp32 on the GPU, float64 in the oracle), so a value
near a rounding boundary can land one bf16 ulp (2^-8 relative) apart and
later layers carry that difference on; bf16 networks are therefore checked
operator by operator on the inputs the GPU stored (assert_close) and end to
end by the normwise error alone (assert_normwise).
"""
from __future__ import annotations

import numpy as np

TOL_F32 = 1e-4
TOL_BF16 = 2e-2


def key_permutation(gpu_keys: np.ndarray, oracle_keys: np.ndarray) -> np.ndarray:
    """gpu2orc[v] = oracle index of GPU vertex v; asserts equal vertex sets."""
    gk = np.asarray(gpu_keys, dtype=np.int64)
    ok = np.asarray(oracle_keys, dtype=np.int64)
    assert gk.shape == ok.shape, f"vertex count {gk.shape[0]} vs oracle {ok.shape[0]}"
    order = np.lexsort(gk.T[::-1])
    assert np.array_equal(gk[order], ok), "vertex sets differ"
    gpu2orc = np.empty(gk.shape[0], dtype=np.int64)
    gpu2orc[order] = np.arange(gk.shape[0])
    return gpu2orc


def remap_index(tab: np.ndarray, gpu2orc: np.ndarray) -> np.ndarray:
    """Map GPU vertex indices (-1 = none) to oracle numbering."""
    t = np.asarray(tab, dtype=np.int64)
    return np.where(t >= 0, gpu2orc[np.maximum(t, 0)], -1)


def rows_in_oracle_order(x: np.ndarray, gpu2orc: np.ndarray) -> np.ndarray:
    out = np.empty_like(x)
    out[gpu2orc] = x
    return out


def assert_close(got, ref, tol, what=""):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, f"{what}: shape {got.shape} vs {ref.shape}"
    if ref.size == 0:
        return
    assert np.isfinite(got).all(), f"{what}: non-finite values"
    rms = float(np.sqrt(np.mean(ref * ref)))
    err = np.abs(got - ref)
    bound = tol * np.abs(ref) + tol * rms
    nrm = float(np.linalg.norm(ref))
    if nrm > 0:
        rel = float(np.linalg.norm(got - ref)) / nrm
        assert rel <= tol, f"{what}: normwise relative error {rel:.3g} > {tol}"
    bad = err > bound
    if bad.any():
        i = np.unravel_index(np.argmax(err / np.maximum(bound, 1e-300)), err.shape)
        raise AssertionError(
            f"{what}: {int(bad.sum())}/{ref.size} entries out of tolerance {tol}; worst at {i}: "
            f"got {got[i]!r} ref {ref[i]!r} (rms {rms:.3g}, max abs err {err.max():.3g})")


def assert_normwise(got, ref, tol, what=""):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, f"{what}: shape {got.shape} vs {ref.shape}"
    assert np.isfinite(got).all(), f"{what}: non-finite values"
    nrm = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(got - ref)) / nrm if nrm > 0 else float(np.linalg.norm(got))
    assert rel <= tol, f"{what}: normwise relative error {rel:.3g} > {tol}"


def max_errors(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    err = np.abs(got - ref)
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    return float(err.max(initial=0.0)), float((err / (np.abs(ref) + rms + 1e-300)).max(initial=0.0))
