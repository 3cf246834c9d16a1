"""ctypes wrapper of the CPU oracle (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg use
this module.  It takes numpy arrays on the host; features are float64.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

from . import build as _build

_lib = None

ERRORS = {0: "OK", -1: "EINVAL", -2: "EUNSUPPORTED", -3: "ENOMEM", -4: "EHASHFULL",
          -5: "EKEYRANGE", -6: "ENONFINITE", -7: "EDEVICE", -8: "ELEVEL"}


class OracleError(RuntimeError):
    def __init__(self, code):
        super().__init__(f"oracle returned {ERRORS.get(code, code)}")
        self.code = code


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = C.CDLL(_build.LIB)
        p, i64, i32, dbl = C.c_void_p, C.c_int64, C.c_int, C.c_double
        sig = {
            "orc_axis_factors": (None, [p, p]),
            "orc_elevate": (i32, [p, i64, p, p]),
            "orc_simplex": (i32, [p, i64, p, p]),
            "orc_create": (i32, [p, i64, i32, p, C.POINTER(C.c_void_p)]),
            "orc_coarsen": (i32, [p, C.POINTER(C.c_void_p)]),
            "orc_destroy": (None, [p]),
            "orc_num_vertices": (i64, [p]),
            "orc_num_points": (i64, [p]),
            "orc_level": (i32, [p]),
            "orc_export_elevated": (None, [p, p]),
            "orc_export_keys": (None, [p, p]),
            "orc_export_simplices": (None, [p, p, p]),
            "orc_export_neighbors": (None, [p, p]),
            "orc_export_down_table": (None, [p, p]),
            "orc_export_up_table": (None, [p, p]),
            "orc_splat": (i32, [p, p, i32, i32, p, p]),
            "orc_conv": (i32, [p, p, p, i64, i32, p, p, i32, i32, p, i64, p, i64]),
            "orc_refine": (i32, [p, p, p, i64, i32, p, p, i32, i32, p, i64, p, i64]),
            "orc_slice_raw": (None, [p, i64, i32, p, p, i64, p, p]),
            "orc_deform_slice_raw": (None, [p, i64, i32, p, p, i64, p, dbl, p, p, p]),
            "orc_slice": (i32, [p, p, i64, i32, p, i64, p]),
            "orc_deform_slice": (i32, [p, p, i64, i32, p, dbl, p, i64, p, p]),
            "orc_round_bf16": (None, [p, i64]),
            "orc_distribute_pointnet": (i32, [p, p, p, i32, p, p, dbl, p, p, i32, p, p, i32, p, p, i32, p]),
            "orc_splat_backward": (i32, [p, p, i32, i32, p]),
            "orc_groupnorm": (i32, [p, i64, i32, i64, i32, p, p, dbl, i32, p, i64]),
            "orc_deform_slice_classify": (i32, [p, p, i64, i32, p, dbl, p, p, i32, p]),
            "orc_slice_backward": (i32, [p, p, i32, p]),
            "orc_conv_backward": (i32, [p, p, p, i32, p, i32, i32, p, p, p, p, p]),
            "orc_deform_slice_backward": (i32, [p, p, i32, p, dbl, p, p, p, p]),
            "orc_groupnorm_backward": (i32, [p, i64, i32, i32, p, p, dbl, i32, p, p, p, p]),
            "orc_distribute_pointnet_backward": (i32, [p, p, p, i32, p, p, dbl, p, p, i32, p, p, i32, p, p, i32, p, p,
                                                       p, p, p, p, p, p, p, p, p]),
            "orc_deform_slice_classify_backward": (i32, [p, p, i32, p, dbl, p, i32, p, p, p, p, p, p]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _check(code):
    if code != 0:
        raise OracleError(code)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def axis_factors(sigma) -> np.ndarray:
    s = _f32(sigma)
    a = np.zeros(3, np.float32)
    lib().orc_axis_factors(_ptr(s), _ptr(a))
    return a


def elevate(pos, sigma) -> np.ndarray:
    pos, sigma = _f32(pos), _f32(sigma)
    y = np.zeros((pos.shape[0], 4), np.float32)
    _check(lib().orc_elevate(_ptr(pos), pos.shape[0], _ptr(sigma), _ptr(y)))
    return y


def simplex(y):
    """Enclosing simplex of elevated points: keys (m,4,4) int32, w (m,4) f32."""
    y = _f32(y).reshape(-1, 4)
    m = y.shape[0]
    keys = np.zeros((m, 4, 4), np.int32)
    w = np.zeros((m, 4), np.float32)
    _check(lib().orc_simplex(_ptr(y), m, _ptr(keys), _ptr(w)))
    return keys, w


def round_bf16(x) -> np.ndarray:
    a = np.array(x, dtype=np.float64, copy=True, order="C")
    lib().orc_round_bf16(_ptr(a), a.size)
    return a


class Lattice:
    """A lattice held by the oracle (std::map numbering = lexicographic keys)."""

    def __init__(self, handle, parent=None):
        self._h = handle
        self.parent = parent
        self.n = int(lib().orc_num_vertices(handle))
        self.m = int(lib().orc_num_points(handle))
        self.level = int(lib().orc_level(handle))

    @classmethod
    def create(cls, pos, sigma, d: int = 3):
        pos, sigma = _f32(pos).reshape(-1, 3) if d == 3 else _f32(pos), _f32(sigma)
        h = C.c_void_p()
        _check(lib().orc_create(_ptr(pos), pos.shape[0], d, _ptr(sigma), C.byref(h)))
        return cls(h)

    def coarsen(self):
        h = C.c_void_p()
        _check(lib().orc_coarsen(self._h, C.byref(h)))
        return Lattice(h, parent=self)

    def __del__(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.orc_destroy(self._h)
            self._h = None

    # ---- structure ----
    def elevated(self):
        y = np.zeros((self.m, 4), np.float32)
        lib().orc_export_elevated(self._h, _ptr(y))
        return y

    def keys(self):
        k = np.zeros((self.n, 4), np.int32)
        lib().orc_export_keys(self._h, _ptr(k))
        return k

    def simplices(self):
        idx = np.zeros((self.m, 4), np.int64)
        w = np.zeros((self.m, 4), np.float32)
        lib().orc_export_simplices(self._h, _ptr(idx), _ptr(w))
        return idx, w

    def neighbors(self):
        nb = np.zeros((self.n, 9), np.int64)
        lib().orc_export_neighbors(self._h, _ptr(nb))
        return nb

    def down_table(self):
        """For a coarsened lattice: fine vertex at 2c + o_t (n_coarse x 9)."""
        nb = np.zeros((self.n, 9), np.int64)
        lib().orc_export_down_table(self._h, _ptr(nb))
        return nb

    def up_table(self):
        """For a coarsened lattice: coarse vertex read by each fine vertex and
        tap (n_fine x 9)."""
        nb = np.zeros((self.parent.n, 9), np.int64)
        lib().orc_export_up_table(self._h, _ptr(nb))
        return nb

    # ---- ops ----
    def splat(self, F, normalize=True):
        F = _f64(F)
        Cc = F.shape[1]
        X = np.zeros((self.n, Cc), np.float64)
        W = np.zeros(self.n, np.float64)
        _check(lib().orc_splat(self._h, _ptr(F), Cc, int(bool(normalize)), _ptr(X), _ptr(W)))
        return X, W

    def distribute_pointnet(self, G, F, layers, gn=None, eps=1e-5):
        """Distribute + PointNet: layers = [(W1, b1), (W2, b2), (W3, b3)],
        W_i laid out [out][in] (the first layer's inputs: d coordinates, then
        the Cf features); gn = None or (gamma, beta), each the concatenated
        per-channel parameters of the three GroupNorms ((d + Cf) + C1 + C2).
        G are the raw positions (divided by the lattice's sigma inside).
        Returns n x C3."""
        G = _f64(G)
        F = _f64(F) if F is not None else np.zeros((G.shape[0], 0))
        (W1, b1), (W2, b2), (W3, b3) = [(_f64(W), None if b is None else _f64(b)) for W, b in layers]
        cf = F.shape[1]
        c1, c2, c3 = W1.shape[0], W2.shape[0], W3.shape[0]
        assert W1.shape[1] == G.shape[1] + cf and W2.shape[1] == c1 and W3.shape[1] == c2
        gam = bet = None
        if gn is not None:
            gam, bet = (None if a is None else _f64(a) for a in gn)
            for a in (gam, bet):
                assert a is None or a.shape == (G.shape[1] + cf + c1 + c2,)
        X = np.zeros((self.n, c3), np.float64)
        _check(lib().orc_distribute_pointnet(self._h, _ptr(G), _ptr(F) if cf else None, cf, _ptr(gam), _ptr(bet),
                                             float(eps), _ptr(W1), _ptr(b1), c1, _ptr(W2), _ptr(b2), c2, _ptr(W3),
                                             _ptr(b3), c3, _ptr(X)))
        return X

    def distribute_pointnet_backward(self, G, F, layers, dX, gn=None, eps=1e-5):
        """Gradients of distribute_pointnet(G, F, layers, gn, eps) for
        dL/dX = dX: a dict with dF (m x Cf), dW1..dW3 ([out][in]),
        db1..db3, dgamma and dbeta (concatenated as gn), and margin (n x C3:
        the largest minus the second largest row of J_v per channel)."""
        G = _f64(G)
        F = _f64(F) if F is not None else np.zeros((G.shape[0], 0))
        (W1, b1), (W2, b2), (W3, b3) = [(_f64(W), None if b is None else _f64(b)) for W, b in layers]
        cf = F.shape[1]
        c1, c2, c3 = W1.shape[0], W2.shape[0], W3.shape[0]
        gam = bet = None
        if gn is not None:
            gam, bet = (None if a is None else _f64(a) for a in gn)
        dX = _f64(dX)
        assert dX.shape == (self.n, c3)
        ng = G.shape[1] + cf + c1 + c2
        out = dict(dF=np.zeros((G.shape[0], cf)), dW1=np.zeros_like(W1), db1=np.zeros(c1), dW2=np.zeros_like(W2),
                   db2=np.zeros(c2), dW3=np.zeros_like(W3), db3=np.zeros(c3), dgamma=np.zeros(ng),
                   dbeta=np.zeros(ng), margin=np.zeros((self.n, c3)))
        _check(lib().orc_distribute_pointnet_backward(
            self._h, _ptr(G), _ptr(F) if cf else None, cf, _ptr(gam), _ptr(bet), float(eps), _ptr(W1), _ptr(b1), c1,
            _ptr(W2), _ptr(b2), c2, _ptr(W3), _ptr(b3), c3, _ptr(dX), _ptr(out["dF"]) if cf else None,
            _ptr(out["dW1"]), _ptr(out["db1"]), _ptr(out["dW2"]), _ptr(out["db2"]), _ptr(out["dW3"]),
            _ptr(out["db3"]), _ptr(out["dgamma"]), _ptr(out["dbeta"]), _ptr(out["margin"])))
        return out

    def conv(self, src: "Lattice", X, W, bias=None, relu=False, rows=None):
        """dst = self.  src is self (1-hop conv) or self.parent (strided)."""
        X, W = _f64(X), _f64(W)
        cin, cout = W.shape[1], W.shape[2]
        assert X.shape[1] == cin
        b = None if bias is None else _f64(bias)
        r = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
        nr = self.n if r is None else r.shape[0]
        Y = np.zeros((nr, cout), np.float64)
        _check(lib().orc_conv(self._h, src._h, _ptr(X), cin, cin, _ptr(W), _ptr(b), cout,
                              int(bool(relu)), _ptr(r), nr, _ptr(Y), cout))
        return Y

    def refine_into(self, coarse: "Lattice", X, W, bias=None, relu=False, rows=None):
        """Upsample coarse (a coarsening of self) values X to self."""
        X, W = _f64(X), _f64(W)
        cin, cout = W.shape[1], W.shape[2]
        assert X.shape[1] == cin
        b = None if bias is None else _f64(bias)
        r = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
        nr = self.n if r is None else r.shape[0]
        Y = np.zeros((nr, cout), np.float64)
        _check(lib().orc_refine(self._h, coarse._h, _ptr(X), cin, cin, _ptr(W), _ptr(b), cout,
                                int(bool(relu)), _ptr(r), nr, _ptr(Y), cout))
        return Y

    # ---- backward ----
    def splat_backward(self, dX, normalize=True):
        """dL/dF of splat for dL/dX = dX (n x C)."""
        dX = _f64(dX)
        Cc = dX.shape[1]
        dF = np.zeros((self.m, Cc), np.float64)
        _check(lib().orc_splat_backward(self._h, _ptr(dX), Cc, int(bool(normalize)), _ptr(dF)))
        return dF

    def slice_backward(self, dOut):
        """dL/dX of slice for dL/dout = dOut (m x C)."""
        dOut = _f64(dOut)
        Cc = dOut.shape[1]
        dX = np.zeros((self.n, Cc), np.float64)
        _check(lib().orc_slice_backward(self._h, _ptr(dOut), Cc, _ptr(dX)))
        return dX

    def conv_backward(self, src: "Lattice", X, W, dY, relu=False, Y=None):
        """Gradients of Y = act(conv(src -> self)(X, W) + bias) for dL/dY = dY:
        (dX, dW, dbias).  src is self, self.parent (strided) or a coarsening
        of self (Upsample into self).  W laid out [tap][c_in][c_out]."""
        X, W, dY = _f64(X), _f64(W), _f64(dY)
        cin, cout = W.shape[1], W.shape[2]
        Yc = None if Y is None else _f64(Y)
        dX = np.zeros((src.n, cin), np.float64)
        dW = np.zeros(W.shape, np.float64)
        db = np.zeros(cout, np.float64)
        _check(lib().orc_conv_backward(self._h, src._h, _ptr(X), cin, _ptr(W), cout, int(bool(relu)), _ptr(Yc),
                                       _ptr(dY), _ptr(dX), _ptr(dW), _ptr(db)))
        return dX, dW, db

    def deform_slice_backward(self, X, wv, beta, dOut):
        """Gradients of deform_slice(X, wv, beta) for dL/dout = dOut:
        (dX, dwv, dbeta)."""
        X, wv, dOut = _f64(X), _f64(wv), _f64(dOut)
        Cc = X.shape[1]
        dX = np.zeros((self.n, Cc), np.float64)
        dwv = np.zeros(Cc, np.float64)
        dbeta = np.zeros(1, np.float64)
        _check(lib().orc_deform_slice_backward(self._h, _ptr(X), Cc, _ptr(wv), float(beta), _ptr(dOut), _ptr(dX),
                                               _ptr(dwv), _ptr(dbeta)))
        return dX, dwv, float(dbeta[0])

    def deform_slice_classify_backward(self, X, wv, beta, Wc, dZ):
        """Gradients of deform_slice_classify(X, wv, beta, Wc, bc) for
        dL/dlogits = dZ: (dX, dwv, dbeta, dWc, dbc)."""
        X, wv, Wc, dZ = _f64(X), _f64(wv), _f64(Wc), _f64(dZ)
        Cc, K = X.shape[1], Wc.shape[0]
        assert Wc.shape[1] == Cc and dZ.shape == (self.m, K)
        dX = np.zeros((self.n, Cc), np.float64)
        dwv = np.zeros(Cc, np.float64)
        dbeta = np.zeros(1, np.float64)
        dWc = np.zeros((K, Cc), np.float64)
        dbc = np.zeros(K, np.float64)
        _check(lib().orc_deform_slice_classify_backward(self._h, _ptr(X), Cc, _ptr(wv), float(beta), _ptr(Wc), K,
                                                        _ptr(dZ), _ptr(dX), _ptr(dwv), _ptr(dbeta), _ptr(dWc),
                                                        _ptr(dbc)))
        return dX, dwv, float(dbeta[0]), dWc, dbc

    def slice(self, X, pts=None):
        X = _f64(X)
        Cc = X.shape[1]
        p = None if pts is None else np.ascontiguousarray(pts, dtype=np.int64)
        npt = self.m if p is None else p.shape[0]
        out = np.zeros((npt, Cc), np.float64)
        _check(lib().orc_slice(self._h, _ptr(X), Cc, Cc, _ptr(p), npt, _ptr(out)))
        return out

    def deform_slice_classify(self, X, wv, beta, Wc, bc=None):
        """DeformSlice fused with a linear classifier: m x K logits,
        Wc [class][channel]."""
        X, wv, Wc = _f64(X), _f64(wv), _f64(Wc)
        Cc, K = X.shape[1], Wc.shape[0]
        assert Wc.shape[1] == Cc
        b = None if bc is None else _f64(bc)
        out = np.zeros((self.m, K), np.float64)
        _check(lib().orc_deform_slice_classify(self._h, _ptr(X), Cc, Cc, _ptr(wv), float(beta), _ptr(Wc), _ptr(b), K,
                                               _ptr(out)))
        return out

    def deform_slice(self, X, wv, beta, pts=None):
        X, wv = _f64(X), _f64(wv)
        Cc = X.shape[1]
        p = None if pts is None else np.ascontiguousarray(pts, dtype=np.int64)
        npt = self.m if p is None else p.shape[0]
        out = np.zeros((npt, Cc), np.float64)
        delta = np.zeros((npt, 4), np.float64)
        _check(lib().orc_deform_slice(self._h, _ptr(X), Cc, Cc, _ptr(wv), float(beta), _ptr(p), npt,
                                      _ptr(out), _ptr(delta)))
        return out, delta


def groupnorm(X, groups, gamma=None, beta=None, eps=1e-5, relu=False):
    """Group Normalization over the rows of X (n x C), optional ReLU."""
    X = _f64(X)
    n, Cc = X.shape
    g = None if gamma is None else _f64(gamma)
    b = None if beta is None else _f64(beta)
    Y = np.zeros_like(X)
    _check(lib().orc_groupnorm(_ptr(X), n, Cc, Cc, int(groups), _ptr(g), _ptr(b), float(eps), int(bool(relu)),
                               _ptr(Y), Cc))
    return Y


def groupnorm_backward(X, dY, groups, gamma=None, beta=None, eps=1e-5, relu=False):
    """Gradients of groupnorm(X, groups, gamma, beta, eps, relu) for
    dL/dY = dY: (dX, dgamma, dbeta)."""
    X, dY = _f64(X), _f64(dY)
    n, Cc = X.shape
    assert dY.shape == X.shape
    g = None if gamma is None else _f64(gamma)
    b = None if beta is None else _f64(beta)
    dX = np.zeros_like(X)
    dg = np.zeros(Cc, np.float64)
    db = np.zeros(Cc, np.float64)
    _check(lib().orc_groupnorm_backward(_ptr(X), n, Cc, int(groups), _ptr(g), _ptr(b), float(eps), int(bool(relu)),
                                        _ptr(dY), _ptr(dX), _ptr(dg), _ptr(db)))
    return dX, dg, db


def slice_raw(X, idx, w):
    X = _f64(X)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    w = _f32(w)
    m, Cc = idx.shape[0], X.shape[1]
    out = np.zeros((m, Cc), np.float64)
    lib().orc_slice_raw(_ptr(X), Cc, Cc, _ptr(idx), _ptr(w), m, None, _ptr(out))
    return out


def deform_slice_raw(X, idx, w, wv, beta):
    X, wv = _f64(X), _f64(wv)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    w = _f32(w)
    m, Cc = idx.shape[0], X.shape[1]
    out = np.zeros((m, Cc), np.float64)
    delta = np.zeros((m, 4), np.float64)
    lib().orc_deform_slice_raw(_ptr(X), Cc, Cc, _ptr(idx), _ptr(w), m, _ptr(wv), float(beta), None,
                               _ptr(out), _ptr(delta))
    return out, delta
