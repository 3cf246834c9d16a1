"""Python binding of liblattice (ctypes).

Argument marshalling only: every lattice operation runs in the library's HIP
kernels.  PyTorch supplies device memory (tensors) and the current HIP
stream.  The library must be built (``python -m paper_1912_05905_amd.build``);
importing this module without it raises, there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblattice.so")

LAT_F32, LAT_BF16 = 0, 1
LAT_RELU = 1
LAT_ON_STREAM = 1
TAPS = 9
STATUS = {0: "LAT_OK", -1: "LAT_EINVAL", -2: "LAT_EUNSUPPORTED", -3: "LAT_ENOMEM",
          -4: "LAT_EHASHFULL", -5: "LAT_EKEYRANGE", -6: "LAT_ENONFINITE", -7: "LAT_EDEVICE",
          -8: "LAT_ELEVEL"}

_lib = None

# exported entry points and their argument types
_P, _I64, _I32, _F32 = C.c_void_p, C.c_int64, C.c_int, C.c_float
SIGNATURES = {
    "lattice_last_error": (C.c_char_p, []),
    "lattice_status_string": (C.c_char_p, [_I32]),
    "lattice_create": (_I32, [_P, _I64, _I32, _P, _I64, _P, C.POINTER(_P)]),
    "lattice_coarsen": (_I32, [_P, _I64, _P, C.POINTER(_P)]),
    "lattice_coarsen_ex": (_I32, [_P, _I64, _I32, _P, C.POINTER(_P)]),
    "lattice_create_hierarchy": (_I32, [_P, _I64, _I32, _P, _I32, _P, _P, C.POINTER(_P)]),
    "lattice_destroy": (_I32, [_P]),
    "lattice_num_vertices": (_I32, [_P, C.POINTER(_I64)]),
    "lattice_num_points": (_I32, [_P, C.POINTER(_I64)]),
    "lattice_level": (_I32, [_P, C.POINTER(_I32)]),
    "lattice_export_keys": (_I32, [_P, _P, _P]),
    "lattice_export_simplices": (_I32, [_P, _P, _P, _P]),
    "lattice_export_neighbors": (_I32, [_P, _P, _P]),
    "lattice_splat": (_I32, [_P, _P, _I64, _I32, _I32, _I32, _P, _I64, _P, _P]),
    "lattice_splat_noalloc": (_I32, [_P, _P, _I64, _I32, _I32, _I32, _P, _I64, _P, _P]),
    "lattice_conv_taps": (_I32, [_P, _P, C.POINTER(_I64), _P]),
    "lattice_conv": (_I32, [_P, _P, _P, _I64, _I32, _P, _P, _I32, _I32, _I32, _P, _I64, _P]),
    "lattice_refine": (_I32, [_P, _P, _P, _I64, _I32, _P, _P, _I32, _I32, _I32, _P, _I64, _P]),
    "lattice_slice": (_I32, [_P, _P, _I64, _I32, _I32, _P, _P]),
    "lattice_deform_slice": (_I32, [_P, _P, _I64, _I32, _I32, _P, _F32, _P, _P, _P]),
    "lattice_slice_and_deform": (_I32, [_P, _P, _I64, _I32, _I32, _P, _F32, _P, _P, _P]),
    "lattice_conv_preact": (_I32, [_P, _P, _P, _I64, _I32, _I32, _P, _P, _F32, _P, _P, _I32, _I32, _I32, _P, _I64,
                                   _P, _I64, _P]),
    "lattice_refine_preact": (_I32, [_P, _P, _P, _I64, _I32, _I32, _P, _P, _F32, _P, _P, _I32, _I32, _I32, _P,
                                     _I64, _P]),
    "lattice_deform_slice_classify": (_I32, [_P, _P, _I64, _I32, _I32, _P, _F32, _P, _P, _I32, _P, _P]),
    "lattice_distribute_pointnet": (_I32, [_P, _P, _P, _I64, _I32, _P, _P, C.c_float, _P, _P, _I32, _P, _P,
                                           _I32, _P, _P, _I32, _I32, _P, _I64, _P]),
    "lattice_splat_backward": (_I32, [_P, _P, _I64, _I32, _I32, _P, _P, _P]),
    "lattice_slice_backward": (_I32, [_P, _P, _I64, _I32, _P, _I64, _P]),
    "lattice_conv_backward": (_I32, [_P, _P, _P, _I64, _I32, _P, _I32, _I32, _P, _I64, _P, _I64, _P, _I64, _P, _P,
                                     _P]),
    "lattice_conv_preact_backward": (_I32, [_P, _P, _P, _I64, _I32, _I32, _P, _P, _F32, _P, _I32, _I32, _P, _I64,
                                            _P, _I64, _P, _I64, _P, _P, _P, _P, _P]),
    "lattice_deform_slice_classify_backward": (_I32, [_P, _P, _I64, _I32, _P, _F32, _P, _I32, _P, _I64, _P, _I64,
                                                      _P, _P, _P, _P, _P]),
    "lattice_distribute_pointnet_backward": (_I32, [_P, _P, _P, _I64, _I32, _P, _P, C.c_float, _P, _P, _I32, _P, _P,
                                                    _I32, _P, _P, _I32, _P, _I64, _P, _I64, _P, _P, _P, _P, _P, _P,
                                                    _P, _P, _P]),
    "lattice_conv_backward_ex": (_I32, [_P, _P, _P, _I64, _I32, _P, _I32, _I32, _I32, _P, _I64, _P, _I64, _P, _I64,
                                        _P, _P, _P]),
    "lattice_deform_slice_backward": (_I32, [_P, _P, _I64, _I32, _P, _F32, _P, _I64, _P, _I64, _P, _P, _P]),
    "lattice_timing_enable": (_I32, [C.c_char_p, _I32]),
    "lattice_timing_read": (_I32, [C.c_char_p, C.POINTER(_I64), C.POINTER(C.c_double)]),
}


class LatticeError(RuntimeError):
    def __init__(self, status: int, text: str):
        super().__init__(text or STATUS.get(status, str(status)))
        self.status = status


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with python -m paper_1912_05905_amd.build")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(status: int):
    if status != 0:
        raise LatticeError(status, lib().lattice_last_error().decode())


# the raw handle of the current stream without building a torch Stream
# object (which costs microseconds per call)
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)
_raw_device = getattr(torch._C, "_cuda_getDevice", None)


def _stream(stream=None):
    if stream is not None:
        return C.c_void_p(stream.cuda_stream)
    if _raw_stream is not None and _raw_device is not None:
        return C.c_void_p(_raw_stream(_raw_device()))
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return LAT_F32
    if t.dtype == torch.bfloat16:
        return LAT_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _rows(t: torch.Tensor):
    """(pointer, row stride) of a row-major matrix or a column slice of one."""
    if t.dim() != 2 or (t.shape[1] > 1 and t.stride(1) != 1):
        raise ValueError("expected a 2-D tensor with unit column stride")
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    return C.c_void_p(t.data_ptr()), t.stride(0)


def timing_enable(family: str, enable: bool = True):
    _check(lib().lattice_timing_enable(family.encode(), int(enable)))


def timing_read(family: str):
    n = C.c_int64()
    ms = C.c_double()
    _check(lib().lattice_timing_read(family.encode(), C.byref(n), C.byref(ms)))
    return int(n.value), float(ms.value)


class Lattice:
    """A sparse permutohedral lattice owned by liblattice."""

    def __init__(self, handle: C.c_void_p, parent: "Lattice | None" = None, m: int | None = None):
        self._h = handle
        self.parent = parent
        self._n = None
        if m is None:
            mm, lv = C.c_int64(), C.c_int()
            _check(lib().lattice_num_points(handle, C.byref(mm)))
            _check(lib().lattice_level(handle, C.byref(lv)))
            self.m, self.level = int(mm.value), int(lv.value)
        else:
            # known to the caller: the points of a new lattice, or of its parent
            self.m, self.level = m, (parent.level + 1 if parent is not None else 0)

    @property
    def n(self) -> int:
        """Vertex count; the first read waits for the lattice's build to
        report it (and raises a device-side build error)."""
        if self._n is None:
            n = C.c_int64()
            _check(lib().lattice_num_vertices(self._h, C.byref(n)))
            self._n = int(n.value)
        return self._n

    # ---- construction ----
    @classmethod
    def create(cls, pos: torch.Tensor, sigma, capacity_hint: int = 0, stream=None) -> "Lattice":
        if pos.dtype != torch.float32 or pos.dim() != 2 or not pos.is_contiguous():
            raise ValueError("positions must be a contiguous m x d float32 tensor")
        sig = (C.c_float * pos.shape[1])(*[float(s) for s in sigma])
        h = C.c_void_p()
        _check(lib().lattice_create(C.c_void_p(pos.data_ptr()), pos.shape[0], pos.shape[1], sig,
                                    int(capacity_hint), _stream(stream), C.byref(h)))
        return cls(h, m=pos.shape[0])

    @classmethod
    def create_hierarchy(cls, pos: torch.Tensor, sigma, levels: int, stream=None, capacity_hints=None) -> list:
        """[level 0, level 1, ...]: create then levels - 1 coarsenings, all
        built on the given (or current) stream in one library call;
        capacity_hints: expected vertex counts per level (0 = automatic)."""
        if pos.dtype != torch.float32 or pos.dim() != 2 or not pos.is_contiguous():
            raise ValueError("positions must be a contiguous m x d float32 tensor")
        sig = (C.c_float * pos.shape[1])(*[float(s) for s in sigma])
        hs = (C.c_void_p * max(int(levels), 1))()
        hints = None
        if capacity_hints is not None:
            if len(capacity_hints) != int(levels):
                raise ValueError("capacity_hints needs one value per level")
            hints = (C.c_int64 * int(levels))(*[int(h) for h in capacity_hints])
        _check(lib().lattice_create_hierarchy(C.c_void_p(pos.data_ptr()), pos.shape[0], pos.shape[1], sig,
                                              int(levels), C.cast(hints, _P) if hints is not None else None,
                                              _stream(stream), hs))
        out = [cls(C.c_void_p(hs[0]), m=pos.shape[0])]
        for l in range(1, int(levels)):
            out.append(Lattice(C.c_void_p(hs[l]), parent=out[-1], m=pos.shape[0]))
        return out

    def coarsen(self, capacity_hint: int = 0, stream=None, on_stream: bool = False) -> "Lattice":
        """Coarser lattice (Downsample).  on_stream=True builds it on the
        given (or current) stream instead of the library's side stream."""
        h = C.c_void_p()
        _check(lib().lattice_coarsen_ex(self._h, int(capacity_hint), LAT_ON_STREAM if on_stream else 0,
                                        _stream(stream), C.byref(h)))
        return Lattice(h, parent=self, m=self.m)

    def destroy(self):
        if getattr(self, "_h", None):
            _check(lib().lattice_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            if getattr(self, "_h", None) and _lib is not None:
                _lib.lattice_destroy(self._h)
                self._h = None
        except Exception:
            pass

    @property
    def handle(self):
        return self._h

    # ---- structure export ----
    def keys(self, stream=None) -> torch.Tensor:
        k = torch.empty((self.n, 4), dtype=torch.int32, device="cuda")
        _check(lib().lattice_export_keys(self._h, C.c_void_p(k.data_ptr()), _stream(stream)))
        return k

    def simplices(self, stream=None):
        idx = torch.empty((self.m, 4), dtype=torch.int32, device="cuda")
        w = torch.empty((self.m, 4), dtype=torch.float32, device="cuda")
        _check(lib().lattice_export_simplices(self._h, C.c_void_p(idx.data_ptr()),
                                              C.c_void_p(w.data_ptr()), _stream(stream)))
        return idx, w

    def neighbors(self, stream=None) -> torch.Tensor:
        nb = torch.empty((self.n, TAPS), dtype=torch.int32, device="cuda")
        _check(lib().lattice_export_neighbors(self._h, C.c_void_p(nb.data_ptr()), _stream(stream)))
        return nb

    # ---- operators ----
    def splat(self, feat: torch.Tensor, normalize: bool = True, out: torch.Tensor | None = None,
              wsum: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        Cc = feat.shape[1]
        if out is None:
            out = torch.empty((self.n, Cc), dtype=feat.dtype, device="cuda")
        fp, fld = _rows(feat)
        op, old = _rows(out)
        _check(lib().lattice_splat(self._h, fp, fld, Cc, _dtype_code(feat), int(bool(normalize)),
                                   op, old, None if wsum is None else C.c_void_p(wsum.data_ptr()),
                                   _stream(stream)))
        return out

    def splat_noalloc(self, feat: torch.Tensor, normalize: bool = True, out: torch.Tensor | None = None,
                      wsum: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        """splat through lattice_splat_noalloc (its partials in the library's
        fixed device scratch; out must be given by callers that cannot
        allocate)."""
        Cc = feat.shape[1]
        if out is None:
            out = torch.empty((self.n, Cc), dtype=feat.dtype, device="cuda")
        fp, fld = _rows(feat)
        op, old = _rows(out)
        _check(lib().lattice_splat_noalloc(self._h, fp, fld, Cc, _dtype_code(feat), int(bool(normalize)),
                                           op, old, None if wsum is None else C.c_void_p(wsum.data_ptr()),
                                           _stream(stream)))
        return out

    def conv_taps(self, src: "Lattice") -> int:
        """(vertex, tap) pairs with an existing neighbour of the convolution
        from src into self (1-hop, strided or Upsample); waits."""
        n = _I64()
        _check(lib().lattice_conv_taps(self._h, src._h, C.byref(n), _stream(None)))
        return int(n.value)

    def conv(self, src: "Lattice", x: torch.Tensor, W: torch.Tensor, bias: torch.Tensor | None = None,
             relu: bool = False, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        """self is the destination lattice: src itself (1-hop) or its parent
        (strided convolution).  W is taps x Cout x Cin."""
        cout, cin = W.shape[1], W.shape[2]
        if out is None:
            out = torch.empty((self.n, cout), dtype=x.dtype, device="cuda")
        xp, xld = _rows(x)
        op, old = _rows(out)
        if not W.is_contiguous() or W.dtype != x.dtype:
            raise ValueError("W must be contiguous with the dtype of x")
        _check(lib().lattice_conv(self._h, src._h, xp, xld, cin, C.c_void_p(W.data_ptr()),
                                  None if bias is None else C.c_void_p(bias.data_ptr()), cout,
                                  _dtype_code(x), LAT_RELU if relu else 0, op, old, _stream(stream)))
        return out

    def refine(self, coarse: "Lattice", x: torch.Tensor, W: torch.Tensor,
               bias: torch.Tensor | None = None, relu: bool = False, out: torch.Tensor | None = None,
               stream=None) -> torch.Tensor:
        """self is the fine lattice; coarse = self.coarsen()."""
        cout, cin = W.shape[1], W.shape[2]
        if out is None:
            out = torch.empty((self.n, cout), dtype=x.dtype, device="cuda")
        xp, xld = _rows(x)
        op, old = _rows(out)
        if not W.is_contiguous() or W.dtype != x.dtype:
            raise ValueError("W must be contiguous with the dtype of x")
        _check(lib().lattice_refine(self._h, coarse._h, xp, xld, cin, C.c_void_p(W.data_ptr()),
                                    None if bias is None else C.c_void_p(bias.data_ptr()), cout,
                                    _dtype_code(x), LAT_RELU if relu else 0, op, old, _stream(stream)))
        return out

    def conv_preact(self, src: "Lattice", x: torch.Tensor, W: torch.Tensor, groups: int = 32,
                    gamma: torch.Tensor | None = None, beta: torch.Tensor | None = None, eps: float = 1e-5,
                    bias: torch.Tensor | None = None, relu: bool = False, out: torch.Tensor | None = None,
                    refine: bool = False, res: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        """conv(relu(GroupNorm(x))) (+ res): self is the destination; src as
        for conv (refine=False) or the coarse lattice of an Upsample
        (refine=True, no residual)."""
        cout, cin = W.shape[1], W.shape[2]
        if out is None:
            out = torch.empty((self.n, cout), dtype=x.dtype, device="cuda")
        xp, xld = _rows(x)
        op, old = _rows(out)
        if not W.is_contiguous() or W.dtype != x.dtype:
            raise ValueError("W must be contiguous with the dtype of x")
        ptr = lambda t: None if t is None else C.c_void_p(t.data_ptr())
        args = [self._h, src._h, xp, xld, cin, int(groups), ptr(gamma), ptr(beta), float(eps), ptr(W), ptr(bias),
                cout, _dtype_code(x), LAT_RELU if relu else 0]
        if refine:
            if res is not None:
                raise ValueError("no residual for an Upsample")
            _check(lib().lattice_refine_preact(*args, op, old, _stream(stream)))
        else:
            rp, rld = _rows(res) if res is not None else (None, 0)
            _check(lib().lattice_conv_preact(*args, rp, rld, op, old, _stream(stream)))
        return out

    def slice(self, x: torch.Tensor, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        Cc = x.shape[1]
        if out is None:
            out = torch.empty((self.m, Cc), dtype=torch.float32, device="cuda")
        xp, xld = _rows(x)
        _check(lib().lattice_slice(self._h, xp, xld, Cc, _dtype_code(x), C.c_void_p(out.data_ptr()),
                                   _stream(stream)))
        return out

    def distribute_pointnet(self, pos: torch.Tensor, feat: torch.Tensor | None, layers, gn=None, eps: float = 1e-5,
                            out: torch.Tensor | None = None, stream=None, dtype=torch.float32) -> torch.Tensor:
        """Distribute + PointNet; layers = [(W1, b1), (W2, b2), (W3, b3)] with
        W_i float32 [out][in] device tensors and optional biases; gn = None or
        (gamma, beta), the concatenated parameters of the three GroupNorms
        ((3 + Cf) + C1 + C2 float32 values each, either may be None).  The
        output is float32 or bfloat16 (out's dtype, else `dtype`)."""
        (W1, b1), (W2, b2), (W3, b3) = layers
        c1, c2, c3 = W1.shape[0], W2.shape[0], W3.shape[0]
        for W in (W1, W2, W3):
            if W.dtype != torch.float32 or not W.is_contiguous():
                raise ValueError("weights must be contiguous float32")
        if pos.dtype != torch.float32 or not pos.is_contiguous():
            raise ValueError("positions must be a contiguous m x d float32 tensor")
        cf = 0 if feat is None else feat.shape[1]
        gam, bet = (None, None) if gn is None else gn
        for a in (gam, bet):
            if a is not None and (a.dtype != torch.float32 or not a.is_contiguous()
                                  or a.numel() != 3 + cf + c1 + c2):
                raise ValueError("GroupNorm parameters must be contiguous float32 of (3 + Cf) + C1 + C2 values")
        fp, fld = (None, 0) if feat is None else _rows(feat)
        if out is None:
            out = torch.empty((self.n, c3), dtype=dtype, device="cuda")
        op, old = _rows(out)
        ptr = lambda t: None if t is None else C.c_void_p(t.data_ptr())
        _check(lib().lattice_distribute_pointnet(self._h, ptr(pos), fp, fld, cf, ptr(gam), ptr(bet), float(eps),
                                                 ptr(W1), ptr(b1), c1, ptr(W2), ptr(b2), c2, ptr(W3), ptr(b3), c3,
                                                 _dtype_code(out), op, old, _stream(stream)))
        return out

    # ---- backward passes (float32) ----
    def splat_backward(self, dx: torch.Tensor, normalize: bool = True, out: torch.Tensor | None = None,
                       wsum: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        """Gradient of splat(feat, normalize) with respect to feat, for
        dL/dvalues = dx (n x C); returns m x C.  wsum: the weight sums the
        forward splat returned (optional)."""
        Cc = dx.shape[1]
        if out is None:
            out = torch.empty((self.m, Cc), dtype=torch.float32, device="cuda")
        xp, xld = _rows(dx)
        _check(lib().lattice_splat_backward(self._h, xp, xld, Cc, int(bool(normalize)),
                                            None if wsum is None else C.c_void_p(wsum.data_ptr()),
                                            C.c_void_p(out.data_ptr()), _stream(stream)))
        return out

    def slice_backward(self, dout: torch.Tensor, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        """Gradient of slice(x) with respect to x, for dL/dout = dout (m x C);
        returns n x C."""
        Cc = dout.shape[1]
        if out is None:
            out = torch.empty((self.n, Cc), dtype=torch.float32, device="cuda")
        gp, gld = _rows(dout)
        op, old = _rows(out)
        _check(lib().lattice_slice_backward(self._h, gp, gld, Cc, op, old, _stream(stream)))
        return out

    def conv_backward(self, src: "Lattice", x: torch.Tensor | None, W: torch.Tensor | None, dy: torch.Tensor,
                      relu: bool = False, y: torch.Tensor | None = None, want_dx: bool = True,
                      want_dw: bool = True, want_dbias: bool = True, dx_out: torch.Tensor | None = None,
                      stream=None):
        """Gradients of the convolution self <- src (1-hop, strided, or
        Upsample when src = self.coarsen()) for dL/dY = dy: (dx, dW, dbias),
        None where not asked for.  W is taps x Cout x Cin."""
        cout = dy.shape[1]
        cin = W.shape[2] if W is not None else x.shape[1]
        dx = dx_out if dx_out is not None else (
            torch.empty((src.n, cin), dtype=torch.float32, device="cuda") if want_dx else None)
        dW = torch.empty((9, cout, cin), dtype=torch.float32, device="cuda") if want_dw else None
        db = torch.empty((cout,), dtype=torch.float32, device="cuda") if want_dbias else None
        xp, xld = _rows(x) if x is not None else (None, 0)
        yp, yld = _rows(y) if y is not None else (None, 0)
        gp, gld = _rows(dy)
        dp, dld = _rows(dx) if dx is not None else (None, 0)
        ptr = lambda t: None if t is None else C.c_void_p(t.data_ptr())
        _check(lib().lattice_conv_backward(self._h, src._h, xp, xld, cin, ptr(W), cout, LAT_RELU if relu else 0,
                                           yp, yld, gp, gld, dp, dld, ptr(dW), ptr(db), _stream(stream)))
        return dx, dW, db

    def conv_backward_bf16(self, src: "Lattice", x: torch.Tensor | None, W: torch.Tensor | None, dy: torch.Tensor,
                           relu: bool = False, y: torch.Tensor | None = None, want_dx: bool = True,
                           want_dw: bool = True, want_dbias: bool = True, stream=None):
        """conv_backward for bfloat16 x, W, y, dy: (dx bfloat16, dW and dbias
        float32), None where not asked for."""
        cout = dy.shape[1]
        cin = W.shape[2] if W is not None else x.shape[1]
        dx = torch.empty((src.n, cin), dtype=torch.bfloat16, device="cuda") if want_dx else None
        dW = torch.empty((9, cout, cin), dtype=torch.float32, device="cuda") if want_dw else None
        db = torch.empty((cout,), dtype=torch.float32, device="cuda") if want_dbias else None
        xp, xld = _rows(x) if x is not None else (None, 0)
        yp, yld = _rows(y) if y is not None else (None, 0)
        gp, gld = _rows(dy)
        dp, dld = _rows(dx) if dx is not None else (None, 0)
        ptr = lambda t: None if t is None else C.c_void_p(t.data_ptr())
        _check(lib().lattice_conv_backward_ex(self._h, src._h, xp, xld, cin, ptr(W), cout, _dtype_code(dy),
                                              LAT_RELU if relu else 0, yp, yld, gp, gld, dp, dld, ptr(dW), ptr(db),
                                              _stream(stream)))
        return dx, dW, db

    def conv_preact_backward(self, src: "Lattice", x: torch.Tensor, W: torch.Tensor, dy: torch.Tensor,
                             groups: int = 32, gamma: torch.Tensor | None = None, beta: torch.Tensor | None = None,
                             eps: float = 1e-5, relu: bool = False, y: torch.Tensor | None = None,
                             want_dx: bool = True, want_dw: bool = True, want_dbias: bool = True,
                             want_dgn: bool = True, stream=None):
        """Gradients of the pre-activated convolution self <- src
        (Y = act(conv(relu(GN(x)), W) + bias)) for dL/dY = dy:
        (dx, dW, dbias, dgamma, dbeta), None where not asked for."""
        cout, cin = dy.shape[1], x.shape[1]
        dev = dict(dtype=torch.float32, device="cuda")
        dx = torch.empty((src.n, cin), **dev) if want_dx else None
        dW = torch.empty((9, cout, cin), **dev) if want_dw else None
        db = torch.empty((cout,), **dev) if want_dbias else None
        dg = torch.empty((cin,), **dev) if want_dgn else None
        dbe = torch.empty((cin,), **dev) if want_dgn else None
        xp, xld = _rows(x)
        yp, yld = _rows(y) if y is not None else (None, 0)
        gp, gld = _rows(dy)
        dp, dld = _rows(dx) if dx is not None else (None, 0)
        ptr = lambda t: None if t is None else C.c_void_p(t.data_ptr())
        _check(lib().lattice_conv_preact_backward(self._h, src._h, xp, xld, cin, int(groups), ptr(gamma), ptr(beta),
                                                  float(eps), ptr(W), cout, LAT_RELU if relu else 0, yp, yld, gp,
                                                  gld, dp, dld, ptr(dW), ptr(db), ptr(dg), ptr(dbe),
                                                  _stream(stream)))
        return dx, dW, db, dg, dbe

    def distribute_pointnet_backward(self, pos: torch.Tensor, feat: torch.Tensor | None, layers, dx: torch.Tensor,
                                     gn=None, eps: float = 1e-5, stream=None) -> dict:
        """Gradients of distribute_pointnet(pos, feat, layers, gn, eps) for
        dL/dx = dx (n x C3): a dict with dF (m x Cf, None without features),
        dW1..dW3 ([out][in]), db1..db3, dgamma and dbeta (concatenated as
        gn)."""
        (W1, b1), (W2, b2), (W3, b3) = layers
        c1, c2, c3 = W1.shape[0], W2.shape[0], W3.shape[0]
        cf = 0 if feat is None else feat.shape[1]
        gam, bet = (None, None) if gn is None else gn
        dev = dict(dtype=torch.float32, device="cuda")
        ng = 3 + cf + c1 + c2
        out = dict(dF=torch.empty((self.m, cf), **dev) if cf else None, dW1=torch.empty_like(W1),
                   db1=torch.empty((c1,), **dev), dW2=torch.empty_like(W2), db2=torch.empty((c2,), **dev),
                   dW3=torch.empty_like(W3), db3=torch.empty((c3,), **dev), dgamma=torch.empty((ng,), **dev),
                   dbeta=torch.empty((ng,), **dev))
        fp, fld = (None, 0) if feat is None else _rows(feat)
        dfp, dfld = (None, 0) if out["dF"] is None else _rows(out["dF"])
        xp, xld = _rows(dx)
        ptr = lambda t: None if t is None else C.c_void_p(t.data_ptr())
        _check(lib().lattice_distribute_pointnet_backward(
            self._h, ptr(pos), fp, fld, cf, ptr(gam), ptr(bet), float(eps), ptr(W1), ptr(b1), c1, ptr(W2), ptr(b2),
            c2, ptr(W3), ptr(b3), c3, xp, xld, dfp, dfld, ptr(out["dW1"]), ptr(out["db1"]), ptr(out["dW2"]),
            ptr(out["db2"]), ptr(out["dW3"]), ptr(out["db3"]), ptr(out["dgamma"]), ptr(out["dbeta"]),
            _stream(stream)))
        return out

    def deform_slice_backward(self, x: torch.Tensor, wv: torch.Tensor, beta: float, dout: torch.Tensor,
                              dx_out: torch.Tensor | None = None, stream=None):
        """Gradients of deform_slice(x, wv, beta) for dL/dout = dout:
        (dx n x C, dwv C, dbeta scalar tensor)."""
        Cc = x.shape[1]
        dx = dx_out if dx_out is not None else torch.empty((self.n, Cc), dtype=torch.float32, device="cuda")
        dwv = torch.empty((Cc,), dtype=torch.float32, device="cuda")
        dbeta = torch.empty((1,), dtype=torch.float32, device="cuda")
        xp, xld = _rows(x)
        gp, gld = _rows(dout)
        dp, dld = _rows(dx)
        _check(lib().lattice_deform_slice_backward(self._h, xp, xld, Cc, C.c_void_p(wv.data_ptr()), float(beta), gp, gld,
                                                   dp, dld, C.c_void_p(dwv.data_ptr()), C.c_void_p(dbeta.data_ptr()),
                                                   _stream(stream)))
        return dx, dwv, dbeta

    def deform_slice_classify_backward(self, x: torch.Tensor, wv: torch.Tensor, beta: float, Wc: torch.Tensor,
                                       dlogits: torch.Tensor, want_dwc: bool = True, stream=None):
        """Gradients of deform_slice_classify(x, wv, beta, Wc, bc) for
        dL/dlogits = dlogits: (dx, dwv, dbeta, dWc, dbc), dWc and dbc None
        unless asked for."""
        Cc, K = x.shape[1], Wc.shape[0]
        dev = dict(dtype=torch.float32, device="cuda")
        dx = torch.empty((self.n, Cc), **dev)
        dwv = torch.empty((Cc,), **dev)
        dbeta = torch.empty((1,), **dev)
        dWc = torch.empty((K, Cc), **dev) if want_dwc else None
        dbc = torch.empty((K,), **dev) if want_dwc else None
        xp, xld = _rows(x)
        zp, zld = _rows(dlogits)
        dp, dld = _rows(dx)
        ptr = lambda t: None if t is None else C.c_void_p(t.data_ptr())
        _check(lib().lattice_deform_slice_classify_backward(self._h, xp, xld, Cc, ptr(wv), float(beta), ptr(Wc), K,
                                                            zp, zld, dp, dld, ptr(dwv), ptr(dbeta), ptr(dWc),
                                                            ptr(dbc), _stream(stream)))
        return dx, dwv, dbeta, dWc, dbc

    def deform_slice_classify(self, x: torch.Tensor, wv: torch.Tensor, beta: float, Wc: torch.Tensor,
                              bc: torch.Tensor | None = None, out: torch.Tensor | None = None,
                              stream=None) -> torch.Tensor:
        """DeformSlice fused with the classifier: m x K logits, Wc K x C."""
        K, Cc = Wc.shape[0], x.shape[1]
        if Wc.dtype != torch.float32 or not Wc.is_contiguous() or Wc.shape[1] != Cc:
            raise ValueError("Wc must be a contiguous K x C float32 tensor")
        if out is None:
            out = torch.empty((self.m, K), dtype=torch.float32, device="cuda")
        xp, xld = _rows(x)
        _check(lib().lattice_deform_slice_classify(self._h, xp, xld, Cc, _dtype_code(x), C.c_void_p(wv.data_ptr()),
                                                   float(beta), C.c_void_p(Wc.data_ptr()),
                                                   None if bc is None else C.c_void_p(bc.data_ptr()), K,
                                                   C.c_void_p(out.data_ptr()), _stream(stream)))
        return out

    def deform_slice(self, x: torch.Tensor, wv: torch.Tensor, beta: float,
                     out: torch.Tensor | None = None, delta: torch.Tensor | None = None,
                     stream=None) -> torch.Tensor:
        Cc = x.shape[1]
        if out is None:
            out = torch.empty((self.m, Cc), dtype=torch.float32, device="cuda")
        xp, xld = _rows(x)
        _check(lib().lattice_deform_slice(self._h, xp, xld, Cc, _dtype_code(x),
                                          C.c_void_p(wv.data_ptr()), float(beta),
                                          C.c_void_p(out.data_ptr()),
                                          None if delta is None else C.c_void_p(delta.data_ptr()),
                                          _stream(stream)))
        return out

    def slice_and_deform(self, x: torch.Tensor, wv: torch.Tensor, beta: float, slice_out: torch.Tensor | None = None,
                         deform_out: torch.Tensor | None = None, stream=None):
        """(slice(x), deform_slice(x, wv, beta)) from one pass over the
        gathered rows."""
        Cc = x.shape[1]
        if slice_out is None:
            slice_out = torch.empty((self.m, Cc), dtype=torch.float32, device="cuda")
        if deform_out is None:
            deform_out = torch.empty((self.m, Cc), dtype=torch.float32, device="cuda")
        xp, xld = _rows(x)
        _check(lib().lattice_slice_and_deform(self._h, xp, xld, Cc, _dtype_code(x), C.c_void_p(wv.data_ptr()),
                                              float(beta), C.c_void_p(slice_out.data_ptr()),
                                              C.c_void_p(deform_out.data_ptr()), _stream(stream)))
        return slice_out, deform_out
