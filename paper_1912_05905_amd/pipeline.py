"""Run a workload's lattice pipeline on the GPU through liblattice.

A workload (see workloads.configs) lists lattice operations; this runner
executes them in order: lattices are created / coarsened per step, values
live in device buffers (row-major, vertices of their level x channels), and
each operation reads / writes a column range of a buffer, which gives channel
concatenation without copies.  All arithmetic happens in the library's
kernels; torch only allocates the buffers.
"""
from __future__ import annotations

import numpy as np
import torch

from . import lattice as _lat
from .lattice import Lattice


class _Buffers(dict):
    """name -> the n x total buffer of a step, sliced from its store when
    first read (the forward operators pass raw pointers instead)."""

    def __init__(self, stores, rows):
        super().__init__()
        self._stores, self._rows = stores, rows

    def __missing__(self, name):
        v = self._stores[name][:self._rows[name]]
        self[name] = v
        return v

    def __contains__(self, name):
        return name in self._rows


class GpuPipeline:
    """overlap=True builds the lattices on a stream of their own and one
    cloud ahead: a step issues the next cloud's hierarchy, then runs this
    cloud's operators on the hierarchy the previous step issued, so the next
    cloud's lattice construction runs while this cloud's operators execute
    (steps are independent; every step builds one hierarchy and runs one
    pass of operators).  A step's lattices are destroyed by finish_step() one
    step later, once the build stream is ordered after the step's operators;
    flush() releases what is still held, the hierarchy built ahead
    included.  Several pipelines (each with its own buffers, and a build
    stream of its own or one they share, given as build_stream) may take
    steps in turn on compute streams of their own, so that consecutive
    clouds' operators overlap as well."""

    def __init__(self, wl, overlap=False, hierarchy=True, build_stream=None):
        self.wl = wl
        self.overlap = overlap
        # levels 0..L-1 created by one library call when the workload's
        # builds are a create followed by coarsenings level by level
        kinds = [(op["op"], op.get("level")) for op in wl.ops if op["op"] in ("create", "coarsen")]
        chain = [("create", 0)] + [("coarsen", l) for l in range(1, len(kinds))]
        self._levels = len(kinds) if hierarchy and kinds == chain else 0
        if overlap:
            self._build_stream = build_stream if build_stream is not None else torch.cuda.Stream()
        else:
            self._build_stream = None
        self._pending: list = []      # (levels, operators-done event) of finished steps
        self._ahead = None            # (levels, built event) of the next cloud
        self._events = [torch.cuda.Event() for _ in range(8)] if overlap else []
        self._next_event = 0
        self._cur = None                    # the caller's stream of the last step
        self._cur_raw = None                # its raw handle
        self.dtype = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
        self.pos = torch.from_numpy(np.ascontiguousarray(wl.positions)).cuda()
        self.feat = torch.from_numpy(np.ascontiguousarray(wl.features)).cuda().to(self.dtype)
        # Distribute reads float32 features (a bf16 workload's are bf16 values)
        self.feat32 = torch.from_numpy(np.ascontiguousarray(wl.features, dtype=np.float32)).cuda()
        # library weight layout: taps x Cout x Cin
        self.weights = {k: torch.from_numpy(np.ascontiguousarray(np.transpose(w, (0, 2, 1))))
                        .cuda().to(self.dtype).contiguous() for k, w in wl.weights.items()}
        self.vectors = {k: (torch.from_numpy(np.ascontiguousarray(v)).cuda(), float(beta))
                        for k, (v, beta) in wl.vectors.items()}
        self.mlp = {k: (torch.from_numpy(np.ascontiguousarray(W, dtype=np.float32)).cuda(),
                        torch.from_numpy(np.ascontiguousarray(b, dtype=np.float32)).cuda())
                    for k, (W, b) in wl.mlp.items()}
        self.grads = {k: torch.from_numpy(np.ascontiguousarray(g)).cuda() for k, g in wl.grads.items()}
        self.norms = {k: (torch.from_numpy(np.ascontiguousarray(g)).cuda(), torch.from_numpy(np.ascontiguousarray(b))
                          .cuda()) for k, (g, b) in wl.norms.items()}
        self.classifiers = {k: (torch.from_numpy(np.ascontiguousarray(W, dtype=np.float32)).cuda(),
                                torch.from_numpy(np.ascontiguousarray(b, dtype=np.float32)).cuda())
                            for k, (W, b) in wl.classifiers.items()}
        self.sigma = [float(s) for s in wl.sigma]
        self._store: dict[str, torch.Tensor] = {}
        self._wsum: torch.Tensor | None = None
        # static arguments of the forward operators, converted once
        self._lib = _lat.lib()
        self._esize = 2 if self.dtype == torch.bfloat16 else 4
        self._dt = _lat.LAT_BF16 if self.dtype == torch.bfloat16 else _lat.LAT_F32
        self._wptr = {k: (w.data_ptr(), w.shape[1], w.shape[2]) for k, w in self.weights.items()}
        self._outs: dict[str, torch.Tensor] = {}
        # a slice followed by a DeformSlice of the same values runs as one pass
        ops = wl.ops
        self._fused = {i for i in range(len(ops) - 1)
                       if ops[i]["op"] == "slice" and ops[i + 1]["op"] == "deform_slice"
                       and ops[i]["level"] == ops[i + 1]["level"] and ops[i]["src"] == ops[i + 1]["src"]}

    def _out(self, name, rows, cols, keep):
        """Point output buffer (float32), kept across steps unless keep."""
        t = None if keep else self._outs.get(name)
        if t is None or t.shape != (rows, cols):
            t = torch.empty((rows, cols), dtype=torch.float32, device="cuda")
            if not keep:
                self._outs[name] = t
        return t

    def _grad(self, name, shape, keep):
        """Gradient output buffer (float32), kept across steps unless keep."""
        t = None if keep else self._outs.get(name)
        if t is None or tuple(t.shape) != tuple(shape):
            t = torch.empty(shape, dtype=torch.float32, device="cuda")
            if not keep:
                self._outs[name] = t
        return t

    def step(self, keep=False, after_op=None):
        """One pass of the pipeline.  Returns (levels, buffers, point outputs).

        The lattice hierarchy (create, coarsen) is issued first: a coarse
        level depends only on the positions, and issuing every build before
        the feature operations keeps the device busy while the host waits
        for vertex counts.  With keep=True the buffers are fresh tensors
        that later steps do not overwrite.  Forward operators are called
        with raw pointers into the buffers (column ranges by offset), which
        keeps the host's cost per operator near the library call itself.
        after_op(i, op, levels, buffers, outputs), if given, is called once
        each operation i has been enqueued (for checks of every operator on
        the inputs it saw)."""
        wl, lib, es, dt = self.wl, self._lib, self._esize, self._dt
        levels: dict[int, Lattice] = {}
        rows: dict[str, int] = {}
        base: dict[str, tuple] = {}
        outs: dict[str, torch.Tensor] = {}
        if keep:
            self._store = {}
        stream = _lat._stream()

        def check(status):
            if status != 0:
                _lat._check(status)

        def ptr(spec):
            name, c0, _ = spec
            b = base.get(name)
            if b is None:
                lv, total = wl.buffers[name]
                n = levels[lv].n
                store = self._store.get(name)
                if store is None or store.shape[0] < n:
                    store = torch.empty((n, total), dtype=self.dtype, device="cuda")
                    self._store[name] = store
                rows[name] = n
                b = base[name] = (store.data_ptr(), total)
            return b[0] + c0 * es, b[1]

        def build(into, bstream=None):
            if self._levels:
                for lv, L in enumerate(Lattice.create_hierarchy(self.pos, self.sigma, self._levels,
                                                                stream=bstream)):
                    into[lv] = L
                return
            for op in wl.ops:
                if op["op"] == "create":
                    into[0] = Lattice.create(self.pos, self.sigma, stream=bstream)
                elif op["op"] == "coarsen":
                    # on a build stream of its own the hierarchy is already off
                    # the operators' stream: no side stream needed
                    into[op["level"]] = into[op["level"] - 1].coarsen(stream=bstream,
                                                                      on_stream=bstream is not None)

        if self.overlap and not keep:
            # Builds run one cloud ahead: this step issues the next cloud's
            # hierarchy on the build stream, then this cloud's operators on
            # the caller's stream, on the hierarchy issued a step earlier.
            # The next build then runs under this cloud's operators, and the
            # vertex counts the operators need are normally home already.
            bs = self._build_stream
            ahead = self._ahead
            if ahead is None:
                first: dict[int, Lattice] = {}
                build(first, bs)
                ev = self._event()
                ev.record(bs)
                ahead = (first, ev)
            # destroy the lattices of all but the last finished step; their
            # buffers return to the build stream's pool once that stream has
            # passed the step's operators
            while len(self._pending) > 1:
                old, done = self._pending.pop(0)
                bs.wait_event(done)
                GpuPipeline.release(old)
            nxt: dict[int, Lattice] = {}
            build(nxt, bs)
            ev = self._event()
            ev.record(bs)
            self._ahead = (nxt, ev)
            levels.update(ahead[0])
            self._cur = self._current_stream()
            self._cur.wait_event(ahead[1])
        else:
            build(levels)

        skip = False
        for i, op in enumerate(wl.ops):
            kind = op["op"]
            if skip:
                skip = False
                continue
            if kind in ("create", "coarsen"):
                continue
            if i in self._fused:
                dop = wl.ops[i + 1]
                L = levels[op["level"]]
                wv, beta = self.vectors[dop["wv"]]
                xp, xld = ptr(op["src"])
                cc = op["src"][2]
                out = outs[op["out"]] = self._out(op["out"], L.m, cc, keep)
                dout = outs[dop["out"]] = self._out(dop["out"], L.m, cc, keep)
                check(lib.lattice_slice_and_deform(L._h, xp, xld, cc, dt, wv.data_ptr(), beta, out.data_ptr(),
                                                   dout.data_ptr(), stream))
                skip = True
                if after_op is not None:
                    after_op(i, op, levels, _Buffers(self._store, rows), outs)
                    after_op(i + 1, dop, levels, _Buffers(self._store, rows), outs)
                continue
            elif kind == "splat":
                L0 = levels[0]
                # the weight sums are kept for a backward pass
                if self._wsum is None or self._wsum.shape[0] < L0.n:
                    self._wsum = torch.empty(L0.n, dtype=torch.float32, device="cuda")
                op_, old = ptr(op["dst"])
                check(lib.lattice_splat(L0._h, self.feat.data_ptr(), self.feat.stride(0), self.feat.shape[1], dt,
                                        int(bool(op["normalize"])), op_, old, self._wsum.data_ptr(), stream))
            elif kind in ("conv", "conv_down", "refine"):
                lv = op["level"]
                xp, xld = ptr(op["src"])
                yp, yld = ptr(op["dst"])
                wp, cout, cin = self._wptr[op["w"]]
                flags = _lat.LAT_RELU if op["relu"] else 0
                dst = levels[lv]
                src = levels[{"conv": lv, "conv_down": lv - 1, "refine": lv + 1}[kind]]
                if "pre" in op:
                    gam, bet = self.norms[op["pre"]["norm"]]
                    args = (dst._h, src._h, xp, xld, cin, int(op["pre"]["groups"]), gam.data_ptr(), bet.data_ptr(),
                            1e-5, wp, None, cout, dt, flags)
                    if kind == "refine":
                        check(lib.lattice_refine_preact(*args, yp, yld, stream))
                    else:
                        rp, rld = ptr(op["res"]) if "res" in op else (None, 0)
                        check(lib.lattice_conv_preact(*args, rp, rld, yp, yld, stream))
                elif kind == "refine":
                    check(lib.lattice_refine(dst._h, src._h, xp, xld, cin, wp, None, cout, dt, flags, yp, yld, stream))
                else:
                    check(lib.lattice_conv(dst._h, src._h, xp, xld, cin, wp, None, cout, dt, flags, yp, yld, stream))
            elif kind == "distribute":
                yp, yld = ptr(op["dst"])
                layers = [self.mlp[n] for n in op["layers"]]
                (W1, b1), (W2, b2), (W3, b3) = layers
                gam, bet = self.norms[op["norm"]]
                check(lib.lattice_distribute_pointnet(
                    levels[op["level"]]._h, self.pos.data_ptr(), self.feat32.data_ptr(), self.feat32.stride(0),
                    self.feat32.shape[1], gam.data_ptr(), bet.data_ptr(), 1e-5, W1.data_ptr(), b1.data_ptr(),
                    W1.shape[0], W2.data_ptr(), b2.data_ptr(), W2.shape[0], W3.data_ptr(), b3.data_ptr(),
                    W3.shape[0], dt, yp, yld, stream))
            elif kind == "slice":
                L = levels[op["level"]]
                xp, xld = ptr(op["src"])
                cc = op["src"][2]
                out = outs[op["out"]] = self._out(op["out"], L.m, cc, keep)
                check(lib.lattice_slice(L._h, xp, xld, cc, dt, out.data_ptr(), stream))
            elif kind == "deform_slice":
                L = levels[op["level"]]
                wv, beta = self.vectors[op["wv"]]
                xp, xld = ptr(op["src"])
                cc = op["src"][2]
                out = outs[op["out"]] = self._out(op["out"], L.m, cc, keep)
                check(lib.lattice_deform_slice(L._h, xp, xld, cc, dt, wv.data_ptr(), beta, out.data_ptr(), None,
                                               stream))
            elif kind == "deform_classify":
                L = levels[op["level"]]
                wv, beta = self.vectors[op["wv"]]
                Wc, bc = self.classifiers[op["cls"]]
                xp, xld = ptr(op["src"])
                cc = op["src"][2]
                out = outs[op["out"]] = self._out(op["out"], L.m, Wc.shape[0], keep)
                check(lib.lattice_deform_slice_classify(L._h, xp, xld, cc, dt, wv.data_ptr(), beta, Wc.data_ptr(),
                                                        bc.data_ptr(), Wc.shape[0], out.data_ptr(), stream))
            elif kind == "conv_bwd":
                lv = op["level"]
                dst = levels[lv]
                src = levels[{"conv": lv, "conv_down": lv - 1, "refine": lv + 1}[op["kind"]]]
                xp, xld = ptr(op["x"])
                gp, gld = ptr(op["src"])
                dp, dld = ptr(op["dst"])
                yp, yld = ptr(op["y"]) if op["relu"] else (None, 0)
                wp, cout, cin = self._wptr[op["w"]]
                dW = self._grad(op["out"], (9, cout, cin), keep)
                db = self._grad("db:" + op["w"], (cout,), keep)
                check(lib.lattice_conv_backward(dst._h, src._h, xp, xld, cin, wp, cout,
                                                _lat.LAT_RELU if op["relu"] else 0, yp, yld, gp, gld, dp, dld,
                                                dW.data_ptr(), db.data_ptr(), stream))
                outs[op["out"]] = dW.transpose(1, 2)          # taps x Cin x Cout, the workload's layout
                outs["db:" + op["w"]] = db
            elif kind == "deform_slice_bwd":
                L = levels[op["level"]]
                wv, beta = self.vectors[op["wv"]]
                xp, xld = ptr(op["x"])
                dp, dld = ptr(op["dst"])
                cc = op["x"][2]
                g = self.grads[op["grad"]]
                dwv = self._grad(op["out"], (cc,), keep)
                dbeta = self._grad("dbeta:" + op["wv"], (1,), keep)
                check(lib.lattice_deform_slice_backward(L._h, xp, xld, cc, wv.data_ptr(), beta, g.data_ptr(),
                                                        g.stride(0), dp, dld, dwv.data_ptr(), dbeta.data_ptr(),
                                                        stream))
                outs[op["out"]], outs["dbeta:" + op["wv"]] = dwv, dbeta
            elif kind == "splat_bwd":
                L0 = levels[0]
                gp, gld = ptr(op["src"])
                cc = op["src"][2]
                out = self._grad(op["out"], (L0.m, cc), keep)
                check(lib.lattice_splat_backward(L0._h, gp, gld, cc, int(bool(op["normalize"])),
                                                 self._wsum.data_ptr(), out.data_ptr(), stream))
                outs[op["out"]] = out
            else:
                raise ValueError(f"unknown op {kind}")
            if after_op is not None:
                after_op(i, op, levels, _Buffers(self._store, rows), outs)
        stores = self._store
        if keep:
            self._store = {}
        return levels, _Buffers(stores, rows), outs

    def finish_step(self, levels):
        """Release a step's lattices: at once, or (overlap) after the next
        step's build has been ordered behind this step's operators."""
        if not self.overlap:
            GpuPipeline.release(levels)
            return
        done = self._event()
        done.record(self._cur)
        self._pending.append((levels, done))

    def _current_stream(self):
        """The current stream as a torch Stream, rebuilt only when the raw
        handle changed (torch.cuda.current_stream() costs microseconds)."""
        raw = _lat._stream().value
        if self._cur is None or self._cur_raw != raw:
            self._cur = torch.cuda.current_stream()
            self._cur_raw = raw
        return self._cur

    def _event(self):
        # a ring of events: a re-record does not affect waits already enqueued,
        # and at most two steps are pending
        e = self._events[self._next_event]
        self._next_event = (self._next_event + 1) % len(self._events)
        return e

    def flush(self):
        """Release every lattice still held (overlap mode)."""
        torch.cuda.synchronize()
        for old, _ in self._pending:
            GpuPipeline.release(old)
        self._pending = []
        if self._ahead is not None:
            GpuPipeline.release(self._ahead[0])
            self._ahead = None

    @staticmethod
    def release(levels):
        """Destroy lattices finest-last (children before parents)."""
        for lv in sorted(levels, reverse=True):
            levels[lv].destroy()
