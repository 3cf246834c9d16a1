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

from .lattice import Lattice


class GpuPipeline:
    def __init__(self, wl):
        self.wl = wl
        self.dtype = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
        self.pos = torch.from_numpy(np.ascontiguousarray(wl.positions)).cuda()
        self.feat = torch.from_numpy(np.ascontiguousarray(wl.features)).cuda().to(self.dtype)
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

    def _view(self, bufs, levels, spec):
        name, c0, cc = spec
        if name not in bufs:
            lv, total = self.wl.buffers[name]
            n = levels[lv].n
            # device buffers are kept across steps (same stream, so a step's
            # kernels finish with a buffer before the next step's reuse it)
            store = self._store.get(name)
            if store is None or store.shape[0] < n:
                store = torch.empty((n, total), dtype=self.dtype, device="cuda")
                self._store[name] = store
            bufs[name] = store[:n]
        return bufs[name][:, c0:c0 + cc]

    def step(self, keep=False):
        """One pass of the pipeline.  Returns (levels, buffers, point outputs).

        The lattice hierarchy (create, coarsen) is issued first: a coarse
        level depends only on the positions, and issuing every build before
        the feature operations keeps the device busy while the host waits
        for vertex counts.  With keep=True the buffers are fresh tensors
        that later steps do not overwrite."""
        levels: dict[int, Lattice] = {}
        bufs: dict[str, torch.Tensor] = {}
        outs: dict[str, torch.Tensor] = {}
        if keep:
            self._store = {}
        for op in self.wl.ops:
            if op["op"] == "create":
                levels[0] = Lattice.create(self.pos, self.sigma)
            elif op["op"] == "coarsen":
                levels[op["level"]] = levels[op["level"] - 1].coarsen()
        for op in self.wl.ops:
            kind = op["op"]
            if kind in ("create", "coarsen"):
                continue
            elif kind == "splat":
                # the weight sums are kept for a backward pass
                if self._wsum is None or self._wsum.shape[0] < levels[0].n:
                    self._wsum = torch.empty(levels[0].n, dtype=torch.float32, device="cuda")
                levels[0].splat(self.feat, normalize=bool(op["normalize"]),
                                out=self._view(bufs, levels, op["dst"]), wsum=self._wsum[:levels[0].n])
            elif kind in ("conv", "conv_down", "refine"):
                lv = op["level"]
                x = self._view(bufs, levels, op["src"])
                y = self._view(bufs, levels, op["dst"])
                W = self.weights[op["w"]]
                if "pre" in op:
                    gam, bet = self.norms[op["pre"]["norm"]]
                    src = levels[{"conv": lv, "conv_down": lv - 1, "refine": lv + 1}[kind]]
                    res = self._view(bufs, levels, op["res"]) if "res" in op else None
                    levels[lv].conv_preact(src, x, W, groups=op["pre"]["groups"], gamma=gam, beta=bet,
                                           relu=op["relu"], out=y, refine=kind == "refine", res=res)
                elif kind == "conv":
                    levels[lv].conv(levels[lv], x, W, relu=op["relu"], out=y)
                elif kind == "conv_down":
                    levels[lv].conv(levels[lv - 1], x, W, relu=op["relu"], out=y)
                else:
                    levels[lv].refine(levels[lv + 1], x, W, relu=op["relu"], out=y)
            elif kind == "distribute":
                levels[op["level"]].distribute_pointnet(self.pos, self.feat, [self.mlp[n] for n in op["layers"]],
                                                        out=self._view(bufs, levels, op["dst"]))
            elif kind == "slice":
                outs[op["out"]] = levels[op["level"]].slice(self._view(bufs, levels, op["src"]))
            elif kind == "deform_slice":
                wv, beta = self.vectors[op["wv"]]
                outs[op["out"]] = levels[op["level"]].deform_slice(
                    self._view(bufs, levels, op["src"]), wv, beta)
            elif kind == "deform_classify":
                wv, beta = self.vectors[op["wv"]]
                Wc, bc = self.classifiers[op["cls"]]
                outs[op["out"]] = levels[op["level"]].deform_slice_classify(
                    self._view(bufs, levels, op["src"]), wv, beta, Wc, bc)
            elif kind == "deform_slice_bwd":
                wv, beta = self.vectors[op["wv"]]
                _, dwv, dbeta = levels[op["level"]].deform_slice_backward(
                    self._view(bufs, levels, op["x"]), wv, beta, self.grads[op["grad"]],
                    dx_out=self._view(bufs, levels, op["dst"]))
                outs[op["out"]], outs["dbeta:" + op["wv"]] = dwv, dbeta
            elif kind == "conv_bwd":
                lv = op["level"]
                dst = levels[lv]
                src = {"conv": lv, "conv_down": lv - 1, "refine": lv + 1}[op["kind"]]
                _, dW, db = dst.conv_backward(levels[src], self._view(bufs, levels, op["x"]), self.weights[op["w"]],
                                              self._view(bufs, levels, op["src"]), relu=op["relu"],
                                              y=self._view(bufs, levels, op["y"]) if op["relu"] else None,
                                              dx_out=self._view(bufs, levels, op["dst"]))
                outs[op["out"]] = dW.transpose(1, 2)          # taps x Cin x Cout, the workload's layout
                outs["db:" + op["w"]] = db
            elif kind == "splat_bwd":
                outs[op["out"]] = levels[0].splat_backward(self._view(bufs, levels, op["src"]),
                                                           normalize=bool(op["normalize"]),
                                                           wsum=self._wsum[:levels[0].n])
            else:
                raise ValueError(f"unknown op {kind}")
        if keep:
            self._store = {}
        return levels, bufs, outs

    @staticmethod
    def release(levels):
        """Destroy lattices finest-last (children before parents)."""
        for lv in sorted(levels, reverse=True):
            levels[lv].destroy()
