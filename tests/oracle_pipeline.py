"""Run a workload's pipeline on the CPU oracle (test infrastructure).

Mirrors the operation list of workloads.configs with the oracle's functions:
float64 buffers, and in bf16 workloads every stored activation is rounded to
bfloat16 where the GPU stores bf16 (splat, convolution outputs).
"""
from __future__ import annotations

import time

import numpy as np

from oracle import oracle as O


class OraclePipeline:
    def __init__(self, wl):
        self.wl = wl
        self.bf16 = wl.dtype == "bf16"

    def _store(self, x):
        return O.round_bf16(x) if self.bf16 else x

    def run(self, stop_after=None, times=None):
        """The whole operation list; `times`, if given, accumulates the
        seconds spent per operation kind."""
        wl = self.wl
        levels, bufs, outs = {}, {}, {}

        def view_src(spec):
            name, c0, cc = spec
            return bufs[name][:, c0:c0 + cc]

        def write(spec, val):
            name, c0, cc = spec
            if name not in bufs:
                lv, total = wl.buffers[name]
                bufs[name] = np.zeros((levels[lv].n, total))
            bufs[name][:, c0:c0 + cc] = self._store(val)

        for i, op in enumerate(wl.ops):
            kind = op["op"]
            t_op = time.perf_counter()
            if kind == "create":
                levels[0] = O.Lattice.create(wl.positions, wl.sigma)
            elif kind == "coarsen":
                levels[op["level"]] = levels[op["level"] - 1].coarsen()
            elif kind == "splat":
                X, _ = levels[0].splat(wl.features.astype(np.float64), normalize=bool(op["normalize"]))
                write(op["dst"], X)
            elif kind in ("conv", "conv_down", "refine"):
                lv = op["level"]
                x = np.ascontiguousarray(view_src(op["src"]))
                W = wl.weights[op["w"]].astype(np.float64)
                if "pre" in op:
                    gam, bet = wl.norms[op["pre"]["norm"]]
                    x = O.groupnorm(x, op["pre"]["groups"], gam.astype(np.float64), bet.astype(np.float64),
                                    eps=1e-5, relu=True)
                    if self.bf16:
                        x = O.round_bf16(x)
                if kind == "conv":
                    y = levels[lv].conv(levels[lv], x, W, relu=op["relu"])
                elif kind == "conv_down":
                    y = levels[lv].conv(levels[lv - 1], x, W, relu=op["relu"])
                else:
                    y = levels[lv].refine_into(levels[lv + 1], x, W, relu=op["relu"])
                if "res" in op:
                    y = y + view_src(op["res"])
                write(op["dst"], y)
            elif kind == "distribute":
                layers = [tuple(a.astype(np.float64) for a in wl.mlp[n]) for n in op["layers"]]
                gn = tuple(a.astype(np.float64) for a in wl.norms[op["norm"]])
                write(op["dst"], levels[op["level"]].distribute_pointnet(
                    wl.positions.astype(np.float64), wl.features.astype(np.float64), layers, gn))
            elif kind == "slice":
                outs[op["out"]] = levels[op["level"]].slice(np.ascontiguousarray(view_src(op["src"])))
            elif kind == "deform_slice":
                wv, beta = wl.vectors[op["wv"]]
                outs[op["out"]], _ = levels[op["level"]].deform_slice(
                    np.ascontiguousarray(view_src(op["src"])), wv.astype(np.float64), beta)
            elif kind == "deform_classify":
                wv, beta = wl.vectors[op["wv"]]
                Wc, bc = wl.classifiers[op["cls"]]
                outs[op["out"]] = levels[op["level"]].deform_slice_classify(
                    np.ascontiguousarray(view_src(op["src"])), wv.astype(np.float64), beta, Wc.astype(np.float64),
                    bc.astype(np.float64))
            elif kind == "deform_slice_bwd":
                wv, beta = wl.vectors[op["wv"]]
                dx, dwv, dbeta = levels[op["level"]].deform_slice_backward(
                    np.ascontiguousarray(view_src(op["x"])), wv.astype(np.float64), beta,
                    wl.grads[op["grad"]].astype(np.float64))
                write(op["dst"], dx)
                outs[op["out"]], outs["dbeta:" + op["wv"]] = dwv, np.array([dbeta])
            elif kind == "conv_bwd":
                lv = op["level"]
                src = {"conv": lv, "conv_down": lv - 1, "refine": lv + 1}[op["kind"]]
                dx, dW, db = levels[lv].conv_backward(
                    levels[src], np.ascontiguousarray(view_src(op["x"])), wl.weights[op["w"]].astype(np.float64),
                    np.ascontiguousarray(view_src(op["src"])), relu=op["relu"],
                    Y=np.ascontiguousarray(view_src(op["y"])) if op["relu"] else None)
                write(op["dst"], dx)
                outs[op["out"]], outs["db:" + op["w"]] = dW, db
            elif kind == "splat_bwd":
                outs[op["out"]] = levels[0].splat_backward(np.ascontiguousarray(view_src(op["src"])),
                                                           normalize=bool(op["normalize"]))
            if times is not None:
                times[kind] = times.get(kind, 0.0) + time.perf_counter() - t_op
            if stop_after is not None and i == stop_after:
                break
        return levels, bufs, outs
