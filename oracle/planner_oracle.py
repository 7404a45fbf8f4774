"""Test infrastructure: a plain reference planner for PartIR:Core propagation.

Only tests may import this module.  It restates, in the paper's order and
vocabulary, what a schedule of ManualPartition tactics does (Sec. 3): each
tactic value-tiles some inputs along a mesh axis (Sec. 5.1, `tile<%v, dim,
axis>`) and then propagates (Sec. 5.2.2) with the tile-mapping registry
(Sec. 5.2.1) until nothing changes:

  * forward propagation -- a TMR entry whose required operand tilings are
    all present (the operands come out of #tile loops or value tiling);
  * backward propagation -- an entry whose result action #tile<d> matches a
    downstream use of the result sliced along d;
  * inference -- only when nothing matches fully: a single entry that matches
    some operands while the others carry no tiling on the axis;
  * conflicts -- two or more candidates: reported, nothing rewritten;
  * an operation is never wrapped twice in loops over the same axis.

``evaluate`` then runs a partitioned program with the loop semantics of App. C
(slice = r-th contiguous chunk, #tile = concatenation, #sum = summation), so
a planner's output can be checked against the unpartitioned program, which
it must equal (value tiling and propagation preserve semantics, Sec. 5).
"""
from __future__ import annotations

import numpy as np

from . import partir_oracle as O

SUM = "sum"

# TMR (Sec. 5.2.1): (operand tiling dims, None = unsliced) -> result action
TMR = {
    "matmul": [((0, None), 0), ((None, 1), 1), ((1, 0), SUM)],
    "add": [((0, 0), 0), ((1, 1), 1)],
    "gelu": [((0,), 0), ((1,), 1)],
    "rmsnorm": [((0,), 0)],
}
ARITY = {"matmul": 2, "add": 2, "gelu": 1, "rmsnorm": 1}


class PlanError(ValueError):
    def __init__(self, status, msg):
        super().__init__(f"{status}: {msg}")
        self.status = status


def parse_program(text):
    """-> (axes [(name, size)], shapes {name: (r, c)}, ops [(out, kind, [ins])], args [names])."""
    axes, shapes, ops, args = [], {}, [], []
    for raw in text.replace(";", "\n").splitlines():
        line = raw.split("#")[0].split()
        if not line:
            continue
        if line[0] == "mesh":
            for item in line[1:]:
                name, size = item.split("=")
                axes.append((name, int(size)))
        elif line[0] == "arg":
            r, c = (int(v) for v in line[2].split("x"))
            shapes[line[1]] = (r, c)
            args.append(line[1])
        elif line[0] == "ret":
            pass
        else:
            out, eq, kind, *ins = line
            if eq != "=" or kind not in ARITY or len(ins) != ARITY[kind]:
                raise PlanError("PARTIR_E_SHAPE", f"cannot parse {raw!r}")
            a = shapes[ins[0]]
            if kind == "matmul":
                b = shapes[ins[1]]
                if a[1] != b[0]:
                    raise PlanError("PARTIR_E_SHAPE", f"matmul {a} . {b}")
                shapes[out] = (a[0], b[1])
            else:
                shapes[out] = a
            ops.append((out, kind, list(ins)))
    return axes, shapes, ops, args


class State:
    """Per-axis partitioning facts of a program."""

    def __init__(self, text):
        self.axes, self.shapes, self.ops, self.args = parse_program(text)
        self.size = dict(self.axes)
        self.tiled = {}      # (value, axis) -> dim: the value is available tiled
        self.sliced = {}     # (value, axis) -> dim: value tiling = a sliced use
        self.nest = {out: [] for out, _, _ in self.ops}      # out -> [(axis, action)], outer first
        self.cuts = {}       # (out, operand index, axis) -> dim
        self.conflicts = set()
        self.log = []

    def action_of(self, out, axis):
        for a, act in self.nest[out]:
            if a == axis:
                return act
        return None

    def parts(self, value, dim, axis, cuts):
        """How many chunks dim `dim` of `value` is split into if `axis` joins
        the axes in `cuts` that split it (TSlice needs exact division)."""
        n = self.size[axis]
        for a, d in cuts.items():
            if a != axis and d == dim:
                n *= self.size[a]
        return n

    def entry_fits(self, out, kind, ins, axis, entry):
        dims, res = entry
        for i, d in enumerate(dims):
            if d is None:
                continue
            cuts = {a: dd for (o, ii, a), dd in self.cuts.items() if o == out and ii == i}
            if self.shapes[ins[i]][d] % self.parts(ins[i], d, axis, cuts):
                return False
        if res != SUM:
            cuts = {a: d for (v, a), d in self.tiled.items() if v == out}
            if self.shapes[out][res] % self.parts(out, res, axis, cuts):
                return False
        return True

    def downstream_slices(self, value, axis):
        dims = set()
        if (value, axis) in self.sliced:
            dims.add(self.sliced[(value, axis)])
        for out, _, ins in self.ops:
            if self.action_of(out, axis) is None:
                continue
            for i, v in enumerate(ins):
                if v == value and (out, i, axis) in self.cuts:
                    dims.add(self.cuts[(out, i, axis)])
        return dims

    def rewrite(self, out, ins, axis, entry, why):
        dims, res = entry
        self.nest[out].append((axis, res))
        for i, d in enumerate(dims):
            if d is not None:
                self.cuts[(out, i, axis)] = d
        if res != SUM:
            self.tiled.setdefault((out, axis), res)
        self.log.append(f"rewrite {out} {axis} {'#sum' if res == SUM else f'#tile<{res}>'} ({why})")

    def try_op(self, out, kind, ins, axis):
        if self.action_of(out, axis) is not None or (out, axis) in self.conflicts:
            return False
        entries = TMR[kind]
        have = [self.tiled.get((v, axis)) for v in ins]
        forward = [e for e in entries
                   if any(d is not None for d in e[0])
                   and all(d is None or have[i] == d for i, d in enumerate(e[0]))]
        uses = self.downstream_slices(out, axis)
        backward = [e for e in entries if e[1] != SUM and e[1] in uses]
        found = forward + [e for e in backward if e not in forward]
        found = [e for e in found if self.entry_fits(out, kind, ins, axis, e)]
        if len(found) == 1:
            self.rewrite(out, ins, axis, found[0], "forward" if found[0] in forward else "backward")
            return True
        if len(found) > 1:
            self.conflicts.add((out, axis))
            self.log.append(f"conflict {out} {axis} {len(found)} entries match")
            return False
        partial = []
        for e in entries:
            hits = [i for i, d in enumerate(e[0]) if d is not None and have[i] == d]
            clash = [i for i, d in enumerate(e[0]) if d is not None and have[i] not in (None, d)]
            if hits and not clash and self.entry_fits(out, kind, ins, axis, e):
                partial.append(e)
        if len(partial) == 1:
            self.rewrite(out, ins, axis, partial[0], "inference")
            return True
        if len(partial) > 1:
            self.conflicts.add((out, axis))
            self.log.append(f"conflict {out} {axis} {len(partial)} partial matches")
        return False

    def propagate(self):
        self.log.append("propagate")
        changed = True
        while changed:
            changed = False
            for axis, _ in self.axes:
                for out, kind, ins in self.ops:
                    changed |= self.try_op(out, kind, ins, axis)
                for out, kind, ins in reversed(self.ops):
                    changed |= self.try_op(out, kind, ins, axis)

    def tile(self, value, dim, axis):
        if axis not in self.size:
            raise PlanError("PARTIR_E_AXIS", f"unknown axis {axis}")
        self.log.append(f"tile {value} {dim} {axis}")
        if (value, axis) in self.tiled and self.tiled[(value, axis)] != dim:
            raise PlanError("PARTIR_E_AXIS", f"{value} already tiled on {axis}")
        cuts = {a: d for (v, a), d in self.tiled.items() if v == value}
        if self.shapes[value][dim] % self.parts(value, dim, axis, cuts):
            raise PlanError("PARTIR_E_DIVISIBILITY", f"{value} dim {dim}")
        self.tiled[(value, axis)] = dim
        self.sliced[(value, axis)] = dim


def run(program, schedule):
    """schedule: [(axis, {name: dim})] ManualPartition tactics, each followed
    by propagation (the desugaring of Sec. 3)."""
    st = State(program)
    for axis, parts in schedule:
        for name, dim in parts.items():
            st.tile(name, dim, axis)
        st.propagate()
    return st


# ---------------------------------------------------------------------------
# executing a partitioned program (App. C loop semantics)
# ---------------------------------------------------------------------------
def _apply(kind, xs):
    if kind == "matmul":
        return O.matmul(xs[0], xs[1])
    if kind == "add":
        return xs[0] + xs[1]
    if kind == "gelu":
        return O.gelu_erf(xs[0])
    if kind == "rmsnorm":
        return O.rmsnorm(xs[0], np.ones(xs[0].shape[1]), 1e-6)
    raise ValueError(kind)


def evaluate(program, args, nest=None, cuts=None, size=None):
    """Evaluate `program` on `args` {name: array}.  With a plan (nest: out ->
    [(axis, action)], cuts: (out, i, axis) -> dim, size: axis -> size) every
    op runs as its loop nest over sliced operands; without, unpartitioned."""
    _, _, ops, _ = parse_program(program)
    env = dict(args)
    for out, kind, ins in ops:
        operands = [env[v] for v in ins]
        if not nest or not nest.get(out):
            env[out] = _apply(kind, operands)
            continue
        loops = nest[out]

        def body(level, xs, _loops=loops, _out=out, _kind=kind):
            if level == len(_loops):
                return _apply(_kind, xs)
            axis, act = _loops[level]
            R = size[axis]

            def iteration(r):
                ys = [O.slice_(x, cuts[(_out, i, axis)], r, R) if (_out, i, axis) in cuts else x
                      for i, x in enumerate(xs)]
                return body(level + 1, ys)

            return O.loop_sum(R, iteration) if act == SUM else O.loop_tile(R, act, iteration)

        env[out] = body(0, operands)
    return env
