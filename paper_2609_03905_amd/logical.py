"""Logical optimization (Section 4) through libea's native planner: a
join-agg spec for every abstract operator of a computation over p
processors, and the block partitions those specs induce, which the join-agg
calls take.

An operator is (spec, extents, inputs, shardable): extents maps each letter
of the einsum spec to its size; inputs names, per input of the spec, the
index of the producing operator (lower than its own) or None for a
computation input; shardable lists the letters that may be split (None:
every letter).  This module only marshals arguments: the dynamic program
runs in ea_logical_plan.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass, field

from . import ea

MAX_INPUTS = 8
MAX_LETTERS = 16


class _Lop(ctypes.Structure):
    _fields_ = [("spec", ctypes.c_char_p), ("extents", ctypes.POINTER(ctypes.c_int64)),
                ("shardable", ctypes.c_char_p), ("input", ctypes.c_int32 * MAX_INPUTS)]


@dataclass
class LogicalOp:
    spec: str
    extents: dict
    inputs: list = field(default_factory=list)
    shardable: str | None = None

    def letters(self) -> list:
        """Distinct letters in order of first appearance (inputs, then output)."""
        out = []
        for ch in self.spec.replace(",", "").replace("->", ""):
            if ch not in out:
                out.append(ch)
        return out


def plan(ops, p: int):
    """(counts, cost): counts[i] maps each letter of operator i to its
    interval count in the chosen join-agg spec; cost is the plan's total
    communication proxy."""
    n = len(ops)
    keep = []
    arr = (_Lop * n)()
    for i, op in enumerate(ops):
        ext = (ctypes.c_int64 * MAX_LETTERS)(*[int(op.extents[ch]) for ch in op.letters()])
        keep.append(ext)
        arr[i].spec = op.spec.encode()
        arr[i].extents = ext
        arr[i].shardable = None if op.shardable is None else op.shardable.encode()
        ins = [-1 if x is None else int(x) for x in op.inputs]
        ins += [-1] * (MAX_INPUTS - len(ins))
        arr[i].input = (ctypes.c_int32 * MAX_INPUTS)(*ins)
    counts = (ctypes.c_int32 * (n * MAX_LETTERS))()
    cost = ctypes.c_int64()
    ea._check(ea.lib().ea_logical_plan(n, ctypes.cast(arr, ctypes.c_void_p), int(p), counts, ctypes.byref(cost)))
    out = []
    for i, op in enumerate(ops):
        out.append({ch: int(counts[i * MAX_LETTERS + j]) for j, ch in enumerate(op.letters())})
    return out, int(cost.value)


def near_equal_splits(extent: int, count: int) -> list:
    """Split points of `count` near-equal intervals of [0, extent)."""
    return [(i * extent) // count for i in range(count)] + [extent]


def partitions(op: LogicalOp, counts: dict) -> list:
    """The partition of every operand (inputs, then output) under the spec."""
    lhs, out = op.spec.split("->")
    return [[near_equal_splits(op.extents[ch], counts[ch]) for ch in operand] for operand in lhs.split(",") + [out]]
