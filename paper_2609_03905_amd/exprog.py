"""Exchange programs (Section 5.2) through libea's native checker: the
closure and validity of Definition "Closure; validity", and the naive valid
program for a set of declarations.  Argument marshalling only."""
from __future__ import annotations

import ctypes

from . import ea


def check(text: str):
    """(valid, why): whether the program is valid; why names the first unmet
    requirement or never-enabled action of an invalid one."""
    valid = ctypes.c_int32()
    why = ctypes.create_string_buffer(512)
    ea._check(ea.lib().ea_exprog_check(text.encode(), ctypes.byref(valid), why, len(why)))
    return bool(valid.value), why.value.decode()


def naive(text: str) -> str:
    """The declarations of `text` with the gather-then-aggregate body."""
    n = ctypes.c_int64()
    rc = ea.lib().ea_exprog_naive(text.encode(), None, 0, ctypes.byref(n))
    if rc not in (ea.OK, -4):
        ea._check(rc)
    buf = ctypes.create_string_buffer(n.value + 1)
    ea._check(ea.lib().ea_exprog_naive(text.encode(), buf, len(buf), ctypes.byref(n)))
    return buf.value.decode()


# MI355X node: every GPU pair on its own xGMI link (about 153 GB/s per link
# and direction), HBM3E at about 8 TB/s
XGMI_LINK_GBS = 153.0
HBM_GBS = 8000.0


def simulate(text: str, link_gbs: float = XGMI_LINK_GBS, hbm_gbs: float = HBM_GBS) -> float:
    """Completion time in seconds of a valid program on a full xGMI mesh."""
    t = ctypes.c_double()
    ea._check(ea.lib().ea_exprog_simulate(text.encode(), float(link_gbs), float(hbm_gbs), ctypes.byref(t)))
    return t.value


def preamble(prod_partition, prod_specs, cons_partition, cons_blocks, n_gpus: int, elem_bytes: int = 0) -> str:
    """Preamble of the exchange program delivering one input (Section 5.3):
    prod_partition / cons_partition are the producer output's and the
    consumer's required tilings (split lists per dim); prod_specs lists the
    producer's function specifications as (output block index, GPU);
    cons_blocks the block each consumer specification reads."""
    rank = len(prod_partition)
    i32, i64 = ctypes.c_int32, ctypes.c_int64
    arr = lambda t, xs: (t * max(1, len(xs)))(*[int(x) for x in xs])
    pn = arr(i32, [len(sp) - 1 for sp in prod_partition])
    psp = arr(i64, [x for sp in prod_partition for x in sp])
    cn = arr(i32, [len(sp) - 1 for sp in cons_partition])
    csp = arr(i64, [x for sp in cons_partition for x in sp])
    pb = arr(i64, [b for b, _ in prod_specs])
    pg = arr(i32, [g for _, g in prod_specs])
    cb = arr(i64, cons_blocks)
    n = ctypes.c_int64()
    args = [rank, pn, psp, len(prod_specs), pb, pg, cn, csp, len(cons_blocks), cb, int(n_gpus), int(elem_bytes)]
    rc = ea.lib().ea_exprog_preamble(*args, None, 0, ctypes.byref(n))
    if rc not in (ea.OK, -4):
        ea._check(rc)
    buf = ctypes.create_string_buffer(n.value + 1)
    ea._check(ea.lib().ea_exprog_preamble(*args, buf, len(buf), ctypes.byref(n)))
    return buf.value.decode()


def synthesize(text: str, link_gbs: float = XGMI_LINK_GBS, hbm_gbs: float = HBM_GBS, iters: int = 2000,
               seed: int = 0):
    """Body synthesis (Section 5.4) for the declarations in text: returns
    (program, simulated seconds).  The search starts from the naive program
    under the cheapest membership and applies the paper's transformations,
    keeping only valid programs."""
    n = ctypes.c_int64()
    t = ctypes.c_double()
    args = [text.encode(), float(link_gbs), float(hbm_gbs), int(iters), int(seed) & (2**64 - 1)]
    rc = ea.lib().ea_exprog_synthesize(*args, None, 0, ctypes.byref(n), ctypes.byref(t))
    if rc not in (ea.OK, -4):
        ea._check(rc)
    buf = ctypes.create_string_buffer(n.value + 1)
    ea._check(ea.lib().ea_exprog_synthesize(*args, buf, len(buf), ctypes.byref(n), ctypes.byref(t)))
    return buf.value.decode(), t.value
