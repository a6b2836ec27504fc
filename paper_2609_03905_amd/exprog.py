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
