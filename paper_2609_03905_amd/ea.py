"""Python binding of libea (the C ABI declared in include/ea.h).

Argument marshalling only: every step of a join-agg or repartition runs in the
HIP kernels of libea.so.  PyTorch provides device memory (uint8 tensors) and
the current HIP stream.  If libea.so has not been built the import of a
compute function raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libea.so")

# ---- codes (mirror include/ea.h) ------------------------------------------
OK = 0
ERR_NAMES = {-1: "EA_ERR_ARG", -2: "EA_ERR_DTYPE", -3: "EA_ERR_PARTITION", -4: "EA_ERR_CAPACITY",
             -5: "EA_ERR_SPEC", -6: "EA_ERR_JOIN", -7: "EA_ERR_UNSUPPORTED", -8: "EA_ERR_HIP",
             -9: "EA_ERR_NOPLAN"}
WS_COUNTER_BYTES = 262144  # EA_WS_COUNTER_BYTES: the counter area at the start of a workspace
F32, BF16, F16 = 0, 1, 2
DTYPES = {"f32": F32, "bf16": BF16, "f16": F16}
ELEM_SIZE = {"f32": 4, "bf16": 2, "f16": 2}
JOIN_MUL, JOIN_ADD = 0, 1
OP_RMSNORM, OP_SOFTMAX, OP_ATTENTION, OP_SWIGLU = 16, 17, 18, 19
AGG_NONE, AGG_SUM, AGG_MAX, AGG_LSE = 0, 1, 2, 3
STORE_CACHED, STORE_STREAM = 0, 1  # output store policy (EA_STORE_*)


class EAError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERR_NAMES.get(code, code)}: {msg}")
        self.code = code


class _Params(ctypes.Structure):
    _fields_ = [("eps", ctypes.c_float), ("scale", ctypes.c_float), ("causal", ctypes.c_int32),
                ("store", ctypes.c_int32), ("residual", ctypes.c_void_p), ("gqa_group", ctypes.c_int32),
                ("n_seq", ctypes.c_int32), ("seq_ends", ctypes.c_void_p)]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2609_03905_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        i32, i64, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
        P = ctypes.POINTER
        L.ea_version.restype = ctypes.c_int
        L.ea_last_error.restype = ctypes.c_char_p
        L.ea_dtype_size.argtypes = [i32]
        L.ea_layout_nbytes.argtypes = [i32, P(i64), i32, P(i32), P(i64), P(i64)]
        L.ea_relation_create.argtypes = [i32, P(i64), i32, P(i32), P(i64), vp, i64, P(vp)]
        L.ea_relation_destroy.argtypes = [vp]
        L.ea_relation_set_data.argtypes = [vp, vp, i64]
        L.ea_relation_num_blocks.argtypes = [vp, P(i64)]
        L.ea_relation_nbytes.argtypes = [vp, P(i64)]
        L.ea_relation_block.argtypes = [vp, i64, P(i64), P(i64), P(i64)]
        L.ea_joinagg.argtypes = [ctypes.c_char_p, i32, i32, i32, P(vp), vp, P(_Params), vp, i64, vp]
        L.ea_joinagg_workspace.argtypes = [ctypes.c_char_p, i32, i32, i32, P(vp), vp, P(_Params), P(i64), vp]
        L.ea_repartition_plan.argtypes = [vp, vp, vp]
        L.ea_joinagg_noalloc.argtypes = [ctypes.c_char_p, i32, i32, i32, P(vp), vp, P(_Params), vp]
        L.ea_join_tuples.argtypes = [ctypes.c_char_p, i32, i32, P(vp), vp, P(_Params), vp, i64, vp, i64,
                                     P(i64), P(i64), vp]
        L.ea_repartition.argtypes = [vp, vp, vp]
        L.ea_repartition_ex.argtypes = [vp, vp, i32, vp]
        L.ea_overlay.argtypes = [i32, P(i32), P(i64), P(i32), P(i64), P(i32), P(i64)]
        L.ea_logical_plan.argtypes = [i32, ctypes.c_void_p, i64, P(i32), P(i64)]
        L.ea_exprog_check.argtypes = [ctypes.c_char_p, P(i32), ctypes.c_char_p, i64]
        L.ea_exprog_naive.argtypes = [ctypes.c_char_p, ctypes.c_char_p, i64, P(i64)]
        L.ea_exprog_simulate.argtypes = [ctypes.c_char_p, ctypes.c_double, ctypes.c_double, P(ctypes.c_double)]
        L.ea_exprog_synthesize.argtypes = [ctypes.c_char_p, ctypes.c_double, ctypes.c_double, i32, ctypes.c_uint64,
                                           ctypes.c_char_p, i64, P(i64), P(ctypes.c_double)]
        L.ea_exprog_preamble.argtypes = [i32, P(i32), P(i64), i32, P(i64), P(i32), P(i32), P(i64), i32, P(i64), i32,
                                         i64, ctypes.c_char_p, i64, P(i64)]
        L.ea_plan_cache_size.restype = i64
        L.ea_plan_cache_clear.restype = ctypes.c_int
        _lib = L
    return _lib


def _check(rc: int):
    if rc != OK:
        raise EAError(rc, lib().ea_last_error().decode())


def _arr(ctype, values):
    values = list(values)
    return (ctype * max(len(values), 1))(*values)


def _partition_args(partition):
    nb = _arr(ctypes.c_int32, [len(s) - 1 for s in partition])
    sp = _arr(ctypes.c_int64, [int(p) for s in partition for p in s])
    return nb, sp


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        if not torch.cuda.is_available():
            return ctypes.c_void_p(None)  # host-side validation still runs; HIP calls then fail
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def version() -> int:
    return int(lib().ea_version())


def layout_nbytes(shape, dtype: str, partition) -> int:
    nb, sp = _partition_args(partition)
    out = ctypes.c_int64(0)
    _check(lib().ea_layout_nbytes(len(shape), _arr(ctypes.c_int64, shape), DTYPES[dtype], nb, sp,
                                  ctypes.byref(out)))
    return int(out.value)


def overlay(part_a, part_b):
    """Per dim, the sorted union of both partitions' split points (Section 5.3)."""
    rank = len(part_a)
    nba, spa = _partition_args(part_a)
    nbb, spb = _partition_args(part_b)
    nbo = (ctypes.c_int32 * rank)()
    spo = (ctypes.c_int64 * sum(len(a) + len(b) for a, b in zip(part_a, part_b)))()
    _check(lib().ea_overlay(rank, nba, spa, nbb, spb, nbo, spo))
    out, k = [], 0
    for d in range(rank):
        out.append([int(spo[k + i]) for i in range(nbo[d] + 1)])
        k += nbo[d] + 1
    return out


class Relation:
    """A tensor relation: a shape, a dtype, a block partition (split points
    per dim) and block-major storage in a torch uint8 device tensor."""

    def __init__(self, shape: Sequence[int], dtype: str, partition, data: torch.Tensor | None = None,
                 device: str | torch.device = "cuda", allocate: bool = True, byte_offset: int = 0):
        self.shape = tuple(int(s) for s in shape)
        self.dtype = dtype
        self.partition = [list(map(int, s)) for s in partition]
        self.nbytes = layout_nbytes(self.shape, dtype, self.partition)
        if data is None and allocate:
            data = torch.empty(max(self.nbytes, 1), dtype=torch.uint8, device=device)
        self.data = data
        self._byte_offset = int(byte_offset)
        ptr, cap = None, 0
        if data is not None:
            ptr = data.data_ptr() + self._byte_offset
            cap = data.numel() * data.element_size() - self._byte_offset
        nb, sp = _partition_args(self.partition)
        h = ctypes.c_void_p()
        _check(lib().ea_relation_create(len(self.shape), _arr(ctypes.c_int64, self.shape), DTYPES[dtype], nb, sp,
                                        ctypes.c_void_p(ptr) if ptr else None, cap, ctypes.byref(h)))
        self.handle = h

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and _lib is not None:
            _lib.ea_relation_destroy(h)
            self.handle = None

    # -- views ---------------------------------------------------------------
    def view(self, byte_offset: int, shape, dtype: str, partition) -> "Relation":
        """Another relation over this relation's storage, starting
        ``byte_offset`` bytes in (for example a per-head slice)."""
        return Relation(shape, dtype, partition, data=self.data, byte_offset=self._byte_offset + byte_offset)

    def bytes(self) -> torch.Tensor:
        """The relation's storage as a uint8 tensor (a view)."""
        return self.data[self._byte_offset:self._byte_offset + self.nbytes]

    # -- introspection -------------------------------------------------------
    def num_blocks(self) -> int:
        n = ctypes.c_int64()
        _check(lib().ea_relation_num_blocks(self.handle, ctypes.byref(n)))
        return int(n.value)

    def block(self, b: int):
        r = len(self.shape)
        lo, hi, off = (ctypes.c_int64 * r)(), (ctypes.c_int64 * r)(), ctypes.c_int64()
        _check(lib().ea_relation_block(self.handle, b, lo, hi, ctypes.byref(off)))
        return list(lo), list(hi), int(off.value)


def _params(eps=0.0, scale=0.0, causal=False, store=0, residual=None, gqa_group=0, seq_ends=None):
    """ea_params plus the host array it points at (kept alive by the caller)."""
    ends = None
    if seq_ends is not None:
        ends = (ctypes.c_int64 * max(1, len(seq_ends)))(*[int(e) for e in seq_ends])
    prm = _Params(eps, scale, int(causal), int(store), residual.handle.value if residual is not None else None,
                  int(gqa_group), 0 if seq_ends is None else len(seq_ends),
                  ctypes.cast(ends, ctypes.c_void_p) if ends is not None else None)
    return prm, ends


def new_workspace(nbytes: int, device=None) -> torch.Tensor:
    """A zeroed device buffer usable as a join-agg workspace of ``nbytes``
    (the counter area must start zeroed; every call leaves it zeroed)."""
    return torch.zeros(max(int(nbytes), 1), dtype=torch.uint8, device=device or "cuda")


_WS = {}  # (device, stream handle) -> workspace tensor of the calls on that stream
_WS_RETIRED = []  # outgrown workspaces: kernels queued earlier may still use them


def _stream_workspace(nbytes: int, stream: ctypes.c_void_p) -> torch.Tensor:
    """The binding's workspace for calls on ``stream``: calls on one stream run
    in order, so they share one buffer, grown (zeroed) when a plan needs more."""
    dev = torch.cuda.current_device()
    key = (dev, stream.value or 0)
    buf = _WS.get(key)
    if buf is None or buf.numel() < nbytes:
        if buf is not None:
            _WS_RETIRED.append(buf)
        buf = new_workspace(max(nbytes, 2 * buf.numel() if buf is not None else nbytes), device=dev)
        torch.cuda.synchronize(dev)  # zeroed before any stream uses it
        _WS[key] = buf
    return buf


def joinagg_workspace(spec: str, join_op: int, agg_op: int, inputs: Sequence[Relation], out: Relation, *,
                      eps: float = 0.0, scale: float = 0.0, causal: bool = False, residual: Relation | None = None,
                      store: int = 0, gqa_group: int = 0, seq_ends=None, stream=None) -> int:
    """Plan a join-agg configuration (first call: allocate the plan, run the
    GPU join, wait for it) and return the workspace bytes its runs need."""
    handles = _arr(ctypes.c_void_p, [r.handle.value for r in inputs])
    prm, _ends = _params(eps, scale, causal, store, residual, gqa_group, seq_ends)
    n = ctypes.c_int64()
    _check(lib().ea_joinagg_workspace(spec.encode(), join_op, agg_op, len(inputs), handles, out.handle,
                                      ctypes.byref(prm), ctypes.byref(n), _stream(stream)))
    return int(n.value)


def joinagg(spec: str, join_op: int, agg_op: int, inputs: Sequence[Relation], out: Relation, *,
            eps: float = 0.0, scale: float = 0.0, causal: bool = False, residual: Relation | None = None,
            store: int = 0, gqa_group: int = 0, seq_ends=None, stream=None,
            workspace: torch.Tensor | None = None) -> None:
    """Run one GPU's share of a join-agg: join the input relations' blocks,
    run the per-tuple kernel, aggregate by output key, store into ``out``.
    ``store``: STORE_CACHED (default) or STORE_STREAM (non-temporal output
    stores, for an output nothing reads soon).  Attention: ``gqa_group``
    query heads per key-value head, ``seq_ends`` the ends of packed
    sequences.  The configuration is planned on first use (see
    joinagg_workspace).  ``workspace``: a device buffer from new_workspace
    for key-split partials; by default one buffer per stream, held by the
    binding."""
    handles = _arr(ctypes.c_void_p, [r.handle.value for r in inputs])
    prm, _ends = _params(eps, scale, causal, store, residual, gqa_group, seq_ends)
    s = _stream(stream)
    need = ctypes.c_int64()
    spec_b = spec.encode()
    _check(lib().ea_joinagg_workspace(spec_b, join_op, agg_op, len(inputs), handles, out.handle, ctypes.byref(prm),
                                      ctypes.byref(need), s))
    ws, nbytes = None, 0
    if need.value:
        buf = workspace if workspace is not None else _stream_workspace(need.value, s)
        ws, nbytes = ctypes.c_void_p(buf.data_ptr()), buf.numel() * buf.element_size()
    _check(lib().ea_joinagg(spec_b, join_op, agg_op, len(inputs), handles, out.handle, ctypes.byref(prm), ws, nbytes,
                            s))


def joinagg_noalloc(spec: str, join_op: int, agg_op: int, inputs: Sequence[Relation], out: Relation, *,
                    eps: float = 0.0, scale: float = 0.0, causal: bool = False, residual: Relation | None = None,
                    store: int = 0, gqa_group: int = 0, seq_ends=None, stream=None) -> None:
    """ea_joinagg_noalloc: run a join-agg planned earlier (joinagg_workspace)
    with the library's own per-device workspace array; allocates nothing.
    Calls that may overlap in time on one GPU race on that array."""
    handles = _arr(ctypes.c_void_p, [r.handle.value for r in inputs])
    prm, _ends = _params(eps, scale, causal, store, residual, gqa_group, seq_ends)
    _check(lib().ea_joinagg_noalloc(spec.encode(), join_op, agg_op, len(inputs), handles, out.handle,
                                    ctypes.byref(prm), _stream(stream)))


def repartition_plan(src: Relation, dst: Relation, stream=None) -> None:
    """Plan the repartition of ``src``'s partition into ``dst``'s (first call:
    build and upload its overlay boxes, wait)."""
    _check(lib().ea_repartition_plan(src.handle, dst.handle, _stream(stream)))


def repartition(src: Relation, dst: Relation, stream=None, *, store: int = 0) -> None:
    """Write ``src``'s dense tensor into ``dst`` under ``dst``'s partition
    (``store`` as for joinagg); planned on first use."""
    s = _stream(stream)
    _check(lib().ea_repartition_plan(src.handle, dst.handle, s))
    _check(lib().ea_repartition_ex(src.handle, dst.handle, int(store), s))


def join_tuples(spec: str, join_op: int, inputs: Sequence[Relation], out: Relation, *, causal: bool = False,
                scale: float = 1.0, eps: float = 1e-6, gqa_group: int = 0, seq_ends=None, stream=None):
    """The GPU-built tuple table and CSR group offsets of a join (synchronous)."""
    handles = _arr(ctypes.c_void_p, [r.handle.value for r in inputs])
    prm, _ends = _params(eps, scale, causal, 0, None, gqa_group, seq_ends)
    n_t, n_g = ctypes.c_int64(), ctypes.c_int64()
    dev = out.data.device if out.data is not None else torch.device("cuda")
    # first call sizes the tables (it fails with EA_ERR_CAPACITY but reports the counts)
    rc = lib().ea_join_tuples(spec.encode(), join_op, len(inputs), handles, out.handle, ctypes.byref(prm), None, 0,
                              None, 0, ctypes.byref(n_t), ctypes.byref(n_g), _stream(stream))
    if rc not in (OK, -1, -4):
        _check(rc)
    tuples = torch.zeros((max(n_t.value, 1), len(inputs) + 1), dtype=torch.int32, device=dev)
    goff = torch.zeros(n_g.value + 1, dtype=torch.int64, device=dev)
    _check(lib().ea_join_tuples(spec.encode(), join_op, len(inputs), handles, out.handle, ctypes.byref(prm),
                                ctypes.c_void_p(tuples.data_ptr()), tuples.shape[0], ctypes.c_void_p(goff.data_ptr()),
                                goff.numel(), ctypes.byref(n_t), ctypes.byref(n_g), _stream(stream)))
    return tuples[:n_t.value], goff


def plan_cache_size() -> int:
    return int(lib().ea_plan_cache_size())


def plan_cache_clear() -> None:
    _check(lib().ea_plan_cache_clear())


# ---- dense <-> relation through the library's own repartition ---------------
def whole_partition(shape):
    return [[0, int(n)] for n in shape]


def from_dense(dense: torch.Tensor, dtype: str, partition, stream=None) -> Relation:
    """A new relation holding ``dense`` (a contiguous device tensor whose bytes
    are the dtype's storage) under ``partition``; the re-blocking runs on the
    GPU (a one-block relation over the dense tensor, repartitioned)."""
    dense = dense.contiguous()
    raw = dense.view(torch.uint8).reshape(-1)
    src = Relation(dense.shape, dtype, whole_partition(dense.shape), data=raw)
    dst = Relation(dense.shape, dtype, partition, device=dense.device)
    repartition(src, dst, stream)
    return dst


def to_dense(rel: Relation, stream=None) -> torch.Tensor:
    """The relation's dense tensor as raw storage (uint8, then viewed by the
    caller), re-blocked on the GPU."""
    dst = Relation(rel.shape, rel.dtype, whole_partition(rel.shape), device=rel.data.device)
    repartition(rel, dst, stream)
    return dst.bytes()
