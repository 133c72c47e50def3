"""MI355X-native sampler of multi-hop query training data (SMORE, arXiv 2110.14890).

Thin Python binding over the C ABI of ``libsmore.so`` (declared in
``include/smore.h``).  It only marshals arguments: graph building, reverse
directional sampling of positives and bidirectional rejection sampling of
negatives all run in the library's HIP kernels.  PyTorch provides device
memory and the current HIP stream.  There is no CPU fallback: if the library
is not built, every call raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsmore.so")

TYPES = ("1p", "2p", "3p", "2i", "3i", "ip", "pi", "2u", "up", "2in", "3in", "inp", "pin", "pni")
ADD_INVERSE = 1
MAX_NEG_TRIES = 4096
OP_ANCHOR, OP_PROJ, OP_AND, OP_OR, OP_NOT = range(5)
ERRORS = {0: "OK", -1: "INVALID_ARG", -2: "RANGE", -3: "UNSUPPORTED", -4: "NOMEM", -5: "HIP",
          -6: "OVERFLOW"}

c_i32, c_i64, c_u32, c_u64, c_vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_void_p


class DagNode(ctypes.Structure):
    _fields_ = [("op", c_i32), ("n_child", c_i32), ("child", c_i32 * 3), ("slot", c_i32)]


class QueryDag(ctypes.Structure):
    _fields_ = [("n_nodes", c_i32), ("root", c_i32), ("node", DagNode * 16)]


class SampleArgs(ctypes.Structure):
    _fields_ = [("batch", c_i32), ("n_neg", c_i32), ("pos_tries", c_i32), ("neg_tries", c_i32),
                ("max_fanout", c_i32), ("seed", c_u64), ("query_offset", c_u64), ("flags", c_u32)]


class SampleOut(ctypes.Structure):
    _fields_ = [(n, c_vp) for n in ("anchors", "relations", "positive", "negatives", "n_valid",
                                    "pos_attempts", "neg_draws")]


SHARED_FIELDS = ("anchors", "relations", "positive", "pos_attempts", "shared", "n_shared", "mask",
                 "n_valid")


class SharedOut(ctypes.Structure):
    _fields_ = [(n, c_vp) for n in SHARED_FIELDS]


OUT_FIELDS = ("anchors", "relations", "positive", "negatives", "n_valid", "pos_attempts",
              "neg_draws")


class SmoreError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                               "(python paper_2110_14890_amd/build.py)")
        L = ctypes.CDLL(LIB_PATH)
        L.smore_last_error.restype = ctypes.c_char_p
        L.smore_build_graph.argtypes = [c_vp, c_i64, c_i32, c_i32, c_u32, ctypes.POINTER(c_vp)]
        L.smore_graph_info.argtypes = [c_vp] + [ctypes.POINTER(c_i64)] * 6
        L.smore_graph_copy.argtypes = [c_vp, c_i32, c_vp, c_i64]
        L.smore_query_preset.argtypes = [ctypes.c_char_p, ctypes.POINTER(QueryDag)]
        L.smore_plan.argtypes = [ctypes.POINTER(QueryDag), c_i32, ctypes.POINTER(c_i32),
                                 ctypes.POINTER(c_i32)]
        L.smore_sample_workspace_bytes.argtypes = [c_vp, ctypes.POINTER(QueryDag),
                                                   ctypes.POINTER(SampleArgs),
                                                   ctypes.POINTER(ctypes.c_size_t)]
        L.smore_sample.argtypes = [c_vp, ctypes.POINTER(QueryDag), ctypes.POINTER(SampleArgs),
                                   ctypes.POINTER(SampleOut), c_vp, ctypes.c_size_t, c_vp]
        L.smore_sample_noalloc.argtypes = [c_vp, ctypes.POINTER(QueryDag), ctypes.POINTER(SampleArgs),
                                           ctypes.POINTER(SampleOut), c_vp]
        L.smore_sample_shared.argtypes = [c_vp, ctypes.POINTER(QueryDag), ctypes.POINTER(SampleArgs),
                                          ctypes.POINTER(SharedOut), c_vp, ctypes.c_size_t, c_vp]
        L.smore_verify.argtypes = [c_vp, ctypes.POINTER(QueryDag), ctypes.POINTER(SampleArgs), c_vp,
                                   c_vp, c_vp, c_vp, c_vp, c_vp, ctypes.c_size_t, c_vp]
        L.smore_sample_positives.argtypes = [c_vp, ctypes.POINTER(QueryDag),
                                             ctypes.POINTER(SampleArgs), ctypes.POINTER(SampleOut),
                                             c_vp]
        L.smore_sample_negatives.argtypes = [c_vp, ctypes.POINTER(QueryDag),
                                             ctypes.POINTER(SampleArgs), ctypes.POINTER(SampleOut),
                                             c_vp, c_vp, ctypes.c_size_t, c_vp]
        L.smore_sample_negatives_part.argtypes = [c_vp, ctypes.POINTER(QueryDag),
                                                  ctypes.POINTER(SampleArgs),
                                                  ctypes.POINTER(SampleOut), c_vp, c_i32, c_vp,
                                                  ctypes.c_size_t, c_vp]
        L.smore_profile_kernel.argtypes = [c_vp, c_vp, c_i32]
        L.smore_wait_before_kernel.argtypes = [c_vp, c_i32]
        L.smore_gather_probe.argtypes = [c_vp, c_i64, c_i64, c_vp, c_i64, c_vp]
        L.smore_free_graph.argtypes = [c_vp]
        L.smore_free_graph.restype = None
        _lib = L
    return _lib


def last_error() -> str:
    return lib().smore_last_error().decode()


def _check(rc: int) -> None:
    if rc != 0:
        raise SmoreError(rc, last_error())


def query_preset(name: str) -> QueryDag:
    d = QueryDag()
    _check(lib().smore_query_preset(name.encode(), ctypes.byref(d)))
    return d


def plan(dag: "QueryDag | str", tie_break: int = 0) -> list:
    if isinstance(dag, str):
        dag = query_preset(dag)
    cut = (c_i32 * 16)()
    n = c_i32()
    _check(lib().smore_plan(ctypes.byref(dag), tie_break, cut, ctypes.byref(n)))
    return [cut[k] for k in range(n.value)]


class Graph:
    """Device adjacency owned by the library (smore_build_graph / smore_free_graph)."""

    def __init__(self, triples, n_entities: int, n_relations: int, add_inverse: bool = False):
        tr = np.ascontiguousarray(triples, dtype=np.int32).reshape(-1, 3)
        h = c_vp()
        _check(lib().smore_build_graph(tr.ctypes.data if len(tr) else None, len(tr), n_entities,
                                       n_relations, ADD_INVERSE if add_inverse else 0,
                                       ctypes.byref(h)))
        self._h = h
        vals = [c_i64() for _ in range(6)]
        _check(lib().smore_graph_info(h, *[ctypes.byref(v) for v in vals]))
        (self.V, self.R, self.E, self.S_fwd, self.S_rev, self.device_bytes) = [v.value for v in vals]

    @property
    def handle(self):
        return self._h

    _SIZES = {0: "V+1", 1: "2*(S_fwd+1)", 2: "E", 3: "V+1", 4: "2*(S_rev+1)", 5: "E", 6: "A"}

    def copy(self, which: int, count: int) -> np.ndarray:
        out = np.zeros(max(count, 1), np.int32)
        _check(lib().smore_graph_copy(self._h, which, out.ctypes.data, count))
        return out[:count]

    def close(self) -> None:
        if getattr(self, "_h", None):
            lib().smore_free_graph(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def build_graph(triples, n_entities: int, n_relations: int, add_inverse: bool = False) -> Graph:
    return Graph(triples, n_entities, n_relations, add_inverse)


def make_args(batch: int, n_neg: int, seed: int = 0, query_offset: int = 0, pos_tries: int = 64,
              neg_tries: int | None = None, max_fanout: int = 0, flags: int = 0) -> SampleArgs:
    if neg_tries is None:
        neg_tries = 4 * n_neg
    return SampleArgs(batch, n_neg, pos_tries, neg_tries, max_fanout, seed, query_offset, flags)


def alloc_outputs(batch: int, n_neg: int, device=None) -> dict:
    import torch
    dev = device if device is not None else torch.device("cuda", torch.cuda.current_device())
    z = lambda *s: torch.empty(s, dtype=torch.int32, device=dev)
    return {"anchors": z(batch, 3), "relations": z(batch, 3), "positive": z(batch),
            "negatives": z(batch, n_neg), "n_valid": z(batch), "pos_attempts": z(batch),
            "neg_draws": z(batch)}


def workspace_bytes(dag: QueryDag, args: SampleArgs) -> int:
    n = ctypes.c_size_t()
    _check(lib().smore_sample_workspace_bytes(None, ctypes.byref(dag), ctypes.byref(args),
                                              ctypes.byref(n)))
    return n.value


class Workspace:
    """Device scratch for the sampling calls, grown on demand (a uint8 torch
    tensor).  One per stream: calls that overlap must not share it."""

    def __init__(self, device=None):
        self.device = device
        self.buf = None

    def get(self, nbytes: int):
        import torch
        if self.buf is None or self.buf.numel() < nbytes:
            dev = self.device if self.device is not None else torch.device(
                "cuda", torch.cuda.current_device())
            self.buf = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
        return self.buf


_default_ws = {}


def _workspace(ws, dag, args, stream=None):
    """The caller's workspace, or a default one per (device, stream) the call
    runs on, so that calls on different streams never share scratch."""
    import torch
    if args.n_neg == 0:        # nothing is drawn: the library needs no workspace
        return None, 0
    if ws is None:
        st = stream if stream is not None else torch.cuda.current_stream()
        key = (st.device, st.cuda_stream)
        ws = _default_ws.setdefault(key, Workspace(st.device))
    buf = ws.get(workspace_bytes(dag, args))
    return c_vp(buf.data_ptr()), buf.numel()


def sample_into(graph: Graph, dag: QueryDag, args: SampleArgs, out: dict, stream=None,
                workspace: "Workspace | None" = None) -> dict:
    """smore_sample into caller-owned torch tensors on the current (or given) stream."""
    _require(out, _sample_shapes(args))
    wp, wn = _workspace(workspace, dag, args, stream)
    _check(lib().smore_sample(graph.handle, ctypes.byref(dag), ctypes.byref(args),
                              ctypes.byref(_out_struct(out)), wp, wn, _stream_handle(stream)))
    return out


NOALLOC_SCRATCH_BYTES = 64 << 20


def sample_noalloc_into(graph: Graph, dag: QueryDag, args: SampleArgs, out: dict,
                        stream=None) -> dict:
    """smore_sample_noalloc: smore_sample without a workspace argument (the
    library's fixed per-device scratch; calls on one GPU must not overlap)."""
    _require(out, _sample_shapes(args))
    _check(lib().smore_sample_noalloc(graph.handle, ctypes.byref(dag), ctypes.byref(args),
                                      ctypes.byref(_out_struct(out)), _stream_handle(stream)))
    return out


def alloc_shared_outputs(batch: int, n_shared: int, device=None) -> dict:
    """Device outputs of sample_shared_into (the mask is int32 storage of the
    uint32 words)."""
    import torch
    dev = device if device is not None else torch.device("cuda", torch.cuda.current_device())
    z = lambda *s: torch.empty(s, dtype=torch.int32, device=dev)
    return {"anchors": z(batch, 3), "relations": z(batch, 3), "positive": z(batch),
            "pos_attempts": z(batch), "shared": z(n_shared), "n_shared": z(1),
            "mask": z(batch, (n_shared + 31) // 32), "n_valid": z(batch)}


def sample_shared_into(graph: Graph, dag: QueryDag, args: SampleArgs, out: dict, stream=None,
                       workspace: "Workspace | None" = None) -> dict:
    """smore_sample_shared: args.n_neg is the size of the shared candidate set."""
    b, n = args.batch, args.n_neg
    _require(out, {"anchors": (b, 3), "relations": (b, 3), "positive": (b,), "pos_attempts": (b,),
                   "shared": (n,), "n_shared": (1,), "mask": (b, (n + 31) // 32), "n_valid": (b,)})
    wp, wn = _workspace(workspace, dag, args, stream)
    st = SharedOut(*[out[k].data_ptr() if out[k].numel() else None for k in SHARED_FIELDS])
    _check(lib().smore_sample_shared(graph.handle, ctypes.byref(dag), ctypes.byref(args),
                                     ctypes.byref(st), wp, wn, _stream_handle(stream)))
    return out


def sample_shared(graph: Graph, qtype: "str | QueryDag", batch: int, n_shared: int, seed: int = 0,
                  query_offset: int = 0, pos_tries: int = 64, neg_tries: int | None = None,
                  max_fanout: int = 0, stream=None) -> dict:
    """A minibatch of `batch` queries sharing one set of `n_shared` candidate
    negatives, with the mask of verified negatives per query."""
    dag = query_preset(qtype) if isinstance(qtype, str) else qtype
    args = make_args(batch, n_shared, seed, query_offset, pos_tries, neg_tries, max_fanout)
    out = alloc_shared_outputs(batch, n_shared)
    return sample_shared_into(graph, dag, args, out, stream)


def verify(graph: Graph, qtype: "str | QueryDag", anchors, relations, candidates, stream=None,
           workspace: "Workspace | None" = None) -> dict:
    """smore_verify: which of the candidates (device int32 [batch, n]) are
    entities outside each query's answer set.  Returns {"mask" (int32
    storage of the uint32 words), "n_valid"}."""
    import torch
    dag = query_preset(qtype) if isinstance(qtype, str) else qtype
    batch, n = candidates.shape
    for name, t, shape in (("anchors", anchors, (batch, 3)), ("relations", relations, (batch, 3)),
                           ("candidates", candidates, (batch, n))):
        if tuple(t.shape) != shape or t.dtype != torch.int32 or not t.is_contiguous() \
                or t.device != candidates.device or not t.is_cuda:
            raise ValueError(f"{name} must be a contiguous int32 device tensor of shape {shape}")
    args = make_args(batch, n, neg_tries=n)
    dev = candidates.device
    out = {"mask": torch.empty((batch, (n + 31) // 32), dtype=torch.int32, device=dev),
           "n_valid": torch.empty(batch, dtype=torch.int32, device=dev)}
    wp, wn = _workspace(workspace, dag, args, stream)
    ptr = lambda t: t.data_ptr() if t.numel() else None
    _check(lib().smore_verify(graph.handle, ctypes.byref(dag), ctypes.byref(args),
                              anchors.data_ptr(), relations.data_ptr(), ptr(candidates),
                              ptr(out["mask"]), out["n_valid"].data_ptr(), wp, wn,
                              _stream_handle(stream)))
    return out


def _require(tensors: dict, shapes: dict, dtype_name: str = "int32") -> None:
    """Caller-provided device buffers must have the sizes the kernels write:
    the C ABI cannot see a device buffer's length."""
    import torch
    dtype = getattr(torch, dtype_name)
    size = {}
    for k, shape in shapes.items():
        n = 1
        for d in shape:
            n *= d
        size[k] = n
        if tensors.get(k) is None and n:
            raise ValueError(f"{k}: missing (needs {n} {dtype_name})")
    dev = None
    for k, shape in shapes.items():
        t, n = tensors.get(k), size[k]
        if t is None:
            continue
        if t.dtype != dtype or not t.is_cuda or not t.is_contiguous() or t.numel() != n:
            raise ValueError(f"{k} must be a contiguous {dtype_name} device tensor of shape "
                             f"{tuple(shape)}, got {t.dtype} {tuple(t.shape)}")
        if dev is not None and t.device != dev:
            raise ValueError(f"{k} is on {t.device}, other buffers on {dev}")
        dev = t.device


def _sample_shapes(args: SampleArgs, negatives: bool = True) -> dict:
    b = args.batch
    shapes = {"anchors": (b, 3), "relations": (b, 3), "positive": (b,), "n_valid": (b,),
              "pos_attempts": (b,)}
    if negatives:
        shapes.update({"negatives": (b, args.n_neg), "neg_draws": (b,)})
    return shapes


def _out_struct(out: dict) -> SampleOut:
    return SampleOut(*[out[k].data_ptr() if k in out and out[k].numel() else None
                       for k in OUT_FIELDS])


def _stream_handle(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return c_vp(stream.cuda_stream)


def sample_positives(graph: Graph, dag: QueryDag, args: SampleArgs, out: dict, stream=None) -> dict:
    """First stage only (smore_sample_positives): anchors, relations, positive,
    pos_attempts, n_valid."""
    _require(out, _sample_shapes(args, negatives=False))
    _check(lib().smore_sample_positives(graph.handle, ctypes.byref(dag), ctypes.byref(args),
                                        ctypes.byref(_out_struct(out)), _stream_handle(stream)))
    return out


NEG_PREPARE, NEG_CANDIDATES, NEG_REST = 0, 1, 2


def sample_negatives(graph: Graph, dag: QueryDag, args: SampleArgs, out: dict, stats=None,
                     stream=None, workspace: "Workspace | None" = None, part=None) -> dict:
    """Second stage only (smore_sample_negatives) on the queries in `out`;
    stats: optional int64 [batch, 4] device tensor: (bytes, 64-byte lines) of
    graph data read per query by the candidate kernel, then by the kernel
    that intersects long lists.  part: None for the whole stage, else one of
    NEG_PREPARE, NEG_CANDIDATES, NEG_REST (smore_sample_negatives_part: the
    caller orders the three parts and passes the same workspace to each)."""
    if part is not None and workspace is None:
        raise ValueError("the parts of one negatives call must share an explicit workspace")
    _require(out, _sample_shapes(args))
    if stats is not None:
        _require({"stats": stats}, {"stats": (args.batch, 4)}, "int64")
    sp = c_vp(stats.data_ptr()) if stats is not None else None
    wp, wn = _workspace(workspace, dag, args, stream)
    if part is None:
        _check(lib().smore_sample_negatives(graph.handle, ctypes.byref(dag), ctypes.byref(args),
                                            ctypes.byref(_out_struct(out)), sp, wp, wn,
                                            _stream_handle(stream)))
    else:
        _check(lib().smore_sample_negatives_part(graph.handle, ctypes.byref(dag), ctypes.byref(args),
                                                 ctypes.byref(_out_struct(out)), sp, part, wp, wn,
                                                 _stream_handle(stream)))
    return out


KERNEL_CANDIDATES, KERNEL_HEAVY, KERNEL_SELECT = 0, 1, 2


def profile_kernel(start_event, stop_event, which: int = KERNEL_CANDIDATES) -> None:
    """Arm torch.cuda.Event objects (enable_timing=True) to be recorded around
    one kernel of the next negatives call on this thread (smore_profile_kernel)."""
    for ev in (start_event, stop_event):
        if not ev.cuda_event:          # torch creates the HIP event on first use
            ev.record()
    _check(lib().smore_profile_kernel(c_vp(start_event.cuda_event), c_vp(stop_event.cuda_event),
                                      which))


def wait_before_kernel(event, which: int = KERNEL_CANDIDATES) -> None:
    """The next negatives call on this thread waits on the torch.cuda.Event
    right before its first candidate kernel (smore_wait_before_kernel);
    None disarms."""
    if event is None:
        _check(lib().smore_wait_before_kernel(None, which))
        return
    if not event.cuda_event:           # torch creates the HIP event on first use
        event.record()
    _check(lib().smore_wait_before_kernel(c_vp(event.cuda_event), which))


def sample(graph: Graph, qtype: "str | QueryDag", batch: int, n_neg: int, seed: int = 0,
           query_offset: int = 0, pos_tries: int = 64, neg_tries: int | None = None,
           max_fanout: int = 0, stream=None) -> dict:
    """Sample `batch` queries: dict of int32 device tensors (see include/smore.h)."""
    dag = query_preset(qtype) if isinstance(qtype, str) else qtype
    args = make_args(batch, n_neg, seed, query_offset, pos_tries, neg_tries, max_fanout)
    out = alloc_outputs(batch, n_neg)
    return sample_into(graph, dag, args, out, stream)


def gather_probe(table, n_reads: int, stream=None):
    """Random-read ceiling probe (smore_gather_probe): n_reads random 4-byte
    reads from the device tensor `table`.  Returns the sink tensor; time it
    with events on `stream`."""
    import torch

    threads = (n_reads + 63) // 64
    sink = torch.empty(threads, dtype=torch.int32, device=table.device)
    st = stream if stream is not None else torch.cuda.current_stream(table.device)
    _check(lib().smore_gather_probe(c_vp(table.data_ptr()), table.numel() * table.element_size(),
                                    n_reads, c_vp(sink.data_ptr()), threads, c_vp(st.cuda_stream)))
    return sink
