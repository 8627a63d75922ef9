"""Python binding of libwb, the gfx950 resharding library (WeightBridge,
arXiv 2609.25442, Sec. 3.1-3.2): layouts as slice-copy source maps, the
routing plan, and the packing and assembly kernels.

Argument marshalling only: every step runs in libwb.so (host planner in C++,
kernels in HIP). Importing this package fails if the library is not built
(``python paper_2609_25442_amd/build.py``); there is no fallback path.
"""

from __future__ import annotations

import atexit
import collections.abc
import ctypes
import os
import weakref
from ctypes import POINTER, byref, c_char_p, c_int32, c_int64, c_size_t, c_uint32, c_uint64, c_void_p

_HERE = os.path.dirname(os.path.abspath(__file__))
# WB_LIB selects another build of the same library (e.g. a tuning variant)
LIB_PATH = os.environ.get("WB_LIB") or os.path.join(_HERE, "libwb.so")

WB_OK, WB_EINVAL, WB_EUNSUPPORTED, WB_ENOMEM, WB_EHIP, WB_ESIZE = 0, -1, -2, -3, -4, -5
DTYPES = {"f32": 0, "bf16": 1, "f8e4m3": 2}
DTYPE_NAMES = {v: k for k, v in DTYPES.items()}
DTYPE_BYTES = {"f32": 4, "bf16": 2, "f8e4m3": 1}
FAMILIES = {"dense": 0, "mixtral": 1, "moe_only": 2}
STYLES = {"fsdp_flat": 0, "megatron": 1, "serving": 2}
SENDER, RECEIVER = 0, 1


class WbError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libwb error {code}: {msg}")
        self.code = code


class ModelShapes(ctypes.Structure):
    _fields_ = [(n, c_int32) for n in ("family", "num_layers", "hidden", "num_heads", "num_kv_heads", "head_dim",
                                       "ffn", "vocab", "num_experts", "num_shared_experts")]


class Parallelism(ctypes.Structure):
    _fields_ = [(n, c_int32) for n in ("style", "dtype", "tp", "ep", "fsdp", "dp", "transposed_row_parallel",
                                       "quant_dtype", "quant_block")]


class Placement(ctypes.Structure):
    _fields_ = [("t", c_int32), ("u", c_int32), ("r0", c_int64), ("r1", c_int64), ("c0", c_int64), ("c1", c_int64),
                ("base", c_int64), ("ld", c_int64), ("transposed", c_int32), ("reserved", c_int32)]


class TensorDesc(ctypes.Structure):
    _fields_ = [("name", c_char_p), ("rows", c_int64), ("cols", c_int64)]


class SegmentInfo(ctypes.Structure):
    _fields_ = [(n, c_int32) for n in ("sender", "receiver", "tensor", "stage", "round", "src_placement",
                                       "dst_placement", "reserved")] + \
               [(n, c_int64) for n in ("r0", "r1", "c0", "c1", "send_offset", "recv_offset", "src_offset", "origin",
                                       "bytes")]


class Field(ctypes.Structure):
    _fields_ = [("data", c_void_p * 3), ("dtype", c_int32), ("passes", c_int32), ("rows", c_int64), ("cols", c_int64)]


class LocalInfo(ctypes.Structure):
    _fields_ = [("name", c_char_p), ("dtype", c_int32), ("quant_block", c_int32), ("batch", c_int64),
                ("rows", c_int64), ("cols", c_int64), ("scale_index", c_int32), ("scales_index", c_int32)]


def _load():
    # libwb.so and torch's HIP extension both need libamdhip64.so.7; whichever is
    # loaded first serves the whole process. Load torch's first so that the
    # tensors' runtime and the library's kernels share one HIP runtime.
    import torch  # noqa: F401

    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python paper_2609_25442_amd/build.py`")
    lib = ctypes.CDLL(LIB_PATH)
    P, L = c_void_p, c_void_p
    sig = {
        "wb_describe_layout": [POINTER(ModelShapes), POINTER(Parallelism), POINTER(L)],
        "wb_layout_create": [POINTER(TensorDesc), c_int32, c_int32, POINTER(L)],
        "wb_layout_add_local": [L, c_int32, c_char_p, c_int32, c_int64, c_int64, c_int64, c_int32, POINTER(c_int32)],
        "wb_layout_add_placement": [L, c_int32, POINTER(Placement)],
        "wb_layout_num_ranks": [L, POINTER(c_int32)],
        "wb_layout_num_tensors": [L, POINTER(c_int32)],
        "wb_layout_tensor": [L, c_int32, POINTER(TensorDesc)],
        "wb_layout_num_locals": [L, c_int32, POINTER(c_int32)],
        "wb_layout_local": [L, c_int32, c_int32, POINTER(LocalInfo)],
        "wb_layout_num_placements": [L, c_int32, POINTER(c_int32)],
        "wb_layout_placement": [L, c_int32, c_int32, POINTER(Placement)],
        "wb_layout_dump": [L, ctypes.c_char_p, c_size_t, POINTER(c_size_t)],
        "wb_plan": [L, L, c_int32, c_int32, POINTER(P)],
        "wb_plan_rounds": [L, L, c_int32, c_int32, c_int64, POINTER(P)],
        "wb_plan_num_rounds": [P, POINTER(c_int32)],
        "wb_plan_round_buffer_bytes": [P, c_int32, POINTER(c_int64)],
        "wb_plan_round_region": [P, c_int32, c_int32, c_int32, POINTER(c_int64), POINTER(c_int64), POINTER(c_int64)],
        "wb_pack_round": [P, c_int32, POINTER(c_void_p), c_void_p, c_void_p],
        "wb_unpack_round": [P, c_int32, c_void_p, POINTER(c_void_p), c_void_p],
        "wb_unpack_round_noalloc": [P, c_int32, c_void_p, POINTER(c_void_p), c_void_p],
        "wb_plan_num_segments": [P, POINTER(c_int64)],
        "wb_plan_buffer_bytes": [P, POINTER(c_int64)],
        "wb_plan_num_peers": [P, POINTER(c_int32)],
        "wb_plan_peer": [P, c_int32, POINTER(c_int32), POINTER(c_int64), POINTER(c_int64)],
        "wb_plan_region": [P, c_int32, c_int32, POINTER(c_int64), POINTER(c_int64), POINTER(c_int64)],
        "wb_plan_rank_buffer_bytes": [P, c_int32, c_int32, POINTER(c_int64)],
        "wb_plan_num_local_tensors": [P, POINTER(c_int32)],
        "wb_plan_workspace_bytes": [P, POINTER(c_int64)],
        "wb_plan_traffic_bytes": [P, POINTER(c_int64), POINTER(c_int64)],
        "wb_plan_work_counts": [P, POINTER(c_int64), POINTER(c_int64), POINTER(c_int64)],
        "wb_plan_work_digest": [P, POINTER(c_uint64)],
        "wb_plan_launch_grid": [P, c_int32, c_int32, POINTER(c_uint32), POINTER(c_uint32), POINTER(c_uint32)],
        "wb_plan_kernel_traffic": [P, c_int32, POINTER(c_int64), POINTER(c_int64)],
        "wb_plan_dump": [P, ctypes.c_char_p, c_size_t, POINTER(c_size_t)],
        "wb_plan_upload": [P, c_void_p, c_size_t, c_void_p],
        "wb_pack": [P, POINTER(c_void_p), c_void_p, c_void_p],
        "wb_unpack": [P, c_void_p, POINTER(c_void_p), c_void_p],
        "wb_plan_exchange": [L, L, c_int32, c_int32, c_int64, c_int32, POINTER(P)],
        "wb_plan_node_size": [P, POINTER(c_int32)],
        "wb_plan_stage_region": [P, c_int32, c_int32, c_int32, c_int32, POINTER(c_int64), POINTER(c_int64),
                                 POINTER(c_int64)],
        "wb_plan_forward_bytes": [P, c_int32, c_int32, POINTER(c_int64)],
        "wb_forward_round": [P, c_int32, c_int32, c_void_p, c_void_p, c_void_p],
        "wb_plan_segment": [P, c_int64, POINTER(SegmentInfo)],
        "wb_plan_local_tensor": [P, c_int32, POINTER(c_int32), POINTER(c_int64)],
        "wb_probe_create": [POINTER(TensorDesc), c_int32, c_int32, POINTER(c_void_p)],
        "wb_probe_chunks": [c_void_p, POINTER(c_int32), POINTER(c_int32)],
        "wb_probe_first_id": [c_void_p, c_int32, POINTER(c_int64)],
        "wb_probe_add_local": [c_void_p, c_char_p, c_int32, c_int64, c_int64, c_int64, POINTER(c_int32)],
        "wb_probe_record": [c_void_p, c_int32, c_int32, c_void_p, c_void_p, c_int64],
        "wb_probe_scan": [c_void_p, L, c_int32],
        "wb_make_ids": [c_void_p, c_int32, c_int64, c_int64, c_int32, c_int32, c_void_p],
        "wb_diff2": [c_void_p, c_int32, c_int64, c_int64, c_void_p, c_void_p, c_int64, c_void_p, c_void_p],
        "wb_diff2_batch_workspace": [POINTER(Field), c_int32, POINTER(c_size_t)],
        "wb_diff2_batch": [POINTER(Field), c_int32, c_void_p, c_size_t, c_void_p, c_void_p, c_int64, c_void_p,
                           c_void_p],
        "wb_diff2_carry_workspace": [POINTER(Field), c_int32, c_int64, POINTER(c_size_t)],
        "wb_diff2_carry": [POINTER(Field), c_int32, c_int32, c_int32, c_int64, c_void_p, c_size_t, c_void_p,
                           c_void_p, c_int64, c_void_p, c_void_p, c_void_p],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = c_int32
    lib.wb_layout_destroy.argtypes = [L]
    lib.wb_layout_destroy.restype = None
    lib.wb_plan_destroy.argtypes = [P]
    lib.wb_plan_destroy.restype = None
    lib.wb_probe_destroy.argtypes = [c_void_p]
    lib.wb_probe_destroy.restype = None
    lib.wb_last_error.restype = c_char_p
    lib.wb_version.restype = c_char_p
    return lib


lib = _load()


def _check(rc: int):
    if rc != WB_OK:
        raise WbError(rc, lib.wb_last_error().decode())


def _text(fn, handle) -> str:
    need = c_size_t(0)
    fn(handle, None, 0, byref(need))
    buf = ctypes.create_string_buffer(need.value)
    _check(fn(handle, buf, need.value, byref(need)))
    return buf.value.decode()


_live = weakref.WeakSet()


@atexit.register
def _release_all():
    # free what is still alive while the interpreter is intact
    for obj in list(_live):
        _release(obj)


def _release(obj):
    """Free a library object once; quiet when the interpreter is shutting down."""
    h, fn = getattr(obj, "_h", None), getattr(obj, "_destroy", None)
    if h is not None and h.value and callable(fn):
        try:
            fn(h)
        except Exception:
            pass
        obj._h = c_void_p()


def _stream_handle(stream) -> int | None:
    if stream is None:
        import torch

        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _ptr(x) -> int:
    return x if isinstance(x, int) else x.data_ptr()


# torch dtypes that hold each library dtype's codes (the value type, or an
# integer view of the same width)
_CODE_TYPES = {"f32": ("float32", "int32", "uint32"), "bf16": ("bfloat16", "int16", "uint16"),
               "f8e4m3": ("float8_e4m3fn", "uint8", "int8")}


def _einval(msg: str):
    raise WbError(WB_EINVAL, msg)


def _check_memory(x, what: str):
    """A tensor handed to a kernel: contiguous, on the GPU or in pinned host
    memory. Raw pointers (ints) are left to the library's own checks."""
    if isinstance(x, int) or x is None:
        return
    if not x.is_contiguous():
        _einval(f"{what} is not contiguous")
    if not (x.is_cuda or x.is_pinned()):
        _einval(f"{what} is neither device memory nor pinned host memory")


def _check_buffer(x, nbytes: int, what: str):
    _check_memory(x, what)
    if not isinstance(x, int) and x is not None and x.numel() * x.element_size() < nbytes:
        _einval(f"{what} is smaller than the plan needs ({x.numel() * x.element_size()} < {nbytes} bytes)")


class Layout:
    """All ranks of one side: a checkpoint catalog and per-rank local tensors
    and placements."""

    def __init__(self, handle: int):
        self._h = c_void_p(handle)
        self._destroy = lib.wb_layout_destroy
        _live.add(self)

    @classmethod
    def describe(cls, model: dict, par: dict) -> "Layout":
        m = ModelShapes(FAMILIES[model["family"]], model["num_layers"], model["hidden"], model.get("num_heads", 0),
                        model.get("num_kv_heads", 0), model.get("head_dim", 0), model.get("ffn", 0),
                        model.get("vocab", 0), model.get("num_experts", 0), model.get("num_shared_experts", 0))
        q = par.get("quant", "")
        p = Parallelism(STYLES[par["style"]], DTYPES[par["dtype"]], par.get("tp", 1), par.get("ep", 1),
                        par.get("fsdp", 1), par.get("dp", 1), int(bool(par.get("transposed_row_parallel", False))),
                        DTYPES[q] if q else -1, par.get("quant_block", 128) if q else 0)
        h = c_void_p()
        _check(lib.wb_describe_layout(byref(m), byref(p), byref(h)))
        return cls(h.value)

    @classmethod
    def create(cls, catalog, nranks: int) -> "Layout":
        """Empty generic layout over ``catalog`` = [(name, rows, cols), ...]."""
        arr = (TensorDesc * max(1, len(catalog)))()
        keep = []
        for i, (n, r, c) in enumerate(catalog):
            b = n.encode()
            keep.append(b)
            arr[i] = TensorDesc(b, r, c)
        h = c_void_p()
        _check(lib.wb_layout_create(arr, len(catalog), nranks, byref(h)))
        return cls(h.value)

    def add_local(self, rank, name, dtype, batch, rows, cols, quant_block=0) -> int:
        out = c_int32()
        _check(lib.wb_layout_add_local(self._h, rank, name.encode(), DTYPES[dtype], batch, rows, cols, quant_block,
                                       byref(out)))
        return out.value

    def add_placement(self, rank, t, r0, r1, c0, c1, u, base, ld, transposed=0):
        p = Placement(t, u, r0, r1, c0, c1, base, ld, transposed, 0)
        _check(lib.wb_layout_add_placement(self._h, rank, byref(p)))

    @property
    def nranks(self) -> int:
        n = c_int32()
        _check(lib.wb_layout_num_ranks(self._h, byref(n)))
        return n.value

    def tensors(self):
        n = c_int32()
        _check(lib.wb_layout_num_tensors(self._h, byref(n)))
        out = []
        for t in range(n.value):
            d = TensorDesc()
            _check(lib.wb_layout_tensor(self._h, t, byref(d)))
            out.append((d.name.decode(), d.rows, d.cols))
        return out

    def locals(self, rank: int):
        n = c_int32()
        _check(lib.wb_layout_num_locals(self._h, rank, byref(n)))
        out = []
        for u in range(n.value):
            i = LocalInfo()
            _check(lib.wb_layout_local(self._h, rank, u, byref(i)))
            out.append(dict(name=i.name.decode(), dtype=DTYPE_NAMES[i.dtype], block=i.quant_block, batch=i.batch,
                            rows=i.rows, cols=i.cols, scale=i.scale_index, scales=i.scales_index,
                            numel=i.batch * i.rows * i.cols))
        return out

    def placements(self, rank: int):
        n = c_int32()
        _check(lib.wb_layout_num_placements(self._h, rank, byref(n)))
        out = []
        for k in range(n.value):
            p = Placement()
            _check(lib.wb_layout_placement(self._h, rank, k, byref(p)))
            out.append((p.t, p.r0, p.r1, p.c0, p.c1, p.u, p.base, p.ld, p.transposed))
        return out

    def dump(self) -> str:
        return _text(lib.wb_layout_dump, self._h)

    def __del__(self):
        # at interpreter teardown the module's globals may already be gone
        if getattr(self, "_h", None) is not None and self._h.value and _release is not None:
            _release(self)


class Plan:
    """The global routing plan seen from one rank (a sender or a receiver)."""

    def __init__(self, trainer: Layout, rollout: Layout, role: int, rank: int, round_budget: int = 0,
                 node_size: int = 0):
        h = c_void_p()
        _check(lib.wb_plan_exchange(trainer._h, rollout._h, role, rank, round_budget, node_size, byref(h)))
        self._h = h
        self._destroy = lib.wb_plan_destroy
        _live.add(self)
        self.role, self.rank = role, rank
        self._workspace = None
        self._locals = None

    def _i64(self, fn):
        v = c_int64()
        _check(fn(self._h, byref(v)))
        return v.value

    @property
    def num_segments(self) -> int:
        return self._i64(lib.wb_plan_num_segments)

    @property
    def buffer_bytes(self) -> int:
        return self._i64(lib.wb_plan_buffer_bytes)

    @property
    def workspace_bytes(self) -> int:
        return self._i64(lib.wb_plan_workspace_bytes)

    @property
    def num_local_tensors(self) -> int:
        v = c_int32()
        _check(lib.wb_plan_num_local_tensors(self._h, byref(v)))
        return v.value

    def local_tensor(self, i: int):
        """(dtype name, element count) of pointer-table entry i."""
        dt, n = c_int32(), c_int64()
        _check(lib.wb_plan_local_tensor(self._h, i, byref(dt), byref(n)))
        return DTYPE_NAMES[dt.value], n.value

    @property
    def num_rounds(self) -> int:
        v = c_int32()
        _check(lib.wb_plan_num_rounds(self._h, byref(v)))
        return v.value

    def round_buffer_bytes(self, rnd: int) -> int:
        v = c_int64()
        _check(lib.wb_plan_round_buffer_bytes(self._h, rnd, byref(v)))
        return v.value

    def round_region(self, rnd: int, sender: int, receiver: int):
        s, r, b = c_int64(), c_int64(), c_int64()
        _check(lib.wb_plan_round_region(self._h, rnd, sender, receiver, byref(s), byref(r), byref(b)))
        return s.value, r.value, b.value

    def _check_locals(self, xs, what: str):
        """The pointer table of a pack or unpack: one tensor (or raw pointer)
        per local tensor of the rank, each of the plan's dtype and size."""
        if self._locals is None:
            self._locals = [self.local_tensor(i) for i in range(self.num_local_tensors)]
        if len(xs) != len(self._locals):
            _einval(f"{what}: {len(xs)} tensors given, the plan's rank has {len(self._locals)} local tensors")
        for i, (x, (dt, numel)) in enumerate(zip(xs, self._locals)):
            if isinstance(x, int) or x is None:
                continue
            name = str(x.dtype).replace("torch.", "")
            if name not in _CODE_TYPES[dt]:
                _einval(f"{what} {i} has dtype {name}; the plan's local tensor is {dt}")
            if x.numel() != numel:
                _einval(f"{what} {i} has {x.numel()} elements: "
                        f"{'smaller' if x.numel() < numel else 'larger'} than the plan's {numel}")
            _check_memory(x, f"{what} {i}")

    def pack_round(self, rnd, src, send_buf, stream=None):
        self._check_locals(src, "local tensor")
        _check_buffer(send_buf, self.round_buffer_bytes(rnd), "send_buf")
        ptrs = (c_void_p * max(1, len(src)))(*[_ptr(x) for x in src])
        _check(lib.wb_pack_round(self._h, rnd, ptrs, _ptr(send_buf), _stream_handle(stream)))

    def unpack_round(self, rnd, recv_buf, dst, stream=None):
        self._check_locals(dst, "local tensor")
        _check_buffer(recv_buf, self.round_buffer_bytes(rnd), "recv_buf")
        ptrs = (c_void_p * max(1, len(dst)))(*[_ptr(x) for x in dst])
        _check(lib.wb_unpack_round(self._h, rnd, _ptr(recv_buf), ptrs, _stream_handle(stream)))

    def unpack_round_noalloc(self, rnd, recv_buf, dst, stream=None):
        """unpack_round without a workspace or upload: the library stages the
        round's tables in its own per-GPU device array (calls that overlap on
        one GPU race; a round whose tables exceed the array raises WB_ESIZE)."""
        self._check_locals(dst, "local tensor")
        _check_buffer(recv_buf, self.round_buffer_bytes(rnd), "recv_buf")
        ptrs = (c_void_p * max(1, len(dst)))(*[_ptr(x) for x in dst])
        _check(lib.wb_unpack_round_noalloc(self._h, rnd, _ptr(recv_buf), ptrs, _stream_handle(stream)))

    @property
    def node_size(self) -> int:
        v = c_int32()
        _check(lib.wb_plan_node_size(self._h, byref(v)))
        return v.value

    def stage_region(self, rnd: int, stage: int, sender: int, receiver: int):
        """(offset in the sender's send or forward buffer, offset in the
        receiver's receive buffer, bytes) of one stage of one round."""
        s, r, b = c_int64(), c_int64(), c_int64()
        _check(lib.wb_plan_stage_region(self._h, rnd, stage, sender, receiver, byref(s), byref(r), byref(b)))
        return s.value, r.value, b.value

    def segments(self):
        """Every segment of the global plan as a dict (the order of dump())."""
        out = []
        for i in range(self.num_segments):
            g = SegmentInfo()
            _check(lib.wb_plan_segment(self._h, i, byref(g)))
            out.append({f: getattr(g, f) for f, _ in SegmentInfo._fields_ if f != "reserved"})
        return out

    def forward_bytes(self, stage: int, rnd: int = -1) -> int:
        v = c_int64()
        _check(lib.wb_plan_forward_bytes(self._h, rnd, stage, byref(v)))
        return v.value

    def forward_round(self, rnd, stage, recv_buf, fwd_buf, stream=None):
        _check_buffer(recv_buf, self.round_buffer_bytes(rnd), "recv_buf")
        _check_buffer(fwd_buf, self.forward_bytes(stage, rnd), "fwd_buf")
        _check(lib.wb_forward_round(self._h, rnd, stage, _ptr(recv_buf), _ptr(fwd_buf) if fwd_buf is not None else 0,
                                    _stream_handle(stream)))

    def rank_buffer_bytes(self, role: int, rank: int) -> int:
        v = c_int64()
        _check(lib.wb_plan_rank_buffer_bytes(self._h, role, rank, byref(v)))
        return v.value

    def peers(self):
        """[(peer rank, offset, bytes)] of the regions in this rank's buffer."""
        n = c_int32()
        _check(lib.wb_plan_num_peers(self._h, byref(n)))
        out = []
        for i in range(n.value):
            p, o, b = c_int32(), c_int64(), c_int64()
            _check(lib.wb_plan_peer(self._h, i, byref(p), byref(o), byref(b)))
            out.append((p.value, o.value, b.value))
        return out

    def region(self, sender: int, receiver: int):
        """(offset in the sender's buffer, offset in the receiver's buffer, bytes)."""
        s, r, b = c_int64(), c_int64(), c_int64()
        _check(lib.wb_plan_region(self._h, sender, receiver, byref(s), byref(r), byref(b)))
        return s.value, r.value, b.value

    def traffic(self):
        r, w = c_int64(), c_int64()
        _check(lib.wb_plan_traffic_bytes(self._h, byref(r), byref(w)))
        return r.value, w.value

    def kernel_traffic(self, launch: int):
        """(read, write) algorithmic bytes of launch 0 (copy/cast), 1 (fp8 blocks),
        2 or 3 (forward packing of exchange stage 1 or 2)."""
        r, w = c_int64(), c_int64()
        _check(lib.wb_plan_kernel_traffic(self._h, launch, byref(r), byref(w)))
        return r.value, w.value

    def work_counts(self):
        a, b, c = c_int64(), c_int64(), c_int64()
        _check(lib.wb_plan_work_counts(self._h, byref(a), byref(b), byref(c)))
        return a.value, b.value, c.value

    def work_digest(self) -> int:
        """64-bit digest of the kernel work tables (equal digests, same work)."""
        v = c_uint64()
        _check(lib.wb_plan_work_digest(self._h, byref(v)))
        return v.value

    def launch_grid(self, launch=0, round=0):
        """(workgroups in x, in y, threads per workgroup) of one launch of one
        round: 0 copy/cast, 1 fp8 blocks, 2 and 3 the forward packings of
        exchange stages 1 and 2."""
        x, y, t = c_uint32(), c_uint32(), c_uint32()
        _check(lib.wb_plan_launch_grid(self._h, launch, round, byref(x), byref(y), byref(t)))
        return x.value, y.value, t.value

    def dump(self) -> str:
        return _text(lib.wb_plan_dump, self._h)

    def upload(self, workspace, stream=None):
        """Copy the work tables into ``workspace`` (a device tensor or pointer of
        at least ``workspace_bytes`` bytes); the plan keeps a reference to it."""
        _check_memory(workspace, "workspace")
        nbytes = workspace.numel() * workspace.element_size() if hasattr(workspace, "numel") else self.workspace_bytes
        _check(lib.wb_plan_upload(self._h, _ptr(workspace), nbytes, _stream_handle(stream)))
        self._workspace = workspace

    def pack(self, src, send_buf, stream=None):
        self._check_locals(src, "local tensor")
        _check_buffer(send_buf, self.buffer_bytes, "send_buf")
        ptrs = (c_void_p * max(1, len(src)))(*[_ptr(x) for x in src])
        _check(lib.wb_pack(self._h, ptrs, _ptr(send_buf), _stream_handle(stream)))

    def unpack(self, recv_buf, dst, stream=None):
        self._check_locals(dst, "local tensor")
        _check_buffer(recv_buf, self.buffer_bytes, "recv_buf")
        ptrs = (c_void_p * max(1, len(dst)))(*[_ptr(x) for x in dst])
        _check(lib.wb_unpack(self._h, _ptr(recv_buf), ptrs, _stream_handle(stream)))

    def __del__(self):
        # at interpreter teardown the module's globals may already be gone
        if getattr(self, "_h", None) is not None and self._h.value and _release is not None:
            _release(self)


class Probe:
    """Source-map probing of one rank (Sec. 3.1; App. B, Algorithm 1): identifier
    chunks are written into a checkpoint, a weight loader copies them into the
    rank's tensors, diff2 entries of every pass are recorded and scanned back
    into placements."""

    def __init__(self, catalog, ckpt_dtype: str):
        arr = (TensorDesc * len(catalog))()
        self._names = []
        for i, (n, r, c) in enumerate(catalog):
            b = n.encode()
            self._names.append(b)
            arr[i] = TensorDesc(b, r, c)
        h = c_void_p()
        _check(lib.wb_probe_create(arr, len(catalog), DTYPES[ckpt_dtype], byref(h)))
        self._h = h
        self._destroy = lib.wb_probe_destroy
        _live.add(self)
        self.catalog = list(catalog)
        self.dtype = ckpt_dtype
        n, b = c_int32(), c_int32()
        _check(lib.wb_probe_chunks(self._h, byref(n), byref(b)))
        self.num_chunks, self.chunk_bits = n.value, b.value

    def first_id(self, t: int) -> int:
        v = c_int64()
        _check(lib.wb_probe_first_id(self._h, t, byref(v)))
        return v.value

    def add_local(self, name, dtype, batch, rows, cols) -> int:
        v = c_int32()
        _check(lib.wb_probe_add_local(self._h, name.encode(), DTYPES[dtype], batch, rows, cols, byref(v)))
        return v.value

    def record(self, local: int, chunk: int, index, value):
        """index and value host arrays (numpy, taken as int64) of one pass, or
        of all passes at once as chunk 0."""
        import numpy as np

        index = np.ascontiguousarray(index, dtype=np.int64)
        value = np.ascontiguousarray(value, dtype=np.int64)
        _check(lib.wb_probe_record(self._h, local, chunk, index.ctypes.data, value.ctypes.data, len(index)))

    def scan(self, layout: "Layout", rank: int):
        _check(lib.wb_probe_scan(self._h, layout._h, rank))

    def __del__(self):
        # at interpreter teardown the module's globals may already be gone
        if getattr(self, "_h", None) is not None and self._h.value and _release is not None:
            _release(self)


def make_ids(dst, dtype: str, first_id: int, chunk: int, stream=None):
    """Write identifier chunk ``chunk`` of first_id, first_id + 1, ... into the
    tensor ``dst`` (every element, in storage order)."""
    _check(lib.wb_make_ids(_ptr(dst), DTYPES[dtype], dst.numel(), first_id, chunk, 16, _stream_handle(stream)))


def diff2(src, dtype: str, rows: int, cols: int, index, value, count, stream=None):
    """Non-zero diff2 entries of a [rows, cols] chunk field into the device
    tensors index (int64), value (int32); count (uint64 device scalar) gets
    their number (which may exceed the arrays' length)."""
    _check(lib.wb_diff2(_ptr(src), DTYPES[dtype], rows, cols, _ptr(index), _ptr(value), index.numel(), _ptr(count),
                        _stream_handle(stream)))


def _field_array(fields):
    """ctypes wb_field array of (tensors, dtype, rows, cols) tuples; an array
    built here before is passed through."""
    if isinstance(fields, ctypes.Array):
        return fields
    arr = (Field * len(fields))()
    for f, (ts, dtype, rows, cols) in enumerate(fields):
        ts = list(ts) if isinstance(ts, (list, tuple)) else [ts]
        if not 1 <= len(ts) <= 3:
            raise ValueError("a field holds 1 to 3 passes")
        arr[f].dtype, arr[f].passes, arr[f].rows, arr[f].cols = DTYPES[dtype], len(ts), rows, cols
        for c, t in enumerate(ts):
            arr[f].data[c] = _ptr(t)
    return arr


def diff2_batch_workspace(fields) -> int:
    """Device workspace bytes of diff2_batch over ``fields``."""
    arr = _field_array(fields)
    v = c_size_t()
    _check(lib.wb_diff2_batch_workspace(arr, len(fields), byref(v)))
    return v.value


def diff2_batch(fields, index, value, count, workspace, stream=None):
    """Non-zero diff2 entries of many fields in one launch. ``fields`` is a list
    of (tensors, dtype, rows, cols); ``tensors`` is one tensor or the list of
    one loaded tensor per probing pass (value sum of 2^(16 k) times pass k).
    Entries go to the device tensors index (int64, position in the
    concatenation of the fields) and value (int64); count (uint64 device
    scalar) gets their number. ``workspace``: a uint8 device tensor of at least
    diff2_batch_workspace(fields) bytes."""
    arr = _field_array(fields)
    nbytes = workspace.numel() if workspace is not None else 0
    _check(lib.wb_diff2_batch(arr, len(fields), _ptr(workspace) if nbytes else None, nbytes, _ptr(index),
                              _ptr(value), index.numel(), _ptr(count), _stream_handle(stream)))


def diff2_carry_workspace(fields, carry_capacity: int) -> int:
    """Device workspace bytes of diff2_carry over one-pass ``fields`` with
    room for ``carry_capacity`` carries per pass."""
    arr = _field_array(fields)
    v = c_size_t()
    _check(lib.wb_diff2_carry_workspace(arr, len(fields), carry_capacity, byref(v)))
    return v.value


def diff2_carry(fields, pass_: int, last: bool, carry_capacity: int, index, value, count, carries, workspace,
                stream=None):
    """One probing pass with carries kept on the device (App. B): entries
    of pass ``pass_`` (values in 1..65535 except in the last pass) into the
    device tensors index and value (int64); count and carries (uint64 device
    scalars) get the number of entries and of carries kept for the next
    pass. ``fields`` as for diff2_batch with one tensor each; ``workspace``
    (uint8, diff2_carry_workspace bytes) is the same tensor every pass."""
    arr = _field_array(fields)
    _check(lib.wb_diff2_carry(arr, len(fields), pass_, int(bool(last)), carry_capacity, _ptr(workspace),
                              workspace.numel(), _ptr(index), _ptr(value), index.numel(), _ptr(count), _ptr(carries),
                              _stream_handle(stream)))


def _view_shape(t):
    if t.dim() == 1:
        return 1, 1, t.shape[0]
    if t.dim() == 2:
        return 1, t.shape[0], t.shape[1]
    if t.dim() == 3:
        return t.shape[0], t.shape[1], t.shape[2]
    raise ValueError("local tensors must be 1-, 2- or 3-D")


def _batched_entries(fields, cap, device):
    """Run diff2_batch over ``fields``, growing the entry arrays until they
    hold every entry; returns host (index, value) arrays."""
    import torch

    count = torch.zeros(1, dtype=torch.int64, device=device)
    ws = torch.empty(max(diff2_batch_workspace(fields), 8), dtype=torch.uint8, device=device)
    while True:
        idx = torch.empty(cap, dtype=torch.int64, device=device)
        val = torch.empty(cap, dtype=torch.int64, device=device)
        diff2_batch(fields, idx, val, count, ws)
        n = int(count.item())
        if n <= cap:
            return idx[:n].cpu().numpy(), val[:n].cpu().numpy()
        cap = n


class _CarryRoom(Exception):
    """A carry pass kept more carries than its tables hold."""

    def __init__(self, need):
        super().__init__(need)
        self.need = need


def _carry_entries(fields, k, last, st, device):
    """Run carry pass k, growing the entry arrays until they hold every entry
    (a pass can be run again on the same workspace); returns host (index,
    value) arrays and the number of carries kept."""
    import torch

    while True:
        diff2_carry(fields, k, last, st["cap"], st["idx"], st["val"], st["count"], st["carries"], st["ws"])
        n, c = int(st["count"].item()), int(st["carries"].item())
        if c > st["cap"]:
            raise _CarryRoom(c)
        if n <= st["idx"].numel():
            return st["idx"][:n].cpu().numpy(), st["val"][:n].cpu().numpy(), c
        st["idx"] = torch.empty(n, dtype=torch.int64, device=device)
        st["val"] = torch.empty(n, dtype=torch.int64, device=device)


def _record_split(probe, chunk, offsets, index, value):
    """Hand batched entries to the probe, local tensor by local tensor."""
    import numpy as np

    order = np.argsort(index, kind="stable")
    index, value = index[order], value[order]
    cut = np.searchsorted(index, offsets)
    for u in range(len(offsets) - 1):
        a, b = cut[u], cut[u + 1]
        probe.record(u, chunk, index[a:b] - offsets[u], value[a:b])


def probe_layout(catalog, ckpt_dtype: str, loaders, names=None, device="cuda", stats=None,
                 hold_passes=False, carry_capacity=None) -> "Layout":
    """Discover a layout from weight loaders: ``loaders[r](ckpt)`` takes the
    checkpoint as {name: tensor} and returns rank r's local tensors (a list of
    1-, 2- or 3-D tensors, always the same shapes, values copied unchanged).
    Returns a Layout with one rank per loader.

    Every pass runs diff2_carry as soon as it is loaded: each pass hands the
    host only the entries next to slice-copy corners and keeps its
    wrap-arounds as device carries for the next pass (``carry_capacity``
    carries per pass, by default about 16 per 2^16 elements; a rank whose
    passes need more is probed again with room for what they needed). With
    ``hold_passes`` a copy of every pass's loaded tensors stays in device
    memory instead and one diff2 launch over all passes runs at the end (the
    chunk wrap-arounds cancel inside it); None holds them when they fit in
    free device memory with a quarter to spare. ``stats`` (a dict) receives
    timings and entry counts when given."""
    tdt = torch_dtype(ckpt_dtype)
    layout = Layout.create(catalog, len(loaders))
    ckpt = _IdCheckpoint(catalog, ckpt_dtype, tdt, device)
    for r, load in enumerate(loaders):
        cap = carry_capacity
        while True:
            try:
                probe, hold = _probe_rank(catalog, ckpt_dtype, tdt, load, r, names, device, stats, hold_passes, cap,
                                          ckpt)
                break
            except _CarryRoom as room:
                cap = room.need + room.need // 4 + 4096
                if stats is not None:
                    stats.setdefault("carry_retries", []).append(cap)
        t4 = _now()
        probe.scan(layout, r)
        if stats is not None:
            stats.setdefault("scan_s", []).append(_now() - t4)
            stats.setdefault("hold_passes", []).append(bool(hold))
        del probe
    return layout


def _now():
    import time

    return time.perf_counter()


class _IdCheckpoint(collections.abc.Mapping):
    """The identifier checkpoint a loader reads, {name: tensor}, made on
    demand: a tensor is allocated the first time any pass reads it and filled
    with the current pass's chunk of its identifiers the first time that pass
    reads it. Tensors no loader reads are never made, so a rank of a checkpoint
    larger than the GPU (a DeepSeek-V3 expert-parallel rank) is probed with
    device memory for its own tensors only."""

    def __init__(self, catalog, ckpt_dtype, tdt, device):
        self._cat = {n: (t, rows, cols) for t, (n, rows, cols) in enumerate(catalog)}
        self._dtype, self._tdt, self._device = ckpt_dtype, tdt, device
        self._tensors, self._filled = {}, set()
        self._probe, self._k = None, 0
        self.ids_s = 0.0

    def start_pass(self, probe, k):
        self._probe, self._k = probe, k
        self._filled.clear()
        self.ids_s = 0.0

    def __getitem__(self, name):
        import torch

        t, rows, cols = self._cat[name]
        x = self._tensors.get(name)
        if x is None:
            x = self._tensors[name] = torch.empty((rows, cols), dtype=self._tdt, device=self._device)
        if name not in self._filled:
            t0 = _now()
            make_ids(x, self._dtype, self._probe.first_id(t), self._k)
            self.ids_s += _now() - t0
            self._filled.add(name)
        return x

    def __contains__(self, name):  # a membership test makes nothing
        return name in self._cat

    def __iter__(self):
        return iter(self._cat)

    def __len__(self):
        return len(self._cat)


def _probe_rank(catalog, ckpt_dtype, tdt, load, r, names, device, stats, hold_passes, carry_capacity, ckpt):
    """Probe one rank; returns the filled Probe and whether passes were held."""
    import numpy as np
    import torch

    probe = Probe(catalog, ckpt_dtype)
    shapes, held, hold, carry = None, [], hold_passes, None
    rec = stats.setdefault(r, []) if stats is not None else None
    if rec is not None:
        rec.clear()
    for k in range(probe.num_chunks):
        last = k + 1 == probe.num_chunks
        ckpt.start_pass(probe, k)
        t1 = _now()
        locs = load(ckpt)
        torch.cuda.synchronize()
        t2 = _now()
        if shapes is None:
            shapes = [_view_shape(x) for x in locs]
            for u, (b, rr, cc) in enumerate(shapes):
                probe.add_local(names[r][u] if names else f"local{u}", ckpt_dtype, b, rr, cc)
            offsets = np.cumsum([0] + [b * rr * cc for b, rr, cc in shapes]).astype(np.int64)
            if hold is None:
                need = (probe.num_chunks - 1) * sum(x.numel() * x.element_size() for x in locs)
                hold = need * 4 <= torch.cuda.mem_get_info()[0] * 3
        for u, x in enumerate(locs):
            if x.dtype != tdt or not x.is_contiguous() or _view_shape(x) != shapes[u]:
                raise ValueError(f"loader of rank {r} returned a changed or non-contiguous tensor {u}")
        entries, carries = 0, 0
        if hold:
            # a loader may write into the same buffers every pass, or hand
            # back checkpoint tensors, which the next pass overwrites
            held.append([x.clone() for x in locs] if not last else locs)
        else:
            fields = [(x, ckpt_dtype, b * rr, cc) for x, (b, rr, cc) in zip(locs, shapes)]
            if carry is None:
                cap = carry_capacity or 16 * (int(offsets[-1]) >> 16) + 64 * len(fields) + 4096
                nbytes = diff2_carry_workspace(fields, cap)
                carry = {"cap": cap, "ws": torch.empty(nbytes, dtype=torch.uint8, device=device),
                         "idx": torch.empty(1 << 16, dtype=torch.int64, device=device),
                         "val": torch.empty(1 << 16, dtype=torch.int64, device=device),
                         "count": torch.zeros(1, dtype=torch.int64, device=device),
                         "carries": torch.zeros(1, dtype=torch.int64, device=device)}
            idx, val, carries = _carry_entries(fields, k, last, carry, device)
            _record_split(probe, k, offsets, idx, val)
            entries = len(idx)
        del locs
        t3 = _now()
        if rec is not None:
            rec.append({"pass": k, "ids_s": ckpt.ids_s, "load_s": t2 - t1 - ckpt.ids_s, "diff2_s": t3 - t2,
                        "entries": entries, "carries": carries})
    if hold:
        t2 = _now()
        fields = [([held[k][u] for k in range(probe.num_chunks)], ckpt_dtype, b * rr, cc)
                  for u, (b, rr, cc) in enumerate(shapes)]
        idx, val = _batched_entries(fields, 1 << 16, device)
        _record_split(probe, 0, offsets, idx, val)
        del fields, held
        if rec is not None:
            rec.append({"pass": "all", "diff2_s": _now() - t2, "entries": len(idx)})
    return probe, hold


def version() -> str:
    return lib.wb_version().decode()


def torch_dtype(name: str):
    import torch

    return {"f32": torch.float32, "bf16": torch.bfloat16, "f8e4m3": torch.float8_e4m3fn}[name]


def allocate_locals(layout: Layout, rank: int, device="cuda", zero=False):
    """Torch tensors for every local tensor of ``rank`` (shape [batch, rows, cols]
    squeezed as the layout gives it)."""
    import torch

    out = []
    for lc in layout.locals(rank):
        shape = (lc["batch"], lc["rows"], lc["cols"]) if lc["batch"] > 1 else (lc["rows"], lc["cols"])
        mk = torch.zeros if zero else torch.empty
        out.append(mk(shape, dtype=torch_dtype(lc["dtype"]), device=device))
    return out
