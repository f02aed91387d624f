"""ctypes binding of librbs.so (the C ABI in include/rbs.h).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  PyTorch provides device memory and the current stream.  The binding
refuses to run when the library is not built; there is no CPU fallback.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# RBS_LIB_PATH points the binding at another build of the same library (for
# comparing builds); the default is the in-tree one.
LIB_PATH = os.environ.get("RBS_LIB_PATH") or os.path.join(_HERE, "librbs.so")

RBS_OK, RBS_ERR_NULL, RBS_ERR_SHAPE, RBS_ERR_UNSUPPORTED, RBS_ERR_ARG, RBS_ERR_ALIGN, RBS_ERR_HIP, RBS_ERR_RANGE = range(8)


class RbsError(RuntimeError):
    def __init__(self, fn: str, status: int, message: str):
        super().__init__(f"{fn} failed with status {status}: {message}")
        self.status = status


class rbs_shape(ctypes.Structure):
    _fields_ = [
        ("n_tokens", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("q_stride_head", ctypes.c_int64),
        ("q_stride_tok", ctypes.c_int64),
        ("kv_stride_head", ctypes.c_int64),
        ("kv_stride_tok", ctypes.c_int64),
    ]


class rbs_stats(ctypes.Structure):
    _fields_ = [
        ("centroids", ctypes.c_void_p),
        ("radii", ctypes.c_void_p),
        ("beta", ctypes.c_void_p),
        ("quantiles", ctypes.c_void_p),
        ("summary", ctypes.c_void_p),
    ]


class rbs_box(ctypes.Structure):
    _fields_ = [
        ("center", ctypes.c_void_p),
        ("half", ctypes.c_void_p),
        ("summary", ctypes.c_void_p),
    ]


class rbs_batch(ctypes.Structure):
    _fields_ = [
        ("n_seqs", ctypes.c_int32),
        ("seq_tokens", ctypes.POINTER(ctypes.c_int32)),
    ]


RBS_MAX_SEQS = 64
RBS_SELECTOR_CENTROID, RBS_SELECTOR_FULL_L2, RBS_SELECTOR_BOX = 1, 2, 3
SELECTORS = {"centroid": RBS_SELECTOR_CENTROID, "full_l2": RBS_SELECTOR_FULL_L2, "box": RBS_SELECTOR_BOX}

_lib = None


def load() -> ctypes.CDLL:
    """Load librbs.so once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_20971_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, F32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_int64, ctypes.c_size_t
    SP = ctypes.POINTER(rbs_shape)
    lib.rbs_summary_bytes.argtypes = [SP]
    lib.rbs_summary_bytes.restype = SZ
    lib.rbs_index_capacity.argtypes = [I32]
    lib.rbs_index_capacity.restype = I64
    lib.rbs_block_stats.argtypes = [SP, P, ctypes.POINTER(rbs_stats), P]
    lib.rbs_block_stats.restype = ctypes.c_int
    lib.rbs_stats_summarize.argtypes = [SP, ctypes.POINTER(rbs_stats), P]
    lib.rbs_stats_summarize.restype = ctypes.c_int
    lib.rbs_select.argtypes = [SP, P, ctypes.POINTER(rbs_stats), F32, F32, I32, I32, I32, P, P, P]
    lib.rbs_select.restype = ctypes.c_int
    lib.rbs_attention_workspace_bytes.argtypes = []
    lib.rbs_attention_workspace_bytes.restype = SZ
    lib.rbs_sparse_prefill.argtypes = [SP, P, P, P, P, P, F32, P, P, P, P]
    lib.rbs_sparse_prefill.restype = ctypes.c_int
    lib.rbs_sparse_prefill_noalloc.argtypes = [SP, P, P, P, P, P, F32, P, P, P]
    lib.rbs_sparse_prefill_noalloc.restype = ctypes.c_int
    lib.rbs_select_attend.argtypes = [SP, P, P, P, ctypes.POINTER(rbs_stats), F32, F32, I32, I32, I32, F32, P, P, P,
                                      P, P, P]
    lib.rbs_select_attend.restype = ctypes.c_int
    lib.rbs_box_summary_bytes.argtypes = [SP]
    lib.rbs_box_summary_bytes.restype = SZ
    lib.rbs_block_box.argtypes = [SP, P, ctypes.POINTER(rbs_box), P]
    lib.rbs_block_box.restype = ctypes.c_int
    lib.rbs_select_variant.argtypes = [SP, P, ctypes.POINTER(rbs_stats), ctypes.POINTER(rbs_box), I32, F32, I32,
                                       I32, I32, P, P, P]
    lib.rbs_select_variant.restype = ctypes.c_int
    lib.rbs_dense_indices.argtypes = [SP, P, P, P]
    lib.rbs_dense_indices.restype = ctypes.c_int
    lib.rbs_fp8_vt_bytes.argtypes = [SP]
    lib.rbs_fp8_vt_bytes.restype = SZ
    lib.rbs_fp8_amax.argtypes = [SP, P, P, P, P, P]
    lib.rbs_fp8_amax.restype = ctypes.c_int
    lib.rbs_fp8_pack.argtypes = [SP, P, P, P, P, P, P, P, P]
    lib.rbs_fp8_pack.restype = ctypes.c_int
    lib.rbs_sparse_prefill_fp8.argtypes = [SP, P, P, P, P, P, P, F32, P, P, P, P]
    lib.rbs_sparse_prefill_fp8.restype = ctypes.c_int
    BP = ctypes.POINTER(rbs_batch)
    lib.rbs_varlen_blocks.argtypes = [SP, BP]
    lib.rbs_varlen_blocks.restype = I32
    lib.rbs_varlen_index_capacity.argtypes = [SP, BP]
    lib.rbs_varlen_index_capacity.restype = I64
    lib.rbs_varlen_summary_bytes.argtypes = [SP, BP]
    lib.rbs_varlen_summary_bytes.restype = SZ
    lib.rbs_block_stats_varlen.argtypes = [SP, BP, P, ctypes.POINTER(rbs_stats), P]
    lib.rbs_block_stats_varlen.restype = ctypes.c_int
    lib.rbs_select_varlen.argtypes = [SP, BP, P, ctypes.POINTER(rbs_stats), F32, F32, I32, I32, I32, P, P, P]
    lib.rbs_select_varlen.restype = ctypes.c_int
    lib.rbs_sparse_prefill_varlen.argtypes = [SP, BP, P, P, P, P, P, F32, P, P, P, P]
    lib.rbs_sparse_prefill_varlen.restype = ctypes.c_int
    lib.rbs_dense_indices_varlen.argtypes = [SP, BP, P, P, P]
    lib.rbs_dense_indices_varlen.restype = ctypes.c_int
    lib.rbs_status_str.argtypes = [ctypes.c_int]
    lib.rbs_status_str.restype = ctypes.c_char_p
    lib.rbs_set_debug.argtypes = [ctypes.c_int]
    lib.rbs_set_debug.restype = ctypes.c_int
    _lib = lib
    return lib


def rbs_status_str(status: int) -> str:
    return load().rbs_status_str(status).decode()


def rbs_set_debug(on: bool) -> bool:
    """Debug mode on or off (process-wide); returns the previous setting.  In
    debug mode every call drains its stream and reports kernel failures, and
    the selection calls reject a Q the selector's f16 operands cannot hold
    (RBS_ERR_RANGE) before launching anything else."""
    return bool(load().rbs_set_debug(1 if on else 0))


def _check(fn: str, status: int):
    if status != RBS_OK:
        raise RbsError(fn, status, rbs_status_str(status))


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


# Attention workspace argument: AUTO takes one cached per (device, stream) --
# calls on one stream are ordered, so they may share it (a stream handle that
# is destroyed and handed out again while work is pending would share it
# with that work; torch's pooled streams are never destroyed) --; None asks
# for the one-workgroup-per-item launch; a device tensor of at least
# rbs_attention_workspace_bytes() bytes is used as given.  Its contents do not
# matter: every call resets the queues on its own stream.
AUTO = "auto"
_workspaces: dict = {}


def attention_workspace(device, stream=None) -> torch.Tensor:
    device = torch.device(device)
    index = device.index if device.index is not None else torch.cuda.current_device()
    key = (index, _stream(stream))
    ws = _workspaces.get(key)
    if ws is None:
        n = int(load().rbs_attention_workspace_bytes())
        ws = torch.empty(n // 4, dtype=torch.int32, device=torch.device("cuda", index))
        _workspaces[key] = ws
    return ws


def _workspace(workspace, device, stream):
    if isinstance(workspace, str):
        if workspace != AUTO:
            raise ValueError(f"workspace must be AUTO, None or a tensor, not {workspace!r}")
        return attention_workspace(device, stream)
    if workspace is None:
        return None
    if workspace.numel() * workspace.element_size() < load().rbs_attention_workspace_bytes():
        raise ValueError("workspace is smaller than rbs_attention_workspace_bytes()")
    dev = torch.device(device)
    if dev.type == "cuda":
        index = dev.index if dev.index is not None else torch.cuda.current_device()
        if workspace.device.type != "cuda" or workspace.device.index != index:
            raise ValueError(f"workspace is on {workspace.device}, the inputs on cuda:{index}")
    return workspace


def make_shape(n_tokens: int, n_q_heads: int, n_kv_heads: int, block_size: int, head_dim: int = 128) -> rbs_shape:
    """Shape with zero (dense) strides; the calls fill the strides in from the
    tensors they are given."""
    return rbs_shape(n_tokens, n_q_heads, n_kv_heads, head_dim, block_size, 0, 0, 0, 0)


# ------------------------------------------------------------------ argument checks
# Every call checks its tensors here, before anything reaches the library:
# dtype, sizes and layout of each tensor first, then that all of them sit on
# one GPU.  Q/K/V/O strides go into the rbs_shape passed on.  A mismatch
# raises ValueError; nothing is launched.

def _device_index(t) -> int:
    if t.device.type != "cuda":
        return -1
    return t.device.index if t.device.index is not None else torch.cuda.current_device()


def _check_tensor(name: str, t, dtype, sizes, contiguous=True):
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch.Tensor, not {type(t).__name__}")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, not {t.dtype}")
    if tuple(t.shape) != tuple(sizes):
        raise ValueError(f"{name} must have shape {tuple(sizes)}, not {tuple(t.shape)}")
    if contiguous and not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() > 0 and t.stride(-1) != 1:
        raise ValueError(f"{name} must have a contiguous last dimension")


def _on_gpu(*named) -> int:
    """All (name, tensor) pairs (None tensors skipped) on one GPU; its index."""
    dev = None
    for name, t in named:
        if t is None:
            continue
        if t.device.type != "cuda":
            raise ValueError(f"{name} must be on a GPU, not {t.device}")
        if dev is None:
            dev = _device_index(t)
        elif _device_index(t) != dev:
            raise ValueError(f"{name} is on cuda:{_device_index(t)}, the other arguments on cuda:{dev}")
    return dev


def _heads_tokens(name: str, t, n_heads: int, n_tokens: int, head_dim: int):
    """A bf16 (head, token, dimension) tensor of any strides with a contiguous
    last dimension; returns its (head stride, token stride)."""
    _check_tensor(name, t, torch.bfloat16, (n_heads, n_tokens, head_dim), contiguous=False)
    return t.stride(0), t.stride(1)


def _with_strides(shape: rbs_shape, q=None, kv=None) -> rbs_shape:
    """A copy of shape with the Q and/or K, V strides of the given tensors.
    Strides already set in shape must agree with the tensors'."""
    out = rbs_shape.from_buffer_copy(shape)
    for pair, fields in ((q, ("q_stride_head", "q_stride_tok")), (kv, ("kv_stride_head", "kv_stride_tok"))):
        if pair is None:
            continue
        for value, field in zip(pair, fields):
            given = getattr(shape, field)
            if given not in (0, value):
                raise ValueError(f"shape.{field} = {given} disagrees with the tensor's stride {value}")
            setattr(out, field, value)
    return out


def _check_q(shape: rbs_shape, Q):
    return _heads_tokens("Q", Q, shape.n_q_heads, shape.n_tokens, shape.head_dim)


def _check_kv(shape: rbs_shape, K, V=None):
    kv = _heads_tokens("K", K, shape.n_kv_heads, shape.n_tokens, shape.head_dim)
    if V is not None:
        v = _heads_tokens("V", V, shape.n_kv_heads, shape.n_tokens, shape.head_dim)
        if v != kv:
            raise ValueError(f"V strides {v} differ from K strides {kv}; the library takes one pair")
    return kv


def _check_out(O, Q):
    """O: bf16 with Q's sizes and strides (the library writes O with Q's strides)."""
    _check_tensor("O", O, torch.bfloat16, tuple(Q.shape), contiguous=False)
    if O.stride() != Q.stride():
        raise ValueError(f"O strides {O.stride()} must equal Q strides {Q.stride()}")


def _check_lse(shape: rbs_shape, lse):
    if lse is not None:
        _check_tensor("lse", lse, torch.float32, (shape.n_q_heads, shape.n_tokens))


def _check_lists(shape: rbs_shape, counts, indices, n_blocks_total=None, capacity=None):
    m = n_blocks(shape) if n_blocks_total is None else n_blocks_total
    cap = rbs_index_capacity(m) if capacity is None else capacity
    _check_tensor("counts", counts, torch.int32, (shape.n_q_heads, m))
    _check_tensor("indices", indices, torch.int32, (shape.n_q_heads, cap))


def _check_stats(shape: rbs_shape, stats, n_blocks_total=None, n_seqs=1, summary_bytes=None, need_fp32=True):
    """The BlockStats tensors a call reads or writes; returns them named, for _on_gpu."""
    if not isinstance(stats, BlockStats):
        raise ValueError("stats must be a BlockStats")
    m = n_blocks(shape) if n_blocks_total is None else n_blocks_total
    hk, d = shape.n_kv_heads, shape.head_dim
    named = []
    if need_fp32:
        _check_tensor("stats.centroids", stats.centroids, torch.float32, (hk, m, d))
        _check_tensor("stats.radii", stats.radii, torch.float32, (hk, m))
        _check_tensor("stats.beta", stats.beta, torch.float32, (hk, m))
        qshape = (hk, 2) if n_blocks_total is None else (n_seqs, hk, 2)
        _check_tensor("stats.quantiles", stats.quantiles, torch.float32, qshape)
        named += [("stats.centroids", stats.centroids), ("stats.radii", stats.radii), ("stats.beta", stats.beta),
                  ("stats.quantiles", stats.quantiles)]
    nbytes = rbs_summary_bytes(shape) if summary_bytes is None else summary_bytes
    _check_tensor("stats.summary", stats.summary, torch.uint8, (nbytes,))
    return named + [("stats.summary", stats.summary)]


def _like_q(Q):
    """An output with Q's sizes and strides (the layout the library writes O in)."""
    return torch.empty_strided(tuple(Q.shape), Q.stride(), dtype=torch.bfloat16, device=Q.device)


def n_blocks(shape: rbs_shape) -> int:
    return -(-shape.n_tokens // shape.block_size)


def rbs_index_capacity(m: int) -> int:
    return int(load().rbs_index_capacity(m))


def rbs_summary_bytes(shape: rbs_shape) -> int:
    return int(load().rbs_summary_bytes(ctypes.byref(shape)))


@dataclass
class BlockStats:
    """Device buffers of rbs_stats (allocated by the caller: here, torch)."""
    shape: rbs_shape
    centroids: torch.Tensor   # fp32 [H_kv][M][d]
    radii: torch.Tensor       # fp32 [H_kv][M]
    beta: torch.Tensor        # fp32 [H_kv][M]
    quantiles: torch.Tensor   # fp32 [H_kv][2]
    summary: torch.Tensor     # uint8 [rbs_summary_bytes]

    @classmethod
    def allocate(cls, shape: rbs_shape, device="cuda") -> "BlockStats":
        m, hk, d = n_blocks(shape), shape.n_kv_heads, shape.head_dim
        f32 = dict(dtype=torch.float32, device=device)
        nbytes = rbs_summary_bytes(shape)
        if nbytes == 0:
            raise RbsError("rbs_summary_bytes", RBS_ERR_SHAPE, "invalid shape")
        return cls(shape, torch.empty((hk, m, d), **f32), torch.empty((hk, m), **f32),
                   torch.empty((hk, m), **f32), torch.empty((hk, 2), **f32),
                   torch.empty(nbytes, dtype=torch.uint8, device=device))

    def as_c(self) -> rbs_stats:
        return rbs_stats(_ptr(self.centroids), _ptr(self.radii), _ptr(self.beta), _ptr(self.quantiles),
                         _ptr(self.summary))


def rbs_block_stats(shape: rbs_shape, K: torch.Tensor, stats: BlockStats | None = None, stream=None) -> BlockStats:
    """Stage 1: centroids, radii, radius quantiles and beta of every key block."""
    kvs = _check_kv(shape, K)
    if stats is None:
        stats = BlockStats.allocate(shape, K.device)
    _on_gpu(("K", K), *_check_stats(shape, stats))
    sh = _with_strides(shape, kv=kvs)
    c = stats.as_c()
    _check("rbs_block_stats", load().rbs_block_stats(ctypes.byref(sh), _ptr(K), ctypes.byref(c), _stream(stream)))
    return stats


def rbs_stats_summarize(shape: rbs_shape, stats: BlockStats, stream=None) -> BlockStats:
    """The select-ready summary from stats.centroids, radii and beta (statistics
    computed elsewhere); rbs_block_stats writes the same summary itself."""
    _on_gpu(*_check_stats(shape, stats))
    c = stats.as_c()
    _check("rbs_stats_summarize", load().rbs_stats_summarize(ctypes.byref(shape), ctypes.byref(c), _stream(stream)))
    return stats


@dataclass
class BoxStats:
    """Device buffers of rbs_box (allocated by the caller: here, torch)."""
    shape: rbs_shape
    center: torch.Tensor   # fp32 [H_kv][M][d]
    half: torch.Tensor     # fp32 [H_kv][M][d]
    summary: torch.Tensor  # uint8 [rbs_box_summary_bytes]

    @classmethod
    def allocate(cls, shape: rbs_shape, device="cuda") -> "BoxStats":
        m, hk, d = n_blocks(shape), shape.n_kv_heads, shape.head_dim
        nbytes = int(load().rbs_box_summary_bytes(ctypes.byref(shape)))
        if nbytes == 0:
            raise RbsError("rbs_box_summary_bytes", RBS_ERR_SHAPE, "invalid shape")
        f32 = dict(dtype=torch.float32, device=device)
        return cls(shape, torch.empty((hk, m, d), **f32), torch.empty((hk, m, d), **f32),
                   torch.empty(nbytes, dtype=torch.uint8, device=device))

    def as_c(self) -> rbs_box:
        return rbs_box(_ptr(self.center), _ptr(self.half), _ptr(self.summary))


def _check_box(shape: rbs_shape, box):
    if not isinstance(box, BoxStats):
        raise ValueError("box must be a BoxStats")
    m, hk, d = n_blocks(shape), shape.n_kv_heads, shape.head_dim
    _check_tensor("box.center", box.center, torch.float32, (hk, m, d))
    _check_tensor("box.half", box.half, torch.float32, (hk, m, d))
    nbytes = int(load().rbs_box_summary_bytes(ctypes.byref(shape)))
    _check_tensor("box.summary", box.summary, torch.uint8, (nbytes,))
    return [("box.center", box.center), ("box.half", box.half), ("box.summary", box.summary)]


def rbs_block_box(shape: rbs_shape, K: torch.Tensor, box: BoxStats | None = None, stream=None) -> BoxStats:
    """Coordinate-wise key box of every block (centre, half-width)."""
    kvs = _check_kv(shape, K)
    if box is None:
        box = BoxStats.allocate(shape, K.device)
    _on_gpu(("K", K), *_check_box(shape, box))
    sh = _with_strides(shape, kv=kvs)
    c = box.as_c()
    _check("rbs_block_box", load().rbs_block_box(ctypes.byref(sh), _ptr(K), ctypes.byref(c), _stream(stream)))
    return box


def rbs_select_variant(shape: rbs_shape, Q: torch.Tensor, stats: BlockStats, selector, param: float,
                       n_sink: int, n_local: int, n_recent: int, box: BoxStats | None = None, counts=None,
                       indices=None, stream=None):
    """A supporting selector ("centroid", "full_l2", "box" or its RBS_SELECTOR_* code)."""
    sel = SELECTORS[selector] if isinstance(selector, str) else int(selector)
    qs = _check_q(shape, Q)
    named = _check_stats(shape, stats)
    if box is not None:
        named += _check_box(shape, box)
    if counts is None or indices is None:
        counts, indices = allocate_lists(shape, Q.device)
    _check_lists(shape, counts, indices)
    _on_gpu(("Q", Q), *named, ("counts", counts), ("indices", indices))
    sh = _with_strides(shape, q=qs)
    c = stats.as_c()
    b = box.as_c() if box is not None else None
    _check("rbs_select_variant", load().rbs_select_variant(
        ctypes.byref(sh), _ptr(Q), ctypes.byref(c), ctypes.byref(b) if b is not None else None, sel,
        float(param), int(n_sink), int(n_local), int(n_recent), _ptr(counts), _ptr(indices), _stream(stream)))
    return counts, indices


def allocate_lists(shape: rbs_shape, device="cuda"):
    m = n_blocks(shape)
    counts = torch.empty((shape.n_q_heads, m), dtype=torch.int32, device=device)
    indices = torch.empty((shape.n_q_heads, rbs_index_capacity(m)), dtype=torch.int32, device=device)
    return counts, indices


def rbs_select(shape: rbs_shape, Q: torch.Tensor, stats: BlockStats, tau_base: float, tau_rescue: float,
               n_sink: int, n_local: int, n_recent: int, counts=None, indices=None, stream=None):
    """Stage 2: per (query head, query block) ascending key-block index lists."""
    qs = _check_q(shape, Q)
    named = _check_stats(shape, stats, need_fp32=False)
    if counts is None or indices is None:
        counts, indices = allocate_lists(shape, Q.device)
    _check_lists(shape, counts, indices)
    _on_gpu(("Q", Q), *named, ("counts", counts), ("indices", indices))
    sh = _with_strides(shape, q=qs)
    c = stats.as_c()
    _check("rbs_select", load().rbs_select(ctypes.byref(sh), _ptr(Q), ctypes.byref(c), float(tau_base),
                                           float(tau_rescue), int(n_sink), int(n_local), int(n_recent),
                                           _ptr(counts), _ptr(indices), _stream(stream)))
    return counts, indices


def rbs_sparse_prefill(shape: rbs_shape, Q, K, V, counts, indices, softmax_scale: float = 0.0, O=None,
                       lse=None, stream=None, workspace=AUTO):
    """Stage 3: causal GQA block-sparse attention; returns O (bf16, Q's sizes and strides)."""
    qs = _check_q(shape, Q)
    kvs = _check_kv(shape, K, V)
    _check_lists(shape, counts, indices)
    if O is not None:
        _check_out(O, Q)
    _check_lse(shape, lse)
    _on_gpu(("Q", Q), ("K", K), ("V", V), ("counts", counts), ("indices", indices), ("O", O), ("lse", lse))
    if O is None:
        O = _like_q(Q)
    ws = _workspace(workspace, Q.device, stream)
    sh = _with_strides(shape, q=qs, kv=kvs)
    _check("rbs_sparse_prefill", load().rbs_sparse_prefill(ctypes.byref(sh), _ptr(Q), _ptr(K), _ptr(V),
                                                           _ptr(counts), _ptr(indices), float(softmax_scale),
                                                           _ptr(O), _ptr(lse), _ptr(ws), _stream(stream)))
    return O


def rbs_sparse_prefill_noalloc(shape: rbs_shape, Q, K, V, counts, indices, O, softmax_scale: float = 0.0,
                               lse=None, stream=None):
    """Stage 3 through the allocation-free entry point (the persistent launch
    with the library's static queue counters): O and lse must be given."""
    qs = _check_q(shape, Q)
    kvs = _check_kv(shape, K, V)
    _check_lists(shape, counts, indices)
    _check_out(O, Q)
    _check_lse(shape, lse)
    _on_gpu(("Q", Q), ("K", K), ("V", V), ("counts", counts), ("indices", indices), ("O", O), ("lse", lse))
    sh = _with_strides(shape, q=qs, kv=kvs)
    _check("rbs_sparse_prefill_noalloc", load().rbs_sparse_prefill_noalloc(
        ctypes.byref(sh), _ptr(Q), _ptr(K), _ptr(V), _ptr(counts), _ptr(indices), float(softmax_scale), _ptr(O),
        _ptr(lse), _stream(stream)))
    return O


def rbs_select_attend(shape: rbs_shape, Q, K, V, stats: BlockStats, tau_base: float, tau_rescue: float,
                      n_sink: int, n_local: int, n_recent: int, softmax_scale: float = 0.0, counts=None,
                      indices=None, O=None, lse=None, stream=None, workspace=AUTO):
    """Stages 2 and 3 in one pass; returns (counts, indices, O) as the two calls would."""
    qs = _check_q(shape, Q)
    kvs = _check_kv(shape, K, V)
    named = _check_stats(shape, stats, need_fp32=False)
    if counts is None or indices is None:
        counts, indices = allocate_lists(shape, Q.device)
    _check_lists(shape, counts, indices)
    if O is not None:
        _check_out(O, Q)
    _check_lse(shape, lse)
    _on_gpu(("Q", Q), ("K", K), ("V", V), *named, ("counts", counts), ("indices", indices), ("O", O),
            ("lse", lse))
    if O is None:
        O = _like_q(Q)
    c = stats.as_c()
    ws = _workspace(workspace, Q.device, stream)
    sh = _with_strides(shape, q=qs, kv=kvs)
    _check("rbs_select_attend", load().rbs_select_attend(
        ctypes.byref(sh), _ptr(Q), _ptr(K), _ptr(V), ctypes.byref(c), float(tau_base), float(tau_rescue),
        int(n_sink), int(n_local), int(n_recent), float(softmax_scale), _ptr(counts), _ptr(indices), _ptr(O),
        _ptr(lse), _ptr(ws), _stream(stream)))
    return counts, indices, O


def rbs_dense_indices(shape: rbs_shape, counts=None, indices=None, stream=None, device="cuda"):
    """Full causal lists: the dense path through the same attention kernel."""
    if counts is None or indices is None:
        counts, indices = allocate_lists(shape, device)
    _check_lists(shape, counts, indices)
    _on_gpu(("counts", counts), ("indices", indices))
    _check("rbs_dense_indices", load().rbs_dense_indices(ctypes.byref(shape), _ptr(counts), _ptr(indices),
                                                         _stream(stream)))
    return counts, indices


# ------------------------------------------------------------------ varlen

class Batch:
    """A batch of independent sequences packed along the token axis (the
    rbs_*_varlen calls).  Holds the host array that rbs_batch points at."""

    def __init__(self, seq_tokens):
        self.seq_tokens = [int(x) for x in seq_tokens]
        self._arr = (ctypes.c_int32 * max(1, len(self.seq_tokens)))(*self.seq_tokens)
        self.c = rbs_batch(len(self.seq_tokens), self._arr)

    @property
    def n_seqs(self) -> int:
        return len(self.seq_tokens)

    @property
    def n_tokens(self) -> int:
        return sum(self.seq_tokens)

    def token_offsets(self) -> list:
        out = [0]
        for n in self.seq_tokens:
            out.append(out[-1] + n)
        return out

    def block_counts(self, block_size: int) -> list:
        return [-(-n // block_size) for n in self.seq_tokens]


def varlen_shape(batch: Batch, n_q_heads: int, n_kv_heads: int, block_size: int, head_dim: int = 128) -> rbs_shape:
    return make_shape(batch.n_tokens, n_q_heads, n_kv_heads, block_size, head_dim)


def rbs_varlen_blocks(shape: rbs_shape, batch: Batch) -> int:
    return int(load().rbs_varlen_blocks(ctypes.byref(shape), ctypes.byref(batch.c)))


def rbs_varlen_index_capacity(shape: rbs_shape, batch: Batch) -> int:
    return int(load().rbs_varlen_index_capacity(ctypes.byref(shape), ctypes.byref(batch.c)))


def rbs_varlen_summary_bytes(shape: rbs_shape, batch: Batch) -> int:
    return int(load().rbs_varlen_summary_bytes(ctypes.byref(shape), ctypes.byref(batch.c)))


def allocate_stats_varlen(shape: rbs_shape, batch: Batch, device="cuda") -> BlockStats:
    """rbs_stats buffers of a batch: block arrays over all sequences' blocks,
    quantiles [n_seqs][H_kv][2]."""
    m, hk, d = rbs_varlen_blocks(shape, batch), shape.n_kv_heads, shape.head_dim
    nbytes = rbs_varlen_summary_bytes(shape, batch)
    if m == 0 or nbytes == 0:
        raise RbsError("rbs_varlen_summary_bytes", RBS_ERR_SHAPE, "invalid shape or batch")
    f32 = dict(dtype=torch.float32, device=device)
    return BlockStats(shape, torch.empty((hk, m, d), **f32), torch.empty((hk, m), **f32),
                      torch.empty((hk, m), **f32), torch.empty((batch.n_seqs, hk, 2), **f32),
                      torch.empty(nbytes, dtype=torch.uint8, device=device))


def allocate_lists_varlen(shape: rbs_shape, batch: Batch, device="cuda"):
    m, cap = rbs_varlen_blocks(shape, batch), rbs_varlen_index_capacity(shape, batch)
    if m == 0:
        raise RbsError("rbs_varlen_blocks", RBS_ERR_SHAPE, "invalid shape or batch")
    counts = torch.empty((shape.n_q_heads, m), dtype=torch.int32, device=device)
    indices = torch.empty((shape.n_q_heads, cap), dtype=torch.int32, device=device)
    return counts, indices


def rbs_block_stats_varlen(shape: rbs_shape, batch: Batch, K: torch.Tensor, stats: BlockStats | None = None,
                           stream=None) -> BlockStats:
    """Stage 1 for every sequence of a batch (one launch)."""
    kvs = _check_kv(shape, K)
    if stats is None:
        stats = allocate_stats_varlen(shape, batch, K.device)
    _on_gpu(("K", K), *_check_stats(shape, stats, n_blocks_total=rbs_varlen_blocks(shape, batch),
                                    n_seqs=batch.n_seqs, summary_bytes=rbs_varlen_summary_bytes(shape, batch)))
    sh = _with_strides(shape, kv=kvs)
    c = stats.as_c()
    _check("rbs_block_stats_varlen", load().rbs_block_stats_varlen(
        ctypes.byref(sh), ctypes.byref(batch.c), _ptr(K), ctypes.byref(c), _stream(stream)))
    return stats


def rbs_select_varlen(shape: rbs_shape, batch: Batch, Q: torch.Tensor, stats: BlockStats, tau_base: float,
                      tau_rescue: float, n_sink: int, n_local: int, n_recent: int, counts=None, indices=None,
                      stream=None):
    """Stage 2 for every sequence of a batch (one launch)."""
    qs = _check_q(shape, Q)
    m, cap = rbs_varlen_blocks(shape, batch), rbs_varlen_index_capacity(shape, batch)
    named = _check_stats(shape, stats, n_blocks_total=m, n_seqs=batch.n_seqs,
                         summary_bytes=rbs_varlen_summary_bytes(shape, batch), need_fp32=False)
    if counts is None or indices is None:
        counts, indices = allocate_lists_varlen(shape, batch, Q.device)
    _check_lists(shape, counts, indices, n_blocks_total=m, capacity=cap)
    _on_gpu(("Q", Q), *named, ("counts", counts), ("indices", indices))
    sh = _with_strides(shape, q=qs)
    c = stats.as_c()
    _check("rbs_select_varlen", load().rbs_select_varlen(
        ctypes.byref(sh), ctypes.byref(batch.c), _ptr(Q), ctypes.byref(c), float(tau_base), float(tau_rescue),
        int(n_sink), int(n_local), int(n_recent), _ptr(counts), _ptr(indices), _stream(stream)))
    return counts, indices


def rbs_sparse_prefill_varlen(shape: rbs_shape, batch: Batch, Q, K, V, counts, indices, softmax_scale: float = 0.0,
                              O=None, lse=None, stream=None, workspace=AUTO):
    """Stage 3 for every sequence of a batch (one launch); returns O."""
    qs = _check_q(shape, Q)
    kvs = _check_kv(shape, K, V)
    _check_lists(shape, counts, indices, n_blocks_total=rbs_varlen_blocks(shape, batch),
                 capacity=rbs_varlen_index_capacity(shape, batch))
    if O is not None:
        _check_out(O, Q)
    _check_lse(shape, lse)
    _on_gpu(("Q", Q), ("K", K), ("V", V), ("counts", counts), ("indices", indices), ("O", O), ("lse", lse))
    if O is None:
        O = _like_q(Q)
    ws = _workspace(workspace, Q.device, stream)
    sh = _with_strides(shape, q=qs, kv=kvs)
    _check("rbs_sparse_prefill_varlen", load().rbs_sparse_prefill_varlen(
        ctypes.byref(sh), ctypes.byref(batch.c), _ptr(Q), _ptr(K), _ptr(V), _ptr(counts), _ptr(indices),
        float(softmax_scale), _ptr(O), _ptr(lse), _ptr(ws), _stream(stream)))
    return O


def rbs_dense_indices_varlen(shape: rbs_shape, batch: Batch, counts=None, indices=None, stream=None,
                             device="cuda"):
    """Full causal lists of every sequence of a batch."""
    if counts is None or indices is None:
        counts, indices = allocate_lists_varlen(shape, batch, device)
    _check_lists(shape, counts, indices, n_blocks_total=rbs_varlen_blocks(shape, batch),
                 capacity=rbs_varlen_index_capacity(shape, batch))
    _on_gpu(("counts", counts), ("indices", indices))
    _check("rbs_dense_indices_varlen", load().rbs_dense_indices_varlen(
        ctypes.byref(shape), ctypes.byref(batch.c), _ptr(counts), _ptr(indices), _stream(stream)))
    return counts, indices


# ------------------------------------------------------------------ FP8 inputs

@dataclass
class Fp8Inputs:
    """E4M3 copies of Q, K, V and their per-head amax (device buffers)."""
    amax: torch.Tensor   # fp32 [H_q + 2 H_kv]
    Q8: torch.Tensor     # uint8 [H_q][N][d]
    K8: torch.Tensor     # uint8 [H_kv][N][d]
    V8t: torch.Tensor    # uint8 [rbs_fp8_vt_bytes]


def rbs_fp8_vt_bytes(shape: rbs_shape) -> int:
    return int(load().rbs_fp8_vt_bytes(ctypes.byref(shape)))


def allocate_fp8(shape: rbs_shape, device="cuda") -> Fp8Inputs:
    nvt = rbs_fp8_vt_bytes(shape)
    if nvt == 0:
        raise RbsError("rbs_fp8_vt_bytes", RBS_ERR_SHAPE, "invalid shape for the FP8 inputs")
    u8 = dict(dtype=torch.uint8, device=device)
    return Fp8Inputs(torch.empty(shape.n_q_heads + 2 * shape.n_kv_heads, dtype=torch.float32, device=device),
                     torch.empty((shape.n_q_heads, shape.n_tokens, shape.head_dim), **u8),
                     torch.empty((shape.n_kv_heads, shape.n_tokens, shape.head_dim), **u8),
                     torch.empty(nvt, **u8))


def _check_fp8(shape: rbs_shape, f8):
    if not isinstance(f8, Fp8Inputs):
        raise ValueError("f8 must be Fp8Inputs")
    n, d = shape.n_tokens, shape.head_dim
    _check_tensor("f8.amax", f8.amax, torch.float32, (shape.n_q_heads + 2 * shape.n_kv_heads,))
    _check_tensor("f8.Q8", f8.Q8, torch.uint8, (shape.n_q_heads, n, d))
    _check_tensor("f8.K8", f8.K8, torch.uint8, (shape.n_kv_heads, n, d))
    _check_tensor("f8.V8t", f8.V8t, torch.uint8, (rbs_fp8_vt_bytes(shape),))
    return [("f8.amax", f8.amax), ("f8.Q8", f8.Q8), ("f8.K8", f8.K8), ("f8.V8t", f8.V8t)]


def rbs_fp8_amax(shape: rbs_shape, Q, K, V, amax, stream=None):
    qs = _check_q(shape, Q)
    kvs = _check_kv(shape, K, V)
    _check_tensor("amax", amax, torch.float32, (shape.n_q_heads + 2 * shape.n_kv_heads,))
    _on_gpu(("Q", Q), ("K", K), ("V", V), ("amax", amax))
    sh = _with_strides(shape, q=qs, kv=kvs)
    _check("rbs_fp8_amax", load().rbs_fp8_amax(ctypes.byref(sh), _ptr(Q), _ptr(K), _ptr(V), _ptr(amax),
                                               _stream(stream)))
    return amax


def rbs_fp8_pack(shape: rbs_shape, Q, K, V, f8: Fp8Inputs, stream=None) -> Fp8Inputs:
    qs = _check_q(shape, Q)
    kvs = _check_kv(shape, K, V)
    _on_gpu(("Q", Q), ("K", K), ("V", V), *_check_fp8(shape, f8))
    sh = _with_strides(shape, q=qs, kv=kvs)
    _check("rbs_fp8_pack", load().rbs_fp8_pack(ctypes.byref(sh), _ptr(Q), _ptr(K), _ptr(V), _ptr(f8.amax),
                                               _ptr(f8.Q8), _ptr(f8.K8), _ptr(f8.V8t), _stream(stream)))
    return f8


def rbs_fp8_prepare(shape: rbs_shape, Q, K, V, f8: Fp8Inputs | None = None, stream=None) -> Fp8Inputs:
    """amax then pack: the E4M3 inputs of rbs_sparse_prefill_fp8."""
    if f8 is None:
        f8 = allocate_fp8(shape, Q.device)
    rbs_fp8_amax(shape, Q, K, V, f8.amax, stream)
    return rbs_fp8_pack(shape, Q, K, V, f8, stream)


def rbs_sparse_prefill_fp8(shape: rbs_shape, f8: Fp8Inputs, counts, indices, softmax_scale: float = 0.0, O=None,
                           lse=None, stream=None, workspace=AUTO):
    """Stage 3 on the E4M3 inputs; returns O (bf16 [H_q][N][d], or the strides of the O given)."""
    named = _check_fp8(shape, f8)
    _check_lists(shape, counts, indices)
    if O is None:
        O = torch.empty((shape.n_q_heads, shape.n_tokens, shape.head_dim), dtype=torch.bfloat16,
                        device=f8.Q8.device)
    qs = _heads_tokens("O", O, shape.n_q_heads, shape.n_tokens, shape.head_dim)
    _check_lse(shape, lse)
    _on_gpu(*named, ("counts", counts), ("indices", indices), ("O", O), ("lse", lse))
    ws = _workspace(workspace, f8.Q8.device, stream)
    sh = _with_strides(shape, q=qs)
    _check("rbs_sparse_prefill_fp8", load().rbs_sparse_prefill_fp8(
        ctypes.byref(sh), _ptr(f8.Q8), _ptr(f8.K8), _ptr(f8.V8t), _ptr(f8.amax), _ptr(counts), _ptr(indices),
        float(softmax_scale), _ptr(O), _ptr(lse), _ptr(ws), _stream(stream)))
    return O
