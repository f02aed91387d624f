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

RBS_OK, RBS_ERR_NULL, RBS_ERR_SHAPE, RBS_ERR_UNSUPPORTED, RBS_ERR_ARG, RBS_ERR_ALIGN, RBS_ERR_HIP = range(7)


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
    lib.rbs_select.argtypes = [SP, P, ctypes.POINTER(rbs_stats), F32, F32, I32, I32, I32, P, P, P]
    lib.rbs_select.restype = ctypes.c_int
    lib.rbs_attention_workspace_bytes.argtypes = []
    lib.rbs_attention_workspace_bytes.restype = SZ
    lib.rbs_sparse_prefill.argtypes = [SP, P, P, P, P, P, F32, P, P, P, P]
    lib.rbs_sparse_prefill.restype = ctypes.c_int
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
    _lib = lib
    return lib


def rbs_status_str(status: int) -> str:
    return load().rbs_status_str(status).decode()


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
    return rbs_shape(n_tokens, n_q_heads, n_kv_heads, head_dim, block_size)


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
    if stats is None:
        stats = BlockStats.allocate(shape, K.device)
    c = stats.as_c()
    _check("rbs_block_stats", load().rbs_block_stats(ctypes.byref(shape), _ptr(K), ctypes.byref(c), _stream(stream)))
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


def rbs_block_box(shape: rbs_shape, K: torch.Tensor, box: BoxStats | None = None, stream=None) -> BoxStats:
    """Coordinate-wise key box of every block (centre, half-width)."""
    if box is None:
        box = BoxStats.allocate(shape, K.device)
    c = box.as_c()
    _check("rbs_block_box", load().rbs_block_box(ctypes.byref(shape), _ptr(K), ctypes.byref(c), _stream(stream)))
    return box


def rbs_select_variant(shape: rbs_shape, Q: torch.Tensor, stats: BlockStats, selector, param: float,
                       n_sink: int, n_local: int, n_recent: int, box: BoxStats | None = None, counts=None,
                       indices=None, stream=None):
    """A supporting selector ("centroid", "full_l2", "box" or its RBS_SELECTOR_* code)."""
    sel = SELECTORS[selector] if isinstance(selector, str) else int(selector)
    if counts is None or indices is None:
        counts, indices = allocate_lists(shape, Q.device)
    c = stats.as_c()
    b = box.as_c() if box is not None else None
    _check("rbs_select_variant", load().rbs_select_variant(
        ctypes.byref(shape), _ptr(Q), ctypes.byref(c), ctypes.byref(b) if b is not None else None, sel,
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
    if counts is None or indices is None:
        counts, indices = allocate_lists(shape, Q.device)
    c = stats.as_c()
    _check("rbs_select", load().rbs_select(ctypes.byref(shape), _ptr(Q), ctypes.byref(c), float(tau_base),
                                           float(tau_rescue), int(n_sink), int(n_local), int(n_recent),
                                           _ptr(counts), _ptr(indices), _stream(stream)))
    return counts, indices


def rbs_sparse_prefill(shape: rbs_shape, Q, K, V, counts, indices, softmax_scale: float = 0.0, O=None,
                       lse=None, stream=None, workspace=AUTO):
    """Stage 3: causal GQA block-sparse attention; returns O (bf16 [H_q][N][d])."""
    if O is None:
        O = torch.empty_like(Q)
    ws = _workspace(workspace, Q.device, stream)
    _check("rbs_sparse_prefill", load().rbs_sparse_prefill(ctypes.byref(shape), _ptr(Q), _ptr(K), _ptr(V),
                                                           _ptr(counts), _ptr(indices), float(softmax_scale),
                                                           _ptr(O), _ptr(lse), _ptr(ws), _stream(stream)))
    return O


def rbs_select_attend(shape: rbs_shape, Q, K, V, stats: BlockStats, tau_base: float, tau_rescue: float,
                      n_sink: int, n_local: int, n_recent: int, softmax_scale: float = 0.0, counts=None,
                      indices=None, O=None, lse=None, stream=None, workspace=AUTO):
    """Stages 2 and 3 in one pass; returns (counts, indices, O) as the two calls would."""
    if counts is None or indices is None:
        counts, indices = allocate_lists(shape, Q.device)
    if O is None:
        O = torch.empty_like(Q)
    c = stats.as_c()
    ws = _workspace(workspace, Q.device, stream)
    _check("rbs_select_attend", load().rbs_select_attend(
        ctypes.byref(shape), _ptr(Q), _ptr(K), _ptr(V), ctypes.byref(c), float(tau_base), float(tau_rescue),
        int(n_sink), int(n_local), int(n_recent), float(softmax_scale), _ptr(counts), _ptr(indices), _ptr(O),
        _ptr(lse), _ptr(ws), _stream(stream)))
    return counts, indices, O


def rbs_dense_indices(shape: rbs_shape, counts=None, indices=None, stream=None, device="cuda"):
    """Full causal lists: the dense path through the same attention kernel."""
    if counts is None or indices is None:
        counts, indices = allocate_lists(shape, device)
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
    if stats is None:
        stats = allocate_stats_varlen(shape, batch, K.device)
    c = stats.as_c()
    _check("rbs_block_stats_varlen", load().rbs_block_stats_varlen(
        ctypes.byref(shape), ctypes.byref(batch.c), _ptr(K), ctypes.byref(c), _stream(stream)))
    return stats


def rbs_select_varlen(shape: rbs_shape, batch: Batch, Q: torch.Tensor, stats: BlockStats, tau_base: float,
                      tau_rescue: float, n_sink: int, n_local: int, n_recent: int, counts=None, indices=None,
                      stream=None):
    """Stage 2 for every sequence of a batch (one launch)."""
    if counts is None or indices is None:
        counts, indices = allocate_lists_varlen(shape, batch, Q.device)
    c = stats.as_c()
    _check("rbs_select_varlen", load().rbs_select_varlen(
        ctypes.byref(shape), ctypes.byref(batch.c), _ptr(Q), ctypes.byref(c), float(tau_base), float(tau_rescue),
        int(n_sink), int(n_local), int(n_recent), _ptr(counts), _ptr(indices), _stream(stream)))
    return counts, indices


def rbs_sparse_prefill_varlen(shape: rbs_shape, batch: Batch, Q, K, V, counts, indices, softmax_scale: float = 0.0,
                              O=None, lse=None, stream=None, workspace=AUTO):
    """Stage 3 for every sequence of a batch (one launch); returns O."""
    if O is None:
        O = torch.empty_like(Q)
    ws = _workspace(workspace, Q.device, stream)
    _check("rbs_sparse_prefill_varlen", load().rbs_sparse_prefill_varlen(
        ctypes.byref(shape), ctypes.byref(batch.c), _ptr(Q), _ptr(K), _ptr(V), _ptr(counts), _ptr(indices),
        float(softmax_scale), _ptr(O), _ptr(lse), _ptr(ws), _stream(stream)))
    return O


def rbs_dense_indices_varlen(shape: rbs_shape, batch: Batch, counts=None, indices=None, stream=None,
                             device="cuda"):
    """Full causal lists of every sequence of a batch."""
    if counts is None or indices is None:
        counts, indices = allocate_lists_varlen(shape, batch, device)
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


def rbs_fp8_amax(shape: rbs_shape, Q, K, V, amax, stream=None):
    _check("rbs_fp8_amax", load().rbs_fp8_amax(ctypes.byref(shape), _ptr(Q), _ptr(K), _ptr(V), _ptr(amax),
                                               _stream(stream)))
    return amax


def rbs_fp8_pack(shape: rbs_shape, Q, K, V, f8: Fp8Inputs, stream=None) -> Fp8Inputs:
    _check("rbs_fp8_pack", load().rbs_fp8_pack(ctypes.byref(shape), _ptr(Q), _ptr(K), _ptr(V), _ptr(f8.amax),
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
    """Stage 3 on the E4M3 inputs; returns O (bf16 [H_q][N][d])."""
    if O is None:
        O = torch.empty((shape.n_q_heads, shape.n_tokens, shape.head_dim), dtype=torch.bfloat16,
                        device=f8.Q8.device)
    ws = _workspace(workspace, f8.Q8.device, stream)
    _check("rbs_sparse_prefill_fp8", load().rbs_sparse_prefill_fp8(
        ctypes.byref(shape), _ptr(f8.Q8), _ptr(f8.K8), _ptr(f8.V8t), _ptr(f8.amax), _ptr(counts), _ptr(indices),
        float(softmax_scale), _ptr(O), _ptr(lse), _ptr(ws), _stream(stream)))
    return O
