"""C-ABI checks that need no GPU: the library loads, exports every symbol that
include/rbs.h declares, and rejects invalid arguments on the host before any
launch (no call here reaches the GPU: each one fails validation first)."""

from __future__ import annotations

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rbs.h")


def _lib():
    import paper_2609_20971_amd as rbs
    if not os.path.exists(rbs.LIB_PATH):
        pytest.fail("librbs.so is not built (run __graft_entry__.build())")
    return rbs, rbs.load()


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\w[\w\s\*]*?\b(rbs_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_three_stage_calls():
    names = _declared()
    for fn in ("rbs_block_stats", "rbs_select", "rbs_sparse_prefill", "rbs_select_attend"):
        assert fn in names


def test_library_exports_every_declared_symbol():
    _, lib = _lib()
    for name in _declared():
        assert hasattr(lib, name), name


def test_status_strings():
    rbs, _ = _lib()
    for code in range(8):
        assert rbs.rbs_status_str(code) != "unknown status"
    assert rbs.rbs_status_str(99) == "unknown status"


def test_debug_switch_is_host_state_and_validation_still_comes_first():
    """rbs_set_debug only flips a flag (no HIP call) and returns the previous
    setting; in debug mode a rejected call still launches nothing."""
    rbs, lib = _lib()
    prev = rbs.rbs_set_debug(True)
    try:
        assert rbs.rbs_set_debug(True) is True
        s = rbs.make_shape(1024, 4, 2, 64)
        st = _stats(rbs)
        assert lib.rbs_select(ctypes.byref(s), None, ctypes.byref(st), 0.9, 0.9, 1, 1, 0, FAKE, FAKE, None) == 1
        assert lib.rbs_select(ctypes.byref(s), FAKE, ctypes.byref(st), 1.5, 0.9, 1, 1, 0, FAKE, FAKE, None) == 4
        assert _fused(lib, s, st, Q=MIS) == 5
        assert rbs.rbs_set_debug(False) is True
        assert rbs.rbs_set_debug(False) is False
    finally:
        rbs.rbs_set_debug(prev)


def test_capacity_and_summary_sizes():
    rbs, _ = _lib()
    assert rbs.rbs_index_capacity(1024) == 1024 * 1025 // 2
    assert rbs.rbs_index_capacity(0) == 0
    s = rbs.make_shape(131072, 32, 4, 128)
    # f16 select-ready centroids + fp32 uplift and centroid norm per block.
    assert rbs.rbs_summary_bytes(s) == 4 * 1024 * 256 + 2 * 4 * 1024 * 4
    assert rbs.rbs_summary_bytes(rbs.make_shape(100, 2, 1, 96)) == 0


FAKE = 0x10000  # aligned, never dereferenced: validation fails before use
MIS = 0x10001


def _stats(rbs, ptr=FAKE, **override):
    vals = dict(centroids=ptr, radii=ptr, beta=ptr, quantiles=ptr, summary=ptr)
    vals.update(override)
    return rbs.rbs_stats(**vals)


@pytest.mark.parametrize("field,value,code", [
    ("head_dim", 64, 3), ("block_size", 96, 3), ("block_size", 32, 3), ("n_tokens", 0, 2),
    ("n_q_heads", 3, 2), ("n_kv_heads", 0, 2), ("n_tokens", 262145, 2),
])
def test_shape_validation(field, value, code):
    rbs, lib = _lib()
    s = rbs.make_shape(1024, 4, 2, 64)
    setattr(s, field, value)
    st = _stats(rbs)
    assert lib.rbs_block_stats(ctypes.byref(s), FAKE, ctypes.byref(st), None) == code
    assert lib.rbs_select(ctypes.byref(s), FAKE, ctypes.byref(st), 0.9, 0.9, 1, 1, 0, FAKE, FAKE, None) == code
    assert lib.rbs_sparse_prefill(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, None, None, None) == code
    assert lib.rbs_dense_indices(ctypes.byref(s), FAKE, FAKE, None) == code
    assert _fused(lib, s, st) == code


def _fused(lib, s, st, Q=FAKE, K=FAKE, V=FAKE, tb=0.9, tr=0.9, sink=1, local=1, recent=0, scale=0.0, counts=FAKE,
           indices=FAKE, O=FAKE, lse=None, workspace=None):
    return lib.rbs_select_attend(ctypes.byref(s), Q, K, V, ctypes.byref(st) if st is not None else None, tb, tr,
                                 sink, local, recent, scale, counts, indices, O, lse, workspace, None)


def test_largest_shape_passes_shape_validation():
    rbs, lib = _lib()
    s = rbs.make_shape(262144, 1, 1, 64)  # M = 4096, the largest allowed
    st = _stats(rbs)
    # Passes the shape checks and stops at the NULL key pointer.
    assert lib.rbs_block_stats(ctypes.byref(s), None, ctypes.byref(st), None) == 1


def test_null_and_alignment_errors():
    rbs, lib = _lib()
    s = rbs.make_shape(1024, 4, 2, 64)
    assert lib.rbs_block_stats(None, FAKE, ctypes.byref(_stats(rbs)), None) == 1
    assert lib.rbs_block_stats(ctypes.byref(s), None, ctypes.byref(_stats(rbs)), None) == 1
    assert lib.rbs_block_stats(ctypes.byref(s), FAKE, None, None) == 1
    for field in ("centroids", "radii", "beta", "quantiles", "summary"):
        assert lib.rbs_block_stats(ctypes.byref(s), FAKE, ctypes.byref(_stats(rbs, **{field: None})), None) == 1
        assert lib.rbs_block_stats(ctypes.byref(s), FAKE, ctypes.byref(_stats(rbs, **{field: MIS})), None) == 5
    assert lib.rbs_block_stats(ctypes.byref(s), MIS, ctypes.byref(_stats(rbs)), None) == 5
    st = _stats(rbs)
    assert lib.rbs_select(ctypes.byref(s), None, ctypes.byref(st), 0.9, 0.9, 1, 1, 0, FAKE, FAKE, None) == 1
    assert lib.rbs_select(ctypes.byref(s), FAKE, ctypes.byref(st), 0.9, 0.9, 1, 1, 0, None, FAKE, None) == 1
    assert lib.rbs_select(ctypes.byref(s), FAKE, ctypes.byref(st), 0.9, 0.9, 1, 1, 0, FAKE, MIS, None) == 5
    assert lib.rbs_sparse_prefill(ctypes.byref(s), FAKE, FAKE, None, FAKE, FAKE, 0.0, FAKE, None, None, None) == 1
    assert lib.rbs_sparse_prefill(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, MIS, None, None, None) == 5
    assert lib.rbs_sparse_prefill(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, MIS, None, None) == 5
    # A misaligned attention workspace is refused before anything is launched.
    assert lib.rbs_sparse_prefill(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, None, MIS, None) == 5
    assert lib.rbs_dense_indices(ctypes.byref(s), FAKE, None, None) == 1
    for arg in ("Q", "K", "V", "counts", "indices", "O"):
        assert _fused(lib, s, st, **{arg: None}) == 1
        assert _fused(lib, s, st, **{arg: MIS}) == 5
    assert _fused(lib, s, None) == 1
    assert _fused(lib, s, _stats(rbs, summary=None)) == 1
    assert _fused(lib, s, _stats(rbs, summary=MIS)) == 5
    assert _fused(lib, s, st, lse=MIS) == 5
    assert _fused(lib, s, st, workspace=MIS) == 5


@pytest.mark.parametrize("tb,tr,sink,local,recent", [
    (-0.1, 0.5, 1, 1, 0), (0.5, 1.5, 1, 1, 0), (float("nan"), 0.5, 1, 1, 0),
    (0.5, 0.5, -1, 1, 0), (0.5, 0.5, 1, 0, 0), (0.5, 0.5, 1, 1, -2),
])
def test_select_argument_errors(tb, tr, sink, local, recent):
    rbs, lib = _lib()
    s = rbs.make_shape(1024, 4, 2, 64)
    st = _stats(rbs)
    assert lib.rbs_select(ctypes.byref(s), FAKE, ctypes.byref(st), tb, tr, sink, local, recent, FAKE, FAKE, None) == 4
    assert _fused(lib, s, st, tb=tb, tr=tr, sink=sink, local=local, recent=recent) == 4


def test_bad_softmax_scale():
    rbs, lib = _lib()
    s = rbs.make_shape(1024, 4, 2, 64)
    for bad in (float("nan"), float("inf")):
        assert lib.rbs_sparse_prefill(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, FAKE, bad, FAKE, None, None, None) == 4
        assert _fused(lib, s, _stats(rbs), scale=bad) == 4


def test_binding_raises_without_library(monkeypatch, tmp_path):
    import paper_2609_20971_amd._lib as L
    monkeypatch.setattr(L, "_lib", None)
    monkeypatch.setattr(L, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="missing"):
        L.load()


def _box(rbs, ptr=FAKE, **override):
    vals = dict(center=ptr, half=ptr, summary=ptr)
    vals.update(override)
    return rbs.rbs_box(**vals)


def _variant(lib, s, st, bx, sel=1, param=0.5, sink=1, local=1, recent=0, Q=FAKE, counts=FAKE, indices=FAKE):
    return lib.rbs_select_variant(ctypes.byref(s), Q, ctypes.byref(st) if st is not None else None,
                                  ctypes.byref(bx) if bx is not None else None, sel, param, sink, local, recent,
                                  counts, indices, None)


def test_box_summary_size_and_validation():
    rbs, lib = _lib()
    s = rbs.make_shape(1000, 4, 2, 64)
    M = 16
    assert lib.rbs_box_summary_bytes(ctypes.byref(s)) >= 2 * 2 * M * 128 * 2
    bad = rbs.make_shape(1000, 4, 2, 96)
    assert lib.rbs_box_summary_bytes(ctypes.byref(bad)) == 0
    assert lib.rbs_block_box(ctypes.byref(bad), FAKE, ctypes.byref(_box(rbs)), None) == 3
    assert lib.rbs_block_box(ctypes.byref(s), None, ctypes.byref(_box(rbs)), None) == 1
    assert lib.rbs_block_box(ctypes.byref(s), FAKE, None, None) == 1
    for field in ("center", "half", "summary"):
        assert lib.rbs_block_box(ctypes.byref(s), FAKE, ctypes.byref(_box(rbs, **{field: None})), None) == 1
        assert lib.rbs_block_box(ctypes.byref(s), FAKE, ctypes.byref(_box(rbs, **{field: MIS})), None) == 5


def test_select_variant_validation():
    rbs, lib = _lib()
    s = rbs.make_shape(1024, 4, 2, 64)
    st, bx = _stats(rbs), _box(rbs)
    for sel in (0, 4, -1):
        assert _variant(lib, s, st, bx, sel=sel) == 4
    for sel, param in ((1, -0.1), (1, 1.5), (2, float("nan")), (3, 0.0), (3, 1.01), (3, -0.5)):
        assert _variant(lib, s, st, bx, sel=sel, param=param) == 4
    assert _variant(lib, s, st, None, sel=3, param=0.1) == 1
    assert _variant(lib, s, st, _box(rbs, summary=None), sel=3, param=0.1) == 1
    assert _variant(lib, s, st, _box(rbs, summary=MIS), sel=3, param=0.1) == 5
    assert _variant(lib, s, _stats(rbs, radii=None), bx, sel=2) == 1
    assert _variant(lib, s, _stats(rbs, radii=MIS), bx, sel=2) == 5
    assert _variant(lib, s, None, bx) == 1
    assert _variant(lib, s, st, bx, Q=None) == 1
    assert _variant(lib, s, st, bx, counts=MIS) == 5
    assert _variant(lib, s, st, bx, local=0) == 4
    bad = rbs.make_shape(1024, 3, 2, 64)
    assert _variant(lib, bad, st, bx) == 2


def _varlen_calls(lib, s, b, st, ptr=FAKE):
    """Status of every varlen call on (shape, batch) with the given pointers."""
    bb = ctypes.byref(b.c) if b is not None else None
    return [
        lib.rbs_block_stats_varlen(ctypes.byref(s), bb, ptr, ctypes.byref(st), None),
        lib.rbs_select_varlen(ctypes.byref(s), bb, ptr, ctypes.byref(st), 0.9, 0.9, 1, 1, 0, ptr, ptr, None),
        lib.rbs_sparse_prefill_varlen(ctypes.byref(s), bb, ptr, ptr, ptr, ptr, ptr, 0.0, ptr, None, None, None),
        lib.rbs_dense_indices_varlen(ctypes.byref(s), bb, ptr, ptr, None),
    ]


def test_varlen_sizes():
    rbs, _ = _lib()
    b = rbs.Batch([700, 1536, 64, 2049, 1])
    s = rbs.varlen_shape(b, 4, 2, 128)
    m = [6, 12, 1, 17, 1]
    assert rbs.rbs_varlen_blocks(s, b) == sum(m)
    assert rbs.rbs_varlen_index_capacity(s, b) == sum(x * (x + 1) // 2 for x in m)
    # rbs_summary_bytes at M = 37: f16 centroids, then uplift and norms, each part 256-aligned
    assert rbs.rbs_varlen_summary_bytes(s, b) == 2 * 37 * 256 + 512 + 2 * 37 * 4
    one = rbs.Batch([4096])
    s1 = rbs.varlen_shape(one, 4, 2, 128)
    assert rbs.rbs_varlen_summary_bytes(s1, one) == rbs.rbs_summary_bytes(s1)
    assert rbs.rbs_varlen_index_capacity(s1, one) == rbs.rbs_index_capacity(32)


@pytest.mark.parametrize("seqs,total,code", [
    ([], None, 2),                      # no sequence
    ([10] * 65, None, 2),               # more than RBS_MAX_SEQS
    ([10, 0, 5], None, 2),              # an empty sequence
    ([10, 262145], None, 2),            # a sequence over the token limit
    ([100, 200], 301, 2),               # lengths do not add up to n_tokens
])
def test_varlen_batch_validation(seqs, total, code):
    rbs, lib = _lib()
    b = rbs.Batch(seqs)
    s = rbs.make_shape(total if total is not None else max(1, sum(seqs)), 4, 2, 64)
    st = _stats(rbs)
    assert _varlen_calls(lib, s, b, st) == [code] * 4
    assert rbs.rbs_varlen_blocks(s, b) == 0 and rbs.rbs_varlen_summary_bytes(s, b) == 0


def test_varlen_null_unsupported_and_alignment():
    rbs, lib = _lib()
    b = rbs.Batch([100, 200])
    s = rbs.varlen_shape(b, 4, 2, 64)
    st = _stats(rbs)
    assert _varlen_calls(lib, s, None, st) == [1] * 4           # no batch
    nb = rbs.Batch([100, 200])
    nb.c.seq_tokens = ctypes.POINTER(ctypes.c_int32)()           # NULL host array
    assert _varlen_calls(lib, s, nb, st) == [1] * 4
    assert _varlen_calls(lib, s, b, st, ptr=None) == [1] * 4
    assert _varlen_calls(lib, s, b, st, ptr=MIS) == [5] * 4
    assert lib.rbs_sparse_prefill_varlen(ctypes.byref(s), ctypes.byref(b.c), FAKE, FAKE, FAKE, FAKE, FAKE, 0.0,
                                         FAKE, None, MIS, None) == 5
    bad = rbs.varlen_shape(b, 4, 2, 96)
    assert _varlen_calls(lib, bad, b, st) == [3] * 4
    assert lib.rbs_select_varlen(ctypes.byref(s), ctypes.byref(b.c), FAKE, ctypes.byref(st), 1.5, 0.9, 1, 1, 0,
                                 FAKE, FAKE, None) == 4
    assert lib.rbs_sparse_prefill_varlen(ctypes.byref(s), ctypes.byref(b.c), FAKE, FAKE, FAKE, FAKE, FAKE,
                                         float("nan"), FAKE, None, None, None) == 4


def test_varlen_largest_batch_passes_validation():
    rbs, lib = _lib()
    b = rbs.Batch([262144] * 2 + [1] * 62)  # RBS_MAX_SEQS sequences, two at the token limit
    s = rbs.varlen_shape(b, 1, 1, 64)
    st = _stats(rbs)
    # Passes the shape and batch checks, stops at the NULL key pointer.
    assert lib.rbs_block_stats_varlen(ctypes.byref(s), ctypes.byref(b.c), None, ctypes.byref(st), None) == 1
    assert rbs.rbs_varlen_blocks(s, b) == 2 * 4096 + 62


def test_fp8_sizes_and_validation():
    rbs, lib = _lib()
    s = rbs.make_shape(1000, 4, 2, 128)
    assert rbs.rbs_fp8_vt_bytes(s) == 2 * 8 * 128 * 128
    assert rbs.rbs_fp8_vt_bytes(rbs.make_shape(1000, 4, 2, 64)) == 2 * 16 * 128 * 64
    assert rbs.rbs_fp8_vt_bytes(rbs.make_shape(1000, 4, 2, 256)) == 2 * 4 * 128 * 256
    assert rbs.rbs_fp8_vt_bytes(rbs.make_shape(1000, 4, 2, 32)) == 0
    S = ctypes.byref(s)
    assert lib.rbs_fp8_amax(S, None, FAKE, FAKE, FAKE, None) == 1
    assert lib.rbs_fp8_amax(S, FAKE, FAKE, FAKE, MIS, None) == 5
    assert lib.rbs_fp8_pack(S, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None) == 1
    assert lib.rbs_fp8_pack(S, FAKE, FAKE, FAKE, FAKE, FAKE, MIS, FAKE, None) == 5
    # Block sizes other than 64/128/256 are refused before anything is launched.
    b32 = rbs.make_shape(1000, 4, 2, 32)
    assert lib.rbs_fp8_pack(ctypes.byref(b32), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == 3
    assert lib.rbs_sparse_prefill_fp8(ctypes.byref(b32), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, None,
                                      None, None) == 3
    assert lib.rbs_sparse_prefill_fp8(S, FAKE, FAKE, None, FAKE, FAKE, FAKE, 0.0, FAKE, None, None, None) == 1
    assert lib.rbs_sparse_prefill_fp8(S, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, float("nan"), FAKE, None, None, None) == 4
    assert lib.rbs_sparse_prefill_fp8(S, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, MIS, None, None) == 5
    assert lib.rbs_sparse_prefill_fp8(S, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, None, MIS, None) == 5
    bad = rbs.make_shape(1000, 3, 2, 128)
    assert lib.rbs_fp8_amax(ctypes.byref(bad), FAKE, FAKE, FAKE, FAKE, None) == 2


def test_attention_workspace_size():
    rbs, lib = _lib()
    assert lib.rbs_attention_workspace_bytes() == 256


def test_binding_workspace_argument():
    """The binding's workspace argument: None passes NULL, a tensor must hold
    rbs_attention_workspace_bytes(), anything else is refused (host checks only)."""
    import torch
    from paper_2609_20971_amd import _lib as L
    _lib()
    assert L._workspace(None, "cpu", 0) is None
    t = torch.zeros(64, dtype=torch.int32)
    assert L._workspace(t, "cpu", 0) is t
    with pytest.raises(ValueError):
        L._workspace(torch.zeros(63, dtype=torch.int32), "cpu", 0)
    with pytest.raises(ValueError):
        L._workspace("cached", "cpu", 0)


# ------------------------------------------------------------------ strides (rbs_shape)

@pytest.mark.parametrize("strides,ok", [
    ((0, 0, 0, 0), True),                                   # dense [H][N][d]
    ((128, 4 * 128, 128, 2 * 128), True),                   # token-major [N][H][d] (H_q = 4, H_kv = 2)
    ((128, 6 * 128, 128, 6 * 128), True),                   # token-major rows of a wider buffer
    ((1024 * 256, 256, 1024 * 256, 256), True),             # head-major with padded rows
    ((128, 128, 0, 0), False),                              # Q rows of different heads overlap
    ((0, 64, 0, 0), False),                                 # token stride shorter than a row
    ((0, 0, 1024 * 128 - 8, 128), False),                   # heads overlap
    ((0, 132, 0, 0), False),                                # not a multiple of 8 elements
    ((0, 0, 128, -256), False),                             # negative
    ((0, 0, 0, (1 << 23) + 8), False),                      # token stride past the copy offsets
])
def test_stride_validation(strides, ok):
    rbs, lib = _lib()
    s = rbs.make_shape(1024, 4, 2, 64)
    s.q_stride_head, s.q_stride_tok, s.kv_stride_head, s.kv_stride_tok = strides
    # NULL counts: a shape that passes reaches the pointer checks (status 1)
    # and launches nothing; a bad one stops at the shape (status 2).
    want = 1 if ok else 2
    assert lib.rbs_sparse_prefill(ctypes.byref(s), FAKE, FAKE, FAKE, None, FAKE, 0.0, FAKE, None, None, None) == want
    assert lib.rbs_block_stats(ctypes.byref(s), None, ctypes.byref(_stats(rbs)), None) == want
    assert (lib.rbs_summary_bytes(ctypes.byref(s)) > 0) == ok


def test_stats_summarize_validation():
    rbs, lib = _lib()
    s = rbs.make_shape(1024, 4, 2, 64)
    assert lib.rbs_stats_summarize(ctypes.byref(s), ctypes.byref(_stats(rbs, beta=None)), None) == 1
    assert lib.rbs_stats_summarize(ctypes.byref(s), None, None) == 1
    assert lib.rbs_stats_summarize(ctypes.byref(s), ctypes.byref(_stats(rbs, summary=MIS)), None) == 5
    bad = rbs.make_shape(1024, 4, 2, 64)
    bad.head_dim = 64
    assert lib.rbs_stats_summarize(ctypes.byref(bad), ctypes.byref(_stats(rbs)), None) == 3


# ------------------------------------------------------------------ binding argument checks
# The Python binding checks dtype, sizes, layout and device of every tensor
# before calling the library; a mismatch raises ValueError and reaches no
# C call.  These run on CPU tensors: every check before the device check is
# exercised with otherwise valid CPU tensors, the device check with a CPU
# tensor that passes the others.

def _cpu_inputs(n=256, hq=4, hkv=2, d=128):
    import torch
    bf = dict(dtype=torch.bfloat16)
    return (torch.zeros(hq, n, d, **bf), torch.zeros(hkv, n, d, **bf), torch.zeros(hkv, n, d, **bf))


def test_binding_rejects_bad_attention_arguments():
    import torch
    rbs, _ = _lib()
    shape = rbs.make_shape(256, 4, 2, 64)
    Q, K, V = _cpu_inputs()
    M = rbs.n_blocks(shape)
    counts = torch.zeros(4, M, dtype=torch.int32)
    indices = torch.zeros(4, rbs.rbs_index_capacity(M), dtype=torch.int32)
    cases = [
        (dict(Q=Q.float()), "must be torch.bfloat16"),
        (dict(Q=Q[:, :128]), "must have shape"),
        (dict(K=K[:1]), "must have shape"),
        (dict(V=V.transpose(0, 1).contiguous().transpose(0, 1)), "differ from K strides"),
        (dict(Q=Q.transpose(1, 2).contiguous().transpose(1, 2)), "contiguous last dimension"),
        (dict(counts=counts.long()), "must be torch.int32"),
        (dict(counts=counts[:, :-1]), "must have shape"),
        (dict(indices=indices[:, :-1]), "must have shape"),
        (dict(indices=indices.t().contiguous().t()), "must be contiguous"),
        (dict(O=torch.zeros(4, 256, 128, dtype=torch.float32)), "must be torch.bfloat16"),
        (dict(lse=torch.zeros(4, 255, dtype=torch.float32)), "must have shape"),
        (dict(), "must be on a GPU"),
    ]
    for override, msg in cases:
        args = dict(Q=Q, K=K, V=V, counts=counts, indices=indices, O=None, lse=None)
        args.update(override)
        with pytest.raises(ValueError, match=msg):
            rbs.rbs_sparse_prefill(shape, args["Q"], args["K"], args["V"], args["counts"], args["indices"],
                                   O=args["O"], lse=args["lse"], workspace=None)


def test_binding_rejects_bad_selection_and_stats_arguments():
    import torch
    rbs, _ = _lib()
    shape = rbs.make_shape(256, 4, 2, 64)
    Q, K, _ = _cpu_inputs()
    with pytest.raises(ValueError, match="must be torch.bfloat16"):
        rbs.rbs_block_stats(shape, K.half())
    with pytest.raises(ValueError, match="must have shape"):
        rbs.rbs_block_stats(shape, K[:, :64])
    with pytest.raises(ValueError, match="must be on a GPU"):
        rbs.rbs_block_stats(shape, K)
    M = rbs.n_blocks(shape)
    f32 = dict(dtype=torch.float32)
    stats = rbs.BlockStats(shape, torch.zeros(2, M, 128, **f32), torch.zeros(2, M, **f32), torch.zeros(2, M, **f32),
                           torch.zeros(2, 2, **f32), torch.zeros(rbs.rbs_summary_bytes(shape), dtype=torch.uint8))
    bad = rbs.BlockStats(shape, stats.centroids, stats.radii, stats.beta, stats.quantiles, stats.summary[:-16])
    with pytest.raises(ValueError, match="stats.summary must have shape"):
        rbs.rbs_select(shape, Q, bad, 0.9, 0.9, 1, 1, 0)
    with pytest.raises(ValueError, match="must be a BlockStats"):
        rbs.rbs_select(shape, Q, object(), 0.9, 0.9, 1, 1, 0)
    with pytest.raises(ValueError, match="Q must be on a GPU"):
        rbs.rbs_select(shape, Q, stats, 0.9, 0.9, 1, 1, 0)
    with pytest.raises(ValueError, match="stats.centroids must have shape"):
        rbs.rbs_stats_summarize(shape, rbs.BlockStats(shape, stats.centroids[:1], stats.radii, stats.beta,
                                                      stats.quantiles, stats.summary))


def test_binding_strides_come_from_the_tensors():
    rbs, _ = _lib()
    shape = rbs.make_shape(256, 4, 2, 64)
    tok_major = rbs._lib._with_strides(shape, q=(128, 512), kv=(128, 256))
    assert (tok_major.q_stride_head, tok_major.q_stride_tok, tok_major.kv_stride_head,
            tok_major.kv_stride_tok) == (128, 512, 128, 256)
    assert shape.q_stride_tok == 0  # the caller's shape is not modified
    shape.q_stride_tok = 384
    with pytest.raises(ValueError, match="disagrees"):
        rbs._lib._with_strides(shape, q=(128, 512))
