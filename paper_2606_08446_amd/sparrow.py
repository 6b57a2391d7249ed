"""Python binding of libsparrow (the C ABI declared in include/sparrow.h).

Argument marshalling only: every step of the sparse-decode path runs in the
library's HIP kernels.  PyTorch provides device memory and the stream.  The
functions named ``sparrow_*`` mirror the C entry points one to one (raw
pointers); the functions without the prefix take torch tensors, allocate the
workspace when none is given, and raise ``SparrowError`` on a negative status.

There is no fallback: if ``libsparrow.so`` has not been built, or no GPU is
visible, the tensor-level calls raise.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
# SPARROW_LIB selects another build of the library (the host-sanitizer build, for instance).
LIB_PATH = os.environ.get("SPARROW_LIB", os.path.join(_PKG, "libsparrow.so"))

SPARROW_OK = 0
SPARROW_EINVAL = -1
SPARROW_EUNSUPPORTED = -2
SPARROW_EWORKSPACE = -3
SPARROW_EHIP = -4
SPARROW_MAX_PAGES_PER_SEQ = 15360
SPARROW_MAX_BATCH = 8192
SPARROW_OUT_F32 = 0
SPARROW_OUT_BF16 = 1
SPARROW_LANDMARK_MINMAX = 0
SPARROW_LANDMARK_MEAN = 1
SPARROW_LOGITS_F32 = 0
SPARROW_LOGITS_BF16 = 1
SPARROW_OP_SCORE_TOPK = 0
SPARROW_OP_SPARSE_ATTN = 1
SPARROW_OP_DENSE_ATTN = 2
SPARROW_OP_DECODE_STEP = 3
SPARROW_NOALLOC_SCRATCH_BYTES = 32 << 20

EXPORTS = ("sparrow_page_meta_update", "sparrow_append_kv", "sparrow_page_score_topk",
           "sparrow_append_score_topk", "sparrow_sparse_decode_attn", "sparrow_dense_decode_attn",
           "sparrow_acceptance_rate", "sparrow_acceptance_rate_topk", "sparrow_tail_stats",
           "sparrow_stream_read", "sparrow_sparse_decode_attn_noalloc", "sparrow_decode_step",
           "sparrow_budget_bound", "sparrow_workspace_size", "sparrow_status_string")


class SparrowError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {status} ({status_string(status)})")
        self.status = status


class Shape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("max_pages_per_seq", ctypes.c_int32),
                ("num_phys_pages", ctypes.c_int64), ("landmark", ctypes.c_int32)]


class Schedule(ctypes.Structure):
    _fields_ = [("bin_tokens", ctypes.c_int32), ("n_bins", ctypes.c_int32),
                ("min_pages", ctypes.c_void_p), ("frac_num", ctypes.c_void_p),
                ("frac_den", ctypes.c_int32), ("sink_pages", ctypes.c_int32),
                ("local_pages", ctypes.c_int32)]


_lib = None
_p = ctypes.c_void_p
_i32 = ctypes.c_int32


def load():
    """Load libsparrow.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2606_08446_amd.build` (no fallback exists)")
    lib = ctypes.CDLL(LIB_PATH)
    sp = ctypes.POINTER(Shape)
    lib.sparrow_page_meta_update.argtypes = [sp, _p, _p, _p, _p, _p, _p]
    lib.sparrow_page_score_topk.argtypes = [sp, _p, _p, _p, _p, ctypes.POINTER(Schedule), _i32,
                                            _p, _p, _p, ctypes.c_size_t, _p]
    lib.sparrow_sparse_decode_attn.argtypes = [sp, _p, _p, _p, _p, _p, _p, _p, _i32,
                                               ctypes.c_float, _p, _i32, _p, ctypes.c_size_t, _p]
    lib.sparrow_dense_decode_attn.argtypes = [sp, _p, _p, _p, _p, _p, ctypes.c_float, _p, _i32,
                                              _p, ctypes.c_size_t, _p]
    lib.sparrow_append_kv.argtypes = [sp, _p, _p, _p, _p, _p, _p, _p, _p]
    lib.sparrow_append_score_topk.argtypes = [sp, _p, _p, _p, _p, _p, _p, _p, _p,
                                              ctypes.POINTER(Schedule), _i32, _p, _p, _p,
                                              ctypes.c_size_t, _p]
    lib.sparrow_acceptance_rate.argtypes = [ctypes.c_int64, _i32, _i32, _p, _p, ctypes.c_float,
                                            _p, _p]
    lib.sparrow_acceptance_rate_topk.argtypes = [ctypes.c_int64, _i32, _p, _p, _p, _p]
    lib.sparrow_tail_stats.argtypes = [ctypes.c_int64, _p, _p, _i32, _i32, ctypes.c_double, _p,
                                       _p, _p, _p]
    lib.sparrow_stream_read.argtypes = [_p, ctypes.c_int64, _p, _p]
    lib.sparrow_sparse_decode_attn_noalloc.argtypes = [sp, _p, _p, _p, _p, _p, _p, _p, _i32,
                                                       ctypes.c_float, _p, _i32, _p]
    lib.sparrow_decode_step.argtypes = [sp, _p, _p, _p, _p, _p, _p, _p, _p,
                                        ctypes.POINTER(Schedule), _i32, ctypes.c_float, _p, _p,
                                        _p, _i32, _p, ctypes.c_size_t, _p]
    for fn in EXPORTS[:12]:
        getattr(lib, fn).restype = ctypes.c_int
    lib.sparrow_budget_bound.argtypes = [_p, ctypes.c_int64, _i32, _i32, _i32, _p, _p, _i32, _p]
    lib.sparrow_budget_bound.restype = ctypes.c_int32
    lib.sparrow_workspace_size.argtypes = [sp, _i32, _i32]
    lib.sparrow_workspace_size.restype = ctypes.c_size_t
    lib.sparrow_status_string.argtypes = [_i32]
    lib.sparrow_status_string.restype = ctypes.c_char_p
    _lib = lib
    return lib


# ------------------------------------------------------------------ raw entry points (C names)
def sparrow_page_meta_update(shape, k_cache, block_table, seq_lens, first_pos, meta, stream):
    return load().sparrow_page_meta_update(ctypes.byref(shape), k_cache, block_table, seq_lens,
                                           first_pos, meta, stream)


def sparrow_page_score_topk(shape, q, meta, block_table, seq_lens, schedule, k_max, out_k,
                            out_idx, workspace, ws_bytes, stream):
    return load().sparrow_page_score_topk(ctypes.byref(shape), q, meta, block_table, seq_lens,
                                          ctypes.byref(schedule), k_max, out_k, out_idx,
                                          workspace, ws_bytes, stream)


def sparrow_append_kv(shape, k_new, v_new, k_cache, v_cache, block_table, seq_lens, meta, stream):
    return load().sparrow_append_kv(ctypes.byref(shape), k_new, v_new, k_cache, v_cache,
                                    block_table, seq_lens, meta, stream)


def sparrow_append_score_topk(shape, q, k_new, v_new, k_cache, v_cache, meta, block_table,
                              seq_lens, schedule, k_max, out_k, out_idx, workspace, ws_bytes,
                              stream):
    return load().sparrow_append_score_topk(ctypes.byref(shape), q, k_new, v_new, k_cache,
                                            v_cache, meta, block_table, seq_lens,
                                            ctypes.byref(schedule), k_max, out_k, out_idx,
                                            workspace, ws_bytes, stream)


def sparrow_sparse_decode_attn(shape, q, k_cache, v_cache, block_table, seq_lens, k, idx, k_max,
                               scale, out, out_dtype, workspace, ws_bytes, stream):
    return load().sparrow_sparse_decode_attn(ctypes.byref(shape), q, k_cache, v_cache,
                                             block_table, seq_lens, k, idx, k_max, scale, out,
                                             out_dtype, workspace, ws_bytes, stream)


def sparrow_sparse_decode_attn_noalloc(shape, q, k_cache, v_cache, block_table, seq_lens, k, idx,
                                       k_max, scale, out, out_dtype, stream):
    return load().sparrow_sparse_decode_attn_noalloc(ctypes.byref(shape), q, k_cache, v_cache,
                                                     block_table, seq_lens, k, idx, k_max, scale,
                                                     out, out_dtype, stream)


def sparrow_decode_step(shape, q, k_new, v_new, k_cache, v_cache, meta, block_table, seq_lens,
                        schedule, k_max, scale, out_k, out_idx, out, out_dtype, workspace,
                        ws_bytes, stream):
    return load().sparrow_decode_step(ctypes.byref(shape), q, k_new, v_new, k_cache, v_cache,
                                      meta, block_table, seq_lens, ctypes.byref(schedule), k_max,
                                      scale, out_k, out_idx, out, out_dtype, workspace, ws_bytes,
                                      stream)


def sparrow_dense_decode_attn(shape, q, k_cache, v_cache, block_table, seq_lens, scale, out,
                              out_dtype, workspace, ws_bytes, stream):
    return load().sparrow_dense_decode_attn(ctypes.byref(shape), q, k_cache, v_cache,
                                            block_table, seq_lens, scale, out, out_dtype,
                                            workspace, ws_bytes, stream)


def sparrow_acceptance_rate(num_tokens, vocab, logits_dtype, target, draft, inv_temperature,
                            alpha, stream):
    return load().sparrow_acceptance_rate(num_tokens, vocab, logits_dtype, target, draft,
                                          inv_temperature, alpha, stream)


def sparrow_acceptance_rate_topk(num_tokens, k, lp_target, lp_draft, alpha, stream):
    return load().sparrow_acceptance_rate_topk(num_tokens, k, lp_target, lp_draft, alpha, stream)


def sparrow_tail_stats(num_tokens, alpha, positions, bin_tokens, n_bins, percentile, quantile,
                       mean, count, stream):
    return load().sparrow_tail_stats(num_tokens, alpha, positions, bin_tokens, n_bins, percentile,
                                     quantile, mean, count, stream)


def sparrow_stream_read(src, nbytes, checksum, stream):
    return load().sparrow_stream_read(src, nbytes, checksum, stream)


def sparrow_budget_bound(seq_lens, num_seqs, page_size, bin_tokens, n_bins, min_pages, frac_num,
                         frac_den, budgets) -> int:
    return int(load().sparrow_budget_bound(seq_lens, num_seqs, page_size, bin_tokens, n_bins,
                                           min_pages, frac_num, frac_den, budgets))


def sparrow_workspace_size(shape, k_max, op) -> int:
    return int(load().sparrow_workspace_size(ctypes.byref(shape), k_max, op))


def sparrow_status_string(status) -> str:
    return load().sparrow_status_string(status).decode()


status_string = sparrow_status_string


# ------------------------------------------------------------------ host helpers
def make_shape(batch, num_q_heads, num_kv_heads, page_size, max_pages_per_seq, num_phys_pages,
               head_dim=128, landmark=SPARROW_LANDMARK_MINMAX) -> Shape:
    return Shape(batch, num_q_heads, num_kv_heads, head_dim, page_size, max_pages_per_seq,
                 num_phys_pages, landmark)


def shape_of(q, k_cache, block_table, landmark=SPARROW_LANDMARK_MINMAX) -> Shape:
    """Shape struct from tensors q [B][Hq][D], k_cache [P][Hkv][ps][D], block_table [B][M]."""
    B, Hq, D = q.shape
    P, Hkv, ps, _ = k_cache.shape
    return make_shape(B, Hq, Hkv, ps, block_table.shape[1], P, head_dim=D, landmark=landmark)


def new_meta(num_phys_pages, num_kv_heads, device, landmark=SPARROW_LANDMARK_MINMAX):
    """A zeroed metadata buffer of the given landmark: bf16 [P][Hkv][2][128] (min/max) or fp32
    [P][Hkv][128] (key sums) - 512 bytes per (page, head) either way."""
    import torch
    if landmark == SPARROW_LANDMARK_MEAN:
        return torch.zeros((num_phys_pages, num_kv_heads, 128), dtype=torch.float32, device=device)
    return torch.zeros((num_phys_pages, num_kv_heads, 2, 128), dtype=torch.bfloat16,
                       device=device)


def _host_i32(values) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(values, dtype=np.int64).astype(np.int32))


def budgets(seq_lens: Sequence[int], page_size: int, bin_tokens: int, min_pages: Sequence[int],
            frac_num: Sequence[int], frac_den: int):
    """(per-sequence schedule budgets int32 [B], their bound) from host-known lengths, computed
    by the library's sparrow_budget_bound (host code, no GPU needed)."""
    lens = _host_i32(seq_lens)
    mp, fn = _host_i32(min_pages), _host_i32(frac_num)
    out = np.zeros(len(lens), dtype=np.int32)
    rc = sparrow_budget_bound(lens.ctypes.data, len(lens), int(page_size), int(bin_tokens),
                              len(mp), mp.ctypes.data, fn.ctypes.data, int(frac_den),
                              out.ctypes.data)
    _check("sparrow_budget_bound", min(rc, 0))
    return out, rc


def budget_bound(seq_lens: Sequence[int], page_size: int, bin_tokens: int,
                 min_pages: Sequence[int], frac_num: Sequence[int], frac_den: int) -> int:
    """Largest schedule budget over host-known lengths (at least 1), to size ``k_max``."""
    return budgets(seq_lens, page_size, bin_tokens, min_pages, frac_num, frac_den)[1]


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(device=None) -> int:
    import torch
    return torch.cuda.current_stream(device).cuda_stream


def _check(fn: str, rc: int) -> None:
    if rc != SPARROW_OK:
        raise SparrowError(fn, rc)


def _workspace(nbytes: int, device):
    import torch
    return torch.empty(max(int(nbytes), 16), dtype=torch.uint8, device=device)


def _require_device(t):
    if not t.is_cuda:
        raise RuntimeError("libsparrow runs on the GPU only: tensors must be on a HIP device")


def _expect(t, name, dtype, shape, device):
    """Raise unless ``t`` is a contiguous tensor on ``device`` with exactly this dtype and shape.

    The C ABI receives bare pointers: the kernels index every buffer with the sizes in the
    shape struct, so a tensor of another dtype, shape or layout would be read or written
    out of bounds.  The tensor-level wrappers check each buffer before any launch."""
    if t is None:
        raise ValueError(f"{name} is required")
    _require_device(t)
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, the other tensors on {device}")
    if t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _expect_cache(q, k_cache, v_cache, block_table, seq_lens):
    """q bf16 [B][Hq][D]; k_cache and v_cache bf16 [P][Hkv][ps][D]; block_table int32
    [B][M]; seq_lens int32 [B].  Returns (B, Hq, Hkv, ps, D, P, M)."""
    import torch
    _require_device(q)
    dev = q.device
    if q.dim() != 3 or k_cache.dim() != 4 or block_table.dim() != 2:
        raise ValueError("q must be [B][Hq][D], the caches [P][Hkv][ps][D], block_table [B][M]")
    B, Hq, D = q.shape
    P, Hkv, ps, _ = k_cache.shape
    M = block_table.shape[1]
    _expect(q, "q", torch.bfloat16, (B, Hq, D), dev)
    _expect(k_cache, "k_cache", torch.bfloat16, (P, Hkv, ps, D), dev)
    if v_cache is not None:
        _expect(v_cache, "v_cache", torch.bfloat16, (P, Hkv, ps, D), dev)
    _expect(block_table, "block_table", torch.int32, (B, M), dev)
    _expect(seq_lens, "seq_lens", torch.int32, (B,), dev)
    return B, Hq, Hkv, ps, D, P, M


def _expect_meta(meta, P, Hkv, D, landmark, device):
    import torch
    if landmark == SPARROW_LANDMARK_MEAN:
        _expect(meta, "meta", torch.float32, (P, Hkv, D), device)
    else:
        _expect(meta, "meta", torch.bfloat16, (P, Hkv, 2, D), device)


def _expect_tables(min_pages, frac_num, device):
    import torch
    if min_pages.dim() != 1:
        raise ValueError("min_pages must be a 1-D table")
    _expect(min_pages, "min_pages", torch.int32, (min_pages.numel(),), device)
    _expect(frac_num, "frac_num", torch.int32, (min_pages.numel(),), device)


def _expect_out(out, out_dtype, shape, device):
    import torch
    dt = torch.float32 if out_dtype == SPARROW_OUT_F32 else torch.bfloat16
    _expect(out, "out", dt, shape, device)


# ------------------------------------------------------------------ tensor-level wrappers
def page_meta_update(k_cache, block_table, seq_lens, meta, first_pos=None, shape=None,
                     landmark=SPARROW_LANDMARK_MINMAX):
    """Rebuild (first_pos None) or update the page metadata in ``meta`` (in place)."""
    import torch
    _require_device(k_cache)
    dev = k_cache.device
    if k_cache.dim() != 4 or block_table.dim() != 2:
        raise ValueError("k_cache must be [P][Hkv][ps][D], block_table [B][M]")
    P, Hkv, ps, D = k_cache.shape
    B, M = block_table.shape
    _expect(k_cache, "k_cache", torch.bfloat16, (P, Hkv, ps, D), dev)
    _expect(block_table, "block_table", torch.int32, (B, M), dev)
    _expect(seq_lens, "seq_lens", torch.int32, (B,), dev)
    if first_pos is not None:
        _expect(first_pos, "first_pos", torch.int32, (B,), dev)
    _expect_meta(meta, P, Hkv, D, landmark, dev)
    if B == 0:   # nothing to launch (an empty tensor's data pointer is null)
        return meta
    if shape is None:
        shape = make_shape(B, Hkv, Hkv, ps, M, P, D, landmark=landmark)
    rc = sparrow_page_meta_update(shape, _ptr(k_cache), _ptr(block_table), _ptr(seq_lens),
                                  _ptr(first_pos), _ptr(meta), _stream(k_cache.device))
    _check("sparrow_page_meta_update", rc)
    return meta


def append_kv(k_new, v_new, k_cache, v_cache, block_table, seq_lens, meta,
              landmark=SPARROW_LANDMARK_MINMAX):
    """Write token ``seq_lens[b] - 1`` of every sequence into the caches and update the
    metadata of its page (all in place)."""
    import torch
    _require_device(k_cache)
    dev = k_cache.device
    if k_cache.dim() != 4 or block_table.dim() != 2:
        raise ValueError("k_cache must be [P][Hkv][ps][D], block_table [B][M]")
    P, Hkv, ps, D = k_cache.shape
    B, M = block_table.shape
    _expect(k_cache, "k_cache", torch.bfloat16, (P, Hkv, ps, D), dev)
    _expect(v_cache, "v_cache", torch.bfloat16, (P, Hkv, ps, D), dev)
    _expect(block_table, "block_table", torch.int32, (B, M), dev)
    _expect(seq_lens, "seq_lens", torch.int32, (B,), dev)
    _expect(k_new, "k_new", torch.bfloat16, (B, Hkv, D), dev)
    _expect(v_new, "v_new", torch.bfloat16, (B, Hkv, D), dev)
    _expect_meta(meta, P, Hkv, D, landmark, dev)
    if B == 0:
        return
    shape = make_shape(B, Hkv, Hkv, ps, M, P, D, landmark=landmark)
    rc = sparrow_append_kv(shape, _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache),
                           _ptr(block_table), _ptr(seq_lens), _ptr(meta), _stream(k_cache.device))
    _check("sparrow_append_kv", rc)


def page_score_topk(q, meta, block_table, seq_lens, k_cache_shape, min_pages, frac_num,
                    frac_den, bin_tokens, k_max, out_k=None, out_idx=None, workspace=None,
                    landmark=SPARROW_LANDMARK_MINMAX, sink_pages=0, local_pages=0):
    """Scores, budgets and top-k page lists.  Returns (k [B] int32, idx [B][Hkv][k_max] int32)."""
    import torch
    _require_device(q)
    dev = q.device
    P, Hkv, ps, D = k_cache_shape
    if q.dim() != 3 or block_table.dim() != 2:
        raise ValueError("q must be [B][Hq][D], block_table [B][M]")
    B, Hq, _ = q.shape
    M = block_table.shape[1]
    _expect(q, "q", torch.bfloat16, (B, Hq, D), dev)
    _expect(block_table, "block_table", torch.int32, (B, M), dev)
    _expect(seq_lens, "seq_lens", torch.int32, (B,), dev)
    _expect_meta(meta, P, Hkv, D, landmark, dev)
    _expect_tables(min_pages, frac_num, dev)
    shape = make_shape(B, Hq, Hkv, ps, M, P, D, landmark=landmark)
    sched = Schedule(int(bin_tokens), int(min_pages.numel()), _ptr(min_pages), _ptr(frac_num),
                     int(frac_den), int(sink_pages), int(local_pages))
    if out_k is None:
        out_k = torch.empty(B, dtype=torch.int32, device=dev)
    if out_idx is None:
        out_idx = torch.empty((B, Hkv, int(k_max)), dtype=torch.int32, device=dev)
    _expect(out_k, "out_k", torch.int32, (B,), dev)
    _expect(out_idx, "out_idx", torch.int32, (B, Hkv, int(k_max)), dev)
    if B == 0:
        return out_k, out_idx
    need = sparrow_workspace_size(shape, int(k_max), SPARROW_OP_SCORE_TOPK)
    if workspace is None:
        workspace = _workspace(need, dev)
    rc = sparrow_page_score_topk(shape, _ptr(q), _ptr(meta), _ptr(block_table), _ptr(seq_lens),
                                 sched, int(k_max), _ptr(out_k), _ptr(out_idx), _ptr(workspace),
                                 workspace.numel() * workspace.element_size(), _stream(dev))
    _check("sparrow_page_score_topk", rc)
    return out_k, out_idx


def sparse_decode_attn(q, k_cache, v_cache, block_table, seq_lens, k, idx, scale=None, out=None,
                       out_dtype=SPARROW_OUT_F32, workspace=None):
    """Attention over the selected pages.  Returns out [B][Hq][D] (fp32 or bf16)."""
    import torch
    B, Hq, Hkv, ps, D, P, M = _expect_cache(q, k_cache, v_cache, block_table, seq_lens)
    if idx.dim() != 3:
        raise ValueError("idx must be [B][Hkv][k_max]")
    k_max = int(idx.shape[2])
    _expect(k, "k", torch.int32, (B,), q.device)
    _expect(idx, "idx", torch.int32, (B, Hkv, k_max), q.device)
    shape = shape_of(q, k_cache, block_table)
    scale = 1.0 / math.sqrt(q.shape[2]) if scale is None else scale
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32 if out_dtype == SPARROW_OUT_F32
                          else torch.bfloat16, device=q.device)
    _expect_out(out, out_dtype, (B, Hq, D), q.device)
    if B == 0:
        return out
    need = sparrow_workspace_size(shape, k_max, SPARROW_OP_SPARSE_ATTN)
    if workspace is None:
        workspace = _workspace(need, q.device)
    rc = sparrow_sparse_decode_attn(shape, _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                    _ptr(block_table), _ptr(seq_lens), _ptr(k), _ptr(idx), k_max,
                                    float(scale), _ptr(out), int(out_dtype), _ptr(workspace),
                                    workspace.numel() * workspace.element_size(),
                                    _stream(q.device))
    _check("sparrow_sparse_decode_attn", rc)
    return out


def dense_decode_attn(q, k_cache, v_cache, block_table, seq_lens, scale=None, out=None,
                      out_dtype=SPARROW_OUT_F32, workspace=None):
    """Dense paged decode attention.  Returns out [B][Hq][D] (fp32 or bf16)."""
    import torch
    B, Hq, Hkv, ps, D, P, M = _expect_cache(q, k_cache, v_cache, block_table, seq_lens)
    shape = shape_of(q, k_cache, block_table)
    scale = 1.0 / math.sqrt(q.shape[2]) if scale is None else scale
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32 if out_dtype == SPARROW_OUT_F32
                          else torch.bfloat16, device=q.device)
    _expect_out(out, out_dtype, (B, Hq, D), q.device)
    if B == 0:
        return out
    need = sparrow_workspace_size(shape, 0, SPARROW_OP_DENSE_ATTN)
    if workspace is None:
        workspace = _workspace(need, q.device)
    rc = sparrow_dense_decode_attn(shape, _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                   _ptr(block_table), _ptr(seq_lens), float(scale), _ptr(out),
                                   int(out_dtype), _ptr(workspace),
                                   workspace.numel() * workspace.element_size(),
                                   _stream(q.device))
    _check("sparrow_dense_decode_attn", rc)
    return out


def acceptance_rate(target, draft, inv_temperature=1.0, alpha=None):
    """Per-token acceptance rate of logit rows ``[T][V]`` (float32 or bfloat16, same dtype).
    Returns alpha fp32 ``[T]``."""
    import torch
    _require_device(target)
    if target.dtype != draft.dtype or target.shape != draft.shape:
        raise ValueError("target and draft logits need the same dtype and shape")
    dt = {torch.float32: SPARROW_LOGITS_F32, torch.bfloat16: SPARROW_LOGITS_BF16}[target.dtype]
    T, V = target.shape
    if not (target.is_contiguous() and draft.is_contiguous()):
        raise ValueError("logit rows must be contiguous")
    _require_device(draft)
    if draft.device != target.device:
        raise ValueError("target and draft logits must be on one device")
    if alpha is None:
        alpha = torch.empty(T, dtype=torch.float32, device=target.device)
    _expect(alpha, "alpha", torch.float32, (T,), target.device)
    if T == 0:   # nothing to launch (an empty tensor's data pointer is null)
        return alpha
    _check("sparrow_acceptance_rate", sparrow_acceptance_rate(
        T, V, dt, _ptr(target), _ptr(draft), float(inv_temperature), _ptr(alpha),
        _stream(target.device)))
    return alpha


def acceptance_rate_topk(lp_target, lp_draft, alpha=None):
    """Top-K approximation from log-probabilities ``[T][K]`` (fp32).  Returns alpha ``[T]``."""
    import torch
    _require_device(lp_target)
    if lp_target.dim() != 2:
        raise ValueError("log-probabilities must be [T][K]")
    T, K = lp_target.shape
    dev = lp_target.device
    _expect(lp_target, "lp_target", torch.float32, (T, K), dev)
    _expect(lp_draft, "lp_draft", torch.float32, (T, K), dev)
    if alpha is None:
        alpha = torch.empty(T, dtype=torch.float32, device=dev)
    _expect(alpha, "alpha", torch.float32, (T,), dev)
    if T == 0:
        return alpha
    _check("sparrow_acceptance_rate_topk", sparrow_acceptance_rate_topk(
        T, K, _ptr(lp_target), _ptr(lp_draft), _ptr(alpha), _stream(lp_target.device)))
    return alpha


def tail_stats(alpha, positions, bin_tokens, n_bins, percentile=5.0):
    """(quantile fp64 [n_bins], mean fp64 [n_bins], count int64 [n_bins]) on the device."""
    import torch
    _require_device(alpha)
    dev = alpha.device
    _expect(alpha, "alpha", torch.float32, (alpha.numel(),), dev)
    _expect(positions, "positions", torch.int32, (alpha.numel(),), dev)
    q = torch.empty(n_bins, dtype=torch.float64, device=dev)
    m = torch.empty(n_bins, dtype=torch.float64, device=dev)
    c = torch.empty(n_bins, dtype=torch.int64, device=dev)
    _check("sparrow_tail_stats", sparrow_tail_stats(
        alpha.numel(), _ptr(alpha), _ptr(positions), int(bin_tokens), int(n_bins),
        float(percentile), _ptr(q), _ptr(m), _ptr(c), _stream(dev)))
    return q, m, c


def stream_read(buf, checksum=None):
    """Read a device buffer once through the library's streaming reference; returns the
    uint32 checksum tensor (sum of the buffer's 32-bit words modulo 2^32, added to
    ``checksum`` when given, else to a new zero)."""
    import torch
    _require_device(buf)
    if not buf.is_contiguous():
        raise ValueError("buf must be contiguous")
    if checksum is None:
        checksum = torch.zeros(1, dtype=torch.int32, device=buf.device)
    _expect(checksum, "checksum", torch.int32, (1,), buf.device)
    _check("sparrow_stream_read", sparrow_stream_read(
        _ptr(buf), buf.numel() * buf.element_size(), _ptr(checksum), _stream(buf.device)))
    return checksum


class SparseDecodeStep:
    """One layer's sparse decode step with preallocated buffers.

    ``run(first_pos)`` enqueues: metadata update of the pages touched since
    ``first_pos`` (skipped when None), page scoring + top-k, sparse attention."""

    def __init__(self, q, k_cache, v_cache, block_table, seq_lens, meta, min_pages, frac_num,
                 frac_den, bin_tokens, k_max, scale=None, landmark=SPARROW_LANDMARK_MINMAX,
                 sink_pages=0, local_pages=0):
        import torch
        B, Hq, Hkv, ps, D, P, M = _expect_cache(q, k_cache, v_cache, block_table, seq_lens)
        _expect_meta(meta, P, Hkv, D, landmark, q.device)
        _expect_tables(min_pages, frac_num, q.device)
        self.q, self.k_cache, self.v_cache = q, k_cache, v_cache
        self.block_table, self.seq_lens, self.meta = block_table, seq_lens, meta
        self.shape = shape_of(q, k_cache, block_table, landmark=landmark)
        self.sched = Schedule(int(bin_tokens), int(min_pages.numel()), _ptr(min_pages),
                              _ptr(frac_num), int(frac_den), int(sink_pages), int(local_pages))
        self._tables = (min_pages, frac_num)
        self.k_max = int(k_max)
        self.scale = 1.0 / math.sqrt(q.shape[2]) if scale is None else float(scale)
        dev = q.device
        B, Hkv = q.shape[0], k_cache.shape[1]
        self.k = torch.empty(B, dtype=torch.int32, device=dev)
        self.idx = torch.empty((B, Hkv, self.k_max), dtype=torch.int32, device=dev)
        self.out = torch.empty(q.shape, dtype=torch.float32, device=dev)
        self.ws_score = _workspace(sparrow_workspace_size(self.shape, self.k_max,
                                                          SPARROW_OP_SCORE_TOPK), dev)
        self.ws_attn = _workspace(sparrow_workspace_size(self.shape, self.k_max,
                                                         SPARROW_OP_SPARSE_ATTN), dev)
        # allocated here, not on first use, so that a first call under graph capture
        # allocates nothing
        self.ws_step = _workspace(sparrow_workspace_size(self.shape, self.k_max,
                                                         SPARROW_OP_DECODE_STEP), dev)

    # Every method takes an optional ``seq_lens`` tensor that replaces the one given at
    # construction for that call (a decode loop advances the lengths step by step).
    def _lens(self, seq_lens):
        import torch
        if seq_lens is None:
            return _ptr(self.seq_lens)
        _expect(seq_lens, "seq_lens", torch.int32, tuple(self.seq_lens.shape), self.q.device)
        return _ptr(seq_lens)

    def _rows(self, k_new, v_new):
        """The decoded token's rows: bf16 [B][Hkv][D] each."""
        import torch
        want = (self.q.shape[0], self.k_cache.shape[1], self.q.shape[2])
        _expect(k_new, "k_new", torch.bfloat16, want, self.q.device)
        _expect(v_new, "v_new", torch.bfloat16, want, self.q.device)

    def meta_update(self, first_pos, stream, seq_lens=None):
        import torch
        if first_pos is not None:
            _expect(first_pos, "first_pos", torch.int32, tuple(self.seq_lens.shape),
                    self.q.device)
        _check("sparrow_page_meta_update", sparrow_page_meta_update(
            self.shape, _ptr(self.k_cache), _ptr(self.block_table), self._lens(seq_lens),
            _ptr(first_pos), _ptr(self.meta), stream))

    def append(self, k_new, v_new, stream, seq_lens=None):
        """Write the decoded token's K/V rows and update its page's metadata."""
        self._rows(k_new, v_new)
        _check("sparrow_append_kv", sparrow_append_kv(
            self.shape, _ptr(k_new), _ptr(v_new), _ptr(self.k_cache), _ptr(self.v_cache),
            _ptr(self.block_table), self._lens(seq_lens), _ptr(self.meta), stream))

    def score_topk(self, stream, seq_lens=None):
        _check("sparrow_page_score_topk", sparrow_page_score_topk(
            self.shape, _ptr(self.q), _ptr(self.meta), _ptr(self.block_table),
            self._lens(seq_lens), self.sched, self.k_max, _ptr(self.k), _ptr(self.idx),
            _ptr(self.ws_score), self.ws_score.numel(), stream))

    def append_score_topk(self, k_new, v_new, stream, seq_lens=None):
        """Append the decoded token (k_new/v_new [B][Hkv][D]) and select pages, fused."""
        self._rows(k_new, v_new)
        _check("sparrow_append_score_topk", sparrow_append_score_topk(
            self.shape, _ptr(self.q), _ptr(k_new), _ptr(v_new), _ptr(self.k_cache),
            _ptr(self.v_cache), _ptr(self.meta), _ptr(self.block_table), self._lens(seq_lens),
            self.sched, self.k_max, _ptr(self.k), _ptr(self.idx), _ptr(self.ws_score),
            self.ws_score.numel(), stream))

    def attend(self, stream, seq_lens=None):
        _check("sparrow_sparse_decode_attn", sparrow_sparse_decode_attn(
            self.shape, _ptr(self.q), _ptr(self.k_cache), _ptr(self.v_cache),
            _ptr(self.block_table), self._lens(seq_lens), _ptr(self.k), _ptr(self.idx),
            self.k_max, self.scale, _ptr(self.out), SPARROW_OUT_F32, _ptr(self.ws_attn),
            self.ws_attn.numel(), stream))

    def decode_step(self, k_new, v_new, stream, seq_lens=None):
        """The whole step in one call (sparrow_decode_step): append the decoded token
        (k_new/v_new [B][Hkv][D], or both None for no append), select pages, attend; the
        same results as append_score_topk (or score_topk) followed by attend."""
        if (k_new is None) != (v_new is None):
            raise ValueError("k_new and v_new are both given or both None")
        if k_new is not None:
            self._rows(k_new, v_new)
        _check("sparrow_decode_step", sparrow_decode_step(
            self.shape, _ptr(self.q), _ptr(k_new), _ptr(v_new), _ptr(self.k_cache),
            _ptr(self.v_cache), _ptr(self.meta), _ptr(self.block_table), self._lens(seq_lens),
            self.sched, self.k_max, self.scale, _ptr(self.k), _ptr(self.idx), _ptr(self.out),
            SPARROW_OUT_F32, _ptr(self.ws_step), self.ws_step.numel(), stream))
        return self.out

    def run(self, first_pos=None, stream=None):
        stream = _stream(self.q.device) if stream is None else stream
        if first_pos is not None:
            self.meta_update(first_pos, stream)
        self.score_topk(stream)
        self.attend(stream)
        return self.out
