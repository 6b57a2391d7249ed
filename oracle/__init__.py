"""CPU oracle for Sparrow's sparse-decode step (arXiv 2606.08446).

TEST INFRASTRUCTURE ONLY: the plain C reference in ``sparrow_oracle.c`` behind
numpy-level wrappers.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package; the GPU library never calls it and
shares no code with it.

Every function takes numpy arrays: bf16 tensors travel as ``uint16`` bit
patterns, indices as ``int32``.  Layouts are those of ``sparrow_oracle.c``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# SPARROW_ORACLE_LIB lets the mutation tests load a deliberately broken build.
_LIB_PATH = os.environ.get("SPARROW_ORACLE_LIB", os.path.join(_HERE, "liboracle.so"))
_lib = None

_i32 = ctypes.c_int32
_p = ctypes.c_void_p


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        subprocess.check_call(["make", "-s", "-C", _HERE])
    lib = ctypes.CDLL(_LIB_PATH)
    lib.oracle_budget.argtypes = [_i32, _i32, _i32, _i32, _p, _p, _i32]
    lib.oracle_budget.restype = _i32
    lib.oracle_budgets.argtypes = [_i32, _p, _i32, _i32, _i32, _p, _p, _i32, _p]
    lib.oracle_budgets.restype = None
    lib.oracle_page_meta.argtypes = [_i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p, _p]
    lib.oracle_page_meta.restype = None
    lib.oracle_append_kv.argtypes = [_i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p, _p, _p, _p]
    lib.oracle_append_kv.restype = None
    lib.oracle_page_scores.argtypes = [_i32, _i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p,
                                       _p, _p]
    lib.oracle_page_scores.restype = None
    lib.oracle_topk.argtypes = [_p, _i32, _i32, _p]
    lib.oracle_topk.restype = None
    lib.oracle_select.argtypes = [_i32, _i32, _i32, _i32, _p, _p, _p, _i32, _p]
    lib.oracle_select.restype = None
    lib.oracle_attention.argtypes = [_i32, _i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p, _p,
                                     _p, _p, _i32, ctypes.c_double, _p]
    lib.oracle_attention.restype = None
    lib.oracle_weight_sum.argtypes = [_i32, ctypes.c_int64, _p, _p, ctypes.c_double]
    lib.oracle_weight_sum.restype = ctypes.c_double
    lib.oracle_acceptance.argtypes = [ctypes.c_int64, _i32, _i32, _p, _p, ctypes.c_double, _p]
    lib.oracle_acceptance.restype = None
    lib.oracle_acceptance_topk.argtypes = [ctypes.c_int64, _i32, _p, _p, _p]
    lib.oracle_acceptance_topk.restype = None
    lib.oracle_tail_stats.argtypes = [ctypes.c_int64, _p, _p, _i32, _i32, ctypes.c_double, _p, _p,
                                      _p]
    lib.oracle_tail_stats.restype = None
    lib.oracle_page_key_sums.argtypes = [_i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p, _p]
    lib.oracle_page_key_sums.restype = None
    lib.oracle_page_scores_mean.argtypes = [_i32, _i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p,
                                            _p, _p]
    lib.oracle_page_scores_mean.restype = None
    lib.oracle_select_forced.argtypes = [_i32, _i32, _i32, _i32, _p, _p, _p, _i32, _i32, _i32, _p]
    lib.oracle_select_forced.restype = None
    lib.oracle_set_num_threads.argtypes = [_i32]
    lib.oracle_set_num_threads.restype = None
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = _i32
    _lib = lib
    return lib


def _c(a, dtype):
    """Contiguous array of ``dtype`` and its address (the array is returned to keep it alive)."""
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's parallel loops from now on (default: every host core)."""
    _load().oracle_set_num_threads(int(n))


def budget(L, ps, bin_tokens, min_pages, frac_num, frac_den) -> int:
    """Page budget of one sequence of ``L`` tokens (Sec. 3.2 schedule)."""
    mp, mpp = _c(min_pages, np.int32)
    fn, fnp = _c(frac_num, np.int32)
    return int(_load().oracle_budget(int(L), int(ps), int(bin_tokens), len(mp), mpp, fnp,
                                     int(frac_den)))


def budgets(seq_lens, ps, bin_tokens, min_pages, frac_num, frac_den) -> np.ndarray:
    sl, slp = _c(seq_lens, np.int32)
    mp, mpp = _c(min_pages, np.int32)
    fn, fnp = _c(frac_num, np.int32)
    out = np.zeros(len(sl), np.int32)
    _load().oracle_budgets(len(sl), slp, int(ps), int(bin_tokens), len(mp), mpp, fnp,
                           int(frac_den), out.ctypes.data)
    return out


def page_meta(k_cache, block_table, seq_lens, first_pos=None, meta=None) -> np.ndarray:
    """Min/max key metadata ``[P][Hkv][2][D]`` (uint16 bf16 bits).

    With ``first_pos`` given, only pages overlapping ``[first_pos[b], L_b)`` are
    recomputed in a copy of ``meta``; otherwise every page is built."""
    P, Hkv, ps, D = k_cache.shape
    B, max_pages = block_table.shape
    kc, kcp = _c(k_cache, np.uint16)
    bt, btp = _c(block_table, np.int32)
    sl, slp = _c(seq_lens, np.int32)
    if meta is None:
        out = np.zeros((P, Hkv, 2, D), np.uint16)
    else:
        out = np.array(meta, dtype=np.uint16, copy=True, order="C")
    fp_arr, fpp = (None, None) if first_pos is None else _c(first_pos, np.int32)
    _load().oracle_page_meta(B, Hkv, D, ps, max_pages, kcp, btp, slp, fpp, out.ctypes.data)
    return out


def append_kv(k_new, v_new, k_cache, v_cache, block_table, seq_lens, meta, inplace=False,
              landmark="minmax"):
    """(k_cache, v_cache, meta) after writing token ``L_b - 1`` of every sequence (rows
    ``k_new``/``v_new`` ``[B][Hkv][D]``) and rebuilding the metadata of its page: copies, or
    the given arrays updated in place (C-contiguous uint16) with ``inplace``.  With
    ``landmark="mean"`` ``meta`` is the fp32 key-sum array ``[P][Hkv][D]``."""
    if landmark == "mean":
        P, Hkv, ps, D = k_cache.shape
        scratch = np.zeros((P, Hkv, 2, D), np.uint16)
        kc, vc, _ = append_kv(k_new, v_new, k_cache, v_cache, block_table, seq_lens, scratch,
                              inplace=inplace)
        lens = np.asarray(seq_lens, np.int32)
        first = np.where((lens >= 1) & (lens <= ps * block_table.shape[1]), lens - 1,
                         np.iinfo(np.int32).max).astype(np.int32)
        sums = page_key_sums(kc, block_table, np.minimum(lens, ps * block_table.shape[1]),
                             first_pos=first, sums=meta, inplace=inplace)
        return kc, vc, sums
    P, Hkv, ps, D = k_cache.shape
    B, max_pages = block_table.shape
    kn, knp = _c(k_new, np.uint16)
    vn, vnp = _c(v_new, np.uint16)
    if inplace:
        for a in (k_cache, v_cache, meta):
            if a.dtype != np.uint16 or not a.flags.c_contiguous:
                raise ValueError("in-place append needs C-contiguous uint16 arrays")
        kc, vc, mt = k_cache, v_cache, meta
    else:
        kc = np.array(k_cache, dtype=np.uint16, copy=True, order="C")
        vc = np.array(v_cache, dtype=np.uint16, copy=True, order="C")
        mt = np.array(meta, dtype=np.uint16, copy=True, order="C")
    bt, btp = _c(block_table, np.int32)
    sl, slp = _c(seq_lens, np.int32)
    _load().oracle_append_kv(B, Hkv, D, ps, max_pages, knp, vnp, kc.ctypes.data, vc.ctypes.data,
                             btp, slp, mt.ctypes.data)
    return kc, vc, mt


def page_scores(q, meta, block_table, seq_lens, ps, fp64=True):
    """(scores32, scores64), each ``[B][Hkv][max_pages]``; entries past ``n_b`` are NaN.
    ``fp64=False`` skips the fp64 adjudication copy (scores64 is then None)."""
    B, Hq, D = q.shape
    P, Hkv, _, _ = meta.shape
    max_pages = block_table.shape[1]
    qq, qp = _c(q, np.uint16)
    mm, mp = _c(meta, np.uint16)
    bt, btp = _c(block_table, np.int32)
    sl, slp = _c(seq_lens, np.int32)
    s32 = np.full((B, Hkv, max_pages), np.nan, np.float32)
    s64 = np.full((B, Hkv, max_pages), np.nan, np.float64) if fp64 else None
    _load().oracle_page_scores(B, Hq, Hkv, D, ps, max_pages, qp, mp, btp, slp,
                               s32.ctypes.data, None if s64 is None else s64.ctypes.data)
    return s32, s64


def topk(scores, k) -> np.ndarray:
    """Indices of the ``k`` largest scores (ties to the lower index), ascending."""
    s, sp = _c(scores, np.float32)
    k = min(int(k), len(s))
    out = np.zeros(max(k, 0), np.int32)
    _load().oracle_topk(sp, len(s), k, out.ctypes.data)
    return out


def select(seq_lens, k_of_seq, scores32, ps, k_max) -> np.ndarray:
    """Top-k page lists ``[B][Hkv][k_max]`` (ascending, padded with -1)."""
    B, Hkv, max_pages = scores32.shape
    sl, slp = _c(seq_lens, np.int32)
    kk, kp = _c(k_of_seq, np.int32)
    s, sp = _c(scores32, np.float32)
    idx = np.zeros((B, Hkv, k_max), np.int32)
    _load().oracle_select(B, Hkv, ps, max_pages, slp, kp, sp, int(k_max), idx.ctypes.data)
    return idx


def attention(q, k_cache, v_cache, block_table, seq_lens, scale, k_of_seq=None, idx=None):
    """fp64 attention output ``[B][Hq][D]``; dense when ``idx`` is None."""
    B, Hq, D = q.shape
    P, Hkv, ps, _ = k_cache.shape
    max_pages = block_table.shape[1]
    qq, qp = _c(q, np.uint16)
    kc, kcp = _c(k_cache, np.uint16)
    vc, vcp = _c(v_cache, np.uint16)
    bt, btp = _c(block_table, np.int32)
    sl, slp = _c(seq_lens, np.int32)
    out = np.zeros((B, Hq, D), np.float64)
    if idx is None:
        kp = ip = None
        k_max = 0
    else:
        kk, kp = _c(k_of_seq, np.int32)
        ii, ip = _c(idx, np.int32)
        k_max = ii.shape[2]
    _load().oracle_attention(B, Hq, Hkv, D, ps, max_pages, qp, kcp, vcp, btp, slp, kp, ip,
                             int(k_max), float(scale), out.ctypes.data)
    return out


def weight_sum(qj, keys, scale) -> float:
    """Sum of the softmax weights of one query over ``keys`` ``[n][D]``."""
    qq, qp = _c(qj, np.uint16)
    kk, kp = _c(keys, np.uint16)
    return float(_load().oracle_weight_sum(kk.shape[1], kk.shape[0], qp, kp, float(scale)))


def sparse_step(q, k_cache, v_cache, block_table, seq_lens, schedule, k_max, scale):
    """The whole sparse step on the CPU: meta, scores, budget, top-k, attention.

    ``schedule`` is ``(bin_tokens, min_pages, frac_num, frac_den)``.
    Returns a dict with every intermediate."""
    ps = k_cache.shape[2]
    bin_tokens, min_pages, frac_num, frac_den = schedule
    meta = page_meta(k_cache, block_table, seq_lens)
    s32, s64 = page_scores(q, meta, block_table, seq_lens, ps)
    k = budgets(seq_lens, ps, bin_tokens, min_pages, frac_num, frac_den)
    k = np.minimum(k, k_max).astype(np.int32)
    idx = select(seq_lens, k, s32, ps, k_max)
    out = attention(q, k_cache, v_cache, block_table, seq_lens, scale, k, idx)
    return {"meta": meta, "scores32": s32, "scores64": s64, "k": k, "idx": idx, "out": out}


# ----------------------------------------------------------------- acceptance rate (Sec. 3.1)
def acceptance(target, draft, inv_temp=1.0) -> np.ndarray:
    """Per-token acceptance rate ``sum_x min(p(x), q(x))`` (Eq. 1), fp64 ``[T]``.

    ``target``/``draft``: logit rows ``[T][V]``, float32 or bf16 bit patterns (uint16)."""
    if target.dtype == np.uint16:
        dtype, npt = 1, np.uint16
    else:
        dtype, npt = 0, np.float32
    tg, tgp = _c(target, npt)
    dr, drp = _c(draft, npt)
    T, V = tg.shape
    out = np.zeros(T, np.float64)
    _load().oracle_acceptance(T, V, dtype, tgp, drp, float(inv_temp), out.ctypes.data)
    return out


def acceptance_topk(lp_target, lp_draft) -> np.ndarray:
    """The top-K approximation from normalised log-probabilities ``[T][K]`` (fp32)."""
    a, ap = _c(lp_target, np.float32)
    b, bp = _c(lp_draft, np.float32)
    T, K = a.shape
    out = np.zeros(T, np.float64)
    _load().oracle_acceptance_topk(T, K, ap, bp, out.ctypes.data)
    return out


def tail_stats(alpha, positions, bin_tokens, n_bins, pct):
    """(quantile fp64 [n_bins], mean fp64 [n_bins], count int64 [n_bins]) of ``alpha`` (fp32)
    grouped by position bin; the ``pct``-percentile with linear interpolation."""
    a, ap = _c(alpha, np.float32)
    ps_, pp = _c(positions, np.int32)
    q = np.zeros(n_bins, np.float64)
    m = np.zeros(n_bins, np.float64)
    c = np.zeros(n_bins, np.int64)
    _load().oracle_tail_stats(len(a), ap, pp, int(bin_tokens), int(n_bins), float(pct),
                              q.ctypes.data, m.ctypes.data, c.ctypes.data)
    return q, m, c


# ----------------------------------------------------------------- selector variants
def page_key_sums(k_cache, block_table, seq_lens, first_pos=None, sums=None, inplace=False):
    """Mean-landmark metadata: fp32 key sums ``[P][Hkv][D]`` of the pages overlapping
    ``[first_pos[b], L_b)`` (all pages without ``first_pos``), updated in a copy of ``sums``
    (or in place)."""
    P, Hkv, ps, D = k_cache.shape
    B, max_pages = block_table.shape
    kc, kcp = _c(k_cache, np.uint16)
    bt, btp = _c(block_table, np.int32)
    sl, slp = _c(seq_lens, np.int32)
    if sums is None:
        out = np.zeros((P, Hkv, D), np.float32)
    elif inplace:
        if sums.dtype != np.float32 or not sums.flags.c_contiguous:
            raise ValueError("in-place update needs a C-contiguous float32 array")
        out = sums
    else:
        out = np.array(sums, dtype=np.float32, copy=True, order="C")
    fp_arr, fpp = (None, None) if first_pos is None else _c(first_pos, np.int32)
    _load().oracle_page_key_sums(B, Hkv, D, ps, max_pages, kcp, btp, slp, fpp, out.ctypes.data)
    return out


def page_scores_mean(q, sums, block_table, seq_lens, ps, fp64=True):
    """Mean-landmark page scores (scores32, scores64), each ``[B][Hkv][max_pages]``;
    ``fp64=False`` skips the fp64 copy (scores64 is then None)."""
    B, Hq, D = q.shape
    P, Hkv, _ = sums.shape
    max_pages = block_table.shape[1]
    qq, qp = _c(q, np.uint16)
    ss, sp_ = _c(sums, np.float32)
    bt, btp = _c(block_table, np.int32)
    sl, slp = _c(seq_lens, np.int32)
    s32 = np.full((B, Hkv, max_pages), np.nan, np.float32)
    s64 = np.full((B, Hkv, max_pages), np.nan, np.float64) if fp64 else None
    _load().oracle_page_scores_mean(B, Hq, Hkv, D, ps, max_pages, qp, sp_, btp, slp,
                                    s32.ctypes.data, None if s64 is None else s64.ctypes.data)
    return s32, s64


def select_forced(seq_lens, k_of_seq, scores32, ps, k_max, sink, local) -> np.ndarray:
    """Top-k page lists with pages ``[0, sink)`` and ``[n - local, n)`` forced first."""
    B, Hkv, max_pages = scores32.shape
    sl, slp = _c(seq_lens, np.int32)
    kk, kp = _c(k_of_seq, np.int32)
    sc, scp = _c(scores32, np.float32)
    out = np.zeros((B, Hkv, k_max), np.int32)
    _load().oracle_select_forced(B, Hkv, ps, max_pages, slp, kp, scp, int(sink), int(local),
                                 int(k_max), out.ctypes.data)
    return out

