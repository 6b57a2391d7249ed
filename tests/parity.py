"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
and compare with the CPU oracle on the same seeded inputs.

Tolerances: page indices bit-exact, except pages whose fp64 score differs from
the k-th score by a nonzero relative gap below 1e-5 (near ties; exact ties are
never excused); attention outputs within 1e-2 max-abs and 2e-3 mean-abs of the
fp64 oracle; metadata bit-exact.
"""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle
from paper_2606_08446_amd import sparrow as S
from paper_2606_08446_amd import workloads as W

MAX_ABS = 1e-2
MEAN_ABS = 2e-3
NEAR_TIE = 1e-5
SCALE = 1.0 / math.sqrt(128.0)


def log(msg):
    print(msg, flush=True)


def gpu_run(inp: W.Inputs, k_max: int, dense=True, out_dtype=S.SPARROW_OUT_F32):
    """Meta rebuild, score + top-k, sparse and dense attention on the GPU; host copies."""
    meta = torch.zeros((inp.num_phys_pages, inp.workload.num_kv_heads, 2, 128),
                       dtype=torch.bfloat16, device=inp.q.device)
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta)
    s = inp.workload.schedule
    k, idx = S.page_score_topk(inp.q, meta, inp.block_table, inp.seq_lens, inp.k_cache.shape,
                               inp.min_pages, inp.frac_num, s.frac_den, s.bin_tokens, k_max)
    out_s = S.sparse_decode_attn(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                                 k, idx, SCALE, out_dtype=out_dtype)
    out_d = None
    if dense:
        out_d = S.dense_decode_attn(inp.q, inp.k_cache, inp.v_cache, inp.block_table,
                                    inp.seq_lens, SCALE, out_dtype=out_dtype)
    torch.cuda.synchronize()
    r = dict(meta=W.bf16_bits(meta), k=k.cpu().numpy(), idx=idx.cpu().numpy(),
             out_sparse=out_s.float().cpu().numpy().astype(np.float64))
    if dense:
        r["out_dense"] = out_d.float().cpu().numpy().astype(np.float64)
    return r


def host(inp: W.Inputs):
    return dict(q=W.bf16_bits(inp.q), k=W.bf16_bits(inp.k_cache), v=W.bf16_bits(inp.v_cache),
                bt=inp.block_table.cpu().numpy(), lens=inp.seq_lens.cpu().numpy())


def used_pages(bt, lens, ps):
    pages = []
    for b, L in enumerate(lens):
        pages.extend(int(x) for x in bt[b, :(int(L) + ps - 1) // ps])
    return np.array(sorted(set(pages)), dtype=np.int64)


def check_meta(gpu_meta, ora_meta, bt, lens, ps):
    pages = used_pages(bt, lens, ps)
    if len(pages):
        np.testing.assert_array_equal(gpu_meta[pages], ora_meta[pages])


def oracle_budgets(lens, ps, bin_tokens, min_pages, frac_num, frac_den, k_max,
                   capped=False):
    """The oracle's schedule budgets, uncapped.  Unless a test caps k_max on purpose
    (capped=True), k_max must cover every budget: a k_max sized below the schedule would
    truncate the budgets on both sides alike and hide the error."""
    k = oracle.budgets(lens, ps, bin_tokens, min_pages, frac_num, frac_den)
    if capped:
        return np.minimum(k, k_max).astype(np.int32)
    assert int(np.max(k, initial=0)) <= k_max, ("k_max below a schedule budget", k_max)
    return k.astype(np.int32)


def rank_boundary(s32_row, s64_row, n, k):
    """fp64 score of the oracle's k-th page (ranking by fp32 score, ties to lower index)."""
    order = sorted(range(n), key=lambda p: (-float(s32_row[p]), p))
    return float(s64_row[order[k - 1]])


def check_indices(gpu_k, gpu_idx, ora_k, ora_idx, s32, s64, lens, ps, k_max):
    """Bit-exact page lists with the near-tie excuse.  Returns the number of excused pages."""
    np.testing.assert_array_equal(gpu_k, ora_k)
    excused = 0
    B, Hkv, _ = gpu_idx.shape
    for b in range(B):
        n = (int(lens[b]) + ps - 1) // ps
        k = int(ora_k[b])
        for h in range(Hkv):
            g = gpu_idx[b, h]
            o = ora_idx[b, h]
            assert (g[k:] == -1).all(), (b, h, "padding")
            gk = g[:k]
            assert (np.diff(gk) > 0).all(), (b, h, "not strictly ascending")
            assert k == 0 or (gk[0] >= 0 and gk[-1] < n), (b, h, "out of range")
            if np.array_equal(gk, o[:k]):
                continue
            diff = set(gk.tolist()) ^ set(o[:k].tolist())
            sk = rank_boundary(s32[b, h], s64[b, h], n, k)
            for p in diff:
                sp = float(s64[b, h, p])
                gap = abs(sp - sk)
                assert 0 < gap < NEAR_TIE * max(abs(sp), abs(sk)), (
                    f"b={b} h={h} page {p}: score {sp!r} vs k-th {sk!r} (gap {gap:.3g})")
                excused += 1
    return excused


def check_out(gpu, ref, what):
    err = np.abs(gpu - ref)
    mx, mean = float(err.max()) if err.size else 0.0, float(err.mean()) if err.size else 0.0
    log(f"  {what}: max abs {mx:.3e}, mean abs {mean:.3e}")
    assert np.isfinite(gpu).all(), what
    assert mx <= MAX_ABS and mean <= MEAN_ABS, (what, mx, mean)


def full_check(inp: W.Inputs, k_max=None, dense=True, out_dtype=S.SPARROW_OUT_F32,
               capped=False):
    """Whole sparse step plus dense on the GPU vs the oracle, every sequence.  ``capped``: the
    test passes a k_max below some budgets on purpose."""
    w = inp.workload
    s = w.schedule
    ps = w.page_size
    lens = inp.lens_host
    if k_max is None:
        k_max = S.budget_bound(lens, ps, s.bin_tokens, s.min_pages, s.frac_num, s.frac_den)
    g = gpu_run(inp, k_max, dense=dense, out_dtype=out_dtype)
    h = host(inp)
    ora_meta = oracle.page_meta(h["k"], h["bt"], h["lens"])
    check_meta(g["meta"], ora_meta, h["bt"], h["lens"], ps)
    s32, s64 = oracle.page_scores(h["q"], ora_meta, h["bt"], h["lens"], ps)
    ora_k = oracle_budgets(h["lens"], ps, s.bin_tokens, s.min_pages, s.frac_num,
                           s.frac_den, k_max, capped=capped)
    ora_idx = oracle.select(h["lens"], ora_k, s32, ps, k_max)
    excused = check_indices(g["k"], g["idx"], ora_k, ora_idx, s32, s64, h["lens"], ps, k_max)
    # attention over the GPU's (validated) page lists
    ref_s = oracle.attention(h["q"], h["k"], h["v"], h["bt"], h["lens"], SCALE, g["k"], g["idx"])
    check_out(g["out_sparse"], ref_s, "sparse")
    if dense:
        ref_d = oracle.attention(h["q"], h["k"], h["v"], h["bt"], h["lens"], SCALE)
        check_out(g["out_dense"], ref_d, "dense")
    return dict(gpu=g, ora_idx=ora_idx, ora_k=ora_k, excused=excused, k_max=k_max)


def sample_inputs(inp: W.Inputs, seqs):
    """Host copies of the sampled sequences only, with a compact block table."""
    w = inp.workload
    ps = w.page_size
    bt_all = inp.block_table.cpu().numpy()
    rows, phys = [], []
    for b in seqs:
        n = (int(inp.lens_host[b]) + ps - 1) // ps
        rows.append(len(phys))
        phys.extend(int(x) for x in bt_all[b, :n])
    max_n = max(1, max((int(inp.lens_host[b]) + ps - 1) // ps for b in seqs))
    bt = np.zeros((len(seqs), max_n), np.int32)
    for i, b in enumerate(seqs):
        n = (int(inp.lens_host[b]) + ps - 1) // ps
        bt[i, :n] = np.arange(rows[i], rows[i] + n)
    pi = torch.as_tensor(np.array(phys, np.int64), device=inp.k_cache.device)
    sel = torch.as_tensor(np.array(seqs, np.int64), device=inp.q.device)
    return dict(q=W.bf16_bits(inp.q[sel]), k=W.bf16_bits(inp.k_cache[pi]),
                v=W.bf16_bits(inp.v_cache[pi]), bt=bt,
                lens=inp.lens_host[list(seqs)].astype(np.int32), phys=np.array(phys, np.int64))
