"""GPU parity of the token append: sparrow_append_kv and the fused
sparrow_append_score_topk, through the C ABI, against the CPU oracle (which
rebuilds the appended page's metadata from its tokens) and against each other.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_08446_amd import sparrow as S
from paper_2606_08446_amd import workloads as W

from parity import (SCALE, check_indices, check_out, host, log, oracle_budgets,
                    sample_inputs)

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(autouse=True)
def _need_gpu(gpu_device):
    S.load()
    yield


def new_rows(B, Hkv, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    k = torch.randn((B, Hkv, 128), generator=g, device=DEV).to(torch.bfloat16)
    v = torch.randn((B, Hkv, 128), generator=g, device=DEV).to(torch.bfloat16)
    return k, v


def append_case(G, Hkv, ps, lengths, seed, schedule=None, skip_last=True):
    """Inputs whose seq_lens count the token to append, and metadata (from the oracle) that
    describes the tokens before it.  With skip_last, the longest sequence gets a length one
    past what the block table addresses (the append must leave it alone)."""
    schedule = schedule or W.fraction_budget(1, 4)
    w = W.small(B=len(lengths), Hq=G * Hkv, Hkv=Hkv, ps=ps, lengths=lengths, seed=seed,
                schedule=schedule)
    inp = W.generate(w, DEV, lengths=list(lengths))
    lens = np.asarray(lengths, np.int32).copy()
    if skip_last:
        b = int(np.argmax(lens))
        lens[b] = ps * inp.max_pages + 1
    h = host(inp)
    meta0 = oracle.page_meta(h["k"], h["bt"], np.maximum(lens - 1, 0).astype(np.int32))
    inp.seq_lens = torch.as_tensor(lens, device=DEV)
    inp.lens_host = lens.astype(np.int64)
    meta = torch.as_tensor(meta0.view(np.int16), device=DEV).view(torch.bfloat16)
    kn, vn = new_rows(len(lengths), Hkv, seed + 1000)
    return inp, meta, meta0, kn, vn


CASES = [  # (G, Hkv, ps, lengths)
    (2, 2, 16, (1, 16, 17, 40, 0, 100)),
    (5, 3, 32, (33, 64, 65, 1, 200)),
    (1, 9, 64, (64, 65, 130, 7, 300)),
    (4, 8, 128, (128, 129, 1, 260, 600)),
    (2, 12, 16, (15, 16, 17, 500)),  # a partial group of 8 heads per scoring workgroup
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_append_matches_oracle(case):
    G, Hkv, ps, lengths = CASES[case]
    log(f"case append G={G} Hkv={Hkv} ps={ps} lengths={lengths}")
    inp, meta, meta0, kn, vn = append_case(G, Hkv, ps, lengths, seed=40 + case)
    h = host(inp)
    S.append_kv(kn, vn, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens, meta)
    torch.cuda.synchronize()
    kc, vc, mt = oracle.append_kv(W.bf16_bits(kn), W.bf16_bits(vn), h["k"], h["v"], h["bt"],
                                  h["lens"], meta0)
    np.testing.assert_array_equal(W.bf16_bits(inp.k_cache), kc)
    np.testing.assert_array_equal(W.bf16_bits(inp.v_cache), vc)
    np.testing.assert_array_equal(W.bf16_bits(meta), mt)


def selection_args(inp, k_max):
    s = inp.workload.schedule
    shape = S.shape_of(inp.q, inp.k_cache, inp.block_table)
    sched = S.Schedule(s.bin_tokens, int(inp.min_pages.numel()), inp.min_pages.data_ptr(),
                       inp.frac_num.data_ptr(), s.frac_den)
    ws = torch.empty(S.sparrow_workspace_size(shape, k_max, S.SPARROW_OP_SCORE_TOPK),
                     dtype=torch.uint8, device=DEV)
    return shape, sched, ws


def run_fused(inp, meta, kn, vn, k_max):
    shape, sched, ws = selection_args(inp, k_max)
    B, Hkv = inp.q.shape[0], inp.k_cache.shape[1]
    k = torch.empty(B, dtype=torch.int32, device=DEV)
    idx = torch.empty((B, Hkv, k_max), dtype=torch.int32, device=DEV)
    stream = torch.cuda.current_stream().cuda_stream
    S._check("sparrow_append_score_topk", S.sparrow_append_score_topk(
        shape, inp.q.data_ptr(), kn.data_ptr(), vn.data_ptr(), inp.k_cache.data_ptr(),
        inp.v_cache.data_ptr(), meta.data_ptr(), inp.block_table.data_ptr(),
        inp.seq_lens.data_ptr(), sched, k_max, k.data_ptr(), idx.data_ptr(), ws.data_ptr(),
        ws.numel(), stream))
    return k, idx


def clone_inputs(inp):
    c = W.Inputs(**{f: getattr(inp, f) for f in inp.__dataclass_fields__})
    c.k_cache = inp.k_cache.clone()
    c.v_cache = inp.v_cache.clone()
    return c


@pytest.mark.parametrize("case", range(len(CASES)))
def test_fused_equals_append_then_select(case):
    G, Hkv, ps, lengths = CASES[case]
    log(f"case fused G={G} Hkv={Hkv} ps={ps} lengths={lengths}")
    # a quarter of the pages with a floor of 2 pages: short sequences are dense (k = n)
    fused_check(G, Hkv, ps, lengths, 60 + case, W.Schedule(1 << 20, (2,), (1,), 4))


@pytest.mark.parametrize("seed", range(8))
def test_fused_random_shapes(seed):
    rng = np.random.default_rng(5000 + seed)
    G = int(rng.choice([1, 2, 4, 5, 8]))
    Hkv = int(rng.integers(1, 11))
    ps = int(rng.choice([16, 32, 64, 128]))
    B = int(rng.integers(1, 7))
    lengths = [int(x) for x in rng.integers(1, 6000, size=B)]
    lengths[int(rng.integers(0, B))] = int(rng.choice([1, ps, ps + 1, 2 * ps]))
    sched = W.fraction_budget(int(rng.integers(1, 4)), int(rng.integers(4, 12)),
                              floor_pages=int(rng.integers(0, 4)))
    log(f"case fused random {seed}: G={G} Hkv={Hkv} ps={ps} lengths={lengths}")
    fused_check(G, Hkv, ps, tuple(lengths), 5100 + seed, sched, skip_last=seed % 2 == 0)


@pytest.mark.parametrize("G,n_bins", [(16, 256), (12, 300)])
def test_fused_large_groups_and_many_bins(G, n_bins):
    # more than 8 query heads per KV head (a second batch of query rows in the scoring
    # prologue) and schedule tables staged in LDS (256 bins) or read from memory (300)
    rng = np.random.default_rng(77 + n_bins)
    sched = W.Schedule(16, tuple(int(x) for x in rng.integers(0, 7, n_bins)),
                       tuple(int(x) for x in rng.integers(1, 10, n_bins)), 20)
    log(f"case fused G={G} with {n_bins} schedule bins")
    fused_check(G, 2, 16, (3000, 4097, 6000, 5), 90 + G, sched)


def fused_check(G, Hkv, ps, lengths, seed, schedule, skip_last=True):
    """The fused append + selection equals the append followed by the selection bit for
    bit, and both match the oracle through attention."""
    inp, meta, meta0, kn, vn = append_case(G, Hkv, ps, lengths, seed=seed, schedule=schedule,
                                           skip_last=skip_last)
    k_max = inp.max_pages
    a = clone_inputs(inp)
    meta_a = meta.clone()
    S.append_kv(kn, vn, a.k_cache, a.v_cache, a.block_table, a.seq_lens, meta_a)
    s = a.workload.schedule
    k_a, idx_a = S.page_score_topk(a.q, meta_a, a.block_table, a.seq_lens, a.k_cache.shape,
                                   a.min_pages, a.frac_num, s.frac_den, s.bin_tokens, k_max)
    b = clone_inputs(inp)
    meta_b = meta.clone()
    k_b, idx_b = run_fused(b, meta_b, kn, vn, k_max)
    torch.cuda.synchronize()
    assert torch.equal(a.k_cache.view(torch.int16), b.k_cache.view(torch.int16))
    assert torch.equal(a.v_cache.view(torch.int16), b.v_cache.view(torch.int16))
    assert torch.equal(meta_a.view(torch.int16), meta_b.view(torch.int16))
    assert torch.equal(k_a, k_b)
    assert torch.equal(idx_a, idx_b)
    # and the fused step against the oracle: append, rebuild, score, select, attend
    h0 = host(inp)
    kc, vc, mt = oracle.append_kv(W.bf16_bits(kn), W.bf16_bits(vn), h0["k"], h0["v"], h0["bt"],
                                  h0["lens"], meta0)
    np.testing.assert_array_equal(W.bf16_bits(meta_b), mt)
    lens_eff = np.minimum(h0["lens"], ps * inp.max_pages).astype(np.int32)
    s32, s64 = oracle.page_scores(h0["q"], mt, h0["bt"], lens_eff, ps)
    ora_k = oracle_budgets(lens_eff, ps, s.bin_tokens, s.min_pages, s.frac_num,
                           s.frac_den, k_max)
    ora_idx = oracle.select(lens_eff, ora_k, s32, ps, k_max)
    check_indices(k_b.cpu().numpy(), idx_b.cpu().numpy(), ora_k, ora_idx, s32, s64, lens_eff,
                  ps, k_max)
    out = S.sparse_decode_attn(b.q, b.k_cache, b.v_cache, b.block_table, b.seq_lens, k_b, idx_b,
                               SCALE)
    torch.cuda.synchronize()
    ref = oracle.attention(h0["q"], kc, vc, h0["bt"], lens_eff, SCALE, k_b.cpu().numpy(),
                           idx_b.cpu().numpy())
    check_out(out.cpu().numpy().astype(np.float64), ref, "fused step sparse")


def test_token_by_token_growth_equals_rebuild():
    log("case append growth")
    G, Hkv, ps = 3, 2, 16
    final = (70, 33, 16, 5)
    T = 40
    w = W.small(B=4, Hq=G * Hkv, Hkv=Hkv, ps=ps, lengths=final, seed=71,
                schedule=W.fraction_budget(1, 3))
    inp = W.generate(w, DEV, lengths=list(final))
    full = np.asarray(final, np.int32)
    start = np.maximum(full - T, 0).astype(np.int32)
    target_k = inp.k_cache.clone()
    target_v = inp.v_cache.clone()
    meta = torch.zeros((inp.num_phys_pages, Hkv, 2, 128), dtype=torch.bfloat16, device=DEV)
    S.page_meta_update(inp.k_cache, inp.block_table, torch.as_tensor(start, device=DEV), meta)
    bt = inp.block_table.cpu().numpy()
    k_max = inp.max_pages
    for t in range(T):
        lens = np.where(start + t < full, start + t + 1, 0).astype(np.int32)  # done: sit out
        kn = torch.zeros((4, Hkv, 128), dtype=torch.bfloat16, device=DEV)
        vn = torch.zeros_like(kn)
        for b in range(4):
            if lens[b] > 0:
                pos = int(lens[b]) - 1
                phys = int(bt[b, pos // ps])
                kn[b] = target_k[phys, :, pos % ps]
                vn[b] = target_v[phys, :, pos % ps]
        inp.seq_lens = torch.as_tensor(lens, device=DEV)
        if t % 2 == 0:
            run_fused(inp, meta, kn, vn, k_max)
        else:
            S.append_kv(kn, vn, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens, meta)
    inp.seq_lens = torch.as_tensor(full, device=DEV)
    rebuilt = torch.zeros_like(meta)
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, rebuilt)
    torch.cuda.synchronize()
    h = host(inp)
    ora = oracle.page_meta(h["k"], h["bt"], h["lens"])
    for b, L in enumerate(full):
        pages = bt[b, :(int(L) + ps - 1) // ps].astype(np.int64)
        np.testing.assert_array_equal(W.bf16_bits(meta)[pages], W.bf16_bits(rebuilt)[pages])
        np.testing.assert_array_equal(W.bf16_bits(meta)[pages], ora[pages])


def test_full_size_c5_fused_append_step():
    log("case full-size c5 fused append")
    w = W.C5
    inp = W.generate(w, DEV)
    meta = torch.zeros((inp.num_phys_pages, w.num_kv_heads, 2, 128), dtype=torch.bfloat16,
                       device=DEV)
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta)
    inp.seq_lens += 1                      # the appended token goes to position L (spare page)
    inp.lens_host = inp.lens_host + 1
    kn, vn = new_rows(w.batch, w.num_kv_heads, 99)
    s = w.schedule
    k_max = S.budget_bound(inp.lens_host, w.page_size, s.bin_tokens, s.min_pages, s.frac_num,
                           s.frac_den)
    k, idx = run_fused(inp, meta, kn, vn, k_max)
    # the same selection from a fresh metadata rebuild of the updated cache
    meta_r = torch.zeros_like(meta)
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta_r)
    k_r, idx_r = S.page_score_topk(inp.q, meta_r, inp.block_table, inp.seq_lens,
                                   inp.k_cache.shape, inp.min_pages, inp.frac_num, s.frac_den,
                                   s.bin_tokens, k_max)
    torch.cuda.synchronize()
    assert torch.equal(k, k_r) and torch.equal(idx, idx_r)
    rng = np.random.default_rng(5)
    seqs = sorted(set([0, w.batch - 1] + [int(x) for x in rng.integers(0, w.batch, 2)]))
    h = sample_inputs(inp, seqs)
    ora_meta = oracle.page_meta(h["k"], h["bt"], h["lens"])
    np.testing.assert_array_equal(W.bf16_bits(meta)[h["phys"]], ora_meta)
    for i, b in enumerate(seqs):   # the appended rows landed where the oracle expects them
        pos = int(h["lens"][i]) - 1
        row = h["k"][h["bt"][i, pos // w.page_size], :, pos % w.page_size]
        np.testing.assert_array_equal(row, W.bf16_bits(kn[b]))
    s32, s64 = oracle.page_scores(h["q"], ora_meta, h["bt"], h["lens"], w.page_size)
    ora_k = oracle_budgets(h["lens"], w.page_size, s.bin_tokens, s.min_pages,
                           s.frac_num, s.frac_den, k_max)
    ora_idx = oracle.select(h["lens"], ora_k, s32, w.page_size, k_max)
    check_indices(k.cpu().numpy()[seqs], idx.cpu().numpy()[seqs], ora_k, ora_idx, s32, s64,
                  h["lens"], w.page_size, k_max)
