"""Block-table entries outside the caches, on the GPU through the C ABI.

An entry outside [0, num_phys_pages) marks an absent page: no kernel reads or writes that
physical page, scoring sees zero metadata for it (score 0), attention leaves its tokens
out, and an append to it writes nothing.  The oracle gets the same inputs with every such
entry pointing at one extra all-zero physical page (zero metadata gives the same score 0)
and, for attention, page lists without those pages.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_08446_amd import sparrow as S
from paper_2606_08446_amd import workloads as W

from parity import SCALE, check_indices, check_out, host, log, oracle_budgets

pytestmark = pytest.mark.gpu

DEV = "cuda"
G, HKV, PS = 2, 2, 16
LENGTHS = (700, 1500, 300)


@pytest.fixture(autouse=True)
def _need_gpu(gpu_device):
    S.load()
    yield


def corrupted_inputs():
    w = W.small(B=len(LENGTHS), Hq=G * HKV, Hkv=HKV, ps=PS, lengths=LENGTHS, seed=19,
                schedule=W.fraction_budget(1, 3))
    inp = W.generate(w, DEV, lengths=list(LENGTHS))
    P = inp.num_phys_pages
    bt = inp.block_table.cpu().numpy().copy()
    n = [(L + PS - 1) // PS for L in LENGTHS]
    # past the cache, negative, the last page of a sequence, the largest int32
    for b, p, v in ((0, 2, P + 7), (0, 10, -5), (1, n[1] - 1, P), (2, 0, 2**31 - 1)):
        bt[b, p] = v
    inp.block_table = torch.as_tensor(bt, device=DEV)
    return inp, bt, n


def oracle_view(h, P):
    """Caches with one extra all-zero page P and the block table with every entry outside
    the cache pointing at it."""
    k = np.concatenate([h["k"], np.zeros_like(h["k"][:1])])
    v = np.concatenate([h["v"], np.zeros_like(h["v"][:1])])
    bt = h["bt"].copy()
    bt[(bt < 0) | (bt >= P)] = P
    return k, v, bt


def absent(bt, b, p, P):
    return not 0 <= int(bt[b, p]) < P


def attention_ref(h, kz, vz, btz, lists):
    """fp64 attention per (sequence, KV head) over the given logical page lists."""
    B = len(lists)
    ref = np.zeros((B, G * HKV, 128))
    for b in range(B):
        for hh in range(HKV):
            pages = lists[b][hh]
            sub = np.full((1, 1, max(len(pages), 1)), -1, np.int32)
            sub[0, 0, :len(pages)] = pages
            ref[b, G * hh:G * hh + G] = oracle.attention(
                h["q"][b:b + 1, G * hh:G * hh + G], kz[:, hh:hh + 1], vz[:, hh:hh + 1],
                btz[b:b + 1], h["lens"][b:b + 1], SCALE, np.array([len(pages)], np.int32),
                sub)[0]
    return ref


def test_block_table_entries_outside_the_cache():
    log("case block-table entries outside the cache")
    inp, bt, n = corrupted_inputs()
    P = inp.num_phys_pages
    h = host(inp)
    kz, vz, btz = oracle_view(h, P)
    lens = h["lens"]
    s = inp.workload.schedule

    # metadata: the pages with valid entries as the oracle builds them, nothing else written
    meta = S.new_meta(P, HKV, DEV)
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta)
    torch.cuda.synchronize()
    g_meta = W.bf16_bits(meta)
    ora_meta = oracle.page_meta(kz, btz, lens)
    np.testing.assert_array_equal(g_meta, ora_meta[:P])

    # selection: absent pages score 0, like the oracle's all-zero page
    k_max = S.budget_bound(lens, PS, s.bin_tokens, s.min_pages, s.frac_num, s.frac_den)
    k, idx = S.page_score_topk(inp.q, meta, inp.block_table, inp.seq_lens, inp.k_cache.shape,
                               inp.min_pages, inp.frac_num, s.frac_den, s.bin_tokens, k_max)
    torch.cuda.synchronize()
    s32, s64 = oracle.page_scores(h["q"], ora_meta, btz, lens, PS)
    ora_k = oracle_budgets(lens, PS, s.bin_tokens, s.min_pages, s.frac_num,
                           s.frac_den, k_max)
    ora_idx = oracle.select(lens, ora_k, s32, PS, k_max)
    check_indices(k.cpu().numpy(), idx.cpu().numpy(), ora_k, ora_idx, s32, s64, lens, PS,
                  k_max)

    # attention: absent pages contribute no tokens
    out = S.sparse_decode_attn(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                               k, idx, SCALE)
    dense = S.dense_decode_attn(inp.q, inp.k_cache, inp.v_cache, inp.block_table,
                                inp.seq_lens, SCALE)
    torch.cuda.synchronize()
    gi, gk = idx.cpu().numpy(), k.cpu().numpy()
    sparse_lists = [[[p for p in gi[b, hh, :gk[b]].tolist() if not absent(bt, b, p, P)]
                     for hh in range(HKV)] for b in range(len(LENGTHS))]
    check_out(out.cpu().numpy().astype(np.float64), attention_ref(h, kz, vz, btz, sparse_lists),
              "sparse, absent pages")
    dense_lists = [[[p for p in range(n[b]) if not absent(bt, b, p, P)]] * HKV
                   for b in range(len(LENGTHS))]
    check_out(dense.cpu().numpy().astype(np.float64), attention_ref(h, kz, vz, btz, dense_lists),
              "dense, absent pages")


def test_append_to_a_page_outside_the_cache_writes_nothing():
    log("case append to a page outside the cache")
    inp, bt, n = corrupted_inputs()
    P = inp.num_phys_pages
    h = host(inp)
    kz, vz, btz = oracle_view(h, P)
    lens = h["lens"]
    s = inp.workload.schedule
    meta0 = oracle.page_meta(kz, btz, np.maximum(lens - 1, 0).astype(np.int32))
    gen = torch.Generator(device=DEV)
    gen.manual_seed(1019)
    kn = torch.randn((len(LENGTHS), HKV, 128), generator=gen, device=DEV).to(torch.bfloat16)
    vn = torch.randn((len(LENGTHS), HKV, 128), generator=gen, device=DEV).to(torch.bfloat16)
    kc, vc, mt = oracle.append_kv(W.bf16_bits(kn), W.bf16_bits(vn), kz, vz, btz, lens, meta0)
    k_max = S.budget_bound(lens, PS, s.bin_tokens, s.min_pages, s.frac_num, s.frac_den)

    def fresh():
        k_cache, v_cache = inp.k_cache.clone(), inp.v_cache.clone()
        meta = torch.as_tensor(meta0[:P].view(np.int16), device=DEV).view(torch.bfloat16)
        return k_cache, v_cache, meta.clone()

    # the append alone: sequence 1's token (its page is outside the cache) goes nowhere; the
    # oracle writes it into the extra page, which is not compared
    k_a, v_a, m_a = fresh()
    S.append_kv(kn, vn, k_a, v_a, inp.block_table, inp.seq_lens, m_a)
    # the fused append + selection
    k_b, v_b, m_b = fresh()
    shape = S.shape_of(inp.q, k_b, inp.block_table)
    sched = S.Schedule(s.bin_tokens, int(inp.min_pages.numel()), inp.min_pages.data_ptr(),
                       inp.frac_num.data_ptr(), s.frac_den)
    ws = torch.empty(S.sparrow_workspace_size(shape, k_max, S.SPARROW_OP_SCORE_TOPK),
                     dtype=torch.uint8, device=DEV)
    kf = torch.empty(len(LENGTHS), dtype=torch.int32, device=DEV)
    idxf = torch.empty((len(LENGTHS), HKV, k_max), dtype=torch.int32, device=DEV)
    S._check("sparrow_append_score_topk", S.sparrow_append_score_topk(
        shape, inp.q.data_ptr(), kn.data_ptr(), vn.data_ptr(), k_b.data_ptr(), v_b.data_ptr(),
        m_b.data_ptr(), inp.block_table.data_ptr(), inp.seq_lens.data_ptr(), sched, k_max,
        kf.data_ptr(), idxf.data_ptr(), ws.data_ptr(), ws.numel(),
        torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    for what, kk, vv, mm in (("append", k_a, v_a, m_a), ("fused", k_b, v_b, m_b)):
        np.testing.assert_array_equal(W.bf16_bits(kk), kc[:P], err_msg=what)
        np.testing.assert_array_equal(W.bf16_bits(vv), vc[:P], err_msg=what)
        np.testing.assert_array_equal(W.bf16_bits(mm), mt[:P], err_msg=what)
    # the fused selection sees every absent page with zero metadata (the oracle's append
    # wrote sequence 1's key into the extra page: clear it again)
    mz = mt.copy()
    mz[P] = 0
    s32, s64 = oracle.page_scores(h["q"], mz, btz, lens, PS)
    ora_k = oracle_budgets(lens, PS, s.bin_tokens, s.min_pages, s.frac_num,
                           s.frac_den, k_max)
    ora_idx = oracle.select(lens, ora_k, s32, PS, k_max)
    check_indices(kf.cpu().numpy(), idxf.cpu().numpy(), ora_k, ora_idx, s32, s64, lens, PS,
                  k_max)


def test_mean_landmark_with_absent_pages():
    log("case mean landmark, absent pages")
    inp, bt, n = corrupted_inputs()
    P = inp.num_phys_pages
    h = host(inp)
    kz, vz, btz = oracle_view(h, P)
    lens = h["lens"]
    s = inp.workload.schedule
    mean = S.SPARROW_LANDMARK_MEAN
    sums = S.new_meta(P, HKV, DEV, landmark=mean)
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, sums, landmark=mean)
    torch.cuda.synchronize()
    ora_sums = oracle.page_key_sums(kz, btz, lens)
    np.testing.assert_array_equal(sums.cpu().numpy().view(np.uint32),
                                  ora_sums[:P].view(np.uint32))
    k_max = S.budget_bound(lens, PS, s.bin_tokens, s.min_pages, s.frac_num, s.frac_den)
    k, idx = S.page_score_topk(inp.q, sums, inp.block_table, inp.seq_lens, inp.k_cache.shape,
                               inp.min_pages, inp.frac_num, s.frac_den, s.bin_tokens, k_max,
                               landmark=mean)
    torch.cuda.synchronize()
    s32, s64 = oracle.page_scores_mean(h["q"], ora_sums, btz, lens, PS)
    ora_k = oracle_budgets(lens, PS, s.bin_tokens, s.min_pages, s.frac_num,
                           s.frac_den, k_max)
    ora_idx = oracle.select(lens, ora_k, s32, PS, k_max)
    check_indices(k.cpu().numpy(), idx.cpu().numpy(), ora_k, ora_idx, s32, s64, lens, PS,
                  k_max)


def test_block_table_entries_past_the_sequence_do_not_matter():
    # the entries past a sequence's last page may be read but never used: garbage there
    # (negative, past the cache, or another sequence's pages) leaves every output unchanged
    log("case garbage past each sequence's pages")
    w = W.small(B=len(LENGTHS), Hq=G * HKV, Hkv=HKV, ps=PS, lengths=LENGTHS, seed=23,
                schedule=W.fraction_budget(1, 3))
    inp = W.generate(w, DEV, lengths=list(LENGTHS))
    s = inp.workload.schedule
    k_max = S.budget_bound(inp.lens_host, PS, s.bin_tokens, s.min_pages, s.frac_num,
                           s.frac_den)
    kn = torch.ones((len(LENGTHS), HKV, 128), device=DEV).to(torch.bfloat16)

    def run(bt):
        kc, vc = inp.k_cache.clone(), inp.v_cache.clone()
        meta = S.new_meta(inp.num_phys_pages, HKV, DEV)
        S.page_meta_update(kc, bt, inp.seq_lens, meta)
        step = S.SparseDecodeStep(inp.q, kc, vc, bt, inp.seq_lens, meta, inp.min_pages,
                                  inp.frac_num, s.frac_den, s.bin_tokens, k_max)
        sp = torch.cuda.current_stream().cuda_stream
        step.append_score_topk(kn, kn, sp)
        step.attend(sp)
        dense = S.dense_decode_attn(inp.q, kc, vc, bt, inp.seq_lens, SCALE)
        torch.cuda.synchronize()
        return [x.cpu() for x in (meta.view(torch.int16), kc.view(torch.int16), step.k,
                                  step.idx, step.out, dense)]

    ref = run(inp.block_table)
    bt = inp.block_table.cpu().numpy().copy()
    rng = np.random.default_rng(3)
    P = inp.num_phys_pages
    for b, L in enumerate(LENGTHS):
        n = (L + PS - 1) // PS
        tail = bt.shape[1] - n
        bt[b, n:] = rng.choice([-1, -(2**31), P, 2**31 - 1, 0, 1, P - 1], size=tail)
    got = run(torch.as_tensor(bt, device=DEV))
    for x, y in zip(got, ref):
        assert torch.equal(x, y)


@pytest.mark.parametrize("whole", [False, True])
def test_negative_lengths_count_as_empty(whole):
    """A negative length is an empty sequence, as 0 is: no pages, budget 0, a zero output
    row, no append; the other sequences are unaffected (separate calls and the whole-step
    call, on the one-kernel and the streaming path)."""
    log(f"case negative lengths, whole-step call {whole}")
    lengths = (900, 0, 2500, 0, 40)
    w = W.small(B=5, Hq=4, Hkv=2, ps=16, lengths=lengths, seed=23, schedule=W.fixed_budget(12))
    outs = []
    for neg in (False, True):
        inp = W.generate(w, DEV, lengths=list(lengths))
        if neg:
            inp.seq_lens[1] = -7
            inp.seq_lens[3] = -(2**31)
        meta = S.new_meta(inp.num_phys_pages, 2, DEV)
        S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta)
        s = w.schedule
        step = S.SparseDecodeStep(inp.q, inp.k_cache, inp.v_cache, inp.block_table,
                                  inp.seq_lens, meta, inp.min_pages, inp.frac_num, s.frac_den,
                                  s.bin_tokens, 12)
        g = torch.Generator(device=DEV)
        g.manual_seed(24)
        kn = torch.randn((5, 2, 128), generator=g, device=DEV).to(torch.bfloat16)
        vn = torch.randn((5, 2, 128), generator=g, device=DEV).to(torch.bfloat16)
        stream = torch.cuda.current_stream().cuda_stream
        if whole:
            step.decode_step(kn, vn, stream)
        else:
            step.append_score_topk(kn, vn, stream)
            step.attend(stream)
        dense = S.dense_decode_attn(inp.q, inp.k_cache, inp.v_cache, inp.block_table,
                                    inp.seq_lens, SCALE)
        torch.cuda.synchronize()
        outs.append((step.k.cpu().numpy(), step.idx.cpu().numpy(), step.out.cpu().numpy(),
                     dense.cpu().numpy(), W.bf16_bits(inp.k_cache), W.bf16_bits(meta)))
    for name, a, b in zip(("k", "idx", "out", "dense", "k_cache", "meta"), outs[0], outs[1]):
        np.testing.assert_array_equal(a, b, err_msg=name)
    assert outs[1][0][1] == 0 and outs[1][0][3] == 0
    assert (outs[1][2][1] == 0).all() and (outs[1][3][3] == 0).all()
