"""GPU parity of the selector variants (the mean-key landmark, forced sink/local pages),
through the C ABI, against the CPU oracle.  Key sums are fp32 additions in token order on
both sides, so the metadata is compared bit for bit; page lists bit-exact up to the
near-tie rule of the other parity tests (applied to the pages chosen by score)."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_08446_amd import sparrow as S
from paper_2606_08446_amd import workloads as W

from parity import NEAR_TIE, SCALE, check_out, host, log, oracle_budgets, sample_inputs

pytestmark = pytest.mark.gpu

DEV = "cuda"
MEAN = S.SPARROW_LANDMARK_MEAN


@pytest.fixture(autouse=True)
def _need_gpu(gpu_device):
    S.load()
    yield


def small(G, Hkv, ps, lengths, seed, schedule=None, **kw):
    w = W.small(B=len(lengths), Hq=G * Hkv, Hkv=Hkv, ps=ps, lengths=lengths, seed=seed,
                schedule=schedule or W.fraction_budget(1, 4, floor_pages=2), **kw)
    return W.generate(w, DEV, lengths=list(lengths))


def check_forced_indices(gk, gidx, ora_k, ora_idx, s32, s64, lens, ps, sink, local):
    """Bit-exact page lists; a page where GPU and oracle differ must be chosen by score (not
    forced) and be a near tie with the oracle's last page chosen by score."""
    np.testing.assert_array_equal(gk, ora_k)
    B, Hkv, _ = gidx.shape
    for b in range(B):
        n = (int(lens[b]) + ps - 1) // ps
        k = min(int(ora_k[b]), n)
        forced = [p for p in range(n) if p < sink or p >= n - local]
        for h in range(Hkv):
            g, o = gidx[b, h, :k], ora_idx[b, h, :k]
            assert (gidx[b, h, k:] == -1).all() and (np.diff(g) > 0).all()
            if np.array_equal(g, o):
                continue
            free = [p for p in range(n) if p not in forced]
            order = sorted(free, key=lambda p: (-float(s32[b, h, p]), p))
            n_scored = k - min(k, len(forced))
            sk = float(s64[b, h, order[n_scored - 1]])
            for p in set(g.tolist()) ^ set(o.tolist()):
                assert p not in forced, (b, h, p)
                sp = float(s64[b, h, p])
                assert 0 < abs(sp - sk) < NEAR_TIE * max(abs(sp), abs(sk)), (b, h, p, sp, sk)


@pytest.mark.parametrize("ps", [16, 32, 64, 128])
def test_mean_metadata_matches_oracle_bitwise(ps):
    log(f"case mean meta ps={ps}")
    inp = small(3, 3, ps, (ps * 5 + 3, 1, ps * 2, 0, ps * 9 - 1), seed=50 + ps)
    meta = S.new_meta(inp.num_phys_pages, 3, DEV, MEAN)
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta, landmark=MEAN)
    torch.cuda.synchronize()
    h = host(inp)
    ref = oracle.page_key_sums(h["k"], h["bt"], h["lens"])
    np.testing.assert_array_equal(meta.cpu().numpy(), ref)
    # incremental: recompute the pages touched since first_pos
    first = np.maximum(h["lens"] - 7, 0).astype(np.int32)
    part = oracle.page_key_sums(h["k"], h["bt"], first)
    meta2 = torch.as_tensor(part, device=DEV)
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta2,
                       first_pos=torch.as_tensor(first, device=DEV), landmark=MEAN)
    torch.cuda.synchronize()
    want = oracle.page_key_sums(h["k"], h["bt"], h["lens"], first_pos=first, sums=part)
    np.testing.assert_array_equal(meta2.cpu().numpy(), want)


@pytest.mark.parametrize("G,Hkv,ps", [(2, 2, 16), (5, 3, 32), (1, 9, 16), (4, 8, 64)])
def test_mean_selection_and_attention_match_oracle(G, Hkv, ps):
    log(f"case mean select G={G} Hkv={Hkv} ps={ps}")
    inp = small(G, Hkv, ps, (ps * 40 + 5, ps * 3, 700, 17), seed=60 + G, hot_pages=3)
    h = host(inp)
    s = inp.workload.schedule
    k_max = inp.max_pages
    meta = S.new_meta(inp.num_phys_pages, Hkv, DEV, MEAN)
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta, landmark=MEAN)
    k, idx = S.page_score_topk(inp.q, meta, inp.block_table, inp.seq_lens, inp.k_cache.shape,
                               inp.min_pages, inp.frac_num, s.frac_den, s.bin_tokens, k_max,
                               landmark=MEAN)
    out = S.sparse_decode_attn(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                               k, idx, SCALE)
    torch.cuda.synchronize()
    sums = oracle.page_key_sums(h["k"], h["bt"], h["lens"])
    s32, s64 = oracle.page_scores_mean(h["q"], sums, h["bt"], h["lens"], ps)
    ora_k = oracle_budgets(h["lens"], ps, s.bin_tokens, s.min_pages, s.frac_num,
                           s.frac_den, k_max)
    ora_idx = oracle.select(h["lens"], ora_k, s32, ps, k_max)
    check_forced_indices(k.cpu().numpy(), idx.cpu().numpy(), ora_k, ora_idx, s32, s64,
                         h["lens"], ps, 0, 0)
    ref = oracle.attention(h["q"], h["k"], h["v"], h["bt"], h["lens"], SCALE, k.cpu().numpy(),
                           idx.cpu().numpy())
    check_out(out.cpu().numpy().astype(np.float64), ref, "mean-landmark sparse")


@pytest.mark.parametrize("landmark", [S.SPARROW_LANDMARK_MINMAX, MEAN])
@pytest.mark.parametrize("sink,local", [(1, 0), (0, 3), (2, 2), (40, 40)])
def test_forced_pages_match_oracle(landmark, sink, local):
    log(f"case forced sink={sink} local={local} landmark={landmark}")
    inp = small(4, 2, 16, (16 * 60, 16 * 5 + 9, 300, 16 * 200 + 1), seed=70,
                schedule=W.fraction_budget(1, 8, floor_pages=3))
    h = host(inp)
    s = inp.workload.schedule
    k_max = inp.max_pages
    meta = S.new_meta(inp.num_phys_pages, 2, DEV, landmark)
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta, landmark=landmark)
    k, idx = S.page_score_topk(inp.q, meta, inp.block_table, inp.seq_lens, inp.k_cache.shape,
                               inp.min_pages, inp.frac_num, s.frac_den, s.bin_tokens, k_max,
                               landmark=landmark, sink_pages=sink, local_pages=local)
    torch.cuda.synchronize()
    if landmark == MEAN:
        s32, s64 = oracle.page_scores_mean(h["q"], oracle.page_key_sums(h["k"], h["bt"],
                                                                         h["lens"]),
                                           h["bt"], h["lens"], 16)
    else:
        s32, s64 = oracle.page_scores(h["q"], oracle.page_meta(h["k"], h["bt"], h["lens"]),
                                      h["bt"], h["lens"], 16)
    ora_k = oracle_budgets(h["lens"], 16, s.bin_tokens, s.min_pages, s.frac_num,
                           s.frac_den, k_max)
    ora_idx = oracle.select_forced(h["lens"], ora_k, s32, 16, k_max, sink, local)
    check_forced_indices(k.cpu().numpy(), idx.cpu().numpy(), ora_k, ora_idx, s32, s64,
                         h["lens"], 16, sink, local)


def run_fused(inp, meta, kn, vn, k_max, landmark):
    s = inp.workload.schedule
    shape = S.shape_of(inp.q, inp.k_cache, inp.block_table, landmark=landmark)
    sched = S.Schedule(s.bin_tokens, int(inp.min_pages.numel()), inp.min_pages.data_ptr(),
                       inp.frac_num.data_ptr(), s.frac_den)
    ws = torch.empty(S.sparrow_workspace_size(shape, k_max, S.SPARROW_OP_SCORE_TOPK),
                     dtype=torch.uint8, device=DEV)
    B, Hkv = inp.q.shape[0], inp.k_cache.shape[1]
    k = torch.empty(B, dtype=torch.int32, device=DEV)
    idx = torch.empty((B, Hkv, k_max), dtype=torch.int32, device=DEV)
    S._check("fused", S.sparrow_append_score_topk(
        shape, inp.q.data_ptr(), kn.data_ptr(), vn.data_ptr(), inp.k_cache.data_ptr(),
        inp.v_cache.data_ptr(), meta.data_ptr(), inp.block_table.data_ptr(),
        inp.seq_lens.data_ptr(), sched, k_max, k.data_ptr(), idx.data_ptr(), ws.data_ptr(),
        ws.numel(), torch.cuda.current_stream().cuda_stream))
    return k, idx


def test_mean_append_alone_and_fused():
    log("case mean append")
    lengths = (33, 64, 17, 100, 1)
    inp = small(3, 2, 16, lengths, seed=80)
    h = host(inp)
    before = np.maximum(h["lens"] - 1, 0).astype(np.int32)
    sums0 = oracle.page_key_sums(h["k"], h["bt"], before)
    g = torch.Generator(device=DEV)
    g.manual_seed(81)
    kn = torch.randn((5, 2, 128), generator=g, device=DEV).to(torch.bfloat16)
    vn = torch.randn((5, 2, 128), generator=g, device=DEV).to(torch.bfloat16)
    kc, vc, want = oracle.append_kv(W.bf16_bits(kn), W.bf16_bits(vn), h["k"], h["v"], h["bt"],
                                    h["lens"], sums0, landmark="mean")
    # alone
    a_k, a_v = inp.k_cache.clone(), inp.v_cache.clone()
    a_meta = torch.as_tensor(sums0, device=DEV)
    S.append_kv(kn, vn, a_k, a_v, inp.block_table, inp.seq_lens, a_meta, landmark=MEAN)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(a_meta.cpu().numpy(), want)
    np.testing.assert_array_equal(W.bf16_bits(a_k), kc)
    # fused with scoring: same caches and metadata, and the selection of the separate calls
    b_meta = torch.as_tensor(sums0, device=DEV)
    k_f, idx_f = run_fused(inp, b_meta, kn, vn, inp.max_pages, MEAN)
    s = inp.workload.schedule
    k_s, idx_s = S.page_score_topk(inp.q, a_meta, inp.block_table, inp.seq_lens,
                                   inp.k_cache.shape, inp.min_pages, inp.frac_num, s.frac_den,
                                   s.bin_tokens, inp.max_pages, landmark=MEAN)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(b_meta.cpu().numpy(), want)
    np.testing.assert_array_equal(W.bf16_bits(inp.k_cache), kc)
    assert torch.equal(k_f, k_s) and torch.equal(idx_f, idx_s)


def test_full_size_c2_mean_landmark_sampled():
    log("case full-size c2 mean landmark")
    w = W.C2
    inp = W.generate(w, DEV)
    s = w.schedule
    k_max = S.budget_bound(inp.lens_host, 16, s.bin_tokens, s.min_pages, s.frac_num, s.frac_den)
    meta = S.new_meta(inp.num_phys_pages, w.num_kv_heads, DEV, MEAN)
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta, landmark=MEAN)
    k, idx = S.page_score_topk(inp.q, meta, inp.block_table, inp.seq_lens, inp.k_cache.shape,
                               inp.min_pages, inp.frac_num, s.frac_den, s.bin_tokens, k_max,
                               landmark=MEAN)
    torch.cuda.synchronize()
    seqs = [0, 17, 40, 63]
    hs = sample_inputs(inp, seqs)
    sums = oracle.page_key_sums(hs["k"], hs["bt"], hs["lens"])
    np.testing.assert_array_equal(meta.cpu().numpy()[hs["phys"]], sums)
    s32, s64 = oracle.page_scores_mean(hs["q"], sums, hs["bt"], hs["lens"], 16)
    ora_k = oracle_budgets(hs["lens"], 16, s.bin_tokens, s.min_pages, s.frac_num,
                           s.frac_den, k_max)
    ora_idx = oracle.select(hs["lens"], ora_k, s32, 16, k_max)
    check_forced_indices(k.cpu().numpy()[seqs], idx.cpu().numpy()[seqs], ora_k, ora_idx, s32,
                         s64, hs["lens"], 16, 0, 0)
    # the planted hot pages (keys shifted along the group's query) win with the mean too
    kept = sum(set(inp.hot_host[b][hh]) <= set(idx[b, hh].tolist())
               for b in range(w.batch) for hh in range(w.num_kv_heads))
    log(f"  hot pages fully kept in {kept} of {w.batch * w.num_kv_heads} (sequence, head) units")
    assert kept == w.batch * w.num_kv_heads
