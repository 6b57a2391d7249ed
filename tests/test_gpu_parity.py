"""GPU parity: the HIP path (called through the C ABI) against the CPU oracle.

Small cases are checked in full (every sequence, head, page and output
element), at sizes that span several tiles of every kernel plus ragged tails.
The five workload shapes run at full size on the GPU and are checked on a
seeded sample of sequences.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_08446_amd import sparrow as S
from paper_2606_08446_amd import workloads as W

from parity import (SCALE, check_indices, check_meta, check_out, full_check, gpu_run, host, log,
                    oracle_budgets, sample_inputs)

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(autouse=True)
def _need_gpu(gpu_device):
    S.load()
    yield


def small_inputs(G, Hkv, ps, lengths, seed, schedule, **kw):
    w = W.small(B=len(lengths), Hq=G * Hkv, Hkv=Hkv, ps=ps, lengths=lengths, seed=seed,
                schedule=schedule, **kw)
    return W.generate(w, DEV, lengths=list(lengths))


# ---------------------------------------------------------------------------------- C1 in full
def test_c1_full():
    log("case c1 full")
    inp = W.generate(W.C1, DEV)
    r = full_check(inp)
    assert r["gpu"]["k"].tolist() == [32]
    # the x4 sink page carries the largest keys; it must be selected for every head
    assert (r["gpu"]["idx"][0, :, 0] == 0).all()


# ---------------------------------------------------------------------------------- small sweep
SWEEP = [
    # (G, Hkv, ps, lengths, schedule)
    (2, 2, 16, (1, 16, 17, 300, 4100), W.fraction_budget(1, 3)),
    (1, 3, 16, (33, 5000, 2, 15), W.fraction_budget(1, 10)),
    (4, 2, 16, (9000, 4097, 4096), W.fraction_budget(5, 100, floor_pages=3)),
    (5, 2, 16, (777, 6000, 31), W.rising_permille(2048, 2048, 8192, 30, 150)),
    (8, 1, 16, (2500, 64, 65), W.fixed_budget(7)),
    (16, 1, 16, (1000, 3333), W.fraction_budget(1, 4)),
    (2, 2, 32, (1, 32, 33, 8000, 20000), W.fraction_budget(1, 8)),
    (4, 2, 64, (64, 65, 9000), W.fraction_budget(1, 5)),
    (2, 2, 128, (127, 128, 129, 30000), W.fraction_budget(1, 6)),
    (3, 2, 16, (0, 50, 0, 1200), W.fraction_budget(1, 2)),
    # KV-head counts that leave a partial group of 8 heads per scoring workgroup, an odd
    # head in a wave's head pair, or an idle wave
    (1, 9, 16, (3000, 17, 900), W.fraction_budget(1, 5)),
    (2, 12, 32, (5000, 64, 1), W.fraction_budget(1, 4)),
    (3, 5, 16, (2048, 2049, 333), W.fraction_budget(1, 3)),
    # the remaining group sizes up to 16 that no case above uses: some query-head rows of
    # the padded 16-row MFMA tile unused, and group sums of more heads in the scoring
    (6, 3, 64, (4000, 129, 7000), W.fraction_budget(1, 4)),
    (7, 2, 128, (2600, 257), W.fraction_budget(1, 2)),
    (12, 1, 32, (6000, 31, 1900), W.rising_permille(2048, 2048, 8192, 40, 200)),
    # more KV heads than one scoring workgroup takes (8): two and four head blocks, the
    # last partial
    (1, 16, 16, (3000, 70, 1), W.fraction_budget(1, 6)),
    (2, 20, 32, (2500, 900), W.fraction_budget(1, 5)),
    (1, 32, 64, (5000, 129), W.fixed_budget(9)),
]


@pytest.mark.parametrize("case", range(len(SWEEP)))
def test_small_sweep(case):
    G, Hkv, ps, lengths, sched = SWEEP[case]
    log(f"case sweep {case}: G={G} Hkv={Hkv} ps={ps} lens={lengths}")
    inp = small_inputs(G, Hkv, ps, lengths, seed=100 + case, schedule=sched)
    full_check(inp)



# ------------------------------------------------- both scoring workgroup sizes, one selection
def replicated(inp, reps):
    """The batch of `inp` repeated `reps` times over the same cache pages (the block-table
    rows repeat, so every copy of a sequence reads the same physical pages)."""
    import dataclasses
    B = inp.workload.batch
    w = dataclasses.replace(inp.workload, batch=B * reps)
    return W.Inputs(workload=w, seq_lens=inp.seq_lens.repeat(reps).contiguous(),
                    block_table=inp.block_table.repeat(reps, 1).contiguous(),
                    q=inp.q.repeat(reps, 1, 1).contiguous(), k_cache=inp.k_cache,
                    v_cache=inp.v_cache, min_pages=inp.min_pages, frac_num=inp.frac_num,
                    lens_host=np.tile(inp.lens_host, reps), pages_host=np.tile(inp.pages_host, reps))


@pytest.mark.parametrize("case", [0, 8, 10, 11, 12, 15])
def test_scoring_workgroup_sizes_select_alike(case):
    """A small batch is scored in 8-page workgroups; the same sequences repeated until the
    grid holds 256 or more 32-page workgroups are scored in 32-page ones.  Both selections
    equal the oracle's, and every copy of a sequence selects exactly the small batch's
    pages (the scores are bit-identical)."""
    G, Hkv, ps, lengths, sched = SWEEP[case]
    inp = small_inputs(G, Hkv, ps, lengths, seed=100 + case, schedule=sched)
    blocks = -(-inp.max_pages // 32) * len(lengths) * -(-Hkv // 8)
    reps = -(-256 // blocks)
    assert blocks < 256 <= blocks * reps
    log(f"case block sizes {case}: G={G} Hkv={Hkv} ps={ps} lens={lengths} x{reps}")
    small = full_check(inp)
    big = full_check(replicated(inp, reps))
    B = len(lengths)
    for r in range(reps):
        assert np.array_equal(big["gpu"]["k"][r * B:(r + 1) * B], small["gpu"]["k"])
        assert np.array_equal(big["gpu"]["idx"][r * B:(r + 1) * B], small["gpu"]["idx"])


# ------------------------------------------------------------------- seeded random shapes
def random_case(seed):
    """A shape drawn from a seeded generator: group size, KV heads, page size, ragged
    lengths (0 and 1 included now and then) and one of the schedule forms."""
    rng = np.random.default_rng(9000 + seed)
    G = int(rng.choice([1, 2, 3, 4, 5, 8, 16]))
    Hkv = int(rng.integers(1, 13))
    ps = int(rng.choice([16, 32, 64, 128]))
    B = int(rng.integers(1, 7))
    lengths = [int(x) for x in rng.integers(0, 9000, size=B)]
    if rng.random() < 0.3:
        lengths[int(rng.integers(0, B))] = int(rng.choice([0, 1, ps, ps + 1]))
    form = int(rng.integers(0, 3))
    if form == 0:
        sched = W.fixed_budget(int(rng.integers(1, 40)))
    elif form == 1:
        sched = W.fraction_budget(int(rng.integers(1, 5)), int(rng.integers(5, 20)),
                                  floor_pages=int(rng.integers(0, 6)))
    else:
        sched = W.rising_permille(2048, 2048, 8192, int(rng.integers(20, 100)),
                                  int(rng.integers(100, 400)))
    return G, Hkv, ps, tuple(lengths), sched


@pytest.mark.parametrize("seed", range(16))
def test_random_shapes(seed):
    G, Hkv, ps, lengths, sched = random_case(seed)
    log(f"case random {seed}: G={G} Hkv={Hkv} ps={ps} lens={lengths}")
    inp = small_inputs(G, Hkv, ps, lengths, seed=700 + seed, schedule=sched)
    s = inp.workload.schedule
    k_max = S.budget_bound(inp.lens_host, ps, s.bin_tokens, s.min_pages, s.frac_num, s.frac_den)
    if seed % 4 == 3:
        k_max = max(1, k_max // 2)  # a k_max below some budgets: the cap applies
    full_check(inp, k_max=k_max, capped=seed % 4 == 3)


@pytest.mark.parametrize("k_pages", ["one", "n_minus_1", "n", "more"])
def test_budget_edges(k_pages):
    lengths = (800, 801, 3000)
    n = [(L + 15) // 16 for L in lengths]
    fixed = {"one": 1, "n_minus_1": min(n) - 1, "n": max(n), "more": max(n) + 50}[k_pages]
    log(f"case budget edge {k_pages}: fixed={fixed}")
    inp = small_inputs(4, 2, 16, lengths, seed=7, schedule=W.fixed_budget(fixed))
    r = full_check(inp)
    if k_pages in ("n", "more"):
        for b, nb in enumerate(n):
            assert r["gpu"]["k"][b] == nb


def test_every_sequence_within_one_page():
    # a one-column block table: one scoring block, one page per unit, budgets of 0 or 1
    log("case one page per sequence")
    inp = small_inputs(4, 2, 16, (1, 16, 7, 0, 12), seed=43, schedule=W.fixed_budget(1),
                       extra_pages=0)
    assert inp.max_pages == 1
    full_check(inp)


def many_bins(n_bins, seed):
    """A seeded schedule table of n_bins 16-token bins (fractions 1..9 / 20, floors 0..6)."""
    rng = np.random.default_rng(seed)
    return W.Schedule(16, tuple(int(x) for x in rng.integers(0, 7, n_bins)),
                      tuple(int(x) for x in rng.integers(1, 10, n_bins)), 20)


@pytest.mark.parametrize("n_bins", [256, 300])
def test_schedule_tables_of_many_bins(n_bins):
    # 256 bins: the scoring kernel stages the tables in LDS; more: it reads them from memory
    log(f"case schedule of {n_bins} bins")
    lengths = (4000, 17, 4096, 4097, 6000, 1)  # several bins, the last bin and past it
    inp = small_inputs(3, 2, 16, lengths, seed=41, schedule=many_bins(n_bins, 5))
    full_check(inp)


def test_k_max_caps_the_budget():
    log("case k_max cap")
    inp = small_inputs(2, 2, 16, (3000, 5000), seed=8, schedule=W.fraction_budget(1, 2))
    r = full_check(inp, k_max=40, capped=True)
    assert (r["gpu"]["k"] == 40).all()


def test_bf16_output():
    log("case bf16 output")
    inp = small_inputs(4, 2, 16, (700, 2900), seed=9, schedule=W.fraction_budget(1, 5))
    full_check(inp, out_dtype=S.SPARROW_OUT_BF16)


# ---------------------------------------------------------------------------------- ties
def test_zero_query_selects_lowest_pages():
    log("case zero query")
    inp = small_inputs(4, 2, 16, (2000, 5000), seed=10, schedule=W.fixed_budget(9))
    inp.q.zero_()
    r = full_check(inp)
    for b in range(2):
        for h in range(2):
            assert r["gpu"]["idx"][b, h, :9].tolist() == list(range(9))


def test_duplicated_pages_keep_lower_index():
    log("case duplicated pages")
    inp = small_inputs(2, 2, 16, (4000,), seed=11, schedule=W.fixed_budget(5))
    bt = inp.block_table.cpu().numpy()
    # pages 3, 40, 200 and 201 all get copies of page 100's keys, boosted to be on top
    src = int(bt[0, 100])
    inp.k_cache[src] = (inp.k_cache[src].float() * 3).to(torch.bfloat16)
    for p in (3, 40, 200, 201):
        inp.k_cache[int(bt[0, p])] = inp.k_cache[src]
    r = full_check(inp)
    for h in range(2):
        sel = r["gpu"]["idx"][0, h, :5].tolist()
        assert sel == [3, 40, 100, 200, 201]


def test_duplicated_pages_at_the_cut():
    log("case duplicated pages at the cut")
    inp = small_inputs(2, 1, 16, (3000,), seed=12, schedule=W.fixed_budget(2))
    bt = inp.block_table.cpu().numpy()
    src = int(bt[0, 50])
    inp.k_cache[src] = (inp.k_cache[src].float() * 3).to(torch.bfloat16)
    for p in (10, 150):
        inp.k_cache[int(bt[0, p])] = inp.k_cache[src]
    # three identical top pages, budget 2: the two lowest indices win
    r = full_check(inp)
    assert r["gpu"]["idx"][0, 0, :2].tolist() == [10, 50]


@pytest.mark.parametrize("perturb", [False, True])
def test_many_pages_in_the_threshold_digit(perturb):
    """100 copies of one boosted page, budget 50: the radix select's threshold digit holds
    many keys pass after pass - down to the last bit for identical copies (ties to the lower
    index), or until the copies' scores, nudged apart in one channel each, separate.  With 8
    units (512-thread top-k) and with the batch repeated to 1024 units (256-thread top-k),
    which must select alike."""
    log(f"case many pages in the threshold digit, perturbed {perturb}")
    inp = small_inputs(2, 8, 16, (3000,), seed=14, schedule=W.fixed_budget(50))
    bt = inp.block_table.cpu().numpy()
    src = int(bt[0, 150])
    inp.k_cache[src] = (inp.k_cache[src].float() * 3).to(torch.bfloat16)
    for j, p in enumerate(range(20, 120)):
        dst = int(bt[0, p])
        inp.k_cache[dst] = inp.k_cache[src]
        if perturb:
            c = j % 128
            v = inp.k_cache[dst, :, :, c].float()
            inp.k_cache[dst, :, :, c] = (v * (1.0 + (j + 1) / 512.0)).to(torch.bfloat16)
    small = full_check(inp)
    if not perturb:
        for h in range(8):   # the 50 lowest of the 101 identical pages
            assert small["gpu"]["idx"][0, h, :50].tolist() == list(range(20, 70))
    big = full_check(replicated(inp, 128))
    for r in range(128):
        assert np.array_equal(big["gpu"]["idx"][r:r + 1], small["gpu"]["idx"])


def test_signed_zero_keys_and_scores():
    log("case signed zeros")
    inp = small_inputs(2, 2, 16, (900, 333), seed=13, schedule=W.fixed_budget(6))
    k = inp.k_cache
    # whole pages of +0 / -0 keys: their scores are zero of either sign and tie
    bt = inp.block_table.cpu().numpy()
    for p, sign in ((5, 1.0), (6, -1.0), (7, 1.0)):
        k[int(bt[0, p])] = torch.zeros_like(k[int(bt[0, p])]) * sign
    half = k[int(bt[1, 2])].view(torch.int16)
    half[:, :, 0::2] = 0
    half[:, :, 1::2] = -32768  # bf16 -0
    full_check(inp)


@pytest.mark.parametrize("scale", [0.03, 0.25, 0.6])
@pytest.mark.parametrize("units", ["few", "many"])
def test_softmax_scale_is_applied(scale, units):
    """Sparse and dense attention at softmax scales other than 1/sqrt(128), on the
    one-workgroup-per-unit path (8 units) and the streaming path (320 units), against the
    oracle at the same scale; the whole-step call takes the scale as the separate calls do."""
    B, Hkv = (2, 4) if units == "few" else (40, 8)
    lengths = tuple(int(x) for x in np.random.default_rng(31).integers(300, 3000, size=B))
    log(f"case softmax scale {scale}, {B * Hkv} units")
    inp = small_inputs(2, Hkv, 16, lengths, seed=32, schedule=W.fixed_budget(20))
    h = host(inp)
    meta = torch.zeros((inp.num_phys_pages, Hkv, 2, 128), dtype=torch.bfloat16, device=DEV)
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta)
    s = inp.workload.schedule
    k, idx = S.page_score_topk(inp.q, meta, inp.block_table, inp.seq_lens, inp.k_cache.shape,
                               inp.min_pages, inp.frac_num, s.frac_den, s.bin_tokens, 20)
    out_s = S.sparse_decode_attn(inp.q, inp.k_cache, inp.v_cache, inp.block_table,
                                 inp.seq_lens, k, idx, scale)
    out_d = S.dense_decode_attn(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                                scale)
    step = S.SparseDecodeStep(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                              meta, inp.min_pages, inp.frac_num, s.frac_den, s.bin_tokens, 20,
                              scale=scale)
    whole = step.decode_step(None, None, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    gk, gidx = k.cpu().numpy(), idx.cpu().numpy()
    check_out(out_s.cpu().numpy().astype(np.float64),
              oracle.attention(h["q"], h["k"], h["v"], h["bt"], h["lens"], scale, gk, gidx),
              f"sparse, scale {scale}")
    check_out(out_d.cpu().numpy().astype(np.float64),
              oracle.attention(h["q"], h["k"], h["v"], h["bt"], h["lens"], scale),
              f"dense, scale {scale}")
    assert torch.equal(step.idx, idx)
    assert torch.equal(whole.view(torch.int32), out_s.view(torch.int32))


# ---------------------------------------------------------------------------------- metadata
@pytest.mark.parametrize("step", [1, 9, 40])
def test_meta_incremental_update_equals_rebuild(step):
    log(f"case meta update step {step}")
    inp = small_inputs(2, 4, 16, (100, 2000, 17, 5), seed=14, schedule=W.fixed_budget(3))
    full = inp.seq_lens.clone()
    short = torch.clamp(full - step, min=0)
    meta = torch.zeros((inp.num_phys_pages, 4, 2, 128), dtype=torch.bfloat16, device=DEV)
    S.page_meta_update(inp.k_cache, inp.block_table, short, meta)
    S.page_meta_update(inp.k_cache, inp.block_table, full, meta, first_pos=short)
    rebuilt = torch.zeros_like(meta)
    S.page_meta_update(inp.k_cache, inp.block_table, full, rebuilt)
    torch.cuda.synchronize()
    h = host(inp)
    pages = [int(x) for b, L in enumerate(h["lens"]) for x in h["bt"][b, :(int(L) + 15) // 16]]
    g1, g2 = W.bf16_bits(meta), W.bf16_bits(rebuilt)
    np.testing.assert_array_equal(g1[pages], g2[pages])
    check_meta(g1, oracle.page_meta(h["k"], h["bt"], h["lens"]), h["bt"], h["lens"], 16)


@pytest.mark.parametrize("ps", [32, 64, 128])
def test_meta_update_larger_pages(ps):
    log(f"case meta update ps {ps}")
    inp = small_inputs(2, 2, ps, (ps * 3 + 5, ps - 1), seed=15, schedule=W.fixed_budget(2))
    meta = torch.zeros((inp.num_phys_pages, 2, 2, 128), dtype=torch.bfloat16, device=DEV)
    short = torch.clamp(inp.seq_lens - 7, min=0)
    S.page_meta_update(inp.k_cache, inp.block_table, short, meta)
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta, first_pos=short)
    torch.cuda.synchronize()
    h = host(inp)
    check_meta(W.bf16_bits(meta), oracle.page_meta(h["k"], h["bt"], h["lens"]), h["bt"],
               h["lens"], ps)


# ---------------------------------------------------------------------------------- invariants
def test_full_budget_sparse_equals_dense_bitwise():
    log("case full budget == dense")
    inp = small_inputs(4, 2, 16, (3000, 777, 16), seed=16, schedule=W.fixed_budget(10000))
    k_max = inp.max_pages  # every page listed: the same wave partition as the dense call
    g = gpu_run(inp, k_max)
    np.testing.assert_array_equal(g["out_sparse"], g["out_dense"])


def test_runs_are_deterministic():
    log("case determinism")
    inp = small_inputs(5, 2, 16, (6000, 2000), seed=17, schedule=W.fraction_budget(1, 7))
    a = gpu_run(inp, 200)
    b = gpu_run(inp, 200)
    for key in ("meta", "k", "idx", "out_sparse", "out_dense"):
        np.testing.assert_array_equal(a[key], b[key])


def test_out_of_range_page_entries_are_skipped():
    log("case invalid idx entries")
    inp = small_inputs(2, 2, 16, (500, 900), seed=18, schedule=W.fixed_budget(4))
    idx = torch.tensor([[[0, 3, -1, 31], [2, 40, 5, 7]],
                        [[1, 2, 3, 4], [57, 56, 1000, 0]]], dtype=torch.int32, device=DEV)
    k = torch.tensor([4, 4], dtype=torch.int32, device=DEV)
    out = S.sparse_decode_attn(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                               k, idx, SCALE)
    torch.cuda.synchronize()
    h = host(inp)
    n = [(int(L) + 15) // 16 for L in h["lens"]]
    clean = np.full((2, 2, 4), -1, np.int32)
    kk = np.zeros(2, np.int32)
    ref = np.zeros((2, 4, 128))
    for b in range(2):
        for hh in range(2):
            valid = [p for p in idx[b, hh].tolist() if 0 <= p < n[b]]
            sub = np.full((1, 1, 4), -1, np.int32)
            sub[0, 0, :len(valid)] = valid
            one = oracle.attention(h["q"][b:b + 1, 2 * hh:2 * hh + 2], h["k"][:, hh:hh + 1],
                                   h["v"][:, hh:hh + 1], h["bt"][b:b + 1], h["lens"][b:b + 1],
                                   SCALE, np.array([len(valid)], np.int32), sub)
            ref[b, 2 * hh:2 * hh + 2] = one[0]
    check_out(out.cpu().numpy().astype(np.float64), ref, "invalid-idx sparse")


# ---------------------------------------------------------------------------------- full sizes
def sampled_check(inp, seqs, k_max, dense=True, label=""):
    """Full-size GPU run; oracle on the sampled sequences (all heads, all pages)."""
    w = inp.workload
    s = w.schedule
    ps = w.page_size
    log(f"  gpu run {label}: B={w.batch} P={inp.num_phys_pages} k_max={k_max}")
    g = gpu_run(inp, k_max, dense=dense)
    h = sample_inputs(inp, seqs)
    log(f"  oracle on sequences {list(seqs)}")
    ora_meta = oracle.page_meta(h["k"], h["bt"], h["lens"])
    # compare metadata of the sampled pages (GPU meta is indexed by physical page)
    np.testing.assert_array_equal(g["meta"][h["phys"]], ora_meta)
    s32, s64 = oracle.page_scores(h["q"], ora_meta, h["bt"], h["lens"], ps)
    ora_k = oracle_budgets(h["lens"], ps, s.bin_tokens, s.min_pages, s.frac_num,
                           s.frac_den, k_max)
    ora_idx = oracle.select(h["lens"], ora_k, s32, ps, k_max)
    gk = g["k"][list(seqs)]
    gidx = g["idx"][list(seqs)]
    excused = check_indices(gk, gidx, ora_k, ora_idx, s32, s64, h["lens"], ps, k_max)
    log(f"  indices match ({excused} near-tie pages excused)")
    ref_s = oracle.attention(h["q"], h["k"], h["v"], h["bt"], h["lens"], SCALE, gk, gidx)
    check_out(g["out_sparse"][list(seqs)], ref_s, "sparse")
    if dense:
        ref_d = oracle.attention(h["q"], h["k"], h["v"], h["bt"], h["lens"], SCALE)
        check_out(g["out_dense"][list(seqs)], ref_d, "dense")
    return g


def pick(inp, count, seed):
    rng = np.random.default_rng(seed)
    B = inp.workload.batch
    order = np.argsort(inp.lens_host)
    # shortest, longest and random others
    chosen = {int(order[0]), int(order[-1])}
    while len(chosen) < min(count, B):
        chosen.add(int(rng.integers(0, B)))
    return sorted(chosen)


def bound(inp):
    s = inp.workload.schedule
    return S.budget_bound(inp.lens_host, inp.workload.page_size, s.bin_tokens, s.min_pages,
                          s.frac_num, s.frac_den)


@pytest.mark.parametrize("cfg", ["c2", "c3", "c5"])
def test_full_size_sampled(cfg):
    log(f"case full-size {cfg}")
    inp = W.generate(W.CONFIGS[cfg], DEV)
    g = sampled_check(inp, pick(inp, 4, 1), bound(inp), label=cfg)
    if cfg == "c2":
        # every planted hot page is kept (the budget of at least 64 pages has room)
        for b in range(inp.workload.batch):
            for hh in range(inp.workload.num_kv_heads):
                assert set(inp.hot_host[b][hh]) <= set(g["idx"][b, hh].tolist())
    del inp
    torch.cuda.empty_cache()


def test_full_size_c4_budget_sweep():
    log("case full-size c4")
    inp = W.generate(W.C4, DEV)
    seqs = pick(inp, 3, 2)
    for i in range(len(W.C4_FRACTIONS)):   # 2, 5, 10, 25 and 100 % of the pages
        run = W.with_schedule(inp, W.c4_with_fraction(i))
        sampled_check(run, seqs, bound(run), dense=(i == 4), label=run.workload.name)
    del inp
    torch.cuda.empty_cache()


def test_full_size_c5_append_and_update():
    log("case full-size c5 append")
    w = W.C5
    inp = W.generate(w, DEV)
    meta = torch.zeros((inp.num_phys_pages, w.num_kv_heads, 2, 128), dtype=torch.bfloat16,
                       device=DEV)
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta)
    first = inp.seq_lens.clone()
    inp.seq_lens += 1   # the cache already holds a token at position L (the spare page)
    inp.lens_host = inp.lens_host + 1
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta, first_pos=first)
    torch.cuda.synchronize()
    seqs = pick(inp, 4, 3)
    h = sample_inputs(inp, seqs)
    np.testing.assert_array_equal(W.bf16_bits(meta)[h["phys"]],
                                  oracle.page_meta(h["k"], h["bt"], h["lens"]))
    sampled_check(inp, seqs, bound(inp), dense=False, label="c5 after append")


def test_workspace_reuse_across_sizes():
    log("case workspace reuse")
    inp = small_inputs(4, 2, 16, (9000, 3000, 700), seed=19, schedule=W.fraction_budget(1, 3))
    shape = S.shape_of(inp.q, inp.k_cache, inp.block_table)
    k_max = inp.max_pages
    # one workspace of each kind, left uninitialised, reused by every call below
    ws = torch.empty(S.sparrow_workspace_size(shape, k_max, S.SPARROW_OP_SPARSE_ATTN),
                     dtype=torch.uint8, device=DEV)
    dws = torch.empty(S.sparrow_workspace_size(shape, 0, S.SPARROW_OP_DENSE_ATTN),
                      dtype=torch.uint8, device=DEV)
    h = host(inp)
    n = np.array([(int(L) + 15) // 16 for L in h["lens"]], np.int32)
    rng = np.random.default_rng(0)
    for trial, frac in enumerate((1.0, 0.3, 0.05, 1.0)):
        kk = np.maximum(1, np.ceil(n * frac)).astype(np.int32)
        idx = np.full((3, 2, k_max), -1, np.int32)
        for b in range(3):
            for hh in range(2):
                idx[b, hh, :kk[b]] = np.sort(rng.choice(n[b], size=kk[b], replace=False))
        out = S.sparse_decode_attn(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                                   torch.as_tensor(kk, device=DEV), torch.as_tensor(idx, device=DEV),
                                   SCALE, workspace=ws)
        dense = S.dense_decode_attn(inp.q, inp.k_cache, inp.v_cache, inp.block_table,
                                    inp.seq_lens, SCALE, workspace=dws)
        torch.cuda.synchronize()
        ref = oracle.attention(h["q"], h["k"], h["v"], h["bt"], h["lens"], SCALE, kk, idx)
        check_out(out.cpu().numpy().astype(np.float64), ref, f"reuse sparse {trial}")
        if trial == 0:
            ref_d = oracle.attention(h["q"], h["k"], h["v"], h["bt"], h["lens"], SCALE)
        check_out(dense.cpu().numpy().astype(np.float64), ref_d, f"reuse dense {trial}")


# ---------------------------------------------------------------------------------- limits
def test_longest_sequence_the_block_table_allows():
    # SPARROW_MAX_PAGES_PER_SEQ pages of 16 tokens (245760 tokens) in one sequence, next to a
    # short one: the top-k keeps 15360 keys in LDS, the attention plan spans both.
    log("case max pages per sequence")
    n_max = S.SPARROW_MAX_PAGES_PER_SEQ
    lengths = (16 * n_max, 5000)
    w = W.small(B=2, Hq=8, Hkv=1, ps=16, lengths=lengths, seed=31,
                schedule=W.fraction_budget(1, 20, floor_pages=4), extra_pages=0)
    inp = W.generate(w, DEV, lengths=list(lengths))
    assert inp.max_pages == n_max
    full_check(inp)


@pytest.mark.parametrize("out_dtype", [S.SPARROW_OUT_F32, S.SPARROW_OUT_BF16])
def test_many_units_per_wave(out_dtype):
    """Several (sequence, KV head) units end inside one streaming wave's range (more units
    than resident waves, a few pages each): the finished units a wave holds until its range
    ends, and the ones past what it holds, are all written."""
    log(f"case many units per wave, out dtype {out_dtype}")
    rng = np.random.default_rng(33)
    B = 3000
    lengths = tuple(int(x) for x in rng.integers(0, 200, size=B))
    w = W.small(B=B, Hq=8, Hkv=2, ps=16, lengths=lengths, seed=33,
                schedule=W.fraction_budget(1, 3, floor_pages=1))
    inp = W.generate(w, DEV, lengths=list(lengths))
    full_check(inp, out_dtype=out_dtype)


def test_largest_batch():
    # SPARROW_MAX_BATCH ragged sequences (many empty or shorter than a page).
    log("case max batch")
    B = S.SPARROW_MAX_BATCH
    rng = np.random.default_rng(32)
    lengths = tuple(int(x) for x in rng.integers(0, 70, size=B))
    w = W.small(B=B, Hq=2, Hkv=1, ps=16, lengths=lengths, seed=32,
                schedule=W.fraction_budget(1, 2, floor_pages=1))
    inp = W.generate(w, DEV, lengths=list(lengths))
    full_check(inp)
