"""GPU parity of sparrow_decode_step, the whole decode step in one call, through the C ABI.

It must give, bit for bit, what sparrow_append_score_topk (or sparrow_page_score_topk when
no token is appended) followed by sparrow_sparse_decode_attn gives on the same inputs:
caches, metadata, budgets, page lists and outputs.  The cases sit on both sides of the
attention's one-workgroup-per-unit switch (at most 256 units, G <= 8, k_max * page_size <=
1024 and a block table of at most 4096 pages), where the step runs the budget, the top-k and
the attention in one kernel after the scoring kernel; they cover forced sink/local pages,
schedule tables too long to stage on chip, the mean-key landmark, bf16 output, empty and
one-token sequences and capped budgets.  One case is checked against the CPU oracle as well.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_08446_amd import sparrow as S
from paper_2606_08446_amd import workloads as W

from parity import SCALE, check_indices, check_out, host, log
from test_gpu_append import append_case, clone_inputs

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(autouse=True)
def _need_gpu(gpu_device):
    S.load()
    yield


def unit_path(inp, k_max):
    w = inp.workload
    return (w.batch * w.num_kv_heads <= 256 and w.group <= 8 and k_max * w.page_size <= 1024
            and inp.max_pages <= 4096)


def sched_of(inp, sink=0, local=0):
    s = inp.workload.schedule
    return S.Schedule(s.bin_tokens, int(inp.min_pages.numel()), inp.min_pages.data_ptr(),
                      inp.frac_num.data_ptr(), s.frac_den, sink, local)


def outputs(inp, k_max, out_dtype):
    B, Hkv = inp.q.shape[0], inp.k_cache.shape[1]
    k = torch.full((B,), -7, dtype=torch.int32, device=DEV)
    idx = torch.full((B, Hkv, k_max), -7, dtype=torch.int32, device=DEV)
    out = torch.full(inp.q.shape, 3.0, dtype=torch.float32 if out_dtype == S.SPARROW_OUT_F32
                     else torch.bfloat16, device=DEV)
    return k, idx, out


def p(t):
    return None if t is None else t.data_ptr()


def run_step(inp, meta, kn, vn, k_max, sink=0, local=0, out_dtype=S.SPARROW_OUT_F32,
             landmark=S.SPARROW_LANDMARK_MINMAX):
    shape = S.shape_of(inp.q, inp.k_cache, inp.block_table, landmark=landmark)
    sched = sched_of(inp, sink, local)
    ws = torch.empty(S.sparrow_workspace_size(shape, k_max, S.SPARROW_OP_DECODE_STEP),
                     dtype=torch.uint8, device=DEV)
    k, idx, out = outputs(inp, k_max, out_dtype)
    S._check("sparrow_decode_step", S.sparrow_decode_step(
        shape, p(inp.q), p(kn), p(vn), p(inp.k_cache), p(inp.v_cache), p(meta),
        p(inp.block_table), p(inp.seq_lens), sched, k_max, SCALE, p(k), p(idx), p(out),
        out_dtype, p(ws), ws.numel(), torch.cuda.current_stream().cuda_stream))
    return k, idx, out


def run_separate(inp, meta, kn, vn, k_max, sink=0, local=0, out_dtype=S.SPARROW_OUT_F32,
                 landmark=S.SPARROW_LANDMARK_MINMAX):
    shape = S.shape_of(inp.q, inp.k_cache, inp.block_table, landmark=landmark)
    sched = sched_of(inp, sink, local)
    ws_s = torch.empty(S.sparrow_workspace_size(shape, k_max, S.SPARROW_OP_SCORE_TOPK),
                       dtype=torch.uint8, device=DEV)
    ws_a = torch.empty(S.sparrow_workspace_size(shape, k_max, S.SPARROW_OP_SPARSE_ATTN),
                       dtype=torch.uint8, device=DEV)
    k, idx, out = outputs(inp, k_max, out_dtype)
    stream = torch.cuda.current_stream().cuda_stream
    if kn is None:
        S._check("sparrow_page_score_topk", S.sparrow_page_score_topk(
            shape, p(inp.q), p(meta), p(inp.block_table), p(inp.seq_lens), sched, k_max, p(k),
            p(idx), p(ws_s), ws_s.numel(), stream))
    else:
        S._check("sparrow_append_score_topk", S.sparrow_append_score_topk(
            shape, p(inp.q), p(kn), p(vn), p(inp.k_cache), p(inp.v_cache), p(meta),
            p(inp.block_table), p(inp.seq_lens), sched, k_max, p(k), p(idx), p(ws_s),
            ws_s.numel(), stream))
    S._check("sparrow_sparse_decode_attn", S.sparrow_sparse_decode_attn(
        shape, p(inp.q), p(inp.k_cache), p(inp.v_cache), p(inp.block_table), p(inp.seq_lens),
        p(k), p(idx), k_max, SCALE, p(out), out_dtype, p(ws_a), ws_a.numel(), stream))
    return k, idx, out


def same_bits(t):
    """A device tensor viewed as integers, so that equality is bitwise."""
    return t.view(torch.int16 if t.element_size() == 2 else torch.int32)


def bits(t):
    """Bit patterns of a device tensor on the host."""
    return same_bits(t).cpu().numpy()


def same_step(inp, meta, kn, vn, k_max, **kw):
    """The whole-step call and the separate calls on copies of the same inputs: every result
    and every buffer they write must be equal bit for bit."""
    a_inp, b_inp = clone_inputs(inp), clone_inputs(inp)
    a_meta, b_meta = meta.clone(), meta.clone()
    a = run_step(a_inp, a_meta, kn, vn, k_max, **kw)
    b = run_separate(b_inp, b_meta, kn, vn, k_max, **kw)
    torch.cuda.synchronize()
    for name, x, y in zip(("k", "idx", "out"), a, b):
        np.testing.assert_array_equal(bits(x), bits(y), err_msg=name)
    # the caches and the metadata are compared on the device (tens of GB at full size)
    for name, x, y in (("k_cache", a_inp.k_cache, b_inp.k_cache),
                       ("v_cache", a_inp.v_cache, b_inp.v_cache), ("meta", a_meta, b_meta)):
        assert torch.equal(same_bits(x), same_bits(y)), name
    assert (a[0].cpu().numpy() >= 0).all()
    return a, a_inp


CASES = [
    # (G, Hkv, ps, lengths, schedule, k_max or None for the schedule's bound)
    (2, 8, 16, (4096, 1000, 513, 1, 0), W.fixed_budget(32), None),
    (4, 2, 32, (700, 33, 8000, 64), W.fraction_budget(1, 8, floor_pages=2), None),
    (8, 1, 64, (64, 65, 3000, 2), W.fraction_budget(1, 4), None),
    (5, 3, 128, (129, 1, 900, 7000), W.fixed_budget(8), None),
    (3, 4, 16, (2000, 17, 16, 15, 9000), W.rising_permille(2048, 2048, 8192, 30, 150), None),
    (1, 2, 16, (5000, 300), W.fraction_budget(1, 2), 20),  # budgets capped at k_max
    # streaming path: a list bound past 1024 tokens, G > 8, more than 256 units
    (2, 8, 16, (4096, 1000, 513, 1, 0), W.fixed_budget(80), None),
    (12, 1, 32, (6000, 31, 1900), W.fraction_budget(1, 16), None),
    (2, 8, 16, tuple(range(40, 40 * 34, 40)), W.fixed_budget(4), None),
]


@pytest.mark.parametrize("append", [True, False])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_step_equals_separate_calls(case, append):
    G, Hkv, ps, lengths, sched, k_max = CASES[case]
    log(f"case decode step {case} append={append}: G={G} Hkv={Hkv} ps={ps} lens={lengths}")
    inp, meta, meta0, kn, vn = append_case(G, Hkv, ps, lengths, seed=500 + case,
                                           schedule=sched, skip_last=False)
    if k_max is None:
        s = inp.workload.schedule
        k_max = S.budget_bound(inp.lens_host, ps, s.bin_tokens, s.min_pages, s.frac_num,
                               s.frac_den)
    log(f"  k_max {k_max}, unit path {unit_path(inp, k_max)}")
    if append:
        same_step(inp, meta, kn, vn, k_max)
    else:
        same_step(inp, meta, None, None, k_max)


def test_step_matches_the_oracle():
    """The one-kernel selection and attention (a batch-1-like unit-path case) against the
    CPU oracle's whole step after its append."""
    log("case decode step vs oracle")
    inp, meta, meta0, kn, vn = append_case(2, 8, 16, (4096, 1000, 513, 1), seed=520,
                                           schedule=W.fixed_budget(32), skip_last=False)
    assert unit_path(inp, 32)
    h = host(inp)
    (k, idx, out), a_inp = same_step(inp, meta, kn, vn, 32)
    kc, vc, _ = oracle.append_kv(W.bf16_bits(kn), W.bf16_bits(vn), h["k"], h["v"], h["bt"],
                                 h["lens"], meta0)
    s = inp.workload.schedule
    ref = oracle.sparse_step(h["q"], kc, vc, h["bt"], h["lens"],
                             (s.bin_tokens, s.min_pages, s.frac_num, s.frac_den), 32, SCALE)
    check_indices(k.cpu().numpy(), idx.cpu().numpy(), ref["k"], ref["idx"], ref["scores32"],
                  ref["scores64"], h["lens"], 16, 32)
    # attention over the GPU's (validated) page lists
    ref_out = oracle.attention(h["q"], kc, vc, h["bt"], h["lens"], SCALE, k.cpu().numpy(),
                               idx.cpu().numpy())
    check_out(out.cpu().numpy().astype(np.float64), ref_out, "decode step")


@pytest.mark.parametrize("sink,local", [(1, 0), (0, 3), (2, 2)])
def test_step_forced_pages(sink, local):
    log(f"case decode step, forced pages sink={sink} local={local}")
    inp, meta, _, kn, vn = append_case(2, 4, 16, (900, 40, 17, 3000), seed=530 + sink + local,
                                       schedule=W.fixed_budget(6), skip_last=False)
    assert unit_path(inp, 6)
    same_step(inp, meta, kn, vn, 6, sink=sink, local=local)


def test_step_schedule_too_long_to_stage():
    """600 schedule bins (more than the 512 the one-kernel step stages on chip): the budget
    is read from the tables in HBM instead."""
    log("case decode step, 600-bin schedule")
    mins = tuple(1 + (i % 7) for i in range(600))
    fracs = tuple(i % 50 for i in range(600))
    sched = W.Schedule(16, mins, fracs, 200)
    inp, meta, _, kn, vn = append_case(2, 4, 16, (9000, 800, 31, 5), seed=540,
                                       schedule=sched, skip_last=False)
    k_max = S.budget_bound(inp.lens_host, 16, 16, mins, fracs, 200)
    k_max = min(k_max, 40)
    assert unit_path(inp, k_max)
    same_step(inp, meta, kn, vn, k_max)


def test_step_bf16_output():
    log("case decode step, bf16 output")
    inp, meta, _, kn, vn = append_case(4, 2, 32, (700, 33, 8000), seed=550,
                                       schedule=W.fixed_budget(10), skip_last=False)
    same_step(inp, meta, kn, vn, 10, out_dtype=S.SPARROW_OUT_BF16)


def test_step_mean_landmark():
    log("case decode step, mean-key landmark")
    lengths = (2000, 300, 16, 4097)
    w = W.small(B=4, Hq=8, Hkv=4, ps=16, lengths=lengths, seed=560,
                schedule=W.fixed_budget(12))
    inp = W.generate(w, DEV, lengths=list(lengths))
    lens = np.asarray(lengths, np.int32)
    meta = S.new_meta(inp.num_phys_pages, 4, DEV, landmark=S.SPARROW_LANDMARK_MEAN)
    S.page_meta_update(inp.k_cache, inp.block_table, torch.as_tensor(lens - 1, device=DEV), meta,
                       landmark=S.SPARROW_LANDMARK_MEAN)
    g = torch.Generator(device=DEV)
    g.manual_seed(561)
    kn = torch.randn((4, 4, 128), generator=g, device=DEV).to(torch.bfloat16)
    vn = torch.randn((4, 4, 128), generator=g, device=DEV).to(torch.bfloat16)
    assert unit_path(inp, 12)
    same_step(inp, meta, kn, vn, 12, landmark=S.SPARROW_LANDMARK_MEAN)


def test_step_through_the_tensor_wrapper():
    """SparseDecodeStep.decode_step gives what append_score_topk + attend give."""
    log("case decode step, tensor wrapper")
    inp, meta, _, kn, vn = append_case(2, 8, 16, (4096, 700), seed=570,
                                       schedule=W.fixed_budget(32), skip_last=False)
    s = inp.workload.schedule
    outs = []
    for whole in (True, False):
        c = clone_inputs(inp)
        m = meta.clone()
        step = S.SparseDecodeStep(c.q, c.k_cache, c.v_cache, c.block_table, c.seq_lens, m,
                                  c.min_pages, c.frac_num, s.frac_den, s.bin_tokens, 32)
        stream = torch.cuda.current_stream().cuda_stream
        if whole:
            step.decode_step(kn, vn, stream)
        else:
            step.append_score_topk(kn, vn, stream)
            step.attend(stream)
        torch.cuda.synchronize()
        outs.append((step.k.cpu().numpy(), step.idx.cpu().numpy(), step.out.cpu().numpy()))
    for x, y in zip(outs[0], outs[1]):
        np.testing.assert_array_equal(x, y)


@pytest.mark.parametrize("cfg", ["c2", "c4-2"])
def test_step_full_size(cfg):
    """Full-size Qwen3-shaped batches (the streaming path): the whole-step call equals the
    separate calls bit for bit, appended token included."""
    log(f"case decode step, full size {cfg}")
    w = W.C2 if cfg == "c2" else W.c4_with_fraction(0)
    inp = W.generate(w, DEV)
    lens = inp.lens_host.astype(np.int32)
    meta = S.new_meta(inp.num_phys_pages, w.num_kv_heads, DEV)
    S.page_meta_update(inp.k_cache, inp.block_table, torch.as_tensor(lens - 1, device=DEV), meta)
    g = torch.Generator(device=DEV)
    g.manual_seed(580)
    kn = torch.randn((w.batch, w.num_kv_heads, 128), generator=g, device=DEV).to(torch.bfloat16)
    vn = torch.randn((w.batch, w.num_kv_heads, 128), generator=g, device=DEV).to(torch.bfloat16)
    s = w.schedule
    k_max = S.budget_bound(inp.lens_host, w.page_size, s.bin_tokens, s.min_pages, s.frac_num,
                           s.frac_den)
    assert not unit_path(inp, k_max)
    same_step(inp, meta, kn, vn, k_max)


@pytest.mark.parametrize("case", [0, 3, 6])
def test_step_sequence_past_the_block_table(case):
    """The longest sequence gets a length one past what its block table addresses: the
    append leaves it alone and its length is clamped, in both forms of the step."""
    G, Hkv, ps, lengths, sched, _ = CASES[case]
    log(f"case decode step {case}, a sequence past its block table")
    inp, meta, _, kn, vn = append_case(G, Hkv, ps, lengths, seed=590 + case, schedule=sched,
                                       skip_last=True)
    s = inp.workload.schedule
    k_max = S.budget_bound(np.minimum(inp.lens_host, ps * inp.max_pages), ps, s.bin_tokens,
                           s.min_pages, s.frac_num, s.frac_den)
    same_step(inp, meta, kn, vn, k_max)


@pytest.mark.parametrize("case", [0, 6])
def test_step_absent_pages(case):
    """Block-table entries outside the cache inside the sequences (absent pages: scored 0,
    left out of the attention, no append to them) give the same results in both forms."""
    G, Hkv, ps, lengths, sched, _ = CASES[case]
    log(f"case decode step {case}, absent pages")
    inp, meta, _, kn, vn = append_case(G, Hkv, ps, lengths, seed=600 + case, schedule=sched,
                                       skip_last=False)
    bt = inp.block_table.clone()
    P = inp.num_phys_pages
    for b, L in enumerate(lengths):
        n = (L + ps - 1) // ps
        if n >= 3:
            bt[b, 1] = P + 3          # past the cache
            bt[b, n - 1] = -2         # negative: the page that takes the appended token
    inp.block_table.copy_(bt)
    s = inp.workload.schedule
    k_max = S.budget_bound(inp.lens_host, ps, s.bin_tokens, s.min_pages, s.frac_num,
                           s.frac_den)
    same_step(inp, meta, kn, vn, k_max)


def random_step_case(seed):
    """A seeded shape for the whole-step call: two seeds in three are drawn inside the
    one-kernel selection and attention's limits (G <= 8, a fixed budget with
    k_max * page_size <= 1024, few units), the third from any shape and schedule form."""
    rng = np.random.default_rng(4200 + seed)
    small = seed % 3 != 2
    G = int(rng.choice([1, 2, 3, 4, 5, 8] if small else [1, 2, 4, 8, 12, 16]))
    Hkv = int(rng.integers(1, 9 if small else 13))
    ps = int(rng.choice([16, 32, 64, 128]))
    B = int(rng.integers(1, 7))
    lengths = [int(x) for x in rng.integers(0, 9000, size=B)]
    if rng.random() < 0.4:
        lengths[int(rng.integers(0, B))] = int(rng.choice([0, 1, ps, ps + 1]))
    if small:
        sched = W.fixed_budget(int(rng.integers(1, 1024 // ps + 1)))
    elif rng.random() < 0.5:
        sched = W.fraction_budget(int(rng.integers(1, 5)), int(rng.integers(5, 20)),
                                  floor_pages=int(rng.integers(0, 6)))
    else:
        sched = W.rising_permille(2048, 2048, 8192, int(rng.integers(20, 100)),
                                  int(rng.integers(100, 400)))
    return G, Hkv, ps, tuple(lengths), sched


@pytest.mark.parametrize("seed", range(12))
def test_random_shapes_whole_step(seed):
    """Seeded random shapes: the whole-step call equals the separate calls bit for bit, and
    its budgets, page lists and outputs match the CPU oracle's step after the append."""
    G, Hkv, ps, lengths, sched = random_step_case(seed)
    inp, meta, meta0, kn, vn = append_case(G, Hkv, ps, lengths, seed=610 + seed,
                                           schedule=sched, skip_last=False)
    s = inp.workload.schedule
    k_max = S.budget_bound(inp.lens_host, ps, s.bin_tokens, s.min_pages, s.frac_num,
                           s.frac_den)
    log(f"case decode step random {seed}: G={G} Hkv={Hkv} ps={ps} lens={lengths} "
        f"k_max {k_max}, unit path {unit_path(inp, k_max)}")
    h = host(inp)
    (k, idx, out), _ = same_step(inp, meta, kn, vn, k_max)
    kc, vc, _ = oracle.append_kv(W.bf16_bits(kn), W.bf16_bits(vn), h["k"], h["v"], h["bt"],
                                 h["lens"], meta0)
    ref = oracle.sparse_step(h["q"], kc, vc, h["bt"], h["lens"],
                             (s.bin_tokens, s.min_pages, s.frac_num, s.frac_den), k_max, SCALE)
    k_h, idx_h = k.cpu().numpy(), idx.cpu().numpy()
    check_indices(k_h, idx_h, ref["k"], ref["idx"], ref["scores32"], ref["scores64"],
                  h["lens"], ps, k_max)
    ref_out = oracle.attention(h["q"], kc, vc, h["bt"], h["lens"], SCALE, k_h, idx_h)
    check_out(out.cpu().numpy().astype(np.float64), ref_out, f"decode step random {seed}")
