"""The C-ABI library: it loads, exports what include/sparrow.h declares, and
rejects bad host-visible arguments with the documented status before any GPU
work is enqueued.  Runs on the CPU (no compute call reaches a kernel)."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2606_08446_amd import sparrow as S
from paper_2606_08446_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sparrow.h")
FAKE = 0x1000  # non-null address that no test call ever dereferences


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^[A-Za-z_][\w \*]*?\b(sparrow_\w+)\s*\(", text, re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(S.LIB_PATH):
        from paper_2606_08446_amd import build
        build.build_library()
    return S.load()


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert set(names) == set(S.EXPORTS)
    for name in names:
        assert hasattr(lib, name), name


def test_struct_layouts_match_the_header():
    # the binding's structs must have the header's field order and sizes
    import ctypes
    assert ctypes.sizeof(S.Shape) == 40 and S.Shape.landmark.offset == 32
    assert S.Schedule.sink_pages.offset == 28 and S.Schedule.local_pages.offset == 32
    assert ctypes.sizeof(S.Schedule) == 40


def test_header_constants_match_binding():
    text = open(HEADER).read()
    consts = dict(re.findall(r"#define (SPARROW_\w+) \(?(-?\d+)\)?", text))
    for name, value in consts.items():
        assert getattr(S, name) == int(value), name


def good_shape(**kw):
    d = dict(batch=4, num_q_heads=16, num_kv_heads=8, page_size=16, max_pages_per_seq=64,
             num_phys_pages=300)
    d.update(kw)
    return S.make_shape(**d)


BAD_SHAPES = [
    (dict(head_dim=64), S.SPARROW_EUNSUPPORTED),
    (dict(num_q_heads=12, num_kv_heads=8), S.SPARROW_EINVAL),
    (dict(page_size=8), S.SPARROW_EUNSUPPORTED),
    (dict(page_size=48), S.SPARROW_EUNSUPPORTED),
    (dict(num_q_heads=136, num_kv_heads=8), S.SPARROW_EUNSUPPORTED),   # G = 17
    (dict(max_pages_per_seq=S.SPARROW_MAX_PAGES_PER_SEQ + 1), S.SPARROW_EUNSUPPORTED),
    (dict(max_pages_per_seq=0), S.SPARROW_EINVAL),
    (dict(batch=-1), S.SPARROW_EINVAL),
    (dict(num_kv_heads=0), S.SPARROW_EINVAL),
    (dict(num_phys_pages=0), S.SPARROW_EINVAL),
    (dict(landmark=2), S.SPARROW_EUNSUPPORTED),
    (dict(landmark=-1), S.SPARROW_EUNSUPPORTED),
]


def sched():
    return S.Schedule(2048, 1, FAKE, FAKE, 10)


def call(fn, shape, **over):
    """Call entry point `fn` with plausible fake pointers, overriding some arguments."""
    ws = over.pop("ws", FAKE)
    ws_bytes = over.pop("ws_bytes", 1 << 40)
    if fn == "meta":
        a = dict(k_cache=FAKE, bt=FAKE, lens=FAKE, first_pos=FAKE, meta=FAKE)
        a.update(over)
        return S.sparrow_page_meta_update(shape, a["k_cache"], a["bt"], a["lens"], a["first_pos"],
                                          a["meta"], None)
    if fn == "append":
        a = dict(k_new=FAKE, v_new=FAKE, k=FAKE, v=FAKE, bt=FAKE, lens=FAKE, meta=FAKE)
        a.update(over)
        return S.sparrow_append_kv(shape, a["k_new"], a["v_new"], a["k"], a["v"], a["bt"],
                                   a["lens"], a["meta"], None)
    if fn == "topk":
        a = dict(q=FAKE, meta=FAKE, bt=FAKE, lens=FAKE, sched=sched(), k_max=8, out_k=FAKE,
                 out_idx=FAKE)
        a.update(over)
        return S.sparrow_page_score_topk(shape, a["q"], a["meta"], a["bt"], a["lens"], a["sched"],
                                         a["k_max"], a["out_k"], a["out_idx"], ws, ws_bytes, None)
    if fn == "fused":
        a = dict(q=FAKE, k_new=FAKE, v_new=FAKE, k=FAKE, v=FAKE, meta=FAKE, bt=FAKE, lens=FAKE,
                 sched=sched(), k_max=8, out_k=FAKE, out_idx=FAKE)
        a.update(over)
        return S.sparrow_append_score_topk(shape, a["q"], a["k_new"], a["v_new"], a["k"], a["v"],
                                           a["meta"], a["bt"], a["lens"], a["sched"], a["k_max"],
                                           a["out_k"], a["out_idx"], ws, ws_bytes, None)
    if fn == "sparse":
        a = dict(q=FAKE, k=FAKE, v=FAKE, bt=FAKE, lens=FAKE, kk=FAKE, idx=FAKE, k_max=8,
                 out=FAKE, dtype=0)
        a.update(over)
        return S.sparrow_sparse_decode_attn(shape, a["q"], a["k"], a["v"], a["bt"], a["lens"],
                                            a["kk"], a["idx"], a["k_max"], 0.088, a["out"],
                                            a["dtype"], ws, ws_bytes, None)
    if fn == "step":
        a = dict(q=FAKE, k_new=FAKE, v_new=FAKE, k=FAKE, v=FAKE, meta=FAKE, bt=FAKE, lens=FAKE,
                 sched=sched(), k_max=8, out_k=FAKE, out_idx=FAKE, out=FAKE, dtype=0)
        a.update(over)
        return S.sparrow_decode_step(shape, a["q"], a["k_new"], a["v_new"], a["k"], a["v"],
                                     a["meta"], a["bt"], a["lens"], a["sched"], a["k_max"], 0.088,
                                     a["out_k"], a["out_idx"], a["out"], a["dtype"], ws, ws_bytes,
                                     None)
    a = dict(q=FAKE, k=FAKE, v=FAKE, bt=FAKE, lens=FAKE, out=FAKE, dtype=0)
    a.update(over)
    return S.sparrow_dense_decode_attn(shape, a["q"], a["k"], a["v"], a["bt"], a["lens"], 0.088,
                                       a["out"], a["dtype"], ws, ws_bytes, None)


@pytest.mark.parametrize("fn", ["meta", "append", "topk", "fused", "sparse", "dense", "step"])
@pytest.mark.parametrize("bad,status", BAD_SHAPES)
def test_bad_shapes_are_rejected(lib, fn, bad, status):
    bad = dict(bad)
    head_dim = bad.pop("head_dim", 128)
    shape = good_shape(**bad)
    shape.head_dim = head_dim
    assert call(fn, shape) == status


NULLS = {
    "meta": ["k_cache", "bt", "lens", "meta"],
    "append": ["k_new", "v_new", "k", "v", "bt", "lens", "meta"],
    "topk": ["q", "meta", "bt", "lens", "out_k", "out_idx"],
    "fused": ["q", "k_new", "v_new", "k", "v", "meta", "bt", "lens", "out_k", "out_idx"],
    "sparse": ["q", "k", "v", "bt", "lens", "kk", "idx", "out"],
    "dense": ["q", "k", "v", "bt", "lens", "out"],
    # (k_new and v_new may both be NULL: no append; one of them alone is refused below)
    "step": ["q", "k", "v", "meta", "bt", "lens", "out_k", "out_idx", "out"],
}


@pytest.mark.parametrize("fn,arg", [(f, a) for f, args in NULLS.items() for a in args])
def test_null_pointers_are_rejected(lib, fn, arg):
    assert call(fn, good_shape(), **{arg: None}) == S.SPARROW_EINVAL


def test_null_shape_and_schedule_are_rejected(lib):
    assert lib.sparrow_page_meta_update(None, FAKE, FAKE, FAKE, None, FAKE, None) == S.SPARROW_EINVAL
    assert call("topk", good_shape(), sched=S.Schedule(0, 1, FAKE, FAKE, 10)) == S.SPARROW_EINVAL
    assert call("topk", good_shape(), sched=S.Schedule(2048, 0, FAKE, FAKE, 10)) == S.SPARROW_EINVAL
    assert call("topk", good_shape(), sched=S.Schedule(2048, 1, FAKE, FAKE, 0)) == S.SPARROW_EINVAL
    assert call("topk", good_shape(), sched=S.Schedule(2048, 1, None, FAKE, 10)) == S.SPARROW_EINVAL
    assert call("topk", good_shape(), k_max=0) == S.SPARROW_EINVAL
    assert call("topk", good_shape(), sched=S.Schedule(2048, 1, FAKE, FAKE, 10, -1, 0)) == \
        S.SPARROW_EINVAL
    assert call("fused", good_shape(), sched=S.Schedule(2048, 1, FAKE, FAKE, 10, 0, -3)) == \
        S.SPARROW_EINVAL
    assert call("fused", good_shape(), k_max=0) == S.SPARROW_EINVAL
    assert call("fused", good_shape(), sched=S.Schedule(2048, 1, FAKE, None, 10)) == \
        S.SPARROW_EINVAL
    assert call("sparse", good_shape(), k_max=0) == S.SPARROW_EINVAL
    assert call("step", good_shape(), k_max=0) == S.SPARROW_EINVAL
    assert call("step", good_shape(), sched=S.Schedule(2048, 1, FAKE, FAKE, 10, 0, -1)) == \
        S.SPARROW_EINVAL
    assert call("step", good_shape(), sched=S.Schedule(2048, 1, None, FAKE, 10)) == \
        S.SPARROW_EINVAL
    assert call("step", good_shape(), k_new=None) == S.SPARROW_EINVAL
    assert call("step", good_shape(), v_new=None) == S.SPARROW_EINVAL
    # no budget exceeds the largest page count, so a longer row is refused
    big = S.SPARROW_MAX_PAGES_PER_SEQ + 1
    for fn in ("topk", "fused", "sparse", "step"):
        assert call(fn, good_shape(), k_max=big) == S.SPARROW_EINVAL
        assert call(fn, good_shape(), k_max=2**31 - 1) == S.SPARROW_EINVAL
    assert call("topk", good_shape(), k_max=S.SPARROW_MAX_PAGES_PER_SEQ, ws_bytes=0) == \
        S.SPARROW_EWORKSPACE


def test_unsupported_output_dtype(lib):
    assert call("sparse", good_shape(), dtype=2) == S.SPARROW_EUNSUPPORTED
    assert call("dense", good_shape(), dtype=7) == S.SPARROW_EUNSUPPORTED
    assert call("step", good_shape(), dtype=2) == S.SPARROW_EUNSUPPORTED


@pytest.mark.parametrize("fn,op", [("topk", S.SPARROW_OP_SCORE_TOPK),
                                   ("fused", S.SPARROW_OP_SCORE_TOPK),
                                   ("sparse", S.SPARROW_OP_SPARSE_ATTN),
                                   ("dense", S.SPARROW_OP_DENSE_ATTN),
                                   ("step", S.SPARROW_OP_DECODE_STEP)])
def test_workspace_checks(lib, fn, op):
    shape = good_shape()
    need = S.sparrow_workspace_size(shape, 8, op)
    assert need > 0
    assert call(fn, shape, ws=None) == S.SPARROW_EWORKSPACE
    assert call(fn, shape, ws_bytes=need - 1) == S.SPARROW_EWORKSPACE


def test_empty_batch_enqueues_nothing(lib):
    shape = good_shape(batch=0)
    for fn in ("meta", "append", "topk", "fused", "sparse", "dense", "step"):
        assert call(fn, shape, ws=None, ws_bytes=0) == S.SPARROW_OK


def test_workspace_size_properties(lib):
    shape = good_shape()
    assert S.sparrow_workspace_size(shape, 8, 99) == 0
    assert S.sparrow_workspace_size(good_shape(page_size=8), 8, 0) == 0
    assert S.sparrow_workspace_size(shape, 0, S.SPARROW_OP_SPARSE_ATTN) == 0
    assert S.sparrow_workspace_size(shape, S.SPARROW_MAX_PAGES_PER_SEQ + 1,
                                    S.SPARROW_OP_SPARSE_ATTN) == 0
    a = S.sparrow_workspace_size(shape, 8, S.SPARROW_OP_SPARSE_ATTN)
    b = S.sparrow_workspace_size(shape, 64, S.SPARROW_OP_SPARSE_ATTN)
    assert 0 < a <= b
    assert S.sparrow_workspace_size(shape, 1, S.SPARROW_OP_SCORE_TOPK) == 4 * 8 * 64 * 4
    # the whole step: the scores (rounded up to 256 bytes), then the attention's workspace
    score = S.sparrow_workspace_size(shape, 8, S.SPARROW_OP_SCORE_TOPK)
    assert S.sparrow_workspace_size(shape, 8, S.SPARROW_OP_DECODE_STEP) == \
        (score + 255) // 256 * 256 + a
    assert S.sparrow_workspace_size(shape, 0, S.SPARROW_OP_DECODE_STEP) == 0


def test_status_strings(lib):
    for code in (0, -1, -2, -3, -4, -99):
        assert isinstance(S.sparrow_status_string(code), str)
    assert S.sparrow_status_string(-3) != S.sparrow_status_string(-1)


def schedule_workloads():
    """Every schedule a workload uses: C1-C5, C4's five fractions, the Table 4 study."""
    ws = [W.CONFIGS[c] for c in ("c1", "c2", "c3", "c4", "c5")]
    ws += [W.c4_with_fraction(i) for i in range(len(W.C4_FRACTIONS))]
    ws += [W.table4(ps, 16384) for ps in (16, 32, 64, 128)]
    return ws


@pytest.mark.parametrize("w", schedule_workloads(), ids=lambda w: w.name)
def test_host_budget_bound_matches_oracle(w):
    # sparrow_budget_bound (the library's schedule arithmetic, run on the host) against the
    # oracle's budgets, per sequence, on lengths over and around the workload's range
    s = w.schedule
    rng = np.random.default_rng(3)
    lens = np.concatenate([rng.integers(w.len_lo, w.len_hi + 1, size=300),
                           [0, 1, w.page_size, w.page_size + 1, w.len_lo, w.len_hi,
                            w.len_hi + 5000, 2048, 2049]])
    want = oracle.budgets(lens, w.page_size, s.bin_tokens, s.min_pages, s.frac_num, s.frac_den)
    got, bound = S.budgets(lens, w.page_size, s.bin_tokens, s.min_pages, s.frac_num, s.frac_den)
    np.testing.assert_array_equal(got, want)
    assert bound == max(1, int(want.max()))
    assert S.budget_bound(lens, w.page_size, s.bin_tokens, s.min_pages, s.frac_num,
                          s.frac_den) == bound


@pytest.mark.parametrize("seed", range(8))
def test_host_budget_bound_random_schedules(seed):
    rng = np.random.default_rng(500 + seed)
    nb = int(rng.integers(1, 300))
    sch = W.Schedule(int(rng.choice([1, 7, 256, 2048])),
                     tuple(int(x) for x in rng.integers(0, 50, size=nb)),
                     tuple(int(x) for x in rng.integers(0, 1200, size=nb)),
                     int(rng.choice([1, 3, 1000])))
    ps = int(rng.choice([16, 32, 64, 128]))
    lens = rng.integers(-3, 60000, size=400)
    want = oracle.budgets(np.maximum(lens, 0), ps, sch.bin_tokens, sch.min_pages, sch.frac_num,
                          sch.frac_den)
    got, bound = S.budgets(lens, ps, sch.bin_tokens, sch.min_pages, sch.frac_num, sch.frac_den)
    np.testing.assert_array_equal(got, want)
    assert bound == max(1, int(want.max()))


def test_host_budget_bound_validates_arguments(lib):
    lens = np.array([100, 200], np.int32)
    mp = np.array([4], np.int32)
    fn = np.array([1], np.int32)

    def call(lens_p=lens.ctypes.data, n=2, ps=16, bt=2048, nb=1, mp_p=mp.ctypes.data,
             fn_p=fn.ctypes.data, den=10, out=None):
        return S.sparrow_budget_bound(lens_p, n, ps, bt, nb, mp_p, fn_p, den, out)
    assert call() == 4                       # ceil(13 / 10) = 2 < floor 4
    assert call(n=0, lens_p=None) == 1
    assert call(lens_p=None) == S.SPARROW_EINVAL
    assert call(n=-1) == S.SPARROW_EINVAL
    for kw in (dict(ps=0), dict(bt=0), dict(nb=0), dict(den=0), dict(mp_p=None),
               dict(fn_p=None)):
        assert call(**kw) == S.SPARROW_EINVAL, kw
    neg = np.array([-1], np.int32)
    assert call(mp_p=neg.ctypes.data) == S.SPARROW_EINVAL
    assert call(fn_p=neg.ctypes.data) == S.SPARROW_EINVAL
    too_long = np.array([16 * S.SPARROW_MAX_PAGES_PER_SEQ + 1], np.int32)
    assert call(lens_p=too_long.ctypes.data, n=1) == S.SPARROW_EINVAL
    longest = np.array([16 * S.SPARROW_MAX_PAGES_PER_SEQ], np.int32)
    assert call(lens_p=longest.ctypes.data, n=1, fn_p=np.array([10], np.int32).ctypes.data) == \
        S.SPARROW_MAX_PAGES_PER_SEQ


def test_tensor_wrappers_refuse_host_tensors():
    import torch
    q = torch.zeros(1, 2, 128, dtype=torch.bfloat16)
    with pytest.raises(RuntimeError):
        S.dense_decode_attn(q, torch.zeros(2, 1, 16, 128, dtype=torch.bfloat16),
                            torch.zeros(2, 1, 16, 128, dtype=torch.bfloat16),
                            torch.zeros(1, 2, dtype=torch.int32), torch.ones(1, dtype=torch.int32))


VEC16 = {"meta": ["k_cache", "meta"], "append": ["k_new", "v_new", "k", "v", "meta"],
         "topk": ["q", "meta", "ws"], "fused": ["q", "k_new", "v_new", "k", "v", "meta", "ws"],
         "sparse": ["q", "k", "v", "out", "ws"], "dense": ["q", "k", "v", "out", "ws"],
         "step": ["q", "k_new", "v_new", "k", "v", "meta", "out", "ws"]}


@pytest.mark.parametrize("fn,arg", [(f, a) for f, args in NULLS.items() for a in args] +
                         [(f, a) for f, args in VEC16.items() for a in args if a == "ws"] +
                         [("meta", "first_pos")])
def test_misaligned_pointers_are_rejected(lib, fn, arg):
    # Every pointer the kernels read or write must be at least 4-byte aligned.
    assert call(fn, good_shape(), **{arg: FAKE + 2}) == S.SPARROW_EINVAL


@pytest.mark.parametrize("fn,arg", [(f, a) for f, args in VEC16.items() for a in args])
def test_vector_pointers_need_16_byte_alignment(lib, fn, arg):
    assert call(fn, good_shape(), **{arg: FAKE + 4}) == S.SPARROW_EINVAL


def test_acceptance_entry_points_validate_arguments(lib):
    f32, bf16 = S.SPARROW_LOGITS_F32, S.SPARROW_LOGITS_BF16
    ok = dict(n=4, v=100, dt=f32, t=FAKE, d=FAKE, tau=1.0, a=FAKE)

    def acc(**kw):
        a = dict(ok, **kw)
        return S.sparrow_acceptance_rate(a["n"], a["v"], a["dt"], a["t"], a["d"], a["tau"],
                                         a["a"], None)
    assert acc(n=0) == S.SPARROW_OK
    assert acc(n=-1) == S.SPARROW_EINVAL
    assert acc(v=0) == S.SPARROW_EINVAL
    assert acc(dt=5) == S.SPARROW_EUNSUPPORTED
    for arg in ("t", "d", "a"):
        assert acc(**{arg: None}) == S.SPARROW_EINVAL
    assert acc(t=FAKE + 2) == S.SPARROW_EINVAL                 # fp32 rows need 4-byte alignment
    assert acc(dt=bf16, t=FAKE + 2, d=FAKE + 18, n=0) == S.SPARROW_OK   # same 16-byte phase
    assert acc(dt=bf16, t=FAKE + 2, d=FAKE + 4) == S.SPARROW_EINVAL     # different phases
    assert acc(tau=float("nan")) == S.SPARROW_EINVAL
    assert acc(tau=float("inf")) == S.SPARROW_EINVAL
    assert S.sparrow_acceptance_rate_topk(0, 20, FAKE, FAKE, FAKE, None) == S.SPARROW_OK
    assert S.sparrow_acceptance_rate_topk(5, 0, FAKE, FAKE, FAKE, None) == S.SPARROW_EINVAL
    assert S.sparrow_acceptance_rate_topk(5, 20, None, FAKE, FAKE, None) == S.SPARROW_EINVAL
    assert S.sparrow_acceptance_rate_topk(5, 20, FAKE + 2, FAKE, FAKE, None) == S.SPARROW_EINVAL

    def tail(**kw):
        a = dict(n=10, al=FAKE, pos=FAKE, bt=2048, nb=20, pct=5.0, q=FAKE, m=FAKE, c=FAKE)
        a.update(kw)
        return S.sparrow_tail_stats(a["n"], a["al"], a["pos"], a["bt"], a["nb"], a["pct"],
                                    a["q"], a["m"], a["c"], None)
    assert tail(n=-1) == S.SPARROW_EINVAL
    assert tail(bt=0) == S.SPARROW_EINVAL
    assert tail(nb=0) == S.SPARROW_EINVAL and tail(nb=65536) == S.SPARROW_EINVAL
    assert tail(pct=-0.5) == S.SPARROW_EINVAL and tail(pct=100.5) == S.SPARROW_EINVAL
    assert tail(pct=float("nan")) == S.SPARROW_EINVAL
    for arg in ("al", "pos", "q", "m", "c"):
        assert tail(**{arg: None}) == S.SPARROW_EINVAL
    assert tail(n=0, q=None) == S.SPARROW_EINVAL
    assert tail(q=FAKE + 4) == S.SPARROW_EINVAL               # fp64 outputs need 8-byte alignment


def test_stream_read_validates_arguments(lib):
    assert S.sparrow_stream_read(FAKE, 0, FAKE, None) == S.SPARROW_OK
    assert S.sparrow_stream_read(None, 0, FAKE, None) == S.SPARROW_OK
    assert S.sparrow_stream_read(None, 16, FAKE, None) == S.SPARROW_EINVAL
    assert S.sparrow_stream_read(FAKE, 16, None, None) == S.SPARROW_EINVAL
    assert S.sparrow_stream_read(FAKE, -16, FAKE, None) == S.SPARROW_EINVAL
    assert S.sparrow_stream_read(FAKE, 24, FAKE, None) == S.SPARROW_EINVAL   # not a multiple of 16
    assert S.sparrow_stream_read(FAKE + 8, 16, FAKE, None) == S.SPARROW_EINVAL
    assert S.sparrow_stream_read(FAKE, 16, FAKE + 2, None) == S.SPARROW_EINVAL


def test_noalloc_attention_validates_arguments(lib):
    # the workspace-free attention entry point checks its arguments like the one with a
    # workspace, and refuses shapes whose workspace exceeds the library's buffer
    shape = good_shape()
    ok = dict(q=FAKE, k=FAKE, v=FAKE, bt=FAKE, lens=FAKE, ksel=FAKE, idx=FAKE, k_max=8,
              out=FAKE, dt=S.SPARROW_OUT_F32)

    def call(shape=shape, **kw):
        a = dict(ok, **kw)
        return S.sparrow_sparse_decode_attn_noalloc(shape, a["q"], a["k"], a["v"], a["bt"],
                                                    a["lens"], a["ksel"], a["idx"], a["k_max"],
                                                    0.088, a["out"], a["dt"], None)
    for arg in ("q", "k", "v", "bt", "lens", "ksel", "idx", "out"):
        assert call(**{arg: None}) == S.SPARROW_EINVAL, arg
        assert call(**{arg: FAKE + 2}) == S.SPARROW_EINVAL, arg
    for arg in ("q", "k", "v", "out"):
        assert call(**{arg: FAKE + 4}) == S.SPARROW_EINVAL, arg
    assert call(k_max=0) == S.SPARROW_EINVAL
    assert call(k_max=S.SPARROW_MAX_PAGES_PER_SEQ + 1) == S.SPARROW_EINVAL
    assert call(dt=7) == S.SPARROW_EUNSUPPORTED
    assert call(shape=good_shape(batch=0)) == S.SPARROW_OK
    for kw, status in BAD_SHAPES:
        assert call(shape=good_shape(**kw)) == status, kw
    big = S.make_shape(8192, 16, 1, 16, 64, 1 << 20)
    assert S.sparrow_workspace_size(big, 8, S.SPARROW_OP_SPARSE_ATTN) > \
        S.SPARROW_NOALLOC_SCRATCH_BYTES
    assert call(shape=big) == S.SPARROW_EWORKSPACE
