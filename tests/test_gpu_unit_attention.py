"""GPU parity of the attention's one-workgroup-per-unit path against the CPU oracle.

A call takes that path when it has at most 256 (sequence, KV head) units, at most 8 query
heads per KV head, a list bound (k_max for the sparse call, the block table's width for
the dense one) of at most 1024 tokens and a block table of at most 4096 pages per
sequence; every other call streams.  The cases below sit on both sides of each of the four
limits, with ragged, empty and one-token sequences,
partial last pages, every page size and group sizes 1..8.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_08446_amd import sparrow as S
from paper_2606_08446_amd import workloads as W

from parity import SCALE, check_out, full_check, gpu_run, host, log

pytestmark = pytest.mark.gpu

DEV = "cuda"
UNIT_MAX_UNITS = 256
UNIT_MAX_TOKENS = 1024
UNIT_MAX_GROUP = 8
UNIT_MAX_BT = 4096


@pytest.fixture(autouse=True)
def _need_gpu(gpu_device):
    S.load()
    yield


def inputs(G, Hkv, ps, lengths, seed, schedule, extra_pages=0):
    w = W.small(B=len(lengths), Hq=G * Hkv, Hkv=Hkv, ps=ps, lengths=lengths, seed=seed,
                schedule=schedule, extra_pages=extra_pages)
    return W.generate(w, DEV, lengths=list(lengths))


def takes_unit_path(inp, list_bound):
    w = inp.workload
    return (w.batch * w.num_kv_heads <= UNIT_MAX_UNITS and w.group <= UNIT_MAX_GROUP
            and list_bound * w.page_size <= UNIT_MAX_TOKENS and inp.max_pages <= UNIT_MAX_BT)


# Sparse and dense both on the unit path: block tables of at most 1024 tokens.
UNIT_CASES = [
    # (G, Hkv, ps, lengths, schedule)
    (1, 2, 16, (1, 16, 17, 300, 512), W.fraction_budget(1, 3)),
    (2, 8, 16, (0, 511, 100, 37), W.fixed_budget(5)),
    (5, 2, 32, (480, 33, 1), W.fraction_budget(1, 2)),
    (8, 1, 64, (512, 65, 200), W.fraction_budget(1, 1)),
    (3, 4, 128, (129, 384, 500), W.fixed_budget(2)),
    (4, 3, 16, (0, 0, 7), W.fraction_budget(1, 4)),
    (7, 2, 32, (250, 31, 449, 2), W.fixed_budget(16)),
    (2, 4, 64, (1024, 1000, 63), W.fraction_budget(1, 3)),
    (6, 2, 16, (1024, 513, 16, 1), W.fixed_budget(64)),
]


@pytest.mark.parametrize("case", range(len(UNIT_CASES)))
def test_unit_path_sparse_and_dense(case):
    G, Hkv, ps, lengths, sched = UNIT_CASES[case]
    log(f"case unit path {case}: G={G} Hkv={Hkv} ps={ps} lens={lengths}")
    inp = inputs(G, Hkv, ps, lengths, seed=400 + case, schedule=sched)
    assert takes_unit_path(inp, inp.max_pages)
    full_check(inp)


@pytest.mark.parametrize("out_dtype", [S.SPARROW_OUT_F32, S.SPARROW_OUT_BF16])
def test_unit_path_full_budget_equals_dense_bitwise(out_dtype):
    log(f"case unit path, full budget == dense, out dtype {out_dtype}")
    inp = inputs(4, 2, 16, (500, 77, 16, 0), seed=410, schedule=W.fixed_budget(10000))
    k_max = inp.max_pages  # the dense call's list bound: both take the unit path
    assert takes_unit_path(inp, k_max)
    g = gpu_run(inp, k_max, out_dtype=out_dtype)
    np.testing.assert_array_equal(g["out_sparse"], g["out_dense"])


def test_unit_path_is_deterministic():
    log("case unit path determinism")
    inp = inputs(6, 2, 16, (480, 300, 9), seed=411, schedule=W.fraction_budget(1, 2))
    a = gpu_run(inp, 16)
    b = gpu_run(inp, 16)
    for key in ("k", "idx", "out_sparse", "out_dense"):
        np.testing.assert_array_equal(a[key], b[key])


def attend(inp, k, idx, k_max):
    """The sparse attention of explicit page lists on the GPU and in the oracle."""
    kk = np.asarray(k, np.int32)
    ii = np.asarray(idx, np.int32)
    assert ii.shape[2] == k_max
    out = S.sparse_decode_attn(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                               torch.as_tensor(kk, device=DEV), torch.as_tensor(ii, device=DEV),
                               SCALE)
    torch.cuda.synchronize()
    h = host(inp)
    ref = oracle.attention(h["q"], h["k"], h["v"], h["bt"], h["lens"], SCALE, kk, ii)
    return out.cpu().numpy().astype(np.float64), ref


@pytest.mark.parametrize("k_max", [64, 65])
def test_sparse_list_bound_at_the_switch(k_max):
    """k_max = 64 pages of 16 tokens (1024 tokens) takes the unit path, 65 streams; the same
    64-page lists give the oracle's output either way."""
    log(f"case list bound at the switch, k_max {k_max}")
    inp = inputs(2, 8, 16, (4096, 1000, 513), seed=412, schedule=W.fixed_budget(64),
                 extra_pages=1)
    assert takes_unit_path(inp, k_max) == (k_max == 64)
    rng = np.random.default_rng(412)
    B, Hkv = 3, 8
    n = [(L + 15) // 16 for L in (4096, 1000, 513)]
    idx = np.full((B, Hkv, k_max), -1, np.int32)
    k = np.array([min(64, x) for x in n], np.int32)
    for b in range(B):
        for h in range(Hkv):
            idx[b, h, :k[b]] = np.sort(rng.choice(n[b], size=k[b], replace=False))
    out, ref = attend(inp, k, idx, k_max)
    check_out(out, ref, f"k_max {k_max}")


@pytest.mark.parametrize("B", [32, 33])
def test_unit_count_at_the_switch(B):
    """256 units (32 sequences x 8 KV heads) take the unit path, 264 stream."""
    log(f"case unit count at the switch, batch {B}")
    rng = np.random.default_rng(413 + B)
    lengths = tuple(int(x) for x in rng.integers(0, 400, size=B))
    inp = inputs(2, 8, 16, lengths, seed=413 + B, schedule=W.fraction_budget(1, 3))
    assert takes_unit_path(inp, inp.max_pages) == (B == 32)
    full_check(inp)


@pytest.mark.parametrize("G", [8, 9])
def test_group_size_at_the_switch(G):
    """8 query heads per KV head take the unit path, 9 stream."""
    log(f"case group size at the switch, G {G}")
    inp = inputs(G, 2, 32, (300, 512, 1), seed=414 + G, schedule=W.fraction_budget(1, 2))
    assert takes_unit_path(inp, inp.max_pages) == (G == 8)
    full_check(inp)


def test_unit_path_skips_out_of_range_entries():
    """Page-list entries outside the sequence and block-table entries outside the cache add
    no tokens, as on the streaming path."""
    log("case unit path, invalid entries")
    inp = inputs(2, 2, 16, (200, 90), seed=415, schedule=W.fixed_budget(4))
    bt = inp.block_table.clone()
    bt[1, 2] = inp.num_phys_pages + 5      # logical page 2 of sequence 1 is absent
    inp.block_table.copy_(bt)
    idx = np.array([[[0, 3, -1, 12], [2, 40, 5, 7]],
                    [[1, 2, 3, 4], [5, 3, 1000, 0]]], np.int32)
    k = np.array([4, 4], np.int32)
    assert takes_unit_path(inp, 4)
    out = S.sparse_decode_attn(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                               torch.as_tensor(k, device=DEV), torch.as_tensor(idx, device=DEV),
                               SCALE)
    torch.cuda.synchronize()
    h = host(inp)
    n = [(int(L) + 15) // 16 for L in h["lens"]]
    ref = np.zeros((2, 4, 128))
    for b in range(2):
        for hh in range(2):
            valid = [p for p in idx[b, hh].tolist()
                     if 0 <= p < n[b] and 0 <= h["bt"][b, p] < inp.num_phys_pages]
            sub = np.full((1, 1, 4), -1, np.int32)
            sub[0, 0, :len(valid)] = valid
            one = oracle.attention(h["q"][b:b + 1, 2 * hh:2 * hh + 2], h["k"][:, hh:hh + 1],
                                   h["v"][:, hh:hh + 1], h["bt"][b:b + 1], h["lens"][b:b + 1],
                                   SCALE, np.array([len(valid)], np.int32), sub)
            ref[b, 2 * hh:2 * hh + 2] = one[0]
    check_out(out.cpu().numpy().astype(np.float64), ref, "unit path, invalid entries")


@pytest.mark.parametrize("pages", [4096, 4201])
def test_block_table_width_at_the_switch(pages):
    """A block-table row is staged in LDS: rows of up to 4096 pages take the unit path,
    wider ones stream."""
    log(f"case block table of {pages} pages")
    inp = inputs(2, 2, 16, (16 * pages - 5, 700), seed=416, schedule=W.fixed_budget(8))
    assert inp.max_pages == pages
    assert takes_unit_path(inp, 8) == (pages <= UNIT_MAX_BT)
    full_check(inp, k_max=8)
