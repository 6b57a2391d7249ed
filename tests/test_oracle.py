"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these tests compares the oracle with itself: each checks it against a
brute-force or library computation written independently here (numpy, scipy,
fractions), a closed form, an invariant, or a value printed in the paper
(``tests/golden``).  All run on the CPU.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.special

import oracle
from paper_2606_08446_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
SCALE = 1.0 / math.sqrt(128.0)


# ----------------------------------------------------------------------------- helpers
def bits_to_f64(a):
    return (np.asarray(a, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f32_to_bf16_bits(x):
    """Round fp32 values to bf16 (nearest even) and return the bit patterns."""
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    return r


def host_inputs(B=3, Hq=4, Hkv=2, ps=16, lengths=(37, 64, 90), seed=0, **kw):
    w = W.small(B=B, Hq=Hq, Hkv=Hkv, ps=ps, lengths=lengths, seed=seed, **kw)
    inp = W.generate(w, "cpu", lengths=list(lengths))
    return dict(
        q=W.bf16_bits(inp.q), k=W.bf16_bits(inp.k_cache), v=W.bf16_bits(inp.v_cache),
        bt=inp.block_table.numpy().copy(), lens=inp.seq_lens.numpy().copy(), w=w, ps=ps)


def tokens_of(d, b, h, pages=None):
    """Logical token list of sequence b, KV head h: (keys fp64 [T][D], values fp64 [T][D])."""
    ps = d["ps"]
    L = int(d["lens"][b])
    n = (L + ps - 1) // ps
    pages = range(n) if pages is None else pages
    ks, vs = [], []
    for p in pages:
        phys = d["bt"][b, p]
        for t in range(ps):
            if p * ps + t < L:
                ks.append(bits_to_f64(d["k"][phys, h, t]))
                vs.append(bits_to_f64(d["v"][phys, h, t]))
    return np.array(ks), np.array(vs)


def order_key(bits):
    """bf16 bit pattern -> integer whose order is the total order of the values (-0 < +0)."""
    b = np.asarray(bits, np.uint16).astype(np.int32)
    neg = (b & 0x8000) != 0
    return np.where(neg, -(b & 0x7FFF) - 1, b)


# ----------------------------------------------------------------------------- metadata
def test_meta_matches_brute_force_total_order():
    d = host_inputs(lengths=(37, 64, 1), seed=1)
    # plant signed zeros so that the -0 < +0 rule is exercised
    k = d["k"].copy()
    k[d["bt"][0, 0], 0, :, 5] = [0x8000, 0x0000] * 8        # whole channel of signed zeros
    k[d["bt"][0, 0], 1, :, 7] = [0x0000, 0x8000] * 8
    d["k"] = k
    meta = oracle.page_meta(d["k"], d["bt"], d["lens"])
    ps = d["ps"]
    for b, L in enumerate(d["lens"]):
        for p in range((L + ps - 1) // ps):
            phys = d["bt"][b, p]
            valid = min(ps, L - p * ps)
            for h in range(d["k"].shape[1]):
                rows = d["k"][phys, h, :valid]                   # [valid][D]
                keys = order_key(rows)
                mn = rows[np.argmin(keys, axis=0), np.arange(rows.shape[1])]
                mx = rows[np.argmax(keys, axis=0), np.arange(rows.shape[1])]
                np.testing.assert_array_equal(meta[phys, h, 0], mn)
                np.testing.assert_array_equal(meta[phys, h, 1], mx)
    assert meta[d["bt"][0, 0], 0, 0, 5] == 0x8000 and meta[d["bt"][0, 0], 0, 1, 5] == 0x0000
    assert meta[d["bt"][0, 0], 1, 0, 7] == 0x8000 and meta[d["bt"][0, 0], 1, 1, 7] == 0x0000


def test_meta_single_token_page_is_the_key():
    d = host_inputs(lengths=(17, 33, 1), seed=2)
    meta = oracle.page_meta(d["k"], d["bt"], d["lens"])
    for b, L in enumerate(d["lens"]):
        p = (L - 1) // 16  # the last page holds exactly one token
        phys = d["bt"][b, p]
        np.testing.assert_array_equal(meta[phys, :, 0], d["k"][phys, :, 0])
        np.testing.assert_array_equal(meta[phys, :, 1], d["k"][phys, :, 0])


@pytest.mark.parametrize("step", [1, 5, 37])
def test_meta_incremental_update_equals_rebuild(step):
    d = host_inputs(lengths=(50, 64, 95), seed=3)
    full = d["lens"].copy()
    short = np.maximum(full - step, 0).astype(np.int32)
    meta_short = oracle.page_meta(d["k"], d["bt"], short)
    updated = oracle.page_meta(d["k"], d["bt"], full, first_pos=short, meta=meta_short)
    rebuilt = oracle.page_meta(d["k"], d["bt"], full)
    # only the pages the sequences use are defined
    for b, L in enumerate(full):
        for p in range((L + 15) // 16):
            np.testing.assert_array_equal(updated[d["bt"][b, p]], rebuilt[d["bt"][b, p]])


# ----------------------------------------------------------------------------- append
def _rand_bits(rng, shape):
    return f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32))


def test_append_writes_exactly_one_row_per_head_and_rebuilds_its_page():
    # lengths: mid-page, first slot of a fresh page, last slot of a page, empty, beyond the table
    d = host_inputs(B=5, lengths=(37, 33, 48, 0, 20), seed=21)
    rng = np.random.default_rng(5)
    B, Hkv, D, ps = 5, 2, 128, 16
    lens = d["lens"].copy()
    cap = ps * d["bt"].shape[1]
    lens[4] = cap + 1                       # cannot be addressed: skipped
    kn, vn = _rand_bits(rng, (B, Hkv, D)), _rand_bits(rng, (B, Hkv, D))
    meta0 = oracle.page_meta(d["k"], d["bt"], np.minimum(lens, cap).astype(np.int32))
    kc, vc, mt = oracle.append_kv(kn, vn, d["k"], d["v"], d["bt"], lens, meta0)
    k_exp, v_exp = d["k"].copy(), d["v"].copy()
    touched = []
    for b, L in enumerate(lens):
        if L < 1 or L > cap:
            continue
        phys, slot = d["bt"][b, (L - 1) // ps], (L - 1) % ps
        k_exp[phys, :, slot], v_exp[phys, :, slot] = kn[b], vn[b]
        touched.append((b, phys, min(ps, L - (L - 1) // ps * ps)))
    np.testing.assert_array_equal(kc, k_exp)        # the new rows and nothing else
    np.testing.assert_array_equal(vc, v_exp)
    for b, phys, valid in touched:
        for h in range(Hkv):
            rows = k_exp[phys, h, :valid]
            keys = order_key(rows)
            np.testing.assert_array_equal(mt[phys, h, 0],
                                          rows[np.argmin(keys, 0), np.arange(D)])
            np.testing.assert_array_equal(mt[phys, h, 1],
                                          rows[np.argmax(keys, 0), np.arange(D)])
    # the in-place form gives the same arrays
    kc2, vc2, mt2 = d["k"].copy(), d["v"].copy(), meta0.copy()
    oracle.append_kv(kn, vn, kc2, vc2, d["bt"], lens, mt2, inplace=True)
    np.testing.assert_array_equal(kc2, kc)
    np.testing.assert_array_equal(vc2, vc)
    np.testing.assert_array_equal(mt2, mt)
    # pages nobody appended to keep their metadata
    untouched = np.ones(mt.shape[0], bool)
    untouched[[t[1] for t in touched]] = False
    np.testing.assert_array_equal(mt[untouched], meta0[untouched])


def test_appending_token_by_token_equals_building_at_once():
    # Grow three sequences from empty, one token per step, and compare with writing the
    # whole sequences into the cache first and building the metadata in one pass.
    d = host_inputs(B=3, lengths=(40, 16, 17), seed=22)
    full = d["lens"].copy()
    B, Hkv = 3, 2
    kc = np.zeros_like(d["k"])
    vc = np.zeros_like(d["v"])
    mt = np.zeros((kc.shape[0], Hkv, 2, 128), np.uint16)
    for t in range(int(full.max())):
        lens = np.minimum(full, t + 1).astype(np.int32)
        grow = (full > t)
        kn = np.zeros((B, Hkv, 128), np.uint16)
        vn = np.zeros((B, Hkv, 128), np.uint16)
        for b in range(B):
            if grow[b]:
                phys = d["bt"][b, t // 16]
                kn[b], vn[b] = d["k"][phys, :, t % 16], d["v"][phys, :, t % 16]
        lens_step = np.where(grow, lens, 0).astype(np.int32)   # finished sequences sit out
        kc, vc, mt = oracle.append_kv(kn, vn, kc, vc, d["bt"], lens_step, mt)
    rebuilt = oracle.page_meta(d["k"], d["bt"], full)
    for b, L in enumerate(full):
        for p in range((L + 15) // 16):
            phys = d["bt"][b, p]
            valid = min(16, L - p * 16)
            np.testing.assert_array_equal(kc[phys, :, :valid], d["k"][phys, :, :valid])
            np.testing.assert_array_equal(vc[phys, :, :valid], d["v"][phys, :, :valid])
            np.testing.assert_array_equal(mt[phys], rebuilt[phys])


# ----------------------------------------------------------------------------- scores
def brute_scores64(d, meta, b, h, G):
    n = (int(d["lens"][b]) + d["ps"] - 1) // d["ps"]
    out = np.zeros(n)
    for p in range(n):
        phys = d["bt"][b, p]
        mn = bits_to_f64(meta[phys, h, 0])
        mx = bits_to_f64(meta[phys, h, 1])
        tot = []
        for g in range(G):
            qj = bits_to_f64(d["q"][b, h * G + g])
            tot.extend(np.maximum(qj * mn, qj * mx))
        out[p] = math.fsum(tot)
    return out


@pytest.mark.parametrize("Hq,Hkv", [(4, 2), (2, 2), (10, 2)])
def test_scores_match_brute_force(Hq, Hkv):
    d = host_inputs(Hq=Hq, Hkv=Hkv, lengths=(37, 130, 16), seed=4)
    meta = oracle.page_meta(d["k"], d["bt"], d["lens"])
    s32, s64 = oracle.page_scores(d["q"], meta, d["bt"], d["lens"], d["ps"])
    G = Hq // Hkv
    for b in range(3):
        for h in range(Hkv):
            ref = brute_scores64(d, meta, b, h, G)
            n = len(ref)
            np.testing.assert_allclose(s64[b, h, :n], ref, rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(s32[b, h, :n], ref, rtol=2e-5, atol=1e-4)


def test_score_upper_bounds_every_token_logit():
    d = host_inputs(Hq=6, Hkv=2, lengths=(77, 100, 20), seed=5)
    meta = oracle.page_meta(d["k"], d["bt"], d["lens"])
    _, s64 = oracle.page_scores(d["q"], meta, d["bt"], d["lens"], d["ps"])
    G = 3
    for b in range(3):
        for h in range(2):
            L = int(d["lens"][b])
            for p in range((L + 15) // 16):
                keys, _ = tokens_of(d, b, h, [p])
                qs = np.stack([bits_to_f64(d["q"][b, h * G + g]) for g in range(G)])
                logits = (keys @ qs.T).sum(axis=1)   # sum over the group of q_j . k_t
                assert s64[b, h, p] >= logits.max() - 1e-9


def test_single_token_page_score_is_the_dot_product():
    d = host_inputs(Hq=4, Hkv=2, lengths=(1, 17, 33), seed=6)
    meta = oracle.page_meta(d["k"], d["bt"], d["lens"])
    _, s64 = oracle.page_scores(d["q"], meta, d["bt"], d["lens"], d["ps"])
    for b in range(3):
        p = (int(d["lens"][b]) - 1) // 16
        for h in range(2):
            k = bits_to_f64(d["k"][d["bt"][b, p], h, 0])
            want = math.fsum(math.fsum(bits_to_f64(d["q"][b, h * 2 + g]) * k) for g in range(2))
            assert abs(s64[b, h, p] - want) <= 1e-12 * max(1.0, abs(want))


def test_scaling_query_by_two_scales_scores_exactly():
    d = host_inputs(lengths=(200, 150, 64), seed=7)
    meta = oracle.page_meta(d["k"], d["bt"], d["lens"])
    s32, _ = oracle.page_scores(d["q"], meta, d["bt"], d["lens"], 16)
    q2 = f32_to_bf16_bits(bits_to_f64(d["q"]).astype(np.float32) * 2)
    t32, _ = oracle.page_scores(q2, meta, d["bt"], d["lens"], 16)
    mask = ~np.isnan(s32)
    np.testing.assert_array_equal(t32[mask], 2 * s32[mask])
    k = np.array([3, 3, 2], np.int32)
    np.testing.assert_array_equal(oracle.select(d["lens"], k, s32, 16, 3),
                                  oracle.select(d["lens"], k, t32, 16, 3))


# ----------------------------------------------------------------------------- budget
def budget_fraction_reference(L, ps, bin_tokens, min_pages, frac_num, frac_den):
    if L <= 0:
        return 0
    n = -(-L // ps)
    b = min((L - 1) // bin_tokens, len(min_pages) - 1)
    want = max(min_pages[b], math.ceil(Fraction(n * frac_num[b], frac_den)))
    return min(max(want, 1), n)


@pytest.mark.parametrize("sched", [W.C1.schedule, W.C2.schedule, W.C3.schedule, W.C5.schedule]
                         + [W.fraction_budget(n, d) for n, d in W.C4_FRACTIONS])
@pytest.mark.parametrize("ps", [16, 32])
def test_budget_matches_integer_reference(sched, ps):
    rng = np.random.default_rng(8)
    lens = np.concatenate([[0, 1, 2, ps - 1, ps, ps + 1, 2047, 2048, 2049, 4096, 65536, 70000],
                           rng.integers(1, 70000, size=300)])
    got = oracle.budgets(lens, ps, sched.bin_tokens, sched.min_pages, sched.frac_num,
                         sched.frac_den)
    want = [budget_fraction_reference(int(L), ps, sched.bin_tokens, sched.min_pages,
                                      sched.frac_num, sched.frac_den) for L in lens]
    np.testing.assert_array_equal(got, want)


def test_c2_budget_depends_only_on_pages():
    # ceil(0.10 * L / 16) == ceil(ceil(L / 16) / 10) for every L
    s = W.C2.schedule
    for L in range(1, 40000, 7):
        k = oracle.budget(L, 16, s.bin_tokens, s.min_pages, s.frac_num, s.frac_den)
        assert k == min(max(64, math.ceil(L / 160)), -(-L // 16))


def _golden_rows(kind):
    rows = []
    with open(os.path.join(GOLDEN, "budget_units.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            parts = line.split()
            if parts[0] == kind:
                nums = []
                for x in parts[1:]:
                    if not x.isdigit():
                        break
                    nums.append(int(x))
                rows.append(nums)
    assert rows, kind
    return rows


def test_golden_budget_units_from_paper():
    for ps, pages, tokens, ctx in _golden_rows("fixed"):
        k = oracle.budget(ctx, ps, 2048, [pages], [0], 1)
        assert k == pages and k * ps == tokens


def test_golden_two_k_bins_from_paper():
    for bin_tokens, length, bins in _golden_rows("bins"):
        # a table whose budget is bin index + 1 exposes the bin of a length
        n_bins = bins + 5
        k = oracle.budget(length, 16, bin_tokens, list(range(1, n_bins + 1)), [0] * n_bins, 1)
        assert k == bins


def test_golden_dense_while_context_fits_budget():
    for ps, pages, ctx, kept in _golden_rows("dense"):
        assert oracle.budget(ctx, ps, 2048, [pages], [0], 1) == kept


# ----------------------------------------------------------------------------- top-k
def brute_topk(s, k):
    return sorted(sorted(range(len(s)), key=lambda i: (-s[i], i))[:k])


@pytest.mark.parametrize("n,k", [(1, 1), (5, 2), (64, 13), (300, 299), (300, 300), (257, 1)])
def test_topk_matches_brute_force(n, k):
    rng = np.random.default_rng(n * 1000 + k)
    s = rng.standard_normal(n).astype(np.float32)
    s[rng.integers(0, n, size=n // 3)] = s[0]          # many exact ties
    got = oracle.topk(s, k)
    assert list(got) == brute_topk([float(x) for x in s], k)
    sel = np.zeros(n, bool)
    sel[got] = True
    assert len(got) == k
    if k < n:
        assert s[sel].min() >= s[~sel].max()


def test_topk_ties_go_to_lower_index_and_signed_zeros_tie():
    assert list(oracle.topk(np.zeros(10, np.float32), 4)) == [0, 1, 2, 3]
    s = np.array([1.0, 2.0, 2.0, 0.5, 2.0], np.float32)
    assert list(oracle.topk(s, 2)) == [1, 2]
    z = np.array([-0.0, 0.0, -0.0, 0.0, -1.0], np.float32)
    assert list(oracle.topk(z, 3)) == [0, 1, 2]


def test_zero_query_selects_first_pages():
    d = host_inputs(lengths=(160, 90, 200), seed=9)
    d["q"][:] = 0
    meta = oracle.page_meta(d["k"], d["bt"], d["lens"])
    s32, _ = oracle.page_scores(d["q"], meta, d["bt"], d["lens"], 16)
    idx = oracle.select(d["lens"], np.array([4, 4, 4], np.int32), s32, 16, 6)
    for b in range(3):
        for h in range(2):
            assert list(idx[b, h]) == [0, 1, 2, 3, -1, -1]


def test_duplicated_pages_lower_index_wins():
    d = host_inputs(B=1, lengths=(160,), seed=10)
    # copy page 7's keys onto pages 2 and 9: identical metadata, identical scores
    for p in (2, 9):
        d["k"][d["bt"][0, p]] = d["k"][d["bt"][0, 7]]
    meta = oracle.page_meta(d["k"], d["bt"], d["lens"])
    s32, _ = oracle.page_scores(d["q"], meta, d["bt"], d["lens"], 16)
    for h in range(2):
        assert s32[0, h, 2] == s32[0, h, 7] == s32[0, h, 9]
        order = sorted(range(10), key=lambda i: (-s32[0, h, i], i))
        # the three copies are adjacent in the order, lowest index first; keep one
        idx = oracle.topk(s32[0, h, :10], order.index(2) + 1)
        assert 2 in idx and 7 not in idx and 9 not in idx


# ----------------------------------------------------------------------------- attention
def textbook_attention(qj, keys, values, scale):
    w = scipy.special.softmax(scale * (keys @ qj))
    return w @ values


def test_dense_attention_matches_textbook_softmax():
    d = host_inputs(Hq=6, Hkv=2, lengths=(37, 64, 90), seed=11)
    out = oracle.attention(d["q"], d["k"], d["v"], d["bt"], d["lens"], SCALE)
    for b in range(3):
        for j in range(6):
            keys, vals = tokens_of(d, b, j // 3)
            ref = textbook_attention(bits_to_f64(d["q"][b, j]), keys, vals, SCALE)
            np.testing.assert_allclose(out[b, j], ref, rtol=1e-11, atol=1e-12)


def test_sparse_attention_matches_textbook_on_selected_pages():
    d = host_inputs(Hq=4, Hkv=2, lengths=(100, 33, 129), seed=12)
    k_of = np.array([3, 2, 4], np.int32)
    rng = np.random.default_rng(0)
    idx = np.full((3, 2, 5), -1, np.int32)
    for b in range(3):
        n = (int(d["lens"][b]) + 15) // 16
        for h in range(2):
            idx[b, h, :k_of[b]] = np.sort(rng.choice(n, size=k_of[b], replace=False))
    out = oracle.attention(d["q"], d["k"], d["v"], d["bt"], d["lens"], SCALE, k_of, idx)
    for b in range(3):
        for j in range(4):
            keys, vals = tokens_of(d, b, j // 2, idx[b, j // 2, :k_of[b]])
            ref = textbook_attention(bits_to_f64(d["q"][b, j]), keys, vals, SCALE)
            np.testing.assert_allclose(out[b, j], ref, rtol=1e-11, atol=1e-12)


def test_softmax_weights_sum_to_one_and_constant_values():
    d = host_inputs(lengths=(333, 1, 64), seed=13)
    keys, _ = tokens_of(d, 0, 1)
    kb = f32_to_bf16_bits(keys.astype(np.float32))
    assert abs(oracle.weight_sum(d["q"][0, 2], kb, SCALE) - 1.0) <= 1e-12
    ones = np.full_like(d["v"], 0x3F80)  # bf16 1.0
    out = oracle.attention(d["q"], d["k"], ones, d["bt"], d["lens"], SCALE)
    np.testing.assert_allclose(out, 1.0, rtol=0, atol=1e-12)


def test_single_token_returns_its_value_exactly():
    d = host_inputs(lengths=(1, 1, 1), seed=14)
    out = oracle.attention(d["q"], d["k"], d["v"], d["bt"], d["lens"], SCALE)
    for b in range(3):
        for j in range(4):
            np.testing.assert_array_equal(out[b, j], bits_to_f64(d["v"][d["bt"][b, 0], j // 2, 0]))


def test_identical_keys_give_mean_of_values():
    d = host_inputs(lengths=(45, 16, 70), seed=15)
    d["k"][:] = d["k"][0, 0, 0]          # every key equal
    out = oracle.attention(d["q"], d["k"], d["v"], d["bt"], d["lens"], SCALE)
    for b in range(3):
        for j in range(4):
            _, vals = tokens_of(d, b, j // 2)
            np.testing.assert_allclose(out[b, j], vals.mean(axis=0), rtol=1e-12, atol=1e-13)


def test_full_budget_sparse_equals_dense_bitwise():
    d = host_inputs(lengths=(100, 16, 250), seed=16)
    n = np.array([(int(L) + 15) // 16 for L in d["lens"]], np.int32)
    kmax = int(n.max())
    idx = np.full((3, 2, kmax), -1, np.int32)
    for b in range(3):
        idx[b, :, :n[b]] = np.arange(n[b])
    dense = oracle.attention(d["q"], d["k"], d["v"], d["bt"], d["lens"], SCALE)
    sparse = oracle.attention(d["q"], d["k"], d["v"], d["bt"], d["lens"], SCALE, n, idx)
    np.testing.assert_array_equal(dense, sparse)
    # and the whole step with a budget at least the page count keeps every page
    meta = oracle.page_meta(d["k"], d["bt"], d["lens"])
    s32, _ = oracle.page_scores(d["q"], meta, d["bt"], d["lens"], 16)
    np.testing.assert_array_equal(oracle.select(d["lens"], n, s32, 16, kmax), idx)


def test_block_table_permutation_and_index_order_invariance():
    d = host_inputs(lengths=(100, 60, 130), seed=17)
    base = oracle.attention(d["q"], d["k"], d["v"], d["bt"], d["lens"], SCALE)
    # move every physical page to a new slot and rewrite the block table
    P = d["k"].shape[0]
    perm = np.random.default_rng(1).permutation(P)
    inv = np.argsort(perm)
    k2, v2 = d["k"][perm], d["v"][perm]
    bt2 = inv[d["bt"]].astype(np.int32)
    moved = oracle.attention(d["q"], k2, v2, bt2, d["lens"], SCALE)
    np.testing.assert_array_equal(base, moved)
    k_of = np.array([5, 3, 6], np.int32)
    idx = np.full((3, 2, 6), -1, np.int32)
    for b in range(3):
        idx[b, :, :k_of[b]] = np.arange(k_of[b])
    fwd = oracle.attention(d["q"], d["k"], d["v"], d["bt"], d["lens"], SCALE, k_of, idx)
    rev = idx.copy()
    for b in range(3):
        rev[b, :, :k_of[b]] = idx[b, :, :k_of[b]][:, ::-1]
    bwd = oracle.attention(d["q"], d["k"], d["v"], d["bt"], d["lens"], SCALE, k_of, rev)
    np.testing.assert_allclose(fwd, bwd, rtol=1e-12, atol=1e-14)


def test_empty_sequence_gives_zero_row():
    d = host_inputs(lengths=(0, 20, 0), seed=18)
    out = oracle.attention(d["q"], d["k"], d["v"], d["bt"], d["lens"], SCALE)
    assert not out[0].any() and not out[2].any() and out[1].any()
    assert list(oracle.budgets(d["lens"], 16, 2048, [4], [0], 1)) == [0, 2, 0]


def test_whole_step_on_planted_hot_pages_keeps_them():
    w = W.small(B=2, Hq=4, Hkv=2, ps=16, lengths=(640, 900), seed=19, hot_pages=4,
                schedule=W.fixed_budget(8))
    inp = W.generate(w, "cpu", lengths=[640, 900])
    r = oracle.sparse_step(W.bf16_bits(inp.q), W.bf16_bits(inp.k_cache), W.bf16_bits(inp.v_cache),
                           inp.block_table.numpy(), inp.seq_lens.numpy(),
                           (2048, [8], [0], 1), 8, SCALE)
    for b in range(2):
        for h in range(2):
            assert set(inp.hot_host[b][h]) <= set(r["idx"][b, h].tolist())


def test_scores_without_the_fp64_copy_are_the_same_fp32_scores():
    # page_scores(fp64=False) skips only the adjudication copy: identical fp32 bits
    w = W.small(B=3, Hq=8, Hkv=2, ps=16, lengths=(700, 33, 2100), seed=71)
    inp = W.generate(w, "cpu", lengths=[700, 33, 2100])
    q = W.bf16_bits(inp.q)
    kc = W.bf16_bits(inp.k_cache)
    bt, lens = inp.block_table.numpy(), inp.seq_lens.numpy()
    meta = oracle.page_meta(kc, bt, lens)
    s32, s64 = oracle.page_scores(q, meta, bt, lens, 16)
    t32, t64 = oracle.page_scores(q, meta, bt, lens, 16, fp64=False)
    assert t64 is None and s64 is not None
    np.testing.assert_array_equal(s32.view(np.uint32), t32.view(np.uint32))
    sums = oracle.page_key_sums(kc, bt, lens)
    m32, _ = oracle.page_scores_mean(q, sums, bt, lens, 16)
    n32, n64 = oracle.page_scores_mean(q, sums, bt, lens, 16, fp64=False)
    assert n64 is None
    np.testing.assert_array_equal(m32.view(np.uint32), n32.view(np.uint32))
