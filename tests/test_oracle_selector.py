"""Pins of the selector-variant oracle: the mean-key landmark (key sums, scores) and top-k
with forced sink/local pages, against numpy's sequential sums, a brute-force fp64 mean, the
order of the two landmarks (a mean never exceeds the min/max bound), and brute-force
sorting."""
import math

import numpy as np
import pytest

import oracle
from paper_2606_08446_amd import workloads as W


def bits_f32(a):
    return (np.asarray(a, np.uint16).astype(np.uint32) << 16).view(np.float32)


def inputs(B=3, Hq=6, Hkv=2, ps=16, lengths=(37, 64, 90), seed=0):
    w = W.small(B=B, Hq=Hq, Hkv=Hkv, ps=ps, lengths=lengths, seed=seed)
    inp = W.generate(w, "cpu", lengths=list(lengths))
    return dict(q=W.bf16_bits(inp.q), k=W.bf16_bits(inp.k_cache), v=W.bf16_bits(inp.v_cache),
                bt=inp.block_table.numpy().copy(), lens=inp.seq_lens.numpy().copy(), ps=ps)


def test_key_sums_are_sequential_fp32_sums():
    d = inputs(seed=1)
    sums = oracle.page_key_sums(d["k"], d["bt"], d["lens"])
    for b, L in enumerate(d["lens"]):
        for p in range((L + 15) // 16):
            phys = d["bt"][b, p]
            valid = min(16, L - p * 16)
            rows = bits_f32(d["k"][phys, :, :valid])            # [Hkv][valid][D]
            seq = np.cumsum(rows, axis=1, dtype=np.float32)[:, -1]  # token by token in fp32
            np.testing.assert_array_equal(sums[phys], seq)


def test_incremental_sums_equal_rebuild():
    d = inputs(seed=2)
    full = d["lens"]
    short = np.maximum(full - 9, 0).astype(np.int32)
    part = oracle.page_key_sums(d["k"], d["bt"], short)
    upd = oracle.page_key_sums(d["k"], d["bt"], full, first_pos=short, sums=part)
    ref = oracle.page_key_sums(d["k"], d["bt"], full)
    for b, L in enumerate(full):
        pages = d["bt"][b, :(L + 15) // 16]
        np.testing.assert_array_equal(upd[pages], ref[pages])


def test_mean_scores_match_brute_force_and_stay_below_the_minmax_bound():
    d = inputs(seed=3)
    sums = oracle.page_key_sums(d["k"], d["bt"], d["lens"])
    s32, s64 = oracle.page_scores_mean(d["q"], sums, d["bt"], d["lens"], 16)
    meta = oracle.page_meta(d["k"], d["bt"], d["lens"])
    _, mm64 = oracle.page_scores(d["q"], meta, d["bt"], d["lens"], 16)
    G = 3
    for b, L in enumerate(d["lens"]):
        for h in range(2):
            for p in range((L + 15) // 16):
                phys = d["bt"][b, p]
                valid = min(16, L - p * 16)
                keys = bits_f32(d["k"][phys, h, :valid]).astype(np.float64)
                mean = sums[phys, h].astype(np.float64) / valid
                qs = bits_f32(d["q"][b, h * G:(h + 1) * G]).astype(np.float64)
                ref = math.fsum(float(x) for x in (qs @ mean))
                assert abs(s64[b, h, p] - ref) <= 1e-9 * max(1.0, abs(ref))
                assert abs(s32[b, h, p] - ref) <= 1e-4 * max(1.0, abs(ref))
                # the mean of q.k over the page's tokens never exceeds the min/max bound
                true_mean = float(np.mean(qs.sum(0) @ keys.T))
                assert true_mean <= mm64[b, h, p] + 1e-9
                assert abs(s64[b, h, p] - true_mean) <= 1e-4 * max(1.0, abs(true_mean))


def test_single_token_page_mean_score_is_the_dot_product():
    d = inputs(lengths=(17, 33, 1), seed=4)
    sums = oracle.page_key_sums(d["k"], d["bt"], d["lens"])
    _, s64 = oracle.page_scores_mean(d["q"], sums, d["bt"], d["lens"], 16)
    for b, L in enumerate(d["lens"]):
        p = (L - 1) // 16
        key = bits_f32(d["k"][d["bt"][b, p], 0, 0]).astype(np.float64)
        qs = bits_f32(d["q"][b, 0:3]).astype(np.float64)
        assert abs(s64[b, 0, p] - float((qs @ key).sum())) <= 1e-9


def brute_forced(s_row, n, k, sink, local):
    order = sorted(range(n), key=lambda p: (0, p, 0.0) if (p < sink or p >= n - local)
                   else (1, 0, -float(s_row[p]), p))
    return sorted(order[:k])


@pytest.mark.parametrize("sink,local", [(0, 0), (1, 0), (0, 2), (1, 2), (4, 4)])
def test_forced_selection_matches_brute_force(sink, local):
    rng = np.random.default_rng(5)
    B, Hkv, M = 4, 2, 40
    lens = np.array([16 * 40, 16 * 7 + 3, 16 * 3, 1], np.int32)
    scores = rng.standard_normal((B, Hkv, M)).astype(np.float32)
    scores[0, 0, 5:12] = 0.5                     # exact ties
    k = np.array([9, 4, 2, 1], np.int32)
    got = oracle.select_forced(lens, k, scores, 16, 12, sink, local)
    for b in range(B):
        n = (int(lens[b]) + 15) // 16
        kk = min(int(k[b]), n)
        for h in range(Hkv):
            want = brute_forced(scores[b, h], n, kk, sink, local)
            assert got[b, h, :kk].tolist() == want
            assert (got[b, h, kk:] == -1).all()
            forced = [p for p in range(n) if p < sink or p >= n - local]
            if kk >= len(forced):
                assert set(forced) <= set(want)
    if sink == local == 0:   # no forced pages: plain top-k
        np.testing.assert_array_equal(got, oracle.select(lens, k, scores, 16, 12))


def test_mean_append_token_by_token_equals_one_pass_sums():
    d = inputs(B=2, lengths=(40, 17), seed=6)
    full = d["lens"].copy()
    kc = np.zeros_like(d["k"])
    vc = np.zeros_like(d["v"])
    sums = np.zeros((kc.shape[0], 2, 128), np.float32)
    for t in range(int(full.max())):
        grow = full > t
        lens = np.where(grow, t + 1, 0).astype(np.int32)
        kn = np.zeros((2, 2, 128), np.uint16)
        vn = np.zeros((2, 2, 128), np.uint16)
        for b in range(2):
            if grow[b]:
                phys = d["bt"][b, t // 16]
                kn[b], vn[b] = d["k"][phys, :, t % 16], d["v"][phys, :, t % 16]
        kc, vc, sums = oracle.append_kv(kn, vn, kc, vc, d["bt"], lens, sums, landmark="mean")
    ref = oracle.page_key_sums(d["k"], d["bt"], full)
    for b, L in enumerate(full):
        pages = d["bt"][b, :(L + 15) // 16]
        np.testing.assert_array_equal(sums[pages], ref[pages])
