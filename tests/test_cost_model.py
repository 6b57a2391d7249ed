"""The cost-model calculator (Sec. 3.3 Eq. dense-cost / Eq. sparse-cost, Appendix F) against
the properties the paper states for it: dense attention while the context fits the budget,
O(K L_out) growth past it, the units of I, and the page-size dependence of scoring."""
import math

import pytest

from paper_2606_08446_amd import cost_model as C
from paper_2606_08446_amd import workloads as W

X = C.Rollout(params=1.7e9, samples=8, l_in=1024, l_out=36864, d=1024, r=2)


def test_intensity_of_mi355x():
    # 2.5 PFLOP/s over 8 TB/s of bf16 elements (2 bytes each)
    assert C.intensity_mi355x() == 625.0
    assert C.intensity_mi355x(4.0e12) == 1250.0


@pytest.mark.parametrize("budget", [X.l_in + X.l_out, X.l_in + X.l_out + 1, 10 ** 9])
def test_appendix_f_budget_covering_the_context_is_dense(budget):
    assert C.dense_len(X.l_in, X.l_out, budget) == X.l_out
    assert C.budget_h(X.l_in, X.l_out, budget) == (2 * X.l_in + X.l_out) * X.l_out
    assert C.appendix_f_costs(X, 4, budget, 625.0) == C.appendix_f_costs(X, 4, None, 625.0)


def test_appendix_f_budget_below_the_prompt_has_no_dense_phase():
    for K in (1, 512, X.l_in):
        assert C.dense_len(X.l_in, X.l_out, K) == 0
        assert C.budget_h(X.l_in, X.l_out, K) == 2 * K * X.l_out


def test_appendix_f_grows_linearly_in_the_budget_after_the_dense_phase():
    K = 4096
    ld = K - X.l_in
    for lo in (ld, ld + 1, ld + 1000, 50000):
        assert C.budget_h(X.l_in, lo + 777, K) - C.budget_h(X.l_in, lo, K) == 2 * K * 777
    # continuity where the two branches meet
    assert C.budget_h(X.l_in, ld, K) == (2 * X.l_in + ld) * ld


def test_sparse_cost_scoring_shrinks_with_page_size():
    I = 625.0
    small = C.sparse_cost(X, I, 4096, 16)
    big = C.sparse_cost(X, I, 4096, 128)
    assert big["attn_mem"] == small["attn_mem"] and big["attn_comp"] == small["attn_comp"]
    assert math.isclose(small["score_mem"], 8 * big["score_mem"], rel_tol=1e-12)
    # the printed prompt term of the scoring memory lacks the page-size divisor
    printed = C.sparse_cost(X, I, 4096, 16, printed_prompt_term=True)
    assert math.isclose(printed["score_mem"] - small["score_mem"],
                        2 * X.l_in * X.d * X.l_out * (1 - 1 / 16), rel_tol=1e-12)
    # two landmark vectors per page (min and max) double the scoring terms
    two = C.sparse_cost(X, I, 4096, 16, landmark_vectors=2)
    assert math.isclose(two["score_mem"], 2 * small["score_mem"], rel_tol=1e-12)


def test_sparse_beats_dense_at_long_generations_and_not_at_full_budget():
    I = C.intensity_mi355x()
    assert C.sparse_cost(X, I, 4096, 16)["total"] < C.dense_cost(X, I)["total"]
    # past the quadratic regime the dense cost grows faster
    long_x = C.Rollout(1.7e9, 8, 1024, 2 * 36864, 1024, 2)
    ratio_short = C.dense_cost(X, I)["total"] / C.sparse_cost(X, I, 4096, 16)["total"]
    ratio_long = C.dense_cost(long_x, I)["total"] / C.sparse_cost(long_x, I, 4096, 16)["total"]
    assert ratio_long > ratio_short


def test_decode_step_elements_match_the_bench_workloads():
    # per layer and step: dense reads every K/V element, sparse its budget plus 2 landmarks per page
    w = W.C2
    lens = [8192, 20000, 32768]
    budgets = [max(64, math.ceil(math.ceil(L / 16) / 10)) * 16 for L in lens]
    dense, sparse = C.decode_step_elements(lens, budgets, 16, 1024)
    assert dense == 2 * sum(lens) * 1024
    assert sparse == sum(2 * k * 1024 + 2 * math.ceil(L / 16) * 1024 for L, k in zip(lens, budgets))
    assert w.page_size == 16
    # a budget at or above the length is read densely, without landmarks
    assert C.decode_step_elements([100], [100], 16, 8) == (1600, 1600)


def test_decode_step_elements_do_not_overflow_on_numpy_inputs():
    import numpy as np
    lens = np.full(256, 40960, np.int32)
    budgets = np.full(256, 320 * 32, np.int32)
    dense, sparse = C.decode_step_elements(lens, budgets, 32, 1024)
    assert dense == 2 * 40960 * 1024 * 256 and sparse > 0 and dense / sparse > 1



# ---------------------------------------------------------------- rollouts under a schedule
R = C.Rollout(params=1.7e9, samples=4, l_in=700, l_out=9000, d=1024, r=2)


def test_rollout_with_a_constant_table_is_appendix_f_summed_per_step():
    # a fixed budget of P pages of ps tokens: attention elements per sequence per D are
    # Appendix F's H(L_in, L_out, K) less its continuous dense phase's extra L_dense
    # (sum over t < L_dense of 2 (L_in + t) = (2 L_in + L_dense) L_dense - L_dense)
    for P, ps in ((64, 16), (200, 32), (30, 16), (1000, 16)):
        K = P * ps
        r = C.rollout_costs(R, 3, (2048, (P,), (0,), 1), ps, 625.0)
        ld = C.dense_len(R.l_in, R.l_out, K)
        assert r["attn_elems"] == 3 * R.samples * R.d * (C.budget_h(R.l_in, R.l_out, K) - ld)
        # steps that read their whole context: L_t <= K (at L_t = K the budget covers every
        # page, so no scoring runs; Appendix F's L_dense counts L_t < K, same attention)
        assert r["dense_steps"] == min(R.l_out, max(0, K - R.l_in + 1))


def test_rollout_whose_budget_covers_the_context_is_dense():
    whole = (2048, (0,), (1,), 1)                 # ceil(n * 1 / 1) = n pages
    d = C.rollout_costs(R, 2, None, 16, 625.0)
    s = C.rollout_costs(R, 2, whole, 16, 625.0)
    assert s == d and s["score_elems"] == 0 and s["dense_steps"] == R.l_out
    assert C.rollout_speedup(R, 2, whole, 16, 625.0)["total"] == 1.0
    # the dense rollout: sum over t of 2 (L_in + t) = (2 L_in + L_out) L_out - L_out
    assert d["attn_elems"] == 2 * R.samples * R.d * \
        ((2 * R.l_in + R.l_out) * R.l_out - R.l_out)


def test_rollout_half_budget_against_brute_force():
    # one-token pages, half the pages: K(L) = ceil(L / 2); scoring reads 2 landmark vectors
    # per page (= per token) on every step whose budget is below its context
    sch = (2048, (0,), (1,), 2)
    r = C.rollout_costs(R, 1, sch, 1, 625.0)
    attn = score = 0
    for t in range(R.l_out):
        L = R.l_in + t
        k = max(1, -(-L // 2))
        attn += 2 * min(L, k)
        if k < L:
            score += 2 * L
    assert r["attn_elems"] == R.samples * R.d * attn
    assert r["score_elems"] == R.samples * R.d * score


def test_rollout_with_a_dense_first_bin():
    # dense through the first 2048-token bin, 10 % of the pages after it
    sch = (2048, (0, 0), (10, 1), 10)
    r = C.rollout_costs(R, 1, sch, 16, 625.0)
    assert r["dense_steps"] == sum(1 for t in range(R.l_out) if R.l_in + t <= 2048)
    sp = C.rollout_speedup(R, 1, sch, 16, 625.0)
    assert 1.0 < sp["attention_memory"] < 10.0
    # a larger table never costs less
    more = C.rollout_costs(R, 1, (2048, (0, 0), (10, 2), 10), 16, 625.0)
    assert more["attn_elems"] >= r["attn_elems"]
