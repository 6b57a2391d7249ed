"""Rollout cost model of Sparrow (arXiv 2606.08446): Eq. dense-cost and Eq. sparse-cost
(Sec. 3.3, Control Study 2) and the budgeted form of Appendix F, in equivalent FLOPs, for a
fixed budget or summed over a rollout whose budget follows a schedule table (Sec. 3.2).

Both forms add compute to memory traffic weighted by an intensity I (FLOPs that one
element of memory traffic is worth): I = peak FLOP/s x element bytes / memory bandwidth.
Memory terms count elements (one K or V channel of one token is one element), like the
paper's, so I converts them.  ``intensity_mi355x`` gives I for the MI355X's published peaks
(dense bf16 2.5 PFLOP/s, 8 TB/s) or for a measured bandwidth.

Readings (where the printed formulas are silent or inconsistent):
* The scoring memory term of Eq. sparse-cost has no page-size divisor on its prompt part;
  the landmark metadata is per page, so by default it is divided by the page size like the
  generated part (``printed_prompt_term=True`` keeps the printed form).
* The paper counts one D-vector of landmark per page; the min/max landmark stores two,
  ``landmark_vectors=2``.
* In Appendix F, L_dense = min(L_out, K - L_in) is clamped at 0: a budget below the prompt
  length leaves no dense phase.
* Sec. 3.3 reads the prompt's KV once per step for all N samples (2 L_in L_out D), Appendix
  F once per sample (B N 2 L_in L_out D); both are implemented as printed.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import math

MI355X_BF16_FLOPS = 2.5e15      # dense bf16 MFMA peak
MI355X_HBM_BYTES_PER_S = 8.0e12


def intensity_mi355x(bandwidth_bytes_per_s: float = MI355X_HBM_BYTES_PER_S,
                     peak_flops: float = MI355X_BF16_FLOPS, element_bytes: int = 2) -> float:
    """I: FLOPs equivalent to moving one element (bf16 by default)."""
    return peak_flops * element_bytes / bandwidth_bytes_per_s


@dataclasses.dataclass(frozen=True)
class Rollout:
    """One rollout setting of Sec. 3.3: P parameters, N samples, prompt / generation lengths
    in tokens, D the width of K (and of V) per token, r the GQA ratio (> 1)."""
    params: float
    samples: int
    l_in: int
    l_out: int
    d: int
    r: float


# Qwen3 attention widths per layer: D = kv_heads x head_dim, r = q_heads / kv_heads.
QWEN3 = {"1.7b": dict(params=1.7e9, d=8 * 128, r=2), "4b": dict(params=4.0e9, d=8 * 128, r=4),
         "8b": dict(params=8.2e9, d=8 * 128, r=4), "14b": dict(params=14.8e9, d=8 * 128, r=5)}


def dense_cost(x: Rollout, I: float) -> dict:
    """Eq. dense-cost: C_comp + I * C_mem."""
    comp = 2 * x.params * x.samples * x.l_out + \
        x.r * (2 * x.l_in + x.l_out) * x.l_out * x.samples * x.d
    mem = 2 * x.l_in * x.l_out * x.d + x.samples * x.l_out ** 2 * x.d
    return {"comp": comp, "mem": mem, "total": comp + I * mem}


def sparse_cost(x: Rollout, I: float, budget: int, page_size: int, landmark_vectors: int = 1,
                printed_prompt_term: bool = False) -> dict:
    """Eq. sparse-cost: the attention over a budget of ``budget`` tokens plus the landmark
    scoring (``landmark_vectors`` D-vectors per page)."""
    N, D, r, Lo, Li = x.samples, x.d, x.r, x.l_out, x.l_in
    att_comp = 2 * N * x.params * Lo + 2 * r * N * D * budget * Lo
    att_mem = 2 * N * D * budget * Lo
    lv = landmark_vectors
    prompt_pages = Li if printed_prompt_term else Li / page_size
    sc_comp = lv * (2 * N * prompt_pages * D * Lo + r * N * D * Lo ** 2 / (2 * page_size))
    sc_mem = lv * (2 * prompt_pages * D * Lo + N * D * Lo ** 2 / (2 * page_size))
    return {"attn_comp": att_comp, "attn_mem": att_mem, "score_comp": sc_comp,
            "score_mem": sc_mem,
            "total": att_comp + I * att_mem + sc_comp + I * sc_mem}


def dense_len(l_in: int, l_out: int, budget: int) -> int:
    """Appendix F: tokens generated while the whole context fits the budget."""
    return max(0, min(l_out, budget - l_in))


def budget_h(l_in: int, l_out: int, budget: int) -> int:
    """Appendix F: H(L_in, L_out, K) = (2 L_in + L_dense) L_dense + 2 K (L_out - L_dense)_+."""
    ld = dense_len(l_in, l_out, budget)
    return (2 * l_in + ld) * ld + 2 * budget * max(0, l_out - ld)


def appendix_f_costs(x: Rollout, batch: int, budget: int | None, I: float) -> dict:
    """Appendix F per-layer costs; budget None = dense attention."""
    B, N, D, Lo, Li = batch, x.samples, x.d, x.l_out, x.l_in
    attn = (2 * Li + Lo) * Lo if budget is None else budget_h(Li, Lo, budget)
    comp = 2 * x.params * B * N * Lo + x.r * B * N * D * attn
    mem = 2 * x.params * Lo + B * N * D * attn
    return {"comp": comp, "mem": mem, "attn_elems": B * N * D * attn, "total": comp + I * mem}


def decode_step_elements(lengths, budgets_tokens, page_size, d, landmark_vectors=2):
    """Per decode step of one layer: (dense, sparse) KV elements read for sequences of the given
    lengths, the sparse side reading its budget of K and V plus the page landmarks of every
    sequence whose budget is below its length (dense while it fits, Appendix F)."""
    dense = sparse = 0
    for L, k in zip(lengths, budgets_tokens):
        L, k = int(L), int(k)   # Python integers: no fixed-width overflow
        dense += 2 * L * d
        if k >= L:
            sparse += 2 * L * d
        else:
            sparse += 2 * k * d + landmark_vectors * math.ceil(L / page_size) * d
    return dense, sparse


def schedule_budget_tokens(lengths, schedule, page_size):
    """Budget in tokens of sequences of the given lengths under a schedule table (the form
    the kernels consume: ``(bin_tokens, min_pages, frac_num, frac_den)``): the library's own
    budget in pages (sparrow_budget_bound, host code) times the page size, capped at the
    length (a budget covering every page reads every token)."""
    import numpy as np

    from . import sparrow
    bin_tokens, min_pages, frac_num, frac_den = schedule
    lens = np.asarray(lengths, dtype=np.int64)
    pages, _ = sparrow.budgets(lens, page_size, bin_tokens, min_pages, frac_num, frac_den)
    return np.minimum(pages.astype(np.int64) * page_size, lens)


def rollout_costs(x: Rollout, batch: int, schedule, page_size: int, I: float,
                  landmark_vectors: int = 2) -> dict:
    """Per-layer cost of a whole rollout with a length-dependent budget (Appendix F's
    per-step attention cost summed over the generation, with K taken from the schedule at
    each step's context length; the scoring term of Eq. sparse-cost per step).

    Step t (t = 0 .. L_out - 1) attends over a context of L_t = L_in + t tokens: dense reads
    2 L_t D elements of K and V; sparse reads 2 min(L_t, K(L_t)) D, plus ``landmark_vectors``
    D-vectors per page of landmarks whenever its budget is below L_t.  Compute: 2 P per
    generated token plus r D per attended element (Appendix F's C_comp).  ``schedule`` None
    gives the dense rollout.  Returns elements and costs for B N sequences."""
    import numpy as np
    B, N, D, Lo, Li = batch, x.samples, x.d, x.l_out, x.l_in
    L = Li + np.arange(Lo, dtype=np.int64)
    if schedule is None:
        k = L
    else:
        k = schedule_budget_tokens(L, schedule, page_size)
    attn = int((2 * k).sum())
    sparse_steps = k < L
    score = int((landmark_vectors * -(-L[sparse_steps] // page_size)).sum())
    comp = 2 * x.params * B * N * Lo + x.r * B * N * D * attn
    mem = 2 * x.params * Lo + B * N * D * (attn + score)
    return {"attn_elems": B * N * D * attn, "score_elems": B * N * D * score,
            "dense_steps": int(Lo - sparse_steps.sum()), "comp": comp, "mem": mem,
            "total": comp + I * mem}


def rollout_speedup(x: Rollout, batch: int, schedule, page_size: int, I: float,
                    landmark_vectors: int = 2) -> dict:
    """Predicted dense / sparse rollout cost ratios of a schedule: whole model (Appendix F's
    total with the weights read once per step) and attention memory only (the part the
    decode kernels move)."""
    d = rollout_costs(x, batch, None, page_size, I, landmark_vectors)
    s = rollout_costs(x, batch, schedule, page_size, I, landmark_vectors)
    return {"total": d["total"] / s["total"],
            "attention_memory": d["attn_elems"] / (s["attn_elems"] + s["score_elems"]),
            "dense": d, "sparse": s}


def main():
    ap = argparse.ArgumentParser(description="Sparrow rollout cost model (eFLOPs)")
    ap.add_argument("--model", default="1.7b", choices=sorted(QWEN3))
    ap.add_argument("--samples", type=int, default=8)
    ap.add_argument("--l-in", type=int, default=1024)
    ap.add_argument("--l-out", type=int, default=36864)
    ap.add_argument("--budget", type=int, default=4096, help="KV budget in tokens")
    ap.add_argument("--page-size", type=int, default=16)
    ap.add_argument("--bandwidth", type=float, default=MI355X_HBM_BYTES_PER_S,
                    help="bytes/s used for I (e.g. a measured copy bandwidth)")
    ap.add_argument("--landmark-vectors", type=int, default=1)
    ap.add_argument("--schedule", choices=("c1", "c2", "c3", "c4", "c5"),
                    help="also integrate the rollout with this workload's schedule table")
    a = ap.parse_args()
    m = QWEN3[a.model]
    x = Rollout(m["params"], a.samples, a.l_in, a.l_out, m["d"], m["r"])
    I = intensity_mi355x(a.bandwidth)
    d = dense_cost(x, I)
    s = sparse_cost(x, I, a.budget, a.page_size, a.landmark_vectors)
    fd = appendix_f_costs(x, 1, None, I)
    fs = appendix_f_costs(x, 1, a.budget, I)
    out = {"I": I, "dense": d, "sparse": s, "speedup": d["total"] / s["total"],
           "appendix_f": {"dense": fd, "sparse": fs, "speedup": fd["total"] / fs["total"]}}
    if a.schedule:
        from . import workloads as W
        w = W.CONFIGS[a.schedule] if a.schedule != "c4" else W.C4
        sch = w.schedule
        r = rollout_speedup(x, 1, (sch.bin_tokens, sch.min_pages, sch.frac_num, sch.frac_den),
                            a.page_size, I, a.landmark_vectors)
        out["rollout_with_schedule"] = {"schedule_of": w.name, "speedup": r["total"],
                                        "attention_memory_speedup": r["attention_memory"],
                                        "dense_steps": r["sparse"]["dense_steps"]}
    print(json.dumps(out))


if __name__ == "__main__":
    main()
