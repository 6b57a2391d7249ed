"""Seeded synthetic workloads for the sparse-decode step.

This module only builds inputs: paged bf16 K/V caches, queries, lengths,
block tables and the budget schedule tables.  It holds none of the method's
arithmetic (no metadata, scores, budgets, selection or attention), so both the
GPU library's tests and the CPU oracle may draw their inputs from it.

Structural randomness (lengths, page permutation, planted pages, outlier
channels) comes from ``numpy.random.default_rng(seed)`` and is identical on
every device.  Values (q, K, V) are standard normal, drawn in fp32 with
``torch`` on the target device and rounded to bf16 (round to nearest even).

Shapes follow the Qwen3 family the paper trains (head_dim 128; 16/8, 32/8 and
40/8 query/KV heads) and the page sizes of Sec. 3.2 and Appendix C.  The
paper's own workload (AIME prompts with long reasoning rollouts, Sec. 4.1) is
not available; lengths drawn uniformly over long-context ranges stand in for
it.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np
import torch

HEAD_DIM = 128


@dataclasses.dataclass(frozen=True)
class Schedule:
    """Budget schedule table over length bins (input data).

    Budget of a sequence of L tokens (n pages), bin = min((L-1)//bin_tokens, n_bins-1):
    clamp(max(min_pages[bin], ceil(n * frac_num[bin] / frac_den)), 1, n)."""
    bin_tokens: int
    min_pages: tuple
    frac_num: tuple
    frac_den: int

    @property
    def n_bins(self) -> int:
        return len(self.min_pages)


def fixed_budget(pages: int) -> Schedule:
    return Schedule(2048, (pages,), (0,), 1)


def fraction_budget(num: int, den: int, floor_pages: int = 0) -> Schedule:
    return Schedule(2048, (floor_pages,), (num,), den)


def rising_permille(bin_tokens: int, len_from: int, len_to: int, pm_from: int,
                    pm_to: int) -> Schedule:
    """Per-mille of pages rising linearly from ``pm_from`` at the bin of ``len_from``
    to ``pm_to`` at the bin of ``len_to`` (integer rounding, half up); flat outside."""
    b0 = (len_from - 1) // bin_tokens
    b1 = (len_to - 1) // bin_tokens
    n_bins = b1 + 1
    pm = []
    for b in range(n_bins):
        if b <= b0:
            pm.append(pm_from)
        else:
            num = (pm_to - pm_from) * (b - b0)
            den = b1 - b0
            pm.append(pm_from + (2 * num + den) // (2 * den))
    return Schedule(bin_tokens, tuple([0] * n_bins), tuple(pm), 1000)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    page_size: int
    len_lo: int
    len_hi: int
    seed: int
    schedule: Schedule
    sink_scale: float = 1.0        # keys of logical page 0 are multiplied by this
    hot_pages: int = 0             # planted pages per (sequence, KV head)
    hot_clusters: int = 0          # 0: scattered; c > 0: c runs of consecutive pages
    hot_shift: float = 6.0         # planted keys get += hot_shift * unit(sum of group queries)
    outlier_channels: int = 0      # key channels per KV head scaled by outlier_scale
    outlier_scale: float = 10.0
    extra_pages: int = 1           # allocated but unused pages per sequence (room to append)
    head_dim: int = HEAD_DIM
    description: str = ""

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads


# The five workloads.  The first is the small single-sequence case; the fourth, the
# Qwen3-8B-shaped batch of 256 swept over five budgets, is the largest on one GPU.
C1 = Workload("c1_b1_l4096_fixed32", 1, 16, 8, 16, 4096, 4096, 11, fixed_budget(32),
              sink_scale=4.0,
              description="batch 1, 16/8 heads, 4096 tokens in 16-token pages, fixed 32-page "
                          "budget, sink page x4")
C2 = Workload("c2_qwen3_1p7b_b64", 64, 16, 8, 16, 8192, 32768, 12,
              fraction_budget(100, 1000, floor_pages=64), hot_pages=8,
              description="Qwen3-1.7B-shaped layer, batch 64, lengths U[8192, 32768], 16-token "
                          "pages, budget max(64, ceil(0.10 n)), 8 planted hot pages per head")
C3 = Workload("c3_qwen3_4b_b128", 128, 32, 8, 16, 4096, 32768, 13,
              rising_permille(2048, 4096, 32768, 50, 200), outlier_channels=4,
              description="Qwen3-4B-shaped layer, batch 128, lengths U[4096, 32768], budget "
                          "5% -> 20% of pages rising with length, 4 key channels x10")
C4_FRACTIONS = ((20, 1000), (50, 1000), (100, 1000), (250, 1000), (1000, 1000))
C4 = Workload("c4_qwen3_8b_b256", 256, 32, 8, 32, 16384, 40960, 14,
              fraction_budget(*C4_FRACTIONS[2]),
              description="Qwen3-8B-shaped layer, batch 256, lengths U[16384, 40960], 32-token "
                          "pages, budgets 2/5/10/25/100% of pages")
C5 = Workload("c5_qwen3_14b_b64", 64, 40, 8, 16, 32768, 65536, 15,
              rising_permille(2048, 32768, 65536, 30, 150), sink_scale=4.0, hot_pages=16,
              hot_clusters=2,
              description="Qwen3-14B-shaped layer, batch 64, lengths U[32768, 65536], budget "
                          "3% -> 15% rising with length, sink page, 2 clusters of 8 hot pages, "
                          "one appended token per step")
CONFIGS = {"c1": C1, "c2": C2, "c3": C3, "c4": C4, "c5": C5}


def table4(page_size: int, length: int, batch: int = 16) -> Workload:
    """The page-size study of Table 4: a Qwen3-1.7B-shaped layer (16/8 heads), ``batch``
    sequences of ``length`` past tokens, a fixed budget of 1024 tokens (1024 / page_size
    pages)."""
    return Workload(f"t4_ps{page_size}_l{length // 1024}k_b{batch}", batch, 16, 8, page_size,
                    length, length, 16, fixed_budget(1024 // page_size),
                    description=f"Table 4 page-size study: {page_size}-token pages x "
                                f"{1024 // page_size}, {length} past tokens, batch {batch}")


def c4_with_fraction(i: int) -> Workload:
    num, den = C4_FRACTIONS[i]
    return dataclasses.replace(C4, schedule=fraction_budget(num, den),
                               name=f"{C4.name}_{num / den * 100:g}pct")


@dataclasses.dataclass
class Inputs:
    """One generated workload.  Tensors live on ``device``."""
    workload: Workload
    seq_lens: torch.Tensor        # int32 [B]
    block_table: torch.Tensor     # int32 [B][max_pages]
    q: torch.Tensor               # bf16 [B][Hq][D]
    k_cache: torch.Tensor         # bf16 [P][Hkv][ps][D]
    v_cache: torch.Tensor         # bf16 [P][Hkv][ps][D]
    min_pages: torch.Tensor       # int32 [n_bins]
    frac_num: torch.Tensor        # int32 [n_bins]
    lens_host: np.ndarray         # int64 [B]
    pages_host: np.ndarray        # int64 [B] allocated pages per sequence
    hot_host: Optional[list] = None  # per (b, h): planted logical pages

    @property
    def max_pages(self) -> int:
        return int(self.block_table.shape[1])

    @property
    def num_phys_pages(self) -> int:
        return int(self.k_cache.shape[0])


def _randn_bf16(shape, gen, device, chunk_rows: int = 1 << 14) -> torch.Tensor:
    """Standard normal values, drawn in fp32 and rounded to bf16, in row chunks."""
    out = torch.empty(shape, dtype=torch.bfloat16, device=device)
    rows = shape[0]
    for r0 in range(0, rows, chunk_rows):
        r1 = min(rows, r0 + chunk_rows)
        sub = (r1 - r0,) + tuple(shape[1:])
        out[r0:r1] = torch.randn(sub, generator=gen, device=device,
                                 dtype=torch.float32).to(torch.bfloat16)
    return out


def _pick_hot(rng, n: int, count: int, clusters: int) -> List[int]:
    """Distinct logical pages in [1, n-2] (scattered, or ``clusters`` runs)."""
    lo, hi = 1, n - 2
    avail = hi - lo + 1
    if count <= 0 or avail < count:
        return []
    if clusters <= 0:
        return sorted(int(x) for x in rng.choice(np.arange(lo, hi + 1), size=count,
                                                  replace=False))
    run = count // clusters
    # non-overlapping runs: choose run starts among slots of width `run`
    slots = avail // run
    starts = sorted(int(s) for s in rng.choice(slots, size=clusters, replace=False))
    pages = []
    for s in starts:
        pages.extend(range(lo + s * run, lo + s * run + run))
    return pages


def generate(w: Workload, device="cpu", lengths=None, seed: Optional[int] = None) -> Inputs:
    """Build the inputs of workload ``w`` on ``device``.

    ``lengths`` overrides the drawn sequence lengths (any list of ints >= 0)."""
    seed = w.seed if seed is None else seed
    rng = np.random.default_rng(seed)
    B, Hq, Hkv, ps, D = w.batch, w.num_q_heads, w.num_kv_heads, w.page_size, w.head_dim
    G = Hq // Hkv
    if lengths is None:
        lens = rng.integers(w.len_lo, w.len_hi + 1, size=B).astype(np.int64)
    else:
        lens = np.asarray(lengths, dtype=np.int64)
        assert len(lens) == B
    n_pages = np.array([(int(L) + ps - 1) // ps for L in lens], dtype=np.int64)
    alloc = n_pages + w.extra_pages
    P = int(alloc.sum())
    max_pages = int(alloc.max()) if B > 0 else 1
    perm = rng.permutation(P).astype(np.int64)
    bt = np.zeros((B, max_pages), dtype=np.int32)  # unallocated slots point at page 0
    off = 0
    for b in range(B):
        bt[b, :alloc[b]] = perm[off:off + alloc[b]]
        off += int(alloc[b])

    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    q = _randn_bf16((B, Hq, D), gen, device)
    k_cache = _randn_bf16((P, Hkv, ps, D), gen, device)
    v_cache = _randn_bf16((P, Hkv, ps, D), gen, device)

    # Sink: keys of logical page 0 scaled.
    if w.sink_scale != 1.0 and B > 0:
        phys0 = torch.as_tensor(bt[n_pages > 0, 0].astype(np.int64), device=device)
        if phys0.numel():
            k_cache[phys0] = (k_cache[phys0].float() * w.sink_scale).to(torch.bfloat16)

    # Outlier key channels, per KV head (the same channels in every sequence).
    if w.outlier_channels > 0:
        for h in range(Hkv):
            ch = rng.choice(D, size=w.outlier_channels, replace=False)
            for c in sorted(int(x) for x in ch):
                k_cache[:, h, :, c] = (k_cache[:, h, :, c].float()
                                       * w.outlier_scale).to(torch.bfloat16)

    # Planted hot pages: keys shifted along the unit direction of the summed group queries.
    hot = None
    if w.hot_pages > 0:
        hot = []
        phys_list, head_list, dir_rows = [], [], []
        qg = q.float().view(B, Hkv, G, D).sum(dim=2)
        qg = qg / qg.norm(dim=-1, keepdim=True).clamp_min(1e-30)
        for b in range(B):
            row = []
            for h in range(Hkv):
                pages = _pick_hot(rng, int(n_pages[b]), w.hot_pages, w.hot_clusters)
                row.append(pages)
                for p in pages:
                    phys_list.append(int(bt[b, p]))
                    head_list.append(h)
                    dir_rows.append(b * Hkv + h)
            hot.append(row)
        if phys_list:
            pi = torch.as_tensor(phys_list, device=device)
            hi = torch.as_tensor(head_list, device=device)
            di = torch.as_tensor(dir_rows, device=device)
            shift = (w.hot_shift * qg.view(B * Hkv, D)[di]).unsqueeze(1)  # [N,1,D]
            k_cache[pi, hi] = (k_cache[pi, hi].float() + shift).to(torch.bfloat16)

    return Inputs(
        workload=w,
        seq_lens=torch.as_tensor(lens.astype(np.int32), device=device),
        block_table=torch.as_tensor(bt, device=device),
        q=q, k_cache=k_cache, v_cache=v_cache,
        min_pages=torch.as_tensor(np.array(w.schedule.min_pages, np.int32), device=device),
        frac_num=torch.as_tensor(np.array(w.schedule.frac_num, np.int32), device=device),
        lens_host=lens, pages_host=alloc, hot_host=hot)


def small(B=2, Hq=4, Hkv=2, ps=16, lengths=(40, 70), seed=0, schedule=None, **kw) -> Workload:
    """A small workload for parity tests (explicit lengths are passed to ``generate``)."""
    schedule = schedule or fraction_budget(1, 3)
    lo = min(lengths) if len(lengths) else 0
    hi = max(lengths) if len(lengths) else 0
    return Workload(f"small_b{B}_h{Hq}x{Hkv}_ps{ps}", B, Hq, Hkv, ps, lo, hi, seed, schedule,
                    **kw)


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor -> numpy uint16 bit patterns (on the host)."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def with_schedule(inp: Inputs, w: Workload) -> Inputs:
    """The same caches and queries under workload ``w``'s budget schedule."""
    dev = inp.q.device
    return dataclasses.replace(
        inp, workload=w,
        min_pages=torch.as_tensor(np.array(w.schedule.min_pages, np.int32), device=dev),
        frac_num=torch.as_tensor(np.array(w.schedule.frac_num, np.int32), device=dev))


# ----------------------------------------------------------------------------------------------
# Paired logit rows for the per-token acceptance rate (Sec. 3.1): for each generated token, the
# target (dense policy) and draft (sparse rollout) logits over the vocabulary, and its position.
# Random inputs only; the acceptance rate itself is computed elsewhere.
# ----------------------------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class LogitWorkload:
    """Synthetic logit rows: target = scale * N(0, 1) with one chosen token raised by a peak
    drawn from U(peak_lo, peak_hi) (confident next-token predictions); draft = target +
    sigma_t * N(0, 1), where sigma_t = noise * exp(noise_sigma * N(0, 1)) * (1 + growth * pos /
    max_pos) is log-normal per token (most tokens barely perturbed, a heavy tail) and grows with
    the position, which is uniform in [0, max_pos)."""
    name: str
    tokens: int
    vocab: int
    max_pos: int
    bin_tokens: int
    n_bins: int
    scale: float = 2.0
    peak_lo: float = 10.0
    peak_hi: float = 20.0
    noise: float = 0.01
    noise_sigma: float = 2.0
    growth: float = 2.0
    dtype: str = "f32"     # "f32" or "bf16"
    seed: int = 31


# Qwen3's vocabulary, 4096 generated tokens over a 40K-token generation in 2K-token bins.
A1 = LogitWorkload("a1_qwen3_vocab_t4096", 4096, 151936, 40960, 2048, 20)
A1_BF16 = dataclasses.replace(A1, name="a1_qwen3_vocab_t4096_bf16", dtype="bf16")
LOGIT_CONFIGS = {"a1": A1, "a1-bf16": A1_BF16}


@dataclasses.dataclass
class LogitInputs:
    workload: LogitWorkload
    target: torch.Tensor      # [T][V] float32 or bf16
    draft: torch.Tensor       # [T][V]
    positions: torch.Tensor   # int32 [T]
    sigma: np.ndarray         # float64 [T] perturbation scale of each token


def generate_logits(lw: LogitWorkload, device="cpu", chunk_rows: int = 256) -> LogitInputs:
    rng = np.random.default_rng(lw.seed)
    T, V = lw.tokens, lw.vocab
    pos = rng.integers(0, lw.max_pos, size=T).astype(np.int32)
    peak_id = rng.integers(0, V, size=T)
    peak = rng.uniform(lw.peak_lo, lw.peak_hi, size=T)
    sigma = lw.noise * np.exp(lw.noise_sigma * rng.standard_normal(T)) * \
        (1.0 + lw.growth * pos / lw.max_pos)
    dt = torch.float32 if lw.dtype == "f32" else torch.bfloat16
    target = torch.empty((T, V), dtype=dt, device=device)
    draft = torch.empty((T, V), dtype=dt, device=device)
    gen = torch.Generator(device=device)
    gen.manual_seed(lw.seed)
    for r0 in range(0, T, chunk_rows):
        r1 = min(T, r0 + chunk_rows)
        z = torch.randn((r1 - r0, V), generator=gen, device=device) * lw.scale
        rows = torch.arange(r1 - r0, device=device)
        z[rows, torch.as_tensor(peak_id[r0:r1], device=device)] += \
            torch.as_tensor(peak[r0:r1], dtype=torch.float32, device=device)
        e = torch.randn((r1 - r0, V), generator=gen, device=device)
        s = torch.as_tensor(sigma[r0:r1], dtype=torch.float32, device=device)[:, None]
        target[r0:r1] = z.to(dt)
        draft[r0:r1] = (z + s * e).to(dt)
    return LogitInputs(lw, target, draft, torch.as_tensor(pos, device=device), sigma)


def small_logits(T=40, V=3000, seed=0, dtype="f32", **kw) -> LogitWorkload:
    return LogitWorkload(f"small_logits_t{T}_v{V}", T, V, kw.pop("max_pos", 12000),
                         kw.pop("bin_tokens", 2048), kw.pop("n_bins", 6), dtype=dtype, seed=seed,
                         **kw)
