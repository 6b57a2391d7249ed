"""Benchmark of the sparse decode step on one MI355X.

One step = one decode step of one attention layer for the whole batch: append
the new token's K/V to the paged cache with its page's metadata, page scoring
+ budget + top-k (fused with the append by default), sparse attention over the
selected pages.  Every step appends one token per sequence, so the lengths
advance by one per step.  The dense decode (append + attention over every
token) is timed beside it on the same steps.  Inputs are resident in HBM
before the timed region starts.

The default workload is the largest single-GPU one, the Qwen3-8B-shaped layer
(batch 256, 16K-40K tokens, 32-token pages), swept over budgets of 2, 5, 10, 25
and 100 % of the pages on one cache; the line's ``value`` is the 10 % budget and
``budget_sweep`` holds every budget with its speedup over the dense step.

Prints ONE JSON line.  ``value`` is decode queries per second per layer
(batch / step time).  ``roofline`` reports the dominant entry point's
algorithmic bytes per launch over its average duration (HIP events around each
launch, on the stream its kernels run on) against the 8 TB/s HBM peak.
``cpu_baseline`` times the CPU oracle on a bounded, seeded sample of the same
workload.
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "sparse decode attn queries/sec per layer + achieved HBM GB/s (% of peak) vs dense"
HBM_PEAK_GBPS = 8000.0
C4_HEADLINE = 2            # index of 10 % in the C4 budget sweep
# kernels and sources behind each entry point (the counter summaries are tied to them)
ENTRY = {
    "sparse_attn": ("k_attn_stream<sparse> + k_attn_merge",
                    ("attention.hip", "common.h", "wave.h")),
    "dense_attn": ("k_attn_stream<dense> + k_attn_merge", ("attention.hip", "common.h", "wave.h")),
    "append_score_topk": ("k_page_score (with append) + k_topk",
                          ("score_topk.hip", "topk.h", "common.h", "wave.h")),
    "score_topk": ("k_page_score + k_topk", ("score_topk.hip", "topk.h", "common.h", "wave.h")),
    "decode_step": ("k_page_score (with append) + k_select_attn_unit, or + k_topk + "
                    "k_attn_stream<sparse> + k_attn_merge",
                    ("score_topk.hip", "attention.hip", "topk.h", "common.h", "wave.h")),
    "append": ("k_append_kv", ("append.hip", "common.h")),
}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="c4",
                    help="c4 (default: the budget sweep 2/5/10/25/100 %%, headline 10 %%), "
                         "c4-2/c4-5/c4-10/c4-25/c4-100, c1, c2, c3, c5; "
                         "t4-<page size>-<16k|24k|32k>[-b<batch>] for the page-size study; "
                         "a1 / a1-bf16 for the acceptance rate over paired logit rows")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="target CPU time of the oracle baseline sample (the single-thread "
                         "run takes half of it)")
    ap.add_argument("--step", choices=("fused", "separate", "whole"), default="fused",
                    help="fused: sparrow_append_score_topk + attention; separate: "
                         "sparrow_append_kv, sparrow_page_score_topk, attention; whole: "
                         "sparrow_decode_step (one call per step)")
    ap.add_argument("--landmark", choices=("minmax", "mean"), default="minmax",
                    help="page landmark: channel-wise key min/max (default) or mean key")
    ap.add_argument("--sink", type=int, default=0, help="forced sink pages [0, s)")
    ap.add_argument("--local", type=int, default=0, help="forced most recent pages")
    ap.add_argument("--layers", type=int, default=1,
                    help="attention layers per step, each with its own cache (value stays per "
                         "layer: batch x layers / step time)")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of the whole step captured in one HIP graph")
    ap.add_argument("--cold", action="store_true",
                    help="also time each step after flushing the caches (default for batches "
                         "of at most 16 sequences)")
    ap.add_argument("--batch", type=int, default=0,
                    help="run the decode workload at this batch size instead of its own (lengths "
                         "drawn the same way; for scaling studies, not the headline)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of known size (for counter scaling)")
    return ap.parse_args()


def workload_list(name):
    """(workloads to run on one cache, index of the headline one)."""
    from paper_2606_08446_amd import workloads as W
    if name == "c4":
        return [W.c4_with_fraction(i) for i in range(len(W.C4_FRACTIONS))], C4_HEADLINE
    if name.startswith("t4-"):   # t4-<page size>-<past tokens in K>[-b<batch>]
        parts = name.split("-")
        batch = int(parts[3][1:]) if len(parts) > 3 else 16
        return [W.table4(int(parts[1]), int(parts[2].rstrip("k")) * 1024, batch)], 0
    if name.startswith("c4-"):
        pct = {"2": 0, "5": 1, "10": 2, "25": 3, "100": 4}[name.split("-")[1]]
        return [W.c4_with_fraction(pct)], 0
    return [W.CONFIGS[name]], 0


def budget_label(w):
    s = w.schedule
    if s.n_bins == 1 and s.min_pages[0] == 0:
        return f"{100.0 * s.frac_num[0] / s.frac_den:g}%"
    if s.n_bins == 1 and s.frac_num[0] == 0:
        return f"{s.min_pages[0]} pages"
    if s.n_bins == 1:
        return f"max({s.min_pages[0]} pages, {100.0 * s.frac_num[0] / s.frac_den:g}%)"
    return (f"{100.0 * s.frac_num[0] / s.frac_den:g}% -> "
            f"{100.0 * s.frac_num[-1] / s.frac_den:g}% over {s.n_bins} bins of "
            f"{s.bin_tokens} tokens")


def sparse_bytes(w, lens, k_host, idx_host):
    """Algorithmic HBM bytes of one sparse decode step at lengths ``lens`` (the appended
    token included), per entry point."""
    ps, Hkv, Hq, D = w.page_size, w.num_kv_heads, w.num_q_heads, 128
    append = 0
    score = 0
    kv = 0
    for b, L in enumerate(lens):
        L = int(L)
        if L <= 0:
            continue
        n = -(-L // ps)
        last_valid = L - (n - 1) * ps
        # new K and V rows read and written; the page's metadata read (unless the token
        # opens the page) and written
        append += Hkv * (2 * (2 * D * 2) + (2 * D * 2 if last_valid > 1 else 0) + 2 * D * 2)
        k = int(k_host[b])
        if k < n:
            score += Hkv * n * 2 * D * 2                              # meta rows
        for h in range(Hkv):
            sel = idx_host[b, h, :k]
            toks = k * ps - (ps - last_valid if (n - 1) in set(sel.tolist()) else 0)
            kv += toks * 2 * D * 2                                    # K and V rows
    q_out = len(lens) * Hq * D * (2 + 4)
    return {"append": append, "score_topk": score + len(lens) * Hq * D * 2,
            "sparse_attn": kv + q_out}


def dense_bytes(w, lens):
    """Algorithmic bytes of the dense step: the append's K/V rows and every valid K/V row."""
    B = len(lens)
    attn = int(sum(int(L) for L in lens)) * w.num_kv_heads * 2 * 128 * 2 + \
        B * w.num_q_heads * 128 * (2 + 4)
    return {"append": B * w.num_kv_heads * 4 * 128 * 2, "dense_attn": attn}


def copy_bandwidth(stream):
    """Read + write bytes per second of a plain 1 GiB device-to-device copy (the runtime's
    copy kernel)."""
    import torch
    n = 1 << 30
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    reps = 5
    for _ in range(reps):
        dst.copy_(src)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del src, dst
    return round(2 * n / (ms * 1e-3) / 1e9, 1)


def stream_bandwidth(stream):
    """Bytes per second of the library's read-only streaming reference (sparrow_stream_read)
    over a 4 GiB buffer: the rate a pure read stream of 16-byte non-temporal loads sustains,
    the practical ceiling of the read-dominated decode kernels."""
    import torch

    from paper_2606_08446_amd import sparrow as S
    words = (1 << 30) - 4                      # 4 GiB - 16 B of the value 7
    n = 4 * words
    buf = torch.full((words,), 7, dtype=torch.int32, device="cuda")
    ck = torch.zeros(1, dtype=torch.int32, device="cuda")
    for _ in range(2):
        S.stream_read(buf, ck)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    reps = 10
    for _ in range(reps):
        S.stream_read(buf, ck)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    assert int(ck.item()) & 0xffffffff == (2 + reps) * words * 7 % 2**32, "stream checksum"
    del buf
    return round(n / (ms * 1e-3) / 1e9, 1)


def source_sha(files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2606_08446_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def read_summary(path):
    vals = {}
    if os.path.exists(path):
        for line in open(path):
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    return vals


def read_traffic(entry, workload_name):
    """HBM traffic per launch of an entry point from its committed counter summary
    (profiles/traffic_<entry>_<workload>.txt), if it was taken on this workload with the
    current sources of its kernels; else None."""
    vals = read_summary(os.path.join(ROOT, "profiles", f"traffic_{entry}_{workload_name}.txt"))
    if vals.get("source_sha256") != source_sha(ENTRY[entry][1]) or \
            vals.get("workload") != workload_name or "traffic_bytes_per_launch" not in vals:
        return None
    return float(vals["traffic_bytes_per_launch"])


def acceptance_traffic(workload_name):
    """HBM traffic per k_acceptance launch from its committed counter summary, if it matches
    the current source."""
    vals = read_summary(os.path.join(ROOT, "profiles",
                                     "traffic_acceptance_a1_qwen3_vocab_t4096.txt"))
    if vals.get("source_sha256") != source_sha(("acceptance.hip", "common.h")):
        return None
    v = vals.get(f"traffic_bytes_per_launch[{workload_name}]")
    return None if v is None else float(v)


def cpu_baseline(inp, w, lens_step, k_new, v_new, k_max, target_s, landmark, sink, local):
    """The oracle's sparse decode step on a seeded sample of sequences, repeated to about
    ``target_s`` seconds on every host core and half that on one: append the new token and
    rebuild its page's landmark, score (fp32, the selection precision), budget, top-k,
    attention.  ``lens_step`` are the lengths of the step (the new token included)."""
    import numpy as np
    import torch

    import oracle
    from paper_2606_08446_amd import workloads as W
    s = w.schedule
    ps = w.page_size
    B = w.batch
    n_seq = min(B, 8)
    seqs = sorted(int(x) for x in np.random.default_rng(w.seed + 7).choice(B, n_seq,
                                                                           replace=False))
    lens = np.asarray([lens_step[b] for b in seqs], np.int32)
    bt_all = inp.block_table.cpu().numpy()
    phys, rows = [], []
    for i, b in enumerate(seqs):
        n = -(-int(lens[i]) // ps)
        rows.append(len(phys))
        phys.extend(int(x) for x in bt_all[b, :n])
    max_n = max(1, max(-(-int(L) // ps) for L in lens))
    bt = np.zeros((n_seq, max_n), np.int32)
    for i in range(n_seq):
        n = -(-int(lens[i]) // ps)
        bt[i, :n] = np.arange(rows[i], rows[i] + n)
    pi = torch.as_tensor(np.array(phys, np.int64), device=inp.k_cache.device)
    sel = torch.as_tensor(np.array(seqs, np.int64), device=inp.q.device)
    q = W.bf16_bits(inp.q[sel])
    kc = W.bf16_bits(inp.k_cache[pi])
    vc = W.bf16_bits(inp.v_cache[pi])
    kn = W.bf16_bits(k_new[sel])
    vn = W.bf16_bits(v_new[sel])
    mean = landmark == "mean"
    # setup: the landmarks of the cache before the step
    meta = oracle.page_key_sums(kc, bt, lens - 1) if mean else \
        oracle.page_meta(kc, bt, (lens - 1).astype(np.int32))
    scale = 1.0 / math.sqrt(128.0)

    def run(seconds):
        reps = 0
        t0 = time.perf_counter()
        while True:
            # in place: re-appending the same token rebuilds the same page landmark
            oracle.append_kv(kn, vn, kc, vc, bt, lens, meta, inplace=True,
                             landmark="mean" if mean else "minmax")
            if mean:
                s32, _ = oracle.page_scores_mean(q, meta, bt, lens, ps, fp64=False)
            else:
                s32, _ = oracle.page_scores(q, meta, bt, lens, ps, fp64=False)
            k = np.minimum(oracle.budgets(lens, ps, s.bin_tokens, s.min_pages, s.frac_num,
                                          s.frac_den), k_max).astype(np.int32)
            if sink or local:
                idx = oracle.select_forced(lens, k, s32, ps, k_max, sink, local)
            else:
                idx = oracle.select(lens, k, s32, ps, k_max)
            oracle.attention(q, kc, vc, bt, lens, scale, k, idx)
            reps += 1
            el = time.perf_counter() - t0
            if el >= seconds:
                return reps, el

    threads = oracle.num_threads()
    reps, el = run(target_s)
    oracle.set_num_threads(1)
    try:
        reps1, el1 = run(target_s / 2)
    finally:
        oracle.set_num_threads(threads)
    what = (f"{n_seq} of {B} sequences of {w.name} drawn with seed {w.seed + 7} "
            f"({', '.join(str(b) for b in seqs)}), whole sparse decode step ({landmark} "
            f"landmark: append of the new token with its page's landmark rebuilt, fp32 scores, "
            f"budget, top-k, fp64 attention)")
    return {"value": round(n_seq * reps / el, 3), "unit": "queries/s", "cores": threads,
            "kind": "oracle", "sample": f"{what} repeated {reps}x in {el:.1f} s",
            "single_thread": {"value": round(n_seq * reps1 / el1, 3), "unit": "queries/s",
                              "cores": 1, "sample": f"the same, repeated {reps1}x in "
                                                    f"{el1:.1f} s on one thread"}}


def copy_calibration():
    """A plain device-to-device copy of known size, for scaling the HBM counters."""
    import torch
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_each_way": n, "launches": 5}), flush=True)


def bench_acceptance(args):
    """Acceptance rate of every token of a logit workload, then the per-bin tail statistic."""
    import numpy as np
    import torch

    from paper_2606_08446_amd import sparrow as S
    from paper_2606_08446_amd import workloads as W
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    lw = W.LOGIT_CONFIGS[args.workload]
    li = W.generate_logits(lw, dev)
    T, V = lw.tokens, lw.vocab
    esz = 4 if lw.dtype == "f32" else 2
    alpha = torch.empty(T, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step():
        S.acceptance_rate(li.target, li.draft, 1.0, alpha=alpha)
        return S.tail_stats(alpha, li.positions, lw.bin_tokens, lw.n_bins, 5.0)

    def timed(fn, count):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(count):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / count

    for _ in range(args.warmup):
        step()
    t_wall = time.perf_counter()
    ms_step = timed(step, args.steps)
    wall = time.perf_counter() - t_wall
    ms_alpha = timed(lambda: S.acceptance_rate(li.target, li.draft, 1.0, alpha=alpha), args.steps)
    ms_tail = timed(lambda: S.tail_stats(alpha, li.positions, lw.bin_tokens, lw.n_bins, 5.0),
                    args.steps)
    q, m, c = step()
    torch.cuda.synchronize()
    alg = T * 2 * V * esz                      # both logit rows of every token, read once
    alg_tail = T * 8
    dom_gbps = alg / (ms_alpha * 1e-3) / 1e9
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        n = 8
        tg = li.target[:n].cpu() if lw.dtype == "f32" else None
        rows_t = tg.numpy() if tg is not None else W.bf16_bits(li.target[:n])
        rows_d = li.draft[:n].cpu().numpy() if lw.dtype == "f32" else W.bf16_bits(li.draft[:n])
        reps, t0 = 0, time.perf_counter()
        while True:
            oracle.acceptance(rows_t, rows_d)
            reps += 1
            el = time.perf_counter() - t0
            if el >= args.cpu_seconds:
                break
        cpu = {"value": round(n * reps / el, 3), "unit": "tokens/s", "cores": oracle.num_threads(),
               "kind": "oracle",
               "sample": f"first {n} of {T} tokens of {lw.name}: fp64 acceptance rate over the "
                         f"{V}-entry vocabulary, repeated {reps}x in {el:.1f} s"}
    result = {
        "metric": "acceptance rate tokens/sec (Eq. 1 over the full vocabulary) + per-bin "
                  "5-percentile, achieved HBM GB/s (% of peak)",
        "value": round(T / (ms_step * 1e-3), 2), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": lw.dtype, "data": "synthetic",
        "config": {"workload": lw.name, "tokens": T, "vocab": V, "bin_tokens": lw.bin_tokens,
                   "n_bins": lw.n_bins, "percentile": 5.0},
        "achieved_GBps": round((alg + alg_tail) / (ms_step * 1e-3) / 1e9, 1),
        "hbm_frac": round((alg + alg_tail) / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
        "phase_ms": {"acceptance_rate": round(ms_alpha, 5), "tail_stats": round(ms_tail, 5)},
        "roofline": {"kernel": f"k_acceptance<{'float' if esz == 4 else 'bf16'}>", "bound": "hbm",
                     "achieved": round(dom_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(dom_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": acceptance_traffic(lw.name)},
        "measured_stream_GBps": stream_bandwidth(stream),
        "tail_5pct_per_bin": [round(float(x), 5) for x in q.cpu().numpy()],
        "mean_per_bin": [round(float(x), 5) for x in m.cpu().numpy()],
        "wall_s_timed": round(wall, 3),
        "cpu_baseline": cpu,
    }
    print(json.dumps(result), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the sparse decode "
              "path runs one process per GPU and has no multi-GPU mode.", file=sys.stderr, flush=True)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.workload.startswith("a1"):
        bench_acceptance(args)
        return
    if args.graph and args.landmark == "mean":
        print("--graph replays re-append the same token, which the mean landmark's key sums "
              "would count again: use --graph with the min/max landmark", file=sys.stderr,
              flush=True)
        sys.exit(2)
    bench_decode(args)


def bench_decode(args):
    import numpy as np
    import torch

    from paper_2606_08446_amd import cost_model
    from paper_2606_08446_amd import sparrow as S
    from paper_2606_08446_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    K, Wm = args.steps, args.warmup
    runs, headline = workload_list(args.workload)
    total = Wm + K
    ps = runs[0].page_size
    # every step appends one token per sequence: spare pages for all of them
    runs = [dataclasses.replace(w, extra_pages=(total + 1 + ps - 1) // ps + 1) for w in runs]
    if args.batch > 0:
        runs = [dataclasses.replace(w, batch=args.batch, name=f"{w.name}_batch{args.batch}")
                for w in runs]
    base = runs[headline]
    B, Hkv = base.batch, base.num_kv_heads
    L_layers = args.layers
    fused = args.step == "fused"
    whole = args.step == "whole"
    landmark = S.SPARROW_LANDMARK_MEAN if args.landmark == "mean" else S.SPARROW_LANDMARK_MINMAX
    stream = torch.cuda.current_stream(dev)
    sp = stream.cuda_stream

    # the lengths the workload generator draws first from its seed; step i appends the token
    # at position lens0 + i, so its lengths are lens0 + i + 1
    lens_host0 = np.random.default_rng(base.seed).integers(base.len_lo, base.len_hi + 1,
                                                           size=B).astype(np.int64)
    lens_host_steps = lens_host0[None, :] + np.arange(1, total + 1)[:, None]
    lens_steps = torch.as_tensor(lens_host_steps.astype(np.int32), device=dev).contiguous()

    class Layer:
        """One attention layer: its own cache, landmarks and new rows; the lengths (and so
        the schedule) are shared by all layers, as in a model."""

        def __init__(self, li):
            seed = base.seed + 1000 * li
            # layer 0 is the workload itself; the others reuse its lengths
            self.inp = W.generate(base, dev, lengths=None if li == 0 else list(lens_host0),
                                  seed=seed)
            assert list(self.inp.lens_host) == list(lens_host0)
            gen = torch.Generator(device=dev)
            gen.manual_seed(seed + 1)
            self.k_new = torch.randn((total, B, Hkv, 128), generator=gen,
                                     device=dev).to(torch.bfloat16)
            self.v_new = torch.randn((total, B, Hkv, 128), generator=gen,
                                     device=dev).to(torch.bfloat16)
            inp = self.inp
            self.meta = S.new_meta(inp.num_phys_pages, Hkv, dev, landmark)
            S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, self.meta,
                               landmark=landmark)
            self.shape = S.shape_of(inp.q, inp.k_cache, inp.block_table, landmark=landmark)
            # landmarks before the first step and before the first timed step: every pass
            # over the steps starts from one of them, so re-running a step appends to the
            # landmarks it saw the first time (the mean landmark's sums are not idempotent)
            self.snap0 = self.meta.clone()
            for i in range(Wm):
                S._check("sparrow_append_kv", S.sparrow_append_kv(
                    self.shape, self.k_new[i].data_ptr(), self.v_new[i].data_ptr(),
                    inp.k_cache.data_ptr(), inp.v_cache.data_ptr(), inp.block_table.data_ptr(),
                    lens_steps[i].data_ptr(), self.meta.data_ptr(), sp))
            self.snap_w = self.meta.clone()
            self.dense_out = torch.empty(inp.q.shape, dtype=torch.float32, device=dev)
            self.dense_ws = torch.empty(max(16, S.sparrow_workspace_size(
                self.shape, 0, S.SPARROW_OP_DENSE_ATTN)), dtype=torch.uint8, device=dev)
            self.step = None

        def restore(self, before_timed):
            self.meta.copy_(self.snap_w if before_timed else self.snap0)

        def use_schedule(self, w, k_max):
            inp = W.with_schedule(self.inp, w)
            s = w.schedule
            self.step = S.SparseDecodeStep(inp.q, inp.k_cache, inp.v_cache, inp.block_table,
                                           inp.seq_lens, self.meta, inp.min_pages, inp.frac_num,
                                           s.frac_den, s.bin_tokens, k_max, landmark=landmark,
                                           sink_pages=args.sink, local_pages=args.local)

        def select(self, i, sp):
            st = self.step
            if fused:
                st.append_score_topk(self.k_new[i], self.v_new[i], sp, seq_lens=lens_steps[i])
            else:
                st.append(self.k_new[i], self.v_new[i], sp, seq_lens=lens_steps[i])
                st.score_topk(sp, seq_lens=lens_steps[i])

        def attend(self, i, sp):
            self.step.attend(sp, seq_lens=lens_steps[i])

        def sparse(self, i, sp):
            if whole:
                self.step.decode_step(self.k_new[i], self.v_new[i], sp, seq_lens=lens_steps[i])
                return
            self.select(i, sp)
            self.attend(i, sp)

        def append_only(self, i, sp):
            inp = self.inp
            S._check("sparrow_append_kv", S.sparrow_append_kv(
                self.shape, self.k_new[i].data_ptr(), self.v_new[i].data_ptr(),
                inp.k_cache.data_ptr(), inp.v_cache.data_ptr(), inp.block_table.data_ptr(),
                lens_steps[i].data_ptr(), self.meta.data_ptr(), sp))

        def dense_attend(self, i, sp):
            inp = self.inp
            S._check("sparrow_dense_decode_attn", S.sparrow_dense_decode_attn(
                self.shape, inp.q.data_ptr(), inp.k_cache.data_ptr(), inp.v_cache.data_ptr(),
                inp.block_table.data_ptr(), lens_steps[i].data_ptr(),
                1.0 / math.sqrt(128.0), self.dense_out.data_ptr(), S.SPARROW_OUT_F32,
                self.dense_ws.data_ptr(), self.dense_ws.numel(), sp))

        def dense(self, i, sp):
            self.append_only(i, sp)
            self.dense_attend(i, sp)

    layers = [Layer(li) for li in range(L_layers)]
    lay0 = layers[0]
    torch.cuda.synchronize()

    def restore(before_timed):
        for lay in layers:
            lay.restore(before_timed)

    def timed(fn, first, count):
        """Average time of fn(i), i = first .. first + count - 1, run back to back between
        two events."""
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for i in range(first, first + count):
            fn(i)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / count

    def per_launch(fns, first, count):
        """Average duration of each entry point fns[j](i) over the steps, every call
        bracketed by its own pair of events on the stream it runs on."""
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(fns) + 1)]
              for _ in range(count)]
        torch.cuda.synchronize()
        for j, i in enumerate(range(first, first + count)):
            ev[j][0].record(stream)
            for f, fn in enumerate(fns):
                fn(i)
                ev[j][f + 1].record(stream)
        torch.cuda.synchronize()
        return [sum(ev[j][f].elapsed_time(ev[j][f + 1]) for j in range(count)) / count
                for f in range(len(fns))]

    def step_times(fn, first, count):
        """Duration of each step fn(i) on its own (one event between consecutive steps), for
        the median and tail; a separate pass from the back-to-back timing."""
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(count + 1)]
        torch.cuda.synchronize()
        ev[0].record(stream)
        for j, i in enumerate(range(first, first + count)):
            fn(i)
            ev[j + 1].record(stream)
        torch.cuda.synchronize()
        return [ev[j].elapsed_time(ev[j + 1]) for j in range(count)]

    def captured(fn, i):
        """fn(layer, i, stream) for every layer captured in one graph; a replay callable."""
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            with torch.cuda.graph(g, stream=side):
                csp = torch.cuda.current_stream().cuda_stream
                for lay in layers:
                    fn(lay, i, csp)
        stream.wait_stream(side)
        torch.cuda.synchronize()
        return lambda _i: g.replay()

    cold = args.cold or B <= 16
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev) if cold else None

    def cold_steps(fn, first, count):
        """Average time of fn(i) run after writing 512 MiB elsewhere, which evicts the L2
        caches and the 256 MB Infinity Cache: every step starts from HBM."""
        e0 = [torch.cuda.Event(enable_timing=True) for _ in range(count)]
        e1 = [torch.cuda.Event(enable_timing=True) for _ in range(count)]
        torch.cuda.synchronize()
        for j, i in enumerate(range(first, first + count)):
            flush.fill_(j & 0xff)
            e0[j].record(stream)
            fn(i)
            e1[j].record(stream)
        torch.cuda.synchronize()
        return sum(a.elapsed_time(b) for a, b in zip(e0, e1)) / count

    def sparse_step(i):
        for lay in layers:
            lay.sparse(i, sp)

    def dense_step(i):
        for lay in layers:
            lay.dense(i, sp)

    lens_last = lens_host_steps[Wm if args.graph else total - 1]
    results = []
    wall = None
    cpu = None
    for ri, w in enumerate(runs):
        s = w.schedule
        k_max = S.budget_bound(lens_host_steps.ravel(), ps, s.bin_tokens, s.min_pages,
                               s.frac_num, s.frac_den)
        for lay in layers:
            lay.use_schedule(w, k_max)
        restore(False)
        for i in range(Wm):
            sparse_step(i)
        torch.cuda.synchronize()
        # ---- timed sparse steps: exactly K steps between two events, nothing else inside
        if args.graph:
            # the graph holds the step at index Wm (all layers); each replay re-appends the
            # same token, which leaves caches and min/max landmarks as they were
            sparse_fn = captured(Layer.sparse, Wm)
        else:
            sparse_fn = sparse_step
        t_wall = time.perf_counter()
        ms_step = timed(sparse_fn, Wm, K)
        if ri == headline:
            wall = time.perf_counter() - t_wall
        # ---- per-entry-point durations of layer 0 over the same steps, from the landmarks
        # the timed loop started from
        restore(True)
        if whole:
            names = ["decode_step"]
            fns = [lambda i: lay0.sparse(i, sp)]
        elif fused:
            names = ["append_score_topk", "sparse_attn"]
            fns = [lambda i: lay0.select(i, sp), lambda i: lay0.attend(i, sp)]
        else:
            names = ["append", "score_topk", "sparse_attn"]
            fns = [lambda i: lay0.step.append(lay0.k_new[i], lay0.v_new[i], sp,
                                              seq_lens=lens_steps[i]),
                   lambda i: lay0.step.score_topk(sp, seq_lens=lens_steps[i]),
                   lambda i: lay0.attend(i, sp)]
        if args.graph:
            phase = dict(zip(names, per_launch(fns, Wm, 1)))   # the step the graph holds
        else:
            phase = dict(zip(names, per_launch(fns, Wm, K)))
        restore(True)
        per_step = np.array(step_times(sparse_fn, Wm, K))
        k_host = lay0.step.k.cpu().numpy()
        idx_host = lay0.step.idx.cpu().numpy()
        ms_cold = None
        if cold and not args.graph:
            restore(True)
            ms_cold = cold_steps(sparse_step, Wm, K)
        by = sparse_bytes(w, lens_last, k_host, idx_host)
        if whole:
            by = {"decode_step": by["append"] + by["score_topk"] + by["sparse_attn"]}
        elif fused:
            by = {"append_score_topk": by["append"] + by["score_topk"],
                  "sparse_attn": by["sparse_attn"]}
        total_bytes = sum(by.values())
        gbps = total_bytes * L_layers / (ms_step * 1e-3) / 1e9
        d_el, s_el = cost_model.decode_step_elements(lens_last, k_host.astype(np.int64) * ps,
                                                     ps, Hkv * 128)
        dominant = max(phase, key=phase.get)
        r = {"workload": w.name, "budget": budget_label(w),
             "budget_pages": [int(k_host.min()), int(k_host.max())], "k_max": int(k_max),
             "queries_per_s": round(B * L_layers / (ms_step * 1e-3), 2),
             "ms_per_step": round(ms_step, 5),
             "p50_ms_per_step": round(float(np.median(per_step)), 5),
             "p90_ms_per_step": round(float(np.percentile(per_step, 90)), 5),
             "achieved_GBps": round(gbps, 1), "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4),
             "algorithmic_bytes_per_step": {k: int(v) for k, v in by.items()},
             "phase_ms": {k: round(v, 5) for k, v in phase.items()},
             "phase_hbm_frac": {k: round(by[k] / (phase[k] * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4)
                                for k in phase},
             "dominant": dominant,
             "predicted_speedup_memory_bound": round(d_el / s_el, 3)}
        if ms_cold is not None:
            r["cold_cache"] = {"ms_per_step": round(ms_cold, 5),
                               "queries_per_s": round(B * L_layers / (ms_cold * 1e-3), 2)}
        results.append(r)
        if ri == headline and not args.no_cpu_baseline:
            cpu = cpu_baseline(lay0.inp, w, lens_last, lay0.k_new[Wm if args.graph else total - 1],
                               lay0.v_new[Wm if args.graph else total - 1], k_max,
                               args.cpu_seconds, args.landmark, args.sink, args.local)
        for lay in layers:
            lay.step = None          # free this budget's page lists and workspaces
        torch.cuda.empty_cache()

    # ---- dense steps over the same appended tokens
    restore(False)
    for i in range(Wm):
        dense_step(i)
    dense_fn = captured(Layer.dense, Wm) if args.graph else dense_step
    ms_dense = timed(dense_fn, Wm, K)
    restore(True)
    dense_steps = np.array(step_times(dense_fn, Wm, K))
    restore(True)
    dphase = dict(zip(["append", "dense_attn"],
                      per_launch([lambda i: lay0.append_only(i, sp),
                                  lambda i: lay0.dense_attend(i, sp)], Wm, 1 if args.graph else K)))
    dby = dense_bytes(base, lens_last)
    dgbps = sum(dby.values()) * L_layers / (ms_dense * 1e-3) / 1e9
    dense = {"queries_per_s": round(B * L_layers / (ms_dense * 1e-3), 2),
             "ms_per_step": round(ms_dense, 5),
             "p50_ms_per_step": round(float(np.median(dense_steps)), 5),
             "bytes_per_step": int(sum(dby.values())),
             "achieved_GBps": round(dgbps, 1), "hbm_frac": round(dgbps / HBM_PEAK_GBPS, 4),
             "phase_ms": {k: round(v, 5) for k, v in dphase.items()},
             "attention_hbm_frac": round(dby["dense_attn"] / (dphase["dense_attn"] * 1e-3) / 1e9
                                         / HBM_PEAK_GBPS, 4),
             "step": "append, dense attention"}
    if cold and not args.graph:
        restore(True)
        dense["cold_cache_ms_per_step"] = round(cold_steps(dense_step, Wm, K), 5)
    for r in results:
        r["speedup_vs_dense"] = round(ms_dense / r["ms_per_step"], 3)
    copy_gbps = copy_bandwidth(stream)
    stream_gbps = stream_bandwidth(stream)

    h = results[headline]
    dom = h["dominant"]
    dom_bytes = h["algorithmic_bytes_per_step"][dom]
    dom_gbps = dom_bytes / (h["phase_ms"][dom] * 1e-3) / 1e9
    w = runs[headline]
    result = {
        "metric": METRIC,
        "value": h["queries_per_s"],
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wm,
        "ms_per_step": h["ms_per_step"],
        "p50_ms_per_step": h["p50_ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": B, "num_q_heads": w.num_q_heads, "num_kv_heads": Hkv,
                   "head_dim": 128, "page_size": ps, "len_range": [w.len_lo, w.len_hi],
                   "budget": h["budget"],
                   "budgets_swept": [r["budget"] for r in results] if len(runs) > 1 else None,
                   "budget_pages": h["budget_pages"], "k_max": h["k_max"],
                   "layers": L_layers, "landmark": args.landmark, "sink_pages": args.sink,
                   "local_pages": args.local, "graph": bool(args.graph),
                   "step": ("append+score+top-k+attention in one call" if whole else
                            "append+score+top-k fused, attention" if fused else
                            "append, score+top-k, attention") +
                           "; one token appended per sequence per step"},
        "achieved_GBps": h["achieved_GBps"],
        "hbm_frac": h["hbm_frac"],
        "measured_copy_GBps": copy_gbps,
        "measured_stream_GBps": stream_gbps,
        "algorithmic_bytes_per_step": h["algorithmic_bytes_per_step"],
        "phase_ms": h["phase_ms"],
        "phase_hbm_frac": h["phase_hbm_frac"],
        "dense": dense,
        "speedup_vs_dense": h["speedup_vs_dense"],
        "cost_model": {"predicted_speedup_memory_bound": h["predicted_speedup_memory_bound"]},
        "roofline": {"kernel": ENTRY[dom][0], "entry_point": dom, "bound": "hbm",
                     "achieved": round(dom_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(dom_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": read_traffic(dom, w.name)},
        "wall_s_timed": round(wall, 3),
        "cpu_baseline": cpu,
    }
    if "cold_cache" in h:
        result["cold_cache"] = h["cold_cache"]
    if len(runs) > 1:
        result["budget_sweep"] = results
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
