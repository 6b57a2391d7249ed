"""Benchmark of the sparse decode step on one MI355X.

One step = one decode step of one attention layer for the whole batch: append
the new token's K/V to the paged cache with its page's metadata, page scoring
+ budget + top-k (fused with the append by default), sparse attention over the
selected pages.  Every step appends one token per sequence, so the lengths
advance by one per step.  The dense decode (append + attention over every
token) is timed beside it on the same steps.  Inputs are resident in HBM
before the timed region starts.

Prints ONE JSON line.  ``value`` is decode queries per second per layer
(batch / step time).  ``roofline`` reports the dominant entry point's
algorithmic bytes per launch over its average duration (HIP events around K
back-to-back launches of that entry point, on the stream its kernels run on)
against the 8 TB/s HBM peak.
``cpu_baseline`` times the CPU oracle on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
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
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_sparse_attn_c2_qwen3_1p7b_b64.txt")


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="c2",
                    help="c1..c5, or c4-2/c4-5/c4-10/c4-25/c4-100; t4-<page size>-<16k|24k|32k>"
                         "[-b<batch>] for the page-size study; a1 / a1-bf16 for the acceptance "
                         "rate over paired logit rows")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="target CPU time of the oracle baseline sample")
    ap.add_argument("--step", choices=("fused", "separate"), default="fused",
                    help="fused: sparrow_append_score_topk + attention; separate: "
                         "sparrow_append_kv, sparrow_page_score_topk, attention")
    ap.add_argument("--landmark", choices=("minmax", "mean"), default="minmax",
                    help="page landmark: channel-wise key min/max (default) or mean key")
    ap.add_argument("--sink", type=int, default=0, help="forced sink pages [0, s)")
    ap.add_argument("--local", type=int, default=0, help="forced most recent pages")
    ap.add_argument("--layers", type=int, default=1,
                    help="attention layers per step, each with its own cache (value stays per "
                         "layer: batch x layers / step time)")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of the whole step captured in one HIP graph")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of known size (for counter scaling)")
    return ap.parse_args()


def workload(name):
    from paper_2606_08446_amd import workloads as W
    if name.startswith("t4-"):   # t4-<page size>-<past tokens in K>[-b<batch>]
        parts = name.split("-")
        batch = int(parts[3][1:]) if len(parts) > 3 else 16
        return W.table4(int(parts[1]), int(parts[2].rstrip("k")) * 1024, batch)
    if name.startswith("c4-"):
        pct = {"2": 0, "5": 1, "10": 2, "25": 3, "100": 4}[name.split("-")[1]]
        return W.c4_with_fraction(pct)
    return W.CONFIGS[name]


def sparse_bytes(inp, lens, k_host, idx_host):
    """Algorithmic HBM bytes of one sparse decode step at lengths ``lens`` (the appended
    token included), per entry point."""
    w = inp.workload
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


def dense_bytes(inp, lens):
    """Algorithmic bytes of the dense step: the append's K/V rows and every valid K/V row."""
    w = inp.workload
    B = len(lens)
    return int(sum(int(L) for L in lens)) * w.num_kv_heads * 2 * 128 * 2 + \
        B * w.num_q_heads * 128 * (2 + 4) + B * w.num_kv_heads * 4 * 128 * 2


def copy_bandwidth(stream):
    """Read + write bytes per second of a plain 1 GiB device-to-device copy (the runtime's
    copy kernel): a practical streaming reference beside the 8 TB/s peak."""
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


def read_traffic(kernel_src_sha, workload_name):
    """HBM traffic per launch from the committed counter summary, if it was taken on this
    workload with the current attention source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    vals = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_sha256") != kernel_src_sha or vals.get("workload") != workload_name or \
            "traffic_bytes_per_launch" not in vals:
        return None
    return float(vals["traffic_bytes_per_launch"])


def acceptance_traffic(workload_name):
    """HBM traffic per k_acceptance launch from its committed counter summary, if it matches
    the current source."""
    path = os.path.join(ROOT, "profiles", "traffic_acceptance_a1_qwen3_vocab_t4096.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_sha256") != source_sha(("acceptance.hip", "common.h")):
        return None
    v = vals.get(f"traffic_bytes_per_launch[{workload_name}]")
    return None if v is None else float(v)


def source_sha(files=("attention.hip", "common.h", "wave.h")):
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2606_08446_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def cpu_baseline(inp, lens_step, k_new, v_new, k_max, target_s):
    """The oracle's sparse decode step on a sample of sequences, repeated to ~target_s
    seconds: append the new token, rebuild its page's metadata, score, budget, top-k,
    attention.  ``lens_step`` are the lengths of the step (the new token included)."""
    import numpy as np
    import torch

    import oracle
    from paper_2606_08446_amd import workloads as W
    w = inp.workload
    s = w.schedule
    ps = w.page_size
    B = w.batch
    n_seq = min(B, 8)
    seqs = list(range(n_seq))
    lens = np.asarray(lens_step[:n_seq], np.int32)
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
    q = W.bf16_bits(inp.q[:n_seq])
    kc = W.bf16_bits(inp.k_cache[pi])
    vc = W.bf16_bits(inp.v_cache[pi])
    kn = W.bf16_bits(k_new[:n_seq])
    vn = W.bf16_bits(v_new[:n_seq])
    meta = oracle.page_meta(kc, bt, (lens - 1).astype(np.int32))  # setup: before the step
    scale = 1.0 / math.sqrt(128.0)
    reps = 0
    t0 = time.perf_counter()
    while True:
        # in place: re-appending the same token leaves the arrays as they were after the first
        oracle.append_kv(kn, vn, kc, vc, bt, lens, meta, inplace=True)
        s32, _ = oracle.page_scores(q, meta, bt, lens, ps)
        k = np.minimum(oracle.budgets(lens, ps, s.bin_tokens, s.min_pages, s.frac_num,
                                      s.frac_den), k_max).astype(np.int32)
        idx = oracle.select(lens, k, s32, ps, k_max)
        oracle.attention(q, kc, vc, bt, lens, scale, k, idx)
        reps += 1
        el = time.perf_counter() - t0
        if el >= target_s:
            break
    return {"value": round(n_seq * reps / el, 3), "unit": "queries/s",
            "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"first {n_seq} of {B} sequences of {w.name}, whole sparse decode step "
                      f"(append of the new token with its page's metadata rebuilt, fp32+fp64 "
                      f"scores, budget, top-k, fp64 attention) repeated {reps}x in {el:.1f} s"}


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

    import dataclasses

    import numpy as np
    import torch

    from paper_2606_08446_amd import sparrow as S
    from paper_2606_08446_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    K, Wm = args.steps, args.warmup
    w = workload(args.workload)
    ps = w.page_size
    # every step appends one token per sequence: spare pages for all of them
    w = dataclasses.replace(w, extra_pages=(Wm + K + 1 + ps - 1) // ps + 1)
    L_layers = args.layers
    s = w.schedule
    B, Hkv = w.batch, w.num_kv_heads
    total = Wm + K
    fused = args.step == "fused"
    landmark = S.SPARROW_LANDMARK_MEAN if args.landmark == "mean" else S.SPARROW_LANDMARK_MINMAX

    class Layer:
        """One attention layer: its own cache, metadata and new rows; the lengths (and so
        the schedule) are shared by all layers, as in a model."""

        def __init__(self, li, lengths):
            seed = w.seed + 1000 * li
            # layer 0 is the workload itself; the others reuse its lengths
            self.inp = W.generate(w, dev, lengths=None if li == 0 else lengths, seed=seed)
            assert list(self.inp.lens_host) == list(lengths)
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
            self.step = S.SparseDecodeStep(inp.q, inp.k_cache, inp.v_cache, inp.block_table,
                                           inp.seq_lens, self.meta, inp.min_pages, inp.frac_num,
                                           s.frac_den, s.bin_tokens, k_max, landmark=landmark,
                                           sink_pages=args.sink, local_pages=args.local)
            self.dense_out = torch.empty(inp.q.shape, dtype=torch.float32, device=dev)
            self.dense_ws = torch.empty(max(16, S.sparrow_workspace_size(
                self.step.shape, 0, S.SPARROW_OP_DENSE_ATTN)), dtype=torch.uint8, device=dev)

        def select(self, i, sp):
            st = self.step
            if fused:
                st.append_score_topk(self.k_new[i], self.v_new[i], sp, seq_lens=lens_steps[i])
            else:
                st.append(self.k_new[i], self.v_new[i], sp, seq_lens=lens_steps[i])
                st.score_topk(sp, seq_lens=lens_steps[i])

        def sparse(self, i, sp):
            self.select(i, sp)
            self.step.attend(sp, seq_lens=lens_steps[i])

        def dense(self, i, sp):
            st, inp = self.step, self.inp
            st.append(self.k_new[i], self.v_new[i], sp, seq_lens=lens_steps[i])
            S._check("sparrow_dense_decode_attn", S.sparrow_dense_decode_attn(
                st.shape, inp.q.data_ptr(), inp.k_cache.data_ptr(), inp.v_cache.data_ptr(),
                inp.block_table.data_ptr(), lens_steps[i].data_ptr(), st.scale,
                self.dense_out.data_ptr(), S.SPARROW_OUT_F32, self.dense_ws.data_ptr(),
                self.dense_ws.numel(), sp))

    # the lengths the workload generator draws first from its seed
    lens_host0 = np.random.default_rng(w.seed).integers(w.len_lo, w.len_hi + 1,
                                                        size=B).astype(np.int64)
    # step i appends the token at position lens0 + i: its lengths are lens0 + i + 1
    lens_host_steps = lens_host0[None, :] + np.arange(1, total + 1)[:, None]
    lens_steps = torch.as_tensor(lens_host_steps.astype(np.int32), device=dev).contiguous()
    k_max = S.budget_bound(lens_host_steps.ravel(), ps, s.bin_tokens, s.min_pages, s.frac_num,
                           s.frac_den)
    layers = [Layer(li, list(lens_host0)) for li in range(L_layers)]
    inp, step = layers[0].inp, layers[0].step
    stream = torch.cuda.current_stream(dev)
    sp = stream.cuda_stream

    def sparse_step(i):
        for lay in layers:
            lay.sparse(i, sp)

    def dense_step(i):
        for lay in layers:
            lay.dense(i, sp)

    def timed(fn, first, count):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for i in range(first, first + count):
            fn(i)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / count

    def captured(fn, i):
        """fn(i) for every layer captured in one graph; returns a replay callable."""
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

    for i in range(Wm):
        sparse_step(i)
    torch.cuda.synchronize()

    # ---- timed sparse steps: exactly K steps between two events, nothing else inside
    if args.graph:
        # the graph holds the step at index Wm (all layers); each replay re-appends the same
        # token, which leaves caches and metadata unchanged: the same work every replay
        sparse_fn = captured(Layer.sparse, Wm)
        dense_fn = captured(Layer.dense, Wm)
    else:
        sparse_fn, dense_fn = sparse_step, dense_step
    t_wall = time.perf_counter()
    ms_step = timed(sparse_fn, Wm, K)
    wall = time.perf_counter() - t_wall
    k_host = step.k.cpu().numpy()
    idx_host = step.idx.cpu().numpy()

    # ---- per-entry-point durations of layer 0 (a separate loop over the same steps;
    # re-running a step rewrites the same token, which leaves caches and metadata unchanged)
    lay0 = layers[0]
    phase = {}
    if fused:
        phase["append_score_topk"] = timed(lambda i: lay0.select(i, sp), Wm, K)
    else:
        phase["append"] = timed(lambda i: step.append(lay0.k_new[i], lay0.v_new[i], sp,
                                                      seq_lens=lens_steps[i]), Wm, K)
        phase["score_topk"] = timed(lambda i: step.score_topk(sp, seq_lens=lens_steps[i]), Wm, K)
    phase["sparse_attn"] = timed(lambda i: step.attend(sp, seq_lens=lens_steps[i]), Wm, K)

    # ---- timed dense steps over the same appended tokens
    ms_dense = timed(dense_fn, Wm, K)
    if args.graph:
        lens_host_steps = lens_host_steps[:Wm + 1]  # every replay ran step Wm
    lens_last = lens_host_steps[-1]
    by = sparse_bytes(inp, lens_last, k_host, idx_host)
    if fused:
        by = {"append_score_topk": by["append"] + by["score_topk"],
              "sparse_attn": by["sparse_attn"]}
    total_bytes = sum(by.values())
    dbytes = dense_bytes(inp, lens_last)
    gbps = total_bytes * L_layers / (ms_step * 1e-3) / 1e9
    dgbps = dbytes * L_layers / (ms_dense * 1e-3) / 1e9
    dominant = max(phase, key=phase.get)
    dom_gbps = by[dominant] / (phase[dominant] * 1e-3) / 1e9
    traffic = read_traffic(source_sha(), w.name) if dominant == "sparse_attn" else None
    copy_gbps = copy_bandwidth(stream)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(inp, lens_last, lay0.k_new[len(lens_host_steps) - 1],
                           lay0.v_new[len(lens_host_steps) - 1], k_max, args.cpu_seconds)

    from paper_2606_08446_amd import cost_model
    d_el, s_el = cost_model.decode_step_elements(lens_last, np.asarray(k_host) * ps, ps, Hkv * 128)
    budgets = np.asarray(k_host)
    kernels = {"sparse_attn": "k_attn_stream<sparse> + k_attn_merge",
               "append_score_topk": "k_page_score (with append) + k_topk",
               "score_topk": "k_page_score + k_topk", "append": "k_append_kv"}
    result = {
        "metric": METRIC,
        "value": round(B * L_layers / (ms_step * 1e-3), 2),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wm,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": B, "num_q_heads": w.num_q_heads,
                   "num_kv_heads": Hkv, "head_dim": 128, "page_size": ps,
                   "len_range": [w.len_lo, w.len_hi], "budget_pages": [int(budgets.min()),
                                                                       int(budgets.max())],
                   "k_max": int(k_max), "layers": L_layers, "landmark": args.landmark,
                   "sink_pages": args.sink, "local_pages": args.local,
                   "graph": bool(args.graph),
                   "step": ("append+score+top-k fused, attention" if fused else
                            "append, score+top-k, attention") +
                           "; one token appended per sequence per step"},
        "achieved_GBps": round(gbps, 1),
        "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4),
        "measured_copy_GBps": copy_gbps,
        "algorithmic_bytes_per_step": {k: int(v) for k, v in by.items()},
        "phase_ms": {k: round(v, 5) for k, v in phase.items()},
        "dense": {"queries_per_s": round(B * L_layers / (ms_dense * 1e-3), 2),
                  "ms_per_step": round(ms_dense, 5),
                  "bytes_per_step": int(dbytes), "achieved_GBps": round(dgbps, 1),
                  "hbm_frac": round(dgbps / HBM_PEAK_GBPS, 4),
                  "step": "append, dense attention"},
        "speedup_vs_dense": round(ms_dense / ms_step, 3),
        "cost_model": {"dense_elements": int(d_el), "sparse_elements": int(s_el),
                       "predicted_speedup_memory_bound": round(d_el / s_el, 3)},
        "roofline": {"kernel": kernels[dominant],
                     "bound": "hbm", "achieved": round(dom_gbps, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(dom_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": traffic},
        "wall_s_timed": round(wall, 3),
        "cpu_baseline": cpu,
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
