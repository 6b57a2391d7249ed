"""A decode step captured in a HIP graph (through torch's graph capture) replays to the
same results as the eager calls.  The library records no memset or allocation, so the
captured kernels are the whole step: several layers, each an append fused with scoring
and top-k, then sparse attention - or each one sparrow_decode_step call, on layers that
take the one-kernel selection and attention and layers that stream."""
import numpy as np
import pytest
import torch

from paper_2606_08446_amd import sparrow as S
from paper_2606_08446_amd import workloads as W

from parity import log

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(autouse=True)
def _need_gpu(gpu_device):
    S.load()
    yield


def make_layer(seed, G=4):
    w = W.small(B=3, Hq=2 * G, Hkv=2, ps=16, lengths=(300, 1000, 17), seed=seed,
                schedule=W.fraction_budget(1, 5, floor_pages=2), hot_pages=2)
    inp = W.generate(w, DEV, lengths=[300, 1000, 17])
    s = w.schedule
    meta = torch.zeros((inp.num_phys_pages, 2, 2, 128), dtype=torch.bfloat16, device=DEV)
    lens_before = inp.seq_lens - 1
    S.page_meta_update(inp.k_cache, inp.block_table, lens_before, meta)
    k_max = S.budget_bound(inp.lens_host, 16, s.bin_tokens, s.min_pages, s.frac_num, s.frac_den)
    step = S.SparseDecodeStep(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                              meta, inp.min_pages, inp.frac_num, s.frac_den, s.bin_tokens, k_max)
    g = torch.Generator(device=DEV)
    g.manual_seed(seed + 7)
    kn = torch.randn((3, 2, 128), generator=g, device=DEV).to(torch.bfloat16)
    vn = torch.randn((3, 2, 128), generator=g, device=DEV).to(torch.bfloat16)
    return step, kn, vn


def run_layers(layers, stream, whole):
    for step, kn, vn in layers:
        if whole:
            step.decode_step(kn, vn, stream)
        else:
            step.append_score_topk(kn, vn, stream)
            step.attend(stream)


@pytest.mark.parametrize("whole", [False, True])
def test_multi_layer_step_graph_replays_match_eager(whole):
    log(f"case graph replay, 4 layers, whole-step call {whole}")
    # group sizes 4 and 10: the whole-step call selects and attends in one kernel on the
    # first, streams on the second (more than 8 query heads per KV head)
    layers = [make_layer(80 + i, G=4 if i % 2 == 0 else 10) for i in range(4)]
    run_layers(layers, torch.cuda.current_stream().cuda_stream, whole)
    torch.cuda.synchronize()
    eager = [(st.idx.clone(), st.k.clone(), st.out.clone(), st.meta.clone()) for st, _, _ in layers]
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            run_layers(layers, torch.cuda.current_stream().cuda_stream, whole)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for rep in range(3):
        for st, _, _ in layers:          # eager work between replays clobbers the outputs
            st.out.zero_()
            st.idx.fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for li, (st, _, _) in enumerate(layers):
            idx, k, out, meta = eager[li]
            assert torch.equal(st.idx, idx), (rep, li)
            assert torch.equal(st.k, k), (rep, li)
            assert torch.equal(st.out, out), (rep, li)        # deterministic: bit-identical
            assert torch.equal(st.meta.view(torch.int16), meta.view(torch.int16)), (rep, li)
        log(f"  replay {rep} matches the eager step")
