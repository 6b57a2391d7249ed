"""sparrow_sparse_decode_attn_noalloc (the attention entry point that takes its workspace
from the library's own per-GPU buffer) against sparrow_sparse_decode_attn with a caller
workspace, through the C ABI: identical outputs, bit for bit, on two calls in a row - the
second with a smaller batch, so the buffer still holds the first call's partials - and
within the oracle's tolerance.  Also the refusal of a shape whose workspace exceeds the
buffer (checked on the host, nothing launched)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_08446_amd import sparrow as S
from paper_2606_08446_amd import workloads as W

from parity import SCALE, check_out, host, log

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(autouse=True)
def _need_gpu(gpu_device):
    S.load()
    yield


def selection(inp):
    s = inp.workload.schedule
    k_max = S.budget_bound(inp.lens_host, inp.workload.page_size, s.bin_tokens, s.min_pages,
                           s.frac_num, s.frac_den)
    meta = S.new_meta(inp.num_phys_pages, inp.workload.num_kv_heads, DEV)
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta)
    k, idx = S.page_score_topk(inp.q, meta, inp.block_table, inp.seq_lens, inp.k_cache.shape,
                               inp.min_pages, inp.frac_num, s.frac_den, s.bin_tokens, k_max)
    return k, idx, k_max


def both(inp, k, idx, k_max, out_dtype):
    """(with a caller workspace, without) outputs of the same call."""
    shape = S.shape_of(inp.q, inp.k_cache, inp.block_table)
    dt = torch.float32 if out_dtype == S.SPARROW_OUT_F32 else torch.bfloat16
    ws = torch.empty(S.sparrow_workspace_size(shape, k_max, S.SPARROW_OP_SPARSE_ATTN),
                     dtype=torch.uint8, device=DEV)
    ref = torch.full(inp.q.shape, float("nan"), dtype=dt, device=DEV)
    got = torch.full(inp.q.shape, float("nan"), dtype=dt, device=DEV)
    sp = torch.cuda.current_stream().cuda_stream
    args = (shape, inp.q.data_ptr(), inp.k_cache.data_ptr(), inp.v_cache.data_ptr(),
            inp.block_table.data_ptr(), inp.seq_lens.data_ptr(), k.data_ptr(), idx.data_ptr(),
            k_max, SCALE)
    assert S.sparrow_sparse_decode_attn(*args, ref.data_ptr(), out_dtype, ws.data_ptr(),
                                        ws.numel(), sp) == S.SPARROW_OK
    assert S.sparrow_sparse_decode_attn_noalloc(*args, got.data_ptr(), out_dtype,
                                                sp) == S.SPARROW_OK
    torch.cuda.synchronize()
    return ref, got


@pytest.mark.parametrize("out_dtype", [S.SPARROW_OUT_F32, S.SPARROW_OUT_BF16])
def test_noalloc_matches_the_workspace_entry_point(out_dtype):
    # a large first call, then a smaller one: the second runs over the first's partials
    cases = [((9000, 17, 4100, 1, 30000, 2049), W.fraction_budget(1, 6, floor_pages=3), 91),
             ((5000, 700), W.fraction_budget(1, 4), 92)]
    for lengths, sched, seed in cases:
        w = W.small(B=len(lengths), Hq=12, Hkv=3, ps=16, lengths=lengths, seed=seed,
                    schedule=sched)
        log(f"case noalloc {w.name} lengths={lengths} out_dtype={out_dtype}")
        inp = W.generate(w, DEV, lengths=list(lengths))
        k, idx, k_max = selection(inp)
        ref, got = both(inp, k, idx, k_max, out_dtype)
        assert torch.equal(ref.view(torch.int16) if out_dtype else ref.view(torch.int32),
                           got.view(torch.int16) if out_dtype else got.view(torch.int32))
        h = host(inp)
        want = oracle.attention(h["q"], h["k"], h["v"], h["bt"], h["lens"], SCALE,
                                k.cpu().numpy(), idx.cpu().numpy())
        check_out(got.float().cpu().numpy().astype(np.float64), want, "noalloc sparse")


def test_noalloc_full_size_c2_then_c1():
    # the Qwen3-1.7B-shaped batch (64 sequences of 8K-32K tokens), then one sequence
    for w in (W.C2, W.C1):
        log(f"case noalloc {w.name}")
        inp = W.generate(w, DEV)
        k, idx, k_max = selection(inp)
        ref, got = both(inp, k, idx, k_max, S.SPARROW_OUT_F32)
        assert torch.equal(ref.view(torch.int32), got.view(torch.int32))
        del inp
        torch.cuda.empty_cache()


def test_noalloc_refuses_a_workspace_above_the_buffer():
    # 16 query heads per KV head and 8192 sequences: a workspace far above 32 MiB
    shape = S.make_shape(8192, 16, 1, 16, 64, 1 << 20)
    assert S.sparrow_workspace_size(shape, 8, S.SPARROW_OP_SPARSE_ATTN) > \
        S.SPARROW_NOALLOC_SCRATCH_BYTES
    fake = 0x1000
    assert S.sparrow_sparse_decode_attn_noalloc(shape, fake, fake, fake, fake, fake, fake, fake,
                                                8, SCALE, fake, S.SPARROW_OUT_F32,
                                                None) == S.SPARROW_EWORKSPACE
