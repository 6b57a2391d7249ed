"""The tensor-level wrappers refuse, before any launch, a buffer whose dtype, shape, layout or
device differs from what the kernels index (they receive bare pointers through the C ABI and
would read or write such a buffer out of bounds); the same calls with the right buffers run."""
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


@pytest.fixture
def case():
    w = W.small(B=3, Hq=8, Hkv=2, ps=16, lengths=(300, 40, 1000), seed=21,
                schedule=W.fixed_budget(6))
    inp = W.generate(w, DEV, lengths=[300, 40, 1000])
    meta = S.new_meta(inp.num_phys_pages, 2, DEV)
    S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta)
    return w, inp, meta


def refused(fn, what, error=ValueError):
    with pytest.raises(error) as e:
        fn()
    log(f"  refused ({what}): {e.value}")


def test_attention_wrappers_check_their_buffers(case):
    w, inp, meta = case
    log("case wrapper checks: attention")
    k = torch.full((3,), 4, dtype=torch.int32, device=DEV)
    idx = torch.arange(4, dtype=torch.int32, device=DEV).repeat(3, 2, 1).contiguous()
    args = (inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens)
    out_bf16 = torch.empty(inp.q.shape, dtype=torch.bfloat16, device=DEV)
    refused(lambda: S.sparse_decode_attn(*args, k, idx, out=out_bf16), "bf16 out, fp32 asked")
    refused(lambda: S.sparse_decode_attn(*args, k, idx.long()), "int64 page lists")
    refused(lambda: S.sparse_decode_attn(*args, k[:2], idx), "k of 2 sequences")
    refused(lambda: S.sparse_decode_attn(inp.q.float(), *args[1:], k, idx), "fp32 q")
    refused(lambda: S.dense_decode_attn(inp.q, inp.k_cache, inp.v_cache[:-1], inp.block_table,
                                        inp.seq_lens), "v_cache with fewer pages")
    wide = torch.zeros((3, 2 * inp.block_table.shape[1]), dtype=torch.int32, device=DEV)
    refused(lambda: S.dense_decode_attn(inp.q, inp.k_cache, inp.v_cache,
                                        wide[:, ::2], inp.seq_lens), "strided block table")
    refused(lambda: S.dense_decode_attn(inp.q, inp.k_cache, inp.v_cache, inp.block_table,
                                        inp.seq_lens.long()), "int64 lengths")
    refused(lambda: S.dense_decode_attn(inp.q, inp.k_cache, inp.v_cache, inp.block_table,
                                        inp.seq_lens.cpu()), "lengths on the host",
            RuntimeError)
    out = S.sparse_decode_attn(*args, k, idx)
    dense = S.dense_decode_attn(*args)
    torch.cuda.synchronize()
    assert torch.isfinite(out).all() and torch.isfinite(dense).all()


def test_metadata_and_selection_wrappers_check_their_buffers(case):
    w, inp, meta = case
    log("case wrapper checks: metadata, append, selection")
    mean_meta = S.new_meta(inp.num_phys_pages, 2, DEV, landmark=S.SPARROW_LANDMARK_MEAN)
    refused(lambda: S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, mean_meta),
            "mean-landmark buffer for min/max")
    refused(lambda: S.page_meta_update(inp.k_cache, inp.block_table, inp.seq_lens, meta,
                                       first_pos=inp.seq_lens[:1]), "first_pos of 1 sequence")
    kn = torch.zeros((3, 2, 128), dtype=torch.bfloat16, device=DEV)
    refused(lambda: S.append_kv(kn[:, :1], kn, inp.k_cache, inp.v_cache, inp.block_table,
                                inp.seq_lens, meta), "k_new of one head")
    refused(lambda: S.append_kv(kn, kn.float(), inp.k_cache, inp.v_cache, inp.block_table,
                                inp.seq_lens, meta), "fp32 v_new")
    s = w.schedule
    refused(lambda: S.page_score_topk(inp.q, meta, inp.block_table, inp.seq_lens,
                                      tuple(inp.k_cache.shape), inp.min_pages,
                                      torch.zeros(2, dtype=torch.int32, device=DEV),
                                      s.frac_den, s.bin_tokens, 6), "frac_num of another length")
    refused(lambda: S.page_score_topk(inp.q, meta, inp.block_table, inp.seq_lens,
                                      tuple(inp.k_cache.shape), inp.min_pages, inp.frac_num,
                                      s.frac_den, s.bin_tokens, 6,
                                      out_idx=torch.empty((3, 2, 5), dtype=torch.int32,
                                                          device=DEV)), "out_idx of k_max 5")
    step = S.SparseDecodeStep(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                              meta, inp.min_pages, inp.frac_num, s.frac_den, s.bin_tokens, 6)
    stream = torch.cuda.current_stream().cuda_stream
    refused(lambda: step.decode_step(kn, None, stream), "k_new without v_new")
    refused(lambda: step.decode_step(kn.transpose(0, 1).contiguous().transpose(0, 1), kn,
                                     stream), "non-contiguous k_new")
    refused(lambda: step.attend(stream, seq_lens=inp.seq_lens[:2]), "lengths of 2 sequences")
    refused(lambda: S.SparseDecodeStep(inp.q, inp.k_cache, inp.v_cache, inp.block_table,
                                       inp.seq_lens, mean_meta, inp.min_pages, inp.frac_num,
                                       s.frac_den, s.bin_tokens, 6), "step with the wrong meta")
    k, idx = S.page_score_topk(inp.q, meta, inp.block_table, inp.seq_lens,
                               tuple(inp.k_cache.shape), inp.min_pages, inp.frac_num,
                               s.frac_den, s.bin_tokens, 6)
    step.decode_step(None, None, stream)
    torch.cuda.synchronize()
    assert torch.equal(step.k, k) and torch.equal(step.idx, idx)


def test_acceptance_wrappers_check_their_buffers():
    log("case wrapper checks: acceptance rate and tail statistic")
    li = W.generate_logits(W.small_logits(T=5, V=3000, seed=2), DEV)
    refused(lambda: S.acceptance_rate(li.target, li.draft,
                                      alpha=torch.empty(4, device=DEV)), "alpha of 4 tokens")
    lp = torch.zeros((5, 20), device=DEV)
    refused(lambda: S.acceptance_rate_topk(lp, lp[:, :19].contiguous()), "draft list of 19")
    refused(lambda: S.acceptance_rate_topk(lp, lp.double()), "fp64 draft list")
    alpha = S.acceptance_rate(li.target, li.draft)
    refused(lambda: S.tail_stats(alpha, li.positions.long(), 2048, 20), "int64 positions")
    refused(lambda: S.tail_stats(alpha, li.positions[:4], 2048, 20), "positions of 4 tokens")
    q, m, c = S.tail_stats(alpha, li.positions, 2048, 20)
    torch.cuda.synchronize()
    assert int(c.sum()) == 5


def test_empty_batches_launch_nothing():
    """A batch of no sequences (or no tokens) returns at once: torch gives an empty tensor a
    null data pointer, which the C ABI would refuse, and there is nothing to compute."""
    log("case wrapper checks: empty batches")
    q = torch.zeros((0, 4, 128), dtype=torch.bfloat16, device=DEV)
    kc = torch.zeros((5, 2, 16, 128), dtype=torch.bfloat16, device=DEV)
    bt = torch.zeros((0, 3), dtype=torch.int32, device=DEV)
    lens = torch.zeros((0,), dtype=torch.int32, device=DEV)
    meta = S.new_meta(5, 2, DEV)
    S.page_meta_update(kc, bt, lens, meta)
    S.append_kv(torch.zeros((0, 2, 128), dtype=torch.bfloat16, device=DEV),
                torch.zeros((0, 2, 128), dtype=torch.bfloat16, device=DEV), kc, kc.clone(), bt,
                lens, meta)
    tables = torch.ones(1, dtype=torch.int32, device=DEV)
    k, idx = S.page_score_topk(q, meta, bt, lens, tuple(kc.shape), tables, tables.clone(), 1,
                               2048, 4)
    assert k.shape == (0,) and idx.shape == (0, 2, 4)
    assert S.sparse_decode_attn(q, kc, kc, bt, lens, k, idx).shape == (0, 4, 128)
    assert S.dense_decode_attn(q, kc, kc, bt, lens).shape == (0, 4, 128)
    logits = torch.zeros((0, 100), device=DEV)
    assert S.acceptance_rate(logits, logits).shape == (0,)
    assert S.acceptance_rate_topk(torch.zeros((0, 20), device=DEV),
                                  torch.zeros((0, 20), device=DEV)).shape == (0,)
    torch.cuda.synchronize()
