"""GPU parity of the acceptance-rate kernels (Sec. 3.1, Eq. 1) and of the per-bin tail
statistic, through the C ABI, against the CPU oracle.

Tolerance of alpha: 2e-5 absolute.  The kernel works in fp32: per-element exp and the
(tau * logit - LSE) difference carry relative errors of a few 1e-7 (|logits| <= ~30), the
log-sum-exp of a row about 1e-6; each perturbs alpha (a sum of at most 1) by a few 1e-6.
The tail statistic is checked on the GPU's own fp32 alpha on both sides: counts and the
quantile (an order statistic and one fp64 interpolation) bit-exact, the mean to 1e-12
relative (fp64 sums in a different order)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_08446_amd import sparrow as S
from paper_2606_08446_amd import workloads as W

from parity import log

pytestmark = pytest.mark.gpu

DEV = "cuda"
ALPHA_TOL = 2e-5


@pytest.fixture(autouse=True)
def _need_gpu(gpu_device):
    S.load()
    yield


def host_rows(t):
    if t.dtype == torch.bfloat16:
        return W.bf16_bits(t)
    return t.cpu().numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("V,tau", [(3000, 1.0), (3001, 1.0), (4099, 0.7), (1, 1.0), (12, 0.0),
                                   (2999, -0.6), (5000, -1.0)])
def test_acceptance_matches_oracle(dtype, V, tau):
    log(f"case acceptance {dtype} V={V} tau={tau}")
    li = W.generate_logits(W.small_logits(T=37, V=V, seed=3, dtype=dtype), DEV)
    got = S.acceptance_rate(li.target, li.draft, tau)
    torch.cuda.synchronize()
    ref = oracle.acceptance(host_rows(li.target), host_rows(li.draft), tau)
    err = np.abs(got.cpu().numpy().astype(np.float64) - ref)
    log(f"  max abs err {err.max():.2e}")
    assert err.max() <= ALPHA_TOL
    if V == 1 or tau == 0.0:
        np.testing.assert_allclose(got.cpu().numpy(), 1.0, rtol=0, atol=2e-6)


@pytest.mark.parametrize("seed", range(8))
def test_acceptance_random_shapes(seed):
    """Seeded random vocabulary sizes, token counts, temperatures and dtypes, with rows
    that start off a 16-byte boundary on odd seeds."""
    rng = np.random.default_rng(6000 + seed)
    dtype = "bf16" if seed % 4 >= 2 else "f32"
    T = int(rng.integers(1, 40))
    V = int(rng.integers(1, 20000))
    tau = 0.0 if seed == 5 else float(rng.uniform(0.2, 2.0))
    off = int(rng.integers(1, 8 if dtype == "bf16" else 4)) if seed % 2 else 0
    log(f"case acceptance random {seed}: {dtype} T={T} V={V} tau={tau:.3f} offset={off}")
    li = W.generate_logits(W.small_logits(T=T + 1, V=V, seed=60 + seed, dtype=dtype), DEV)
    t = li.target.view(-1)[off:off + T * V].view(T, V)
    d = li.draft.view(-1)[off:off + T * V].view(T, V)
    got = S.acceptance_rate(t, d, tau)
    torch.cuda.synchronize()
    ref = oracle.acceptance(host_rows(t), host_rows(d), tau)
    err = np.abs(got.cpu().numpy().astype(np.float64) - ref)
    log(f"  max abs err {err.max():.2e}")
    assert err.max() <= ALPHA_TOL


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("off", [0, 1])
def test_acceptance_masked_entries(dtype, off):
    # runs of -inf logits (masked vocabulary entries) where every thread's first vector is
    # masked (the first 1024 16-byte vectors), in the scalar head and tail of unaligned rows,
    # a row whose only finite entry is the last, and rows masked differently on the two
    # sides (probability 0 under one distribution only)
    log(f"case acceptance masked {dtype} offset={off}")
    T, V = 6, 13001
    li = W.generate_logits(W.small_logits(T=T + 1, V=V, seed=80, dtype=dtype), DEV)
    t = li.target.view(-1)[off:off + T * V].view(T, V)   # a view: rows keep the offset
    d = li.draft.view(-1)[off:off + T * V].view(T, V)
    per_vec = 4 if dtype == "f32" else 8
    ninf = float("-inf")
    t[0, :1024 * per_vec + 5] = ninf
    d[0, :1024 * per_vec + 5] = ninf
    t[1, :3] = ninf
    d[1, :3] = ninf
    t[1, -7:] = ninf
    d[1, -7:] = ninf
    t[2, :-1] = ninf
    d[2, :-1] = ninf
    t[3, 100:6000] = ninf
    d[4, 2000:9000] = ninf
    t[5, ::2] = ninf
    d[5, ::2] = ninf
    for tau in (1.0, 0.7):
        got = S.acceptance_rate(t, d, tau)
        torch.cuda.synchronize()
        ref = oracle.acceptance(host_rows(t), host_rows(d), tau)
        g = got.cpu().numpy().astype(np.float64)
        assert np.isfinite(g).all(), g
        err = np.abs(g - ref)
        log(f"  tau={tau} max abs err {err.max():.2e}")
        assert err.max() <= ALPHA_TOL
        assert abs(g[2] - 1.0) <= 2e-6     # one finite entry in both rows: alpha = 1


# Vocabulary sizes around the kernel's on-chip boundaries: each thread of the 1024 keeps the
# first 4 16-byte vectors of each row in LDS and the next 12 (fp32) or 10 (bf16) in
# registers between the two passes, and reads the rest again - so rows end just before and
# just after 4096 and 16384 (fp32) or 14336 (bf16) vectors, and well past them.
ONCHIP_V = {"f32": (16383, 16385, 65535, 65537, 80001),
            "bf16": (32767, 32769, 114687, 114689, 130001)}


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("vi", range(5))
@pytest.mark.parametrize("off", [0, 1])
def test_acceptance_around_the_on_chip_boundaries(dtype, vi, off):
    V = ONCHIP_V[dtype][vi]
    log(f"case acceptance on-chip boundary {dtype} V={V} offset={off}")
    T = 4
    li = W.generate_logits(W.small_logits(T=T + 1, V=V, seed=90 + vi, dtype=dtype), DEV)
    t = li.target.view(-1)[off:off + T * V].view(T, V)
    d = li.draft.view(-1)[off:off + T * V].view(T, V)
    per_vec = 4 if dtype == "f32" else 8
    edge = 4096 * per_vec
    t[1, edge - 300:edge + 300] = float("-inf")   # a masked run across the LDS boundary
    t[2, : V * 4 // 5] = float("-inf")             # most of both rows masked
    d[2, : V * 4 // 5] = float("-inf")
    for tau in (1.0, 0.6):
        got = S.acceptance_rate(t, d, tau)
        torch.cuda.synchronize()
        ref = oracle.acceptance(host_rows(t), host_rows(d), tau)
        err = np.abs(got.cpu().numpy().astype(np.float64) - ref)
        log(f"  tau={tau} max abs err {err.max():.2e}")
        assert err.max() <= ALPHA_TOL


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_acceptance_is_deterministic_and_takes_no_tokens(dtype):
    """Two runs give the same bits (fixed reduction order), the rate of a token does not
    depend on the others in the launch, and zero tokens enqueue nothing."""
    log(f"case acceptance determinism {dtype}")
    li = W.generate_logits(W.small_logits(T=9, V=70001, seed=5, dtype=dtype), DEV)
    a = S.acceptance_rate(li.target, li.draft, 0.9)
    b = S.acceptance_rate(li.target, li.draft, 0.9)
    one = S.acceptance_rate(li.target[4:5], li.draft[4:5], 0.9)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    assert torch.equal(a[4:5].view(torch.int32), one.view(torch.int32))
    keep = torch.full((3,), -5.0, device=DEV)
    S.acceptance_rate(li.target[:0], li.draft[:0], 1.0, alpha=keep[:0])
    torch.cuda.synchronize()
    assert (keep == -5.0).all()


def test_acceptance_unaligned_row_starts():
    # views whose rows start off a 16-byte boundary (both rows in the same phase)
    li = W.generate_logits(W.small_logits(T=9, V=2051, seed=4), DEV)
    for off in (1, 2, 3):
        t = li.target.view(-1)[off:off + 8 * 2051].view(8, 2051)
        d = li.draft.view(-1)[off:off + 8 * 2051].view(8, 2051)
        got = S.acceptance_rate(t, d)
        torch.cuda.synchronize()
        ref = oracle.acceptance(t.cpu().numpy(), d.cpu().numpy())
        assert np.abs(got.cpu().numpy() - ref).max() <= ALPHA_TOL, off


def test_acceptance_topk_matches_oracle():
    rng = np.random.default_rng(6)
    T, K = 1000, 20
    lp = np.log(rng.dirichlet(np.ones(K) * 0.3, size=T) * 0.97).astype(np.float32)
    lq = np.log(rng.dirichlet(np.ones(K) * 0.3, size=T) * 0.97).astype(np.float32)
    got = S.acceptance_rate_topk(torch.as_tensor(lp, device=DEV), torch.as_tensor(lq, device=DEV))
    torch.cuda.synchronize()
    ref = oracle.acceptance_topk(lp, lq)
    assert np.abs(got.cpu().numpy() - ref).max() <= 1e-6


def tail_case(alpha, pos, bin_tokens, n_bins, pct):
    a = torch.as_tensor(alpha, device=DEV)
    p = torch.as_tensor(pos, device=DEV)
    q, m, c = S.tail_stats(a, p, bin_tokens, n_bins, pct)
    torch.cuda.synchronize()
    rq, rm, rc = oracle.tail_stats(alpha, pos, bin_tokens, n_bins, pct)
    np.testing.assert_array_equal(c.cpu().numpy(), rc)
    np.testing.assert_array_equal(q.cpu().numpy(), rq)          # NaN == NaN for empty bins
    gm = m.cpu().numpy()
    ok = rc > 0
    np.testing.assert_allclose(gm[ok], rm[ok], rtol=1e-12, atol=0)
    assert np.isnan(gm[~ok]).all()


@pytest.mark.parametrize("pct", [0.0, 5.0, 12.5, 50.0, 100.0])
def test_tail_stats_match_oracle(pct):
    log(f"case tail stats pct={pct}")
    rng = np.random.default_rng(7)
    T = 20000
    alpha = (1.0 - rng.beta(0.3, 4.0, size=T) * 0.7).astype(np.float32)
    alpha[::7] = np.float32(1.0)                     # many exact ties
    alpha[3::11] = np.round(alpha[3::11], 2)
    pos = rng.integers(-100, 50000, size=T).astype(np.int32)   # negatives, past the last bin
    pos[(pos >= 6144) & (pos < 8192)] = 9000                   # bin 3 empty
    tail_case(alpha, pos, 2048, 20, pct)


def test_tail_stats_small_and_degenerate():
    tail_case(np.array([0.25], np.float32), np.array([5], np.int32), 2048, 3, 5.0)
    tail_case(np.array([0.5, 0.5, 0.5, 0.5], np.float32), np.array([0, 1, 2, 3], np.int32),
              2048, 1, 5.0)
    tail_case(np.array([0.0, -0.0, 1.0], np.float32), np.array([0, 1, 2], np.int32), 2048, 1, 50.0)
    tail_case(np.zeros(0, np.float32), np.zeros(0, np.int32), 2048, 4, 5.0)


@pytest.mark.parametrize("cfg", ["a1", "a1-bf16"])
def test_full_size_acceptance_and_tail(cfg):
    lw = W.LOGIT_CONFIGS[cfg]
    log(f"case full-size {lw.name}")
    li = W.generate_logits(lw, DEV)
    alpha = S.acceptance_rate(li.target, li.draft)
    q, m, c = S.tail_stats(alpha, li.positions, lw.bin_tokens, lw.n_bins, 5.0)
    torch.cuda.synchronize()
    a = alpha.cpu().numpy()
    rng = np.random.default_rng(8)
    sample = np.sort(rng.choice(lw.tokens, size=48, replace=False))
    sel = torch.as_tensor(sample, device=DEV)
    ref = oracle.acceptance(host_rows(li.target[sel]), host_rows(li.draft[sel]))
    err = np.abs(a[sample].astype(np.float64) - ref)
    log(f"  sampled alpha max abs err {err.max():.2e}")
    assert err.max() <= ALPHA_TOL
    rq, rm, rc = oracle.tail_stats(a, li.positions.cpu().numpy(), lw.bin_tokens, lw.n_bins, 5.0)
    np.testing.assert_array_equal(c.cpu().numpy(), rc)
    np.testing.assert_array_equal(q.cpu().numpy(), rq)
    np.testing.assert_allclose(m.cpu().numpy(), rm, rtol=1e-12)
    log(f"  5-percentile per bin: {np.round(rq, 4).tolist()}")
    del li
    torch.cuda.empty_cache()
