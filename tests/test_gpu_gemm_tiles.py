"""GPU checks of the bf16 GEMM kernel's tile forms through the C ABI
(dlm_debug_gemm): every tile configuration, with whole tiles, against the
fp64 product of the same bf16 operands (plain store, residual add and the
SwiGLU epilogue, the feed-forward of "Background and Challenges", Diffusion
Language Models), its K-split slices against the fp64 partial products, and,
for every last-round sub-tile split a configuration allows, bit for bit
against its whole-tile launch (sub-tiles accumulate each output element over
the same k order). Shapes span several tiles with ragged row and column
tails."""
import numpy as np
import pytest
import torch

import oracle
from kernel_checks import U, gemm_tol, half_ulp
from paper_2606_29094_amd import dlm

pytestmark = pytest.mark.gpu


def _configs():
    out = []
    for cfg in range(128):
        info = dlm.debug_gemm_info(cfg)
        if info is not None:
            out.append((cfg,) + info)
    return out


def _operands(gpu, M, N, K, seed):
    g = torch.Generator().manual_seed(seed)
    a = (torch.randn(M, K, generator=g) * 0.5).to(torch.bfloat16)
    b = (torch.randn(N, K, generator=g) * 0.05).to(torch.bfloat16)
    return a, b, a.to(gpu), b.to(gpu)


def _shape(bm, bn, K=320):
    # two and a bit row tiles, three column tiles plus a 64-wide ragged one
    return 2 * bm + 37, 3 * bn + 64, K


def _run(gpu, cfg, epi, a_d, b_d, c0, sub=0, n_tail=0, group_m=0):
    c = c0.clone()
    dlm.debug_gemm(cfg, epi, a_d, b_d, c, sub=sub, n_tail=n_tail, group_m=group_m)
    torch.cuda.synchronize()
    return c


def test_configurations_exist(gpu):
    cfgs = _configs()
    assert len(cfgs) >= 8
    assert any(s & 4 for _, _, _, s in cfgs) and any(s & 2 for _, _, _, s in cfgs)
    assert any(s & 8 for _, _, _, s in cfgs)


@pytest.mark.parametrize("cfg,bm,bn,subs", _configs(), ids=lambda v: str(v))
def test_whole_tiles_match_fp64_product(gpu, cfg, bm, bn, subs):
    M, N, K = _shape(bm, bn)
    a, b, a_d, b_d = _operands(gpu, M, N, K, seed=cfg)
    A = a.double().numpy()
    B = b.double().numpy()
    P = A @ B.T
    tol = gemm_tol(A, B, 1, "bf16")
    # plain store
    c = _run(gpu, cfg, 0, a_d, b_d, torch.zeros(M, N, device=gpu)).cpu().double().numpy()
    assert np.all(np.abs(c - P) <= tol), (cfg, float(np.max(np.abs(c - P) - tol)))
    # residual add: c0 + P with one more rounding of the sum
    c0 = torch.randn(M, N, generator=torch.Generator().manual_seed(7))
    c = _run(gpu, cfg, 2, a_d, b_d, c0.to(gpu)).cpu().double().numpy()
    ref = c0.double().numpy() + P
    assert np.all(np.abs(c - ref) <= tol + U * np.abs(ref)), cfg
    # SwiGLU: silu(gate) * up, rounded to bf16 (configurations whose wave
    # tiles hold an odd number of column fragments reject it)
    F = N // 2
    if subs & 8:
        with pytest.raises(dlm.DlmError):
            _run(gpu, cfg, 1, a_d, b_d, torch.zeros(M, F, dtype=torch.bfloat16, device=gpu))
        return
    y = _run(gpu, cfg, 1, a_d, b_d, torch.zeros(M, F, dtype=torch.bfloat16, device=gpu))
    y = y.cpu().double().numpy()
    g, u = P[:, :F], P[:, F:]
    ref = oracle.silu(g) * u
    # fp32 value before the bf16 store: the errors of g and u through
    # silu(g) * u (|d silu| <= 1.1), plus the exp, the hardware reciprocal and
    # two products (a few ulp of fp32); then the bf16 rounding of that value
    slack = 1.1 * tol[:, :F] * np.abs(u) + np.abs(oracle.silu(g)) * tol[:, F:] \
        + tol[:, :F] * tol[:, F:] + 8 * U * np.abs(ref)
    err = half_ulp(np.abs(ref) + slack, "bf16") + slack
    assert np.all(np.abs(y - ref) <= err), (cfg, float(np.max(np.abs(y - ref) / err)))


@pytest.mark.parametrize("cfg,bm,bn,subs", _configs(), ids=lambda v: str(v))
def test_k_slices_match_fp64_partial_products(gpu, cfg, bm, bn, subs):
    """K-split launches (the plain fp32 store of one slice per K range, which
    the RoPE kernel or the residual norm sums): every slice against the fp64
    product over its own k range, for 2, 4 and 8 slices of 8 k-tiles, in both
    tile orders; slices start as NaN, so an unwritten element fails."""
    M, N, K = _shape(bm, bn, K=512)
    a, b, a_d, b_d = _operands(gpu, M, N, K, seed=200 + cfg)
    A = a.double().numpy()
    B = b.double().numpy()
    for s in (2, 4, 8):
        w = K // s
        parts = [A[:, z * w:(z + 1) * w] @ B[:, z * w:(z + 1) * w].T for z in range(s)]
        tols = [gemm_tol(A[:, z * w:(z + 1) * w], B[:, z * w:(z + 1) * w], 1, "bf16")
                for z in range(s)]
        for group_m in (0, 2):
            c = torch.full((s, M, N), float("nan"), device=gpu)
            dlm.debug_gemm(cfg, 0, a_d, b_d, c, group_m=group_m, splits=s)
            torch.cuda.synchronize()
            c = c.cpu().double().numpy()
            for z in range(s):
                assert np.all(np.abs(c[z] - parts[z]) <= tols[z]), (cfg, s, group_m, z)


def _split_cases():
    out = []
    for cfg, bm, bn, subs in _configs():
        for sub in (2, 4):
            if subs & sub:
                out.append((cfg, bm, bn, sub, subs))
    return out


@pytest.mark.parametrize("cfg,bm,bn,sub,subs", _split_cases(), ids=lambda v: str(v))
def test_sub_tiles_equal_whole_tiles_bitwise(gpu, cfg, bm, bn, sub, subs):
    M, N, K = _shape(bm, bn)
    tiles = -(-M // bm) * -(-N // bn)
    a, b, a_d, b_d = _operands(gpu, M, N, K, seed=100 + cfg)
    c0 = torch.randn(M, N, generator=torch.Generator().manual_seed(8)).to(gpu)
    epis = [(0, torch.zeros(M, N, device=gpu)), (2, c0)]
    if not subs & 8:
        epis.append((1, torch.zeros(M, N // 2, dtype=torch.bfloat16, device=gpu)))
    for epi, init in epis:
        for group_m in (0, 2):
            whole = _run(gpu, cfg, epi, a_d, b_d, init, group_m=group_m)
            for n_tail in (1, 3, tiles):
                split = _run(gpu, cfg, epi, a_d, b_d, init, sub=sub, n_tail=n_tail,
                             group_m=group_m)
                assert torch.equal(whole, split), (cfg, sub, epi, group_m, n_tail)


def test_rejects_invalid_launches(gpu):
    a = torch.zeros(64, 128, dtype=torch.bfloat16, device=gpu)
    b = torch.zeros(96, 128, dtype=torch.bfloat16, device=gpu)
    c = torch.zeros(64, 96, device=gpu)
    cfgs = _configs()
    no_quarter = [cfg for cfg, _, _, s in cfgs if not s & 4]
    with pytest.raises(dlm.DlmError):
        dlm.debug_gemm(999, 0, a, b, c)
    if no_quarter:
        with pytest.raises(dlm.DlmError):
            dlm.debug_gemm(no_quarter[0], 0, a, b, c, sub=4, n_tail=1)
    quarter = [cfg for cfg, _, _, s in cfgs if s & 4][0]
    with pytest.raises(dlm.DlmError):
        dlm.debug_gemm(quarter, 0, a, b, c, sub=4, n_tail=10 ** 6)
    with pytest.raises(dlm.DlmError):
        dlm.debug_gemm(quarter, 0, a[:, :100].contiguous(), b[:, :100].contiguous(), c)
    with pytest.raises(dlm.DlmError):    # SwiGLU width 40 is not a multiple of 16
        dlm.debug_gemm(quarter, 1, a, b[:80].contiguous(), torch.zeros(64, 40, dtype=torch.bfloat16,
                                                                       device=gpu))
