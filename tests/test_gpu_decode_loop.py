"""A generation loop on the GPU: per-sequence cache lengths, one token appended per
step with its block representative maintained incrementally (phsa_cache_append),
and a decode step at every length (phsa_decode_varlen), checked against the oracle.

Cache slots past each sequence's length hold NaN, so any read of them would show."""
import numpy as np
import pytest
import torch

import oracle
from paper_2601_02819_amd import phsa
from tests.gpu_common import O_TOL, check_sel, log, to_np

pytestmark = pytest.mark.gpu

M, D, HQ, HKV = 64, 128, 4, 2


def _nan_tail(x, lens):
    for b, n in enumerate(lens):
        x[b, n:] = float("nan")
    return x


def _check_step(q, kcache, vcache, pcache, kc, clen, sel, o, lse, cfg, step):
    scale = D ** -0.5
    kh, vh = kcache.float().cpu().numpy(), vcache.float().cpu().numpy()
    ph, qh, kc_g = pcache.cpu().numpy(), q.float().cpu().numpy(), kc.cpu().numpy()
    sel_g, o_g, lse_g = sel.cpu().numpy(), to_np(o), lse.cpu().numpy()
    for b, n in enumerate(clen.cpu().tolist()):
        full = n // M                           # complete blocks: maintained representatives
        if full:
            ref = oracle.compress(kh[b:b + 1, :full * M], ph[b:b + 1, :full * M], M, cfg.lam)
            np.testing.assert_allclose(kc_g[b:b + 1, :, :full], ref, atol=1e-5, rtol=1e-5)
        pad = -(-n // M) * M
        kpad = oracle.compress(np.nan_to_num(kh[b:b + 1, :pad]), ph[b:b + 1, :pad], M, cfg.lam)
        if full:
            kpad[:, :, :full] = oracle.compress(kh[b:b + 1, :full * M], ph[b:b + 1, :full * M], M, cfg.lam)
        ref_sel, kth, gap = oracle.select(qh[b:b + 1], kpad, M, cfg.top_k, cfg.n_init_blocks, cfg.window, scale, pad,
                                          q_pos0=n - 1)
        check_sel(sel_g[b:b + 1], ref_sel, kth, gap,
                  lambda idx: oracle.score_row(qh[b:b + 1], kpad, M, scale, pad, 0, 0, idx[1]))
        o_r, lse_r = oracle.attn_fwd(qh[b:b + 1], kh[b:b + 1, :pad], vh[b:b + 1, :pad], sel_g[b:b + 1], M, scale,
                                     q_pos0=n - 1)
        np.testing.assert_allclose(o_g[b:b + 1], o_r, atol=O_TOL["bf16"], rtol=0)
        np.testing.assert_allclose(lse_g[b:b + 1], lse_r, atol=O_TOL["bf16"], rtol=0)
    log(f"[decode-loop] step {step}: lengths {clen.cpu().tolist()} checked")


def test_generation_loop_with_block_cache():
    cap = 2048
    prefix = [1, 63, 64, 65, 700, cap - 3]      # one sequence fills its cache during the loop
    B = len(prefix)
    cfg = phsa.Config(block_size=M, top_k=6, n_init_blocks=1, window=64)
    g = torch.Generator().manual_seed(31)
    kcache = _nan_tail(torch.randn(B, cap, HKV, D, generator=g), prefix).to(torch.bfloat16).cuda()
    vcache = _nan_tail(torch.randn(B, cap, HKV, D, generator=g), prefix).to(torch.bfloat16).cuda()
    pcache = (torch.rand(B, cap, generator=g) < 0.1).to(torch.uint8).cuda()
    clen = torch.tensor(prefix, dtype=torch.int32).cuda()
    # representatives of the prefilled prefixes (blocks holding NaN slots are never scored)
    kc = phsa.compress(kcache, pcache, cfg)
    steps = 70
    for step in range(steps):
        kn = torch.randn(B, HKV, D, generator=g).to(torch.bfloat16).cuda()
        vn = torch.randn(B, HKV, D, generator=g).to(torch.bfloat16).cuda()
        pn = (torch.rand(B, generator=g) < 0.15).to(torch.uint8).cuda()
        q = (torch.randn(B, 1, HQ, D, generator=g) * 0.3).to(torch.bfloat16).cuda()
        phsa.cache_append(kn, vn, pn, kcache, vcache, pcache, clen, kc, cfg)
        sel, o, lse = phsa.decode_varlen(q, kcache, vcache, kc, clen, cfg)
        if step in (0, 1, 2, 3, steps - 1):
            torch.cuda.synchronize()
            assert clen.cpu().tolist() == [min(n + step + 1, cap) for n in prefix]
            _check_step(q, kcache, vcache, pcache, kc, clen, sel, o, lse, cfg, step)


def test_decode_varlen_uniform_equals_decode():
    """All lengths equal to the capacity: phsa_decode_varlen is phsa_decode, bit for bit."""
    B, cap = 4, 4096
    cfg = phsa.Config(block_size=M, top_k=12, n_init_blocks=1, window=0)
    g = torch.Generator().manual_seed(32)
    k = torch.randn(B, cap, HKV, D, generator=g).to(torch.bfloat16).cuda()
    v = torch.randn(B, cap, HKV, D, generator=g).to(torch.bfloat16).cuda()
    p = (torch.rand(B, cap, generator=g) < 0.08).to(torch.uint8).cuda()
    q = torch.randn(B, 1, HQ, D, generator=g).to(torch.bfloat16).cuda()
    kc = phsa.compress(k, p, cfg)
    a = phsa.decode(q, k, v, kc, cfg)
    b = phsa.decode_varlen(q, k, v, kc, torch.full((B,), cap, dtype=torch.int32).cuda(), cfg)
    for x, y in zip(a, b):
        assert torch.equal(x, y)
