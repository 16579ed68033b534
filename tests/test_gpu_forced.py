"""The forced blocks of Algorithm 1 (the init blocks and the local window) go
to the band kernels for every row whose selection holds all of them, when the
window spans at least one 64-key tile; without a window they stay in the sparse
kernels.  These tests hand the attention a selection that mixes such rows with
rows missing one init block or one local block (all their blocks stay in the
sparse kernels) and rows inside the init blocks, and check forward and
backward against the oracle.  The shapes cover several init tiles, init blocks
ending inside a 64-key tile (whose later keys are the windows of early rows),
init tiles whose rows are split over several segments (sequences of 2048 and
4096 tokens), and window 0 (all sparse)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2601_02819_amd import phsa
from tests.gpu_common import GRAD_REL_L2, O_TOL, log, rel_l2, to_np

pytestmark = pytest.mark.gpu


def mixed_selection(B, Hkv, L, m, n_init, window, top_k, ks, seed, drop_all=False):
    """Ascending causal block lists: forced blocks plus up to top_k random picks;
    every fourth row (from row 1) drops one init block and every fourth (from
    row 3) one local block, when the row keeps another block.  drop_all: every
    row that keeps another block drops one of its forced blocks."""
    rng = np.random.default_rng(seed)
    sel = -np.ones((B, Hkv, L, ks), np.int32)
    dropped = [0, 0]
    for b in range(B):
        for g in range(Hkv):
            for i in range(L):
                cur = i // m
                ninit = min(n_init, cur + 1)
                a = max(max(0, cur - window // m), ninit)
                row = set(range(ninit)) | set(range(a, cur + 1))
                free = np.arange(ninit, a)
                if free.size and i % 7 != 5:
                    row |= set(rng.choice(free, size=min(top_k, free.size), replace=False).tolist())
                if (drop_all or i % 4 == 1) and ninit >= 1 and len(row) > 1:
                    row.discard(int(rng.integers(0, ninit)))
                    dropped[0] += 1
                elif (drop_all or i % 4 == 3) and cur >= a and len(row) > 1:
                    row.discard(int(rng.integers(a, cur + 1)))
                    dropped[1] += 1
                row = sorted(row)
                assert 1 <= len(row) <= ks
                sel[b, g, i, :len(row)] = row
    return sel, dropped


@pytest.mark.parametrize("m,n_init,window,top_k,L,G", [
    (64, 1, 64, 6, 2048, 2),     # one init tile, a one-block window
    (64, 3, 128, 4, 2048, 4),    # three init tiles
    (16, 2, 64, 8, 2048, 2),     # init keys end inside tile 0, whose later keys are windows of early rows
    (32, 5, 64, 6, 1024, 1),     # init ends at key 160 (tile 2), window of two blocks
    (64, 2, 128, 5, 4096, 2),    # four row segments per init tile
    (64, 1, 0, 6, 2048, 2),      # window 0 (the 4 x 32k training geometry, small): all sparse
])
def test_forced_blocks_mixed_rows(m, n_init, window, top_k, L, G):
    B, Hkv, d = 2, 2, 128
    Hq = G * Hkv
    cfg = phsa.Config(block_size=m, top_k=top_k, n_init_blocks=n_init, window=window)
    ks = cfg.ksel
    log(f"[forced] m={m} init={n_init} w={window} k={top_k} L={L} G={G}")
    gen = torch.Generator().manual_seed(41)
    q = torch.randn(B, L, Hq, d, generator=gen).to(torch.bfloat16)
    k = torch.randn(B, L, Hkv, d, generator=gen).to(torch.bfloat16)
    v = torch.randn(B, L, Hkv, d, generator=gen).to(torch.bfloat16)
    do = torch.randn(B, L, Hq, d, generator=gen).to(torch.bfloat16)
    sel, dropped = mixed_selection(B, Hkv, L, m, n_init, window, top_k, ks, 7)
    assert min(dropped) > L // 16, dropped
    sel_t = torch.from_numpy(sel).cuda()
    o, lse = phsa.attn_fwd(q.cuda(), k.cuda(), v.cuda(), sel_t, cfg)
    dq, dk, dv = phsa.attn_bwd(q.cuda(), k.cuda(), v.cuda(), o, do.cuda(), lse, sel_t, cfg)
    torch.cuda.synchronize()
    log(f"[forced] m={m}: GPU done, oracle next")
    qh, kh, vh, doh = (x.float().numpy() for x in (q, k, v, do))
    scale = d ** -0.5
    o_r, lse_r = oracle.attn_fwd(qh, kh, vh, sel, m, scale)
    np.testing.assert_allclose(to_np(o), o_r, atol=O_TOL["bf16"], rtol=0)
    np.testing.assert_allclose(to_np(lse), lse_r, atol=O_TOL["bf16"], rtol=0)
    dq_r, dk_r, dv_r = oracle.attn_bwd(qh, kh, vh, doh, sel, m, scale)
    errs = (rel_l2(to_np(dq), dq_r), rel_l2(to_np(dk), dk_r), rel_l2(to_np(dv), dv_r))
    log(f"[forced] m={m} init={n_init} w={window}: grad rel-L2 {errs}")
    assert max(errs) < GRAD_REL_L2["bf16"], errs
    # the init keys, where every row's gradient meets: dK and dV of the first
    # 64 keys on their own
    ni = min(64, n_init * m)
    e0 = (rel_l2(to_np(dk)[:, :ni], dk_r[:, :ni]), rel_l2(to_np(dv)[:, :ni], dv_r[:, :ni]))
    assert max(e0) < GRAD_REL_L2["bf16"], e0


def test_forced_blocks_no_band_rows():
    """Every row that can lose a forced block does: apart from the first
    tokens (a single block), no row is in the band, so most workgroups of the
    band forward attend to no tile and only merge their rows' sparse
    partials."""
    B, Hkv, d, G, L, m = 2, 2, 128, 2, 2048, 64
    Hq = G * Hkv
    cfg = phsa.Config(block_size=m, top_k=6, n_init_blocks=1, window=128)
    log(f"[forced] no band rows: L={L}")
    gen = torch.Generator().manual_seed(43)
    q = torch.randn(B, L, Hq, d, generator=gen).to(torch.bfloat16)
    k = torch.randn(B, L, Hkv, d, generator=gen).to(torch.bfloat16)
    v = torch.randn(B, L, Hkv, d, generator=gen).to(torch.bfloat16)
    do = torch.randn(B, L, Hq, d, generator=gen).to(torch.bfloat16)
    sel, dropped = mixed_selection(B, Hkv, L, m, 1, 128, 6, cfg.ksel, 9, drop_all=True)
    assert dropped[0] > L, dropped
    sel_t = torch.from_numpy(sel).cuda()
    o, lse = phsa.attn_fwd(q.cuda(), k.cuda(), v.cuda(), sel_t, cfg)
    dq, dk, dv = phsa.attn_bwd(q.cuda(), k.cuda(), v.cuda(), o, do.cuda(), lse, sel_t, cfg)
    torch.cuda.synchronize()
    qh, kh, vh, doh = (x.float().numpy() for x in (q, k, v, do))
    o_r, lse_r = oracle.attn_fwd(qh, kh, vh, sel, m, d ** -0.5)
    np.testing.assert_allclose(to_np(o), o_r, atol=O_TOL["bf16"], rtol=0)
    np.testing.assert_allclose(to_np(lse), lse_r, atol=O_TOL["bf16"], rtol=0)
    dq_r, dk_r, dv_r = oracle.attn_bwd(qh, kh, vh, doh, sel, m, d ** -0.5)
    errs = (rel_l2(to_np(dq), dq_r), rel_l2(to_np(dk), dk_r), rel_l2(to_np(dv), dv_r))
    log(f"[forced] no band rows: grad rel-L2 {errs}")
    assert max(errs) < GRAD_REL_L2["bf16"], errs
