"""The scratch-free selection entry point (phsa_select_noalloc) called through
the C ABI, against phsa_select with a caller's workspace on the same inputs:
the selected block indices must be identical (integer work, bit-exact).  Two
calls in a row share the library's fixed scratch, the second with a smaller
problem, so stale contents of the first call must not leak into the second."""
import dataclasses

import numpy as np
import pytest
import torch

from paper_2601_02819_amd import phsa
from paper_2601_02819_amd.inputs import WORKLOADS, make_inputs

pytestmark = pytest.mark.gpu


def _cfg(wl, softmax_sum=False):
    return phsa.Config(block_size=wl.block_size, top_k=wl.top_k, n_init_blocks=wl.n_init_blocks, window=wl.window,
                       lam=wl.lam, softmax_sum=softmax_sum)


def _compare(wl, seed, softmax_sum=False):
    print(f"[noalloc] {wl.name} B{wl.batch} L{wl.seqlen_q} m{wl.block_size} softmax_sum={softmax_sum}", flush=True)
    host = make_inputs(wl, seed, with_grad_out=False)
    q, k, punct = host["q"].cuda(), host["k"].cuda(), host["punct"].cuda()
    cfg = _cfg(wl, softmax_sum)
    kc = phsa.compress(k, punct, cfg)
    p = phsa.make_params(cfg, wl.batch, wl.seqlen_q, wl.seqlen_k, wl.n_heads_q, wl.n_heads_kv, wl.head_dim,
                         q.dtype)
    need = phsa.workspace_size(p, phsa.OP_SELECT)
    assert 0 < need <= phsa.NOALLOC_SCRATCH_BYTES
    ref = phsa.select(q, kc, wl.seqlen_k, cfg)
    out = torch.full_like(ref, -7)
    got = phsa.select_noalloc(q, kc, wl.seqlen_k, cfg, sel=out)
    torch.cuda.synchronize()
    assert got.data_ptr() == out.data_ptr()
    np.testing.assert_array_equal(got.cpu().numpy(), ref.cpu().numpy())
    return need


def test_noalloc_matches_select_two_calls():
    # first call: the paper's geometry at 4 x 32k (2048 blocks per sequence, 33.8 MB of scratch)
    n1 = _compare(WORKLOADS["train_32k_paper"], 0)
    # second call: a smaller problem (64-token blocks, 8k tokens, 0.5 MB) over the same scratch
    n2 = _compare(WORKLOADS["prefill_8k"], 1)
    assert n2 < n1
    # and a third, smaller still, in the softmax-sum mode, which scores with the same split copies
    _compare(dataclasses.replace(WORKLOADS["prefill_8k"], name="prefill_2k", seqlen_q=2048, seqlen_k=2048), 2,
             softmax_sum=True)


def test_noalloc_rejects_oversized_problem():
    wl = dataclasses.replace(WORKLOADS["prefill_32k"], batch=64)   # 64 x 8 x 512 blocks: 135 MB of scratch
    q = torch.zeros(1, dtype=torch.bfloat16, device="cuda")
    p = phsa.make_params(_cfg(wl), wl.batch, wl.seqlen_q, wl.seqlen_k, wl.n_heads_q, wl.n_heads_kv, wl.head_dim,
                         torch.bfloat16)
    import ctypes
    st = phsa.lib().phsa_select_noalloc(ctypes.byref(p), ctypes.c_void_p(q.data_ptr()),
                                        ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(q.data_ptr()), None)
    assert st == phsa.ERR_SCRATCH_LIMIT
