"""Shared helpers for the GPU parity tests (compare the HIP path with the oracle)."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2601_02819_amd import phsa
from paper_2601_02819_amd.inputs import Workload, make_inputs

SEL_GAP_TOL = 1e-4      # rows whose k-th / (k+1)-th oracle score gap is below this are exempt
O_TOL = {"bf16": 2e-2, "fp32": 1e-4}
GRAD_REL_L2 = {"bf16": 5e-2, "fp32": 1e-4}


def log(msg: str) -> None:
    print(msg, flush=True)


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy()


def cfg_of(wl: Workload) -> phsa.Config:
    return phsa.Config(block_size=wl.block_size, top_k=wl.top_k, n_init_blocks=wl.n_init_blocks,
                       window=wl.window, lam=wl.lam)


def device_inputs(wl: Workload, seed: int = 0, with_grad_out=None):
    host = make_inputs(wl, seed, with_grad_out=with_grad_out)
    dev = {k: v.cuda() for k, v in host.items()}
    return host, dev


def rel_l2(a: np.ndarray, b: np.ndarray) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


def check_sel(gpu, ref, kth, gap, score_fn, tol=SEL_GAP_TOL):
    """Index parity: rows must be equal, except rows whose oracle top-k boundary gap is
    below tol, where every block in the symmetric difference must score within tol of
    the oracle's k-th score.  Returns the number of exempt rows."""
    gpu = np.asarray(gpu)
    ref = np.asarray(ref)
    bad = np.nonzero((gpu != ref).any(-1))
    exempt = 0
    for idx in zip(*bad):
        a = set(int(x) for x in gpu[idx] if x >= 0)
        b = set(int(x) for x in ref[idx] if x >= 0)
        assert gap[idx] < tol, f"row {idx}: gpu {sorted(a)} oracle {sorted(b)} gap {gap[idx]}"
        sc = score_fn(idx)
        for t in a ^ b:
            assert abs(sc[t] - kth[idx]) < tol, f"row {idx}: block {t} score {sc[t]} vs k-th {kth[idx]}"
        assert len(a) == len(b), f"row {idx}: set sizes differ"
        exempt += 1
    return exempt


def oracle_inputs(host):
    return {k: (v.float().numpy() if v.dtype != torch.uint8 else v.numpy()) for k, v in host.items()}
