"""The C ABI without a GPU: the library loads, exports every symbol the header
declares, and rejects bad arguments on the host before anything is launched."""
import ctypes
import os
import re
import subprocess

import pytest
import torch

from paper_2601_02819_amd import phsa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "phsa.h")
PROF_HEADER = os.path.join(ROOT, "include", "phsa_prof.h")


def declared_functions(header=HEADER):
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(phsa_[a-z_]+)\s*\(", text)))


def exported_c_functions(path):
    """Unmangled function symbols in the dynamic symbol table of a library."""
    out = subprocess.run(["nm", "-D", "--defined-only", path], capture_output=True, text=True, check=True).stdout
    return sorted({f[2] for f in (ln.split() for ln in out.splitlines()) if len(f) == 3 and f[1] == "T"
                   and not f[2].startswith("_")})


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(phsa.EXPORTS)
    assert declared_functions(PROF_HEADER) == sorted(phsa.PROF_EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(phsa.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_library_exports_only_the_c_abi():
    """libphsa.so exports exactly the calls of phsa.h (no profiling or timing
    calls); the profiling build adds those of phsa_prof.h and nothing else."""
    assert exported_c_functions(phsa.LIB_PATH) == declared_functions()
    assert exported_c_functions(phsa.PROF_LIB_PATH) == sorted(declared_functions() + declared_functions(PROF_HEADER))


# The one exception: phsa_select_noalloc's static device scratch (its host-side
# stand-in) and the per-GPU table of its device address, set once per GPU.
NOALLOC_STATE = {"phsa::(anonymous namespace)::scratch", "phsa::(anonymous namespace)::g_scratch_ptr",
                 "phsa::(anonymous namespace)::g_scratch_mu"}


def test_library_keeps_no_mutable_state():
    """Every writable data symbol of the library's own namespace is a kernel
    handle that the HIP runtime fills in when it registers the code object, or
    the scratch-free entry point's fixed scratch: the ABI layer holds no other
    namespace-scope state, so calls are reentrant."""
    out = subprocess.run(["nm", "-C", phsa.LIB_PATH], capture_output=True, text=True, check=True).stdout
    data = [ln.split(" ", 2)[2] for ln in out.splitlines() if re.match(r"^[0-9a-f]+ [bBdD] ", ln)]
    ours = [n for n in data if n.startswith("phsa::")]
    assert ours, "expected the kernel handles"
    other = [n for n in ours if not re.match(r"phsa::\w+_kernel[<(]", n)]
    assert set(other) == NOALLOC_STATE, other


def _p(**kw):
    base = dict(batch=1, seqlen_q=1024, seqlen_k=1024, n_heads_q=2, n_heads_kv=1, head_dim=64, block_size=64,
                top_k=2, n_init_blocks=1, window=0, lam=0.5, softmax_scale=0.0, dtype=phsa.BF16, flags=0)
    base.update(kw)
    return phsa.Params(*[base[f] for f, _ in phsa.Params._fields_])


@pytest.mark.parametrize("kw,op,code", [
    ({}, phsa.OP_ATTN_FWD, phsa.OK),
    ({"dtype": phsa.FP32}, phsa.OP_ATTN_BWD, phsa.OK),
    ({"dtype": 7}, phsa.OP_COMPRESS, phsa.ERR_DTYPE),
    ({"seqlen_k": 1000}, phsa.OP_COMPRESS, phsa.ERR_SHAPE),             # Lk % m != 0
    ({"n_heads_q": 3, "n_heads_kv": 2}, phsa.OP_SELECT, phsa.ERR_SHAPE),  # Hq % Hkv != 0
    ({"seqlen_q": 2048}, phsa.OP_SELECT, phsa.ERR_SHAPE),               # Lq > Lk
    ({"batch": 0}, phsa.OP_SELECT, phsa.ERR_SHAPE),
    ({"window": 10}, phsa.OP_SELECT, phsa.ERR_INVALID_ARG),             # w % m != 0
    ({"top_k": -1}, phsa.OP_SELECT, phsa.ERR_INVALID_ARG),
    ({"lam": 1.5}, phsa.OP_COMPRESS, phsa.ERR_INVALID_ARG),
    ({"lam": float("nan")}, phsa.OP_COMPRESS, phsa.ERR_INVALID_ARG),
    ({"softmax_scale": float("inf")}, phsa.OP_SELECT, phsa.ERR_INVALID_ARG),
    ({"head_dim": 96}, phsa.OP_SELECT, phsa.ERR_UNSUPPORTED),
    ({"top_k": 40}, phsa.OP_SELECT, phsa.ERR_UNSUPPORTED),
    ({"block_size": 8}, phsa.OP_ATTN_FWD, phsa.ERR_UNSUPPORTED),
    ({"block_size": 32}, phsa.OP_ATTN_FWD, phsa.OK),
    ({"block_size": 16, "n_init_blocks": 8, "window": 512, "top_k": 16}, phsa.OP_ATTN_BWD, phsa.OK),
    ({"block_size": 16, "seqlen_k": 1040, "seqlen_q": 1040}, phsa.OP_ATTN_FWD, phsa.ERR_UNSUPPORTED),  # Lk % 64
    ({"block_size": 16, "seqlen_k": 1040, "seqlen_q": 1040, "dtype": phsa.FP32}, phsa.OP_ATTN_FWD, phsa.OK),
    ({"block_size": 16, "seqlen_k": 1040, "seqlen_q": 1}, phsa.OP_DECODE, phsa.OK),
    ({"block_size": 32}, phsa.OP_SELECT, phsa.OK),
    ({"n_heads_q": 6, "n_heads_kv": 2}, phsa.OP_ATTN_FWD, phsa.ERR_UNSUPPORTED),   # G = 3
    ({"seqlen_q": 2}, phsa.OP_DECODE, phsa.ERR_SHAPE),
    ({"seqlen_q": 1}, phsa.OP_DECODE, phsa.OK),
    ({}, 17, phsa.ERR_INVALID_ARG),
    ({"flags": phsa.FLAG_REUSE_INDEX}, phsa.OP_ATTN_BWD, phsa.OK),
    ({"flags": 4}, phsa.OP_ATTN_BWD, phsa.ERR_INVALID_ARG),                 # unknown flag bit
    ({"flags": phsa.FLAG_SELECT_SOFTMAX_SUM}, phsa.OP_SELECT, phsa.OK),
    ({"flags": phsa.FLAG_SELECT_SOFTMAX_SUM}, phsa.OP_DECODE, phsa.ERR_SHAPE),   # still needs Lq = 1
    ({"n_heads_q": 6, "n_heads_kv": 2}, phsa.OP_SELECT, phsa.OK),                # G = 3, summed logits
    ({"n_heads_q": 6, "n_heads_kv": 2, "flags": phsa.FLAG_SELECT_SOFTMAX_SUM}, phsa.OP_SELECT,
     phsa.ERR_UNSUPPORTED),                                                      # G = 3, softmax sum
    ({"batch": 40000, "n_heads_q": 2, "n_heads_kv": 2}, phsa.OP_SELECT, phsa.ERR_UNSUPPORTED),  # B * Hkv > 65535
])
def test_validate(kw, op, code):
    assert phsa.lib().phsa_validate(ctypes.byref(_p(**kw)), op) == code


def test_ksel_and_workspace():
    L = phsa.lib()
    p = _p(n_init_blocks=2, window=128, top_k=5)
    assert L.phsa_ksel(ctypes.byref(p)) == 2 + 2 + 1 + 5
    assert phsa.workspace_size(_p(), phsa.OP_COMPRESS) == 0
    # bf16 hi/lo copies of K_comp and the norms of both parts per block, rounded up to 256 bytes
    assert phsa.workspace_size(_p(), phsa.OP_SELECT) == -(-16 * (2 * 64 * 2 + 8) // 256) * 256
    assert phsa.workspace_size(_p(dtype=phsa.FP32), phsa.OP_SELECT) == 0
    # the softmax-sum mode scores with the same split copies
    assert phsa.workspace_size(_p(flags=phsa.FLAG_SELECT_SOFTMAX_SUM), phsa.OP_SELECT) == \
        phsa.workspace_size(_p(), phsa.OP_SELECT)
    assert phsa.workspace_size(_p(), phsa.OP_FORWARD) >= phsa.workspace_size(_p(), phsa.OP_SELECT)
    fwd = phsa.workspace_size(_p(), phsa.OP_ATTN_FWD)
    assert fwd > 0 and fwd % 256 == 0
    assert phsa.workspace_size(_p(batch=2), phsa.OP_ATTN_FWD) > fwd
    assert phsa.workspace_size(_p(dtype=phsa.FP32), phsa.OP_ATTN_FWD) == 0
    assert phsa.workspace_size(_p(seqlen_q=1), phsa.OP_DECODE) == 0          # decode needs no scratch
    assert phsa.workspace_size(_p(head_dim=96), phsa.OP_ATTN_FWD) == 0     # invalid -> 0
    # 16-token blocks without a local window are indexed on 64-key tiles, at most
    # min(Ksel, Lk / 64) per row, regrouped as the index reads sel: the
    # workspace is laid out as for 64-token blocks with the same Ksel
    big = dict(seqlen_q=8192, seqlen_k=8192)                               # 128 tiles
    w16 = phsa.workspace_size(_p(block_size=16, n_init_blocks=8, top_k=16, **big), phsa.OP_ATTN_FWD)  # Ksel 25
    w64 = phsa.workspace_size(_p(top_k=23, **big), phsa.OP_ATTN_FWD)                                  # Ksel 25
    assert w16 == w64 > 0
    # with a local window (the band kernels) both block sizes use the same tile
    # layout: Ksel = 57 tile slots plus the band slot, and the band flags
    p16 = phsa.workspace_size(_p(block_size=16, n_init_blocks=8, window=512, top_k=16, **big), phsa.OP_ATTN_BWD)
    p64 = phsa.workspace_size(_p(top_k=24, window=31 * 64, **big), phsa.OP_ATTN_BWD)
    assert p16 == p64 > 0
    assert L.phsa_validate(None, phsa.OP_SELECT) == phsa.ERR_NULL


def test_entry_points_reject_before_launch():
    """Every error return happens on the host: no device pointer is touched."""
    L = phsa.lib()
    bogus = ctypes.c_void_p(0x1000)
    good = _p()
    bad = _p(seqlen_k=1000)
    assert L.phsa_compress(ctypes.byref(bad), bogus, bogus, bogus, None) == phsa.ERR_SHAPE
    assert L.phsa_compress(ctypes.byref(good), None, bogus, bogus, None) == phsa.ERR_NULL
    assert L.phsa_select(ctypes.byref(good), bogus, None, bogus, None, 0, None) == phsa.ERR_NULL
    assert L.phsa_attn_fwd(ctypes.byref(good), bogus, bogus, bogus, bogus, bogus, bogus, None, 0,
                           None) == phsa.ERR_WORKSPACE
    assert L.phsa_attn_fwd(ctypes.byref(good), bogus, bogus, bogus, bogus, bogus, bogus, bogus, 16,
                           None) == phsa.ERR_WORKSPACE
    assert L.phsa_attn_bwd(ctypes.byref(_p(dtype=5)), *([bogus] * 11), 0, None) == phsa.ERR_DTYPE
    assert L.phsa_forward(ctypes.byref(good), *([bogus] * 8), None, 0, None) == phsa.ERR_WORKSPACE
    assert L.phsa_decode(ctypes.byref(good), *([bogus] * 7), None, 0, None) == phsa.ERR_SHAPE  # Lq != 1


def test_punct_mask_rejects_before_launch():
    L = phsa.lib()
    bogus = ctypes.c_void_p(0x1000)
    assert L.phsa_punct_mask(bogus, -1, bogus, 1, bogus, None) == phsa.ERR_INVALID_ARG
    assert L.phsa_punct_mask(bogus, 10, bogus, -3, bogus, None) == phsa.ERR_INVALID_ARG
    assert L.phsa_punct_mask(bogus, 10, bogus, phsa.MAX_PUNCT_IDS + 1, bogus, None) == phsa.ERR_UNSUPPORTED
    assert L.phsa_punct_mask(None, 10, bogus, 1, bogus, None) == phsa.ERR_NULL
    assert L.phsa_punct_mask(bogus, 10, None, 1, bogus, None) == phsa.ERR_NULL
    assert L.phsa_punct_mask(None, 0, None, 0, None, None) == phsa.OK     # nothing to do, nothing launched


def test_select_noalloc_rejects_before_launch():
    """The scratch-free selection validates like phsa_select and refuses a
    problem whose scratch would not fit its fixed array, before any GPU call."""
    L = phsa.lib()
    bogus = ctypes.c_void_p(0x1000)
    assert L.phsa_select_noalloc(ctypes.byref(_p(seqlen_k=1000)), bogus, bogus, bogus, None) == phsa.ERR_SHAPE
    assert L.phsa_select_noalloc(ctypes.byref(_p()), None, bogus, bogus, None) == phsa.ERR_NULL
    # B * Hkv * T blocks at (2 * 2 * d + 4) bytes: 64 x 8 x 512 blocks at d = 128 is 135 MB > 64 MiB
    big = _p(batch=64, n_heads_q=16, n_heads_kv=8, head_dim=128, seqlen_q=32768, seqlen_k=32768, top_k=12)
    assert phsa.workspace_size(big, phsa.OP_SELECT) > phsa.NOALLOC_SCRATCH_BYTES
    assert L.phsa_select_noalloc(ctypes.byref(big), bogus, bogus, bogus, None) == phsa.ERR_SCRATCH_LIMIT
    # the 4 x 32k workloads fit, in both geometries
    for kw in (dict(top_k=12), dict(block_size=16, n_init_blocks=8, window=512, top_k=16)):
        p = _p(batch=4, n_heads_q=16, n_heads_kv=8, head_dim=128, seqlen_q=32768, seqlen_k=32768, **kw)
        assert 0 < phsa.workspace_size(p, phsa.OP_SELECT) <= phsa.NOALLOC_SCRATCH_BYTES


def test_status_strings():
    for s in range(9):
        assert isinstance(phsa.status_string(s), str) and phsa.status_string(s)
    assert phsa.status_string(99) == "unknown status"


def test_missing_library_raises(monkeypatch):
    """No fallback: without the built library the binding raises instead of computing."""
    monkeypatch.setattr(phsa, "_active", None)
    monkeypatch.setattr(phsa, "_libs", {})
    monkeypatch.setattr(phsa, "LIB_PATH", os.path.join(ROOT, "no_such_dir", "libphsa.so"))
    with pytest.raises(RuntimeError, match="missing"):
        phsa.lib()
    with pytest.raises(RuntimeError, match="missing"):
        phsa.workspace_size(_p(), phsa.OP_ATTN_FWD)
    # CPU tensors are refused before any library call
    k = torch.zeros(1, 64, 1, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        phsa.compress(k, torch.zeros(1, 64, dtype=torch.uint8), phsa.Config())
