"""PHSA hot-path benchmark on one MI355X.

A step is one training pass of PHSA attention over the 32k-token workload
(batch 4 x 32768 tokens, 16 query / 8 KV heads, head dim 128, 64-token
blocks, 14 blocks per query = 97.3% sparsity): block compression, scoring +
top-k selection, the inverted index, sparse attention forward and backward.
Inputs are seeded synthetic tensors already resident in HBM.

The JSON line reports whole-step selected-block TFLOP/s (4*d*m FLOPs per
(query row, head, selected block) forward, 2.5x that backward) from the timed
steps (HIP events around each step give its median and p90), the GPU clocks
sampled while they run, per-kernel durations from a second timed pass through
the profiling build of the library (HIP events around every launch on its
stream), the roofline of the dominant kernel, a decode-step measurement, and
the fp64 CPU oracle timed on one (batch, KV head) slice of the same workload.
"""
from __future__ import annotations

import argparse
import dataclasses
import glob
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2601_02819_amd import phsa  # noqa: E402
from paper_2601_02819_amd.inputs import WORKLOADS, make_inputs  # noqa: E402

METRIC = "PHSA fwd+bwd ms & selected-block TFLOP/s at L=32k, 97.3% sparsity; % MFMA peak"
CSRC = os.path.join(ROOT, "paper_2601_02819_amd", "csrc")
# kernel name in the timing hooks -> its source file (the traffic record is void once that changes)
KERNEL_SOURCE = {"phsa_attn_bwd_sparse": "attn_bwd.hip", "phsa_attn_fwd_sparse": "attn_fwd.hip",
                 "phsa_select": "select.hip", "phsa_compress": "compress.hip",
                 "phsa_attn_fwd_combine": "attn_fwd.hip", "phsa_attn_bwd_dq_combine": "attn_bwd.hip"}
# rocprofv3 kernel-name fragment of each timed kernel
KERNEL_SYMBOL = {"phsa_attn_bwd_sparse": "attn_bwd_sparse_kernel", "phsa_attn_fwd_sparse": "attn_fwd_sparse_kernel",
                 "phsa_select": "select_mfma_kernel", "phsa_compress": "compress_kernel",
                 "phsa_attn_fwd_combine": "attn_fwd_combine_kernel", "phsa_attn_bwd_dq_combine": "dq_combine_kernel"}


def code_text(src: str) -> str:
    """Source text without // comments and blank lines (what the compiler sees
    of a kernel file, up to comment edits)."""
    import re
    lines = (re.sub(r"\s*//.*$", "", ln).rstrip() for ln in src.splitlines())
    return "\n".join(ln for ln in lines if ln)


def source_hash(kernel: str) -> str:
    """Hash of the code a kernel is built from; measured traffic is reported only
    while it matches the hash stored with the measurement."""
    import hashlib
    h = hashlib.sha256()
    for f in (KERNEL_SOURCE[kernel], "common.h", "launch.h"):
        h.update(code_text(open(os.path.join(CSRC, f)).read()).encode())
    return h.hexdigest()[:16]


def summarize_traffic(fetch_csv: str, write_csv: str, copy_mb: int, out_json: str) -> None:
    """Turns two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE; KiB per dispatch) into
    calibrated HBM bytes per launch: each counter is scaled by what it reads for the
    plain elementwise copy of copy_mb MiB that --calib-copy-mb runs first."""
    import csv
    import statistics

    def per_kernel(path):
        d = {}
        for r in csv.DictReader(open(path)):
            d.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return d

    fd, wd = per_kernel(fetch_csv), per_kernel(write_csv)
    copy_kib = copy_mb * 1024.0
    cal = [n for n in fd if "MulFunctor" in n or "mul" in n.split("(")[0].lower()]
    big = [n for n in cal if max(fd[n]) > 0.25 * copy_kib]
    if not big:
        raise SystemExit("calibration copy kernel not found in " + fetch_csv)
    fetch_factor = copy_kib / max(fd[big[0]])
    write_factor = copy_kib / max(wd[big[0]])
    rec = {"calibration_kernel": big[0].split("(")[0], "copy_mib": copy_mb,
           "fetch_factor": fetch_factor, "write_factor": write_factor, "kernels": {}}
    for k, sym in KERNEL_SYMBOL.items():
        names = [n for n in fd if sym in n]
        if not names:
            continue
        f = statistics.median(fd[names[0]]) * 1024 * fetch_factor
        w = statistics.median(wd[names[0]]) * 1024 * write_factor
        rec["kernels"][k] = {"symbol": names[0].split("(")[0], "fetch_bytes": f, "write_bytes": w,
                             "bytes_per_launch": f + w, "source_hash": source_hash(k)}
    json.dump(rec, open(out_json, "w"), indent=1)
    print(json.dumps(rec, indent=1))
# Three rocprofv3 --pmc passes (at most 8 SQ counters and one GRBM counter each)
# whose counter_collection.csv files --summarize-counters turns into a table.
COUNTER_PASSES = (
    "SQ_VALU_MFMA_BUSY_CYCLES SQ_VALU_MFMA_COEXEC_CYCLES SQ_WAVE_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_ANY "
    "SQ_WAIT_INST_LDS SQ_ACTIVE_INST_ANY SQ_BUSY_CU_CYCLES GRBM_GUI_ACTIVE",
    "SQ_INSTS_VALU SQ_INSTS_MFMA SQ_INSTS_LDS SQ_INSTS_SALU SQ_INSTS_VMEM SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE "
    "SQ_ACTIVE_INST_LDS GRBM_GUI_ACTIVE",
    "SQ_INSTS_VALU_TRANS_F32 SQ_LDS_ADDR_CONFLICT SQ_LDS_DATA_FIFO_FULL SQ_LDS_CMD_FIFO_FULL SQ_INSTS_VMEM_RD "
    "SQ_INSTS_VMEM_WR SQ_INSTS_SMEM SQ_ACTIVE_INST_VALU GRBM_GUI_ACTIVE",
)


def summarize_counters(out_md: str, csvs) -> None:
    """Per-kernel table from rocprofv3 --pmc counter_collection.csv files (the
    passes of COUNTER_PASSES, any order), written after the preamble of an
    existing out_md.  Values are medians over a kernel's
    dispatches; the topology (XCCs, SIMDs, CUs) comes from the agent_info.csv
    written beside each counter file.  Derived columns:
      MFMA busy   SQ_VALU_MFMA_BUSY_CYCLES / (kernel cycles x SIMDs), kernel
                  cycles = GRBM_GUI_ACTIVE / XCCs (GRBM counts on every XCC)
      co-exec     share of MFMA-busy cycles in which a VALU instruction issued
      VALU/MFMA, LDS/MFMA, exp/MFMA   instruction counts per MFMA instruction
                  (SQ_INSTS_VALU counts MFMA instructions too)
      bank confl. SQ_LDS_BANK_CONFLICT / (SQ_LDS_IDX_ACTIVE - SQ_LDS_BANK_CONFLICT)
      waits       SQ_WAIT_INST_LDS, SQ_WAIT_INST_ANY, SQ_WAIT_ANY as shares of
                  SQ_WAVE_CYCLES (all in quad-cycles)
      waves/CU    resident waves per CU on average (4 SQ_WAVE_CYCLES / cycles / CUs)"""
    import csv
    import glob
    import statistics

    per, dur, topo = {}, {}, {}
    for path in csvs:
        for ai in glob.glob(os.path.join(os.path.dirname(path), "*agent_info.csv")):
            for r in csv.DictReader(open(ai)):
                if r.get("Name", "").startswith("gfx"):
                    topo = {k: int(r[k]) for k in ("Num_Xcc", "Simd_Count", "Cu_Count")}
        for r in csv.DictReader(open(path)):
            sym = r["Kernel_Name"].split("(")[0].replace("void ", "")
            per.setdefault(sym, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
            if r["Counter_Name"] == "GRBM_GUI_ACTIVE":
                dur.setdefault(sym, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-6)
    if not topo:
        raise SystemExit("no gfx agent in the agent_info.csv files beside " + " ".join(csvs))

    def ratio(a, b):
        return a / b if b else float("nan")

    rows = []
    for sym, c in per.items():
        m = {k: statistics.median(v) for k, v in c.items()}
        need = ("GRBM_GUI_ACTIVE", "SQ_INSTS_MFMA", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_WAVE_CYCLES")
        if any(k not in m for k in need) or m["SQ_INSTS_MFMA"] == 0 and "phsa::" not in sym:
            continue
        cyc = m["GRBM_GUI_ACTIVE"] / topo["Num_Xcc"]
        ms = statistics.median(dur[sym])
        wc = m["SQ_WAVE_CYCLES"]
        rows.append((ms, sym, [
            f"{ms:.3f}", f"{cyc / ms * 1e-6:.2f}",
            f"{100 * ratio(m['SQ_VALU_MFMA_BUSY_CYCLES'], cyc * topo['Simd_Count']):.1f}",
            f"{100 * ratio(m.get('SQ_VALU_MFMA_COEXEC_CYCLES', 0), m['SQ_VALU_MFMA_BUSY_CYCLES']):.0f}",
            f"{ratio(m.get('SQ_INSTS_VALU', 0), m['SQ_INSTS_MFMA']):.2f}",
            f"{ratio(m.get('SQ_INSTS_LDS', 0), m['SQ_INSTS_MFMA']):.2f}",
            f"{ratio(m.get('SQ_INSTS_VALU_TRANS_F32', 0), m['SQ_INSTS_MFMA']):.2f}",
            f"{100 * ratio(m.get('SQ_LDS_BANK_CONFLICT', 0), m.get('SQ_LDS_IDX_ACTIVE', 0) - m.get('SQ_LDS_BANK_CONFLICT', 0)):.0f}",
            f"{100 * ratio(m.get('SQ_WAIT_INST_LDS', 0), wc):.0f}",
            f"{100 * ratio(m.get('SQ_WAIT_INST_ANY', 0), wc):.0f}",
            f"{100 * ratio(m.get('SQ_WAIT_ANY', 0), wc):.0f}",
            f"{4 * wc / cyc / topo['Cu_Count']:.1f}",
            f"{m['SQ_INSTS_MFMA']:.3g}", f"{m.get('SQ_INSTS_VALU', float('nan')):.3g}",
            f"{m.get('SQ_INSTS_LDS', float('nan')):.3g}"]))
    rows.sort(reverse=True)
    head = ["kernel", "ms", "GHz", "MFMA busy %", "co-exec %", "VALU/MFMA", "LDS/MFMA", "exp/MFMA",
            "bank confl. %", "wait LDS %", "wait inst %", "wait any %", "waves/CU", "MFMA insts", "VALU insts",
            "LDS insts"]
    lines = ["| " + " | ".join(head) + " |", "|" + "---|" * len(head)]
    lines += ["| `" + sym + "` | " + " | ".join(v) + " |" for _, sym, v in rows]
    text = "\n".join(lines) + "\n"
    # an existing summary keeps its preamble (title, commands, legend) and gets the new table
    pre = ""
    if os.path.exists(out_md):
        old = open(out_md).read()
        pre = old[:old.index("| kernel |")] if "| kernel |" in old else old
    open(out_md, "w").write(pre + text)
    print(text)


PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0


TRAIN_TEXT = {
    "train_32k": "train_32k: PHSA fwd+bwd, batch 4 x 32768 tokens, 16 query / 8 KV heads, head dim 128, "
                 "block 64, 1 init + 1 local + 12 top-k blocks (97.3% sparse)",
    "train_32k_paper": "train_32k_paper: PHSA fwd+bwd, batch 4 x 32768 tokens, 16 query / 8 KV heads, head dim 128, "
                       "16-token blocks, 8 init blocks, 512-token window, 16 top-k blocks (57 blocks = 912 tokens "
                       "per query, 97.2% sparse)",
}


def cfg_of(wl):
    return phsa.Config(block_size=wl.block_size, top_k=wl.top_k, n_init_blocks=wl.n_init_blocks, window=wl.window,
                       lam=wl.lam)


def selected_blocks(sel: torch.Tensor, seqlen_k: int, block: int) -> int:
    """Sum over (b, g, query row) of the number of valid selected blocks."""
    Lq = sel.shape[2]
    cur = ((seqlen_k - Lq + torch.arange(Lq, device=sel.device)) // block).view(1, 1, Lq, 1)
    return int(((sel >= 0) & (sel <= cur)).sum().item())


def dist(xs):
    """avg / median / p90 of a list of durations (ms)."""
    a = np.asarray(xs, dtype=np.float64)
    return {"avg_ms": float(a.mean()), "median_ms": float(np.median(a)), "p90_ms": float(np.percentile(a, 90)),
            "launches": int(a.size)}


def kernel_stats(times, names, steps):
    out = {}
    for n in names:
        d = times.durations(n)
        if d:
            out[n] = dist(d)
            out[n]["total_ms"] = float(np.sum(d))
            out[n]["per_step"] = len(d) / steps
    return out


def gpu_clocks():
    """Current shader (sclk) and memory (mclk) clock levels of the GPU, read from
    the amdgpu driver's sysfs files (no process is started: reading a file is
    safe once the GPU is in use)."""
    try:
        pr = torch.cuda.get_device_properties(0)
        dev = "/sys/bus/pci/devices/%04x:%02x:%02x.0" % (pr.pci_domain_id, pr.pci_bus_id, pr.pci_device_id)
        if not os.path.isdir(dev):
            cands = glob.glob("/sys/class/drm/card*/device")
            dev = cands[0] if len(cands) == 1 else dev
        out = {"sysfs": dev}
        for key in ("pp_dpm_sclk", "pp_dpm_mclk"):
            with open(os.path.join(dev, key)) as f:
                cur = [ln.split(":", 1)[1].replace("*", "").strip() for ln in f if ln.rstrip().endswith("*")]
            out[key[-4:]] = cur[0] if cur else None
        return out
    except Exception as e:  # no GPU, no sysfs files, another driver
        return {"unavailable": type(e).__name__}


KERNELS = ["phsa_compress", "phsa_select_split", "phsa_select", "phsa_index_count", "phsa_index_scan_tiles", "phsa_index_scan_lists",
           "phsa_index_fill", "phsa_attn_fwd_sparse", "phsa_attn_fwd_band", "phsa_attn_fwd_combine",
           "phsa_attn_bwd_pre", "phsa_attn_bwd_band_dkv_init", "phsa_attn_bwd_band_init_reduce", "phsa_attn_bwd_band_dkv",
           "phsa_attn_bwd_band_dq", "phsa_attn_bwd_sparse",
           "phsa_attn_bwd_dkv_finalize", "phsa_attn_bwd_dq_combine"]


def selected_tiles(sel: torch.Tensor, seqlen_k: int, block: int) -> int:
    """Sum over (b, g, query row) of the distinct 64-key tiles holding the row's
    valid selected blocks (the attention kernels' work items; = selected_blocks
    for 64-token blocks)."""
    Lq = sel.shape[2]
    cur = ((seqlen_k - Lq + torch.arange(Lq, device=sel.device)) // block).view(1, 1, Lq, 1)
    valid = (sel >= 0) & (sel <= cur)
    tc = torch.div(sel, 64 // block, rounding_mode="floor")
    same = (tc[..., 1:] == tc[..., :-1]) & valid[..., 1:] & valid[..., :-1]
    return int(valid.sum().item() - same.sum().item())


def band_blocks(sel: torch.Tensor, seqlen_k: int, block: int, n_init: int, window: int):
    """Per (b, g, query row): how many of its selected blocks the band kernels
    take (bf16 attention).  A row whose selection holds all its forced blocks,
    the init blocks 0 .. ninit - 1 (ninit = min(n_init, cur + 1)) and the local
    window A .. cur with A = max(cur - window / block, ninit), leaves them to
    the band; other rows keep all their blocks in the sparse kernels.  Returns
    the counts, A, and the counts' init blocks, per row (0 for other rows)."""
    Lq = sel.shape[2]
    cur = ((seqlen_k - Lq + torch.arange(Lq, device=sel.device)) // block).view(1, 1, Lq)
    ninit = torch.clamp(cur + 1, max=n_init)
    a = torch.maximum((cur - window // block).clamp(min=0), ninit)
    valid = (sel >= 0) & (sel <= cur.unsqueeze(-1))
    forced = valid & ((sel < ninit.unsqueeze(-1)) | (sel >= a.unsqueeze(-1)))
    need = ninit + cur - a + 1
    ok = forced.sum(-1) == need
    zero = torch.zeros_like(cur)
    return torch.where(ok, need, zero), a, torch.where(ok, ninit, zero)


def sparse_part(sel: torch.Tensor, nb: torch.Tensor, a: torch.Tensor, ninit: torch.Tensor) -> torch.Tensor:
    """sel without the blocks that band_blocks gives to the band kernels."""
    band_row = (nb > 0).unsqueeze(-1)
    forced = (sel < ninit.unsqueeze(-1)) | (sel >= a.unsqueeze(-1))
    return torch.where(band_row & forced, torch.full_like(sel, -1), sel)


def bench_train(steps: int, warmup: int, seed: int, name: str = "train_32k"):
    wl = WORKLOADS[name]
    cfg = cfg_of(wl)
    host = make_inputs(wl, seed, with_grad_out=True)
    dev = {k: v.cuda() for k, v in host.items()}
    B, L, Hq, Hkv, d, m, T = wl.batch, wl.seqlen_q, wl.n_heads_q, wl.n_heads_kv, wl.head_dim, wl.block_size, wl.n_blocks
    G = Hq // Hkv
    p = phsa.make_params(cfg, B, L, L, Hq, Hkv, d, torch.bfloat16)
    # one workspace for both passes: the backward reuses the forward's inverted index
    ws = torch.empty(max(phsa.workspace_size(p, phsa.OP_FORWARD), phsa.workspace_size(p, phsa.OP_ATTN_BWD)),
                     dtype=torch.uint8, device="cuda")

    def step():
        kc, sel, o, lse = phsa.forward(dev["q"], dev["k"], dev["v"], dev["punct"], cfg, ws=ws)
        dq, dk, dv = phsa.attn_bwd(dev["q"], dev["k"], dev["v"], o, dev["do"], lse, sel, cfg, ws=ws, reuse_index=True)
        return sel

    for _ in range(warmup):
        sel = step()
    torch.cuda.synchronize()
    nsel = selected_blocks(sel, L, m)
    band = wl.window >= 64 and L % 64 == 0 and min(wl.ksel, L // 64) <= 63  # the library's rule for bf16 attention
    if band:
        nb, a, ni = band_blocks(sel, L, m, wl.n_init_blocks, wl.window)
        sparse_sel = sparse_part(sel, nb, a, ni)
        nband, nband_init = int(nb.sum().item()), int(ni.sum().item())
    else:
        sparse_sel, nband, nband_init = sel, 0, 0
    ntile = selected_tiles(sparse_sel, L, m)  # the sparse kernels' tiles
    # headline: `steps` steps of the product library, one HIP event between steps
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record()
    for i in range(steps):
        step()
        evs[i + 1].record()
    clocks = gpu_clocks()   # sampled while the enqueued steps run
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / steps
    step_ms = [evs[i].elapsed_time(evs[i + 1]) for i in range(steps)]
    # per-kernel durations: the same steps again through the profiling build,
    # which records HIP events around every launch on the launch stream
    prof_steps = max(steps, 50)
    with phsa.profiling() as times:
        for _ in range(prof_steps):
            step()
        torch.cuda.synchronize()
        ks = kernel_stats(times, KERNELS, prof_steps)
        times.reset()

    fwd_flop = 4.0 * d * m * nsel * G
    bwd_flop = 2.5 * fwd_flop
    # the forced blocks' share, attended by the band kernels (same convention);
    # the init tiles' dK/dV run in a launch of their own
    band_fwd_flop = 4.0 * d * m * nband * G
    band_init_fwd_flop = 4.0 * d * m * nband_init * G
    sparse_fwd_flop = fwd_flop - band_fwd_flop
    # MFMA work the kernels execute: whole 64-key tiles (blocks below 64 tokens
    # share tiles, the unselected quarters of a tile are masked)
    tile_fwd_flop = 4.0 * d * 64 * ntile * G
    # Bytes the key-block-major kernels must move per launch: every (row, tile)
    # pair gathers its query rows (and dO rows) and leaves a bf16 partial (plus
    # the forward's (m, l)); every work unit loads its K/V tile once.  This is
    # the schedule's own traffic floor, above the method's algorithmic minimum.
    unit_tokens = 64 * (64 // G)
    T64 = L // 64
    units = B * Hkv * T64 + ntile // unit_tokens
    kv_bytes = units * 64 * d * 2 * 2
    pair_row = G * d * 2
    design_bytes = {"phsa_attn_fwd_sparse": ntile * (2 * pair_row + G * 8 + 4) + kv_bytes,
                    "phsa_attn_bwd_sparse": ntile * (3 * pair_row + G * 8 + 4) + kv_bytes + B * L * Hkv * d * 2 * 2}
    bytes_compress = B * L * Hkv * d * 2 + B * L + B * Hkv * T * d * 4
    bytes_select = B * L * Hq * d * 2 + B * Hkv * T * d * 4 + B * Hkv * L * wl.ksel * 4
    # each attention kernel is credited with the selected-block FLOPs it covers;
    # the band's backward is split as executed: dK/dV 8 d, dQ 6 d per (row, head, key)
    work = {"phsa_attn_fwd_sparse": ("TFLOP/s", sparse_fwd_flop / 1e12),
            "phsa_attn_bwd_sparse": ("TFLOP/s", 2.5 * sparse_fwd_flop / 1e12),
            "phsa_compress": ("GB/s", bytes_compress / 1e9), "phsa_select": ("GB/s", bytes_select / 1e9)}
    if nband:
        work.update({"phsa_attn_fwd_band": ("TFLOP/s", band_fwd_flop / 1e12),
                     "phsa_attn_bwd_band_dkv": ("TFLOP/s", 2.0 * (band_fwd_flop - band_init_fwd_flop) / 1e12),
                     "phsa_attn_bwd_band_dkv_init": ("TFLOP/s", 2.0 * band_init_fwd_flop / 1e12),
                     "phsa_attn_bwd_band_dq": ("TFLOP/s", 1.5 * band_fwd_flop / 1e12)})
    for n, (unit, amount) in work.items():
        if n in ks:
            rate = amount / (ks[n]["avg_ms"] / 1e3)
            peak = PEAK_BF16_TFLOPS if unit == "TFLOP/s" else PEAK_HBM_GBS
            ks[n].update(rate=rate, unit=unit, frac=rate / peak)
            if n in design_bytes:
                # attainable = min(MFMA peak, intensity x HBM peak) for this schedule's
                # traffic and executed tile work, in selected-block FLOP/s
                flop = work[n][1] * 1e12
                exec_flop = tile_fwd_flop * (1.0 if "fwd" in n else 2.5)
                t_min = max(exec_flop / (PEAK_BF16_TFLOPS * 1e12), design_bytes[n] / (PEAK_HBM_GBS * 1e9))
                att = flop / 1e12 / t_min
                ks[n].update(schedule_bytes=design_bytes[n],
                             schedule_GB_per_s=design_bytes[n] / 1e9 / (ks[n]["avg_ms"] / 1e3),
                             attainable_tflops=att, frac_of_attainable=rate / att)
    dom = max(ks, key=lambda n: ks[n]["total_ms"])
    return {
        "ms_per_step": ms_step,
        "step_ms": {k: v for k, v in dist(step_ms).items() if k != "launches"},
        "gpu_clocks": clocks,
        "kernel_timing": f"{prof_steps} steps through libphsa_prof.so (HIP events around each launch)",
        "value": (fwd_flop + bwd_flop) / 1e12 / (ms_step / 1e3),
        "fwd_flop": fwd_flop, "bwd_flop": bwd_flop, "selected_blocks": nsel, "band_blocks": nband,
        "band_init_blocks": nband_init,
        "sparse_tiles": ntile,
        "tile_fwd_flop": tile_fwd_flop,
        # the paper's convention: active tokens of the last query over the sequence length
        "sparsity_last_query": 1.0 - wl.ksel * m / L,
        "sparsity_causal_mean": 1.0 - nsel * m / (B * Hkv * L * (L + 1) / 2),
        "kernels": ks, "dominant": dom, "host": host,
    }


def bench_decode(iters: int, seed: int):
    """One decode step (64 sequences x 1 query vs a 32k cache).  The representatives
    (134 MB) and a step's selected K/V blocks (235 MB) would fit the 256 MB
    last-level cache if one step were simply repeated, so the timed loop rotates
    four query sets (each selects different blocks of the 8.6 GB cache) and four
    copies of the representatives (536 MB)."""
    wl = WORKLOADS["decode_32k"]
    cfg = cfg_of(wl)
    host = make_inputs(wl, seed, with_grad_out=False)
    dev = {k: v.cuda() for k, v in host.items()}
    kc0 = phsa.compress(dev["k"], dev["punct"], cfg)      # block cache representatives, untimed
    R = 4
    gen = torch.Generator(device="cpu")
    gen.manual_seed(seed + 1)
    qs = [dev["q"]] + [torch.randn(dev["q"].shape, generator=gen).to(torch.bfloat16).cuda() for _ in range(R - 1)]
    kcs = [kc0] + [kc0.clone() for _ in range(R - 1)]
    for r in range(R):
        sel, o, lse = phsa.decode(qs[r], dev["k"], dev["v"], kcs[r], cfg)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for i in range(iters):
        sel, o, lse = phsa.decode(qs[i % R], dev["k"], dev["v"], kcs[i % R], cfg)
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / iters
    nsel = selected_blocks(sel, wl.seqlen_k, wl.block_size)
    B, Hq, Hkv, d, T, m = wl.batch, wl.n_heads_q, wl.n_heads_kv, wl.head_dim, wl.n_blocks, wl.block_size
    nbytes = B * Hkv * T * d * 4 + nsel * m * d * 2 * 2 + 2 * B * Hq * d * 2 + B * Hkv * wl.ksel * 4
    return {"workload": "decode_32k: 64 sequences x 1 query vs a 32768-token cache, 16/8 heads, d 128, 14 blocks",
            "ms_per_step": ms, "algorithmic_bytes": nbytes, "GB_per_s": nbytes / 1e9 / (ms / 1e3),
            "frac_hbm_peak": nbytes / 1e9 / (ms / 1e3) / PEAK_HBM_GBS,
            "timing": f"{iters} steps rotating {R} query sets and {R} copies of the representatives"}


def bench_generation(iters: int, seed: int):
    """One generation step with per-sequence cache lengths: append a token to every
    sequence's block cache (maintaining the representative of a block it completes),
    then decode it.  64 sequences, 32k capacity, lengths 30000-32700."""
    wl = WORKLOADS["decode_32k"]
    cfg = cfg_of(wl)
    B, cap, Hq, Hkv, d = wl.batch, wl.seqlen_k, wl.n_heads_q, wl.n_heads_kv, wl.head_dim
    host = make_inputs(wl, seed, with_grad_out=False)
    k, v, punct = host["k"].cuda(), host["v"].cuda(), host["punct"].cuda()
    kc = phsa.compress(k, punct, cfg)
    gen = torch.Generator(device="cpu")
    gen.manual_seed(seed + 2)
    clen = torch.randint(30000, 32700, (B,), generator=gen, dtype=torch.int32).cuda()
    R = 4
    qs = [torch.randn(B, 1, Hq, d, generator=gen).to(torch.bfloat16).cuda() for _ in range(R)]
    kn = [torch.randn(B, Hkv, d, generator=gen).to(torch.bfloat16).cuda() for _ in range(R)]
    vn = [torch.randn(B, Hkv, d, generator=gen).to(torch.bfloat16).cuda() for _ in range(R)]
    pn = [(torch.rand(B, generator=gen) < 0.08).to(torch.uint8).cuda() for _ in range(R)]
    for r in range(R):
        phsa.cache_append(kn[r], vn[r], pn[r], k, v, punct, clen, kc, cfg)
        phsa.decode_varlen(qs[r], k, v, kc, clen, cfg)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for i in range(iters):
        phsa.cache_append(kn[i % R], vn[i % R], pn[i % R], k, v, punct, clen, kc, cfg)
        phsa.decode_varlen(qs[i % R], k, v, kc, clen, cfg)
    ev1.record()
    torch.cuda.synchronize()
    return {"workload": "64 sequences, 32k-token block caches at lengths 30000-32700: append one token "
                        "(block representative maintained) + decode it", "ms_per_step": ev0.elapsed_time(ev1) / iters}


def bench_punct(seed: int):
    """Token ids -> punctuation mask for the 4 x 32768 training batch (60 punctuation ids)."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(seed + 3)
    ids = torch.randint(0, 151936, (4, 32768), generator=gen, dtype=torch.int32).cuda()
    pset = torch.sort(torch.randperm(151936, generator=gen)[:60].to(torch.int32)).values.cuda()
    for _ in range(3):
        phsa.punct_mask(ids, pset)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(50):
        phsa.punct_mask(ids, pset)
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / 50
    nbytes = ids.numel() * 5
    return {"workload": "4 x 32768 token ids, 60 punctuation ids", "ms": ms, "GB_per_s": nbytes / 1e9 / (ms / 1e3)}


def bench_select_modes(seed: int):
    """Block selection alone on the 4 x 32768 training batch in both group
    aggregation modes: summed logits (the training step's mode) and summed
    per-head softmax.  The softmax mode computes, per (row, head), a logit for
    every complete causal block (normaliser) and again for every candidate."""
    wl = WORKLOADS["train_32k"]
    B, L, Hq, Hkv, d, m = wl.batch, wl.seqlen_k, wl.n_heads_q, wl.n_heads_kv, wl.head_dim, wl.block_size
    gen = torch.Generator(device="cpu")
    gen.manual_seed(seed + 5)
    q = torch.randn(B, L, Hq, d, generator=gen).to(torch.bfloat16).cuda()
    k = torch.randn(B, L, Hkv, d, generator=gen).to(torch.bfloat16).cuda()
    punct = (torch.rand(B, L, generator=gen) < 0.08).to(torch.uint8).cuda()
    out = {"workload": "train_32k selection: 4 x 32768 queries, 16/8 heads, d 128, 512 blocks, 12 free picks"}
    cur = np.arange(L) // m
    G = Hq // Hkv
    cand = np.maximum(cur - wl.n_init_blocks - wl.window // m, 0).sum()
    for name, sm in (("summed_logits", False), ("softmax_sum", True)):
        cfg = dataclasses.replace(cfg_of(wl), softmax_sum=sm)
        kc = phsa.compress(k, punct, cfg)
        for _ in range(2):
            phsa.select(q, kc, L, cfg)
        torch.cuda.synchronize()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record()
        for _ in range(5):
            phsa.select(q, kc, L, cfg)
        ev1.record()
        torch.cuda.synchronize()
        ms = ev0.elapsed_time(ev1) / 5
        if sm:
            flop = 2.0 * d * B * Hkv * G * (cur.sum() + cand)   # fp32 FMAs on the vector units
        else:
            flop = 2.0 * d * B * Hkv * cand                     # one dot per (row, group, candidate)
        out[name] = {"ms": ms, "score_tflop": flop / 1e12, "TFLOP_per_s": flop / 1e12 / (ms / 1e3)}
    return out


def cpu_baseline(host, wl, total_blocks: int, b: int = 0, g: int = 0):
    """The fp64 oracle, end to end (compress, select, forward, backward), on one
    (batch, KV head) slice of the workload: batch b, KV head g and its G query
    heads, all query rows.  PHSA is independent per (batch, KV head) and every
    slice has the same shape, so this is a complete sub-problem; the time of the
    whole workload is extrapolated by the ratio of selected-block FLOPs
    (total_blocks: the workload's selected (row, group, block) count)."""
    import oracle

    oracle.build()
    G = wl.n_heads_q // wl.n_heads_kv
    q = host["q"][b:b + 1, :, g * G:(g + 1) * G].float().numpy()
    k = host["k"][b:b + 1, :, g:g + 1].float().numpy()
    v = host["v"][b:b + 1, :, g:g + 1].float().numpy()
    do = host["do"][b:b + 1, :, g * G:(g + 1) * G].float().numpy()
    punct = host["punct"][b:b + 1].numpy()
    d, m, L = wl.head_dim, wl.block_size, wl.seqlen_k
    scale = d ** -0.5
    threads = oracle.num_threads()
    t0 = time.perf_counter()
    kc = oracle.compress(k, punct, m, wl.lam)
    sel, _, _ = oracle.select(q, kc, m, wl.top_k, wl.n_init_blocks, wl.window, scale, L)
    oracle.attn_fwd(q, k, v, sel, m, scale)
    oracle.attn_bwd(q, k, v, do, sel, m, scale)
    dt = time.perf_counter() - t0
    cur = (np.arange(L) // m)[None, None, :, None]
    nsel = int(((sel >= 0) & (sel <= cur)).sum())
    flop = 4.0 * d * m * nsel * G * 3.5
    full = dt * total_blocks / nsel
    return {"value": flop / 1e12 / dt, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "seconds": dt, "extrapolated_full_seconds": full,
            "sample": f"batch {b}, KV head {g} with its {G} query heads, all {L} query rows of the "
                      f"{wl.batch}x{L} training workload: 1 of its {wl.batch * wl.n_heads_kv} independent "
                      f"(batch, KV head) slices, fp64 compress+select+forward+backward; the full workload's "
                      f"time is extrapolated by the selected-block FLOP ratio ({total_blocks / nsel:.2f}x)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-paper-geometry", action="store_true")
    ap.add_argument("--train-workload", default="train_32k", choices=sorted(TRAIN_TEXT),
                    help="training workload of the headline line (train_32k_paper: for profiling that geometry)")
    ap.add_argument("--calib-copy-mb", type=int, default=0,
                    help="run one device-to-device copy of this many MiB first (a known-size kernel for "
                         "calibrating rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="measured HBM traffic of the dominant kernel (from rocprofv3 counters)")
    ap.add_argument("--summarize-counters", nargs="+", metavar=("OUT_MD", "CSV"),
                    help="write a per-kernel counter table (markdown) from rocprofv3 --pmc counter_collection.csv "
                         "files of the COUNTER_PASSES passes and exit")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write --traffic from two rocprofv3 --pmc counter_collection.csv files and exit")
    args = ap.parse_args()
    if args.summarize_counters:
        if len(args.summarize_counters) < 2:
            ap.error("--summarize-counters OUT_MD CSV [CSV ...]")
        summarize_counters(args.summarize_counters[0], args.summarize_counters[1:])
        return
    if args.summarize_traffic:
        summarize_traffic(args.summarize_traffic[0], args.summarize_traffic[1], args.calib_copy_mb or 1024,
                          args.traffic)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the PHSA path shards by (batch, KV head) with no exchange, "
              "and the library has no multi-GPU mode.", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    phsa.lib()
    wl0 = WORKLOADS[args.train_workload]
    if args.calib_copy_mb > 0:
        # plain elementwise copy (reads N bytes, writes N bytes) for counter calibration
        n = args.calib_copy_mb * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst

    tr = bench_train(args.steps, args.warmup, args.seed, args.train_workload)
    dom = tr["dominant"]
    dk = tr["kernels"][dom]
    traffic = None
    if os.path.exists(args.traffic):
        try:
            tk = json.load(open(args.traffic)).get("kernels", {}).get(dom)
            if tk and tk.get("source_hash") == source_hash(dom):
                traffic = tk["bytes_per_launch"]
        except (OSError, ValueError, KeyError):
            traffic = None
    roofline = {"bound": "mfma" if dk.get("unit") == "TFLOP/s" else "hbm", "kernel": dom,
                "achieved": dk.get("rate"), "peak": PEAK_BF16_TFLOPS if dk.get("unit") == "TFLOP/s" else PEAK_HBM_GBS,
                "unit": dk.get("unit"), "frac": dk.get("frac"), "traffic": traffic,
                "avg_ms": dk["avg_ms"], "median_ms": dk["median_ms"], "p90_ms": dk["p90_ms"]}
    for key in ("schedule_bytes", "attainable_tflops", "frac_of_attainable"):
        if key in dk:
            roofline[key] = dk[key]
    result = {
        "metric": METRIC, "value": tr["value"], "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": tr["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "step_ms": tr["step_ms"], "gpu_clocks": tr["gpu_clocks"],
        "config": {"workload": TRAIN_TEXT[args.train_workload],
                   "batch": wl0.batch, "seq_len": wl0.seqlen_k, "heads_q": wl0.n_heads_q, "heads_kv": wl0.n_heads_kv,
                   "head_dim": wl0.head_dim, "block": wl0.block_size,
                   "blocks_per_query": wl0.ksel, "sparsity_last_query": tr["sparsity_last_query"],
                   "sparsity_causal_mean": tr["sparsity_causal_mean"]},
        "selected_block_gflop": {"fwd": tr["fwd_flop"] / 1e9, "bwd": tr["bwd_flop"] / 1e9},
        "frac_mfma_peak_step": tr["value"] / PEAK_BF16_TFLOPS,
        "roofline": roofline,
        "kernel_timing": tr["kernel_timing"],
        "kernels": tr["kernels"],
    }
    host0 = tr.pop("host")
    if not args.no_paper_geometry and args.train_workload != "train_32k_paper":
        pg = bench_train(max(2, args.steps // 2), max(1, args.warmup), args.seed, "train_32k_paper")
        del pg["host"]
        pg.pop("dominant")
        pg["value_unit"] = "TFLOP/s (selected-block)"
        pg["workload"] = TRAIN_TEXT["train_32k_paper"]
        result["train_32k_paper_geometry"] = pg
    if not args.no_decode:
        result["decode"] = bench_decode(40, args.seed)
        result["generation_step"] = bench_generation(40, args.seed)
        result["punct_mask"] = bench_punct(args.seed)
        result["select_modes"] = bench_select_modes(args.seed)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(host0, wl0, tr["selected_blocks"])
    print(json.dumps(result))


if __name__ == "__main__":
    main()
