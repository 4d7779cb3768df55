"""Benchmark of the encoder-layer kernel chain on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config vit22b]

One step is one forward + backward pass of one encoder layer over one
micro-batch of synthetic tokens, launched kernel by kernel through the C ABI
(the separately schedulable units; the composite entry points run the same
kernels and are bit-identical).  Every launch is bracketed by HIP events on
the stream it runs on, so the timed region also yields each kernel's p50
latency.  Prints one JSON line: fwd+bwd TFLOP/s of the whole chain (and its
fraction of the bf16 MFMA peak), per-kernel p50 latencies, the roofline of
the dominant kernel, and the float64 oracle timed on the host cores over a
bounded sample of the same workload.
"""

import argparse
import json
import os
import platform
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6  # 256 CU x 2.4 GHz x 4096 dense bf16 flop/clk/CU
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="vit22b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget-s", type=float, default=15.0)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--fit-config", default="vit22b_tp8",
                    help="a second workload whose chain is timed briefly and packed into the synthetic "
                         "TP-bubble trace beside the main one ('' or 'none' to skip)")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip timing the ViT-22B-style parallel block at the same shape")
    ap.add_argument("--no-corun", action="store_true",
                    help="skip the co-run measurement (encoder chain beside a GEMM load on a second stream)")
    ap.add_argument("--encoder-layers", type=int, default=48,
                    help="also time the whole encoder (patch embedding + this many layers + final LayerNorm) "
                         "at the workload's shape; 0 skips it")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip timing the layer chain at the other workloads (ViT-Tiny/Base/Huge, TP shard)")
    ap.add_argument("--no-isolated", action="store_true",
                    help="skip timing every kernel on its own, launched back to back")
    ap.add_argument("--no-flush", action="store_true",
                    help="skip timing the memory-bound kernels after a 512 MiB cache flush")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip the measured MFMA-only and device-copy reference kernels")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after the timed region, run one device copy of this many MiB "
                         "(a known-size reference for the HBM byte counters)")
    ap.add_argument("--summarize", metavar="DIR",
                    help="print a per-dispatch summary of a rocprofv3 output directory and exit")
    ap.add_argument("--pmc-traffic", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of this bench with "
                         "--copy-mib into per-kernel HBM bytes and print them as markdown")
    ap.add_argument("--pmc-summary", metavar="DIR",
                    help="per chain entry, the counters of one rocprofv3 --pmc run of this bench (averaged over "
                         "its steps) with the matrix-core busy fraction and wait fractions, as markdown")
    return ap.parse_args()


# GPU kernels of each chain entry, in launch order (a substring of each
# dispatch's kernel name; every library kernel lives in namespace optimus).
# A product whose contraction is split adds its reduction kernel.
_GEMM = ("gemm_",)
_GEMM_SPLIT = ("gemm_", "splitk_")
_LN_BWD = ("ln_bwd_kernel", "ln_bwd_reduce_kernel")
ENTRY_KERNELS = {"ln1_fwd": ("ln_fwd_kernel",), "qkv_fwd": _GEMM, "attn_fwd": ("attn_fwd_kernel",),
                 "oproj_fwd": _GEMM, "ln2_fwd": ("ln_fwd_kernel",), "mlp_up_fwd": _GEMM, "mlp_down_fwd": _GEMM,
                 "mlp_down_bwd_data": _GEMM, "mlp_down_bwd_weight": _GEMM, "mlp_up_bwd_data": _GEMM,
                 "mlp_up_bwd_weight": _GEMM, "ln2_bwd": _LN_BWD, "oproj_bwd_data": _GEMM,
                 "oproj_bwd_weight": _GEMM, "attn_bwd": ("attn_bwd_dq_kernel", "attn_bwd_dkdv_kernel"),
                 "qkv_bwd_data": _GEMM, "qkv_bwd_weight": _GEMM, "ln1_bwd": _LN_BWD}
DISPATCHES = {n: len(k) for n, k in ENTRY_KERNELS.items()}


def gemm_products(cfg):
    """Each GEMM entry's product as its workspace query takes it: ("fwd", M,
    N, K) for a forward or input-gradient product with output [M, N] and
    contraction K; ("wgrad", M, N, K) for the gradient dW[N, K] of a linear
    layer over M tokens."""
    Bn, S, H, nh, d, F = (cfg[k] for k in ("batch", "seq", "hidden", "heads", "head_dim", "mlp"))
    M, A = Bn * S, nh * d
    return {"qkv_fwd": ("fwd", M, 3 * A, H), "oproj_fwd": ("fwd", M, H, A), "mlp_up_fwd": ("fwd", M, F, H),
            "mlp_down_fwd": ("fwd", M, H, F), "mlp_down_bwd_data": ("fwd", M, F, H),
            "mlp_down_bwd_weight": ("wgrad", M, H, F), "mlp_up_bwd_data": ("fwd", M, H, F),
            "mlp_up_bwd_weight": ("wgrad", M, F, H), "oproj_bwd_data": ("fwd", M, A, H),
            "oproj_bwd_weight": ("wgrad", M, H, A), "qkv_bwd_data": ("fwd", M, H, 3 * A),
            "qkv_bwd_weight": ("wgrad", M, 3 * A, H)}


def _tile_of(pid, nb, tiles_m, tiles_n):
    """Output tile of workgroup pid in an unsplit GEMM grid of nb workgroups,
    in the kernels' order (workgroup i runs on XCD i % 8): with an even grid,
    two M-halves of four XCDs each, every XCD walking its block in groups of
    4 row tiles; otherwise one contiguous range of tiles per XCD, in groups
    of 8 row tiles."""
    xcd, local = pid & 7, pid >> 3
    if tiles_m % 2 == 0 and tiles_n % 4 == 0:
        rows_p, cols_x = tiles_m // 2, tiles_n // 4
        g, in_g = divmod(local, 4 * cols_x)
        gm = min(rows_p - 4 * g, 4)
        return (xcd >> 2) * rows_p + 4 * g + in_g % gm, (xcd & 3) * cols_x + in_g // gm
    per, rem = nb >> 3, nb & 7
    logical = xcd * (per + 1) + local if xcd < rem else rem * (per + 1) + (xcd - rem) * per + local
    g, in_g = divmod(logical, 8 * tiles_n)
    gm = min(tiles_m - 8 * g, 8)
    return 8 * g + in_g % gm, in_g // gm


def _split_item(pid, nb, tiles_m, tiles_n):
    """(split, row tile, column tile) of workgroup pid in a split grid: work
    items split-major and M-fastest, one contiguous range per XCD."""
    xcd, local = pid & 7, pid >> 3
    per, rem = nb >> 3, nb & 7
    item = xcd * (per + 1) + local if xcd < rem else rem * (per + 1) + (xcd - rem) * per + local
    split, t = divmod(item, tiles_m * tiles_n)
    return split, t % tiles_m, t // tiles_m


def fetch_floor(rows, cols, K, bm, bn, splits):
    """Operand bytes the eight L2s must fetch at least for one GEMM launch
    (output rows x cols, contraction K, bf16 operands): the workgroups of a
    round run together (one per CU, two for 128x128 tiles), the eighth of
    them on one XCD share its L2, and an operand panel (a tile row's or tile
    column's slice of the contraction) outlives neither its round nor its
    XCD.  Each round's distinct panels per XCD, summed."""
    per_round = 512 if (bm, bn) == (128, 128) else 256
    tm, tn = -(-rows // bm), -(-cols // bn)
    nb = tm * tn * splits
    kc = -(-K // splits) if splits > 1 else K
    if splits > 1:
        kc = -(-kc // 64) * 64
    total = 0
    for r0 in range(0, nb, per_round):
        panels = {}
        for pid in range(r0, min(nb, r0 + per_round)):
            sp, a, b = _split_item(pid, nb, tm, tn) if splits > 1 else (0, *_tile_of(pid, nb, tm, tn))
            klen = min(K - sp * kc, kc)
            rs, cs = panels.setdefault(pid & 7, (set(), set()))
            rs.add((a, sp, min(bm, rows - a * bm) * klen))
            cs.add((b, sp, min(bn, cols - b * bn) * klen))
        total += sum(2 * (sum(x[2] for x in rs) + sum(x[2] for x in cs)) for rs, cs in panels.values())
    return total


def gemm_fetch_floors(cfg):
    """fetch_floor of every GEMM entry under the library's own launch plan."""
    from paper_2408_03505_amd import binding as B
    out = {}
    for n, (kind, m, nn, k) in gemm_products(cfg).items():
        if kind == "wgrad":  # dW[nn, k] over m tokens
            bm, bn, sp = B.linear_plan(B.LAYOUT_WGRAD, m, nn, k)
            out[n] = fetch_floor(nn, k, m, bm, bn, sp)
        else:
            layout = B.LAYOUT_DGRAD if n.endswith("_bwd_data") else B.LAYOUT_FWD
            bm, bn, sp = B.linear_plan(layout, m, nn, k)
            out[n] = fetch_floor(m, nn, k, bm, bn, sp)
    return out


def use_config(cfg):
    """Set the dispatch map for the chain of workload cfg: a product the
    library splits (it asks for a workspace, which the chain provides) runs
    as two dispatches."""
    from paper_2408_03505_amd import binding as B
    global ENTRY_KERNELS, DISPATCHES
    ek = dict(ENTRY_KERNELS)
    for n, (kind, m, nn, k) in gemm_products(cfg).items():
        need = B.linear_workspace_bytes(m, nn, k) if kind == "fwd" else B.linear_bwd_weight_workspace_bytes(m, nn, k)
        ek[n] = _GEMM_SPLIT if need > 0 else _GEMM
    ENTRY_KERNELS = ek
    DISPATCHES = {n: len(k) for n, k in ek.items()}


def is_lib_kernel(name):
    """A kernel of the layer chain (the measurement reference kernels excluded)."""
    return "optimus::" in name and "calib_" not in name


def map_dispatches(lib):
    """Split library dispatches [(dispatch id, kernel name, value)] into chain
    steps and return per step a dict entry -> summed value; every dispatch's
    name is checked against the entry it is attributed to."""
    lib = sorted(lib)
    per_step = sum(DISPATCHES.values())
    if not lib or len(lib) % per_step:
        raise RuntimeError(f"{len(lib)} library dispatches is not a whole number of {per_step}-dispatch steps")
    steps = []
    for st in range(len(lib) // per_step):
        i, step = st * per_step, {}
        for n, kernels in ENTRY_KERNELS.items():
            for j, k in enumerate(kernels):
                if k not in lib[i + j][1]:
                    raise RuntimeError(f"step {st}: dispatch {lib[i + j][0]} ({lib[i + j][1][:80]}) is not {n}/{k}")
            step[n] = sum(v for _, _, v in lib[i:i + len(kernels)])
            i += len(kernels)
        steps.append(step)
    return steps


TRAFFIC_MD = os.path.join(ROOT, "profiles", "vit22b_layer_hbm_traffic.md")


# Sources each chain entry's kernels are built from (device code, the
# argument structs they receive and the launch geometry): traffic counters
# describe these files only.
_COMMON_SRC = ("common.hpp", "lds_dma.hpp", "kernels.hpp", "geometry.hpp")
_FAMILY_SRC = {"gemm": ("gemm.hip",), "attention": ("attention.hip",), "layernorm": ("layernorm.hip",)}


def entry_family(entry):
    if entry.startswith("ln"):
        return "layernorm"
    if entry.startswith("attn"):
        return "attention"
    return "gemm"


def source_hash(family):
    """sha256 over the sources of one kernel family."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2408_03505_amd", "csrc")
    for f in sorted(_FAMILY_SRC[family] + _COMMON_SRC):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def _latest_rows(d, pattern):
    """Rows of the newest rocprofv3 csv matching pattern under d (an output
    folder may still hold the files of earlier runs)."""
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", pattern), recursive=True)
    if not files:
        return []
    with open(max(files, key=os.path.getmtime)) as fh:
        return list(csv.DictReader(fh))


def _counter_rows(d):
    return _latest_rows(d, "*counter_collection.csv")


def pmc_entries(d):
    """Per chain entry and counter, the counter's average over the steps of
    one rocprofv3 --pmc run (each dispatch's value as reported, i.e. summed
    over the GPU's instances)."""
    rows = _counter_rows(d)
    out = {}
    for ctr in sorted({r["Counter_Name"] for r in rows}):
        steps = map_dispatches([(int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"]))
                                for r in rows if r["Counter_Name"] == ctr and is_lib_kernel(r["Kernel_Name"])])
        for n in DISPATCHES:
            out.setdefault(n, {})[ctr] = sum(st[n] for st in steps) / len(steps)
    return out


def pmc_utilisation(c, xcds=8, simds=1024):
    """Derived fractions of one entry's counters: matrix-core busy cycles
    over (GPU-active cycles of one XCD x SIMDs), and the waves' instruction
    waits over their cycles."""
    out = {}
    if "SQ_VALU_MFMA_BUSY_CYCLES" in c and "GRBM_GUI_ACTIVE" in c:
        out["mfma_busy"] = c["SQ_VALU_MFMA_BUSY_CYCLES"] / (c["GRBM_GUI_ACTIVE"] / xcds * simds)
    if "SQ_WAVE_CYCLES" in c and c["SQ_WAVE_CYCLES"] > 0:
        for k in ("SQ_WAIT_INST_ANY", "SQ_WAIT_INST_LDS", "SQ_WAIT_ANY"):
            if k in c:
                out[k.lower().replace("sq_", "") + "_per_wave_cycle"] = c[k] / c["SQ_WAVE_CYCLES"]
    return out


def pmc_traffic(fetch_dir, write_dir, copy_bytes):
    """Per-entry HBM bytes per launch from FETCH_SIZE / WRITE_SIZE (KiB per
    dispatch), each scaled by what the counter reports for a device copy of
    copy_bytes in the same run."""
    vals = {}
    for d, ctr in ((fetch_dir, "FETCH_SIZE"), (write_dir, "WRITE_SIZE")):
        rows = [r for r in _counter_rows(d) if r["Counter_Name"] == ctr]
        copies = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]]
        scale = copy_bytes / (max(copies) * 1024.0)
        steps = map_dispatches([(int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"]))
                                for r in rows if is_lib_kernel(r["Kernel_Name"])])
        out = {n: sum(st[n] for st in steps) * 1024.0 * scale / len(steps) for n in DISPATCHES}
        vals[ctr] = (out, scale)
    return vals


def read_traffic(entry):
    """HBM bytes per launch of one entry from the committed profile, or None
    when the profile is missing or was taken on different kernel sources."""
    if not os.path.exists(TRAFFIC_MD):
        return None
    text = open(TRAFFIC_MD).read()
    fam = entry_family(entry)
    if f"source-sha256 {fam}: {source_hash(fam)}" not in text:
        return None
    for line in text.splitlines():
        cells = [c.strip() for c in line.strip().strip("|").split("|")]
        if len(cells) >= 4 and cells[0] == entry:
            try:
                return float(cells[3])
            except ValueError:
                return None
    return None


def summarize(d, skip_steps=0):
    """Per (kernel, grid) duration and counter summary of a rocprofv3 csv run;
    for a kernel trace of this bench also the average duration of each chain
    entry (dispatches mapped by launch order, the first skip_steps steps,
    i.e. the warm-up, left out)."""
    import re

    def rows(pattern):
        return _latest_rows(d, pattern)

    def short(name):
        name = re.sub(r"\(anonymous namespace\)::", "", name)
        name = re.sub(r"\(.*\)$", "", name)
        return name.replace("optimus::", "").replace("void ", "")

    trace = rows("*kernel_trace.csv")
    lib = [(int(r["Dispatch_Id"]), r["Kernel_Name"], (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
           for r in trace if is_lib_kernel(r["Kernel_Name"])]
    if lib:
        steps = map_dispatches(lib)[skip_steps:]
        print(f"per chain entry, steps {skip_steps}..{skip_steps + len(steps) - 1} (device time of its dispatches):\n")
        print("| entry | dispatches | avg us | min us | max us |")
        print("|---|---|---|---|---|")
        for n in DISPATCHES:
            v = [st[n] for st in steps]
            print(f"| {n} | {DISPATCHES[n]} | {np.mean(v):.2f} | {min(v):.2f} | {max(v):.2f} |")
        print()
    groups = {}
    for r in trace:
        key = (short(r["Kernel_Name"]), int(r.get("Grid_Size_X", r.get("Grid_Size", 0)) or 0))
        groups.setdefault(key, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    if groups:
        print("| kernel | grid | calls | avg us | min us | max us |")
        print("|---|---|---|---|---|---|")
        for (k, g), v in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
            print(f"| {k} | {g} | {len(v)} | {np.mean(v):.2f} | {min(v):.2f} | {max(v):.2f} |")
    pmc = rows("*counter_collection.csv")
    if pmc:
        agg = {}
        for r in pmc:
            key = (short(r["Kernel_Name"]), int(r.get("Grid_Size", 0) or 0), r["Counter_Name"])
            agg.setdefault(key, []).append(float(r["Counter_Value"]))
        print("\n| kernel | grid | counter | dispatches | avg value |")
        print("|---|---|---|---|---|")
        for (k, g, c), v in sorted(agg.items()):
            print(f"| {k} | {g} | {c} | {len(v)} | {np.mean(v):.1f} |")


def measure_ceilings(dev, reps=3):
    """Sustained rates of the library's two reference kernels on this GPU: an
    MFMA-only bf16 loop (changing operands) and a 1 GiB device copy."""
    from paper_2408_03505_amd import binding as B

    def best_ms(fn):
        fn()
        times = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1))
        return min(times)

    blocks, iters = 1024, 2000
    out = torch.empty(blocks * 256, dtype=torch.float32, device=dev)
    ms = best_ms(lambda: B.enc_calib_mfma(blocks, iters, out))
    mfma = B.calib_mfma_flops(blocks, iters) / (ms * 1e-3) / 1e12
    n = 1 << 30
    src = torch.ones(n, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    ms = best_ms(lambda: B.enc_calib_copy(src, dst))
    copy = 2 * n / (ms * 1e-3) / 1e9
    del src, dst
    props = torch.cuda.get_device_properties(dev)
    return {"mfma_bf16_tflops": round(mfma, 1), "copy_gbs": round(copy, 1),
            "compute_units": props.multi_processor_count,
            "note": "best of 3; MFMA-only loop of v_mfma_f32_32x32x16_bf16 with changing operands; "
                    "copy counts bytes read plus bytes written"}


FWD_ENTRIES = ("ln1_fwd", "qkv_fwd", "attn_fwd", "oproj_fwd", "ln2_fwd", "mlp_up_fwd", "mlp_down_fwd")


def synthetic_tp_trace(seed=0, n=400):
    """LLM timeline of alternating computation and tensor-parallel bubbles:
    bubbles uniform in [200, 400] us (about 300 us on average, the TP bubble
    length the paper profiles), computation uniform in [300, 900] us."""
    rng = np.random.default_rng(seed)
    lengths, bubble = [], []
    for _ in range(n):
        lengths += [float(rng.uniform(300, 900)), float(rng.uniform(200, 400))]
        bubble += [False, True]
    return lengths, bubble


def bubble_fit(p50, seed=0):
    """Pack the chain's forward and backward kernels (per-kernel p50, chain
    order) into the synthetic TP-bubble trace with the library's packer."""
    from paper_2408_03505_amd import binding as B
    lengths, bubble = synthetic_tp_trace(seed)
    starts = np.concatenate([[0.0], np.cumsum(lengths)[:-1]])
    out = {}
    for part, names in (("fwd", [n for n in p50 if n in FWD_ENTRIES]),
                        ("bwd", [n for n in p50 if n not in FWD_ENTRIES])):
        kus = [p50[n] for n in names]
        where, off, placed = B.enc_schedule_kernels(kus, lengths, bubble)
        r = {"kernels": len(names), "placed": placed, "kernel_us": round(sum(kus), 1)}
        if placed:
            used = sorted(set(where[:placed]))
            r["bubbles_used"] = len(used)
            r["fill"] = round(sum(kus[:placed]) / sum(lengths[j] for j in used), 3)
            last = placed - 1
            r["span_us"] = round(float(starts[where[last]] + off[last] + kus[last] - starts[where[0]]), 1)
        if placed < len(names):
            r["blocked_at"] = names[placed]
            r["blocked_kernel_us"] = round(kus[placed], 1)
        out[part] = r
    return out


def time_chain(chain, steps, warmup):
    """Per-entry p50 (us) of a chain, events around every launch."""
    names = [n for n, _ in chain.kernels]
    for _ in range(warmup):
        for _, fn in chain.kernels:
            fn()
    torch.cuda.synchronize()
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in names]
          for _ in range(steps)]
    for k in range(steps):
        for i, (_, fn) in enumerate(chain.kernels):
            ev[k][i][0].record()
            fn()
            ev[k][i][1].record()
    torch.cuda.synchronize()
    return {n: float(np.median([ev[k][i][0].elapsed_time(ev[k][i][1]) * 1e3 for k in range(steps)]))
            for i, n in enumerate(names)}


def time_isolated(chain, p50_chain, reps=20, warmup=3):
    """Every chain entry launched reps times back to back on its own (its
    inputs stay warm in the caches), p50 and p90 in us, beside its p50
    inside the chain."""
    out = {}
    for n, fn in chain.kernels:
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in ev:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        us = [a.elapsed_time(b) * 1e3 for a, b in ev]
        out[n] = {"p50_us": round(float(np.median(us)), 2), "p90_us": round(float(np.percentile(us, 90)), 2),
                  "chain_p50_us": round(p50_chain[n], 2)}
    return out


MEM_BOUND = ("ln1_fwd", "ln2_fwd", "ln2_bwd", "ln1_bwd")


def time_flushed(chain, work, reps=20, flush_mib=512):
    """The memory-bound entries timed on their own: warm (launches back to
    back) and cold (each launch after writing a 512 MiB buffer, which evicts
    the 256 MB Infinity Cache and the L2s).  p50 of reps launches each."""
    fns = dict(chain.kernels)
    flush = torch.empty(flush_mib << 20, dtype=torch.uint8, device=chain.x.device)
    out = {}
    for n in MEM_BOUND:
        fn = fns[n]
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        res = {}
        for mode in ("warm", "flushed"):
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
            for i in range(reps):
                if mode == "flushed":
                    flush.fill_(i & 255)
                ev[i][0].record()
                fn()
                ev[i][1].record()
            torch.cuda.synchronize()
            us = float(np.median([a.elapsed_time(b) * 1e3 for a, b in ev]))
            res[f"{mode}_p50_us"] = round(us, 2)
            res[f"{mode}_gbs"] = round(work[n][1] / (us * 1e-6) / 1e9, 1)
        out[n] = res
    del flush
    return out


def time_configs(main, dev, seed, steps=10, warmup=3):
    """The layer chain at every other workload: step time (sum of per-kernel
    p50), rate, and the slowest kernel."""
    from paper_2408_03505_amd.synthetic import CONFIGS, layer_inputs
    out = {}
    for name, cfg in CONFIGS.items():
        if name == main:
            continue
        x, params, dout = layer_inputs(cfg, seed=seed)
        ch = Chain(cfg, x.to(dev), {n: params[n].to(dev) for n in params}, dout.to(dev))
        p50 = time_chain(ch, steps=steps, warmup=warmup)
        ms = sum(p50.values()) / 1e3
        worst = max(p50, key=p50.get)
        out[name] = {"sum_kernel_p50_ms": round(ms, 4),
                     "tflops": round(step_flops(cfg) / (ms * 1e-3) / 1e12, 1),
                     "max_kernel_p50_us": round(p50[worst], 2), "max_kernel": worst}
        del ch
    return out


def time_parallel_block(cfg, dev, steps=10, warmup=3):
    """Forward+backward of the ViT-22B-style parallel block (composite entry
    points) at the same shape, plus its two QK-norm kernels on their own."""
    from paper_2408_03505_amd import binding as B
    from paper_2408_03505_amd.synthetic import PPARAM_ORDER, parallel_block_inputs
    x, p, d = parallel_block_inputs(cfg, seed=0)
    gx, gd = x.to(dev), d.to(dev)
    gp = {n: p[n].to(dev) for n in PPARAM_ORDER}
    out, saved = B.encoder_parallel_fwd(cfg, gp, gx)
    dx, grads = B.encoder_parallel_bwd(cfg, gp, gx, saved, gd)
    ws = torch.empty(B.parallel_workspace_bytes(cfg), dtype=torch.uint8, device=dev)

    def step():
        B.encoder_parallel_fwd(cfg, gp, gx, out=out, saved=saved)
        B.encoder_parallel_bwd(cfg, gp, gx, saved, gd, grads=grads, dx=dx, ws=ws)

    def p50_ms(fn, n):
        ts = []
        for _ in range(n):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts))

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    ms = p50_ms(step, steps)
    flops = step_flops(cfg)
    v = B.parallel_saved_views(cfg, saved)
    nh, dd, M = cfg["heads"], cfg["head_dim"], cfg["batch"] * cfg["seq"]
    qkvn, st = v["qkvn"].clone(), v["qkstats"].clone()
    fwd = lambda: B.enc_qk_norm_fwd(nh, dd, v["qkv"], gp["qn_g"], gp["qn_b"], gp["kn_g"], gp["kn_b"],  # noqa: E731
                                    cfg["ln_eps"], qkvn=qkvn, stats=st)
    dq = torch.empty_like(qkvn)
    qg = {n: torch.empty(dd, dtype=torch.float32, device=dev) for n in ("qn_g", "qn_b", "kn_g", "kn_b")}
    bwd = lambda: B.enc_qk_norm_bwd(nh, dd, qkvn, v["qkv"], st, gp["qn_g"], gp["kn_g"], dqkv=dq,  # noqa: E731
                                    grads=qg)
    for f in (fwd, bwd):
        f()
    fwd_us, bwd_us = p50_ms(fwd, 20) * 1e3, p50_ms(bwd, 20) * 1e3
    A = nh * dd
    fwd_bytes = M * 3 * A * 2 * 2 + M * nh * 16            # read qkv, write qkvn, stats
    bwd_bytes = M * 3 * A * 2 * 2 + M * 2 * A * 2 + M * nh * 16  # read dqkvn, q/k, stats; write dqkv
    return {"ms_per_step": round(ms, 4), "tflops": round(flops / (ms * 1e-3) / 1e12, 2),
            "frac_of_bf16_peak": round(flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "qk_norm_fwd": {"p50_us": round(fwd_us, 2), "gbs": round(fwd_bytes / (fwd_us * 1e-6) / 1e9, 1)},
            "qk_norm_bwd": {"p50_us": round(bwd_us, 2), "gbs": round(bwd_bytes / (bwd_us * 1e-6) / 1e9, 1)},
            "note": "ViT-22B-style block (shared LN, parallel branches, QK LayerNorm, no QKV bias) at the same "
                    "shape; composite entry points, p50 of 10 steps; flops counted as for the sequential layer"}


def corun(chain, p50_alone, dev, steps=5, n=8192):
    """The encoder chain on one stream while a loop of n x n x n bf16 GEMMs
    (torch.matmul, standing in for the LLM's computation) runs on another;
    per-kernel p50 under load against p50_alone, and the load's own rate
    alone and beside the chain.  Both streams have the default priority."""
    a = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
    b = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
    c = torch.empty(n, n, device=dev, dtype=torch.bfloat16)
    load, enc = torch.cuda.Stream(device=dev), torch.cuda.Stream(device=dev)
    gemm_flops = 2.0 * n ** 3

    def run_load(k):
        with torch.cuda.stream(load):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(k):
                torch.matmul(a, b, out=c)
            e1.record()
        return e0, e1

    e0, e1 = run_load(3)
    torch.cuda.synchronize()
    e0, e1 = run_load(20)
    torch.cuda.synchronize()
    load_alone = 20 * gemm_flops / (e0.elapsed_time(e1) * 1e-3) / 1e12
    names = [nm for nm, _ in chain.kernels]
    step_ms_alone = sum(p50_alone.values()) / 1e3
    # enough load to outlast the chain even if sharing the GPU slows it eightfold
    k_load = max(8, int(8.0 * steps * step_ms_alone / max(1e-3, gemm_flops / (load_alone * 1e12) * 1e3)))
    torch.cuda.synchronize()
    l0, l1 = run_load(k_load)
    ev = []
    with torch.cuda.stream(enc):
        s0 = torch.cuda.Event(enable_timing=True)
        s0.record()
        for _ in range(steps):
            row = []
            for _, fn in chain.kernels:
                k0, k1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                k0.record()
                fn()
                k1.record()
                row.append((k0, k1))
            ev.append(row)
        s1 = torch.cuda.Event(enable_timing=True)
        s1.record()
    torch.cuda.synchronize()
    per = {nm: float(np.median([ev[k][i][0].elapsed_time(ev[k][i][1]) * 1e3 for k in range(steps)]))
           for i, nm in enumerate(names)}
    enc_ms = s0.elapsed_time(s1) / steps
    load_busy = k_load * gemm_flops / (l0.elapsed_time(l1) * 1e-3) / 1e12
    covered = l0.elapsed_time(s0) >= 0 and s1.elapsed_time(l1) >= 0  # the load spans the whole chain
    return {"load": f"bf16 GEMM {n}x{n}x{n} (torch.matmul) looped on a second stream, {k_load} launches",
            "load_covers_encoder": bool(covered),
            "encoder_step_ms_alone": round(step_ms_alone, 4), "encoder_step_ms_corun": round(enc_ms, 4),
            "step_slowdown": round(enc_ms / step_ms_alone, 3),
            "kernel_slowdown": {nm: round(per[nm] / p50_alone[nm], 2) for nm in names},
            "load_tflops_alone": round(load_alone, 1), "load_tflops_corun": round(load_busy, 1)}


def cu_mask_words(per_word, words=8):
    """A CU mask (32-bit words) with per_word bits set in each word, word w
    holding bits w, w + 8, w + 16, ... (residue w mod 8).  Whichever way the
    runtime spreads mask bits over MI355X's eight XCDs (32 consecutive bits
    per XCD, or bit i on XCD i mod 8), every XCD keeps per_word CUs of the
    mask and 32 - per_word of its complement, so no XCD is left without CUs
    for either stream."""
    assert 1 <= per_word <= 4
    mask = [0] * words
    for w in range(words):
        for k in range(per_word):
            mask[w] |= 1 << (w % 8 + 8 * k)
    return mask


def _hip_runtime():
    """The HIP runtime library this process already uses (torch's)."""
    import ctypes
    paths = sorted({ln.split()[-1] for ln in open("/proc/self/maps") if "libamdhip64" in ln})
    if not paths:
        raise RuntimeError("no HIP runtime mapped in this process")
    return ctypes.CDLL(paths[0])


def corun_masked(chain, p50_alone, dev, per_word=4, steps=3, n=8192):
    """CU-masked co-run: the encoder chain on a stream restricted to a slice
    of the CUs (per_word bits of every 32-bit mask word: 32 of 256 CUs for
    per_word = 4) and the GEMM load of corun() on a stream restricted to the
    complement.  Reports the chain's step time on the slice alone and beside
    the load, and the load's rate on the complement alone and beside the
    chain.  Both streams are created with the default priority."""
    import ctypes
    hip = _hip_runtime()
    hip.hipExtStreamCreateWithCUMask.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint32,
                                                 ctypes.POINTER(ctypes.c_uint32)]
    hip.hipExtStreamGetCUMask.argtypes = [ctypes.c_void_p, ctypes.c_uint32, ctypes.POINTER(ctypes.c_uint32)]
    hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
    ncu = torch.cuda.get_device_properties(dev).multi_processor_count
    words = (ncu + 31) // 32
    if words != 8:
        return {"skipped": f"the mask layout assumes 256 CUs in 8 XCDs (this device has {ncu} CUs)"}
    enc_mask = cu_mask_words(per_word, words)
    load_mask = [(~m) & 0xFFFFFFFF for m in enc_mask]
    handles = []

    def make(mask):
        arr = (ctypes.c_uint32 * words)(*mask)
        h = ctypes.c_void_p()
        err = hip.hipExtStreamCreateWithCUMask(ctypes.byref(h), words, arr)
        if err != 0:
            raise RuntimeError(f"hipExtStreamCreateWithCUMask failed ({err})")
        handles.append(h)
        got = (ctypes.c_uint32 * words)()
        hip.hipExtStreamGetCUMask(h, words, got)
        return torch.cuda.ExternalStream(h.value, device=dev), sum(bin(v).count("1") for v in got)

    try:
        enc, enc_cus = make(enc_mask)
        load, load_cus = make(load_mask)
        a = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
        b = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
        c = torch.empty(n, n, device=dev, dtype=torch.bfloat16)
        gemm_flops = 2.0 * n ** 3

        def run_load(k):
            with torch.cuda.stream(load):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(k):
                    torch.matmul(a, b, out=c)
                e1.record()
            return e0, e1

        def run_chain(k):
            with torch.cuda.stream(enc):
                s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                s0.record()
                for _ in range(k):
                    for _, fn in chain.kernels:
                        fn()
                s1.record()
            return s0, s1

        torch.cuda.synchronize()
        run_chain(1)  # warm-up on the slice
        torch.cuda.synchronize()
        s0, s1 = run_chain(steps)
        torch.cuda.synchronize()
        enc_alone = s0.elapsed_time(s1) / steps
        run_load(2)
        torch.cuda.synchronize()
        e0, e1 = run_load(10)
        torch.cuda.synchronize()
        load_alone = 10 * gemm_flops / (e0.elapsed_time(e1) * 1e-3) / 1e12
        k_load = max(10, int(1.5 * steps * enc_alone / (gemm_flops / (load_alone * 1e12) * 1e3)))
        torch.cuda.synchronize()
        l0, l1 = run_load(k_load)
        s0, s1 = run_chain(steps)
        torch.cuda.synchronize()
        enc_busy = s0.elapsed_time(s1) / steps
        load_busy = k_load * gemm_flops / (l0.elapsed_time(l1) * 1e-3) / 1e12
        covered = l0.elapsed_time(s0) >= 0 and s1.elapsed_time(l1) >= 0
        step_full = sum(p50_alone.values()) / 1e3
        return {"encoder_mask": [f"{m:08x}" for m in enc_mask], "encoder_cus": enc_cus, "load_cus": load_cus,
                "load": f"bf16 GEMM {n}x{n}x{n} (torch.matmul) looped on the complement, {k_load} launches",
                "load_covers_encoder": bool(covered),
                "encoder_step_ms_full_gpu": round(step_full, 4),
                "encoder_step_ms_slice_alone": round(enc_alone, 4),
                "encoder_step_ms_slice_with_load": round(enc_busy, 4),
                "slice_isolation": round(enc_busy / enc_alone, 3),
                "load_tflops_complement_alone": round(load_alone, 1),
                "load_tflops_complement_with_encoder": round(load_busy, 1)}
    finally:
        torch.cuda.synchronize()
        for h in handles:
            hip.hipStreamDestroy(h)


def time_whole_encoder(cfg, layers, dev, steps=2, warmup=1, img=224, patch=14, channels=3):
    """Forward+backward of a whole ViT encoder on one micro-batch: patch
    embedding of img x img images (no class token), `layers` sequential
    layers (distinct weights) and a final LayerNorm, on this one GPU."""
    from paper_2408_03505_amd import binding as B
    Bn, H = cfg["batch"], cfg["hidden"]
    if (img // patch) ** 2 != cfg["seq"]:
        return {"skipped": f"seq {cfg['seq']} is not ({img}/{patch})^2"}
    K, kp = channels * patch * patch, B.patch_kp(channels, patch)
    bf, f32 = dict(dtype=torch.bfloat16, device=dev), dict(dtype=torch.float32, device=dev)
    torch.cuda.reset_peak_memory_stats(dev)
    images = torch.randn(Bn, channels, img, img, **bf)
    w_pe = torch.zeros(H, kp, **bf)
    w_pe[:, :K].normal_(0, 0.02)
    b_pe, pos = torch.empty(H, **bf).normal_(0, 0.02), torch.empty(cfg["seq"], H, **bf).normal_(0, 0.02)
    shapes = B.param_shapes(cfg)
    params = [{n: torch.empty(shapes[n], **bf).normal_(1.0 if n in ("ln1_g", "ln2_g") else 0.0, 0.02)
               for n in B.PARAM_ORDER} for _ in range(layers)]
    grads = [{n: torch.empty(shapes[n], **f32) for n in B.PARAM_ORDER} for _ in range(layers)]
    lnf_g, lnf_b = torch.ones(H, **bf), torch.zeros(H, **bf)
    lnf_grads = (torch.empty(H, **f32), torch.empty(H, **f32))
    dout = torch.randn(Bn * cfg["seq"], H, **bf)
    x0, patches = B.enc_patch_embed_fwd(images, patch, w_pe, b_pe, pos)
    out, saved = B.encoder_stack_fwd(cfg, params, lnf_g, lnf_b, x0)
    ws = torch.empty(B.stack_workspace_bytes(cfg, layers), dtype=torch.uint8, device=dev)
    dx0 = torch.empty_like(x0)
    pe_grads = B.enc_patch_embed_bwd(tuple(images.shape), patch, dout, patches, False)

    def step():
        B.enc_patch_embed_fwd(images, patch, w_pe, b_pe, pos, patches=patches, x0=x0)
        B.encoder_stack_fwd(cfg, params, lnf_g, lnf_b, x0, out=out, saved=saved)
        B.encoder_stack_bwd(cfg, params, lnf_g, x0, saved, dout, grads=grads, lnf_grads=lnf_grads, dx0=dx0, ws=ws)
        B.enc_patch_embed_bwd(tuple(images.shape), patch, dx0, patches, False, grads=pe_grads)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    M = Bn * cfg["seq"]
    flops = layers * step_flops(cfg) + 3 * 2 * M * H * K
    return {"layers": layers, "image": f"{img}x{img}, {patch}x{patch} patches, {channels} channels",
            "ms_per_step": round(ms, 2), "tflops": round(flops / (ms * 1e-3) / 1e12, 1),
            "frac_of_bf16_peak": round(flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "peak_memory_gb": round(torch.cuda.max_memory_allocated(dev) / 1e9, 1),
            "note": "patch embedding + layers + final LayerNorm, forward and backward with fp32 gradients of "
                    "every parameter, one micro-batch, all on this GPU"}


class Chain:
    """Preallocated buffers and the kernel-by-kernel layer step."""

    def __init__(self, cfg, x, params, dout):
        from paper_2408_03505_amd import binding as B
        self.B, self.cfg, self.x, self.p, self.dout = B, cfg, x, params, dout
        Bn, S, H, nh, d, F = (cfg[k] for k in ("batch", "seq", "hidden", "heads", "head_dim", "mlp"))
        M, A = Bn * S, nh * d
        dev = x.device
        bf = dict(dtype=torch.bfloat16, device=dev)
        f32 = dict(dtype=torch.float32, device=dev)
        e = torch.empty
        self.t = t = {
            "y1": e((M, H), **bf), "mean1": e((M,), **f32), "rstd1": e((M,), **f32), "qkv": e((M, 3 * A), **bf),
            "o": e((M, A), **bf), "lse": e((Bn, nh, S), **f32), "h": e((M, H), **bf), "y2": e((M, H), **bf),
            "mean2": e((M,), **f32), "rstd2": e((M,), **f32), "u": e((M, F), **bf), "g": e((M, F), **bf),
            "out": e((M, H), **bf), "du": e((M, F), **bf), "dy2": e((M, H), **bf), "dh": e((M, H), **bf),
            "do": e((M, A), **bf), "dqkv": e((M, 3 * A), **bf), "dy1": e((M, H), **bf), "dx": e((M, H), **bf),
        }
        self.g = {n: torch.zeros(tuple(params[n].shape), **f32) for n in params}
        self.ln_ws = e((B.ln_bwd_workspace_bytes(M, H),), dtype=torch.uint8, device=dev)
        self.attn_ws = e((B.attn_bwd_workspace_bytes(Bn, S, nh, d),), dtype=torch.uint8, device=dev)
        # one workspace for the four weight gradients (split token sums of small outputs)
        wg = max(B.linear_bwd_weight_workspace_bytes(M, n, k) for n, k in ((H, F), (F, H), (H, A), (3 * A, H)))
        self.wg_ws = e((max(wg, 256),), dtype=torch.uint8, device=dev)
        self.M, self.A = M, A
        self.kernels = self._kernels()

    def _kernels(self):
        B, c, x, p, dout, t, g = self.B, self.cfg, self.x, self.p, self.dout, self.t, self.g
        Bn, S, nh, d, eps = c["batch"], c["seq"], c["heads"], c["head_dim"], c["ln_eps"]
        return [
            ("ln1_fwd", lambda: B.enc_ln_fwd(x, p["ln1_g"], p["ln1_b"], eps, t["y1"], t["mean1"], t["rstd1"])),
            ("qkv_fwd", lambda: B.enc_qkv_fwd(t["y1"], p["w_qkv"], p["b_qkv"], t["qkv"])),
            ("attn_fwd", lambda: B.enc_attn_fwd(Bn, S, nh, d, t["qkv"], t["o"], t["lse"])),
            ("oproj_fwd", lambda: B.enc_oproj_fwd(t["o"], p["w_o"], p["b_o"], x, t["h"])),
            ("ln2_fwd", lambda: B.enc_ln_fwd(t["h"], p["ln2_g"], p["ln2_b"], eps, t["y2"], t["mean2"], t["rstd2"])),
            ("mlp_up_fwd", lambda: B.enc_mlp_up_fwd(t["y2"], p["w_1"], p["b_1"], t["u"], t["g"])),
            ("mlp_down_fwd", lambda: B.enc_mlp_down_fwd(t["g"], p["w_2"], p["b_2"], t["h"], t["out"])),
            ("mlp_down_bwd_data", lambda: B.enc_mlp_down_bwd_data(dout, p["w_2"], t["u"], t["du"])),
            ("mlp_down_bwd_weight", lambda: B.enc_mlp_down_bwd_weight(dout, t["g"], g["w_2"], g["b_2"],
                                                                                  ws=self.wg_ws)),
            ("mlp_up_bwd_data", lambda: B.enc_mlp_up_bwd_data(t["du"], p["w_1"], t["dy2"])),
            ("mlp_up_bwd_weight", lambda: B.enc_mlp_up_bwd_weight(t["du"], t["y2"], g["w_1"], g["b_1"],
                                                                              ws=self.wg_ws)),
            ("ln2_bwd", lambda: B.enc_ln_bwd(t["dy2"], t["h"], t["mean2"], t["rstd2"], p["ln2_g"], dout, t["dh"],
                                             g["ln2_g"], g["ln2_b"], ws=self.ln_ws)),
            ("oproj_bwd_data", lambda: B.enc_oproj_bwd_data(t["dh"], p["w_o"], t["do"])),
            ("oproj_bwd_weight", lambda: B.enc_oproj_bwd_weight(t["dh"], t["o"], g["w_o"], g["b_o"],
                                                                            ws=self.wg_ws)),
            ("attn_bwd", lambda: B.enc_attn_bwd(Bn, S, nh, d, t["qkv"], t["o"], t["lse"], t["do"], t["dqkv"],
                                                ws=self.attn_ws)),
            ("qkv_bwd_data", lambda: B.enc_qkv_bwd_data(t["dqkv"], p["w_qkv"], t["dy1"])),
            ("qkv_bwd_weight", lambda: B.enc_qkv_bwd_weight(t["dqkv"], t["y1"], g["w_qkv"], g["b_qkv"],
                                                                          ws=self.wg_ws)),
            ("ln1_bwd", lambda: B.enc_ln_bwd(t["dy1"], x, t["mean1"], t["rstd1"], p["ln1_g"], t["dh"], t["dx"],
                                             g["ln1_g"], g["ln1_b"], ws=self.ln_ws)),
        ]


def kernel_work(cfg):
    """Algorithmic work of each kernel: (flops, bytes)."""
    Bn, S, H, nh, d, F = (cfg[k] for k in ("batch", "seq", "hidden", "heads", "head_dim", "mlp"))
    M, A = Bn * S, nh * d
    att = 4 * Bn * nh * S * S * d
    ln_f = 4 * M * H + 8 * M + 4 * H
    ln_b = 8 * M * H + 8 * M + 2 * H + 8 * H
    gemm = lambda m, n, k: 2 * m * n * k  # noqa: E731
    return {
        "ln1_fwd": (0, ln_f), "qkv_fwd": (gemm(M, 3 * A, H), 2 * (M * H + 3 * A * H + M * 3 * A)),
        "attn_fwd": (att, 2 * (3 * M * A + M * A) + 4 * Bn * nh * S),
        "oproj_fwd": (gemm(M, H, A), 2 * (M * A + H * A + 2 * M * H)), "ln2_fwd": (0, ln_f),
        "mlp_up_fwd": (gemm(M, F, H), 2 * (M * H + F * H + 2 * M * F)),
        "mlp_down_fwd": (gemm(M, H, F), 2 * (M * F + H * F + 2 * M * H)),
        "mlp_down_bwd_data": (gemm(M, F, H), 2 * (M * H + H * F + 2 * M * F)),
        "mlp_down_bwd_weight": (gemm(H, F, M), 2 * (M * H + M * F) + 4 * (H * F + H)),
        "mlp_up_bwd_data": (gemm(M, H, F), 2 * (M * F + F * H + M * H)),
        "mlp_up_bwd_weight": (gemm(F, H, M), 2 * (M * F + M * H) + 4 * (F * H + F)),
        "ln2_bwd": (0, ln_b), "oproj_bwd_data": (gemm(M, A, H), 2 * (M * H + H * A + M * A)),
        "oproj_bwd_weight": (gemm(H, A, M), 2 * (M * H + M * A) + 4 * (H * A + H)),
        "attn_bwd": (2 * att, 2 * (3 * M * A + 2 * M * A + 3 * M * A) + 4 * Bn * nh * S),
        "qkv_bwd_data": (gemm(M, H, 3 * A), 2 * (M * 3 * A + 3 * A * H + M * H)),
        "qkv_bwd_weight": (gemm(3 * A, H, M), 2 * (M * 3 * A + M * H) + 4 * (3 * A * H + 3 * A)),
        "ln1_bwd": (0, ln_b),
    }


def step_flops(cfg):
    """Algorithmic flops of one layer forward + backward (three times the
    forward: the backward has two products per forward product)."""
    return sum(f for f, _ in kernel_work(cfg).values())


def hardware_flops(cfg):
    """Flops the kernels execute where they differ from the algorithmic
    count: the attention backward recomputes S (in both of its kernels) and
    dP (in both), so it runs seven 2*B*heads*S^2*d products (dQ kernel: S,
    dP, dQ; dK/dV kernel: S, dP, dV, dK) against the four counted."""
    Bn, S, nh, d = (cfg[k] for k in ("batch", "seq", "heads", "head_dim"))
    return {"attn_bwd": 7 * 2 * Bn * nh * S * S * d}


def cpu_model():
    """The host CPU's model name (first processor in /proc/cpuinfo)."""
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.lower().startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def _oracle_seconds(cfg, x, params, dout, budget_s, max_seqs=None):
    """Time the float64 oracle's forward+backward on whole sequences of cfg,
    one after another, until the budget would be exceeded (at least one).
    Returns (flops, seconds, sequences)."""
    import oracle

    S = cfg["seq"]
    p64 = {n: params[n].to(torch.float64).numpy() for n in params}
    one = dict(cfg, batch=1)
    f1 = 3 * oracle.layer_flops(one)
    limit = cfg["batch"] if max_seqs is None else min(cfg["batch"], max_seqs)
    done, t_used = 0, 0.0
    while done < limit:
        xs = x[done * S:(done + 1) * S].to(torch.float64).numpy()
        ds = dout[done * S:(done + 1) * S].to(torch.float64).numpy()
        t0 = time.perf_counter()
        out, saved = oracle.layer_fwd(one, p64, xs)
        oracle.layer_bwd(one, p64, xs, saved, ds)
        t_used += time.perf_counter() - t0
        done += 1
        if t_used + t_used / done > budget_s:
            break
    return f1 * done, t_used, done


def cpu_baseline(cfg, x, params, dout, budget_s, name=None, seed=0, configs=None):
    """The float64 oracle (numpy with the host BLAS's threads for matmul,
    scipy for erf; as it stands, not tuned) timed on the host cores: the
    headline on whole sequences of the benchmarked workload within the time
    budget; one sequence of every other workload with all threads; and one
    sequence of the three ViT-sized workloads on a single thread."""
    from threadpoolctl import threadpool_info, threadpool_limits

    from paper_2408_03505_amd.synthetic import CONFIGS, layer_inputs

    flops, secs, done = _oracle_seconds(cfg, x, params, dout, budget_s)
    pools = threadpool_info()
    threads = max([i.get("num_threads", 1) for i in pools] or [1])
    res = {"value": flops / secs / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
           "sample": f"float64 oracle forward+backward of {done} of {cfg['batch']} sequences "
                     f"({done * cfg['seq']} tokens) of the same layer, {secs:.1f} s",
           "oracle": "float64 numpy: BLAS matmul on the host's threads, scipy erf, everything else numpy",
           "cpu_model": cpu_model(), "host_cpus": len(os.sched_getaffinity(0)),
           "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
           "blas": [{k: i.get(k) for k in ("internal_api", "version", "num_threads", "threading_layer")}
                    for i in pools]}
    per, single = {}, {}
    for cname in (configs if configs is not None else CONFIGS):
        ccfg = CONFIGS[cname]
        if cname == name:
            cx, cp, cd = x, params, dout
        else:
            cx, cp, cd = layer_inputs(ccfg, seed=seed)
        f, t, n = _oracle_seconds(ccfg, cx, cp, cd, budget_s=0.0, max_seqs=1)
        per[cname] = {"tflops": round(f / t / 1e12, 4), "s_per_sequence": round(t / n, 4),
                      "sample": f"{n} of {ccfg['batch']} sequences"}
        if cname in ("vit_tiny", "vit_base", "vit_huge"):
            with threadpool_limits(limits=1):
                f, t, n = _oracle_seconds(ccfg, cx, cp, cd, budget_s=0.0, max_seqs=1)
            single[cname] = {"tflops": round(f / t / 1e12, 4), "s_per_sequence": round(t / n, 4),
                             "sample": f"{n} of {ccfg['batch']} sequences, 1 thread"}
        del cx, cp, cd
    res["per_config"] = per
    res["single_thread"] = single
    return res


def main():
    args = parse()
    from paper_2408_03505_amd.synthetic import CONFIGS
    use_config(CONFIGS[args.config])
    if args.summarize:
        summarize(args.summarize, skip_steps=args.warmup)
        return
    if args.pmc_summary:
        ent = pmc_entries(args.pmc_summary)
        ctrs = sorted({k for v in ent.values() for k in v})
        derived = sorted({k for n in DISPATCHES for k in pmc_utilisation(ent[n])})
        print("| entry | " + " | ".join(ctrs + derived) + " |")
        print("|---" * (1 + len(ctrs) + len(derived)) + "|")
        for n in DISPATCHES:
            u = pmc_utilisation(ent[n])
            print(f"| {n} | " + " | ".join([f"{ent[n][k]:.4g}" for k in ctrs] +
                                           [f"{u[k]:.3f}" if k in u else "" for k in derived]) + " |")
        return
    if args.pmc_traffic:
        from paper_2408_03505_amd.synthetic import CONFIGS
        vals = pmc_traffic(args.pmc_traffic[0], args.pmc_traffic[1], args.copy_mib << 20)
        work = kernel_work(CONFIGS[args.config])
        (fetch, fs), (write, ws) = vals["FETCH_SIZE"], vals["WRITE_SIZE"]
        for fam in sorted(_FAMILY_SRC):
            print(f"source-sha256 {fam}: {source_hash(fam)}")
        print(f"copy-reference-bytes: {args.copy_mib << 20}  fetch-scale: {fs:.4f}  write-scale: {ws:.4f}\n")
        floors = gemm_fetch_floors(CONFIGS[args.config])
        print("`fetch floor`: for each GEMM, the operand bytes that the eight XCD caches must fetch at least "
              "under its launch plan, since each XCD's concurrent workgroups share one L2 and an operand "
              "panel outlives neither its round of tiles nor its XCD.\n")
        print("| entry | FETCH bytes | WRITE bytes | traffic bytes | algorithmic bytes | traffic / algorithmic "
              "| fetch floor | FETCH / floor |")
        print("|---|---|---|---|---|---|---|---|")
        for n in DISPATCHES:
            t = fetch[n] + write[n]
            fl = f"{floors[n]} | {fetch[n] / floors[n]:.2f}" if n in floors else " | "
            print(f"| {n} | {fetch[n]:.0f} | {write[n]:.0f} | {t:.0f} | {work[n][1]} | {t / work[n][1]:.2f} | {fl} |")
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; multi-GPU runs are out of scope "
                                   "(--gpus must be 1)"}), flush=True)
        sys.exit(2)
    from paper_2408_03505_amd.synthetic import CONFIGS, layer_inputs

    cfg = CONFIGS[args.config]
    x, params, dout = layer_inputs(cfg, seed=args.seed)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    gx, gd = x.to(dev), dout.to(dev)
    gp = {n: params[n].to(dev) for n in params}
    chain = Chain(cfg, gx, gp, gd)
    names = [n for n, _ in chain.kernels]
    K, W = args.steps, args.warmup

    for _ in range(W):
        for _, fn in chain.kernels:
            fn()
    torch.cuda.synchronize()

    # Per-kernel latencies: K steps with HIP events around every launch (all
    # on the current stream, where the library launches).  Each event record
    # leaves a small gap between kernels, so this pass is not the timed one.
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in names]
          for _ in range(K)]
    for k in range(K):
        for i, (_, fn) in enumerate(chain.kernels):
            ev[k][i][0].record()
            fn()
            ev[k][i][1].record()
    torch.cuda.synchronize()
    per = {n: [ev[k][i][0].elapsed_time(ev[k][i][1]) * 1e3 for k in range(K)] for i, n in enumerate(names)}
    p50 = {n: float(np.median(v)) for n, v in per.items()}
    # the dominant kernel: the single-dispatch entry with the largest average time
    dom = max((n for n in names if DISPATCHES[n] == 1), key=lambda n: float(np.mean(per[n])))
    di = names.index(dom)

    # Timed region: K steps of the chain as it runs in training; only the
    # dominant kernel's launches are bracketed by events, for its live
    # average duration.
    dev_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(K):
        for i, (_, fn) in enumerate(chain.kernels):
            if i == di:
                dev_ev[k][0].record()
                fn()
                dev_ev[k][1].record()
            else:
                fn()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dom_us = [a.elapsed_time(b) * 1e3 for a, b in dev_ev]

    work = kernel_work(cfg)
    flops_step = step_flops(cfg)
    ms = wall / K * 1e3
    tflops = flops_step / (wall / K) / 1e12
    avg = {n: float(np.mean(v)) for n, v in per.items()}
    avg[dom] = float(np.mean(dom_us))
    dflops = work[dom][0]
    achieved = dflops / (avg[dom] * 1e-6) / 1e12
    per_kernel = {n: {"p50_us": round(p50[n], 2), "p90_us": round(float(np.percentile(per[n], 90)), 2),
                      "tflops": round(work[n][0] / (p50[n] * 1e-6) / 1e12, 1) if work[n][0] else None,
                      "gbs": round(work[n][1] / (p50[n] * 1e-6) / 1e9, 1),
                      "frac": round((work[n][0] / (p50[n] * 1e-6) / 1e12) / PEAK_BF16_TFLOPS, 3) if work[n][0]
                      else round(work[n][1] / (p50[n] * 1e-6) / 1e9 / PEAK_HBM_GBS, 3)} for n in names}
    for n, hw in hardware_flops(cfg).items():
        per_kernel[n]["hw_tflops"] = round(hw / (p50[n] * 1e-6) / 1e12, 1)

    res = {
        "metric": "encoder layer fwd+bwd TFLOPS (% bf16 MFMA peak) + per-kernel p50 latency (us)",
        "value": round(tflops, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{args.config} encoder layer fwd+bwd", **{k: cfg[k] for k in (
            "batch", "seq", "hidden", "heads", "head_dim", "mlp")}},
        "frac_of_bf16_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
        "sum_kernel_p50_ms": round(sum(p50.values()) / 1e3, 4),
        "max_kernel_p50_us": round(max(p50.values()), 2),
        "per_kernel": per_kernel,
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": read_traffic(dom) if args.config == "vit22b" else None,
                     "avg_launch_us": round(avg[dom], 2)},
    }
    def section(fn):
        """Run an optional part of the report; a failure is recorded, not raised,
        so that the measurement line above always gets printed."""
        try:
            return fn()
        except Exception as e:  # noqa: BLE001
            torch.cuda.synchronize()
            return {"error": f"{type(e).__name__}: {str(e)[:300]}"}
        finally:
            torch.cuda.empty_cache()

    def fit_report():
        fit = {"trace": "synthetic LLM timeline: TP bubbles uniform in [200, 400] us alternating with "
                        "LLM computation uniform in [300, 900] us (seed 0); kernels = per-kernel p50",
               args.config: bubble_fit(p50)}
        if args.fit_config not in ("", "none", args.config):
            fcfg = CONFIGS[args.fit_config]
            fx, fp, fd = layer_inputs(fcfg, seed=args.seed)
            fchain = Chain(fcfg, fx.to(dev), {n: fp[n].to(dev) for n in fp}, fd.to(dev))
            fp50 = time_chain(fchain, steps=10, warmup=3)
            fit[args.fit_config] = bubble_fit(fp50)
            fit[args.fit_config]["p50_us"] = {n: round(v, 2) for n, v in fp50.items()}
        return fit

    res["bubble_fit"] = section(fit_report)
    if not args.no_corun:
        res["corun"] = section(lambda: corun(chain, p50, dev))
        res["corun_cu_mask"] = section(lambda: corun_masked(chain, p50, dev))
    if not args.no_variants:
        res["variants"] = section(lambda: {f"{args.config}_parallel_block": time_parallel_block(cfg, dev)})
    if args.encoder_layers > 0:
        res["whole_encoder"] = section(lambda: time_whole_encoder(cfg, args.encoder_layers, dev))
    if not args.no_isolated:
        res["isolated"] = section(lambda: time_isolated(chain, p50))
    if not args.no_flush:
        res["memory_bound"] = section(lambda: time_flushed(chain, work))
    if not args.no_configs:
        res["configs"] = section(lambda: time_configs(args.config, dev, args.seed))
    if not args.no_ceilings:
        ceil = section(lambda: measure_ceilings(dev))
        res["ceilings"] = ceil
        if "mfma_bf16_tflops" in ceil:
            res["roofline"]["measured_peak"] = ceil["mfma_bf16_tflops"]
            res["roofline"]["frac_of_measured"] = round(achieved / ceil["mfma_bf16_tflops"], 4)
    if args.copy_mib:
        src = torch.empty(args.copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        res["copy_reference_bytes"] = args.copy_mib << 20
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(cfg, x, params, dout, args.cpu_budget_s, args.config, args.seed)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
