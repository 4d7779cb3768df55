"""Host-side logic of bench.py (no GPU): dispatch-to-entry mapping of a
kernel trace, FETCH/WRITE scaling against the copy reference, the committed
traffic table and its source hash, the bubble packing report, and the refusal
of multi-GPU runs."""
import csv
import json
import os
import subprocess
import sys

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _one_step_names():
    """Kernel names of one chain step, as a trace would show them."""
    out = []
    for entry, kernels in bench.ENTRY_KERNELS.items():
        for k in kernels:
            out.append(f"void optimus::(anonymous namespace)::{k}<256, 3>(int, int)")
    return out


def test_map_dispatches_sums_each_entry_per_step():
    names = _one_step_names()
    per_step = len(names)
    lib = [(i, names[i % per_step], float(i)) for i in range(2 * per_step)]
    steps = bench.map_dispatches(lib[::-1])  # order of the input does not matter
    assert len(steps) == 2
    i = 0
    for n in bench.ENTRY_KERNELS:
        d = bench.DISPATCHES[n]
        for st in range(2):
            want = sum(float(st * per_step + i + j) for j in range(d))
            assert steps[st][n] == want, (n, st)
        i += d


def test_map_dispatches_rejects_partial_steps_and_wrong_kernels():
    names = _one_step_names()
    lib = [(i, names[i], 1.0) for i in range(len(names))]
    with pytest.raises(RuntimeError, match="whole number"):
        bench.map_dispatches(lib[:-1])
    swapped = list(lib)
    swapped[1], swapped[2] = (1, names[2], 1.0), (2, names[1], 1.0)  # qkv GEMM <-> attention
    with pytest.raises(RuntimeError, match="is not"):
        bench.map_dispatches(swapped)


def test_use_config_counts_the_split_reduction_kernels(monkeypatch):
    """Products that the library splits at a workload run as two dispatches
    (the GEMM, then the split reduction); the dispatch map follows."""
    from paper_2408_03505_amd.synthetic import CONFIGS
    monkeypatch.setattr(bench, "ENTRY_KERNELS", dict(bench.ENTRY_KERNELS))
    monkeypatch.setattr(bench, "DISPATCHES", dict(bench.DISPATCHES))
    gemms = set(bench.gemm_products(CONFIGS["vit22b"]))
    split_at = {"vit22b": set(), "vit22b_tp8": {"oproj_bwd_data"},
                "vit_base": {"mlp_down_bwd_weight", "mlp_up_bwd_weight", "oproj_bwd_weight", "qkv_bwd_weight"}}
    for name, split in split_at.items():
        bench.use_config(CONFIGS[name])
        for n in gemms:
            assert bench.ENTRY_KERNELS[n] == (("gemm_", "splitk_") if n in split else ("gemm_",)), (name, n)
        names = _one_step_names()
        steps = bench.map_dispatches([(i, names[i], 1.0) for i in range(len(names))])
        assert all(steps[0][n] == (2.0 if n in split else 1.0) for n in gemms), name


def _write_counters(d, counter, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "1_counter_collection.csv"), "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (name, value) in enumerate(rows):
            w.writerow({"Dispatch_Id": i, "Kernel_Name": name, "Counter_Name": counter, "Counter_Value": value})


def test_pmc_traffic_scales_by_the_copy_reference(tmp_path):
    names = _one_step_names()
    copy_bytes = 1 << 30
    # the copy's FETCH_SIZE reads half its bytes (KiB), WRITE_SIZE all of them
    fetch = [("__amd_rocclr_copyBuffer", copy_bytes / 2 / 1024)] + [(n, 100.0) for n in names]
    write = [("__amd_rocclr_copyBuffer", copy_bytes / 1024)] + [(n, 10.0) for n in names]
    _write_counters(str(tmp_path / "f"), "FETCH_SIZE", fetch)
    _write_counters(str(tmp_path / "w"), "WRITE_SIZE", write)
    vals = bench.pmc_traffic(str(tmp_path / "f"), str(tmp_path / "w"), copy_bytes)
    f, fs = vals["FETCH_SIZE"]
    w, ws = vals["WRITE_SIZE"]
    assert fs == pytest.approx(2.0) and ws == pytest.approx(1.0)
    for n in bench.ENTRY_KERNELS:
        d = bench.DISPATCHES[n]
        assert f[n] == pytest.approx(d * 100.0 * 1024 * 2.0)
        assert w[n] == pytest.approx(d * 10.0 * 1024)


def test_committed_traffic_table_is_keyed_by_the_sources():
    # an entry has a traffic figure exactly when the committed table was taken
    # on its family's current sources, and a changed source hash voids it
    text = open(bench.TRAFFIC_MD).read()
    for n in bench.ENTRY_KERNELS:
        fam = bench.entry_family(n)
        current = f"source-sha256 {fam}: {bench.source_hash(fam)}" in text
        t = bench.read_traffic(n)
        assert (t is not None and t > 0) if current else t is None, n
    real = bench.source_hash
    try:
        bench.source_hash = lambda fam: "0" * 64
        assert bench.read_traffic("qkv_fwd") is None
    finally:
        bench.source_hash = real


def test_kernel_work_covers_every_entry():
    from paper_2408_03505_amd.synthetic import CONFIGS
    for cfg in CONFIGS.values():
        work = bench.kernel_work(cfg)
        assert set(work) == set(bench.ENTRY_KERNELS)
        assert all(f >= 0 and b > 0 for f, b in work.values())
        # memory-bound entries carry no flops; every other entry does
        assert all((work[n][0] == 0) == (n in bench.MEM_BOUND) for n in work)
        # the attention backward's kernels run 7 products where 4 are counted
        assert bench.hardware_flops(cfg)["attn_bwd"] * 4 == work["attn_bwd"][0] * 7


def test_bubble_fit_packs_in_chain_order():
    # a 150 us kernel fits any 200-400 us bubble; a 500 us kernel fits none
    p50 = {n: 150.0 for n in bench.ENTRY_KERNELS}
    r = bench.bubble_fit(p50)
    assert r["fwd"]["placed"] == r["fwd"]["kernels"] and r["bwd"]["placed"] == r["bwd"]["kernels"]
    assert 0 < r["fwd"]["fill"] <= 1 and 0 < r["bwd"]["fill"] <= 1
    p50["qkv_fwd"] = 500.0
    r = bench.bubble_fit(p50)
    assert r["fwd"]["blocked_at"] == "qkv_fwd" and r["fwd"]["placed"] == 1


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in line["error"]


def test_cu_mask_leaves_every_xcd_cus_for_both_streams():
    # the slice and its complement each keep CUs on all eight XCDs whether mask
    # bits go to XCDs in 32-bit blocks or round-robin by bit index
    for per_word in (1, 2, 3, 4):
        mask = bench.cu_mask_words(per_word)
        comp = [(~m) & 0xFFFFFFFF for m in mask]
        bits = lambda ws: [32 * w + b for w, m in enumerate(ws) for b in range(32) if (m >> b) & 1]
        sel, rest = bits(mask), bits(comp)
        assert len(sel) == 8 * per_word and len(rest) == 256 - 8 * per_word
        for xcd in range(8):
            assert sum(1 for i in sel if i // 32 == xcd) == per_word
            assert sum(1 for i in sel if i % 8 == xcd) == per_word
            assert sum(1 for i in rest if i // 32 == xcd) == 32 - per_word
            assert sum(1 for i in rest if i % 8 == xcd) == 32 - per_word


def test_pmc_summary_per_entry_and_busy_fraction(tmp_path):
    # two steps; per dispatch: MFMA busy 51200 cycles over 8 XCDs x 100 active cycles
    names = _one_step_names()
    rows = []
    for st in range(2):
        for n in names:
            rows += [(n, "SQ_VALU_MFMA_BUSY_CYCLES", 512.0 * 100), (n, "GRBM_GUI_ACTIVE", 8 * 100.0),
                     (n, "SQ_WAVE_CYCLES", 10.0), (n, "SQ_WAIT_ANY", 3.0)]
    d = tmp_path / "p"
    os.makedirs(d)
    with open(d / "1_counter_collection.csv", "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (n, c, v) in enumerate(rows):
            w.writerow({"Dispatch_Id": i // 4, "Kernel_Name": n, "Counter_Name": c, "Counter_Value": v})
    ent = bench.pmc_entries(str(d))
    for n in bench.ENTRY_KERNELS:
        k = bench.DISPATCHES[n]
        assert ent[n]["GRBM_GUI_ACTIVE"] == pytest.approx(800.0 * k)
        u = bench.pmc_utilisation(ent[n])
        assert u["mfma_busy"] == pytest.approx(0.5)
        assert u["wait_any_per_wave_cycle"] == pytest.approx(0.3)


def test_cpu_baseline_reports_host_and_per_config_figures():
    from paper_2408_03505_amd.synthetic import CONFIGS, layer_inputs
    cfg = CONFIGS["vit_tiny"]
    x, params, dout = layer_inputs(cfg, seed=0)
    r = bench.cpu_baseline(cfg, x, params, dout, budget_s=0.5, name="vit_tiny", configs=["vit_tiny", "vit_base"])
    assert r["kind"] == "oracle" and r["value"] > 0 and r["cores"] >= 1
    assert r["cpu_model"] and r["host_cpus"] >= 1 and "float64" in r["oracle"]
    assert set(r["per_config"]) == {"vit_tiny", "vit_base"} and set(r["single_thread"]) == {"vit_tiny", "vit_base"}
    for v in list(r["per_config"].values()) + list(r["single_thread"].values()):
        assert v["tflops"] > 0 and v["s_per_sequence"] > 0


@pytest.mark.parametrize("tm,tn", [(8, 96), (8, 72), (16, 18), (9, 5), (1, 1), (24, 32)])
def test_tile_order_model_covers_every_tile_once(tm, tn):
    nb = tm * tn
    seen = [bench._tile_of(p, nb, tm, tn) for p in range(nb)]
    assert sorted(seen) == [(a, b) for a in range(tm) for b in range(tn)]


@pytest.mark.parametrize("tm,tn,S", [(16, 6, 5), (3, 12, 7), (10, 10, 4)])
def test_split_order_model_covers_every_item_once(tm, tn, S):
    nb = tm * tn * S
    seen = [bench._split_item(p, nb, tm, tn) for p in range(nb)]
    assert sorted(seen) == [(s, a, b) for s in range(S) for a in range(tm) for b in range(tn)]


def test_fetch_floor_bounds():
    # ViT-22B MLP-up forward on 256x256 tiles: 8 x 96 tiles, three rounds; in
    # a round each XCD runs 4 row tiles x 8 column tiles and fetches those
    # 12 panels of 256 rows x 6144 bf16
    assert bench.fetch_floor(2048, 24576, 6144, 256, 256, 1) == 8 * 3 * 12 * 256 * 6144 * 2
    for rows, cols, K, bm, bn, sp in ((2048, 18432, 6144, 256, 192, 1), (6304, 768, 768, 128, 128, 1),
                                      (768, 768, 6304, 128, 128, 12), (2000, 72 * 8, 1024, 128, 128, 1)):
        f = bench.fetch_floor(rows, cols, K, bm, bn, sp)
        once = 2 * K * (rows + cols)  # each operand fetched once
        tiles = -(-rows // bm) * -(-cols // bn)
        assert once <= f <= tiles * sp * 2 * (bm + bn) * -(-K // sp), (rows, cols, K)
