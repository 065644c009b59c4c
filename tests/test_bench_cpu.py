"""Host logic of the benchmark, no GPU: the one-GPU guard, the algorithmic work per launch
that the roofline figures divide by, and the rocprofv3 counter summary behind `traffic`
(synthetic counter files)."""
import csv
import json
import os
import subprocess
import sys

import bench
import synth


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(bench.ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""  # no JSON line that could be read as a measurement


def test_algorithmic_work_of_the_8b_step():
    # 64 sessions of a 2048-slot prefix and a 17-row tree (1088 rows, 704 parent rows)
    w = synth.get("8b-bf16")
    B, n1, P = 64, 17, 704
    S_tot = B * 2048 + B * n1
    work = bench.kernel_work(w, B, n1, P, S_tot)
    # products of the [1088, 4096] activations with the layer weights
    assert work["gemm_gate_up"] == (2.0 * 1088 * 28672 * 4096, 28672 * 4096 * 2)
    assert work["gemm_gate_up"][0] == 255_550_554_112.0
    assert work["gemm_down"] == (2.0 * 1088 * 4096 * 14336, 4096 * 14336 * 2)
    assert work["gemm_qkv"] == (2.0 * 1088 * 6144 * 4096, 6144 * 4096 * 2)
    assert work["gemm_o"] == (2.0 * 1088 * 4096 * 4096, 4096 * 4096 * 2)
    # the LM head also writes the fp32 logits once
    assert work["gemm_lm_head"][1] == 128256 * 4096 * 2 + 1088 * 128256 * 4
    # attention reads K and V (bf16) of 64 x 2065 slots of 8 kv heads of 128 dims once
    assert work["tree_attention"][1] == 2 * 64 * 2065 * 8 * 128 * 2 == 541_327_360
    # the vocabulary kernel reads every row's logits and every parent row's draft q once
    assert work["vocab_verify"][1] == 4 * 128256 * (1088 + 704) == 919_339_008


def _write_counters(d, rows):
    os.makedirs(d)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Value"])
        wr.writeheader()
        for r in rows:
            wr.writerow(r)


# one decoder layer with a sliced QKV product, one with the fused QKV epilogue, then the
# LM head and the vocabulary kernel, with a foreign kernel in between
_STEP = [
    ("rmsnorm_kernel", "rmsnorm"),
    ("gemm_f16w_kernelILi3EDF16b", "gemm_qkv"),
    ("tile_fixup_kernelILi3E", "+"),
    ("rope_kv_kernel", "+"),
    ("tree_attn_mfma_kernelILi128E", "tree_attention"),
    ("gemm_f16w_kernelILi1EDF16b", "gemm_o"),
    ("fixup_resid_norm_kernel", "+"),
    ("gemm_f16w_kernelILi2EDF16b", "gemm_gate_up"),
    ("gemm_f16w_kernelILi1EDF16b", "gemm_down"),
    ("fixup_resid_norm_kernel", "+"),
    ("at::native::elementwise_kernel", None),
    ("gemm_f16w_kernelILi4EDF16b", "gemm_qkv"),
    ("tree_attn_t32_kernelILi128E", "tree_attention"),
    ("attn_combine_kernel", "+"),
    ("gemm_f16w_kernelILi5EDF16b", "gemm_lm_head"),
    ("vocab_verify_kernel", "vocab_verify"),
]


def test_dispatch_labels_follow_the_launch_order():
    rows = [{"Dispatch_Id": str(i), "Kernel_Name": n, "Counter_Value": "0"}
            for i, (n, _) in enumerate(_STEP)]
    assert bench._label_dispatches(rows) == [k for _, k in _STEP]
    # a sliced fp32 product right before the vocabulary kernel is the LM head
    rows = [{"Dispatch_Id": "0", "Kernel_Name": "gemm_f16w_kernelILi3EDF16b", "Counter_Value": "0"},
            {"Dispatch_Id": "1", "Kernel_Name": "tile_fixup_kernelILi3E", "Counter_Value": "0"},
            {"Dispatch_Id": "2", "Kernel_Name": "vocab_verify_kernel", "Counter_Value": "0"}]
    assert bench._label_dispatches(rows) == ["gemm_lm_head", "+", "vocab_verify"]


def test_counter_summary_scales_by_the_copy_and_folds_fixups(tmp_path):
    fetch = {i: 10.0 * (i + 1) for i in range(len(_STEP))}
    write = {i: 1.0 * (i + 1) for i in range(len(_STEP))}
    # dispatch order comes from Dispatch_Id, not from the file order
    order = list(reversed(range(len(_STEP))))
    _write_counters(str(tmp_path / "f"), [{"Dispatch_Id": str(i), "Kernel_Name": _STEP[i][0],
                                          "Counter_Value": str(fetch[i])} for i in order])
    _write_counters(str(tmp_path / "w"), [{"Dispatch_Id": str(i), "Kernel_Name": _STEP[i][0],
                                          "Counter_Value": str(write[i])} for i in order])
    # a 1 MiB copy: FETCH_SIZE reads half the bytes read, WRITE_SIZE all the bytes written
    _write_counters(str(tmp_path / "cf"), [{"Dispatch_Id": "0", "Kernel_Name": "copy",
                                           "Counter_Value": "512"}])
    _write_counters(str(tmp_path / "cw"), [{"Dispatch_Id": "0", "Kernel_Name": "copy",
                                           "Counter_Value": "1024"}])
    out = bench.summarize_pmc(str(tmp_path / "f"), str(tmp_path / "w"), str(tmp_path / "cf"),
                              str(tmp_path / "cw"), 1)
    assert out["fetch_scale"] == 2.0 and out["write_scale"] == 1.0
    k = out["kinds"]
    assert set(k) == {"rmsnorm", "gemm_qkv", "tree_attention", "gemm_o", "gemm_gate_up",
                      "gemm_down", "gemm_lm_head", "vocab_verify"}

    def per_launch(idx_groups):
        f = sum(sum(fetch[i] for i in g) for g in idx_groups) / len(idx_groups)
        w = sum(sum(write[i] for i in g) for g in idx_groups) / len(idx_groups)
        return f, w

    # the sliced QKV carries its fixup and RoPE dispatches; the fused one stands alone
    f, w = per_launch([(1, 2, 3), (11,)])
    assert k["gemm_qkv"]["launches"] == 2
    assert k["gemm_qkv"]["fetch_kib"] == round(f, 1)
    assert k["gemm_qkv"]["hbm_bytes_per_launch"] == round((f * 2.0 + w) * 1024)
    f, w = per_launch([(5, 6)])
    assert k["gemm_o"]["hbm_bytes_per_launch"] == round((f * 2.0 + w) * 1024)
    f, w = per_launch([(8, 9)])
    assert k["gemm_down"]["hbm_bytes_per_launch"] == round((f * 2.0 + w) * 1024)
    assert k["vocab_verify"]["source_sha"] == bench.kind_source_hash("vocab_verify")


def test_traffic_is_dropped_for_a_kernel_whose_sources_changed(tmp_path, monkeypatch):
    blob = {"kinds": {
        "gemm_o": {"hbm_bytes_per_launch": 123, "source_sha": bench.kind_source_hash("gemm_o")},
        "vocab_verify": {"hbm_bytes_per_launch": 456, "source_sha": "0000000000000000"}}}
    os.makedirs(tmp_path / "profiles")
    (tmp_path / "profiles" / "hbm_traffic_x.md").write_text(
        "# table\n\n```json\n" + json.dumps(blob) + "\n```\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.load_traffic("x") == {"gemm_o": 123}
    assert bench.load_traffic("missing") == {}


def test_committed_traffic_tables_name_known_kernels():
    d = os.path.join(bench.ROOT, "profiles")
    tables = [f for f in os.listdir(d) if f.startswith("hbm_traffic_") and f.endswith(".md")]
    assert tables
    for f in tables:
        text = open(os.path.join(d, f)).read()
        i = text.index("```json")
        blob = json.loads(text[i + 7: text.index("```", i + 7)])
        assert set(blob["kinds"]) <= set(bench.KIND_SOURCES)
        for v in blob["kinds"].values():
            assert v["hbm_bytes_per_launch"] > 0 and len(v["source_sha"]) == 16


def test_mfma_summary_averages_per_kind_and_skips_fixups(tmp_path, monkeypatch):
    # one MfmaUtil value per dispatch (percent), in dispatch order
    util = {i: 5.0 * (i + 1) for i in range(len(_STEP))}
    rows = [{"Dispatch_Id": str(i), "Kernel_Name": _STEP[i][0], "Counter_Value": str(util[i])}
            for i in reversed(range(len(_STEP)))]
    _write_counters(str(tmp_path / "m"), rows)
    out = bench.summarize_mfma(str(tmp_path / "m"))
    k = out["kinds"]
    assert k["gemm_qkv"] == {"launches": 2, "mfma_busy_pct": round((util[1] + util[11]) / 2, 2),
                             "source_sha": bench.kind_source_hash("gemm_qkv")}
    assert k["gemm_o"]["mfma_busy_pct"] == util[5]          # its fixup is not averaged in
    assert k["gemm_gate_up"]["mfma_busy_pct"] == util[7]
    assert "+" not in k and None not in k
    # committed summaries are read back only for kinds whose sources are unchanged
    blob = {"counter": "MfmaUtil", "kinds": {
        "gemm_o": {"launches": 1, "mfma_busy_pct": 41.5, "source_sha": bench.kind_source_hash("gemm_o")},
        "tree_attention": {"launches": 1, "mfma_busy_pct": 9.0, "source_sha": "0000000000000000"}}}
    os.makedirs(tmp_path / "profiles")
    (tmp_path / "profiles" / "mfma_util_x.md").write_text(
        "# table\n\n```json\n" + json.dumps(blob) + "\n```\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.load_mfma("x") == {"gemm_o": 41.5}
    assert bench.load_mfma("missing") == {}


def test_committed_mfma_tables_name_known_kernels():
    d = os.path.join(bench.ROOT, "profiles")
    tables = [f for f in os.listdir(d) if f.startswith("mfma_util_") and f.endswith(".md")]
    assert tables
    for f in tables:
        blob = bench._profile_blob(f)
        assert blob["counter"] == "MfmaUtil"
        assert set(blob["kinds"]) <= set(bench.KIND_SOURCES)
        for v in blob["kinds"].values():
            assert 0.0 <= v["mfma_busy_pct"] <= 100.0 and len(v["source_sha"]) == 16


def test_lds_probe_patterns_stay_in_bounds():
    """The LDS probe's lane offset tables fit the probe kernel's 16 KB window, are 16-byte
    aligned, and the swizzles only permute pieces within each row (one piece of every
    lane group's row per lane)."""
    import bench
    pats = dict(bench.lds_patterns())
    for name, offs in pats.items():
        assert len(offs) == 64 and len(set(offs)) == 64, name
        assert all(0 <= o < 16384 and o % 16 == 0 for o in offs), name
    # a permutation of the unswizzled layout's pieces within each row
    base = sorted(((l & 15) * 64 + ((l >> 4) << 4)) for l in range(64))
    assert sorted(pats["GEMM 64-byte rows, piece ^ (row / 2)"]) == base
    assert sorted(pats["GEMM 64-byte rows, piece ^ (row / 4)"]) == base
