"""Throughput of the tree-verify step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 8b-bf16]

A step is one acespec_verify_tree call over a batch of drafted trees (embedding, all
decoder layers with tree attention, LM head, fused vocabulary verify, path walk), on
synthetic inputs already resident in HBM.  Prints one JSON line: verified tree tokens/s
(sessions x drafted nodes / step time), the roofline of the dominant kernel from the
library's own HIP-event timing over the timed steps, and the float64 oracle timed on the
host cores on a bounded sample (cpu_baseline).
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_MFMA_TFLOPS = 2500.0   # MI355X dense fp16 / bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def kernel_work(w, B, n1, P, S_tot):
    """Algorithmic work per launch of each kernel kind: (flops, bytes)."""
    R = B * n1
    d, H, Hkv, hd, F, V = w.d, w.H, w.Hkv, w.hd, w.F, w.V
    qkvn = (H + 2 * Hkv) * hd
    wb = 2  # bf16 weights
    return {
        "gemm_qkv": (2.0 * R * qkvn * d, qkvn * d * wb),
        "gemm_o": (2.0 * R * d * H * hd, d * H * hd * wb),
        "gemm_gate_up": (2.0 * R * 2 * F * d, 2 * F * d * wb),
        "gemm_down": (2.0 * R * d * F, d * F * wb),
        "gemm_lm_head": (2.0 * R * V * d, V * d * wb + R * V * 4),
        # K and V of every session's prefix and tree slots, read once
        "tree_attention": (4.0 * w.G * n1 * hd * S_tot * Hkv, 2.0 * S_tot * Hkv * hd * 2),
        # logits of every row once, draft distribution of every parent row once
        "vocab_verify": (0.0, 4.0 * R * V + 4.0 * P * V),
    }


# ---------------------------------------------------------------------------------------
# HBM traffic from rocprofv3 counters
# ---------------------------------------------------------------------------------------
CSRC = os.path.join(ROOT, "paper_2609_02514_amd", "csrc")
# source files whose change invalidates a kernel kind's measured counters
KIND_SOURCES = {
    "tree_attention": ["attention.hip"], "gemm_qkv": ["gemm.hip"], "gemm_o": ["gemm.hip"],
    "gemm_gate_up": ["gemm.hip"], "gemm_down": ["gemm.hip"], "gemm_lm_head": ["gemm.hip"],
    "vocab_verify": ["vocab.hip"], "rmsnorm": ["elementwise.hip"], "rope_table": ["elementwise.hip"],
}


def kind_source_hash(kind):
    import hashlib
    h = hashlib.sha256()
    for f in KIND_SOURCES.get(kind, []) + ["common.h"]:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _pmc_rows(run_dir):
    import csv
    path = os.path.join(run_dir, "run_counter_collection.csv")
    rows = list(csv.DictReader(open(path)))
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    return rows


def _label_dispatches(rows):
    """Kernel kind of every dispatch of the verify library, from the symbol and the fixed
    launch order of a step (per layer: QKV, O, gate/up, down; LM head right before the
    vocabulary kernel).  A K-slice fixup or RoPE dispatch that completes the product
    launched just before it is labelled "+" (its bytes belong to that launch)."""
    labels, resid_seen = [], 0
    for i, r in enumerate(rows):
        n = r["Kernel_Name"]
        kind = None
        if "tree_attn_mfma_kernel" in n or "tree_attn_t32_kernel" in n:
            kind = "tree_attention"
        elif "attn_combine_kernel" in n or "tile_fixup_kernel" in n or \
                "fixup_resid_norm_kernel" in n or "rope_kv_kernel" in n:
            kind = "+"
        elif "gemm_f16w_kernelILi2E" in n:
            kind = "gemm_gate_up"
        elif "gemm_f16w_kernelILi1E" in n:
            kind = "gemm_o" if resid_seen % 2 == 0 else "gemm_down"
            resid_seen += 1
        elif "gemm_f16w_kernelILi4E" in n:          # QKV with its RoPE epilogue
            kind = "gemm_qkv"
        elif "gemm_f16w_kernelILi5E" in n:          # LM head with row maxima
            kind = "gemm_lm_head"
        elif "gemm_f16w_kernelILi3E" in n:          # fp32 store: QKV (sliced) or LM head
            nxt = next((rows[j]["Kernel_Name"] for j in range(i + 1, len(rows))
                        if "fixup" not in rows[j]["Kernel_Name"]), "")
            kind = "gemm_lm_head" if "vocab_verify" in nxt else "gemm_qkv"
        elif "vocab_verify_kernel" in n:
            kind = "vocab_verify"
        elif "rmsnorm_kernel" in n:
            kind = "rmsnorm"
        labels.append(kind)
    return labels


def summarize_pmc(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, copy_mib):
    """Per-kind HBM bytes per launch: FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each
    scaled by what the counter reads for a plain copy of copy_mib MiB."""
    copy_kib = copy_mib * 1024.0
    cf = sum(float(r["Counter_Value"]) for r in _pmc_rows(copy_fetch_dir))
    cw = sum(float(r["Counter_Value"]) for r in _pmc_rows(copy_write_dir))
    f_scale, w_scale = copy_kib / cf, copy_kib / cw
    out = {"copy_mib": copy_mib, "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4),
           "kinds": {}}
    acc = {}
    for which, d in (("fetch", fetch_dir), ("write", write_dir)):
        rows = _pmc_rows(d)
        last = None   # (kind, index) of the last product launch
        for kind, r in zip(_label_dispatches(rows), rows):
            v = float(r["Counter_Value"])
            if kind == "+":
                if last is not None:
                    acc[last[0]][which][last[1]] += v
                continue
            if kind is None:
                last = None
                continue
            e = acc.setdefault(kind, {"fetch": [], "write": []})
            e[which].append(v)
            last = (kind, len(e[which]) - 1)
    for kind, e in sorted(acc.items()):
        fk = sum(e["fetch"]) / max(len(e["fetch"]), 1)
        wk = sum(e["write"]) / max(len(e["write"]), 1)
        out["kinds"][kind] = {
            "launches": len(e["fetch"]), "fetch_kib": round(fk, 1), "write_kib": round(wk, 1),
            "hbm_bytes_per_launch": round((fk * f_scale + wk * w_scale) * 1024.0),
            "source_sha": kind_source_hash(kind)}
    return out


def summarize_mfma(run_dir):
    """Per-kind MFMA pipe utilisation from one rocprofv3 pass of rocprofiler's derived
    counter MfmaUtil (SQ_VALU_MFMA_BUSY_CYCLES summed over the SIMDs / (GRBM_GUI_ACTIVE x
    SIMDs), in percent per dispatch): the hardware's view of how busy the matrix cores are,
    independent of the clock the power limit sets."""
    rows = [r for r in _pmc_rows(run_dir) if r.get("Counter_Name", "MfmaUtil") == "MfmaUtil"]
    acc = {}
    for kind, r in zip(_label_dispatches(rows), rows):
        if kind is None or kind == "+":
            continue
        acc.setdefault(kind, []).append(float(r["Counter_Value"]))
    return {"counter": "MfmaUtil", "kinds": {
        k: {"launches": len(v), "mfma_busy_pct": round(sum(v) / len(v), 2),
            "source_sha": kind_source_hash(k)} for k, v in sorted(acc.items())}}


def _profile_blob(name):
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    i = text.find("```json")
    if i < 0:
        return None
    return json.loads(text[i + 7: text.index("```", i + 7)])


def load_mfma(workload):
    """Measured MFMA busy percentage per kernel kind from the committed counter summary, or
    {} -- a kind whose sources changed since the counters were taken is dropped."""
    blob = _profile_blob(f"mfma_util_{workload}.md")
    if blob is None:
        return {}
    return {k: v["mfma_busy_pct"] for k, v in blob["kinds"].items()
            if v.get("source_sha") == kind_source_hash(k)}


def load_traffic(workload):
    """Measured HBM bytes per launch per kernel kind from the committed counter summary,
    or {} -- a kind whose sources changed since the counters were taken is dropped."""
    blob = _profile_blob(f"hbm_traffic_{workload}.md")
    if blob is None:
        return {}
    return {k: v["hbm_bytes_per_launch"] for k, v in blob["kinds"].items()
            if v.get("source_sha") == kind_source_hash(k)}


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _threads_in_use():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        return os.cpu_count() or 1


def one_thread(fn, *a):
    """fn(*a) with numpy's BLAS and torch's intra-op pool limited to one thread."""
    import torch
    from threadpoolctl import threadpool_limits
    nt = torch.get_num_threads()
    torch.set_num_threads(1)
    try:
        with threadpool_limits(1):
            return fn(*a)
    finally:
        torch.set_num_threads(nt)


def cpu_baseline(w, W, batch, n_sessions, sessions=None):
    """The oracle as it stands on n_sessions whole sessions: the tree forward through every
    layer, the verify stage of every row and the walk."""
    import numpy as np
    from oracle import model as om
    from oracle import verify as ov
    cores = _threads_in_use()
    sess = (list(sessions) if sessions is not None
            else list(range(min(n_sessions, batch.tokens.shape[0]))))
    # host copies of everything the sample reads, taken before the oracle clock starts
    Wh = type(W)(W.embed.cpu(), [{k: v.cpu() for k, v in lw.items()} for lw in W.layers],
                 W.final_norm.cpu(), W.lm_head.cpu())
    S = {b: int(batch.prefix_len[b]) for b in sess}
    kv = {(l, b): (om.k_prefix(batch.kv_k, l, b, S[b]), om.v_prefix(batch.kv_v, l, b, S[b]))
          for l in range(w.L) for b in sess}
    toks, pars = batch.tokens.cpu(), batch.parents.cpu()
    q = batch.q[sess].cpu().numpy().astype(np.float64)
    u = batch.u[sess].cpu().numpy().astype(np.float64)
    t0 = time.perf_counter()
    z = om.forward_tree_batch(Wh, om.dims_of(w), toks, pars, batch.prefix_len.cpu(),
                              lambda l, b: kv[(l, b)], sess)
    for i, b in enumerate(sess):
        tk = [int(t) for t in toks[b]]
        pr = [int(p) for p in pars[b]]
        res = ov.verify_session(z[i], q[i], tk, pr, u[i], w.T, w.top_p, w.top_k)
        ov.walk(tk, pr, res)
    t = time.perf_counter() - t0
    n_tok = len(sess) * (toks.shape[1] - 1)
    B = batch.tokens.shape[0]
    return {"value": n_tok / t, "unit": "verified tree tokens/s", "cores": int(cores),
            "kind": "oracle", "cpu_model": cpu_model(),
            "extrapolated": (f"linear in sessions (each session's outputs depend on its own "
                             f"inputs only): {len(sess)} of {B} sessions timed")
            if len(sess) < B else None,
            "sample": (f"{len(sess)} of {B} sessions of {w.name} "
                       f"({n_tok} drafted nodes): full float64 forward through all {w.L} "
                       f"layers, verify stage of every row, walk; {t:.1f} s")}


def cpu_baseline_tail(w, W, batch, n_chains):
    """The oracle as it stands on n_chains whole chains of the LM-head tail: logits of every
    row in float64, the verify stage of every row and the chain walk."""
    import numpy as np
    from oracle import model as om
    from oracle import verify as ov
    cores = _threads_in_use()
    rows = list(range(min(n_chains * w.chain_len, w.rows)))
    Wh = type(W)(None, [], None, W.lm_head.cpu())
    hid = batch.hidden[rows].cpu()
    q = batch.q[rows].cpu().numpy().astype(np.float64)
    u = batch.u[rows].cpu().numpy().astype(np.float64)
    d = batch.draft_tokens[rows].cpu().numpy()
    t0 = time.perf_counter()
    z = om.lm_head_tail(Wh, hid)
    res = ov.verify_tail(z, q, d, u, w.T, w.top_p, w.top_k, w.chain_len)
    ov.walk_tail(res["accept"], res["resample"], w.chain_len)
    t = time.perf_counter() - t0
    return {"value": len(rows) / t, "unit": "verified tree tokens/s", "cores": int(cores),
            "kind": "oracle", "cpu_model": cpu_model(),
            "extrapolated": (f"linear in rows (each row's outputs depend on its own inputs "
                             f"only): {len(rows)} of {w.rows} rows timed")
            if len(rows) < w.rows else None,
            "sample": (f"{len(rows) // w.chain_len} of {w.rows // w.chain_len} chains of {w.name} "
                       f"({len(rows)} rows): float64 LM head, verify stage of every row, chain "
                       f"walk; {t:.1f} s")}


# ---------------------------------------------------------------------------------------
# Achievable peaks: what this chip sustains, measured beside the published figures
# ---------------------------------------------------------------------------------------


def calibrate(reps=5):
    """Median rate of (a) a plain 1 GiB device copy and (b) the MFMA pipe on random fp16
    operands (v_mfma_f32_16x16x32_f16, 16 independent accumulators a wave, no memory
    traffic in the loop), both timed with HIP events on the current stream."""
    import ctypes
    import statistics
    import torch
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2609_02514_amd", "libacespec_calib.so"))
    lib.acespec_calib_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                       ctypes.c_int, ctypes.c_void_p]
    lib.acespec_calib_mfma.argtypes = [ctypes.c_uint32, ctypes.c_void_p, ctypes.c_int,
                                       ctypes.c_int, ctypes.c_void_p]
    lib.acespec_calib_read.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                       ctypes.c_int, ctypes.c_void_p]
    stream = torch.cuda.current_stream()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    nbytes = 1 << 30
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").normal_()
    dst = torch.empty_like(src)
    blocks, iters = 2 * cus, 30000      # 2 waves a SIMD
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")

    def timed(fn):
        ts = []
        for _ in range(reps + 1):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            rc = fn()
            e1.record(stream)
            torch.cuda.synchronize()
            assert rc == 0, rc
            ts.append(e0.elapsed_time(e1))
        return statistics.median(ts[1:])   # the first run warms up

    ms_copy = timed(lambda: lib.acespec_calib_copy(src.data_ptr(), dst.data_ptr(), nbytes,
                                                   cus * 16, stream.cuda_stream))
    rblocks = cus * 32
    rout = torch.empty(rblocks * 4, dtype=torch.float32, device="cuda")
    ms_read = timed(lambda: lib.acespec_calib_read(src.data_ptr(), rout.data_ptr(), nbytes,
                                                   rblocks, stream.cuda_stream))
    ms_mfma = timed(lambda: lib.acespec_calib_mfma(12345, out.data_ptr(), blocks, iters,
                                                   stream.cuda_stream))
    flops = blocks * 4 * iters * 16 * 16384.0
    del src, dst, out
    return {"hbm_copy_gbs": round(2 * nbytes / (ms_copy / 1e3) / 1e9, 1),
            "hbm_read_gbs": round(nbytes / (ms_read / 1e3) / 1e9, 1),
            "mfma_f16_loop_tflops": round(flops / (ms_mfma / 1e3) / 1e12, 1),
            "method": (f"median of {reps} HIP-event-timed runs: a 1 GiB device copy "
                       f"(16-byte loads and stores, read + write bytes counted), a 1 GiB "
                       f"streaming read (eight nontemporal 16-byte loads in flight a thread), and "
                       f"{blocks} workgroups x 4 waves x {iters} x 16 MFMAs 16x16x32 f16 on "
                       f"random operands generated in registers")}


def lds_patterns():
    """Lane byte offsets of the verify kernels' 16-byte LDS fragment reads (lane l reads
    row l % 16, logical piece l / 16 of a 16-row block), under the XOR swizzles tried."""
    def gemm(rowb, sw):
        return [(l & 15) * rowb + (((l >> 4) ^ sw(l & 15)) << 4) for l in range(64)]

    def key_of_row(kk, m):
        return (kk >> 1) * 32 + (m >> 2) * 8 + (kk & 1) * 4 + (m & 3)

    def attn_k(sw, kk=1, s=0):   # 256-byte key rows (head dim 128), fp16 elements
        out = []
        for l in range(64):
            key = key_of_row(kk, l & 15)
            out.append(2 * (key * 128 + (((s * 4 + (l >> 4)) ^ sw(key)) << 3)))
        return out

    def p32(r):   # key held by A row r of the 32-row-tile kernel's 32 x 32 score block
        return ((r >> 4) & 1) * 16 + ((r >> 2) & 1) * 8 + ((r >> 3) & 1) * 4 + (r & 3)

    def attn_k32(sw, s=0):   # its key fragments: row p32(l % 32), logical piece 2 s + l / 32
        return [2 * (p32(l & 31) * 128 + (((2 * s + (l >> 5)) ^ sw(p32(l & 31))) << 3))
                for l in range(64)]

    def attn_v(sw, ks=0, nb=0):  # 128-byte V^T rows (64 slots)
        out = []
        for l in range(64):
            row = nb * 16 + (l & 15)
            out.append(2 * (row * 64 + (((ks * 4 + (l >> 4)) ^ sw(row)) << 3)))
        return out

    return [
        ("contiguous 1 KB", [16 * l for l in range(64)]),
        ("GEMM 64-byte rows, piece ^ (row / 4)", gemm(64, lambda r: (r >> 2) & 3)),
        ("GEMM 64-byte rows, piece ^ (row / 2)", gemm(64, lambda r: (r >> 1) & 3)),
        ("GEMM 128-byte rows, piece ^ (row / 2)", gemm(128, lambda r: (r >> 1) & 7)),
        ("attention K rows, key swizzle", attn_k(lambda k: (((k >> 3) & 3) << 2) | (k & 3))),
        ("attention V^T rows, row ^ (row / 8)", attn_v(lambda r: (r & 7) ^ ((r >> 3) & 1))),
        ("attention V^T rows, row / 2", attn_v(lambda r: (r >> 1) & 7)),
        ("attention 32-row tiles, K rows, its key swizzle",
         attn_k32(lambda k: (k & 0xB) | ((((k >> 2) ^ (k >> 4)) & 1) << 2))),
        ("attention 32-row tiles, K rows, the 16-row kernel's key swizzle",
         attn_k32(lambda k: (((k >> 3) & 3) << 2) | (k & 3))),
        ("attention 32-row tiles, K rows, piece ^ (key % 16)", attn_k32(lambda k: k & 15)),
    ]


def lds_probe(reps=3):
    """Read rate of every pattern of lds_patterns() (best of reps), B/clk/CU at 2.4 GHz."""
    import ctypes
    import torch
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2609_02514_amd", "libacespec_calib.so"))
    lib.acespec_calib_lds.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                      ctypes.c_int, ctypes.c_void_p]
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    blocks, iters = 4 * cus, 4096
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    res = []
    for name, offs in lds_patterns():
        assert len(offs) == 64 and all(0 <= o < 16384 and o % 16 == 0 for o in offs), name
        d = torch.tensor(offs, dtype=torch.int32, device="cuda")
        best = 1e30
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            rc = lib.acespec_calib_lds(d.data_ptr(), out.data_ptr(), blocks, iters,
                                       stream.cuda_stream)
            e1.record(stream)
            torch.cuda.synchronize()
            assert rc == 0, rc
            best = min(best, e0.elapsed_time(e1))
        nbytes = blocks * 256 * iters * 8 * 16
        res.append((name, round(best, 3), round(nbytes / (best * 1e-3) / cus / 2.4e9, 1)))
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="8b-bf16")
    ap.add_argument("--layout", choices=("auto", "packed", "rows"), default="auto",
                    help="dense weight matrices of the tree step: packed fragment order "
                         "(acespec_pack_weight) or row-major bf16; auto = packed for bf16 "
                         "models (measured faster from 272 to 4096 rows), row-major for fp32")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="capture one step into a HIP graph (stream capture) and time its "
                         "replays; the dominant kernel's launches are then timed in as many "
                         "eager steps run right after the timed replays")
    ap.add_argument("--cpu-sessions", type=int, default=4)
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run one plain device-to-device copy of MIB MiB (the reference "
                         "kernel that scales the FETCH_SIZE / WRITE_SIZE counters)")
    ap.add_argument("--summarize-pmc", nargs=4, metavar=("FETCH", "WRITE", "COPY_FETCH", "COPY_WRITE"),
                    help="print the per-kernel HBM traffic summary of four rocprofv3 --pmc "
                         "output directories (bench FETCH_SIZE, bench WRITE_SIZE, copy "
                         "FETCH_SIZE, copy WRITE_SIZE)")
    ap.add_argument("--copy-mib", type=int, default=1024)
    ap.add_argument("--lds-probe", action="store_true",
                    help="only measure the LDS read rate of the kernels' fragment patterns")
    ap.add_argument("--calibrate", action="store_true",
                    help="only measure the achievable copy, read and MFMA rates")
    ap.add_argument("--summarize-mfma", metavar="DIR",
                    help="print the per-kernel MFMA busy summary of one rocprofv3 "
                         "--pmc MfmaUtil output directory")
    args = ap.parse_args()
    if args.summarize_pmc:
        print(json.dumps(summarize_pmc(*args.summarize_pmc, args.copy_mib), indent=1))
        return
    if args.summarize_mfma:
        print(json.dumps(summarize_mfma(args.summarize_mfma), indent=1))
        return
    if args.lds_probe:
        for name, ms, bpc in lds_probe():
            print(json.dumps({"pattern": name, "ms": ms, "bytes_per_clk_per_cu_at_2.4GHz": bpc}))
        return
    if args.calibrate:
        print(json.dumps(calibrate()))
        return
    if args.copy_calibration:
        import torch
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.empty(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n * 4, "read_bytes": n * 4, "write_bytes": n * 4}))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus}): the verify step "
              "shards by session with no collectives, and only the one-GPU step is built "
              "and measured", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    from paper_2609_02514_amd.acespec import (Verifier, acespec_timing_enable, acespec_timing_only,
                                              acespec_timing_read)

    torch.cuda.set_device(0)
    w = synth.get(args.workload)
    tail = w.tree == "tail"
    log(f"generating {w.name} on the GPU")
    W = synth.make_weights(w, "cuda", progress=log)
    batch = synth.make_batch(w, "cuda", progress=log)
    v = Verifier.for_workload(w)
    if args.layout == "auto":
        args.layout = "packed" if w.dtype == "bf16" else "rows"
    if tail:
        # LM head + vocabulary verify over given hidden states: every row is the parent of
        # one drafted token (acespec_verify_tail); B chains of chain_len rows.
        R = w.rows
        B, n1 = R // w.chain_len, w.chain_len
        P, S_tot = R, 0
        outs = v.alloc_outputs(R, B, n1, w.top_k, w.V, "cuda", False)
        packed = args.layout == "packed"
        Wg = v.pack_weights(W, drop_source=args.no_cpu_baseline) if packed else W
        torch.cuda.synchronize()

        def step():
            v.verify_tail(Wg.lm_head, None, batch.hidden, batch.draft_tokens, batch.q, batch.u,
                          w.chain_len, w.T, w.top_p, w.top_k, outs, packed=packed)
    else:
        B, n1 = batch.tokens.shape
        parents = synth.tree_parents(w)
        P = sum(1 for c in synth.children_lists(parents) if c) * B
        S_tot = int(batch.prefix_len.sum().item()) + B * n1
        # packed: the dense matrices re-laid out once, before anything is timed (a server
        # does this when it loads the model); the row-major W stays for the oracle
        # (without the oracle's CPU baseline nothing reads the row-major copy again: it is
        # released as it is packed, which lets the 70B-class shape fit one GPU packed)
        Wg = (v.pack_weights(W, drop_source=args.no_cpu_baseline) if args.layout == "packed"
              else W)
        torch.cuda.synchronize()
        ws = v.weights_struct(Wg)
        outs = v.alloc_outputs(B * n1, B, n1, w.top_k, w.V, "cuda", False)

        def step():
            v.verify_tree(ws, batch.kv_k, batch.kv_v, batch.cap, batch.prefix_len, batch.tokens,
                          batch.parents, batch.q, batch.u, w.T, w.top_p, w.top_k, outs)

    log(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    work = kernel_work(w, B, n1, P, S_tot)

    def breakdown(per_kernel, nsteps):
        kernels = {}
        for name, (ms, cnt) in per_kernel.items():
            avg = ms / max(cnt, 1)
            ent = {"ms_per_step": round(ms / nsteps, 4), "avg_launch_ms": round(avg, 5),
                   "launches_per_step": cnt // nsteps}
            if name in work:
                fl, by = work[name]
                if fl and name.startswith("gemm"):
                    ent["tflops"] = round(fl / (avg / 1e3) / 1e12, 1)
                    ent["mfma_frac"] = round(ent["tflops"] / PEAK_MFMA_TFLOPS, 4)
                if by:
                    ent["gbs"] = round(by / (avg / 1e3) / 1e9, 1)
                    ent["hbm_frac"] = round(ent["gbs"] / PEAK_HBM_GBS, 4)
            kernels[name] = ent
        return kernels

    graph = None
    if args.graph:
        # The step enqueues kernel launches only (no allocation, memset, synchronisation
        # or, with timing off, events), so it captures as it is.
        acespec_timing_enable(v.ctx, False)
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            step()
        stream.wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        log("captured one step into a graph")

    # Per-kernel breakdown: the same steps with HIP events around every kernel (each
    # recorded pair costs stream time, so this pass is kept out of the timed region).
    acespec_timing_only(v.ctx, None)
    acespec_timing_enable(v.ctx, True)
    acespec_timing_read(v.ctx)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    kernels = breakdown(acespec_timing_read(v.ctx), args.steps)
    dom = max(kernels, key=lambda k: kernels[k]["ms_per_step"])

    # Timed region: exactly K steps, each bracketed by its own HIP event pair on the launch
    # stream, with the L2 and MALL flushed before every step outside its events (a 512 MB
    # buffer is read and written: 2x the 256 MB MALL), so no step finds the previous one's
    # weights or KV in cache; ms/step is the median.  The library records events around
    # the dominant kernel kind only, and only in about five of the steps (each recorded
    # pair costs stream time); their launches give the roofline's average duration,
    # measured live on the launch stream.
    import statistics
    acespec_timing_only(v.ctx, dom)
    acespec_timing_read(v.ctx)
    every = max(1, args.steps // 5)
    flush = torch.zeros((512 << 20) // 4, dtype=torch.float32, device="cuda")
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    if args.graph:
        acespec_timing_enable(v.ctx, False)
        for i in range(args.steps):
            flush.add_(1.0)
            ev[i][0].record(stream)
            graph.replay()
            ev[i][1].record(stream)
        torch.cuda.synchronize()
        t_wall = time.perf_counter() - t_wall
        for i in range(0, args.steps, every):   # the dominant kind, in eager steps
            flush.add_(1.0)
            acespec_timing_enable(v.ctx, True)
            step()
        acespec_timing_enable(v.ctx, False)
        torch.cuda.synchronize()
    else:
        for i in range(args.steps):
            flush.add_(1.0)
            acespec_timing_enable(v.ctx, i % every == 0)
            ev[i][0].record(stream)
            step()
            ev[i][1].record(stream)
        torch.cuda.synchronize()
        t_wall = time.perf_counter() - t_wall
    step_ms = [a.elapsed_time(b) for a, b in ev]
    timed_steps = len(range(0, args.steps, every))
    dk = breakdown(acespec_timing_read(v.ctx), timed_steps)[dom]
    acespec_timing_enable(v.ctx, False)
    acespec_timing_only(v.ctx, None)
    del flush
    ms_step = statistics.median(step_ms)
    tokens = B * n1 if tail else B * (n1 - 1)   # drafted tokens verified per step
    value = tokens / (ms_step / 1e3)
    log(f"{args.steps} steps: median {ms_step:.3f} ms/step (mean {statistics.mean(step_ms):.3f}, "
        f"min {min(step_ms):.3f}, max {max(step_ms):.3f}; wall incl. flushes "
        f"{t_wall / args.steps * 1e3:.3f}), {value:.0f} tok/s; "
        f"status {outs['status'].tolist()[:4]}...")
    ach = calibrate()
    log(f"achievable: copy {ach['hbm_copy_gbs']} GB/s, read {ach['hbm_read_gbs']} GB/s, MFMA loop "
        f"{ach['mfma_f16_loop_tflops']} TFLOP/s")

    traffic = load_traffic(w.name)
    mfma_busy = load_mfma(w.name)
    for name, ent in kernels.items():
        if name in traffic:
            ent["hbm_traffic_bytes_per_launch"] = traffic[name]
        if name in mfma_busy:
            ent["mfma_busy_pct_pmc"] = mfma_busy[name]
    for name, ent in kernels.items():
        if "tflops" in ent:
            ent["mfma_frac_achievable"] = round(ent["tflops"] / ach["mfma_f16_loop_tflops"], 4)
        if "gbs" in ent:
            ent["hbm_frac_achievable"] = round(ent["gbs"] / ach["hbm_read_gbs"], 4)
    if dom.startswith("gemm"):
        roof = {"kernel": dom, "bound": "mfma", "achieved": dk["tflops"],
                "peak": PEAK_MFMA_TFLOPS, "unit": "TFLOP/s", "frac": dk["mfma_frac"],
                "traffic": traffic.get(dom), "achievable": ach["mfma_f16_loop_tflops"],
                "frac_of_achievable": round(dk["tflops"] / ach["mfma_f16_loop_tflops"], 4)}
    else:
        roof = {"kernel": dom, "bound": "hbm", "achieved": dk["gbs"], "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": dk["hbm_frac"], "traffic": traffic.get(dom),
                "achievable": ach["hbm_read_gbs"],
                "frac_of_achievable": round(dk["gbs"] / ach["hbm_read_gbs"], 4)}
    roof["traffic_unit"] = "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)"
    roof["algorithmic_per_launch"] = {"flops": work[dom][0], "bytes": work[dom][1]} if dom in work else None

    # The commit that follows a verify round (Algorithm 1, COMPACT_KV), timed on its own
    # over the kept paths of the last verify step.
    commit = None
    if w.L > 0:
        new_len = torch.empty(B, dtype=torch.int32, device="cuda")
        acespec_timing_enable(v.ctx, True)
        acespec_timing_read(v.ctx)
        for _ in range(args.steps):
            v.commit_kv(batch.kv_k, batch.kv_v, batch.cap, batch.prefix_len, outs["path"],
                        outs["path_len"], outs["status"], new_len)
        ck = acespec_timing_read(v.ctx).get("commit_kv")
        acespec_timing_enable(v.ctx, False)
        kept = int(outs["path_len"].sum().item())
        moved = 2 * 2 * kept * w.L * w.Hkv * w.hd * 2   # K and V, read + write, bf16
        if ck:
            avg = ck[0] / max(ck[1], 1)
            commit = {"avg_launch_ms": round(avg, 5), "kept_rows": kept,
                      "algorithmic_bytes": moved, "gbs": round(moved / (avg / 1e3) / 1e9, 1)}

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the oracle on the host (bounded sample)")
        cpu = (cpu_baseline_tail(w, W, batch, args.cpu_sessions * 32) if tail
               else cpu_baseline(w, W, batch, args.cpu_sessions))
        log(f"oracle: {cpu['value']:.3f} tok/s on {cpu['cores']} threads")
        # per core: one thread on one session (one chain of the tail)
        one = one_thread(cpu_baseline_tail, w, W, batch, 1) if tail else \
            one_thread(cpu_baseline, w, W, batch, 1, [min(args.cpu_sessions, B - 1)])
        cpu["per_core"] = {"value": one["value"], "threads": 1, "sample": one["sample"]}
        log(f"oracle, one thread: {one['value']:.3f} tok/s")

    line = {
        "metric": ("verified tree tokens/s on 1 MI355X (8B shape)" if w.name == "8b-bf16"
                   else f"verified tree tokens/s on 1 MI355X ({w.name})"),
        "value": round(value, 1),
        "unit": "verified tree tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "step_ms_stats": {"median": round(ms_step, 4), "mean": round(statistics.mean(step_ms), 4),
                          "min": round(min(step_ms), 4), "max": round(max(step_ms), 4),
                          "timing": "one HIP event pair per step on the launch stream; L2 and "
                                    "MALL flushed (512 MB touched) before each step, outside "
                                    "its events" + ("; each step a replay of one captured "
                                                    "HIP graph" if args.graph else "")},
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 weights/KV, fp16 activations on f16 MFMA, fp32 accumulate",
        "data": "synthetic (seeded random-init weights, KV prefix, drafted trees, draft q)",
        "config": ({"workload": w.name, "d_model": w.d, "vocab": w.V, "rows": B * n1,
                    "chain_len": n1, "temperature": w.T, "top_p": w.top_p, "top_k": w.top_k,
                    "weight_layout": args.layout}
                   if tail else
                   {"workload": w.name, "layers": w.L, "d_model": w.d, "heads": w.H,
                    "kv_heads": w.Hkv, "head_dim": w.hd, "d_ff": w.F, "vocab": w.V,
                    "sessions": B, "prefix_len": w.S, "drafted_nodes": n1 - 1,
                    "temperature": w.T, "top_p": w.top_p, "top_k": w.top_k,
                    "weight_layout": args.layout}),
        "roofline": roof,
        "cpu_baseline": cpu,
        "kernels": kernels,
        "kernels_timing": "separate pass of the same steps with HIP events around every kernel "
                          "(the timed region records events around the roofline kernel only, "
                          "in about five of its steps)",
        "commit_kv": commit,
        "achievable_peaks": ach,
    }
    print(json.dumps(line), flush=True)
    v.close()


if __name__ == "__main__":
    main()
