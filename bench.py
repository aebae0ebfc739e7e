"""Throughput of the DiT denoising step on one MI355X.

Default workload: the video DiT step, 17550 latent tokens (13 frames x 30 x 45
patches of a 16-channel latent), batch 1, 30 blocks, hidden 3072, 24 heads x
128, MLP 12288, bf16 weights and GEMM operands with fp32 accumulation, a
given 3072-d conditioning vector.  One step = adaLN for all blocks + patch
embedding + 30 DiT blocks + final layer, all in the HIP library
(include/ditmi.h), inputs resident in HBM.  Weights are random-init
(N(0, 0.02), drawn on the device), latents N(0, 1).  --config selects the
other workloads (c1, c2: DiT-XL/2 at 256 and 1024 tokens; c3: the joint
text-image DiT).

Prints ONE JSON line on stdout with steps/s, the roofline of the dominant
kernel (measured with HIP events around its launches on the launch stream
during a repeat of the timed steps) and the fp64 CPU oracle timed on a
bounded sample; progress lines go to stderr.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "DiT denoising steps/sec at 1 GPU; GEMM+attention TFLOP/s as % of bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
CSRC = os.path.join(ROOT, "paper_2605_25550_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")

# kernel class -> (regex of its kernel symbol in rocprofv3 output, source file).  The
# GEMM classes differ in the last template argument (the fused epilogue), for
# both GEMM kernels (gemm_bf16_kernel<BM, BN, WGM, WGN, STAGES, EPI>,
# gemm_bf16_144_kernel<EPI>).
def _gemm_re(epi: int) -> str:
    # generic kernel: epilogue is the last of six template arguments; the
    # 64x144 kernel: <epilogue, k-groups>
    return rf"gemm_bf16_(?:kernel<(?:\d+, ){{5}}{epi}>|144_kernel<{epi}, \d+>)"


CLASSES = {
    "gemm_qkv": (_gemm_re(0), "gemm_bf16.hip"),
    "attention": (r"attn_bf16_\w*kernel<", "attention_bf16.hip"),
    "gemm_out": (_gemm_re(2), "gemm_bf16.hip"),
    "gemm_fc1": (_gemm_re(1), "gemm_bf16.hip"),
    "gemm_fc2": (_gemm_re(4), "gemm_bf16.hip"),
    "ln_mod": (r"ln_mod_kernel<", "elementwise.hip"),
    "adaln": (r"adaln\w*_kernel", "elementwise.hip"),
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="c4", help="workload key (c4, the largest, is the reported one)")
    ap.add_argument("--batch", type=int, default=0, help="override the workload's batch size (0: as configured)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-blocks", type=int, default=28,
                    help="oracle blocks in the CPU sample of the DiT-XL/2 workloads (one block for c3/c4)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="also run a plain device copy of this size (counter calibration runs)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="no GPU work: turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of this "
                         "command with --copy-probe-mib into profiles/<kernel>_<workload>_traffic.json")
    ap.add_argument("--kernel-class", default=None, help="kernel class for --summarize-pmc")
    ap.add_argument("--blas-ref", nargs="+", metavar="MxNxK",
                    help="time torch.matmul (hipBLASLt, bf16, no epilogue) at these GEMM shapes, for comparison "
                         "with paper_2605_25550_amd/gemm_probe; prints one line per shape")
    ap.add_argument("--summarize-profile", nargs=6,
                    metavar=("CONFIG", "TRACE_DIR", "PMC_DIR", "FETCH_DIR", "WRITE_DIR", "BENCH_JSON"),
                    help="no GPU work: write profiles/counters_<config>.md (and per-class traffic records) from a "
                         "kernel-trace run, a --pmc run of PMC_COUNTERS, FETCH_SIZE and WRITE_SIZE runs and the "
                         "bench line of the trace run")
    ap.add_argument("--serve", type=int, default=0,
                    help="time N requests through dit_serve (copies in order vs overlapped on a second "
                         "stream) with --sample-steps (default 1) Euler steps each")
    ap.add_argument("--sp-share", type=int, default=0, metavar="N",
                    help="time one GPU's part of an N-way sequence-parallel step of --config: the token share "
                         "(GEMMs, LayerNorm, embeddings on ceil(T/N) tokens, adaLN in full) and the head share "
                         "(attention of H/N heads over all T tokens); the all-to-alls are not run")
    ap.add_argument("--sample-steps", type=int, default=0,
                    help="instead of single steps, time the multi-step Euler sampler loop of this many steps "
                         "(eager and replayed from a captured HIP graph)")
    return ap.parse_args()


def progress(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def source_hash(fname: str) -> str:
    h = hashlib.sha256()
    for f in (fname, "common.h", "kernels.h"):
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_from_profile(kclass: str, workload: str):
    """HBM bytes per launch from the committed counter summary, if it was taken
    on the current kernel source; else None."""
    path = os.path.join(PROFILES, f"{kclass}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("source_hash") != source_hash(CLASSES[kclass][1]):
        return None
    return rec.get("hbm_bytes_per_launch")


def _pmc_rows(d):
    import csv
    import glob
    rows = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            rows += list(csv.DictReader(fh))
    return rows


def summarize_pmc(fetch_dir, write_dir, kclass, workload, copy_mib):
    """Per-launch HBM bytes of one kernel class from FETCH_SIZE / WRITE_SIZE
    (KiB per dispatch), each scaled by what the counter reads for a plain copy of
    copy_mib MiB (the largest copy dispatch of the run)."""
    import re
    pat = re.compile(CLASSES[kclass][0])
    out = {"kernel_class": kclass, "workload": workload, "source_hash": source_hash(CLASSES[kclass][1])}
    copy_bytes = copy_mib * (1 << 20)
    for name, d, counter in (("fetch", fetch_dir, "FETCH_SIZE"), ("write", write_dir, "WRITE_SIZE")):
        rows = [r for r in _pmc_rows(d) if r["Counter_Name"] == counter]
        kern = [float(r["Counter_Value"]) * 1024 for r in rows if pat.search(r["Kernel_Name"])]
        copies = [float(r["Counter_Value"]) * 1024 for r in rows
                  if "elementwise" in r["Kernel_Name"] or "copy" in r["Kernel_Name"].lower()]
        if not kern or not copies:
            raise SystemExit(f"no {counter} rows for {kclass} or for the copy probe in {d}")
        probe = max(copies)
        factor = probe / copy_bytes   # counter bytes per true byte (read once, or written once)
        out[f"{name}_counter_bytes_per_launch"] = sum(kern) / len(kern)
        out[f"{name}_copy_counter_bytes"] = probe
        out[f"{name}_factor"] = factor
        out[f"{name}_bytes_per_launch"] = out[f"{name}_counter_bytes_per_launch"] / factor
        out[f"{name}_launches"] = len(kern)
    out["hbm_bytes_per_launch"] = out["fetch_bytes_per_launch"] + out["write_bytes_per_launch"]
    path = os.path.join(PROFILES, f"{kclass}_{workload}_traffic.json")
    with open(path, "w") as fh:
        json.dump(out, fh, indent=1)
    print(json.dumps(out))


PMC_COUNTERS = ("MfmaUtil LdsUtil LDSBankConflict VALUBusy SQ_INSTS_VALU_MFMA_MOPS_BF16 "
                "SQ_VALU_MFMA_COEXEC_CYCLES GRBM_GUI_ACTIVE")


def summarize_profile(key, trace_dir, pmc_dir, fetch_dir, write_dir, bench_json, copy_mib):
    """profiles/counters_<key>.md: per kernel class, the kernel-trace average
    (from trace_dir), the counters of one --pmc pass (MFMA and LDS
    utilisation, VALU busy, MFMA ops, GRBM active cycles as the clock) and the
    HBM bytes of the FETCH_SIZE / WRITE_SIZE passes scaled by a plain copy of
    copy_mib MiB; algorithmic work per launch comes from the bench line of
    the trace run.  Also writes profiles/<class>_<key>_traffic.json for the
    bench's roofline.traffic."""
    import csv
    import glob
    import re
    import statistics

    import synth
    cfg = synth.CONFIGS[key]
    with open(bench_json) as fh:
        bench = json.loads([l for l in fh if l.startswith("{")][-1])
    alg = bench["kernel_algorithmic_per_launch"]
    stats = []
    for f in glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True):
        with open(f) as fh:
            stats += list(csv.DictReader(fh))
    pmc = _pmc_rows(pmc_dir)
    fetch = [r for r in _pmc_rows(fetch_dir) if r["Counter_Name"] == "FETCH_SIZE"]
    write = [r for r in _pmc_rows(write_dir) if r["Counter_Name"] == "WRITE_SIZE"]

    def copy_factor(rows):
        c = [float(r["Counter_Value"]) * 1024 for r in rows
             if "elementwise" in r["Kernel_Name"] or "copy" in r["Kernel_Name"].lower()]
        return max(c) / (copy_mib * (1 << 20)), max(c)

    f_fac, f_probe = copy_factor(fetch)
    w_fac, w_probe = copy_factor(write)
    out_rows = []
    for k, (rx, src) in CLASSES.items():
        pat = re.compile(rx)
        st = [r for r in stats if pat.search(r["Name"])]
        if not st:
            continue
        calls = sum(int(r["Calls"]) for r in st)
        avg_us = sum(float(r["TotalDurationNs"]) for r in st) / calls / 1e3
        names = sorted({r["Name"].split("(")[0].replace("void ditmi::", "") for r in st})
        a = alg.get(k, {})
        fl, by = a.get("flops", 0.0), a.get("bytes", 0.0)

        def per_dispatch(rows, counter):
            vals = [float(r["Counter_Value"]) for r in rows if r["Counter_Name"] == counter and pat.search(r["Kernel_Name"])]
            return statistics.mean(vals) if vals else None

        def mean_dur_ns(rows):
            d = {}
            for r in rows:
                if pat.search(r["Kernel_Name"]):
                    d[r["Dispatch_Id"]] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
            return statistics.mean(d.values()) if d else None

        row = {"class": k, "kernels": names, "calls": calls, "trace_avg_us": avg_us, "alg_flops": fl, "alg_bytes": by}
        for c in ("MfmaUtil", "LdsUtil", "LDSBankConflict", "VALUBusy", "SQ_INSTS_VALU_MFMA_MOPS_BF16",
                  "SQ_VALU_MFMA_COEXEC_CYCLES", "GRBM_GUI_ACTIVE"):
            row[c] = per_dispatch(pmc, c)
        dur = mean_dur_ns(pmc)
        row["pmc_dispatch_us"] = dur / 1e3 if dur else None
        # GRBM_GUI_ACTIVE is summed over the 8 XCDs.  It also counts the
        # counter pass's own per-dispatch overhead, so it gives the clock
        # only for dispatches long against that (>= 100 us).
        long_enough = dur is not None and dur >= 100e3
        row["clock_ghz"] = row["GRBM_GUI_ACTIVE"] / 8 / dur if long_enough and row["GRBM_GUI_ACTIVE"] else None
        fb, wb = per_dispatch(fetch, "FETCH_SIZE"), per_dispatch(write, "WRITE_SIZE")
        row["fetch_bytes"] = fb * 1024 / f_fac if fb is not None else None
        row["write_bytes"] = wb * 1024 / w_fac if wb is not None else None
        out_rows.append(row)
        if row["fetch_bytes"] is not None and row["write_bytes"] is not None:
            rec = {"kernel_class": k, "workload": key, "source_hash": source_hash(src),
                   "fetch_bytes_per_launch": row["fetch_bytes"], "write_bytes_per_launch": row["write_bytes"],
                   "hbm_bytes_per_launch": row["fetch_bytes"] + row["write_bytes"], "fetch_factor": f_fac,
                   "write_factor": w_fac, "copy_probe_mib": copy_mib}
            with open(os.path.join(PROFILES, f"{k}_{key}_traffic.json"), "w") as fh:
                json.dump(rec, fh, indent=1)

    def f(v, fmt):
        return "-" if v is None else format(v, fmt)

    cmds = [
        f"rocprofv3 --kernel-trace --stats -f csv -d {trace_dir} -o t -- python -u bench.py --config {key} "
        f"--no-cpu-baseline > {bench_json}",
        f"rocprofv3 --kernel-trace --pmc {PMC_COUNTERS} -f csv -d {pmc_dir} -o a -- python -u bench.py --config {key} "
        f"--no-cpu-baseline --steps 2 --warmup 1",
        f"rocprofv3 --pmc FETCH_SIZE -f csv -d {fetch_dir} -o f -- python -u bench.py --config {key} --no-cpu-baseline "
        f"--steps 2 --warmup 1 --copy-probe-mib {copy_mib}",
        f"rocprofv3 --pmc WRITE_SIZE -f csv -d {write_dir} -o w -- python -u bench.py --config {key} --no-cpu-baseline "
        f"--steps 2 --warmup 1 --copy-probe-mib {copy_mib}",
        f"python bench.py --summarize-profile {key} {trace_dir} {pmc_dir} {fetch_dir} {write_dir} {bench_json} "
        f"--copy-probe-mib {copy_mib}",
    ]
    L = [f"# Kernel counters: {cfg.name}", "",
         f"Workload {key}: batch {cfg.batch}, {cfg.tokens} tokens"
         f"{' + %d text tokens' % cfg.text_tokens if cfg.joint else ''}, hidden {cfg.hidden}, "
         f"{cfg.heads} x {cfg.head_dim} heads, MLP {cfg.mlp_hidden}, {cfg.n_blocks} blocks, bf16.  "
         f"Step: {bench['ms_per_step']} ms ({bench['value']} steps/s) in the trace run.", "",
         "Commands (repo root, one MI355X):", "", "```", *cmds, "```", "",
         "Columns: trace average per launch; algorithmic TFLOP/s and % of the 2.5 PFLOP/s dense bf16 peak; "
         "MfmaUtil = MFMA-busy cycles / (GRBM active cycles x SIMDs); MFMA ops / algorithmic flops "
         "(MOPS x 512; above 1 where MFMA tiles are padded, e.g. head_dim 72 -> 80); clock = GRBM active "
         "cycles per XCD / dispatch time in the counter pass, shown for dispatches of at least 100 us only (the "
         "GRBM count includes the counter pass's per-dispatch overhead, which also makes MfmaUtil understate "
         "short dispatches); LDS = LdsUtil and LDSBankConflict (% of "
         "active cycles); VALU = VALUBusy; HBM = FETCH_SIZE and WRITE_SIZE per launch, each divided by "
         f"what the counter reads for a {copy_mib} MiB device copy (fetch factor {f_fac:.3f}, write factor "
         f"{w_fac:.3f}), against the algorithmic bytes of the launch.", "",
         "| class | kernel | launches | avg us | TFLOP/s | % peak | MfmaUtil % | MFMA/alg | clock GHz | LDS util % | "
         "LDS conflict % | VALU % | fetch MB | write MB | HBM GB/s | alg MB | HBM/alg |",
         "|" + "---|" * 17]
    for r in out_rows:
        tf = r["alg_flops"] / (r["trace_avg_us"] * 1e-6) / 1e12 if r["alg_flops"] else None
        hbm = (r["fetch_bytes"] or 0) + (r["write_bytes"] or 0) if r["fetch_bytes"] is not None else None
        mops = r["SQ_INSTS_VALU_MFMA_MOPS_BF16"]
        L.append("| " + " | ".join([
            r["class"], "<br>".join(f"`{n}`" for n in r["kernels"]), str(r["calls"]), f(r["trace_avg_us"], ".2f"),
            f(tf, ".1f"), f(tf / PEAK_BF16_TFLOPS * 100 if tf else None, ".1f"), f(r["MfmaUtil"], ".1f"),
            f(mops * 512 / r["alg_flops"] if mops and r["alg_flops"] else None, ".3f"), f(r["clock_ghz"], ".2f"),
            f(r["LdsUtil"], ".1f"), f(r["LDSBankConflict"], ".2f"), f(r["VALUBusy"], ".1f"),
            f(r["fetch_bytes"] / 1e6 if r["fetch_bytes"] is not None else None, ".1f"),
            f(r["write_bytes"] / 1e6 if r["write_bytes"] is not None else None, ".1f"),
            f(hbm / (r["trace_avg_us"] * 1e-6) / 1e9 if hbm else None, ".0f"),
            f(r["alg_bytes"] / 1e6 if r["alg_bytes"] else None, ".1f"),
            f(hbm / r["alg_bytes"] if hbm and r["alg_bytes"] else None, ".2f")]) + " |")
    L += ["", f"Copy probe: FETCH_SIZE {f_probe / 2**20:.1f} MiB, WRITE_SIZE {w_probe / 2**20:.1f} MiB for a "
              f"{copy_mib} MiB copy.", ""]
    path = os.path.join(PROFILES, f"counters_{key}.md")
    with open(path, "w") as fh:
        fh.write("\n".join(L))
    print(path)


class Workload:
    def __init__(self, cfg, torch, dm):
        if cfg.grid is not None and cfg.grid[0] * cfg.grid[1] != cfg.tokens:
            # the step reads one position row per token
            raise ValueError(f"{cfg.name}: position grid {cfg.grid} does not match {cfg.tokens} tokens")
        self.cfg = cfg
        self.torch = torch
        self.dm = dm
        self.shape = dm.shape_of(cfg)
        self.dt = dm.weight_dtype(self.shape)
        D, F = cfg.hidden, cfg.mlp_hidden
        g = torch.Generator(device="cuda")
        g.manual_seed(2605)

        def rnd(*s, std=0.02):
            return (torch.randn(*s, device="cuda", generator=g) * std).to(self.dt)

        def stream():
            return {"w_ada": rnd(6 * D, D), "b_ada": rnd(6 * D), "w_qkv": rnd(3 * D, D), "b_qkv": rnd(3 * D),
                    "w_o": rnd(D, D), "b_o": rnd(D), "w_fc1": rnd(F, D), "b_fc1": rnd(F), "w_fc2": rnd(D, F),
                    "b_fc2": rnd(D)}

        self.blocks, structs = [], []
        for _ in range(cfg.n_blocks):
            img = stream()
            txt = stream() if cfg.joint else None
            self.blocks.append((img, txt))
            structs.append(dm.block_struct(img, txt, self.dt))
        self.step_w = {"w_patch": rnd(D, cfg.patch_in), "b_patch": rnd(D), "w_ada_final": rnd(2 * D, D),
                       "b_ada_final": rnd(2 * D), "w_final": rnd(cfg.patch_out, D), "b_final": rnd(cfg.patch_out)}
        self.pos = None
        if cfg.grid is not None:
            self.pos = torch.empty((cfg.grid[0] * cfg.grid[1], D), dtype=torch.float32, device="cuda")
            dm.pos_embed_2d(cfg.grid[0], cfg.grid[1], D, self.pos)
        self.table = dm.StepWeightTable(self.step_w, structs, self.dt, self.pos)
        self.ws = dm.alloc_workspace(self.shape, dm.DIT_WS_STEP)
        B, T = cfg.batch, cfg.tokens
        self.patches = torch.randn(B, T, cfg.patch_in, device="cuda", generator=g)
        self.x_txt = torch.randn(B, cfg.text_tokens, D, device="cuda", generator=g) if cfg.joint else None
        self.out = torch.empty(B, T, cfg.patch_out, device="cuda")
        if cfg.cond == "class":
            self.cond_w = {"w_t1": rnd(D, cfg.freq_dim), "b_t1": rnd(D), "w_t2": rnd(D, D), "b_t2": rnd(D),
                           "class_table": rnd(cfg.n_classes + 1, D)}
            self.t = torch.randint(0, 1000, (B,), device="cuda", generator=g).float()
            self.y = torch.randint(0, cfg.n_classes, (B,), device="cuda", generator=g).int()
            self.ws_cond = self.dm.alloc_workspace(self.shape, dm.DIT_WS_COND)
            self.cond = torch.empty(B, D, device="cuda")
        else:
            self.cond = torch.randn(B, D, device="cuda", generator=g)

    def step(self):
        if self.cfg.cond == "class":
            self.dm.cond_embed(self.shape, self.t, self.y, self.cond_w, self.cond, self.ws_cond)
        self.dm.step_forward(self.shape, self.table, self.patches, self.cond, self.out, self.ws, x_txt=self.x_txt)


def algorithmic_flops(cfg) -> float:
    """GEMMs (2 B T D (3D + D + 2 F) per stream-block: QKV, output projection,
    fc1 and fc2 with MLP width F; 24 B T D^2 at F = 4D) + attention
    (4 B Tj^2 D per block over the joint sequence Tj)."""
    T, Tt, B, D, F = cfg.tokens, cfg.text_tokens, cfg.batch, cfg.hidden, cfg.mlp_hidden
    return cfg.n_blocks * (2.0 * B * (T + Tt) * D * (4 * D + 2 * F) + 4.0 * B * (T + Tt) ** 2 * D)


def host_info() -> dict:
    """CPU model, core count and library versions of the host the oracle runs on."""
    import platform

    import numpy as np
    model = platform.processor() or "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    rocm = None
    for f in ("/opt/rocm/.info/version", "/opt/rocm/.info/version-dev"):
        if os.path.exists(f):
            with open(f) as fh:
                rocm = fh.read().strip()
            break
    return {"cpu_model": model, "cpu_count": os.cpu_count(), "numpy": np.__version__, "rocm": rocm}


def cpu_baseline(cfg, n_blocks_sample: int):
    """fp64 oracle on the host.  DiT-XL/2 workloads: conditioning + patch embed +
    n_blocks_sample blocks (one block's weights reused) + final layer at the
    full batch, scaled to the full block count.  Joint and video workloads:
    one full-size block, timed once, times the block count (labelled
    extrapolated; the embedding and final layer are below 0.1% of a block)."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import synth
    from oracle import dit_oracle as O

    scfg = synth.CONFIGS[cfg.key]
    info = host_info()
    threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    bw = synth.block_weights(scfg, 0)
    blk = {k: {n: a.astype(np.float64) for n, a in v.items()} for k, v in bw.items()}
    inp = synth.inputs(scfg)
    if scfg.key in ("c3", "c4"):
        t0 = time.perf_counter()
        if scfg.joint:
            O.joint_block(inp["x"], inp["x_txt"], inp["cond"], blk["img"], blk["txt"], scfg.heads, scfg.ln_eps)
        else:
            O.dit_block(inp["x"], inp["cond"], blk["img"], scfg.heads, scfg.ln_eps)
        t_block = time.perf_counter() - t0
        sec_per_step = t_block * scfg.n_blocks
        return {"value": 1.0 / sec_per_step, "unit": "steps/s", "cores": threads, "kind": "oracle",
                "extrapolated": True, **info,
                "sample": f"fp64 numpy oracle, one full-size block ({scfg.tokens} tokens"
                          f"{' + %d text' % scfg.text_tokens if scfg.joint else ''}, block 0's weights) timed once "
                          f"at {t_block:.2f} s, extrapolated x {scfg.n_blocks} blocks ({sec_per_step:.1f} s/step)"}
    sw = {k: v.astype(np.float64) for k, v in synth.step_weights(scfg).items()}
    blocks = [blk] * n_blocks_sample
    pos = O.pos_embed_2d(*scfg.grid, scfg.hidden) if scfg.grid else None
    t0 = time.perf_counter()
    if scfg.cond == "class":
        c = O.class_conditioning(inp["t"], inp["y"], sw["w_t1"], sw["b_t1"], sw["w_t2"], sw["b_t2"], sw["class_table"])
    else:
        c = inp["cond"]
    t_cond = time.perf_counter() - t0
    t1 = time.perf_counter()
    passes = 0
    while True:  # at least one pass, and at least ~10 s of oracle work
        O.dit_step(scfg.with_(n_blocks=n_blocks_sample), inp["patches"], c, sw, blocks, x_txt=inp.get("x_txt"),
                   pos=pos)
        passes += 1
        if time.perf_counter() - t1 >= 10.0:
            break
    t_step = (time.perf_counter() - t1) / passes
    # per-block share of the sampled run, extrapolated to all blocks (prologue/epilogue counted once)
    sec_per_step = t_cond + t_step * (scfg.n_blocks / n_blocks_sample)
    return {"value": 1.0 / sec_per_step, "unit": "steps/s", "cores": threads, "kind": "oracle",
            "extrapolated": n_blocks_sample != scfg.n_blocks, **info,
            "sample": f"fp64 numpy oracle, full batch {scfg.batch}: conditioning + patch embed + "
                      f"{n_blocks_sample} of {scfg.n_blocks} blocks (one block's weights) + final layer, "
                      f"{passes} pass(es) at {t_step:.2f} s each, scaled to {scfg.n_blocks} blocks "
                      f"({sec_per_step:.2f} s/step)"}


def sampler_bench(wl, args, torch, dm):
    """Denoising steps per second inside a K-step Euler sampler loop (the
    DiT stage's per-request work), launched eagerly and replayed from a
    captured HIP graph."""
    cfg = wl.cfg
    K = args.sample_steps
    sigmas = [1.0 - i / K for i in range(K + 1)]
    ws = dm.alloc_workspace(wl.shape, dm.DIT_WS_SAMPLE)
    kw = {"x_txt": wl.x_txt}
    if cfg.cond == "class":
        kw.update(cond_w=wl.cond_w, y=wl.y)
    else:
        kw["cond"] = wl.cond
    z0 = wl.patches.clone()
    z = z0.clone()

    def loop():
        dm.sample_euler(wl.shape, wl.table, z, sigmas, ws, **kw)

    loop()
    torch.cuda.synchronize()
    reps = max(1, args.steps // K)
    t0 = time.perf_counter()
    for _ in range(reps):
        z.copy_(z0)
        loop()
    torch.cuda.synchronize()
    eager_s = (time.perf_counter() - t0) / reps
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        loop()
    graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        z.copy_(z0)
        graph.replay()
    torch.cuda.synchronize()
    graph_s = (time.perf_counter() - t0) / reps
    print(json.dumps({
        "metric": f"DiT denoising steps/sec inside a {K}-step Euler sampler loop (per-step conditioning)",
        "value": round(K / eager_s, 3), "unit": "steps/s", "n_gpus": 1, "higher_is_better": True,
        "loop_ms": round(eager_s * 1e3, 3), "graph_value": round(K / graph_s, 3),
        "graph_loop_ms": round(graph_s * 1e3, 3), "loops_timed": reps, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": cfg.name, "blocks": cfg.n_blocks, "batch": cfg.batch, "tokens": cfg.tokens,
                   "sampler": "euler", "steps": K}}), flush=True)


def serve_bench(wl, args, torch, dm):
    """Requests through the DiT stage with host<->device latent copies in order
    and overlapped with compute on a second stream; reports how much of the
    copy time the overlap hides."""
    cfg = wl.cfg
    K = max(1, args.sample_steps)
    N = args.serve
    sigmas = [1.0 - i / K for i in range(K + 1)]
    ws = dm.alloc_workspace(wl.shape, dm.DIT_WS_SERVE)
    cond_w = wl.cond_w if cfg.cond == "class" else None
    reqs = []
    for i in range(N):
        r = {"z_in": wl.patches.cpu().pin_memory(), "z_out": torch.empty_like(wl.patches, device="cpu").pin_memory()}
        if cond_w is not None:
            r["y"] = wl.y.cpu()
        else:
            r["cond"] = wl.cond.cpu()
        reqs.append(r)
    cs = torch.cuda.Stream()

    def run(overlap):
        dm.serve(wl.shape, wl.table, reqs, sigmas, ws, cond_w=cond_w, overlap=overlap, copy_stream=cs)
        torch.cuda.synchronize()

    def timed(fn, reps=3):
        fn()
        t0 = time.perf_counter()
        for _ in range(reps):
            fn()
        return (time.perf_counter() - t0) / reps

    serial = timed(lambda: run(False))
    overlapped = timed(lambda: run(True))
    zd = wl.patches.clone()

    def copies():  # the same copies alone
        for r in reqs:
            zd.copy_(r["z_in"], non_blocking=True)
            r["z_out"].copy_(zd, non_blocking=True)
        torch.cuda.synchronize()

    copy_s = timed(copies)
    # the hidden share of the copy time is only resolvable when the copies are
    # a visible part of a request's time
    hidden = (serial - overlapped) / copy_s if copy_s > 0.05 * serial else None
    print(json.dumps({
        "metric": f"requests/sec through the DiT stage ({K}-step Euler loop each) with overlapped latent copies",
        "value": round(N / overlapped, 3), "unit": "requests/s", "n_gpus": 1, "higher_is_better": True,
        "serial_ms_per_request": round(serial / N * 1e3, 4), "overlapped_ms_per_request": round(overlapped / N * 1e3, 4),
        "copy_only_ms_per_request": round(copy_s / N * 1e3, 4),
        "copy_fraction_hidden": None if hidden is None else round(hidden, 3),
        "latent_bytes_each_way": int(wl.patches.numel() * 4), "requests": N, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": cfg.name, "blocks": cfg.n_blocks, "batch": cfg.batch, "tokens": cfg.tokens,
                   "sampler": "euler", "steps": K}}), flush=True)


def sp_share_bench(cfg, args, torch, dm):
    """One GPU's part of an N-way Ulysses sequence-parallel step, measured on
    one GPU.  Between the two all-to-alls of a block a GPU holds either
    ceil(T/N) tokens with all heads (LayerNorm, the four GEMMs, patch embed,
    final layer) or all T tokens of H/N heads (attention); the adaLN GEMV is
    replicated.  Token share: a full step at ceil(T/N) tokens, minus its own
    attention.  Head share: the attention launches of a step at H/N heads
    (hidden D/N) over all T tokens.  Both are timed with HIP events on the
    launch stream; the all-to-alls are not run (one GPU)."""
    import math
    N = args.sp_share
    if cfg.joint or cfg.heads % N or cfg.hidden % (64 * N):
        raise SystemExit("--sp-share needs a single-stream config with heads and hidden/64 divisible by N")
    cfg_tok = cfg.with_(tokens=math.ceil(cfg.tokens / N))
    cfg_head = cfg.with_(hidden=cfg.hidden // N, heads=cfg.heads // N, mlp_hidden=cfg.mlp_hidden // N)

    def measure(c, classes):
        wl = Workload(c, torch, dm)
        for _ in range(args.warmup):
            wl.step()
        st = torch.cuda.current_stream()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(st)
        for _ in range(args.steps):
            wl.step()
        ev1.record(st)
        torch.cuda.synchronize()
        step_ms = ev0.elapsed_time(ev1) / args.steps
        per = {}
        for k in classes:
            dm.timing_enable(k, 8192)
            for _ in range(args.steps):
                wl.step()
            torch.cuda.synchronize()
            ms, n, _, _ = dm.timing_read()
            dm.timing_disable()
            per[k] = ms / args.steps
        del wl
        torch.cuda.empty_cache()
        return step_ms, per

    tok_ms, tok_cls = measure(cfg_tok, ["attention"])
    _, head_cls = measure(cfg_head, ["attention"])
    share_ms = tok_ms - tok_cls["attention"] + head_cls["attention"]
    attn_flops = 4.0 * cfg.batch * (cfg.heads // N) * cfg.tokens ** 2 * cfg.head_dim * cfg.n_blocks
    print(json.dumps({
        "metric": f"one GPU's share of an {N}-way sequence-parallel DiT step (all-to-alls excluded), steps/s",
        "value": round(1000.0 / share_ms, 3), "unit": "steps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(share_ms, 4), "higher_is_better": True,
        "token_share_step_ms": round(tok_ms, 4), "token_share_attention_ms": round(tok_cls["attention"], 4),
        "head_share_attention_ms": round(head_cls["attention"], 4),
        "head_share_attention_tflops": round(attn_flops / (head_cls["attention"] * 1e-3) / 1e12, 1),
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{cfg.name}_sp{N}_share", "blocks": cfg.n_blocks, "tokens": cfg.tokens,
                   "token_share": cfg_tok.tokens, "heads": cfg.heads, "head_share": cfg_head.heads,
                   "hidden": cfg.hidden, "head_dim": cfg.head_dim, "mlp_hidden": cfg.mlp_hidden}}), flush=True)


def main():
    args = parse()
    if args.summarize_profile:
        summarize_profile(*args.summarize_profile, args.copy_probe_mib or 256)
        return
    if args.summarize_pmc:
        import synth
        summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1], args.kernel_class,
                      synth.CONFIGS[args.config].key, args.copy_probe_mib or 256)
        return
    if args.blas_ref:
        import torch
        torch.cuda.set_device(0)
        for spec in args.blas_ref:
            M, N, K = (int(v) for v in spec.lower().split("x"))
            a = torch.randn(M, K, device="cuda", dtype=torch.bfloat16)
            w = torch.randn(N, K, device="cuda", dtype=torch.bfloat16)
            for _ in range(5):
                c = a @ w.t()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(30):
                c = a @ w.t()
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / 30
            tf = 2.0 * M * N * K / (us * 1e-6) / 1e12
            print(f"torch.matmul bf16 {M}x{N}x{K}: {us:.2f} us  {tf:.1f} TFLOP/s  {100 * tf / PEAK_BF16_TFLOPS:.1f}%",
                  flush=True)
            del a, w, c
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (run with --gpus 1)",
              file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2605_25550_amd as dm
    import synth

    cfg = synth.CONFIGS[args.config]
    if args.batch and args.batch != cfg.batch:  # its own workload name; no traffic record applies
        cfg = cfg.with_(batch=args.batch, key=f"{cfg.key}_batch{args.batch}", name=f"{cfg.name}_batch{args.batch}")
    if cfg.dtype != "bf16":
        raise SystemExit("bench.py times the bf16 workloads (c1..c4)")
    torch.cuda.set_device(0)
    dm.lib()
    if args.sp_share:
        sp_share_bench(cfg, args, torch, dm)
        return
    progress(f"workload {cfg.name}: drawing weights on the device")
    wl = Workload(cfg, torch, dm)
    st = torch.cuda.current_stream()
    if args.serve:
        serve_bench(wl, args, torch, dm)
        return
    if args.sample_steps:
        sampler_bench(wl, args, torch, dm)
        return

    # warmup; afterwards measure each kernel class once to find the dominant one
    progress(f"warmup ({args.warmup} steps)")
    for _ in range(args.warmup):
        wl.step()
    torch.cuda.synchronize()
    share, alg = {}, {}
    for k in CLASSES:
        dm.timing_enable(k, 4096)
        wl.step()
        torch.cuda.synchronize()
        ms, n, fl, by = dm.timing_read()
        dm.timing_disable()
        share[k] = ms
        alg[k] = {"launches_per_step": n, "flops": fl / max(n, 1), "bytes": by / max(n, 1)}
    dominant = max(share, key=share.get)

    # timed region: K steps between synchronisations, events on the launch stream
    progress(f"timing {args.steps} steps")
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(st)
    for _ in range(args.steps):
        wl.step()
    ev1.record(st)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = ev0.elapsed_time(ev1)
    ms_per_step = gpu_ms / args.steps

    # roofline: the same K steps again with every launch of the dominant kernel
    # bracketed by HIP events on its launch stream (the library's timing hook);
    # kept out of the region above because the events add a little time per launch.
    progress(f"{ms_per_step:.3f} ms/step; timing every launch of {dominant}")
    dm.timing_enable(dominant, 8192)
    for _ in range(args.steps):
        wl.step()
    torch.cuda.synchronize()
    k_ms, k_n, k_flops, k_bytes = dm.timing_read()
    dm.timing_disable()

    if args.copy_probe_mib:
        n = args.copy_probe_mib * (1 << 20) // 4
        a = torch.ones(n, device="cuda")
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()

    per_launch_ms = k_ms / max(k_n, 1)
    flops_per_launch = k_flops / max(k_n, 1)
    bytes_per_launch = k_bytes / max(k_n, 1)
    mfma_bound = dominant.startswith("gemm") or dominant == "attention"
    if mfma_bound:
        achieved = flops_per_launch / (per_launch_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4)}
    else:
        achieved = bytes_per_launch / (per_launch_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4)}
    roof["traffic"] = traffic_from_profile(dominant, cfg.key)
    roof["kernel"] = dominant
    roof["launch_ms"] = round(per_launch_ms, 5)
    roof["launches"] = k_n
    roof["algorithmic_per_launch"] = flops_per_launch if mfma_bound else bytes_per_launch

    flops = algorithmic_flops(cfg)
    result = {
        "metric": METRIC,
        "value": round(1000.0 / ms_per_step, 3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": cfg.name, "blocks": cfg.n_blocks, "batch": cfg.batch, "tokens": cfg.tokens,
                   "text_tokens": cfg.text_tokens, "hidden": cfg.hidden, "heads": cfg.heads,
                   "head_dim": cfg.head_dim, "mlp_hidden": cfg.mlp_hidden, "conditioning": cfg.cond,
                   "parallelism": "single GPU"},
        "step_tflops": round(flops / (ms_per_step * 1e-3) / 1e12, 2),
        "step_frac_of_bf16_peak": round(flops / (ms_per_step * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "wall_s_timed": round(wall, 3),
        "kernel_ms_per_step": {k: round(v, 4) for k, v in share.items()},
        "kernel_algorithmic_per_launch": alg,
        "roofline": roof,
    }
    if not args.no_cpu_baseline and cfg.key in ("c1", "c2", "c3", "c4"):
        progress("timing the fp64 CPU oracle")
        result["cpu_baseline"] = cpu_baseline(cfg, min(args.cpu_blocks, cfg.n_blocks))
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
