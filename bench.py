#!/usr/bin/env python3
"""Throughput of K-Forcing joint next-k-token decoding on one MI355X.

A step is one kf_generate call over the whole batch: the prefill (prompt +
k noise rows) and every decode block (k emitted tokens + k fresh noise rows)
until L new tokens per sequence exist.  Default workload: the LM1B-shaped
GPT-2-small backbone in bf16 (12 layers, d=768, 12 heads, MLP 3072,
vocab 30522, context 128), batch 64, prompt 16 Zipf(1.1) tokens, k = 4,
112 new tokens (28 forward passes).  Weights, prompts and noise are seeded and
synthetic.

Printed (one JSON line): generated tokens/s at k (value), the k=1
autoregressive baseline on the same workload, the roofline position of the
dominant kernel class (HIP events on the library's stream), and the CPU oracle
timed on a bounded sample on the host.

    python bench.py [--steps K] [--warmup W] [--workload lm1b|owt|large|toy]
                    [--batch B] [--k K] [--no-cpu] [--no-ar]
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import kf_synth as S  # noqa: E402

PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_MFMA_TFLOPS = {1: 2500.0,  # dense bf16
                    0: 157.3}   # fp32 (matrix and vector)
METRIC = "generated tokens/sec at k=4 vs k=1 per batch size; HBM GB/s / MFMA util"
CLASSES = ["embed", "noise", "norm", "qkv", "attn", "oproj", "mlp_up", "mlp_down", "head",
           "select"]


# --------------------------------------------------------------------------
# Algorithmic cost of each kernel class (minimum bytes moved, flops)
# --------------------------------------------------------------------------

def step_costs(cfg: S.ModelConfig, B: int, nr: int, k: int, C: int) -> dict:
    """Per kernel class: the algorithmic (bytes, flops) of one step with B
    sequences, nr real rows and k noise rows per sequence over C committed
    positions -- what the method itself must move or compute:

      bytes: the weights each class reads once, the cached K/V the attention
             reads (C rows of 2 d elements per sequence and layer) and the K/V
             the QKV GEMM appends (every new row);
      flops: 2 M K N for each GEMM (M = B (nr + k) body rows, B k head rows, or
             B for an AR step), the noise encoder's two GEMMs on the B k noise
             rows, and 4 d per visible (query, key) pair of the attention.

    Activations, the fp32 residual stream and partial results are an
    implementation's own traffic and are not counted (operand_costs does)."""
    es = 2 if cfg.dtype == S.DTYPE_BF16 else 4
    d, f, V, L = cfg.d_model, cfg.d_mlp, cfg.vocab, cfg.n_layer
    R = nr + k
    M = B * R
    Mh = B * k if k > 0 else B
    c = {n: [0.0, 0.0] for n in CLASSES}

    def add(n, by, fl):
        c[n][0] += by
        c[n][1] += fl

    if k > 0:
        add("noise", 8 * d * d * es, 2 * B * k * 8 * d * d)
    visible = sum(C + i + 1 for i in range(R))  # keys seen by the R queries of a sequence
    for _ in range(L):
        add("qkv", 3 * d * d * es + B * R * 2 * d * es, 2 * M * 3 * d * d)
        add("attn", B * C * 2 * d * es, 4 * B * visible * d)
        add("oproj", d * d * es, 2 * M * d * d)
        add("mlp_up", f * d * es, 2 * M * f * d)
        add("mlp_down", d * f * es, 2 * M * d * f)
    add("head", V * d * es, 2 * Mh * V * d)
    return c


def operand_costs(cfg: S.ModelConfig, B: int, nr: int, k: int, C: int) -> dict:
    """A diagnostic beside step_costs: bytes of every operand of this
    implementation's kernels read or written once (weights, bf16 activations
    in and out, the fp32 residual stream read and written by out-proj and
    MLP-down, the cached rows each attention workgroup reads, Q and O).  Not a
    roofline: the activations are the implementation's own traffic."""
    es = 2 if cfg.dtype == S.DTYPE_BF16 else 4
    d, f, V, L = cfg.d_model, cfg.d_mlp, cfg.vocab, cfg.n_layer
    R = nr + k
    M = B * R
    Mk = B * k
    Mh = Mk if k > 0 else B
    c = {n: [0.0, 0.0] for n in CLASSES}

    def add(n, by):
        c[n][0] += by

    add("embed", B * nr * (2 * d * es + 4 * d))
    if k > 0:
        add("noise", Mk * d * es + 4 * d * d * es + Mk * 4 * d * es)
        add("noise", 4 * d * d * es + Mk * 4 * d * es + Mk * d * (4 + es))
    for _ in range(L):
        add("qkv", 3 * d * d * es + M * d * es + M * 3 * d * es)
        add("attn", B * (C + R) * 2 * d * es + 2 * M * d * es)
        add("oproj", d * d * es + M * d * es + 2 * M * d * 4)
        add("mlp_up", f * d * es + M * d * es + M * f * es)
        add("mlp_down", d * f * es + M * f * es + 2 * M * d * 4)
    add("head", V * d * es + Mh * d * es)
    add("select", Mh * 8)
    return c


def generate_costs(cfg, B, N, L, k, per_step=step_costs) -> dict:
    """Summed per-class costs of a kf_generate call: the prefill (N prompt rows
    + k noise rows, C = 0) and L/k - 1 decode blocks (k + k rows at
    C = N, N + k, ...)."""
    tot = {n: [0.0, 0.0] for n in CLASSES}
    steps = [(N, k, 0)] + [(k, k, N + (s - 1) * k) for s in range(1, L // k)]
    for nr, kk, C in steps:
        for n, (by, fl) in per_step(cfg, B, nr, kk, C).items():
            tot[n][0] += by
            tot[n][1] += fl
    return tot


def generate_ar_costs(cfg, B, N, L, per_step=step_costs) -> dict:
    """Summed per-class costs of a kf_generate_ar call (one row per step)."""
    tot = {n: [0.0, 0.0] for n in CLASSES}
    steps = [(N, 0)] + [(1, N + s - 1) for s in range(1, L)]
    for nr, C in steps:
        for n, (by, fl) in per_step(cfg, B, nr, 0, C).items():
            tot[n][0] += by
            tot[n][1] += fl
    return tot


# --------------------------------------------------------------------------

def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="lm1b", choices=sorted(S.WORKLOADS))
    ap.add_argument("--batch", type=int, default=None)
    ap.add_argument("--k", type=int, default=None)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-ar", action="store_true", help="skip the k=1 AR baseline")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the OpenWebText-shaped batch sweep and k comparison")
    ap.add_argument("--sweep-batches", default="1,16,32,64,256,512")
    ap.add_argument("--no-large", action="store_true",
                    help="skip the 24-layer backbone at batch 256")
    ap.add_argument("--large-only", action="store_true",
                    help="only the 24-layer backbone at batch 256 (one JSON line)")
    ap.add_argument("--no-serving", action="store_true",
                    help="skip the continuous-batching run")
    ap.add_argument("--serving-only", action="store_true",
                    help="only the continuous-batching run (one JSON line)")
    ap.add_argument("--no-train-attn", action="store_true",
                    help="skip the training-mask attention measurement")
    ap.add_argument("--train-attn-only", action="store_true",
                    help="measure only the training-mask attention and print its JSON")
    ap.add_argument("--no-teacher", action="store_true",
                    help="skip the distillation-target measurement")
    ap.add_argument("--teacher-only", action="store_true",
                    help="measure only the distillation targets and print their JSON")
    ap.add_argument("--no-rollout", action="store_true",
                    help="skip the self-forcing target measurement")
    ap.add_argument("--rollout-only", action="store_true",
                    help="measure only the self-forcing targets and print their JSON")
    ap.add_argument("--cpu-blocks", type=int, default=28,
                    help="decode blocks per sequence in the CPU oracle sample")
    ap.add_argument("--summarize", metavar="DIR", default=None,
                    help="print a markdown summary of rocprofv3 CSV output under DIR "
                         "(kernel stats, and FETCH_SIZE / WRITE_SIZE counter runs) and exit")
    ap.add_argument("--write-traffic", metavar="JSON", default=None,
                    help="with --summarize: also store the per-class traffic for bench.py")
    return ap.parse_args()


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def cpu_model_name() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(blob, prompt, k, seed, blocks):
    """The oracle's fp32 instantiation (the same loop nest as the parity
    oracle, OpenMP over sequences) on bounded samples, on this host's cores:

      value      -- the benchmark workload: one sequence per thread (up to the
                    batch), prefill + `blocks` - 1 decode blocks at k;
      one_thread -- the same with one thread on one sequence, 8 passes;
      toy        -- the whole 2-layer toy workload (batch 4, 64 new tokens);
      owt_k4_extrapolated -- the OWT-shaped model: 3 decode blocks at k = 4 at
                    the mean context length of its generate (C = 572), on one
                    copy per thread of a single sequence's context (built by an
                    untimed prefill); tokens/s = sequences * k * 3 / time, an
                    extrapolation of the whole generate from its mean step."""
    import ctypes
    import oracle as O
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))
    threads = max(1, min(threads, len(os.sched_getaffinity(0))))
    os.environ["OMP_NUM_THREADS"] = str(threads)
    O.lib()
    try:
        gomp = ctypes.CDLL("libgomp.so.1")
    except OSError:
        gomp = None

    def set_threads(n):
        if gomp is not None:
            gomp.omp_set_num_threads(n)

    set_threads(threads)
    nseq = min(prompt.shape[0], threads)
    m = O.Model(blob, "f32")
    L = blocks * k
    t0 = time.perf_counter()
    O.generate_batched(m, prompt[:nseq], L, k, seed)
    dt = time.perf_counter() - t0
    res = {"value": nseq * L / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
           "cpu": cpu_model_name(), "host_cpus": os.cpu_count(),
           "sample": (f"fp32 oracle loop nest, {nseq} sequences x {L} new tokens "
                      f"(prefill + {blocks - 1} decode blocks at k={k}), {dt:.1f} s"),
           "seconds": round(dt, 2)}
    # one thread, one sequence
    set_threads(1)
    L1 = 8 * k
    t0 = time.perf_counter()
    O.generate_batched(m, prompt[:1], L1, k, seed)
    dt1 = time.perf_counter() - t0
    res["one_thread"] = {"value": L1 / dt1, "unit": "tokens/s", "cores": 1,
                         "sample": f"1 sequence x {L1} new tokens (prefill + 7 blocks), {dt1:.1f} s"}
    set_threads(threads)
    del m
    # the toy workload end to end
    tw = S.WORKLOADS["toy"]
    tcfg = tw["cfg"]
    tm = O.Model(S.pack_blob(tcfg, S.make_weights(tcfg, seed=0)), "f32")
    tp = S.make_prompts(tw["prompts"], 1, tw["B"], tw["N"], tcfg.vocab)
    t0 = time.perf_counter()
    O.generate_batched(tm, tp, tw["L"], tw["k"], seed)
    dtt = time.perf_counter() - t0
    res["toy"] = {"value": tw["B"] * tw["L"] / dtt, "unit": "tokens/s", "cores": min(threads, tw["B"]),
                  "sample": f"whole toy workload: {tw['B']} x {tw['L']} tokens at k={tw['k']}, "
                            f"{dtt * 1e3:.0f} ms"}
    # OWT-shaped k = 4: three decode blocks at C = 572
    ow = S.WORKLOADS["owt"]
    ocfg = ow["cfg"]
    om = O.Model(owt_blob(), "f32")
    C0, kk = 572, 4
    op = S.make_prompts(ow["prompts"], 1, 1, C0 + kk, ocfg.vocab)[0]
    base = om.seq()
    t0 = time.perf_counter()
    base.step(list(op[:C0]), [], commit=True)
    t_pre = time.perf_counter() - t0
    seqs = [base.copy() for _ in range(threads)]
    pend = np.tile(op[C0:C0 + kk], (threads, 1))
    t0 = time.perf_counter()
    for st in range(3):
        u = S.noise_block(seed, threads, C0 + (st + 1) * kk, kk)
        pend = O.decode_batched(seqs, pend, kk, u)
    dto = time.perf_counter() - t0
    res["owt_k4_extrapolated"] = {
        "value": threads * kk * 3 / dto, "unit": "tokens/s", "cores": threads,
        "sample": (f"OWT-shaped fp32 oracle, {threads} sequences x 3 decode blocks at k={kk} "
                   f"from C={C0} (the generate's mean context), {dto:.1f} s; context built by "
                   f"an untimed {t_pre:.1f} s prefill; an extrapolation of the whole generate")}
    return res


def _short(name: str) -> str:
    import re
    n = name.replace("_ZN2kf12_GLOBAL__N_1", "").replace("kf::(anonymous namespace)::", "")
    m = re.match(r"\d+(\w+?)I(.*)", n)
    if m and "gemm_kernel" in m.group(1):
        t = re.findall(r"Li(\d+)E", m.group(2))
        ep = re.search(r"NS0_\d+(Ep\w+?)I|NS0_\d+(Ep\w+?)E", m.group(2))
        epn = (ep.group(1) or ep.group(2)) if ep else "?"
        kg = re.search(r"ELi([24])EEEvNS0_5GemmA", n)  # K groups per workgroup
        groups = f" {kg.group(1)}g" if kg else ""
        return f"gemm {'x'.join(t[:2])}{groups} {epn}" + (" bf16" if "DF16b" in n else " f32")
    if m and "gemm_skinny_kernel" in m.group(1):
        t = re.findall(r"Li(\d+)E", m.group(2))
        ep = re.search(r"NS0_\d+(Ep\w+?)I|NS0_\d+(Ep\w+?)E", m.group(2))
        epn = (ep.group(1) or ep.group(2)) if ep else "?"
        norm = "+LN " if "Lb1E" in m.group(2) else ""
        return f"gemm skinny {t[0] if t else '?'}w {norm}{epn}" + (" bf16" if "DF16b" in n else " f32")
    if m:
        return m.group(1) + (" bf16" if "DF16b" in n else "")
    return n.split("(")[0]


KERNEL_SOURCES = os.path.join(ROOT, "paper_2606_10820_amd", "csrc")
# the training-mask attention source holds no kernel of the decode step
DECODE_EXCLUDED = ("kf_blockattn.hip",)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_lm1b_b64_k4.json")


def kernel_source_hash() -> str:
    """sha256 over the sources of the decode step's kernels and their launch
    code, with comments and whitespace removed: counter figures taken from
    different code are not reported (an edit of a comment does not change the
    kernels)."""
    import hashlib
    import re
    h = hashlib.sha256()
    for fn in sorted(os.listdir(KERNEL_SOURCES)):
        if fn in DECODE_EXCLUDED:
            continue
        with open(os.path.join(KERNEL_SOURCES, fn), encoding="utf-8") as f:
            src = f.read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        src = " ".join(src.split())
        h.update(fn.encode() + b"\0" + src.encode())
    return h.hexdigest()


def kernel_class(name: str, state: dict):
    """Kernel class of one dispatch, from its name and the launch order of a
    step: out-proj and MLP-down share one GEMM instantiation and alternate;
    a split-K part belongs to the reduction that follows it."""
    if "embed_real_kernel" in name:
        return "embed"
    if "noise_sinusoid" in name or "EpNoiseOut" in name:
        return "noise"
    if "attention_mfma_kernel" in name or "attention_combine_kernel" in name:
        return "attn"
    if "EpQKV" in name:
        return "qkv"
    if "EpHead" in name:
        return "head"
    if any(k in name for k in ("argmax_select_kernel", "icdf_select_kernel", "commit_kernel")):
        return "select"
    if "EpPartial" in name:
        return "pending"
    if "EpResidual" in name:
        if "splitk_reduce" in name or "gemm_kernel" in name or "gemm_skinny_kernel" in name:
            role = "oproj" if state.get("residual", 0) % 2 == 0 else "mlp_down"
            state["residual"] = state.get("residual", 0) + 1
            return role
    if "EpBias" in name:
        return "mlp_up" if "Lb1E" in name else "noise"
    return None


def class_times(path: str) -> None:
    """Kernel time per class launch from a kernel trace, in dispatch order
    (kernel_class): out-projection and MLP-down share one GEMM instantiation
    and alternate; a split-K part is counted with the reduction that follows
    it (a part with no reduction after it is the noise encoder's fp32 output
    GEMM); an attention combine with the attention before it."""
    import csv
    rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Dispatch_Id"]))
    state, pending, cls = {}, 0.0, {}
    for r in rows:
        name = r["Kernel_Name"]
        us = (float(r["End_Timestamp"]) - float(r["Start_Timestamp"])) / 1e3
        c = kernel_class(name, state)
        if pending and "splitk_reduce" not in name:  # a part with no reduction
            e = cls.setdefault("noise", [0, 0.0])
            e[0] += 1
            e[1] += pending
            pending = 0.0
        if c == "pending":
            pending = us
            continue
        if c is None:
            continue
        e = cls.setdefault(c, [0, 0.0])
        helper = "attention_combine" in name or "splitk_reduce" in name
        if not helper or pending:
            e[0] += 1
        e[1] += us + pending
        pending = 0.0
    if not cls:
        return
    tot = sum(v[1] for v in cls.values())
    print(f"### kernel time per class launch ({os.path.basename(path)}; split-K parts and "
          "reductions, attention and its combine counted together)\n")
    print("| class | launches | avg us per launch | share |\n|---|---|---|---|")
    for c, (n, t) in sorted(cls.items(), key=lambda kv: -kv[1][1]):
        print(f"| {c} | {n} | {t / max(n, 1):.2f} | {t / tot * 100:.1f}% |")
    print()


def summarize(root: str, write_json: str = None) -> None:
    """Markdown summary of rocprofv3 --stats / --pmc CSV output (no GPU needed),
    with HBM traffic per kernel class; write_json stores the per-launch class
    traffic for bench.py."""
    import csv
    import glob
    stats = glob.glob(os.path.join(root, "**", "*_kernel_stats.csv"), recursive=True)
    for path in stats:
        rows = list(csv.DictReader(open(path)))
        tot = sum(float(r["TotalDurationNs"]) for r in rows)
        print(f"### kernel time ({os.path.relpath(path, root)})\n")
        print("| kernel | calls | avg us | min us | share |\n|---|---|---|---|---|")
        for r in rows[:16]:
            print(f"| {_short(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                  f"{float(r['MinNs']) / 1e3:.2f} | {float(r['TotalDurationNs']) / tot * 100:.1f}% |")
        print()
    for path in glob.glob(os.path.join(root, "**", "*_kernel_trace.csv"), recursive=True):
        class_times(path)
    pmc, seq = {}, {}
    for path in glob.glob(os.path.join(root, "**", "*_counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(path)):
            key = (_short(r["Kernel_Name"]), int(r["Grid_Size"]))
            pmc.setdefault(r["Counter_Name"], {}).setdefault(key, []).append(float(r["Counter_Value"]))
            seq.setdefault(r["Counter_Name"], []).append(
                (int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"])))
    if not pmc:
        return
    other = sorted(c for c in pmc if c not in ("FETCH_SIZE", "WRITE_SIZE"))
    if other:
        # mean per dispatch of every other counter, by kernel, and the MFMA busy
        # fraction: SQ_VALU_MFMA_BUSY_CYCLES is summed over the 1024 SIMDs, so
        # busy / 1024 / (kernel cycles) with the kernel's mean duration from a
        # kernel trace in the same directory at the 2.4 GHz peak engine clock
        durs = {}
        for path in glob.glob(os.path.join(root, "**", "*_kernel_trace.csv"), recursive=True):
            for r in csv.DictReader(open(path)):
                if "Grid_Size" in r:
                    grid = int(r["Grid_Size"])
                else:
                    grid = int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])
                key = (_short(r["Kernel_Name"]), grid)
                durs.setdefault(key, []).append(float(r["End_Timestamp"]) - float(r["Start_Timestamp"]))
        keys = sorted({k for c in other for k in pmc[c]},
                      key=lambda k: -np.mean(pmc[other[0]].get(k, [0])))
        print("| kernel | grid | dispatches | " + " | ".join(other) +
              (" | mean us | MFMA busy |" if "SQ_VALU_MFMA_BUSY_CYCLES" in other else " |"))
        print("|---|---|---|" + "---|" * len(other) +
              ("---|---|" if "SQ_VALU_MFMA_BUSY_CYCLES" in other else ""))
        for k in keys[:20]:
            n = max(len(pmc[c].get(k, [])) for c in other)
            vals = [np.mean(pmc[c][k]) if k in pmc[c] else float("nan") for c in other]
            line = f"| {k[0]} | {k[1]} | {n} | " + " | ".join(f"{v:.4g}" for v in vals) + " |"
            if "SQ_VALU_MFMA_BUSY_CYCLES" in other:
                mb = np.mean(pmc["SQ_VALU_MFMA_BUSY_CYCLES"].get(k, [float("nan")]))
                us = np.mean(durs[k]) / 1e3 if k in durs else float("nan")
                line += f" {us:.2f} | {mb / 1024 / (us * 1e-6 * 2.4e9):.3f} |"
            print(line)
        print()
    if "FETCH_SIZE" not in pmc and "WRITE_SIZE" not in pmc:
        return
    # calibration: fp32 -> bf16 weight conversion of the token table reads 4n, writes 2n bytes
    conv = [k for k in pmc.get("FETCH_SIZE", {}) if k[0].startswith("convert_kernel")]
    cal = max(conv, key=lambda k: k[1]) if conv else None
    f_scale = w_scale = None
    if cal:
        n = cal[1]
        f_scale = 4 * n / 1024 / np.mean(pmc["FETCH_SIZE"][cal])
        if "WRITE_SIZE" in pmc and cal in pmc["WRITE_SIZE"]:
            w_scale = 2 * n / 1024 / np.mean(pmc["WRITE_SIZE"][cal])
        ws = f"{w_scale:.4f}" if w_scale else "n/a"
        print(f"calibration on {cal[0]} over {n} elements: FETCH_SIZE x {f_scale:.4f}, "
              f"WRITE_SIZE x {ws} (true bytes / counter bytes)\n")
    print("| kernel | grid | dispatches | FETCH KiB | WRITE KiB | scaled MB read | scaled MB written |")
    print("|---|---|---|---|---|---|---|")
    keys = sorted(set(pmc.get("FETCH_SIZE", {})) | set(pmc.get("WRITE_SIZE", {})),
                  key=lambda k: -np.mean(pmc.get("FETCH_SIZE", {}).get(k, [0])))
    for k in keys[:16]:
        fv = pmc.get("FETCH_SIZE", {}).get(k)
        wv = pmc.get("WRITE_SIZE", {}).get(k)
        fm = np.mean(fv) if fv else float("nan")
        wm = np.mean(wv) if wv else float("nan")
        print(f"| {k[0]} | {k[1]} | {len(fv or wv)} | {fm:.1f} | {wm:.1f} | "
              f"{fm * 1024 * (f_scale or 1) / 1e6:.2f} | {wm * 1024 * (w_scale or 1) / 1e6:.2f} |")
    # per kernel class: scaled bytes per class launch (a class launch may run a
    # helper kernel too: split-K reduction, attention combine)
    cls = {}
    for counter, scale in (("FETCH_SIZE", f_scale), ("WRITE_SIZE", w_scale)):
        state, pending = {}, 0.0
        for _, name, v in sorted(seq.get(counter, [])):
            c = kernel_class(name, state)
            b = v * 1024 * (scale or 1.0)
            if c is None:
                continue
            if c == "pending":
                pending += b
                continue
            e = cls.setdefault(c, {"launches": {}, "bytes": {}})
            split = pending > 0.0  # the reduction of a split-K launch
            e["bytes"][counter] = e["bytes"].get(counter, 0.0) + b + pending
            pending = 0.0
            helper = "attention_combine" in name or "splitk_reduce" in name
            if not helper or split:
                e["launches"][counter] = e["launches"].get(counter, 0) + 1
    print("\n| class | launches | MB read / launch | MB written / launch |\n|---|---|---|---|")
    out = {}
    for c, e in sorted(cls.items()):
        n = e["launches"].get("FETCH_SIZE") or e["launches"].get("WRITE_SIZE") or 1
        rd = e["bytes"].get("FETCH_SIZE", float("nan")) / n
        wr = e["bytes"].get("WRITE_SIZE", float("nan")) / max(e["launches"].get("WRITE_SIZE", n), 1)
        print(f"| {c} | {n} | {rd / 1e6:.2f} | {wr / 1e6:.2f} |")
        out[c] = {"launches": n, "read_bytes_per_launch": rd, "write_bytes_per_launch": wr}
    if write_json:
        with open(write_json, "w") as f:
            json.dump({"workload": "lm1b B=64 k=4 (bench.py defaults)",
                       "source_sha256": kernel_source_hash(),
                       "calibration": {"kernel": cal[0] if cal else None,
                                       "fetch_scale": f_scale, "write_scale": w_scale},
                       "classes": out}, f, indent=1)
            f.write("\n")


def load_traffic(dom: str, workload: str, B: int, k: int):
    """Per-launch HBM bytes of class dom from the committed counter summary,
    or None when the summary is for another workload or an older build."""
    if workload != "lm1b" or B != S.WORKLOADS["lm1b"]["B"] or k != S.WORKLOADS["lm1b"]["k"]:
        return None
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_sha256") != kernel_source_hash() or dom not in t.get("classes", {}):
        return None
    c = t["classes"][dom]
    return c["read_bytes_per_launch"] + c["write_bytes_per_launch"]


def step_roof_ms(costs, dtype) -> float:
    by = sum(v[0] for v in costs.values())
    fl = sum(v[1] for v in costs.values())
    return max(by / (PEAK_HBM_GBS * 1e9), fl / (PEAK_MFMA_TFLOPS[dtype] * 1e12)) * 1e3


def time_calls(fn, reps):
    import torch
    fn()  # warm-up (also captures the decode-step graph)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        fn()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / reps


_OWT_BLOB = {}


def owt_blob():
    """The OWT-shaped model's seeded weights (kept for the CPU baseline)."""
    if "blob" not in _OWT_BLOB:
        cfg = S.WORKLOADS["owt"]["cfg"]
        log("[bench] generating OWT-shaped weights")
        _OWT_BLOB["blob"] = S.pack_blob(cfg, S.make_weights(cfg, seed=0))
    return _OWT_BLOB["blob"]


def owt_sweep(batches, stream):
    """OpenWebText-shaped model (12 layers, d=768, vocab 50257, context 1024,
    bf16), prompt 128 Zipf(1.1) tokens, generation to the full context (896 new
    tokens): K-Forcing at k = 4, 2 and 1 and the k = 1 AR baseline at every
    batch size.  Each figure is whole-generate throughput with its step-level
    roofline fraction t_roof / t_meas (t_roof from step_costs: max of bytes /
    HBM peak and flops / bf16 MFMA peak, summed over the generate's passes)."""
    import torch
    from paper_2606_10820_amd import binding as Bd
    w = S.WORKLOADS["owt"]
    cfg = w["cfg"]
    N, L, seed = w["N"], w["L"], 2
    blob = owt_blob()
    dev = torch.device("cuda:0")

    def ctx(B):
        kc = Bd.make_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_mlp, cfg.vocab,
                            cfg.n_ctx, cfg.dtype, B, 4, N, 0)
        kf = Bd.KForcing(kc, device="cuda:0", stream=stream)
        kf.load_weights(blob)
        return kf

    def run(kf, B, k, reps):
        prompt = torch.as_tensor(S.make_prompts(w["prompts"], 1, B, N, cfg.vocab), device=dev)
        out = torch.empty((B, L), dtype=torch.int32, device=dev)
        if k == 0:
            dt = time_calls(lambda: kf.generate_ar(prompt, L, seed, out=out), reps)
            roof = step_roof_ms(generate_ar_costs(cfg, B, N, L), cfg.dtype)
        else:
            dt = time_calls(lambda: kf.generate(prompt, L, k, seed, out=out), reps)
            roof = step_roof_ms(generate_costs(cfg, B, N, L, k), cfg.dtype)
        return {"tokens_s": round(B * L / dt, 1), "ms_per_generate": round(dt * 1e3, 3),
                "roofline_ms": round(roof, 3), "roofline_frac": round(roof / (dt * 1e3), 4)}

    rows = []
    for B in batches:
        kf = ctx(B)
        r = {"batch": B}
        r["k4"] = run(kf, B, 4, 2)
        r["k2"] = run(kf, B, 2, 1)
        r["k1"] = run(kf, B, 1, 1)
        r["ar_k1"] = run(kf, B, 0, 1)
        for kk in ("k4", "k2", "k1"):
            r[f"speedup_{kk}_vs_ar"] = round(r[kk]["tokens_s"] / r["ar_k1"]["tokens_s"], 3)
        rows.append(r)
        log(f"[bench] sweep B={B}: k=4 {r['k4']['tokens_s']:,.0f} tok/s "
            f"({r['k4']['roofline_frac']:.1%} of step roofline), k=2 {r['k2']['tokens_s']:,.0f}, "
            f"k=1 {r['k1']['tokens_s']:,.0f}, AR {r['ar_k1']['tokens_s']:,.0f} tok/s, "
            f"k=4/AR x{r['speedup_k4_vs_ar']:.2f}")
        del kf
        torch.cuda.empty_cache()
    return {"workload": (f"OWT-shaped: {cfg.n_layer} layers, d={cfg.d_model}, vocab {cfg.vocab}, "
                         f"context {cfg.n_ctx}, prompt {N} Zipf(1.1), {L} new tokens, bf16"),
            "by_batch": rows}


def teacher_costs(cfg: S.ModelConfig, B: int, N: int) -> dict:
    """Per kernel class (bytes, flops) of one kf_teacher_targets call: an AR
    prefill of N tokens per sequence whose head runs over every row."""
    c = operand_costs(cfg, B, N, 0, 0)
    for n, (_, fl) in step_costs(cfg, B, N, 0, 0).items():
        c[n][1] = fl
    es = 2 if cfg.dtype == S.DTYPE_BF16 else 4
    d, V, M = cfg.d_model, cfg.vocab, B * N
    nt = (V + 255) // 256 * 2
    c["head"] = [V * d * es + M * d * es + M * nt * 36, 2.0 * M * V * d]
    c["select"] = [M * (nt * 36 + 16 * d * es + d * es + 8), 2.0 * M * 16 * d]
    return c


def teacher_bench(reps: int = 3):
    """Stage-1 distillation targets (kf_teacher_targets) at one GPU's share of
    the paper's training batch (64 sequences) for the LM1B-shaped (N = 128)
    and OWT-shaped (N = 1024) models: targets per second and the fraction of
    the call's algorithmic roofline (max of bytes / HBM peak and flops / bf16
    MFMA peak, counted by teacher_costs)."""
    import torch
    from paper_2606_10820_amd import binding as Bd
    dev = torch.device("cuda:0")
    out = []
    for name in ("lm1b", "owt"):
        w = S.WORKLOADS[name]
        cfg = w["cfg"]
        B, N = 64, cfg.n_ctx
        log(f"[bench] teacher targets {name}: B={B}, N={N}")
        blob = S.pack_blob(cfg, S.make_weights(cfg, seed=0))
        kc = Bd.make_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_mlp, cfg.vocab, cfg.n_ctx,
                            cfg.dtype, B, 1, N, Bd.KF_FLAG_TEACHER)
        kf = Bd.KForcing(kc, device="cuda:0")
        kf.load_weights(blob)
        tokens = torch.as_tensor(S.make_prompts(w["prompts"], 3, B, N, cfg.vocab), device=dev)
        tau = torch.as_tensor(np.random.default_rng(5).uniform(0.5, 1.5, B).astype(np.float32),
                              device=dev)
        u = torch.as_tensor(S.noise_block(3, B, 0, N), device=dev)
        tg = torch.empty((B, N), dtype=torch.int32, device=dev)
        L = kf.L
        call = lambda: L.kf_teacher_targets(kf.h, B, N, kf._p(tokens), kf._p(tau), kf._p(u),
                                            kf._p(tg))
        assert call() == 0
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            call()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) / reps * 1e3
        kf.set_timing(Bd.KF_TIMING_ALL)
        call()
        per = {n: round(kf.kernel_time(ci)[0], 4) for ci, n in enumerate(CLASSES)}
        kf.set_timing(0)
        costs = teacher_costs(cfg, B, N)
        by = sum(v[0] for v in costs.values())
        fl = sum(v[1] for v in costs.values())
        roof = max(by / (PEAK_HBM_GBS * 1e9), fl / (PEAK_MFMA_TFLOPS[cfg.dtype] * 1e12)) * 1e3
        hb, hf = costs["head"]
        out.append({"workload": f"{name}-shaped teacher, B={B}, N={N} (every position sampled)",
                    "ms": round(ms, 3), "targets_per_s": round(B * N / (ms * 1e-3), 1),
                    "algorithmic_flops": fl, "algorithmic_bytes": by,
                    "roofline_ms": round(roof, 4), "roofline_frac": round(roof / ms, 4),
                    "head_tflops": round(hf / (per["head"] * 1e-3) / 1e12, 1),
                    "kernel_ms": per})
        log(f"[bench] teacher {name}: {ms:.3f} ms, {B * N / (ms * 1e-3):,.0f} targets/s, "
            f"{roof / ms:.1%} of its roofline; head {out[-1]['head_tflops']} TFLOP/s")
        del kf
        torch.cuda.empty_cache()
    return {"entry": "kf_teacher_targets", "cases": out}


def rollout_costs(cfg: S.ModelConfig, B: int, N: int, k: int):
    """(bytes, flops) of one kf_selfforcing_targets call: per round, the body
    GEMMs over its rows, the block-sparse attention over its visible pairs,
    the noise MLP over N*k rows and the head over N*k rows (the step formulas
    of step_costs applied to the rounds' row counts)."""
    es = 2 if cfg.dtype == S.DTYPE_BF16 else 4
    d, f, V, L = cfg.d_model, cfg.d_mlp, cfg.vocab, cfg.n_layer
    nk = N * k
    ctx = N * (N + 1) // 2
    noise = k * N * (N + 1) // 2 + nk * (k + 1) // 2
    rounds = ((N + nk, ctx + noise, N + nk), (2 * nk, 2 * noise + nk * k, N + 2 * nk))
    by = fl = 0.0
    for rows, pairs, keys in rounds:
        M = B * rows
        fl += L * (2.0 * M * (4 * d * d + 2 * d * f) + 4.0 * d * B * pairs)
        by += L * ((4 * d * d + 2 * d * f) * es + M * (6 * d * es + 2 * f * es + 4 * d * 4)
                   + B * keys * 2 * d * es)
        fl += 2.0 * B * nk * (8 * d * d) + 2.0 * B * nk * V * d
        by += 8 * d * d * es + V * d * es + B * nk * (6 * d * es + 8)
    return by, fl


def rollout_bench(reps: int = 2):
    """Stage-2 self-forcing targets (kf_selfforcing_targets), teacher window
    k = 2 (the PFLM(2) -> PFLM(4) stage), 64 sequences of the LM1B-shaped
    (N = 128 - 2k) and OWT-shaped (N = 1024 - 2k) models: targets per second
    (2k per context position) and the call's roofline fraction."""
    import torch
    from paper_2606_10820_amd import binding as Bd
    dev = torch.device("cuda:0")
    out = []
    k = 2
    for name in ("lm1b", "owt"):
        w = S.WORKLOADS[name]
        cfg = w["cfg"]
        B, N = 64, cfg.n_ctx - 2 * k
        log(f"[bench] self-forcing targets {name}: B={B}, N={N}, k={k}")
        blob = S.pack_blob(cfg, S.make_weights(cfg, seed=0))
        kc = Bd.make_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_mlp, cfg.vocab, cfg.n_ctx,
                            cfg.dtype, B, k, N, Bd.KF_FLAG_ROLLOUT)
        kf = Bd.KForcing(kc, device="cuda:0")
        kf.load_weights(blob)
        tokens = torch.as_tensor(S.make_prompts(w["prompts"], 3, B, N, cfg.vocab), device=dev)
        g = torch.Generator(device=dev)
        g.manual_seed(7)
        z1 = torch.rand((B, N, k), device=dev, generator=g)
        z2 = torch.rand((B, N, k), device=dev, generator=g)
        x1 = torch.empty((B, N, k), dtype=torch.int32, device=dev)
        x2 = torch.empty_like(x1)
        L = kf.L
        call = lambda: L.kf_selfforcing_targets(kf.h, B, N, k, kf._p(tokens), kf._p(z1),
                                                kf._p(z2), kf._p(x1), kf._p(x2))
        assert call() == 0
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            call()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) / reps * 1e3
        kf.set_timing(Bd.KF_TIMING_ALL)
        call()
        per = {n: round(kf.kernel_time(ci)[0], 4) for ci, n in enumerate(CLASSES)}
        kf.set_timing(0)
        by, fl = rollout_costs(cfg, B, N, k)
        roof = max(by / (PEAK_HBM_GBS * 1e9), fl / (PEAK_MFMA_TFLOPS[cfg.dtype] * 1e12)) * 1e3
        out.append({"workload": f"{name}-shaped teacher, B={B}, N={N}, k={k} (2k targets per position)",
                    "ms": round(ms, 3), "targets_per_s": round(B * N * 2 * k / (ms * 1e-3), 1),
                    "algorithmic_flops": fl, "algorithmic_bytes": by,
                    "tflops": round(fl / (ms * 1e-3) / 1e12, 1),
                    "roofline_ms": round(roof, 4), "roofline_frac": round(roof / ms, 4),
                    "kernel_ms": per})
        log(f"[bench] self-forcing {name}: {ms:.2f} ms, {B * N * 2 * k / (ms * 1e-3):,.0f} targets/s, "
            f"{fl / (ms * 1e-3) / 1e12:.0f} TFLOP/s, {roof / ms:.1%} of its roofline")
        del kf
        torch.cuda.empty_cache()
    return {"entry": "kf_selfforcing_targets", "cases": out}


def serving_bench(stream, reps: int = 2):
    """Continuous batching (kf_serve_*) on the LM1B-shaped model: 128 sequences
    (prompt 16 Zipf tokens, 112 new tokens each, k = 4) through 64 slots.
    Sequences arrive in waves of 16 every 7 steps; a finished sequence is
    released and the next waiting one is admitted into its slot at the
    following step.  Tokens per second over the whole run, host calls
    included, beside the lock-step kf_generate of the same sequences."""
    import torch
    from paper_2606_10820_amd import binding as Bd
    w = S.WORKLOADS["lm1b"]
    cfg = w["cfg"]
    slots_n, n_seq, N, L, k = 64, 128, w["N"], w["L"] - w["L"] % 4, 4
    dev = torch.device("cuda:0")
    blob = S.pack_blob(cfg, S.make_weights(cfg, seed=0))
    kc = Bd.make_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_mlp, cfg.vocab, cfg.n_ctx,
                        cfg.dtype, slots_n, k, N, Bd.KF_FLAG_SERVING)
    kf = Bd.KForcing(kc, device="cuda:0", stream=stream)
    kf.load_weights(blob)
    prompts = torch.as_tensor(S.make_prompts(w["prompts"], 5, n_seq, N, cfg.vocab), device=dev)
    g = torch.Generator(device=dev)
    g.manual_seed(11)
    noise = torch.rand((4096, slots_n, k), device=dev, generator=g)
    out = torch.empty((slots_n, k), dtype=torch.int32, device=dev)
    L_ = kf.L
    passes = L // k

    def run():
        nxt, done, tick = 0, 0, 0
        age = {}                      # slot -> passes done
        free = list(range(slots_n))
        calls = rows = 0
        while done < n_seq:
            # arrivals: waves of 16 every 7 steps; a freed slot takes the next waiting sequence
            arrived = min(n_seq, 16 * (tick // 7 + 1))
            take = min(len(free), arrived - nxt)
            new = []
            if take > 0:
                new = [free.pop() for _ in range(take)]
                arr = np.asarray(new, np.int32)
                rc = L_.kf_serve_admit(kf.h, take, arr.ctypes.data_as(ctypes.c_void_p), N,
                                       kf._p(prompts[nxt:nxt + take]), k,
                                       kf._p(noise[tick % 4096]), kf._p(out))
                assert rc == 0, kf.L.kf_last_error(kf.h)
                nxt += take
                calls += 1
                rows += take
                for q in new:
                    age[q] = 1
            live = [q for q in age if q not in new]  # the admitted made their first pass
            if live:
                arr = np.asarray(live, np.int32)
                rc = L_.kf_serve_step(kf.h, len(live), arr.ctypes.data_as(ctypes.c_void_p), k,
                                      kf._p(noise[(tick + 1) % 4096]), kf._p(out))
                assert rc == 0, kf.L.kf_last_error(kf.h)
                calls += 1
                rows += len(live)
                for q in live:
                    age[q] += 1
            fin = [q for q in age if age[q] >= passes]
            if fin:
                arr = np.asarray(fin, np.int32)
                assert L_.kf_serve_release(kf.h, len(fin), arr.ctypes.data_as(ctypes.c_void_p)) == 0
                for q in fin:
                    del age[q]
                    free.append(q)
                done += len(fin)
            tick += 1
        return tick, calls, rows

    run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        ticks, calls, rows = run()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) / reps * 1e3
    toks = n_seq * L
    res = {"workload": (f"lm1b-shaped, {n_seq} sequences (prompt {N}, {L} new tokens, k={k}) "
                        f"through {slots_n} slots, arrivals of 16 every 7 steps"),
           "ms": round(ms, 3), "tokens_per_s": round(toks / (ms * 1e-3), 1),
           "steps": ticks, "calls": calls, "sequence_passes": rows}
    log(f"[bench] serving: {ms:.2f} ms for {toks} tokens -> {toks / (ms * 1e-3):,.0f} tokens/s "
        f"({ticks} steps, {calls} calls)")
    del kf
    torch.cuda.empty_cache()
    return res


def large_bench(stream, reps: int = 2):
    """The 24-layer backbone (d 1024, 16 heads, MLP 4096, vocab 50257, context
    1024, bf16): 256 sequences, prompt 256 Zipf(1.1) tokens, 768 new tokens at
    k = 4 (192 passes).  Tokens/s, the step roofline fraction, and the body
    GEMMs' MFMA rate (algorithmic flops of each class over its HIP-event time;
    at M = 2048 rows per decode pass these GEMMs are MFMA-bound)."""
    import torch
    from paper_2606_10820_amd import binding as Bd
    w = S.WORKLOADS["large"]
    cfg = w["cfg"]
    B, N, k = w["B"], w["N"], w["k"]
    L = w["L"] - w["L"] % k
    dev = torch.device("cuda:0")
    log(f"[bench] large backbone: generating weights ({S.n_params(cfg) / 1e6:.1f} M params)")
    blob = S.pack_blob(cfg, S.make_weights(cfg, seed=0))
    kc = Bd.make_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_mlp, cfg.vocab, cfg.n_ctx,
                        cfg.dtype, B, k, N, 0)
    kf = Bd.KForcing(kc, device="cuda:0", stream=stream)
    kf.load_weights(blob)
    prompt = torch.as_tensor(S.make_prompts(w["prompts"], 1, B, N, cfg.vocab), device=dev)
    out = torch.empty((B, L), dtype=torch.int32, device=dev)
    run = lambda: kf.generate(prompt, L, k, 2, out=out)
    run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        run()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) / reps * 1e3
    kf.set_timing(Bd.KF_TIMING_ALL)
    run()
    per = {n: kf.kernel_time(ci)[0] for ci, n in enumerate(CLASSES)}
    kf.set_timing(0)
    costs = generate_costs(cfg, B, N, L, k)
    roof = step_roof_ms(costs, cfg.dtype)
    gemm = {n: round(costs[n][1] / (per[n] * 1e-3) / 1e12, 1)
            for n in ("qkv", "oproj", "mlp_up", "mlp_down", "head") if per[n] > 0}
    fl = sum(costs[n][1] for n in ("qkv", "oproj", "mlp_up", "mlp_down"))
    tms = sum(per[n] for n in ("qkv", "oproj", "mlp_up", "mlp_down"))
    res = {"workload": (f"large backbone: {cfg.n_layer} layers, d={cfg.d_model}, {cfg.n_head} heads, "
                        f"MLP {cfg.d_mlp}, vocab {cfg.vocab}, context {cfg.n_ctx}; batch {B}, "
                        f"prompt {N}, k={k}, {L} new tokens"),
           "ms_per_generate": round(ms, 2), "tokens_per_s": round(B * L / (ms * 1e-3), 1),
           "roofline_ms": round(roof, 3), "roofline_frac": round(roof / ms, 4),
           "gemm_tflops_by_class": gemm,
           "body_gemm_tflops": round(fl / (tms * 1e-3) / 1e12, 1),
           "body_gemm_mfma_frac": round(fl / (tms * 1e-3) / 1e12 / PEAK_MFMA_TFLOPS[cfg.dtype], 4),
           "kernel_ms_per_generate": {n: round(v, 3) for n, v in per.items()}}
    log(f"[bench] large backbone: {ms:.1f} ms per generate, {B * L / (ms * 1e-3):,.0f} tokens/s, "
        f"{roof / ms:.1%} of the step roofline; body GEMMs {res['body_gemm_tflops']} TFLOP/s")
    del kf
    torch.cuda.empty_cache()
    return res


def training_attention_bench(reps: int = 10):
    """Block-sparse attention of the training masks (SingleForward M_S and
    DoubleForward M_D, Appendix C.2) at one GPU's share of the paper's
    training batch (global batch 512 over 8 GPUs: 64 sequences; 12 heads,
    d_head 64, k = 4) for the OWT (N = 1024) and LM1B (N = 128) sequence
    lengths.  Inputs are seeded N(0, 1) bf16 tensors.  Work counted: 4 d_head
    flops per visible (query, key) pair, against the bf16 MFMA peak; bytes:
    Q, K, V read and O written once, against the HBM peak.  The roofline time
    is the larger of the two."""
    import torch
    from paper_2606_10820_amd import binding as Bd
    dev = torch.device("cuda:0")
    peak = PEAK_MFMA_TFLOPS[S.DTYPE_BF16]
    cases = []
    for name, (B, H, N, k, dh) in (("OWT", (64, 12, 1024, 4, 64)), ("LM1B", (64, 12, 128, 4, 64))):
        for mask, mname in ((Bd.KF_MASK_SINGLE, "single"), (Bd.KF_MASK_DOUBLE, "double")):
            rows, keys = Bd.training_attention_shapes(mask, N, k)
            g = torch.Generator(device=dev)
            g.manual_seed(1)
            q = torch.randn((B, H, rows, dh), device=dev, generator=g).to(torch.bfloat16)
            kk = torch.randn((B, H, keys, dh), device=dev, generator=g).to(torch.bfloat16)
            v = torch.randn((B, H, keys, dh), device=dev, generator=g).to(torch.bfloat16)
            out = torch.empty_like(q)
            for _ in range(3):
                Bd.training_attention(mask, q, kk, v, N, k, dh ** -0.5, out=out)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                Bd.training_attention(mask, q, kk, v, N, k, dh ** -0.5, out=out)
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / reps
            ent = Bd.training_attention_entries(mask, N, k)
            fl = 4.0 * ent * dh * B * H
            tf = fl / (ms * 1e-3) / 1e12
            by = 2.0 * B * H * dh * (2 * rows + 2 * keys)
            t_mem, t_fl = by / (PEAK_HBM_GBS * 1e9) * 1e3, fl / (peak * 1e12) * 1e3
            roof = max(t_mem, t_fl)
            cases.append({"workload": f"{name} training share: B={B}, H={H}, N={N}, k={k}, d_head={dh}",
                          "mask": mname, "ms": round(ms, 4), "tflops": round(tf, 1),
                          "frac": round(tf / peak, 4), "hbm_bytes": by,
                          "gbs": round(by / (ms * 1e-3) / 1e9, 1),
                          "roofline_ms": round(roof, 4), "bound": "hbm" if t_mem >= t_fl else "mfma",
                          "roofline_frac": round(roof / ms, 4), "visible_pairs_per_head": ent,
                          "dense_pairs_per_head": rows * keys})
            log(f"[bench] training attention {name} {mname}: {ms:.3f} ms, {tf:.1f} TFLOP/s "
                f"({tf / peak:.1%} of bf16 MFMA peak), {by / (ms * 1e-3) / 1e9:.0f} GB/s; "
                f"{roof / ms:.1%} of its roofline ({'HBM' if t_mem >= t_fl else 'MFMA'}-bound)")
            del q, kk, v, out
    torch.cuda.empty_cache()
    return {"kernel": "kf_training_attention", "peak_tflops": peak, "peak_gbs": PEAK_HBM_GBS,
            "work": "4 * d_head flops per visible (query, key) pair; Q, K, V, O once each",
            "cases": cases}


def main():
    a = parse()
    if a.summarize:
        summarize(a.summarize, a.write_traffic)
        return
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {a.gpus}); the decode path "
              "shards by sequence and is measured at one GPU's share.", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2606_10820_amd import binding as Bd

    if a.train_attn_only:
        print(json.dumps(training_attention_bench(max(a.steps, 1))), flush=True)
        return
    if a.teacher_only:
        print(json.dumps(teacher_bench(max(a.steps, 1))), flush=True)
        return
    if a.rollout_only:
        print(json.dumps(rollout_bench(max(a.steps, 1))), flush=True)
        return
    if a.large_only:
        st = torch.cuda.Stream(device=torch.device("cuda:0"))
        torch.cuda.set_stream(st)
        print(json.dumps(large_bench(st, max(a.steps, 1))), flush=True)
        return
    if a.serving_only:
        st = torch.cuda.Stream(device=torch.device("cuda:0"))
        torch.cuda.set_stream(st)
        print(json.dumps(serving_bench(st, max(a.steps, 1))), flush=True)
        return

    w = S.WORKLOADS[a.workload]
    cfg: S.ModelConfig = w["cfg"]
    B = a.batch or w["B"]
    k = a.k or w["k"]
    N, L = w["N"], w["L"] - (w["L"] % k)
    seed = 2
    dev = torch.device("cuda:0")

    log(f"[bench] workload {a.workload}: generating weights ({S.n_params(cfg) / 1e6:.1f} M params)")
    blob = S.pack_blob(cfg, S.make_weights(cfg, seed=0))
    prompt = S.make_prompts(w["prompts"], 1, B, N, cfg.vocab)
    kc = Bd.make_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_mlp, cfg.vocab, cfg.n_ctx,
                        cfg.dtype, B, max(k, 1), N, 0)
    stream = torch.cuda.Stream(device=dev)  # a real stream: decode blocks replay as a HIP graph
    torch.cuda.set_stream(stream)
    kf = Bd.KForcing(kc, device="cuda:0", stream=stream)
    kf.load_weights(blob)
    dprompt = torch.as_tensor(prompt, device=dev)
    out = torch.empty((B, L), dtype=torch.int32, device=dev)

    def run_kf():
        kf.generate(dprompt, L, k, seed, out=out)

    def run_ar():
        kf.generate_ar(dprompt, L, seed, out=out)

    def timed(fn, steps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            fn()
        torch.cuda.synchronize()
        return time.perf_counter() - t0

    log(f"[bench] warmup {a.warmup} x kf_generate (B={B}, N={N}, L={L}, k={k})")
    for _ in range(a.warmup):
        run_kf()
    dt = timed(run_kf, a.steps)
    tokens = B * L * a.steps
    value = tokens / dt
    ms_step = dt / a.steps * 1e3
    log(f"[bench] k={k}: {value:,.0f} tokens/s, {ms_step:.3f} ms per generate")

    # per-class kernel time over one generate (all classes bracketed)
    kf.set_timing(Bd.KF_TIMING_ALL)
    run_kf()
    per = {}
    for ci, name in enumerate(CLASSES):
        ms, n = kf.kernel_time(ci)
        per[name] = (ms, n)
    kf.set_timing(0)
    costs = generate_costs(cfg, B, N, L, k)
    opcosts = generate_costs(cfg, B, N, L, k, per_step=operand_costs)
    dom = max(CLASSES, key=lambda n: per[n][0])
    # the timed region again, with only the dominant class bracketed by events
    di = CLASSES.index(dom)
    kf.set_timing(1 << di)
    timed(run_kf, a.steps)
    dom_ms, dom_n = kf.kernel_time(di)
    kf.set_timing(0)
    by, fl = costs[dom]
    by *= a.steps
    fl *= a.steps
    peak_f = PEAK_MFMA_TFLOPS[cfg.dtype]
    t_mem, t_fl = by / (PEAK_HBM_GBS * 1e9), fl / (peak_f * 1e12)
    if t_fl >= t_mem and fl > 0:
        roof = {"bound": "mfma", "achieved": fl / (dom_ms * 1e-3) / 1e12, "peak": peak_f,
                "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": by / (dom_ms * 1e-3) / 1e9, "peak": PEAK_HBM_GBS,
                "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    # HBM bytes per launch of the class from rocprofv3 FETCH_SIZE / WRITE_SIZE
    # (calibrated), when taken on this build of the kernels
    roof["traffic"] = load_traffic(dom, a.workload, B, k)
    roof["kernel_class"] = dom
    roof["launches"] = dom_n
    roof["avg_launch_us"] = dom_ms * 1e3 / max(dom_n, 1)
    roof["algorithmic_per_launch"] = {"bytes": by / max(dom_n, 1), "flops": fl / max(dom_n, 1)}
    roof["operand_bytes_per_launch"] = opcosts[dom][0] * a.steps / max(dom_n, 1)
    gen_bytes = sum(v[0] for v in costs.values())
    gen_flops = sum(v[1] for v in costs.values())
    step_roof_ms = max(gen_bytes / (PEAK_HBM_GBS * 1e9), gen_flops / (peak_f * 1e12)) * 1e3

    res = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == S.DTYPE_BF16 else "fp32",
        "data": "synthetic (seeded N(0,0.02) weights, Zipf/uniform prompts, Philox noise)",
        "config": {"workload": (f"{a.workload}-shaped: {cfg.n_layer} layers, d={cfg.d_model}, "
                                f"{cfg.n_head} heads, MLP {cfg.d_mlp}, vocab {cfg.vocab}, "
                                f"context {cfg.n_ctx}; batch {B}, prompt {N}, k={k}, "
                                f"{L} new tokens per sequence"),
                   "batch": B, "k": k, "prompt": N, "new_tokens": L, "passes": L // k},
        "roofline": roof,
        "step_roofline": {"generate_algorithmic_bytes": gen_bytes,
                          "generate_algorithmic_flops": gen_flops,
                          "roofline_ms": round(step_roof_ms, 4),
                          "frac": round(step_roof_ms / ms_step, 4),
                          "generate_operand_bytes": sum(v[0] for v in opcosts.values())},
        "kernel_ms_per_generate": {n: round(per[n][0], 4) for n in CLASSES},
    }

    if not a.no_ar:
        ar_steps = max(1, a.steps // 4)
        run_ar()
        dt_ar = timed(run_ar, ar_steps)
        v_ar = B * L * ar_steps / dt_ar
        res["k1_ar_baseline"] = {"value": round(v_ar, 1), "unit": "tokens/s",
                                 "ms_per_step": round(dt_ar / ar_steps * 1e3, 4),
                                 "passes": L, "speedup_k_vs_ar": round(value / v_ar, 3)}
        log(f"[bench] AR k=1: {v_ar:,.0f} tokens/s -> speedup {value / v_ar:.2f}x")

    if not a.no_sweep:
        res["owt_sweep"] = owt_sweep([int(x) for x in a.sweep_batches.split(",") if x], stream)

    if not a.no_large:
        res["large_backbone"] = large_bench(stream)

    if not a.no_serving:
        res["serving"] = serving_bench(stream)
        res["serving"]["lockstep_tokens_per_s"] = round(value, 1)

    if not a.no_train_attn:
        res["training_attention"] = training_attention_bench()
    if not a.no_teacher:
        res["teacher_targets"] = teacher_bench()
    if not a.no_rollout:
        res["selfforcing_targets"] = rollout_bench()

    if not a.no_cpu:
        log("[bench] CPU oracle sample ...")
        res["cpu_baseline"] = cpu_baseline(blob, prompt, k, seed, a.cpu_blocks)
        log(f"[bench] CPU oracle: {res['cpu_baseline']['value']:.1f} tokens/s")
    else:
        res["cpu_baseline"] = None
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
