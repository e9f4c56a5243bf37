"""bench.py's trace tooling on a synthetic kernel trace (no GPU): the
per-class launch table separates the out-projection from MLP-down (one GEMM
instantiation, alternating in dispatch order), counts a split-K part with the
reduction that follows it, an attention combine with its attention, and a
part with no reduction after it (the noise encoder's fp32 output GEMM) as
noise."""
import csv

import bench

_NS = "_ZN2kf12_GLOBAL__N_1"
GEMM = _NS + "11gemm_kernelIDF16bLi32ELi64ELi2ELi2ELi4ELi0E"
KERNELS = [  # (name, duration in ns), the launch order of one pass
    (_NS + "17embed_real_kernelIDF16bEEvPfPT_", 3000),
    (GEMM + "Lb1ENS0_5EpQKVIDF16bEELi1EEEvNS0_5GemmAEPKT_iiiiT7_i", 10000),
    (_NS + "21attention_mfma_kernelILi64ELi4ELi0EEEvPKDF16b", 6000),
    (_NS + "24attention_combine_kernelILi64EEEvPDF16b", 2000),
    (GEMM + "Lb0ENS0_10EpResidualIDF16bLb0EEELi2EEEvNS0_5GemmAEPKT_iiiiT7_i", 6000),
    (GEMM + "Lb1ENS0_6EpBiasIDF16bEELi1EEEvNS0_5GemmAEPKT_iiiiT7_i", 9000),
    (GEMM + "Lb0ENS0_9EpPartialELi1EEEvNS0_5GemmAEPKT_iiiiT7_i", 8000),
    (_NS + "20splitk_reduce_kernelILi2ENS0_10EpResidualIDF16bLb0EEEEEvPKfiiT0_", 4000),
    (_NS + "11gemm_kernelIDF16bLi128ELi128ELi2ELi2ELi2ELi1ELb1ENS0_6EpHeadELi1EEEv", 20000),
    (_NS + "20argmax_select_kernelEPKfPKiiNS_10KfStepGeomE", 4000),
    (GEMM + "Lb0ENS0_9EpPartialELi1EEEvNS0_5GemmAEPKT_iiiiT7_i", 5000),
    (_NS + "17embed_real_kernelIDF16bEEvPfPT_", 3000),
]


def _trace(path):
    t = 1_000_000
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        for i, (name, ns) in enumerate(KERNELS):
            w.writerow([i + 1, name, t, t + ns])
            t += ns + 500


def _table(out):
    rows = {}
    for line in out.splitlines():
        cells = [c.strip() for c in line.strip().strip("|").split("|")]
        if len(cells) == 4 and cells[1].isdigit():
            rows[cells[0]] = (int(cells[1]), float(cells[2]))
    return rows


def test_class_times_separates_and_merges(tmp_path, capsys):
    p = tmp_path / "run_kernel_trace.csv"
    _trace(p)
    bench.class_times(str(p))
    rows = _table(capsys.readouterr().out)
    assert rows["embed"] == (2, 3.0)
    assert rows["qkv"] == (1, 10.0)
    assert rows["attn"] == (1, 8.0)          # attention + its combine
    assert rows["oproj"] == (1, 6.0)         # the first residual GEMM of the layer
    assert rows["mlp_up"] == (1, 9.0)
    assert rows["mlp_down"] == (1, 12.0)     # split-K part + its reduction
    assert rows["head"] == (1, 20.0)
    assert rows["select"] == (1, 4.0)
    assert rows["noise"] == (1, 5.0)         # a part with no reduction after it


def test_short_names_show_k_groups():
    two = GEMM + "Lb0ENS0_10EpResidualIDF16bLb0EEELi2EEEvNS0_5GemmAEPKT_iiiiT7_i"
    one = GEMM + "Lb1ENS0_6EpBiasIDF16bEELi1EEEvNS0_5GemmAEPKT_iiiiT7_i"
    assert bench._short(two) == "gemm 32x64 2g EpResidual bf16"
    assert bench._short(one) == "gemm 32x64 EpBias bf16"
