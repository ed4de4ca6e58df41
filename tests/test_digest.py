"""The rocprofv3 digests used for the committed profiles (measurement
tooling): parsed from small hand-made trace files."""
import csv

from paper_2602_11456_amd.probes import rocprof_digest


def _trace(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Kernel_Name", "Stream_Id", "Start_Timestamp", "End_Timestamp"])
        for r in rows:
            w.writerow(r)


def test_pipeline_digest_splits_calls_at_the_reset_kernel(tmp_path, capsys):
    k = "void aurora::{}(aurora::ExtractArgs)"
    rows = [
        (k.format("run_reset_kernel"), 3, 0, 1_000),
        (k.format("stage_kernel<false, true, true>"), 1, 1_000, 101_000),
        (k.format("coded_group_kernel"), 2, 101_000, 111_000),
        (k.format("finalize_coded_kernel<false, true, true>"), 2, 111_000, 161_000),
        (k.format("deliver_kernel"), 3, 161_000, 261_000),
        ("__amd_rocclr_copyBuffer(...)", 0, 300_000, 305_000),
        (k.format("run_reset_kernel"), 3, 400_000, 401_000),
        (k.format("stage_kernel<false, true, false>"), 1, 401_000, 651_000),
        (k.format("finalize_kernel<long, false, true, true>"), 2, 651_000, 831_000),
        (k.format("deliver_kernel"), 3, 831_000, 1_091_000),
    ]
    p = tmp_path / "kernel_trace.csv"
    _trace(p, rows)
    rocprof_digest.pipeline(str(p))
    out = capsys.readouterr().out
    assert "call 0 (coded): 5 kernels, first kernel start to last kernel end 0.26 ms" in out
    assert "call 1 (plain): 4 kernels, first kernel start to last kernel end 0.69 ms" in out
    assert "copyBuffer" not in out
    assert "stream 3: 2 kernels, busy   0.10 ms" in out
