"""The CPU-side summarisers of bench.py that turn rocprofv3 traces and
time-model tables into the committed profiles (synthetic inputs)."""
import csv
import io
import contextlib

import bench

FIELDS = ["Kind", "Kernel_Name", "Start_Timestamp", "End_Timestamp", "Workgroup_Size_X", "Grid_Size_X"]


def _trace(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for name, t0, dur, wgs in rows:
            w.writerow(dict(Kind="KERNEL_DISPATCH", Kernel_Name=name, Start_Timestamp=t0, End_Timestamp=t0 + dur,
                            Workgroup_Size_X=256, Grid_Size_X=256 * wgs))


def test_trace_groups_split_runs_by_idle_time(tmp_path):
    p = tmp_path / "k.csv"
    k = "void stmoe::(anonymous namespace)::ffn_gate_up<true, 64, 1, 1, true>(stmoe::FfnArgs, int, int)"
    rows = [(k, 1000 * i, 500, 1536) for i in range(8)]                     # run 0
    rows += [("void at::native::fill_kernel(float*)", 9000, 100, 4)]        # ignored: not this library's
    rows += [(k, 5_000_000 + 1000 * i, 700, 1536) for i in range(4)]        # run 1, after a 5 ms pause
    _trace(p, rows)
    g = bench.trace_groups(str(p))
    assert sorted(g) == [(0, "stmoe::ffn_gate_up<true, 64, 1, 1, true>", 1536),
                         (1, "stmoe::ffn_gate_up<true, 64, 1, 1, true>", 1536)]
    assert g[(0, "stmoe::ffn_gate_up<true, 64, 1, 1, true>", 1536)] == [0.5] * 8
    med, kept = bench._median_kept([9.0, 1.0, 2.0, 3.0])        # the first quarter is dropped
    assert kept == [1.0, 2.0, 3.0] and med == 2.0


def test_summarize_policy_pivots_rows(tmp_path):
    p = tmp_path / "pb.md"
    p.write_text("| workload | link GB/s | copy ms | attention ms/layer | policy | copies | wasted copy-ms | "
                 "stall ms/token | stall vs on-demand |\n|---|---|---|---|---|---|---|---|---|\n"
                 "| w (layer 0.1 ms) | 57 (measured) | 6.0 | 0.00 | demand | 10 | 0.0 | 4.00 | +0.000 |\n"
                 "| w (layer 0.1 ms) | 57 (measured) | 6.0 | 0.00 | optimum | 8 | 0.0 | 3.00 | +0.250 |\n")
    out = io.StringIO()
    with contextlib.redirect_stdout(out):
        bench.summarize_policy(str(p))
    lines = out.getvalue().strip().splitlines()
    assert lines[0].startswith("| workload | link GB/s | attention ms/layer | on-demand stall ms/token | optimum |")
    assert lines[2] == "| w | 57 (measured) | 0.00 | 4.00 | +0.250 |"


def test_summarize_floor_interpolates_the_read_floor(tmp_path):
    from paper_2606_15453_amd import workload as W
    rf = tmp_path / "rf.csv"
    # 32 KiB per workgroup: 768 workgroups = 24 MiB in 6 us, 1536 = 48 MiB in 10 us
    calib = "void stmoe::(anonymous namespace)::calib_read_blocked_kernel<2048ul>(char const*, unsigned long, unsigned*)"
    _trace(rf, [(calib, 1000 * i, 6000, 768) for i in range(4)] + [(calib, 10_000_000 + 20_000 * i, 10000, 1536)
                                                                   for i in range(4)])
    fs = tmp_path / "fs.csv"
    rows, t = [], 0
    for name in bench.SWEEP_CONFIGS:
        cfg = W.CONFIGS[name]
        _, _, _, sel = bench.sweep_routing(cfg)
        nb = len(sel) + cfg.n_shared
        esz = 2 if cfg.dtype == "bf16" else 4
        up = nb * 2 * cfg.H * cfg.I * esz
        for i in range(4):
            # gate/up at exactly 5 TB/s, down at 4 TB/s
            rows.append(("void stmoe::(anonymous namespace)::ffn_gate_up<x>(stmoe::FfnArgs)", t, int(up / 5e3), 64))
            t += int(up / 5e3) + 10
            rows.append(("void stmoe::(anonymous namespace)::ffn_down_rows<x>(stmoe::FfnArgs)", t,
                         int(up / 2 / 4e3), 32))
            t += int(up / 2 / 4e3) + 10
        t += 10_000_000
    _trace(fs, rows)
    out = io.StringIO()
    with contextlib.redirect_stdout(out):
        bench.summarize_floor(str(rf), str(fs))
    txt = out.getvalue()
    assert "| 24 | 6.00 |" in txt and "| 48 | 10.00 |" in txt
    gu = [l for l in txt.splitlines() if "`ffn_gate_up<x>`" in l]
    dn = [l for l in txt.splitlines() if "`ffn_down_rows<x>`" in l]
    assert len(gu) == len(dn) == len(bench.SWEEP_CONFIGS)
    for l in gu:       # GB/s from the algorithmic bytes (durations rounded to whole ns)
        assert abs(float(l.split("|")[6]) - 5000) <= 0.01 * 5000, l
    for l in dn:
        assert abs(float(l.split("|")[6]) - 4000) <= 0.01 * 4000, l


def test_strip_c_comments_keeps_code_and_literals():
    """The FFN source hash ignores comments: line and block comments go,
    string and character literals (which may hold comment markers) stay."""
    import bench
    src = ('int a = 1; // line\n/* block\n over lines */ const char* s = "x // y /* z */";\n'
           "char q = '\"'; char e = '\\\\'; int b; /**/ int c;\n")
    out = bench.strip_c_comments(src)
    assert "line" not in out and "block" not in out and "over lines" not in out
    assert '"x // y /* z */"' in out and "'\"'" in out and "'\\\\'" in out
    assert "int a = 1;" in out and "int b;" in out and "int c;" in out
    # a comment-only edit leaves the stripped text unchanged
    assert bench.strip_c_comments(src.replace("// line", "// another note")) == out


def test_repeat_summary():
    """Rates of repeated timed runs: the first is the reported value, the
    median and the spread summarise all of them."""
    import bench
    r = bench.repeat_summary(200, [0.8, 0.5, 1.0])
    assert r["runs"] == 3 and r["tokens_per_s"] == [250.0, 400.0, 200.0]
    assert r["median"] == 250.0 and r["spread"] == round((400 - 200) / 250, 4)


def test_timing_cadence():
    """Event-timed tokens: every TIMING_EVERY-th of a long run, at least two
    of a short one, every token of a run of one to three."""
    import bench
    assert bench.timing_cadence(200) == bench.TIMING_EVERY
    assert bench.timing_cadence(100) == bench.TIMING_EVERY
    assert bench.timing_cadence(10) == 5
    assert bench.timing_cadence(3) == 1 and bench.timing_cadence(1) == 1
    for steps in range(1, 300):
        c = bench.timing_cadence(steps)
        timed = len(range(0, steps, c))
        assert 1 <= c <= bench.TIMING_EVERY and (timed >= 2 or steps == 1)
