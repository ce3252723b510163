"""Host logic of bench.py that needs no GPU: the one-GPU rule, the amd-smi
parser behind the clock and power readings, and the kernel-trace summary
that the committed profiles are made with."""
import csv
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


SMI_TEXT = """GPU: 0
    POWER:
        SOCKET_POWER: 1362 W
        GFX_VOLTAGE: N/A
    CLOCK:
        GFX_0:
            CLK: 1901 MHz
            MIN_CLK: 500 MHz
            MAX_CLK: 2400 MHz
        GFX_1:
            CLK: 1957 MHz
            MIN_CLK: 500 MHz
            MAX_CLK: 2400 MHz
        MEM_0:
            CLK: 2000 MHz
        VCLK_0:
            CLK: 59 MHz
"""


def test_smi_parser_takes_socket_power_and_gfx_clocks_only():
    got = bench.parse_smi_metric(SMI_TEXT)
    assert got == {"power_W": 1362.0, "gfx_MHz": [1901, 1957]}
    # no GFX section: no reading
    assert bench.parse_smi_metric("GPU: 0\n    POWER:\n        SOCKET_POWER: 900 W\n") is None
    # a power field the tool cannot read
    got = bench.parse_smi_metric(SMI_TEXT.replace("1362 W", "N/A"))
    assert got["power_W"] is None and got["gfx_MHz"] == [1901, 1957]


def test_trace_summary_separates_detail_and_timed_launches(tmp_path, capsys):
    """A kernel with 2 launches per step: warm-up 1 + 4 one-stream detail
    steps, then the settle steps, 1 warm-up and 3 timed steps; launches after
    those (other measurements) are left out."""
    per, warm, timed = 2, 1, 3
    one = warm + 4
    total = one + 6 + warm + timed
    durs = ([10.0] * per * warm + [20.0] * per * 4 + [25.0] * per * 6 + [30.0] * per * warm +
            [40.0] * per * timed + [99.0] * 5)
    path = tmp_path / "trace.csv"
    t = 1_000_000
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        for d in durs:
            w.writerow(["void fg::dma::wgrad_dma_kernel<fg::dma::K<32, 4, 2, 4, 256>, true>"
                        "(fg::WgradArgs, fg::dma::TileMap)", t, t + int(d * 1000)])
            w.writerow(["fg::split_reduce_kernel(float const*, int, long, unsigned short*, "
                        "int*)", t + 100_000, t + 105_000])
            t += 200_000
    bench.summarize_trace(str(path), "wgrad_dma_kernel<true>", per, timed, warm, 6)
    out = capsys.readouterr().out
    assert f"{per * total} launches in the {total} steps" in out
    assert "one-stream detail steps: 8 launches, average 20.00 us" in out
    assert f"timed region (last {timed} steps): 6 launches, average 40.00 us" in out


def test_traffic_record_is_keyed_by_kernel_and_planner_sources(tmp_path, monkeypatch):
    """recorded_traffic reads the committed profile's line for the kernel only
    while the hash of the kernel's source and the planner's matches."""
    prof = tmp_path / "profiles"
    prof.mkdir()
    k = "wgrad_dma_kernel<true>"
    good = bench.source_hash(k)
    (prof / "fcn_step_hbm_traffic.md").write_text(
        f"traffic: kernel={k} src_sha256_16={good} bytes_per_launch=123\n"
        f"traffic: kernel=data_conv_dma_kernel<true, false> src_sha256_16=0000000000000000 "
        f"bytes_per_launch=456\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    # source_hash reads the sources under ROOT: give the temporary root the
    # real source files
    csrc = tmp_path / "paper_1909_11150_amd" / "csrc"
    csrc.mkdir(parents=True)
    for f in ("conv_dma.hip", "conv_igemm.hip"):
        (csrc / f).write_bytes(open(os.path.join(ROOT, "paper_1909_11150_amd", "csrc", f),
                                    "rb").read())
    assert bench.recorded_traffic(k) == 123
    assert bench.recorded_traffic("data_conv_dma_kernel<true, false>") is None
    # an edit to the planner's file invalidates the record
    (csrc / "conv_igemm.hip").write_bytes(b"// edited\n" + (csrc / "conv_igemm.hip").read_bytes())
    assert bench.recorded_traffic(k) is None


def test_ceiling_summary_prints_every_section(tmp_path, capsys):
    """summarize_ceiling turns the --ceiling JSON line into the three tables
    of the committed ceiling profile; the total row's ratio is the vendor
    time over this library's."""
    clk = {"samples": 9, "gfx_MHz_median": 1920, "gfx_MHz_min": 1850, "gfx_MHz_max": 2010,
           "socket_power_W_median": 1398.0}
    d = {"step": {"ms": 5.2, "tflops": 1060.0, **clk},
         "gemm_8192": {"ms": 0.86, "tflops": 1280.0, **clk},
         "passes": [{"pass": "E1b.fwd", "gemm_mnk": [65536, 512, 4608], "ours_us": 226.9,
                     "ours_tflops": 1362.9, "gemm_us": 264.8, "gemm_tflops": 1167.8}],
         "passes_total": {"ours_us": 200.0, "gemm_us": 250.0, "ours_tflops": 1.0,
                          "gemm_tflops": 1.0},
         "sustained_passes": [{"pass": "E1b.dW", "kernel": "wgrad_dma_kernel<true>",
                               "us": 251.0, "tflops": 1232.0, "frac_of_peak_at_clock": 0.616,
                               **clk}]}
    path = tmp_path / "ceiling.json"
    path.write_text("warm-up text\n" + json.dumps(d) + "\n")
    bench.summarize_ceiling(str(path))
    out = capsys.readouterr().out
    assert "| encoder-decoder step, 3 streams | 5.2000 | 1060.0 | 42.4% | 1920 (1850-2010)" in out
    assert "the same, A about half zero" not in out  # absent runs are left out
    assert "| E1b.dW | `wgrad_dma_kernel<true>` | 251.0 | 1232.0 | 1920 (1850-2010) " \
           "| 1398.0 | 0.616 |" in out
    assert "| E1b.fwd | 65536 x 512 x 4608 | 226.9 |" in out
    assert out.rstrip().endswith("| 1.25 |")


def test_kernel_names_from_the_trace_match_the_library_names():
    """rocprofv3's demangled names map to the names fg_conv_kernel_name
    reports: namespaces and arguments dropped, the pipeline configuration
    dropped unless its tile is not 256, anonymous namespaces too."""
    f = bench.short_kernel_name
    assert f("void fg::dma::wgrad_dma_kernel<fg::dma::K<32, 4, 2, 4, 256>, true>"
             "(fg::WgradArgs, fg::dma::WgradDiv, fg::dma::TileMap)") == "wgrad_dma_kernel<true>"
    assert f("void fg::dma::data_conv_dma_kernel<fg::dma::K<32, 5, 2, 2, 128>, false, true>"
             "(fg::DataConvArgs, fg::dma::TileMap)") == "data_conv_dma_kernel<128, false, true>"
    assert f("fg::(anonymous namespace)::mfma_loop_kernel(float*, int, int)") == \
        "mfma_loop_kernel"
    assert f("fg::split_reduce_kernel(float const*, int, long, unsigned short*, int*)") == \
        "split_reduce_kernel"
