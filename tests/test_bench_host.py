"""Host logic of bench.py (no GPU): the per-call HBM traffic it reports beside the roofline, from
recorded per-dispatch counter values."""
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _setup(tmp_path, monkeypatch, kernels, sources=("k_attn.hip", "k_copy.hip")):
    csrc = tmp_path / "paper_2606_01751_amd" / "csrc"
    csrc.mkdir(parents=True)
    for f in sources:
        (csrc / f).write_text(f"// {f}\n")
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    rec = {"workload": "w", "kernels": {}}
    for sym, (n, nbytes, src_changed) in kernels.items():
        src = bench.KERNELS[sym][1]
        h = "stale" if src_changed else bench.source_hash(src)
        rec["kernels"][sym] = {"entry_point": bench.KERNELS[sym][0], "source_sha256": h, "dispatches": n,
                               "fetch_kib": 0.0, "write_kib": 0.0, "bytes_per_dispatch": nbytes}
    (tmp_path / "profiles" / "traffic_w.json").write_text(json.dumps(rec))


def test_kernels_inside_a_call_add_up(tmp_path, monkeypatch):
    # the scoring call runs the probe gather, the column sums and the head sum: bytes per call are
    # the sum of the three
    _setup(tmp_path, monkeypatch, {"colsum_kernel<128, 2>": (3, 100.0, False),
                                   "probe_gather_kernel<128>": (3, 20.0, False),
                                   "head_reduce_kernel": (3, 5.0, False)})
    assert bench.load_traffic("w") == pytest.approx({"sx_sparseq_score": 125.0})


def test_several_dispatches_of_one_kernel_per_call_add_up(tmp_path, monkeypatch):
    # dispatches per call come from the dispatch count over the calls: with the histogram kernel
    # dispatched twice per call (6 over 3 calls) and per-dispatch means of 10, 20 and 30 bytes, a
    # call moves 2 x 10 + 20 + 30 = 70 bytes
    _setup(tmp_path, monkeypatch, {"topk_hist_kernel": (6, 10.0, False), "topk_bound_kernel": (3, 20.0, False),
                                   "topk_write_kernel": (3, 30.0, False)},
           sources=("k_topk.hip",))
    assert bench.load_traffic("w") == pytest.approx({"sx_topk_select": 70.0})


def test_entry_without_counted_calls_or_with_stale_source_is_dropped(tmp_path, monkeypatch):
    # the row-mark kernel alone is not a call of sx_realign_scatter; a kernel whose source changed
    # since its counters were taken makes its whole entry point unreported
    _setup(tmp_path, monkeypatch, {"mark_rows_kernel": (2, 7.0, False),
                                   "scatter_kernel": (4, 50.0, True),
                                   "attn_mfma_kernel<128, true, true, true>": (28, 300.0, False)})
    assert bench.load_traffic("w") == pytest.approx({"sx_sparse_attn": 300.0})


def test_missing_file_reports_nothing(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.load_traffic("w") == {}


def test_every_kernel_symbol_names_a_source_that_exists():
    for sym, (entry, src, is_call) in bench.KERNELS.items():
        assert entry.startswith("sx_"), sym
        assert os.path.exists(os.path.join(ROOT, "paper_2606_01751_amd", "csrc", src)), sym


def test_every_kernel_symbol_matches_a_kernel_of_its_source():
    # the profiler names a template kernel with all its arguments, so a symbol with too few of them
    # would match no dispatch: the kernel must be a __global__ of the named file, with as many
    # template parameters as the symbol has arguments (a symbol without arguments stands for every
    # instantiation)
    import re
    for sym, (entry, src, is_call) in bench.KERNELS.items():
        text = open(os.path.join(ROOT, "paper_2606_01751_amd", "csrc", src)).read()
        name, _, args = sym.partition("<")
        m = re.search(r"(template <([^>]*)>\s*)?__global__\s+(__launch_bounds__\([^)]*\)\s+)?void\s+"
                      + re.escape(name) + r"\(", text)
        assert m, sym
        if args:
            assert m.group(2) and len(m.group(2).split(",")) == len(args.rstrip(">").split(",")), sym


def test_more_than_one_gpu_is_refused_with_a_message():
    # the step runs on one GPU; asking for more exits with status 2 and says so, before any GPU use
    import subprocess
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_source_hash_ignores_comments_and_layout_but_not_code():
    a = "// kernel\nint f(int x) {  /* block\n comment */ return x + 1; }\n"
    b = "int f(int x) {\n  return x + 1;   // trailing\n}\n"
    c = "int f(int x) { return x + 2; }"
    assert bench.source_code(a) == bench.source_code(b)
    assert bench.source_code(a) != bench.source_code(c)
