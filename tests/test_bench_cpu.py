"""Host-side checks of bench.py's accounting (no GPU): every kernel the
library times on the measured path has algorithmic bytes, the combined
launches are the sums of their parts, and the counter map names them."""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2606_14782_amd import counters, inputs  # noqa: E402

PROMPT_KERNELS = ["window_lse_kr", "lse_merge", "window_score_calib_kr",
                  "window_score_calib_lse_kr", "window_score_calib_lse", "segment_calib",
                  "segment_score", "segment_cand", "final_topk", "segment_calib_cand",
                  "segment_score_final"]


@pytest.mark.parametrize("name", PROMPT_KERNELS)
def test_kernels_of_the_measured_path_have_bytes(name):
    assert bench.kernel_bytes(name, inputs.workload(3)) > 0


def test_combined_launches_are_sums_of_their_jobs():
    wl = inputs.workload(3)
    kb = lambda n: bench.kernel_bytes(n, wl)
    assert kb("window_score_calib_lse_kr") == pytest.approx(kb("window_score_calib_kr")
                                                          + kb("window_lse_kr"))
    assert kb("segment_calib_cand") == pytest.approx(kb("segment_calib") + kb("segment_cand")
                                                   + kb("lse_merge"))
    assert kb("segment_score_final") == pytest.approx(kb("segment_score") + kb("final_topk"))


@pytest.mark.parametrize("kernel,name", [
    ("void bacon::k_krdual<128, true, 4>(bacon::PassArgs, bacon::PassArgs, bacon::SeqTable)",
     "window_score_calib_lse_kr"),
    ("void bacon::k_pass_dual<true, 128, true>(bacon::PassArgs, bacon::PassArgs, bacon::SeqTable)",
     "window_score_calib_lse"),
    ("bacon::k_sel_a(bacon::SegArgs, bacon::SegArgs, bacon::PassArgs, bacon::SeqTable, int, int)",
     "segment_calib_cand"),
    ("bacon::k_sel_b(bacon::SegArgs, bacon::SegArgs, bacon::SeqTable, int)", "segment_score_final"),
    ("bacon::k_segcal(bacon::SegArgs, bacon::SeqTable)", "segment_calib"),
])
def test_counter_names(kernel, name):
    assert counters.library_name(kernel) == name


def test_bench_refuses_more_than_one_gpu(monkeypatch, capsys):
    monkeypatch.setattr(sys, "argv", ["bench.py", "--gpus", "2"])
    with pytest.raises(SystemExit) as e:
        bench.main()
    assert e.value.code == 2
    assert "one GPU" in capsys.readouterr().err
