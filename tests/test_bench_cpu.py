"""Host-side checks of bench.py's accounting (no GPU): the roofline counts a
layer's K once (K + Q_win + E written for the launch that completes a
layer's K pass), the launches of a layer add up to the per-layer
algorithmic bytes, combined launches are the sums of their jobs, and the
counter map names every kernel."""
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
def test_kernels_of_the_measured_path_are_accounted(name):
    wl = inputs.workload(3)
    kb, db = bench.kernel_bytes(name, wl), bench.design_bytes(name, wl)
    if name in bench.DESIGN_ONLY:
        assert kb == 0.0
    else:
        assert kb > 0
    assert db >= kb


def test_score_pass_counts_one_layer_of_k():
    """The dual launch (pass 2 of layer l, pass 1 of l+1) completes one layer's
    K pass: K once, Q_win and E written -- 68,419,584 bytes on the 32K video
    workload, 0.24 of 8 TB/s at 35.40 us; its design bytes read K twice."""
    wl = inputs.workload(3)
    K = 32768 * 8 * 128 * 2
    Q = 32 * 32 * 128 * 2
    vec = 32768 * 8 * 4
    for name in bench.SCORE_PASSES:
        assert bench.kernel_bytes(name, wl) == K + Q + vec
    assert bench.kernel_bytes("window_score_calib_lse_kr", wl) == 68419584
    assert bench.design_bytes("window_score_calib_lse_kr", wl) == 2 * (K + Q) + 2 * vec
    frac = 68419584 / 35.40e-6 / 8e12
    assert frac == pytest.approx(0.2416, abs=1e-3)


@pytest.mark.parametrize("idx", range(5))
def test_launches_of_a_layer_add_up_to_its_algorithmic_bytes(idx):
    """Prompt schedule: one score launch, the calibration launch and the
    score/final launch per layer carry exactly the per-layer bytes (K once,
    Q_win, the E history read and written, the gather, the indices)."""
    wl = inputs.workload(idx)
    kb = lambda n: bench.kernel_bytes(n, wl)
    total = kb("window_score_calib_lse_kr") + kb("segment_calib_cand") + kb("segment_score_final")
    assert total == pytest.approx(bench.algorithmic_bytes(wl)["layer_mean"], rel=1e-12)


def test_combined_launches_are_sums_of_their_jobs():
    wl = inputs.workload(3)
    kb = lambda n: bench.kernel_bytes(n, wl)
    assert kb("window_score_calib_lse_kr") == pytest.approx(kb("window_score_calib_kr")
                                                          + kb("window_lse_kr"))
    db = lambda n: bench.design_bytes(n, wl)
    assert db("window_score_calib_lse_kr") == pytest.approx(db("window_score_calib_kr")
                                                          + db("window_lse_kr"))
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
