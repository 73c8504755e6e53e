"""The hybrid data/model-parallel projection (Section 3, Equations 1-6), pinned
to the numbers the paper's evaluation reports and to the pipeline-bubble
closed form.  Host arithmetic only."""
import json
import math
import random

import pytest

from paper_1907_13257_amd import hybrid


def test_eq2_reduces_to_eq3_for_a_constant_per_device_batch():
    # Section 3: with the per-device mini-batch fixed, S_1 / S_N = N and
    # T_1 / T_N is the scaling efficiency SE_N
    T1, TN, N, E1, EN = 2.0, 2.5, 16, 4.0, 5.0
    S1 = 1000.0
    a = hybrid.dp_speedup_from_times(T1, TN, S1, S1 / N, E1, EN)
    b = hybrid.dp_speedup(T1 / TN, N, E1, EN)
    assert a == pytest.approx(b, rel=1e-15)
    # Equation 1: the speedup is the ratio of training times
    assert hybrid.training_time(T1, S1, E1) / hybrid.training_time(TN, S1 / N, EN) == pytest.approx(a, rel=1e-15)


def test_eq6_is_eq5_against_eq4():
    rng = random.Random(7)
    for _ in range(2000):
        m = rng.choice([2, 3, 4, 8])
        n = rng.choice([1, 2, 4, 16, 128])
        su_m = rng.uniform(0.5, 3.0)
        se_n, se_mn = rng.uniform(0.5, 1.0), rng.uniform(0.3, 1.0)
        e1 = rng.uniform(1, 10)
        e_n = e1 * rng.uniform(1, 3)
        e_mn = e_n * rng.uniform(1, 4)
        lhs = hybrid.hybrid_speedup(su_m, se_n, n, e1, e_n)
        rhs = hybrid.dp_speedup(se_mn, m * n, e1, e_mn)
        if abs(lhs - rhs) > 1e-9 * rhs:
            assert hybrid.hybrid_wins(su_m, m, se_n, se_mn, e_n, e_mn) == (lhs > rhs)


def test_inception_hybrid_beats_dp_at_64_gpus_by_15_5_percent():
    # Evaluation: epochs rise from four to seven once the global batch grows
    # past 32 GPUs; Table 1: 2-way MP speedup 1.32x; SE_N = 1 as assumed in the
    # evaluation.  The paper projects the hybrid (32-way DP of 2-way MP) at
    # least 15.5% ahead of 64-way DP.
    e = {1: 4.0, 32: 4.0, 64: 7.0}
    ratio = hybrid.hybrid_speedup(1.32, 1.0, 32, e[1], e[32]) / hybrid.dp_speedup(1.0, 64, e[1], e[64])
    assert ratio == pytest.approx(1.155, abs=5e-4)
    assert hybrid.hybrid_wins(1.32, 2, 1.0, 1.0, e[32], e[64])
    assert hybrid.hybrid_threshold(2, 1.0, 1.0, e[32], e[64]) == pytest.approx(2 * 4 / 7)


def test_biglstm_hybrid_at_32_gpus():
    # Evaluation: 32-way DP needs 3.2x the epochs of 16-way DP; Table 1: 2-way
    # pipeline speedup 1.22x.  The hybrid on 32 GPUs is 1.22x the best DP-only
    # scale (16 GPUs), and far ahead of 32-way DP.
    e = {1: 1.0, 16: 1.0, 32: 3.2}
    rows = {r["devices"]: r for r in hybrid.project(e, 1.22, 2)}
    assert rows[32]["hybrid"] / rows[16]["dp"] == pytest.approx(1.22, rel=1e-12)
    assert rows[32]["hybrid_wins"] is True
    assert rows[32]["hybrid"] / rows[32]["dp"] == pytest.approx(1.22 * 3.2 / 2, rel=1e-12)
    assert rows[16]["hybrid"] is None   # E_8 not given
    # with no statistical-efficiency loss, MP must beat M itself (Equation 6)
    assert not hybrid.hybrid_wins(1.99, 2, 1.0, 1.0, 5.0, 5.0)
    assert hybrid.hybrid_wins(2.01, 2, 1.0, 1.0, 5.0, 5.0)


def test_pipeline_bubble_closed_form():
    # a step time proportional to the batch: SU = m*S / (m + S - 1)
    lin = {b: 0.01 * b for b in (8, 16, 32, 64, 128, 256)}
    for S in (2, 4):
        for m in (1, 2, 4, 8, 16):
            assert hybrid.pipeline_mp_speedup(lin, 128, m, S) == pytest.approx(m * S / (m + S - 1), rel=1e-12)
    # a step time independent of the batch (latency-bound): SU = S / (m + S - 1) <= 1
    flat = {b: 3.0 for b in (16, 32, 64, 128)}
    for m in (1, 2, 4, 8):
        assert hybrid.pipeline_mp_speedup(flat, 128, m, 2) == pytest.approx(2 / (m + 1), rel=1e-12)
    # one micro-batch: the stages run one after another, no gain
    assert hybrid.pipeline_mp_speedup({64: 1.7}, 64, 1, 2) == pytest.approx(1.0)
    # transfers between stages lengthen the pipelined step
    assert hybrid.pipeline_mp_speedup(lin, 128, 4, 2, comm_ms=0.2) < hybrid.pipeline_mp_speedup(lin, 128, 4, 2)


def test_best_pipeline_picks_the_fastest_split():
    t = {64: 1.7, 128: 2.3, 256: 4.7, 512: 9.7}
    micro, su = hybrid.best_pipeline(t, 512)
    cand = {m: hybrid.pipeline_mp_speedup(t, 512, m) for m in (1, 2, 4, 8)}
    assert micro == max(cand, key=cand.get) and su == pytest.approx(max(cand.values()))
    assert hybrid.best_pipeline({128: 2.0}, 96) is None


@pytest.mark.parametrize("bad", [
    lambda: hybrid.dp_speedup(1.0, 0, 1.0, 1.0),
    lambda: hybrid.dp_speedup(-1.0, 2, 1.0, 1.0),
    lambda: hybrid.hybrid_threshold(2, 1.0, 1.0, 0.0, 1.0),
    lambda: hybrid.pipeline_mp_speedup({64: 1.0, 128: 2.0}, 128, 3),
    lambda: hybrid.pipeline_mp_speedup({64: 1.0, 128: 2.0}, 128, 2, comm_ms=-1),
    lambda: hybrid.pipeline_mp_speedup({128: 2.0}, 128, 2),
    lambda: hybrid.training_time(float("nan"), 1.0, 1.0),
])
def test_invalid_inputs_raise(bad):
    with pytest.raises((ValueError, KeyError)):
        bad()


def test_cli_reads_bench_lines(tmp_path, capsys):
    paths = []
    for b, ms in ((64, 1.7), (128, 2.3), (256, 4.65)):
        p = tmp_path / f"b{b}.json"
        p.write_text("noise\n" + json.dumps({"ms_per_step": ms, "config": {"B": b}}) + "\n")
        paths.append(str(p))
    assert hybrid.main(["--sweep", *paths, "--epochs", "1:1,2:1,4:1.5"]) == 0
    out = json.loads(capsys.readouterr().out)
    assert out["step_ms"] == {"64": 1.7, "128": 2.3, "256": 4.65}
    assert out["su_m"]["256"]["micro_batches"] == 2
    assert out["su_m"]["256"]["su_m"] == pytest.approx(4.65 / (3 * 2.3 / 2))
    assert out["su_m"]["128"]["su_m"] == pytest.approx(max(1.0, 2.3 / (3 * 1.7 / 2)))
    proj = out["projection"]["256"]
    assert [r["devices"] for r in proj] == [1, 2, 4]
    assert math.isclose(proj[2]["dp"], 4 / 1.5)
