"""Host-side pieces of bench.py (CPU): the one-GPU contract, and the work
accounting its rooflines divide by, checked against the per-step figures of
the scope table the workloads come from (projection and attention flops of one
forward, LM-head bytes) for the four bf16 workloads."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2608_22646_amd import synth  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


# per forward: projection flops, attention flops (4 B Hq L^2 hd per layer), LM-head bytes (weights + rows + out)
SCOPE = {
    "llada_b1": (7.147e12, 1.374e11, 1.036e9),
    "llada_b8": (1.1435e14, 4.398e12, 1.038e9),
    "dream_b1": (1.0023e13, 2.368e11, 1.090e9),
    "dream_long": (1.1025e14, 2.865e13, 1.090e9),
}


@pytest.mark.parametrize("name", sorted(SCOPE))
def test_work_per_forward_matches_the_scope_table(name):
    wl = synth.WORKLOADS[name]
    cfg = wl.model
    f = bench.forward_flops(cfg, wl.batch, wl.prompt_len + wl.gen_len)
    gemm, attn, head = SCOPE[name]
    assert f["layer_gemm"] * cfg.n_layers == pytest.approx(gemm, rel=2e-3)
    assert f["attn"] * cfg.n_layers == pytest.approx(attn, rel=2e-3)
    assert f["total"] == pytest.approx(gemm + attn, rel=2e-3)
    assert bench.head_bytes(cfg, wl.batch * wl.block_len) == pytest.approx(head, rel=2e-3)


def test_traffic_is_reported_only_for_the_workload_its_counters_cover():
    for kernel in bench.TRAFFIC:
        assert bench.measured_traffic("dream_b1", kernel) is None


def test_profile_utilisation_summary(tmp_path, capsys):
    """profsum util on a hand-made counter CSV: one kernel, two dispatches of
    10 us; 8 XCDs x 20000 busy cycles (2.0 GHz), the MFMA busy on half of the
    1024 SIMDs' cycles, the texture-address units 3/4 busy, waves waiting a
    third of their cycles."""
    from paper_2608_22646_amd import profsum
    cyc = 20000
    vals = {"GRBM_GUI_ACTIVE": 8 * cyc, "SQ_VALU_MFMA_BUSY_CYCLES": 0.5 * cyc * 256 * 4,
            "TA_TA_BUSY_sum": 0.75 * cyc * 256, "SQ_WAIT_INST_ANY": 100.0, "SQ_WAVE_CYCLES": 300.0}
    lines = ["Dispatch_Id,Kernel_Name,Counter_Name,Counter_Value,Start_Timestamp,End_Timestamp"]
    for d in (1, 2):
        for k, v in vals.items():
            lines.append(f'{d},"void dllm::(anonymous namespace)::gemm_wd_kernel<X, 2>(dllm::GemmArgs)",{k},{v},'
                         f'{1000000 * d},{1000000 * d + 10000}')
    path = tmp_path / "c.csv"
    path.write_text("\n".join(lines) + "\n")
    profsum.util(str(path), 256, 8, "cmd")
    row = [ln for ln in capsys.readouterr().out.splitlines() if "gemm_wd_kernel<X, 2>" in ln]
    assert len(row) == 1
    n, us, ghz, mf, ta, wt = row[0].split()[:6]
    assert (int(n), float(us), float(ghz)) == (2, 10.0, 2.0)
    assert (float(mf), float(ta), float(wt)) == (0.5, 0.75, 0.333)
