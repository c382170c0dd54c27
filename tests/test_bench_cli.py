"""bench.py's command line (no GPU): more than one GPU is refused with a
message before anything touches the device."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run(*args, env=None):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=120, env=env)


def test_more_than_one_gpu_is_refused():
    r = run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_a_distributed_launch_is_refused():
    env = dict(os.environ, WORLD_SIZE="4")
    r = run(env=env)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_unknown_workload_is_rejected():
    r = run("--workload", "no_such_workload")
    assert r.returncode != 0 and "invalid choice" in r.stderr


def test_profiled_figures_belong_to_these_kernel_sources():
    """The HBM traffic and VALU count that bench.py reports come from the
    committed counter runs, and only while the kernel sources hash to the ones
    profiled: a kernel change needs new counter runs (profiles/traffic.json)."""
    import importlib.util
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    bench = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bench)
    traffic = bench.profiled_traffic("llama3_8b_kv")
    valu = bench.profiled_traffic("llama3_8b_kv", "valu_insts_per_block")
    assert traffic is not None and valu is not None, "kernel sources changed since profiles/traffic.json"
    # the algorithmic bytes of the workload's seal kernel, and at most 1% above them
    assert 18123587584 <= traffic <= 1.01 * 18123587584
    assert 300 < valu < 600
    mix = bench.profiled_traffic("llama3_8b_kv", "valu_mix_per_block")
    assert mix is not None and 0 < mix["v_perm_b32"] + mix["v_bitop3_b32"] < valu
    assert bench.profiled_traffic("tamper") is None  # profiled on one workload only


def _bench_module():
    import importlib.util
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    bench = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bench)
    return bench


def test_lds_and_valu_ceilings():
    """The ceilings bench.py reports beside the HBM roofline.  LDS: 197
    four-byte reads at r32 lane-reads per CU-clock plus 512 B at r128 B per
    CU-clock per 16-byte block.  VALU: each named instruction at its probed
    rate, the rest at 64 lane-ops per CU-clock; with every rate at 64 (or no
    probe) it is the 64-lane figure, and the weighting is a harmonic mean."""
    bench = _bench_module()
    probe = {"b32_lane_reads_per_clk": 32.0, "b128_bytes_per_clk": 256.0,
             "valu_perm_lane_ops_per_clk": 64.0, "valu_bitop3_lane_ops_per_clk": 64.0}
    gbps, cycles = bench.lds_ceiling(probe, 256)
    assert cycles == 197 / 32 + 2  # 8.15625 CU-clocks per block
    assert abs(gbps - 16 * 256 * 2.4 / cycles) < 1e-9
    assert abs(bench.lds_ceiling(probe, 256, 1.2e9)[0] - gbps / 2) < 1e-9
    mix = {"v_perm_b32": 206, "v_bitop3_b32": 156}
    nominal = 16 * 256 * 64 * 2.4 / 420.0
    for p, m in ((probe, mix), (None, mix), (probe, None)):
        g, lane_ops = bench.valu_ceiling(420.0, m, p, 256)
        assert lane_ops == 64.0 and abs(g - nominal) < 1e-9
    fast = dict(probe, valu_bitop3_lane_ops_per_clk=128.0, valu_perm_lane_ops_per_clk=32.0)
    g, lane_ops = bench.valu_ceiling(420.0, mix, fast, 256)
    clk = 206 / 32 + 156 / 128 + 58 / 64
    assert abs(lane_ops - 420 / clk) < 1e-12 and abs(g - 16 * 256 * lane_ops * 2.4 / 420) < 1e-9
