"""bench.py's host-side contract that needs no GPU: it measures one GPU and
refuses a multi-GPU request (or a multi-rank launch) with a message and exit
status 2, before touching torch or the library."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(args, env_extra=None):
    env = dict(os.environ)
    env.update(env_extra or {})
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + args,
                          capture_output=True, text=True, timeout=120, env=env, cwd=ROOT)


def test_bench_refuses_more_than_one_gpu():
    r = _run(["--gpus", "2"])
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_bench_refuses_a_multi_rank_launch():
    r = _run([], {"WORLD_SIZE": "4"})
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_cpu_baseline_fields_small_block():
    """The CPU baseline (the oracle timed on the step) on a small dense block:
    the reported fields and a positive rate."""
    sys.path.insert(0, ROOT)
    import bench
    import synthgen as sg
    cfg = sg.small_dense(batch=2, seq=32, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=384)
    r = bench.cpu_baseline(cfg, sg.block_weights(cfg, 0), sg.activations(cfg, 0))
    assert r["kind"] == "oracle" and r["unit"] == "block-steps/s"
    assert r["value"] > 0 and r["cores"] >= 1
    assert abs(r["value"] * r["seconds_per_step"] - 1.0) < 1e-9
    assert "all rows" in r["sample"] and "2 of the 2 samples" in r["sample"]
