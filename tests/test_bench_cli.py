"""bench.py's command line (CPU): one GPU only, workloads known."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_every_workload_has_the_keys_bench_reads():
    sys.path.insert(0, ROOT)
    import synth
    for name, wl in synth.WORKLOADS.items():
        for key in ("unet", "N", "guidance", "weight_seed", "batch", "cond_seed", "uncond_seed"):
            assert key in wl, (name, key)
        if "n_cache" in wl:
            for key in ("d", "clusters", "sigma", "cache_seed", "query_seed", "thresholds"):
                assert key in wl, (name, key)
        if synth.unet_config(wl["unet"]).get("pooled_dim"):
            assert "pooled_seed" in wl, name
