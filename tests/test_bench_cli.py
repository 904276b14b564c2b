"""bench.py's command line on the CPU: the one-GPU guard answers before any GPU work."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and "--gpus 2" in r.stderr
    assert r.stdout == ""


def test_algorithmic_work_of_c4():
    # the roofline's per-stage work: layer lane-ops 2 (2^k - 1) w W, bytes (w_in + w) N / 8
    sys.path.insert(0, ROOT)
    import bench
    from paper_2602_07400_amd.workloads import CONFIGS
    cfg = CONFIGS["c4_cifar100_wide"]
    n = cfg.n
    W = n // 64
    st = bench.algorithmic(cfg, n, fused_head=True)
    assert st["layer1"]["ops"] == 2 * 63 * 64000 * W
    assert st["layer1"]["bytes"] == (21504 + 64000) * W * 8
    assert st["layer2"]["ops"] == 2 * 63 * 64000 * W + n * 64000 // 32
    assert st["layer2"]["bytes"] == 64000 * W * 8
    assert st["encode"]["bytes"] == n * 3072 + 21504 * W * 8
    assert st["head"]["bytes"] == 4 * n * 100 + 4 * n
    # a specialized layer counts 2^k' - 1 multiplexers per node
    hist = [None, [1000, 0, 0, 63000, 0, 0, 0]]
    sp = bench.algorithmic(cfg, n, fused_head=True, fanin_hist=hist)
    assert sp["layer2"]["ops"] == 2 * 7 * 63000 * W + n * 64000 // 32
    assert sp["layer1"]["ops"] == st["layer1"]["ops"]
