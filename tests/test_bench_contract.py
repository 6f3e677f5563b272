"""Host-side checks of the benchmark script (no GPU): it refuses more than
one GPU before touching a device, and the committed counter summary it reads
the dominant kernel's HBM traffic from is well formed and plausible."""
import os
import re
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# gate/up weight bytes of the 32 kept Qwen3-shaped experts (2 I d bf16 each)
GATEUP_BYTES = 32 * 2 * 768 * 2048 * 2


def test_more_than_one_gpu_is_refused():
    for argv, env in ((["--gpus", "2"], {}), (["--gpus", "1"], {"WORLD_SIZE": "4"})):
        r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv],
                           capture_output=True, text=True, timeout=120,
                           env={**os.environ, **env})
        assert r.returncode == 2
        assert "one GPU" in r.stderr
        assert r.stdout.strip() == ""        # no JSON line


def test_counter_summary_is_well_formed():
    path = os.path.join(ROOT, "profiles", "counters_ffn_gateup_qwen3_b256_be32.md")
    txt = open(path).read()
    assert re.search(r"kernel_source_sha256_16:\s*[0-9a-f]{16}\b", txt)
    m = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", txt)
    assert m
    traffic = float(m.group(1))
    # the measured bytes cover the weights once, plus tokens, activations
    # and re-reads that miss L2: more than the weights, well under 1.5 times
    assert GATEUP_BYTES <= traffic <= 1.5 * GATEUP_BYTES
    # every rocprofv3 command it quotes runs committed files only
    for cmd in re.findall(r"^\s+(rocprofv3 .*)$", txt, re.M):
        assert "_work" not in cmd and " -- python3 bench.py" in cmd
