"""bench.py's host-side contract (no GPU): more than one GPU is refused with a
message and exit status 2, before anything touches a device; the committed
counter summary's machine-readable fields are well formed."""
import json
import os
import re
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_profile_summary_fields():
    text = open(os.path.join(ROOT, "profiles", "mla_online_step_256k.md")).read()
    sha = re.search(r"attend_source_sha256_16: ([0-9a-f]+)", text)
    traffic = re.search(r"attend_traffic_bytes_per_launch: ([0-9]+)", text)
    assert sha and len(sha.group(1)) == 16
    # HBM-side bytes of one attention launch: above the latent stream and the
    # partials it must move (about 8.4 GB), below what 8 TB/s allows in one second
    assert traffic and 8.4e9 < int(traffic.group(1)) < 8e12
