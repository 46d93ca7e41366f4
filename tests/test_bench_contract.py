"""bench.py's command-line contract and the counter records it reads (CPU only)."""
import json
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), (["--gpus", "8"], {}),
                                      ([], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_is_refused_before_any_gpu_work(argv, env):
    e = dict(os.environ, **env)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv], env=e,
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2, r.stderr
    assert "one GPU only" in r.stderr and r.stdout == ""


@pytest.mark.parametrize("record", [bench.TRAFFIC_RECORD, bench.PICARD64_RECORD, bench.MFMA_RECORD])
def test_counter_records_are_well_formed(record):
    """Each committed counter summary carries a JSON record naming the kernel sources it was
    taken with (bench.py uses it only while their hash matches)."""
    text = open(record).read()
    rec = json.loads(re.search(r"```json\n(.*?)```", text, re.S).group(1))
    assert rec["kernel"] and len(rec["source_sha256"]) == 64
    for src in rec["sources"]:
        assert os.path.exists(os.path.join(ROOT, src)), src
    assert "rocprofv3" in text            # the command that produced it
