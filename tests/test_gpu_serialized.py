"""Launch-order independence: the layer and decoder block sweeps of tests/serialized_case.py run
once in this process and once in a child process with every kernel launch serialized
(AMD_SERIALIZE_KERNEL=3: the runtime waits for the device before and after each launch;
HIP_LAUNCH_BLOCKING=1), and every output must agree bit for bit.  A result that depended on
launches overlapping, or on a missing ordering between them, would differ."""
import os
import subprocess
import sys

import numpy as np
import pytest

from tests import serialized_case

pytestmark = pytest.mark.gpu


def test_serialized_launches_give_identical_outputs(rq, ctx, tmp_path):
    print("\n[gpu-case] serialized launches: in-process run", flush=True)
    ref = serialized_case.run(rq, ctx)
    path = tmp_path / "serialized.npz"
    env = dict(os.environ, AMD_SERIALIZE_KERNEL="3", HIP_LAUNCH_BLOCKING="1", PYTHONUNBUFFERED="1")
    print("[gpu-case] serialized launches: child process", flush=True)
    proc = subprocess.run([sys.executable, os.path.abspath(serialized_case.__file__), str(path)], env=env,
                          capture_output=True, text=True, timeout=240)
    print(proc.stdout[-2000:], proc.stderr[-2000:], flush=True)
    assert proc.returncode == 0
    got = np.load(path)
    assert sorted(got.files) == sorted(ref)
    for k, v in ref.items():
        assert np.array_equal(got[k], v, equal_nan=True), k
