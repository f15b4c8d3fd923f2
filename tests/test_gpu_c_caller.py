"""The library driven from plain C (tests/c_caller/realq_layer_c.c: HIP runtime C API for memory and
the stream, one realq_quantize_layer call, no PyTorch), checked against the float64 oracle on the
same seeded inputs."""
import subprocess

import numpy as np
import pytest

import oracle
import synth
from tests import parity as P
from tests.c_caller import compile_c_caller

pytestmark = pytest.mark.gpu

def test_c_caller_matches_oracle(tmp_path):
    import torch
    exe = tmp_path / "realq_layer_c"
    r = compile_c_caller(exe)
    assert r.returncode == 0, r.stderr
    L = synth.make_module("single_512", m=96, n=384, T=1024, seed=3)
    m, n = L.W0.shape
    T = L.X.shape[0]
    steps, lr = 2, 1e-3
    inp, out = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(inp, "wb") as f:
        f.write(np.array([m, n, T, steps], dtype=np.int64).tobytes())
        f.write(np.array([lr], dtype=np.float32).tobytes())
        f.write(np.ascontiguousarray(L.W0, dtype=np.float32).tobytes())
        f.write(synth.bf16_bits(L.X).tobytes())
        f.write(synth.bf16_bits(L.Xhat).tobytes())
        f.write(np.ascontiguousarray(L.s, dtype=np.float32).tobytes())
    print(f"\n[gpu-case] C caller on a {m}x{n} layer, {T} tokens", flush=True)
    run = subprocess.run([str(exe), str(inp), str(out)], capture_output=True, text=True, timeout=120)
    print(run.stdout, run.stderr, flush=True)
    assert run.returncode == 0, run.stderr
    g = -(-n // 128)
    buf = open(out, "rb").read()
    o = 0

    def take(count, dtype):
        nonlocal o
        a = np.frombuffer(buf, dtype=dtype, count=count, offset=o)
        o += a.nbytes
        return a

    res = type("R", (), {})()
    res.codes = torch.from_numpy(take(m * n, np.uint8).reshape(m, n).copy())
    res.scales = torch.from_numpy(take(m * g, np.float32).reshape(m, g).copy())
    res.zeros = torch.from_numpy(take(m * g, np.uint8).reshape(m, g).copy())
    res.W_hat = torch.from_numpy(take(m * n, np.float32).reshape(m, n).copy())
    loss = float(take(1, np.float64)[0])
    assert o == len(buf)
    ref = oracle.quantize_layer(L.W0, L.X, L.Xhat, L.s, steps=steps, lr=lr)
    met = P.compare(res, ref)
    print(met, "loss", loss, ref.loss_final, flush=True)
    assert met["code_identity"] >= P.CODE_IDENTITY
    assert met["first_group_agreement"] >= P.CODE_IDENTITY
    assert met["group_param_agreement"] >= P.GROUP_AGREEMENT_AFTER_BGD
    assert abs(loss - ref.loss_final) <= P.LOSS_RTOL * abs(ref.loss_final)
