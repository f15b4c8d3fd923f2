"""The C ABI: the built library loads and exports every entry point the header declares.

No compute call is made here (this runs without a GPU).
"""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "realq.h")
LIB = os.path.join(ROOT, "paper_2609_00049_amd", "librealq.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(realq_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_five_sweep_calls():
    names = declared_functions()
    for f in ["realq_hessian_accum", "realq_chol_inverse", "realq_quantize_block", "realq_bgd_step",
              "realq_quantize_layer"]:
        assert f in names


def test_header_compiles_as_c_and_cxx(tmp_path):
    for compiler, ext in (("gcc", "c"), ("g++", "cpp")):
        src = tmp_path / f"t.{ext}"
        src.write_text('#include "realq.h"\nint main(void){ realq_qparams q; realq_qparams_default(&q); return 0; }\n')
        r = subprocess.run([compiler, "-fsyntax-only", "-Wall", "-Werror", f"-I{os.path.dirname(HEADER)}", str(src)],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr


def test_binding_structs_match_the_c_layout(tmp_path):
    """sizeof and field offsets of the parameter, descriptor and output structs as the C compiler
    lays them out, against the ctypes mirrors of the binding."""
    from paper_2609_00049_amd import realq
    structs = {"realq_qparams": realq.QParams, "realq_bgd_params": realq.BgdParams,
               "realq_layer_desc": realq.LayerDesc, "realq_layer_out": realq.LayerOut,
               "realq_mlp_block": realq.MLPBlock, "realq_mlp_desc": realq.MLPDesc, "realq_mlp_out": realq.MLPOut,
               "realq_decoder_block": realq.DecoderBlock, "realq_decoder_desc": realq.DecoderDesc,
               "realq_decoder_out": realq.DecoderOut, "realq_decoder_fwd_out": realq.DecoderFwdOut}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "realq.h"', 'int main(void) {']
    for cname, py in structs.items():
        lines.append(f'printf("{cname} size %zu\\n", sizeof({cname}));')
        for fname, _ in py._fields_:
            lines.append(f'printf("{cname} {fname} %zu\\n", offsetof({cname}, {fname}));')
    lines += ['return 0;', '}']
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    r = subprocess.run(["gcc", "-Wall", "-Werror", f"-I{os.path.dirname(HEADER)}", str(src), "-o", str(exe)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l.strip()}
    for cname, py in structs.items():
        assert got[(cname, "size")] == ctypes.sizeof(py), cname
        for fname, _ in py._fields_:
            assert got[(cname, fname)] == getattr(py, fname).offset, (cname, fname)


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(LIB)
    missing = [f for f in declared_functions() if not hasattr(lib, f)]
    assert not missing, missing


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_binding_signatures_cover_the_header():
    from paper_2609_00049_amd import realq
    assert sorted(realq.EXPORTS) == declared_functions()


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_defaults_and_host_side_errors_without_gpu():
    """Calls that touch no device memory: defaults, NULL-argument validation."""
    from paper_2609_00049_amd import realq
    lib = realq.lib()
    q = realq.QParams()
    lib.realq_qparams_default(ctypes.byref(q))
    assert (q.bits, q.group, q.block, q.grid) == (4, 128, 128, 80) and abs(q.damp - 0.01) < 1e-9
    b = realq.BgdParams()
    lib.realq_bgd_params_default(ctypes.byref(b))
    assert b.form == realq.BGD_TOKENS
    assert (b.beta1, b.beta2) == (pytest.approx(0.9), pytest.approx(0.999)) and b.eps == pytest.approx(1e-8)
    assert lib.realq_ctx_create(None, None) == -1
    assert lib.realq_hessian_accum(None, None, None, 0, 0, None) == -1
    assert lib.realq_quantize_layer(None, None, None) == -1


def test_plain_c_caller_compiles_and_links(tmp_path):
    """tests/c_caller/realq_layer_c.c uses the header and the library from C11 with the HIP runtime's C
    API only (no C++, no PyTorch); it must compile warning-free and link."""
    from tests.c_caller import compile_c_caller
    r = compile_c_caller(tmp_path / "realq_layer_c")
    assert r.returncode == 0, r.stderr


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_binding_rejects_wrong_dtypes_and_shapes_before_the_call():
    """The binding checks the dtype and exact shape of every tensor it hands to the C ABI (which
    reads each buffer with the layout the sizes imply) and raises ValueError before any call; the
    checks come before the device check, so they run here on host tensors."""
    import torch
    from paper_2609_00049_amd import realq as rq

    class NoCall:           # stands in for a Context: any call into the library fails the test
        h = None

        def check(self, rc):
            raise AssertionError("the C ABI was called")

    ctx = NoCall()
    m, n, T = 8, 16, 32
    W0 = torch.zeros((m, n), dtype=torch.float32)
    X = torch.zeros((T, n), dtype=torch.bfloat16)
    cases = [
        dict(W0=W0.to(torch.bfloat16), X=X, Xhat=X),                         # bf16 weights
        dict(W0=W0, X=X.float(), Xhat=X),                                     # float32 activations
        dict(W0=W0, X=X, Xhat=X[:, :8].contiguous()),                         # Xhat narrower than X
        dict(W0=W0, X=X, Xhat=X, s=torch.ones(T - 1)),                        # short s
        dict(W0=W0, X=X, Xhat=X, M=torch.eye(m + 1)),                         # wrong metric size
        dict(W0=W0, X=X, Xhat=X, P=torch.eye(m, dtype=torch.float64)),        # float64 partner metric
    ]
    for kw in cases:
        with pytest.raises(ValueError):
            rq.quantize_layer(ctx, **kw)
    with pytest.raises(ValueError):
        rq.hessian_accum(ctx, X, None, torch.zeros((n, n), dtype=torch.float32))
    with pytest.raises(ValueError):
        rq.chol_inverse(ctx, torch.zeros((n, n), dtype=torch.float64), T, 0.01, torch.zeros((n, n + 1)))
    with pytest.raises(ValueError):
        rq.handoff(ctx, W0, X, torch.zeros((T, m), dtype=torch.float32))
    with pytest.raises(ValueError):
        rq.mlp_block_sweep(ctx, X, X, torch.ones(n), torch.zeros((24, n)), torch.zeros((24, n)),
                           torch.zeros((24, n)))                             # Wd must be [d, f]
