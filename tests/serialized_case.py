"""The workload of test_gpu_serialized.py, importable by the test and runnable as a child process:
a layer sweep with Block-GD under a dense metric (residual, gradient, metric, Adam and lock GEMMs)
and a decoder block sweep at a shape that takes the LDS-staged attention kernels.  Run as a
script it writes its outputs to the .npz file named on the command line."""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

DECODER = dict(T=4096, d=512, f=768, n_heads=8, n_kv=2, head_dim=64, seq_len=256)


def run(rq, ctx):
    import torch
    import synth
    out = {}
    L = synth.make_module("single_512", m=256, n=384, T=2048)
    g = np.random.default_rng(5)
    A = g.standard_normal((256, 512))
    M = (A @ A.T / 512).astype(np.float32)
    dev = lambda a, bf16=False: (torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda().to(torch.bfloat16)
                                 if bf16 else torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda())
    r = rq.quantize_layer(ctx, dev(L.W0), dev(L.X, True), dev(L.Xhat, True), dev(L.s), dev(M), None,
                          qp=rq.qparams(), bgd=rq.bgd_params(steps=2, lr=1e-3))
    torch.cuda.synchronize()
    out["layer_codes"] = r.codes.cpu().numpy()
    out["layer_W_hat"] = r.W_hat.cpu().numpy()
    out["layer_loss"] = np.array([r.loss_final])
    print("[serialized-case] layer sweep done", flush=True)
    s = DECODER
    inp = synth.make_decoder_block(s["T"], s["d"], s["f"], s["n_heads"], s["n_kv"], s["head_dim"], s["seq_len"],
                                   seed=3, dense_F=True)
    blk = {k: (None if v is None else dev(v)) for k, v in inp.w.items()}
    res = rq.decoder_block_sweep(ctx, dev(inp.X, True), dev(inp.Xhat, True), blk, None, n_heads=inp.n_heads,
                                 n_kv=inp.n_kv, head_dim=inp.head_dim, seq_len=inp.seq_len, window=False,
                                 qp=rq.qparams(), bgd=rq.bgd_params(steps=1, lr=1e-5))
    torch.cuda.synchronize()
    for name, mod in res.modules.items():
        out[f"dec_{name}_codes"] = mod.codes.cpu().numpy()
        out[f"dec_{name}_W_hat"] = mod.W_hat.cpu().numpy()
    out["dec_loss"] = np.array([res.loss_final])
    print("[serialized-case] decoder sweep done", flush=True)
    return out


if __name__ == "__main__":
    import torch
    from paper_2609_00049_amd import realq as rq
    torch.cuda.set_device(0)
    c = rq.Context()
    np.savez(sys.argv[1], **run(rq, c))
    c.close()
