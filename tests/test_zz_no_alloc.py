"""lact_forward_noalloc (the entry point for callers that cannot allocate)
against lact_forward on the same inputs, through the C ABI: three calls in a
row, each smaller than the one before, so every call after the first runs on
the fixed scratch array as the previous call left it. The same kernels run on
the same values in both entry points, so the outputs agree bitwise."""
import numpy as np
import pytest
import torch

import paper_2505_23884_amd as P
from lact_synth import CONFIGS, make_inputs

pytestmark = pytest.mark.gpu

CASES = [
    # one LM sequence with Muon (116 MiB of the 128 MiB array; split gradient, per-product Newton-Schulz)
    CONFIGS["lm32k_muon"].with_(name="noalloc_lm_muon", B=1, H=4, n_kv=4096, n_q=4096),
    # gradient and update in one kind, ragged tiles, update-then-apply with a tail
    CONFIGS["lm32k"].with_(name="noalloc_fused", B=1, H=13, d=320, h=288, n_kv=700, n_q=760, chunk=256, order=1),
    # narrow tiles, a partial last chunk and a tail
    CONFIGS["lm32k"].with_(name="noalloc_small", B=1, H=2, d=128, h=256, n_kv=700, n_q=760, chunk=256),
]


def _on_device(cfg, x):
    sh = lambda a: np.ascontiguousarray(a.reshape(cfg.B, cfg.H, *a.shape[1:]))
    io = torch.bfloat16 if cfg.io == "bf16" else torch.float32
    dev = lambda a, dt: torch.from_numpy(sh(a)).to("cuda", dt)
    return (dev(x["q"], io), dev(x["k"], io), dev(x["v"], io), dev(x["eta"], torch.float32),
            [dev(x[w], torch.float32) for w in ("W1", "W2", "W3")])


def test_noalloc_matches_forward_on_successively_smaller_calls():
    sizes = []
    for i, cfg in enumerate(CASES):
        desc = P.binding.make_desc(cfg.B, cfg.H, cfg.d, cfg.h, cfg.n_kv, cfg.n_q, cfg.chunk, cfg.order, cfg.use_muon,
                                   cfg.ns_steps, P.IO_BF16)
        sizes.append(P.workspace_bytes(desc))
        assert sizes[-1] <= P.binding.NOALLOC_SCRATCH_BYTES
        print(f"[gpu] noalloc call {i}: {cfg.name} B={cfg.B} H={cfg.H} d={cfg.d} h={cfg.h} n_kv={cfg.n_kv} "
              f"n_q={cfg.n_q} chunk={cfg.chunk} muon={cfg.use_muon} scratch used {sizes[-1] / 2**20:.1f} MiB",
              flush=True)
        x = make_inputs(cfg, 100 + i)
        q, k, v, eta, W = _on_device(cfg, x)
        kw = dict(chunk=cfg.chunk, order=cfg.order, use_muon=bool(cfg.use_muon), ns_steps=cfg.ns_steps)
        W_ref = [w.clone() for w in W]
        o_ref = P.forward(q, k, v, eta, *W_ref, **kw)
        W_na = [w.clone() for w in W]
        o_na = torch.empty_like(q)
        torch.cuda.synchronize()
        before = torch.cuda.memory_stats().get("allocation.all.allocated", 0)
        P.forward_noalloc(q, k, v, eta, *W_na, out=o_na, **kw)
        torch.cuda.synchronize()
        assert torch.cuda.memory_stats().get("allocation.all.allocated", 0) == before
        diff = {"o": int((o_na != o_ref).sum())}
        diff.update({f"W{j + 1}": int((a != b).sum()) for j, (a, b) in enumerate(zip(W_na, W_ref))})
        print(f"[gpu] noalloc call {i}: differing elements {diff}", flush=True)
        assert all(n == 0 for n in diff.values()), diff
        assert bool(torch.isfinite(o_na.float()).all())
    assert sizes[0] > sizes[1] > sizes[2]
