"""Helpers shared by the GPU tests: device upload and oracle comparison."""
import sys

import numpy as np
import torch

from oracle import compare as cmp
from oracle import kbest_oracle as ko

TOL = {"f32": 1e-4, "bf16": 2e-2}   # absolute, in log space


def say(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(inp, dev="cuda"):
    if inp.dtype == "bf16":
        h = torch.from_numpy(np.ascontiguousarray(inp.h).view(np.int16)).view(torch.bfloat16).to(dev)
        W = torch.from_numpy(np.ascontiguousarray(inp.W).view(np.int16)).view(torch.bfloat16).to(dev)
    else:
        h = torch.from_numpy(np.ascontiguousarray(inp.h)).to(dev)
        W = torch.from_numpy(np.ascontiguousarray(inp.W)).to(dev)
    b = torch.from_numpy(np.ascontiguousarray(inp.b, dtype=np.float32)).to(dev)
    prev = torch.from_numpy(np.ascontiguousarray(inp.prev, dtype=np.float32)).to(dev)
    off = torch.from_numpy(np.ascontiguousarray(inp.off, dtype=np.int32)).to(dev)
    return h, W, b, prev, off


def run_step(kb, inp, dev="cuda", row_lse=False, ws=None):
    h, W, b, prev, off = to_dev(inp, dev)
    lse = torch.full((inp.N,), float("nan"), dtype=torch.float32, device=dev) if row_lse else None
    tok, par, sc = kb.kbest_step(h, W, b, prev, off, inp.k, row_lse=lse, ws=ws)
    torch.cuda.synchronize()
    res = (tok.cpu().numpy(), par.cpu().numpy(), sc.cpu().numpy())
    return res + ((lse.cpu().numpy(),) if row_lse else ())


def check(inp, dev_out, sentences=None, tol=None):
    """Oracle comparison with rules (i)-(iii); returns the report (asserting ok)."""
    tol = TOL[inp.dtype] if tol is None else tol
    if sentences is None:
        ref = ko.kbest_step(inp.h, inp.W, inp.b, inp.prev, inp.off, inp.k, dtype=inp.dtype)
        tok, par, sc = dev_out[:3]
    else:
        ref = ko.kbest_step_threshold(inp.h, inp.W, inp.b, inp.prev, inp.off, inp.k, dtype=inp.dtype,
                                      sentences=sentences)
        tok, par, sc = dev_out[:3]
    rs = cmp.make_rescorer(inp.h, inp.W, inp.b, inp.prev, inp.dtype, ref.lse)
    rep = cmp.compare_step(tok, par, sc, ref, inp.off, inp.V, tol, rescore=rs, sentences=sentences)
    assert rep.ok, f"{inp.name}: " + "; ".join(rep.errors)
    if len(dev_out) > 3:
        lse = dev_out[3]
        rows = np.isfinite(ref.lse)
        err = np.abs(lse[rows] - ref.lse[rows]).max()
        assert err <= tol, f"{inp.name}: row LSE error {err}"
    return rep, ref
