"""Shared helpers of the GPU tests: move inputs to the device, run the
library through its C-ABI binding, bring results back, compare."""
import sys

import numpy as np

import paper_2509_02197_amd as adst

NP_DTYPE = {adst.ADST_F64: np.float64, adst.ADST_F32: np.float32}
TOL = {adst.ADST_F64: 1e-12, adst.ADST_F32: 1e-5}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (nb if nb > 0 else 1.0))


def dev(a):
    import torch
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    import torch
    if t is None:
        return None
    if torch.is_tensor(t):
        return t.detach().cpu().numpy()
    return t


def gpu_vjp(kind, inp, steps, loss, budget=None, sched=adst.ADST_SCHED_AUTO, want_dK=False,
            flags=0, params=None, ws=None, keep_ws=False, want_xT=True, want_dparams=False,
            lim=None):
    import torch
    out = adst.vjp(kind, dev(inp["x0"]), dev(inp.get("K")), steps, loss, dev(inp.get("aux")),
                   budget, sched, want_dK, params, flags, ws=ws, want_xT=want_xT,
                   want_dparams=want_dparams, lim=lim)
    torch.cuda.synchronize()
    res = {k: host(v) for k, v in out.items() if k not in ("ws", "info")}
    res["loss"] = float(res["loss"])
    res["info"] = out["info"].as_dict()
    if keep_ws:
        res["ws"] = out["ws"]
    return res
