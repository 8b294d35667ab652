"""Helpers of the GPU tests: move a workload to the device, call the library
through its binding, and compare every output bit-exactly with the oracle."""
import numpy as np
import torch

import oracle
import paper_2608_03447_amd as asd


def device_logits(logits, dev):
    if logits.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(logits).view(np.int16)).to(dev).view(
            torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(logits)).to(dev)


def gpu_verify(logits, draft, lens, tau, cap, budget, row_offsets=None, dev="cuda:0",
               workspace=None, stream=None, flags=None):
    """One asd_verify call (asd_verify_ex when ``flags`` is given); returns
    numpy outputs (budget = updated ledger)."""
    dev = torch.device(dev)
    n = len(lens)
    rows = logits.shape[0]
    tl = device_logits(logits, dev)
    td = torch.from_numpy(np.ascontiguousarray(draft, dtype=np.int32)).to(dev)
    tk = torch.from_numpy(np.ascontiguousarray(lens, dtype=np.int32)).to(dev)
    tt = torch.from_numpy(np.array(np.broadcast_to(np.asarray(tau, np.float32), (n,)))).to(dev)
    tc = torch.from_numpy(np.array(np.broadcast_to(np.asarray(cap, np.int32), (n,)))).to(dev)
    tb = torch.from_numpy(np.array(budget, dtype=np.float32).reshape(n, 2)).to(dev)
    to = None if row_offsets is None else torch.from_numpy(
        np.ascontiguousarray(row_offsets, dtype=np.int64)).to(dev)
    amax = torch.full((rows,), -7, dtype=torch.int32, device=dev)
    regret = torch.full((rows,), float("nan"), dtype=torch.float32, device=dev)
    if flags is not None:
        acc, nxt = asd.asd_verify_ex(tl, td, tk, tt, tc, tb, flags=flags, workspace=workspace,
                                     row_offsets=to, out_argmax=amax, out_regret=regret)
    elif workspace is None:
        acc, nxt = asd.asd_verify(tl, td, tk, tt, tc, tb, row_offsets=to, out_argmax=amax,
                                  out_regret=regret)
    else:
        acc, nxt = asd.asd_verify_ws(tl, td, tk, tt, tc, tb, workspace, row_offsets=to,
                                     out_argmax=amax, out_regret=regret)
    torch.cuda.synchronize(dev)
    return {"accept_len": acc.cpu().numpy(), "next_token": nxt.cpu().numpy(),
            "argmax": amax.cpu().numpy(), "regret": regret.cpu().numpy(),
            "budget": tb.cpu().numpy()}


def oracle_verify(logits, draft, lens, tau, cap, budget, row_offsets=None, raw_gate=False):
    return oracle.verify(logits, draft, lens, tau, cap, budget, row_offsets, raw_gate=raw_gate)


def mismatches(gpu, ref):
    """Names of outputs that differ in any bit (regret rows the oracle leaves
    unwritten hold NaN on both sides and are compared as such)."""
    bad = []
    for k in ("accept_len", "next_token", "argmax"):
        if not np.array_equal(gpu[k], ref[k]):
            bad.append(k)
    if not np.array_equal(gpu["regret"].view(np.uint32), ref["regret"].view(np.uint32)):
        g, r = gpu["regret"], ref["regret"]
        both_nan = np.isnan(g) & np.isnan(r)
        if not np.array_equal(g.view(np.uint32)[~both_nan], r.view(np.uint32)[~both_nan]):
            bad.append("regret")
    if not np.array_equal(gpu["budget"].view(np.uint32), ref["budget"].view(np.uint32)):
        bad.append("budget")
    return bad


def describe(gpu, ref, limit=5):
    lines = []
    for k in ("accept_len", "next_token", "argmax"):
        idx = np.flatnonzero(gpu[k] != ref[k])[:limit]
        if idx.size:
            lines.append("%s at %s: gpu %s oracle %s" % (k, idx.tolist(), gpu[k][idx].tolist(),
                                                         ref[k][idx].tolist()))
    gb, rb = gpu["regret"].view(np.uint32), ref["regret"].view(np.uint32)
    idx = np.flatnonzero(gb != rb)[:limit]
    if idx.size:
        lines.append("regret at %s: gpu %s oracle %s" % (idx.tolist(), gpu["regret"][idx].tolist(),
                                                         ref["regret"][idx].tolist()))
    return "; ".join(lines)
