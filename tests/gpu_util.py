"""Shared helpers of the GPU parity tests: run a stage through the C ABI on
seeded inputs and compare with the oracle."""

import sys

import numpy as np

from paper_2606_19163_amd import configs, synth
from paper_2606_19163_amd import stage as S


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def rel_l2(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    nb = np.linalg.norm(b.ravel())
    return np.linalg.norm((a - b).ravel()) / max(nb, 1e-300)


def tol_for(desc):
    return 1e-4 if desc["dtype"] == configs.F32 else 2e-2


def device_boundary(st, b):
    import torch
    out = {k: st.to_dev(v) for k, v in b.items()}
    return out


def run_gpu(desc, params, b, want_cache=True, mb=0):
    """Full F_enc, F_dec, B_dec, B_enc through the library.  With
    ``want_cache`` a second pass reads the skip activations and skip
    gradients out of the cache (take) before releasing the microbatch."""
    import torch
    st = S.Stage(desc)
    st.set_params(params)
    st.zero_grads()
    db = device_boundary(st, b)
    dtemb = torch.zeros((desc["batch"], desc["temb_dim"]), dtype=torch.float32, device="cuda")
    out = S.run_microbatch(st, mb, db, dtemb=dtemb)
    torch.cuda.synchronize()
    res = {k: v.float().cpu().numpy() for k, v in out.items()}
    res["dtemb"] = dtemb.cpu().numpy()
    res["grads"] = st.grads_dict()
    if want_cache:
        res["skips"], res["dskips"] = {}, {}
        st.forward(S.ENC, mb, db["x"], db["temb"])
        st.forward(S.DEC, mb, db["u"], db["temb"])
        st.backward(S.DEC, mb, db["g_dec"])
        for slot in st.slot_ch:
            res["skips"][slot] = st.take(mb, slot, S.SKIP_ACT).float().cpu().numpy()
            if st.state(mb, slot) & S.GRAD_PRESENT:
                res["dskips"][slot] = st.take(mb, slot, S.SKIP_GRAD).cpu().numpy()
        st.release(mb)
        torch.cuda.synchronize()
    return res, st


def compare(desc, gpu, ref, tol=None, grads=True, skip_rows=None, label="", log_all=False):
    """rel L2 per output; returns the dict of errors and asserts each <= tol.
    ``log_all`` prints every tensor's error, not only the worst."""
    tol = tol_for(desc) if tol is None else tol
    errs = {}
    sl = (slice(None) if skip_rows is None else skip_rows)
    for k in ("y_enc", "y_dec", "dx", "du", "dtemb"):
        errs[k] = rel_l2(gpu[k][sl], ref[k])
    if grads:
        for k, v in ref["grads"].items():
            errs["grad." + k] = rel_l2(gpu["grads"][k], v)
    for slot, v in ref.get("skips", {}).items():
        if slot in gpu.get("skips", {}):
            errs[f"skip{slot}"] = rel_l2(gpu["skips"][slot][sl], v)
    for slot, v in ref.get("dskips", {}).items():
        if slot in gpu.get("dskips", {}):
            errs[f"dskip{slot}"] = rel_l2(gpu["dskips"][slot][sl], v)
    worst = max(errs, key=errs.get)
    if log_all:
        for k in sorted(errs):
            log(f"  {label} {k} = {errs[k]:.3e}")
    log(f"  {label} worst {worst} = {errs[worst]:.3e} (tol {tol:g})")
    bad = {k: v for k, v in errs.items() if not (v <= tol)}
    assert not bad, bad
    return errs
