"""Helpers for the GPU parity tests: device tensors from numpy, error
reports (L2, infinity norm, max-abs-relative) against the float64 oracle."""
import sys

import numpy as np
import pytest


def torch_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def dev(torch, a, dtype=None):
    a = np.ascontiguousarray(a)
    if dtype is None:
        dtype = torch.int32 if a.dtype.kind in "iu" else torch.float32
    if dtype == torch.float32:
        a = a.astype(np.float32)
    elif dtype == torch.int32:
        a = a.astype(np.int32)
    return torch.from_numpy(a).to("cuda")


def host(t):
    import torch
    torch.cuda.synchronize()
    return t.detach().cpu().numpy().astype(np.float64)


def err_report(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    d = got - ref
    scale = max(float(np.abs(ref).max()), 1e-30)
    return dict(maxabs_rel=float(np.abs(d).max()) / scale,
                l2_rel=float(np.linalg.norm(d)) / max(float(np.linalg.norm(ref)), 1e-30),
                inf=float(np.abs(d).max()), scale=scale)


def assert_close_maxabs(got, ref, tol, what="", scale=None):
    """|got - ref| <= tol * max|ref| element-wise (the bar used for every
    floating-point tensor).  `scale` overrides max|ref| where the reference
    is identically zero in exact arithmetic (then its natural magnitude is
    the scale of the inputs that cancel)."""
    r = err_report(got, ref)
    if scale is not None:
        r["maxabs_rel"] = r["inf"] / scale
    print(f"[parity] {what}: maxabs_rel={r['maxabs_rel']:.3e} l2_rel={r['l2_rel']:.3e}", file=sys.stderr)
    assert np.isfinite(np.asarray(got)).all(), f"{what}: non-finite values"
    assert r["maxabs_rel"] <= tol, f"{what}: max-abs-relative error {r['maxabs_rel']:.3e} > {tol:.1e}"
    return r


def say(msg):
    print(msg, file=sys.stderr, flush=True)


def progress(msg):
    """A progress line of a long test: to stderr, and appended to the file
    named by BT_PROGRESS_LOG when it is set (pytest holds the test's own
    output until it ends, so a file shows how far a long run got)."""
    import os
    say(msg)
    path = os.environ.get("BT_PROGRESS_LOG")
    if not path:
        return
    try:
        os.makedirs(os.path.dirname(os.path.abspath(path)), exist_ok=True)
        with open(path, "a") as f:
            f.write(msg + "\n")
    except OSError:
        pass
