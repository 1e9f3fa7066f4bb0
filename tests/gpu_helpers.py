"""Shared helpers for the GPU parity tests: run the HIP path through the C ABI and
the fp64 oracle on the same seeded inputs, and compare."""
from __future__ import annotations

import math
import sys

import numpy as np

import oracle as O
from paper_2602_04361_amd.synth import make_qkv

TOL = {"bf16": dict(max_abs=2e-2, mean_abs=2e-3), "f32": dict(max_abs=1e-5, mean_abs=1e-5)}
INF_SIDES = [1, 2, 4, 6, 8, 12, 16, 20, 24, 32, 40, 48, 64]


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def scale_of(d):
    return float(np.float32(1.0 / math.sqrt(d)))


def torch_dtype(name):
    import torch

    return torch.bfloat16 if name == "bf16" else torch.float32


def make_case(h, w, B, H, d, F, ns, seed, dtype):
    q, k, v = make_qkv(h, w, B, H, d, F, ns, seed=seed, bf16=(dtype == "bf16"))
    return q, k, v


def to_dev(x, dtype):
    import torch

    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(torch_dtype(dtype))


def csr_rows(row_ptr, col_idx, padded=False):
    """Rows of a CSR pair; with padded=True, drop the -1 entries that end each row
    (after checking that -1 only appears as trailing padding)."""
    rp = row_ptr.cpu().numpy().astype(np.int64)
    ci = col_idx.cpu().numpy().astype(np.int64)
    rows = [ci[rp[i]:rp[i + 1]].tolist() for i in range(len(rp) - 1)]
    if padded:
        out = []
        for r in rows:
            n = len(r) - (r[::-1].index(next(x for x in r[::-1] if x != -1)) if any(x != -1 for x in r) else len(r))
            assert all(x == -1 for x in r[n:]) and all(x != -1 for x in r[:n]), r
            out.append(r[:n])
        rows = out
    return rows


def assert_close(got, want, dtype, what):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite values"
    err = np.abs(got - want)
    tol = TOL[dtype]
    assert err.max() <= tol["max_abs"], f"{what}: max abs err {err.max():.3e} > {tol['max_abs']}"
    assert err.mean() <= tol["mean_abs"], f"{what}: mean abs err {err.mean():.3e} > {tol['mean_abs']}"
    return float(err.max()), float(err.mean())


def oracle_geometry(h, w, b, ns):
    return O.Geometry(h, w, b, ns)
