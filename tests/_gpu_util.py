"""Helpers shared by the GPU parity tests (device transfer, packing, comparisons)."""
import sys

import numpy as np

from oracle import formats as F
from oracle import resq as Q

Y_TOL = 1e-5  # normwise relative error bound for float32 outputs


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def dev_bf16(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()


def dev_f32(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def host(t):
    return t.cpu().numpy()


def host_scales(fmt, t):
    a = host(t)
    return a.view(np.uint32) if fmt == "hif4" else a.astype(np.uint8)


def assert_codes_equal(gpu_codes, oracle_codes, what=""):
    want = F.pack_nibbles(oracle_codes)
    got = host(gpu_codes)
    if not np.array_equal(got, want):
        bad = np.argwhere(got != want)
        raise AssertionError(f"{what}: {len(bad)} code bytes differ, first at {bad[:5].tolist()}")


def assert_scales_equal(fmt, gpu_scales, oracle_scales, what=""):
    got = host_scales(fmt, gpu_scales)
    want = np.asarray(oracle_scales).astype(got.dtype)
    if not np.array_equal(got, want):
        bad = np.argwhere(got != want)
        raise AssertionError(f"{what}: {len(bad)} scales differ, first at {bad[:5].tolist()}")


def normwise_err(got, want):
    want = np.asarray(want, dtype=np.float64)
    den = np.linalg.norm(want)
    return np.linalg.norm(np.asarray(got, dtype=np.float64) - want) / (den if den > 0 else 1.0)


def assert_close(got, want, what="", tol=Y_TOL):
    err = normwise_err(got, want)
    assert err <= tol, f"{what}: normwise relative error {err:.3e} > {tol:.0e}"
    return err


def pack_bits(mask):
    return Q.pack_bits(mask)
