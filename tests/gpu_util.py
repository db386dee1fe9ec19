"""Helpers for the GPU parity tests: host <-> device copies, bf16 operands
built by the library's own conversion kernel, workspaces, error metrics."""
import sys

import numpy as np
import pytest
import torch

from paper_1912_06680_amd import o5

# Tolerances: relative error max|Y_gpu - Y_ref| / max|Y_ref| per output tensor.
TOL_F32 = 1e-4
TOL_BF16 = 3e-2


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def banner(msg):
    """Name the case before any GPU work, flushed, so a crash log names it."""
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def dev_f32(a):
    return dev(np.asarray(a, dtype=np.float32))


def dev_bf16(a):
    """Upload as fp32 and round on the device with o5_f32_to_bf16."""
    src = dev_f32(a)
    dst = torch.empty(src.shape, dtype=torch.bfloat16, device="cuda")
    o5.o5_f32_to_bf16(src.numel(), src, dst)
    return dst


def dev_dt(a, bf16):
    return dev_bf16(a) if bf16 else dev_f32(a)


def host(t):
    torch.cuda.synchronize()
    return t.detach().to(torch.float64).cpu().numpy() if t.dtype != torch.bfloat16 else \
        t.detach().float().to(torch.float64).cpu().numpy()


def empty_dt(shape, bf16):
    return torch.empty(shape, dtype=torch.bfloat16 if bf16 else torch.float32, device="cuda")


def workspace(nbytes):
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device="cuda")


def rel_err(gpu, ref):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    assert np.all(np.isfinite(gpu)), "non-finite GPU output"
    den = np.max(np.abs(ref))
    return float(np.max(np.abs(gpu - ref)) / (den if den > 0 else 1.0))


def assert_close(name, gpu, ref, tol):
    e = rel_err(gpu, ref)
    print(f"    {name}: rel_err={e:.3e} (tol {tol:g})", flush=True)
    assert e <= tol, f"{name}: rel_err {e:.3e} > {tol:g}"


def assert_close_both(name, gpu, ref, ref_plain, tol):
    """bf16 path: compare with the oracle that rounds where the device stores
    a bf16 operand (``ref``) and with the plain definition that rounds only
    the inputs (``ref_plain``); both at ``tol``, both printed."""
    e = rel_err(gpu, ref)
    e2 = rel_err(gpu, ref_plain)
    print(f"    {name}: rel_err={e:.3e} storage-point oracle, {e2:.3e} plain oracle (tol {tol:g})", flush=True)
    assert e <= tol, f"{name}: rel_err {e:.3e} > {tol:g} (storage-point oracle)"
    assert e2 <= tol, f"{name}: rel_err {e2:.3e} > {tol:g} (plain oracle)"


def tile_rows(B, tile=256):
    """One row inside every `tile`-row block of B rows (its middle, or the
    middle of the partial last block), plus the first and last row."""
    rows = {0, B - 1}
    for t0 in range(0, B, tile):
        rows.add(min(t0 + tile // 2, (t0 + B - 1) // 2 if t0 + tile > B else t0 + tile // 2))
    return sorted(rows)
