"""Helpers shared by the GPU parity tests (not a test module)."""

import numpy as np
import torch

ATOL, RTOL, NORMWISE = 2e-2, 1e-2, 1e-2


def dev_bf16(a):
    """float32 array already on the bf16 grid -> bf16 device tensor (exact)."""
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda", torch.bfloat16)


def dev_f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda")


def dev_i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to("cuda")


def host(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def assert_close(got, want, what="", atol=ATOL, rtol=RTOL, normwise=NORMWISE):
    """Element-wise |got - want| <= atol + rtol |want| and normwise relative
    error <= normwise (the parity bar for floating-point outputs)."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = np.abs(got - want)
    bad = err > atol + rtol * np.abs(want)
    if bad.any():
        idx = np.unravel_index(np.argmax(err - (atol + rtol * np.abs(want))), err.shape)
        raise AssertionError(f"{what}: {bad.sum()} elements out of tolerance; worst at {idx}: "
                             f"got {got[idx]!r} want {want[idx]!r}")
    denom = np.linalg.norm(want)
    if denom > 0:
        rel = np.linalg.norm(got - want) / denom
        assert rel <= normwise, f"{what}: normwise relative error {rel:.3g} > {normwise}"
    return float(err.max()) if err.size else 0.0


def tile_rows(off, seed, block=128):
    """One random row of every `block`-row block of every request, plus the
    request's first and last row, sorted."""
    rng = np.random.default_rng(seed)
    rows = []
    for r in range(len(off) - 1):
        a, b = int(off[r]), int(off[r + 1])
        if b == a:
            continue
        starts = np.arange(a, b, block)
        ends = np.minimum(starts + block, b)
        rows.extend(rng.integers(starts, ends).tolist())
        rows.extend([a, b - 1])
    return np.array(sorted(set(rows)), dtype=np.int64)
