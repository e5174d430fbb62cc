"""Shared helpers of the GPU parity tests (imported by tests marked `gpu` only)."""
import sys

import numpy as np


def say(*a):
    """Name the case before a GPU step (flushed, so a lost box still shows it)."""
    print("[gpu-case]", *a, flush=True)
    sys.stdout.flush()


def rel_inf(y, ref):
    """Normwise relative error ||y - ref||_inf / ||ref||_inf (complex: modulus)."""
    y = np.asarray(y, np.complex128 if np.iscomplexobj(ref) or np.iscomplexobj(y) else np.float64)
    ref = np.asarray(ref, y.dtype)
    den = np.abs(ref).max()
    return float(np.abs(y - ref).max() / (den if den > 0 else 1.0))


def oracle_model(case):
    return {"kind": case.kind, **case.params}


def masks_to_bool(words, H):
    """[B, T, W] uint32/int32 words -> [B, T, H] bool (bit j of word j // 32)."""
    w = np.asarray(words).astype(np.int64) & 0xFFFFFFFF
    B, T, W = w.shape
    bits = ((w[..., :, None] >> np.arange(32)) & 1).reshape(B, T, W * 32)
    return bits[..., :H].astype(bool)


def tie_band_check(got, u, rel, what):
    """GPU ReLU decisions `got` against the float64 pre-activations `u`: equal wherever
    |u| > rel max|u|; inside that band the decisions may differ (the two sides round
    differently), but at most max(2, 1e-4 of all decisions) of them.  Returns the in-band
    mismatch count."""
    u = np.asarray(u)
    scale = max(float(np.abs(u).max()), 1e-30)
    far = np.abs(u) > rel * scale
    ref = u > 0
    assert np.array_equal(got[far], ref[far]), what
    nin = int((got[~far] != ref[~far]).sum())
    print(f"[gpu-case] {what}: {int((~far).sum())} in-band decisions of {far.size}, {nin} differ", flush=True)
    assert nin <= max(2, int(1e-4 * far.size)), (what, nin)
    return nin
