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
