"""Shared set-up for the GPU tests: seeded inputs (from synth) on host and device."""
from __future__ import annotations

import numpy as np

import synth


def torch_mod():
    import torch
    return torch


def device_tensor(a: np.ndarray, dtype: str = "f32"):
    """Upload a float32 numpy array as float32 or bfloat16 (values must already be bf16-representable)."""
    torch = torch_mod()
    if dtype == "bf16":
        bits = synth.bf16_bits(a).view(np.int16)
        return torch.from_numpy(bits.copy()).to("cuda").view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda")


def make_inputs(n, k, q, r, s, seed, dtype="f32", integer=False, a_std=1.0):
    """(P, A, X) float64/float32 host arrays with device-dtype values."""
    if integer:
        P = synth.integer_parity_matrix(n, k, seed)
        A = synth.integers((q, r), seed, synth.STREAM_A)
        X = synth.integers((r, s), seed, synth.STREAM_X)
    else:
        P = synth.parity_matrix(n, k, seed, dtype=dtype)
        A = synth.gaussian((q, r), seed, synth.STREAM_A, std=a_std)
        X = synth.gaussian((r, s), seed, synth.STREAM_X)
        if dtype == "bf16":
            A = synth.bf16_round(A)
            X = synth.bf16_round(X)
    return P, A, X


def normwise_rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    """max over columns of ||got - ref||_inf / ||ref||_inf."""
    got = np.asarray(got, dtype=np.float64).reshape(ref.shape[0], -1)
    ref = np.asarray(ref, dtype=np.float64).reshape(ref.shape[0], -1)
    den = np.max(np.abs(ref), axis=0)
    den[den == 0] = 1.0
    return float(np.max(np.max(np.abs(got - ref), axis=0) / den))
