"""Helpers of the GPU tests: moving seeded inputs to the host and comparing
the library's outputs with the oracle under the stated tolerances."""
import sys

import numpy as np
import torch

import oracle

# Floored relative error bound of the method's parity (max over elements of
# |g - o| / max(|o|, 1e-3 * sum_k |w_k| |F_k|)).  float16 storage: one
# rounding of the output (2^-11) plus fp32 weights and accumulation, at most
# 10^3 (n + 2) 2^-24 once floored, about 1.1e-3 for n = 8 entries.
TOL = {"bf16": 1e-2, "f16": 2e-3, "f32": 1e-5}


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_host_bits(t: torch.Tensor) -> np.ndarray:
    """Exact host copy of a device tensor's storage: uint16 patterns for
    bfloat16 and float16, float32 values for float32."""
    t = t.detach().contiguous()
    if t.dtype in (torch.bfloat16, torch.float16):
        return t.view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1)
    if t.dtype == torch.float32:
        return t.cpu().numpy().reshape(-1)
    raise TypeError(t.dtype)


def decode(host, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return oracle.bf16_to_f64(host)
    if dtype == "f16":
        return oracle.f16_to_f64(host)
    return np.asarray(host, dtype=np.float64)


def oracle_combine(host_entries, w, dtype: str):
    if dtype == "bf16":
        return oracle.extrapolate_bf16(host_entries, w)
    if dtype == "f16":
        return oracle.extrapolate_f16(host_entries, w)
    return oracle.extrapolate_f32(host_entries, w)


def check_parity(got_host, host_entries, w_oracle, dtype: str, label=""):
    """Compare a device result (host copy) with the oracle on the same inputs."""
    expect, mag = oracle_combine(host_entries, w_oracle, dtype)
    got = decode(got_host, dtype)
    e, unfl, normwise, frac = oracle.parity_error(got, expect, mag)
    assert np.all(np.isfinite(got)), f"{label}: non-finite output"
    assert e <= TOL[dtype], (f"{label}: floored error {e:.3e} > {TOL[dtype]:.0e} "
                             f"(normwise {normwise:.2e}, floored fraction {frac:.2e})")
    return e, normwise
