"""Shared helpers of the GPU tests (no arithmetic of the method)."""
import numpy as np
import torch

from synth import gen

# Score tolerance of the bf16 path: |gpu - ref| <= ATOL + RTOL * |ref| (the stated
# parity bar); the fp32 path must agree within F32_ATOL absolutely.
BF16_ATOL, BF16_RTOL = 2e-2, 1e-2
F32_ATOL = 1e-5


def bf16_host(t: torch.Tensor) -> np.ndarray:
    """bf16 device tensor -> uint16 bit patterns on the host."""
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def f64(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return gen.bf16_to_f64(bf16_host(t))
    return t.detach().cpu().double().numpy()


def dev(a: np.ndarray, device="cuda") -> torch.Tensor:
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def assert_scores_close(got: np.ndarray, ref: np.ndarray, dtype: str, what: str = "") -> dict:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    inf_ref = np.isinf(ref)
    assert np.array_equal(np.isinf(got), inf_ref), f"{what}: +inf entries differ"
    assert np.all(got[inf_ref] == ref[inf_ref]), f"{what}: infinite entries differ in sign"
    fin = ~inf_ref
    assert np.all(np.isfinite(got[fin])), f"{what}: non-finite score where the oracle is finite"
    err = np.abs(got[fin] - ref[fin])
    stats = {"max_abs": float(err.max(initial=0.0)),
             "max_rel": float((err / np.maximum(np.abs(ref[fin]), 1e-30)).max(initial=0.0))}
    if dtype == "bf16":
        bad = err > BF16_ATOL + BF16_RTOL * np.abs(ref[fin])
    else:
        bad = err > F32_ATOL
    assert not bad.any(), f"{what}: {int(bad.sum())} scores out of tolerance; {stats}"
    return stats
