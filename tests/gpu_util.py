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


# Second bar of the bf16 fast-variant scores, one that a 10% error in the attention output
# fails.  The stated bar above is dominated by its relative term (|s| is about ln V), while
# a score depends on its row's attention output only through deviations of the logits of
# size sigma_z, the spread of z = W_lm u over the vocabulary (about 0.05 for rows that
# attend to thousands of keys): scaling u by 0.9 moves the score by 0.1 (z_x - E_P z),
# about 0.1 sigma_z.  The path rounds the probabilities P, the attention output y and
# u = W_o y to bf16 (unit roundoff 2^-8; random, so 2^-8 / sqrt(3) standard deviation per
# element) and accumulates in fp32, so u carries a random relative error of about 2^-8,
# the logits an error W_lm du of spread 2^-8 sigma_z, and the score
# sum_v P_v dz_v - dz_x of about sqrt(2) 2^-8 sigma_z = 0.0055 sigma_z (one standard
# deviation).  The bar is 6 of those, plus an absolute 2e-5 for the fp32 log-sum-exp over
# the vocabulary.  A 10% attention error exceeds it on about 3 rows in 4.
SPREAD_K, SPREAD_ATOL = 0.035, 2e-5

# Second bar of bf16 attention outputs, per element: |o - ref| <= 2^-8 |ref| +
# 2^-6 rms(ref) + 1e-6, rms over the head_dim outputs of the (row, head).  The output is
# rounded to bf16 (2^-8 |o|); the probabilities enter P V rounded to bf16, which moves each
# output by a random sum whose standard deviation is about 2^-8 / sqrt(3) times the row's
# scale, and 2^-6 is seven of those.  The stated tolerance (2e-2 + 1e-2 |ref|) cannot see a
# 10% error on rows that attend to thousands of keys, whose outputs are around 0.01.
ATT_REL, ATT_ROW, ATT_ATOL = 2.0 ** -8, 2.0 ** -6, 1e-6


def assert_scores_close(got: np.ndarray, ref: np.ndarray, dtype: str, what: str = "",
                        spread=None) -> dict:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    inf_ref = np.isinf(ref)
    assert np.array_equal(np.isinf(got), inf_ref), f"{what}: +inf entries differ"
    assert np.all(got[inf_ref] == ref[inf_ref]), f"{what}: infinite entries differ in sign"
    fin = ~inf_ref
    assert np.all(np.isfinite(got[fin])), f"{what}: non-finite score where the oracle is finite"
    # a surprisal -log P is never negative
    assert np.all(got[fin] >= 0), f"{what}: negative score {got[fin].min()}"
    err = np.abs(got[fin] - ref[fin])
    stats = {"max_abs": float(err.max(initial=0.0)),
             "max_rel": float((err / np.maximum(np.abs(ref[fin]), 1e-30)).max(initial=0.0))}
    if dtype == "bf16":
        bad = err > BF16_ATOL + BF16_RTOL * np.abs(ref[fin])
    else:
        bad = err > F32_ATOL
    assert not bad.any(), f"{what}: {int(bad.sum())} scores out of tolerance; {stats}"
    if spread is not None:
        sp = np.asarray(spread, dtype=np.float64)[fin]
        ratio = err / np.maximum(sp, 1e-30)
        stats["max_err_over_spread"] = float(ratio.max(initial=0.0))
        bad2 = err > SPREAD_K * sp + SPREAD_ATOL
        assert not bad2.any(), (f"{what}: {int(bad2.sum())} scores outside the spread bar "
                                f"({SPREAD_K} sigma_z + {SPREAD_ATOL}); {stats}")
    return stats


def spread_bar_failures(got: np.ndarray, ref: np.ndarray, spread: np.ndarray) -> int:
    """Finite rows whose score error exceeds the spread bar."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    fin = np.isfinite(ref)
    err = np.abs(got[fin] - ref[fin])
    return int((err > SPREAD_K * np.asarray(spread, dtype=np.float64)[fin] + SPREAD_ATOL).sum())


def attention_bar_failures(got: np.ndarray, ref: np.ndarray) -> int:
    """Elements of attention outputs [rows][Hq][d] outside the attention bar."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    rms = np.sqrt((ref ** 2).mean(axis=-1, keepdims=True))
    return int((np.abs(got - ref) > ATT_REL * np.abs(ref) + ATT_ROW * rms + ATT_ATOL).sum())


def assert_attention_close(got: np.ndarray, ref: np.ndarray, what: str = "") -> dict:
    """bf16 attention outputs: the stated tolerance and the per-row bar above."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    np.testing.assert_allclose(got, ref, rtol=1e-2, atol=2e-2)
    rms = np.sqrt((ref ** 2).mean(axis=-1, keepdims=True))
    err = np.abs(got - ref)
    stats = {"max_abs": float(err.max(initial=0.0)),
             "max_err_over_row_rms": float((err / np.maximum(rms, 1e-30)).max(initial=0.0))}
    n_bad = attention_bar_failures(got, ref)
    assert n_bad == 0, f"{what}: {n_bad} outputs outside the per-row bar; {stats}"
    return stats
