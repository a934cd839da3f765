"""Helpers shared by the GPU parity tests: host copies for the oracle and the tolerance
checks.  Nothing here computes any part of the method."""
import math

import numpy as np
import torch

# Attention: bf16 inputs, fp32 accumulation -> per row max|diff| <= 2e-2 and
# ||diff||_2 / ||ref||_2 <= 1e-2 against the fp64 oracle.
ATTN_ABS = 2e-2
ATTN_REL = 1e-2
# Score: fp32 logits / exp / sums against fp64: |diff| <= 1e-4 * max(|ref|, 1/N_b).
SCORE_REL = 1e-4


def bits(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor (any device) -> host uint16 bit patterns."""
    return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().cpu().numpy()


def check_attention(out_rows: np.ndarray, ref_rows: np.ndarray, label: str = ""):
    """out_rows / ref_rows: float [R, d].  Raises with the worst row on failure."""
    diff = np.abs(out_rows.astype(np.float64) - ref_rows)
    row_max = diff.max(axis=1)
    ref_norm = np.linalg.norm(ref_rows, axis=1)
    row_rel = np.linalg.norm(out_rows.astype(np.float64) - ref_rows, axis=1) / np.maximum(ref_norm, 1e-30)
    bad = np.nonzero((row_max > ATTN_ABS) | (row_rel > ATTN_REL))[0]
    if len(bad):
        r = bad[0]
        raise AssertionError(f"{label}: {len(bad)} of {len(row_max)} rows out of tolerance; row {r}: "
                             f"max|d|={row_max[r]:.3e} rel={row_rel[r]:.3e}")
    return float(row_max.max()), float(row_rel.max())


def gpu_rows(out: torch.Tensor, rows: np.ndarray) -> np.ndarray:
    """Gather (b, t, h) rows of a bf16 [B, T, H, d] output as float64 [R, d]."""
    o = out.float().cpu().numpy()
    return o[rows[:, 0], rows[:, 1], rows[:, 2]].astype(np.float64)


def check_score(gpu: np.ndarray, ref: np.ndarray, n: int, label: str = ""):
    tol = SCORE_REL * np.maximum(np.abs(ref.astype(np.float64)), 1.0 / max(n, 1))
    d = np.abs(gpu.astype(np.float64) - ref.astype(np.float64))
    bad = np.nonzero(d > tol)[0]
    if len(bad):
        i = bad[0]
        raise AssertionError(f"{label}: {len(bad)} of {n} scores out of tolerance; pos {i}: "
                             f"gpu={gpu[i]!r} ref={ref[i]!r}")


def scale_of(d: int) -> float:
    return 1.0 / math.sqrt(d)
