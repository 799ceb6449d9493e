"""Helpers shared by the GPU parity tests (host-side comparison logic only)."""
from __future__ import annotations

import numpy as np
import torch

from oracle import cs_oracle as o

FP32_REL_TOL = 1e-5    # |y_gpu - y_ref| <= 1e-5 * sum_i |w_i x_i| per output


def dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t: torch.Tensor) -> np.ndarray:
    torch.cuda.synchronize()
    return t.cpu().numpy()


def assert_f32_close(y: np.ndarray, ref: np.ndarray, S: np.ndarray, what: str = "") -> None:
    """Per-output bound 1e-5 * S; S == 0 requires an exact zero."""
    y = y.astype(np.float64)
    err = np.abs(y - ref)
    bound = FP32_REL_TOL * S
    bad = err > bound
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {bad.sum()} outputs out of tolerance, first at {tuple(i)}: "
                             f"gpu={y[tuple(i)]!r} ref={ref[tuple(i)]!r} S={S[tuple(i)]!r}")


def pool_S(S: np.ndarray) -> np.ndarray:
    """Tolerance scale of a 2x2 max-pooled output: the largest scale in the window."""
    return o.maxpool2x2_nhwc(S)


def check_kwta_f32(acc_gpu: np.ndarray, out_gpu: np.ndarray, ref_acc: np.ndarray,
                   S: np.ndarray, k: int) -> int:
    """k-WTA parity for fp32 (several answers can be right at a near-tie).

    (1) the GPU's mask must be exactly the top-k (lower-index ties) of the
        GPU's own sums, and winners keep their value bit for bit;
    (2) an element may be in one winner set and not the other only if its
        oracle value is within tolerance of the oracle's k-th largest value.
    Returns the number of such near-tie rows.
    """
    c = acc_gpu.shape[-1]
    a = acc_gpu.reshape(-1, c)
    og = out_gpu.reshape(-1, c)
    win_gpu = o.kwta_winners(a, k)
    exp_out = np.where(win_gpu, a, np.float32(0))
    assert np.array_equal(og, exp_out), "GPU k-WTA is not the exact top-k of its own sums"
    ra = ref_acc.reshape(-1, c)
    rS = S.reshape(-1, c)
    win_ref = o.kwta_winners(ra, k)
    diff = np.nonzero((win_gpu != win_ref).any(axis=1))[0]
    for r in diff:
        order = np.argsort(-ra[r], kind="stable")
        if k == 0 or k == c:
            raise AssertionError("winner sets cannot differ for k in {0, c}")
        ik = order[k - 1]                       # the oracle's k-th largest
        for i in np.nonzero(win_gpu[r] != win_ref[r])[0]:
            gap = abs(ra[r, i] - ra[r, ik])
            tol = FP32_REL_TOL * (rS[r, i] + rS[r, ik])
            assert gap <= tol, f"row {r}: element {i} swapped but its gap {gap} to the k-th > {tol}"
    return len(diff)
