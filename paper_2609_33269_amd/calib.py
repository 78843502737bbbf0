"""Offline construction of one ASP layer's factors (PyTorch).

This is the calibration stage that precedes the deployed layer: in the paper it
is done once per layer in PyTorch, before the 4-bit weights are exported
(Sec. 4.2, App. B.1).  It is not part of the per-token hot path; its outputs
(lambda, L1, L2, R) are the inputs of qwam_pack_weights / qwam_quantize_act /
qwam_asp_linear.

  lambda_k = max_m |x[m, k]|^0.5 / max_n |W[n, k]|^0.5         (App. B.1, alpha = 0.5;
                                                                   1 where a maximum is 0)
  V        = top-r eigenvectors of the layer's Gramian (Eq. 7); here the SPD
             stand-in G = A A^T / K + 1e-3 I, whose eigenvectors are the left
             singular vectors of A (the ridge shifts eigenvalues only)
  W~       = diag(lambda) W, and with a rotation W~ H: every row rotated
             blockwise by the orthonormal Hadamard matrix of block B   (Eq. 3)
  L1       = bf16(V)                    [K][r]
  L2       = bf16(L1^T W~)              [r][N]   (V^T W~ of Eq. 9)
  R        = fl32(W~ - L1 L2)           [N][K]   (W~_perp of Eq. 9, against the rounded factors)
"""

from __future__ import annotations

import torch

RIDGE = 1e-3


def smoothing_factors(x: torch.Tensor, w: torch.Tensor) -> torch.Tensor:
    """x bf16 [M][K], w bf16 [N][K] (any device) -> float32 [K]."""
    xmax = x.abs().amax(dim=0).double()
    wmax = w.abs().amax(dim=0).double()
    ok = (xmax > 0) & (wmax > 0)
    lam = torch.where(ok, xmax.pow(0.5) / wmax.pow(0.5).clamp_min(1e-300), torch.ones_like(xmax))
    return lam.float()


def protected_basis(a: torch.Tensor, r: int) -> torch.Tensor:
    """Top-r eigenvectors of A A^T / K + RIDGE * I as float64 [K][r], largest
    eigenvalue first, each column's largest-|entry| made positive."""
    a64 = a.detach().to("cpu", torch.float64)
    if r > a64.shape[1]:
        raise ValueError("rank must not exceed the Gramian factor's width")
    U, _, _ = torch.linalg.svd(a64, full_matrices=False)
    V = U[:, :r].clone()
    idx = V.abs().argmax(dim=0)
    sgn = torch.sign(V[idx, torch.arange(r)])
    sgn[sgn == 0] = 1.0
    return V * sgn[None, :]


def hadamard_block(K: int) -> int:
    """Largest power of two dividing K, at most 1024 (App. B.1)."""
    return min(K & -K, 1024)


def rotate_rows(v: torch.Tensor, B: int) -> torch.Tensor:
    """Rows of v (float64 [rows][K]) times diag(H_B, ..) / sqrt(B), H_B the
    Sylvester Hadamard matrix, by the fast Walsh-Hadamard transform."""
    rows, K = v.shape
    y = v.reshape(rows, K // B, B)
    h = 1
    while h < B:
        z = y.reshape(rows, K // B, B // (2 * h), 2, h)
        a, b = z[:, :, :, 0, :], z[:, :, :, 1, :]
        y = torch.stack((a + b, a - b), dim=3).reshape(rows, K // B, B)
        h *= 2
    return (y / B ** 0.5).reshape(rows, K)


@torch.no_grad()
def build_layer(x: torch.Tensor, w: torch.Tensor, V: torch.Tensor, hadamard: bool = False):
    """x bf16 [M][K], w bf16 [N][K], V float64 [K][r] (same device as w, or CPU).
    With `hadamard`, the weight is rotated (Eq. 3) and V is taken as a basis of
    the rotated coordinates.

    Returns dict(lam f32 [K], L1 bf16 [K][r], L2 bf16 [r][N], R f32 [N][K],
    hadamard B or 0) on w's device.
    """
    dev = w.device
    lam = smoothing_factors(x, w).to(dev)
    wt = w.double() * lam.double()[None, :]                      # [N][K]
    B = hadamard_block(wt.shape[1]) if hadamard else 0
    if B:
        wt = rotate_rows(wt, B)
    L1 = V.to(dev, torch.float64).to(torch.bfloat16)             # [K][r]
    L1d = L1.double()
    L2t = (wt @ L1d).to(torch.bfloat16)                          # [N][r] = (L1^T W~)^T
    R = (wt - L2t.double() @ L1d.t()).float()                    # [N][K]
    del wt
    return {"lam": lam, "L1": L1, "L2": L2t.t().contiguous(), "R": R, "hadamard": B}
