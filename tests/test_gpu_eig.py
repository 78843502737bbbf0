"""GPU parity of the protected-subspace eigensolve (Sec. 4.2, Eq. 7; the
procedure of the probe estimator; Prop. of App. A.3) through the C ABI,
against the oracle's eigendecomposition (numpy eigh, float64) of the same
G~ = scale H diag(lam) A diag(lam) H.

The eigenvectors are unique up to sign only where the eigenvalues are
separated, so the comparisons are: the subspace overlap ||V^T V_ref||_F^2 / r
(the paper's calibration-overlap metric), the Ky Fan identity
tr(V^T G~ V) = sum of the top-r eigenvalues, the eigenvalues themselves, the
orthonormality of V, single eigenvectors where their eigenvalue is isolated,
and the sign convention (largest-magnitude entry positive).
"""

import numpy as np
import pytest
import torch

from oracle import qwam_oracle as O
from paper_2609_33269_amd import qwam as Q

from parity_helpers import bf16_dev, f32_dev, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    Q.lib()


def _check_basis(V, ev, G, r, overlap_tol=1e-6, ev_tol=1e-5, vec_tol=1e-5):
    """V float [d][r], ev float [r] from the GPU against eigh of G (float64)."""
    V = V.astype(np.float64)
    ev = ev.astype(np.float64)
    Vr, evr = O.protected_basis_eigh(G, r)
    top = evr[:r]
    overlap = float(np.linalg.norm(V.T @ Vr) ** 2 / r)
    kyfan = float(np.trace(V.T @ G @ V))
    orth = float(np.abs(V.T @ V - np.eye(r)).max())
    log(f"    overlap 1 - {1 - overlap:.2e}, Ky Fan rel {abs(kyfan - top.sum()) / top.sum():.2e}, "
        f"eigenvalue rel {np.abs(ev - top).max() / top[0]:.2e}, orthonormality {orth:.2e}")
    assert overlap >= 1 - overlap_tol
    assert abs(kyfan - top.sum()) <= 1e-6 * top.sum()
    assert np.abs(ev - top).max() <= ev_tol * top[0]
    assert (np.diff(ev) <= 0).all(), "eigenvalues descending"
    assert orth <= 1e-5
    # isolated eigenvalues: the eigenvector itself, with the oracle's sign
    gaps = np.minimum(np.abs(np.diff(evr[:r + 1], prepend=np.inf))[:r], np.abs(np.diff(evr[:r + 1]))[:r])
    for i in range(r):
        if gaps[i] > 1e-3 * top[0]:
            c = float(V[:, i] @ Vr[:, i])
            assert abs(c) >= 1 - vec_tol, (i, c)
            srt = np.sort(np.abs(Vr[:, i]))
            if srt[-1] - srt[-2] > 1e-4 * srt[-1]:       # the largest entry is unambiguous
                assert c > 0, f"sign of eigenvector {i}"
    # the sign convention on the GPU's own vectors
    idx = np.argmax(np.abs(V), axis=0)
    assert (V[idx, np.arange(r)] > 0).all()


def _stand_in(d, width=64, seed=0):
    a = np.random.default_rng(seed).standard_normal((d, width))
    return O.gramian(a)


def _run(A64, r, iters, scale=1.0, lam=None, B=0):
    A = f32_dev(A64)
    lam_d = None if lam is None else f32_dev(lam)
    V, ev = Q.aog_protected_basis(A, r, iters=iters, scale=scale, lam=lam_d, hadamard=B)
    torch.cuda.synchronize()
    return V.cpu().numpy(), ev.cpu().numpy()


@pytest.mark.parametrize("d,r", [(4096, 32), (3072, 16), (1024, 48), (128, 16)])
def test_stand_in_gramian(d, r):
    """G = A A^T / K + 1e-3 I (the seeded stand-in of the calibration), on the
    GPU as float32; the reference is eigh of the same float32 values."""
    log(f"  eigensolve stand-in Gramian d={d} r={r}")
    G = _stand_in(d, seed=d + r).astype(np.float32).astype(np.float64)
    V, ev = _run(G, r, iters=8)
    _check_basis(V, ev, G, r)


def test_rotated_aog_from_accumulated_probes():
    """The whole procedure: probe VJPs accumulated by qwam_aog_accumulate
    (A += g g^T), then G~ = H diag(lam) (A / (N P)) diag(lam) H and its top
    eigenvectors, against the oracle's aog_accumulate, aog_estimate,
    rotated_aog and eigh."""
    d, n, r, B = 3072, 512, 32, 1024
    rng = np.random.default_rng(77)
    basis = rng.standard_normal((d, 48)) * np.exp(-np.arange(48) / 12.0)[None, :]
    g = basis @ rng.standard_normal((48, n)) + 0.05 * rng.standard_normal((d, n))
    g_bits = O.f64_to_bf16_bits(g)
    lam = np.exp(rng.uniform(-1.0, 1.0, size=d)).astype(np.float32)
    A = torch.zeros((d, d), dtype=torch.float32, device="cuda:0")
    Q.aog_accumulate(bf16_dev(g_bits), A)
    V, ev = Q.aog_protected_basis(A, r, iters=12, scale=1.0 / n, lam=f32_dev(lam), hadamard=B)
    torch.cuda.synchronize()
    Gt = O.rotated_aog(O.aog_estimate(O.aog_accumulate(np.zeros((d, d)), g_bits), n, 1), lam, B)
    log(f"  eigensolve of the rotated AOG d={d} n={n} r={r} B={B}")
    _check_basis(V.cpu().numpy(), ev.cpu().numpy(), Gt, r, overlap_tol=1e-5, ev_tol=1e-4, vec_tol=1e-4)


def test_small_block_rotation_and_smoothing():
    d, r, B = 256, 16, 64
    rng = np.random.default_rng(5)
    G = _stand_in(d, width=40, seed=5)
    lam = np.exp(rng.uniform(-0.5, 0.5, size=d)).astype(np.float32)
    Gf = G.astype(np.float32).astype(np.float64)
    V, ev = _run(Gf, r, iters=10, scale=0.25, lam=lam, B=B)
    _check_basis(V, ev, O.rotated_aog(0.25 * Gf, lam, B), r)


def test_deterministic_and_workspace_reuse():
    """Two calls with one workspace give bit-identical results; iters = 0
    (Rayleigh-Ritz on the start block) still gives an orthonormal basis."""
    d, r = 1024, 32
    A = f32_dev(_stand_in(d, seed=3).astype(np.float32))
    ws = torch.empty(Q.aog_protected_basis_workspace(d, r), dtype=torch.uint8, device="cuda:0")
    V1, e1 = Q.aog_protected_basis(A, r, iters=6, workspace=ws)
    V2, e2 = Q.aog_protected_basis(A, r, iters=6, workspace=ws)
    V0, _ = Q.aog_protected_basis(A, r, iters=0, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(V1, V2) and torch.equal(e1, e2)
    V0 = V0.cpu().double().numpy()
    assert np.abs(V0.T @ V0 - np.eye(r)).max() <= 1e-5


def test_max_size_known_spectrum():
    """The largest size the entry point takes (d = 16384, r = 48), on a matrix
    whose eigenpairs are known in closed form: A = U diag(e) U^T + 1e-3 I with
    U orthonormal (QR of a seeded Gaussian d x 64 block, each column's
    largest-magnitude entry made positive) and e_i = 2^(-i/8).  Its top-48
    eigenvectors are U's first columns and its eigenvalues e_i + 1e-3 (the
    float32 rounding of A moves them by ~1e-7, far inside the tolerances)."""
    d, r, p = 16384, 48, 64
    log(f"  eigensolve at the maximum size d={d} r={r} (known spectrum)")
    U, _ = np.linalg.qr(np.random.default_rng(16384).standard_normal((d, p)))
    idx = np.argmax(np.abs(U), axis=0)
    U = U * np.sign(U[idx, np.arange(p)])[None, :]
    e = 2.0 ** (-np.arange(p) / 8.0)
    Ud = torch.from_numpy(U).to("cuda:0")
    A64 = (Ud * torch.from_numpy(e).to("cuda:0")[None, :]) @ Ud.T.contiguous()
    A64.diagonal().add_(1e-3)
    A = A64.float().contiguous()
    del A64
    V, ev = Q.aog_protected_basis(A, r, iters=10)
    torch.cuda.synchronize()
    # Ky Fan on the GPU in float64: tr(V^T A V)
    Vd = V.double()
    kyfan = float(torch.trace(Vd.T @ (A.double() @ Vd)))
    del A
    V = V.cpu().numpy().astype(np.float64)
    ev = ev.cpu().numpy().astype(np.float64)
    top = e[:r] + 1e-3
    overlap = float(np.linalg.norm(V.T @ U[:, :r]) ** 2 / r)
    orth = float(np.abs(V.T @ V - np.eye(r)).max())
    dots = np.einsum("ij,ij->j", V, U[:, :r])
    log(f"    overlap 1 - {1 - overlap:.2e}, Ky Fan rel {abs(kyfan - top.sum()) / top.sum():.2e}, "
        f"eigenvalue rel {np.abs(ev - top).max() / top[0]:.2e}, min |v.u| {np.abs(dots).min():.8f}, "
        f"orthonormality {orth:.2e}")
    assert overlap >= 1 - 1e-6
    assert abs(kyfan - top.sum()) <= 1e-6 * top.sum()
    assert np.abs(ev - top).max() <= 1e-5 * top[0]
    assert (np.diff(ev) <= 0).all()
    assert orth <= 1e-5
    assert (dots >= 1 - 1e-5).all(), "each eigenvector, with the sign of the largest entry"
    idx = np.argmax(np.abs(V), axis=0)
    assert (V[idx, np.arange(r)] > 0).all()


def test_small_hadamard_block_and_largest_rank():
    """r = 48 (the largest rank) with the smallest rotation block (B = 16) and
    smoothing, against the oracle's eigh of the same G~.  The rank-80 stand-in
    decays slowly (lambda_65 / lambda_48 = 0.76 here), and subspace iteration
    with a 64-vector block converges by that factor per product, so this case
    takes 30 iterations (12 leave ~1e-4 in the overlap, in exact arithmetic
    as well)."""
    d, r, B = 1024, 48, 16
    rng = np.random.default_rng(48)
    G = _stand_in(d, width=80, seed=48)
    lam = np.exp(rng.uniform(-0.7, 0.7, size=d)).astype(np.float32)
    Gf = G.astype(np.float32).astype(np.float64)
    log(f"  eigensolve d={d} r={r} B={B} with smoothing")
    V, ev = _run(Gf, r, iters=30, scale=0.5, lam=lam, B=B)
    _check_basis(V, ev, O.rotated_aog(0.5 * Gf, lam, B), r)
