"""Shared helpers of the GPU parity tests: move seeded inputs and oracle-built
layer factors to the GPU, run the library through its C ABI, and compare."""

from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import qwam_oracle as O
from paper_2609_33269_amd import qwam as Q

U32 = 2.0 ** -24


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def bf16_dev(bits: np.ndarray) -> torch.Tensor:
    """uint16 bf16 bits (numpy) -> bf16 tensor on cuda:0 (bit-exact)."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to("cuda:0")


def scale_pieces(s: np.ndarray) -> np.ndarray:
    """The weight scales in the two-piece form the weight pack writes (wsp in
    include/qwam.h): hi = bf16(s), lo = bf16(s - hi), both to nearest even,
    packed as hi | lo << 16 (uint32)."""
    s = np.asarray(s, dtype=np.float32).astype(np.float64)
    hi = O.f64_to_bf16_bits(s)
    lo = O.f64_to_bf16_bits(s - O.bf16_bits_to_f64(hi))     # s - hi is exact
    return hi.astype(np.uint32) | (lo.astype(np.uint32) << np.uint32(16))


def check_weight_scales(layer, sw_ref: np.ndarray) -> None:
    """ws bit-exact against the oracle's [N][G] scales, and wsp their pieces."""
    assert (layer.ws.cpu().numpy() == sw_ref.T).all(), "weight scales"
    assert (layer.wsp.cpu().numpy().view(np.uint32) == scale_pieces(sw_ref.T)).all(), "weight-scale pieces"


def f32_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda:0")


def bits(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor -> uint16 bits (numpy)."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def oracle_factors(draws, r=None, hadamard=False):
    r = draws.shape.r if r is None else r
    V = O.protected_basis_from_factor(draws.a, r)
    return O.build_layer(draws.x, draws.w, V, hadamard=hadamard)


def gpu_layer(factors, bias_bits=None) -> Q.PackedLayer:
    """Pack the oracle-built factors with the library (qwam_pack_weights)."""
    L1 = bf16_dev(factors["L1"])
    L2 = bf16_dev(factors["L2"])
    bias = None if bias_bits is None else bf16_dev(bias_bits)
    return Q.make_layer(f32_dev(factors["R"]), f32_dev(factors["lam"]), L1, L2, bias,
                        hadamard=int(factors.get("hadamard", 0)), group=int(factors.get("group", 64)))


def rel_fro(a: np.ndarray, b: np.ndarray) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (nb if nb > 0 else 1.0))


Y_TOL = 2e-3


def y_tolerance(y_ref: np.ndarray) -> float:
    """Relative Frobenius tolerance of y against the unrounded float64 oracle:
    2e-3, unless the output is so small that its own bf16 rounding (the
    correctly rounded bf16 of y_ref) is already further away; then that
    rounding error plus 1e-4 for the float32 accumulation."""
    return max(Y_TOL, rel_fro(O.round_to_bf16(y_ref), y_ref) + 1e-4)


def check_y(y_gpu_bits: np.ndarray, y_ref: np.ndarray) -> float:
    err = rel_fro(O.bf16_bits_to_f64(y_gpu_bits), y_ref)
    tol = y_tolerance(y_ref)
    log(f"    y rel Frobenius error {err:.3e} (tolerance {tol:.3e})")
    assert err <= tol
    return err


def bf16_ulp(v: np.ndarray) -> np.ndarray:
    """Spacing of bf16 numbers at |v| (2**-133 below the normal range)."""
    v = np.abs(np.asarray(v, dtype=np.float64))
    _, e = np.frexp(v)
    e = np.maximum(e, -125)
    return np.ldexp(np.ones_like(v), e - 8)


def check_t(t_gpu_bits, t_ref_bits, xt, L1_bits, frac_over_1ulp=1e-3):
    """t from the GPU (bf16 of a float32 accumulation) against the oracle's
    bf16 of the exact sum.

    Rigorous per element: |t_gpu - t_ref| <= ulp(t) + K 2^-24 sum_k |bf16(x~_k) L1[k, j]|
    (rounding of both to bf16 plus the worst-case error of a float32 sum of K
    terms).  Statistically: at most `frac_over_1ulp` of the elements differ by
    more than one bf16 ulp (that only happens where the sum nearly cancels).
    """
    tg = O.bf16_bits_to_f64(t_gpu_bits)
    tr = O.bf16_bits_to_f64(t_ref_bits)
    K = xt.shape[1]
    absterms = np.abs(O.round_to_bf16(xt)) @ np.abs(O.bf16_bits_to_f64(L1_bits))
    ulp = np.maximum(bf16_ulp(tr), bf16_ulp(tg))
    diff = np.abs(tg - tr)
    bound = ulp + K * U32 * absterms
    assert (diff <= bound).all(), f"t outside the rounding bound at {np.argwhere(diff > bound)[:5].tolist()}"
    over = float(np.mean(diff > ulp))
    assert over <= frac_over_1ulp, f"{over:.2e} of t elements differ by more than 1 bf16 ulp"
    return over


def run_gpu(layer: Q.PackedLayer, x_bits: np.ndarray, deflate: bool = False):
    """quantize_act (or quantize_act_deflated) + asp_linear on cuda:0; returns
    device tensors."""
    x = bf16_dev(x_bits)
    xq, xs, t = (Q.quantize_act_deflated if deflate else Q.quantize_act)(layer, x)
    y = Q.asp_linear(layer, xq, xs, t)
    torch.cuda.synchronize()
    return x, xq, xs, t, y


def y_abs_terms(sx, sw, P, t_bits, L2_bits, bias_bits=None) -> np.ndarray:
    """sum_g |sx sw P| + sum_j |t_j L2[j, n]| (+ |bias|) per output: the scale
    of the float32 error of y (float64)."""
    a = np.einsum("mg,ng,mng->mn", np.abs(np.asarray(sx, np.float64)), np.abs(np.asarray(sw, np.float64)),
                  np.abs(P).astype(np.float64))
    a += np.abs(O.bf16_bits_to_f64(t_bits)) @ np.abs(O.bf16_bits_to_f64(L2_bits))
    if bias_bits is not None:
        a += np.abs(O.bf16_bits_to_f64(bias_bits))[None, :]
    return a


def check_y_elements(y_gpu_bits, y_ref, abs_terms, n_groups, rank, min_identical=0.99):
    """Element by element: bf16(y_gpu) against the correctly rounded bf16 of the
    float64 oracle.  Every element within one bf16 ulp plus the float32 error
    bound of the kernel's arithmetic: each group's scale product is formed from
    two-piece bf16 splits of the two scales (within 2^-15 of sx * sw), and the
    G + r + 1 float32 roundings of the accumulation each add at most 2^-24 of
    the terms' magnitude.  And at least `min_identical` of the elements equal
    to bf16(y_ref): the error bound is far below a bf16 ulp, so y only differs
    where y_ref lies next to a rounding boundary."""
    yg = O.bf16_bits_to_f64(y_gpu_bits)
    yr = O.round_to_bf16(y_ref)
    ulp = np.maximum(bf16_ulp(yr), bf16_ulp(yg))
    bound = ulp + y_float32_bound(abs_terms, n_groups, rank)
    diff = np.abs(yg - yr)
    bad = np.argwhere(diff > bound)
    assert bad.size == 0, f"y outside one ulp + float32 bound at {bad[:5].tolist()}"
    same = float(np.mean(yg == yr))
    log(f"    y elements equal to bf16(y_ref): {same:.5f}")
    assert same >= min_identical, f"only {same:.4f} of y elements equal bf16(y_ref)"
    return same


def y_float32_bound(abs_terms, n_groups, rank) -> np.ndarray:
    """Per-element bound on the kernel's float32 result before its bf16
    rounding: the two-piece bf16 splits of the scales (within 2^-15 of
    sx * sw) and the G + r + 2 float32 roundings of the accumulation."""
    return (2.0 ** -15 + (n_groups + rank + 2) * U32) * np.asarray(abs_terms, dtype=np.float64)


def check_y_per_token(y_gpu_bits, y_ref, abs_terms, n_groups, rank):
    """Relative Frobenius error of every token's output row within its
    tolerance: 2e-3, or, where larger, the row's error when each element takes
    the farther of the bf16 values that a float32 result within the kernel's
    accumulation bound of y_ref can round to (+1e-4).  An element whose bound
    interval does not contain a bf16 rounding midpoint can only take the
    correctly rounded value, so for most rows that is the row's own bf16
    rounding error; a row of few outputs with one element next to a midpoint
    may need more than 2e-3."""
    yg = O.bf16_bits_to_f64(y_gpu_bits)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    eb = y_float32_bound(abs_terms, n_groups, rank)
    worst = np.maximum(np.abs(O.round_to_bf16(y_ref - eb) - y_ref), np.abs(O.round_to_bf16(y_ref + eb) - y_ref))
    nref = np.linalg.norm(y_ref, axis=1)
    nref = np.where(nref > 0, nref, 1.0)
    errs = np.linalg.norm(yg - y_ref, axis=1) / nref
    tols = np.maximum(Y_TOL, np.linalg.norm(worst, axis=1) / nref + 1e-4)
    worst_row = int(np.argmax(errs / tols))
    log(f"    worst token error {errs[worst_row]:.3e} (tolerance {tols[worst_row]:.3e}); "
        f"{int(np.sum(tols > Y_TOL))} of {len(tols)} rows above 2e-3 by rounding")
    bad = np.flatnonzero(errs > tols)
    assert bad.size == 0, f"tokens {bad[:8].tolist()} exceed their tolerance"


def sample_rows(M: int, seed: int, extra: int = 64) -> np.ndarray:
    """Token sample of a large layer: the first and last token, one token in
    every 128-token tile and `extra` more at random; more than 64 tokens for
    M >= 128, so that the debug partials run on the large-tile GEMM."""
    rng = np.random.default_rng(seed)
    rows = {0, M - 1}
    for tile in range(0, M, 128):
        rows.add(int(min(M - 1, tile + rng.integers(0, 128))))
    rows.update(int(v) for v in rng.choice(M, size=min(M, extra), replace=False))
    return np.array(sorted(rows))


def check_sampled_rows(layer, xq, y, xq_ref, sx_ref, t_bits, wq, sw, L2_bits, rows, bias_bits=None):
    """y and the int32 group partials of sampled tokens of a large layer against
    the oracle computed from the same codes and scales and the t the GEMM ran
    with (t_bits: the GPU's own, checked against the oracle's by the caller):
    Frobenius error over the sample, every token's own error, every element
    (check_y_elements), and the partials bit for bit through the debug entry
    point on the sampled rows."""
    t_ref = t_bits
    y_ref, P_ref = O.asp_output_rows(xq_ref[rows], sx_ref[rows], t_ref[rows], wq, sw, L2_bits, bias_bits)
    sel = torch.from_numpy(rows).cuda()
    yb = bits(y[sel])
    err = rel_fro(O.bf16_bits_to_f64(yb), y_ref)
    log(f"    y rel Frobenius error on {len(rows)} sampled tokens {err:.3e}")
    assert err <= y_tolerance(y_ref)
    at = y_abs_terms(sx_ref[rows], sw, P_ref, t_ref[rows], L2_bits, bias_bits)
    check_y_per_token(yb, y_ref, at, P_ref.shape[2], np.asarray(L2_bits).shape[0])
    check_y_elements(yb, y_ref, at, P_ref.shape[2], np.asarray(L2_bits).shape[0])
    P = Q.debug_group_partials(layer, xq[sel].contiguous())
    torch.cuda.synchronize()
    assert (P.cpu().numpy() == P_ref).all(), "int32 group partials of sampled tokens"
    del P
