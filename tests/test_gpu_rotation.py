"""GPU parity of the rotated activation path (Eq. 3, block Hadamard rotation
applied online with the fast Walsh-Hadamard transform), with and without
deflation (Eq. 8 / Eq. 9).

Bit-exact: the rotated activation codes, packed bytes and scales (the float32
transform follows the oracle's butterfly order), the int32 group partials, and
with deflation also t.  Without deflation t is checked against its rounding
bound (parity_helpers.check_t) on the rotated x~.  y within relative Frobenius
error 2e-3 of the float64 oracle on the same codes.
"""

import numpy as np
import pytest
import torch

from oracle import qwam_oracle as O
from paper_2609_33269_amd import inputs as I
from paper_2609_33269_amd import qwam as Q

from parity_helpers import (bf16_dev, bits, check_sampled_rows, check_t, check_y, gpu_layer, log, oracle_factors,
                            run_gpu, sample_rows)

pytestmark = pytest.mark.gpu



@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    Q.lib()


def _rotated_parity(draws, factors, bias_bits=None, deflate=False, check_partials=True):
    M, K, N = draws.shape.M, draws.shape.K, draws.shape.N
    B = factors["hadamard"]
    log(f"  rotated parity {draws.shape.name}: M={M} K={K} N={N} r={factors['L1'].shape[1]} B={B} "
        f"deflate={deflate} bias={bias_bits is not None}")
    ref = O.asp_linear(draws.x, factors, bias_bits=bias_bits, deflate=deflate)
    layer = gpu_layer(factors, bias_bits)
    assert layer.hadamard == B
    x, xq, xs, t, y = run_gpu(layer, draws.x, deflate=deflate)
    assert (xq.cpu().numpy() == ref["xq"]).all(), "packed rotated activation bytes"
    assert (xs.cpu().numpy() == ref["sx"].T).all(), "rotated activation scales"
    if deflate:
        assert (bits(t) == ref["t"]).all(), "t (bf16 of the exact sum)"
    else:
        xt = O.transformed_activations(draws.x, ref["inv_lam"], B)
        check_t(bits(t), ref["t"], xt, factors["L1"])
    if check_partials:
        P = Q.debug_group_partials(layer, xq)
        torch.cuda.synchronize()
        assert (P.cpu().numpy() == ref["P"]).all(), "int32 group partials"
    check_y(bits(y), ref["y"])
    return ref, (xq, xs, t, y)


ROTATED_SHAPES = [
    # M, K, N, r, bias          block B, tile width
    (1, 64, 16, 16, False),     # B 64,  T 64
    (15, 128, 48, 32, True),    # B 128, T 128
    (17, 192, 144, 48, False),  # B 64,  T 192
    (129, 256, 272, 64, True),  # B 256, T 256
    (200, 320, 400, 32, False),  # B 64, T 320
    (130, 1024, 1040, 16, True),  # B 1024, T 1024
    (40, 640, 96, 32, False),   # B 128, T 640
    (33, 3072, 64, 32, True),   # B 1024, three tiles
    (20, 16448, 32, 64, False),  # B 64, T 64, 257 tiles
    (33, 65536, 64, 64, True),   # B 1024, 64 tiles: the largest K
]

def test_rotated_largest_m():
    """M = 2^20, the largest M the entry points take (B = 64)."""
    d = I.custom(M=1 << 20, K=64, N=16, r=16, seed=29, n_outliers=1)
    _rotated_parity(d, oracle_factors(d, 16, hadamard=True))


# block sizes below App. B.1's choice, which the ABI also accepts: the first
# butterfly stages stay inside a lane, or end at the lane-pair exchange
SMALL_BLOCK_SHAPES = [
    # M, K, N, r, bias, B
    (5, 64, 32, 16, False, 16),
    (19, 256, 48, 32, True, 32),
    (70, 1024, 80, 16, False, 16),
    (33, 3072, 64, 32, True, 32),
]


@pytest.mark.parametrize("deflate", [False, True])
@pytest.mark.parametrize("M,K,N,r,bias", ROTATED_SHAPES)
def test_rotated_shapes(M, K, N, r, bias, deflate):
    d = I.custom(M=M, K=K, N=N, r=r, seed=M * 13 + K, n_outliers=max(1, K // 100), with_bias=bias)
    _rotated_parity(d, oracle_factors(d, r, hadamard=True), d.bias, deflate=deflate)


@pytest.mark.parametrize("deflate", [False, True])
@pytest.mark.parametrize("M,K,N,r,bias,B", SMALL_BLOCK_SHAPES)
def test_rotated_small_blocks(M, K, N, r, bias, B, deflate):
    d = I.custom(M=M, K=K, N=N, r=r, seed=M * 17 + K + B, n_outliers=max(1, K // 100), with_bias=bias)
    _rotated_parity(d, oracle_factors(d, r, hadamard=B), d.bias, deflate=deflate)


# one workgroup per token (M <= 64, r = 16 up to K = 2048, r = 32 up to K = 1024)
FEW_TOKEN_SHAPES = [
    # M, K, N, r, bias          block B, rotation waves
    (16, 1024, 256, 16, False),  # B 1024, one wave: the action-expert K
    (64, 1024, 128, 32, True),  # B 1024, the most tokens and the largest K of r = 32
    (7, 1536, 64, 16, True),    # B 512, the second wave half past K
    (3, 2048, 48, 16, False),   # B 1024, two waves: the largest K of r = 16
    (9, 320, 32, 32, False),    # B 64, K below the kernel's channel capacity
    (2, 192, 32, 16, True),     # B 64
    (65, 1024, 64, 16, False),  # one token past: the 16-token kernel
]


@pytest.mark.parametrize("deflate", [False, True])
@pytest.mark.parametrize("M,K,N,r,bias", FEW_TOKEN_SHAPES)
def test_rotated_few_tokens(M, K, N, r, bias, deflate):
    d = I.custom(M=M, K=K, N=N, r=r, seed=M * 23 + K, n_outliers=max(1, K // 100), with_bias=bias)
    _rotated_parity(d, oracle_factors(d, r, hadamard=True), d.bias, deflate=deflate)


def test_rotated_one_hot_closed_form():
    """x = e_k (lambda = 1, B = 1024): the rotated token is +-2^-5 on the whole
    block, so every code of that block is +-7 with the sign of row k of H and
    every scale is fl32(2^-5 / 7); the other block is zero."""
    M, K, N, r = 4, 2048, 32, 16
    ks = [3, 1024 + 77, 700, 2047]
    xf = np.zeros((M, K))
    for m, k in enumerate(ks):
        xf[m, k] = 1.0
    xb = O.f64_to_bf16_bits(xf)
    L1b = O.f64_to_bf16_bits(np.eye(K)[:, :r])
    layer = Q.make_layer(torch.zeros((N, K), dtype=torch.float32, device="cuda:0"),
                         torch.ones(K, dtype=torch.float32, device="cuda:0"), bf16_dev(L1b),
                         bf16_dev(np.zeros((r, N), dtype=np.uint16)), hadamard=1024)
    xq, xs, t = Q.quantize_act(layer, bf16_dev(xb))
    torch.cuda.synchronize()
    codes = O.unpack_codes(xq.cpu().numpy())
    scales = xs.cpu().numpy().T
    s7 = np.float32(np.float32(2.0 ** -5) / np.float32(7.0))
    j = np.arange(1024)
    for m, k in enumerate(ks):
        blk, kk = divmod(k, 1024)
        signs = np.array([(-1) ** bin(int(v) & kk).count("1") for v in j])
        assert (codes[m, blk * 1024:(blk + 1) * 1024] == 7 * signs).all()
        assert not np.delete(codes[m], np.arange(blk * 1024, (blk + 1) * 1024)).any()
        assert (scales[m, blk * 16:(blk + 1) * 16] == s7).all()


@pytest.mark.parametrize("deflate", [False, True])
def test_rotated_full_size(deflate):
    """The FFN up-projection at full size (B = 1024, three tiles per token
    row): every code and scale compared (and t with deflation); y and the
    partials on sampled tokens."""
    draws = I.video_dit_ffn_up()
    M, K, N = draws.shape.M, draws.shape.K, draws.shape.N
    log(f"  rotated full size {draws.shape.name} deflate={deflate}")
    f = oracle_factors(draws, hadamard=True)
    _, sw = O.quantize_groups(f["R"])
    inv_lam = O.inverse_smoothing(f["lam"])
    layer = gpu_layer(f)
    wq = layer.wq.cpu().numpy()
    x, xq, xs, t, y = run_gpu(layer, draws.x, deflate=deflate)
    quant = O.quantize_activations_deflated if deflate else O.quantize_activations
    xq_ref, sx_ref, t_ref, _, xt = quant(draws.x, inv_lam, f["L1"], f["hadamard"])
    assert (xq.cpu().numpy() == xq_ref).all(), "packed rotated activation bytes"
    assert (xs.cpu().numpy() == sx_ref.T).all(), "rotated activation scales"
    if deflate:
        assert (bits(t) == t_ref).all(), "t"
    else:
        check_t(bits(t), t_ref, O.transformed_activations(draws.x, inv_lam, f["hadamard"]), f["L1"])
    check_sampled_rows(layer, xq, y, xq_ref, sx_ref, bits(t), wq, sw, f["L2"], sample_rows(M, seed=M + 7))
    del x, xq, xs, t, y, layer
    torch.cuda.empty_cache()


def test_rotated_action_expert_layer():
    d = I.action_expert(32, 4096)
    _rotated_parity(d, oracle_factors(d, hadamard=True))
