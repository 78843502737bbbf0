"""GPU parity of the deflated activation path (Eq. 8 / Eq. 9): the 4-bit
path quantizes x~_perp = x~ - L1 t instead of x~.

Bit-exact: t (accumulated in float64 on the GPU, so its bf16 rounding is that
of the exact sum, as in the oracle), the deflated codes, packed bytes and
scales, and the int32 group partials.  y within relative Frobenius error 2e-3
of the float64 oracle on the same codes.
"""

import numpy as np
import pytest
import torch

from oracle import qwam_oracle as O
from paper_2609_33269_amd import inputs as I
from paper_2609_33269_amd import qwam as Q

from parity_helpers import (bf16_dev, bits, check_sampled_rows, check_y, f32_dev, gpu_layer, log, oracle_factors,
                            rel_fro, run_gpu, sample_rows, y_tolerance)

pytestmark = pytest.mark.gpu



@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    Q.lib()


def _deflated_parity(draws, factors, bias_bits=None, check_partials=True):
    M, K, N = draws.shape.M, draws.shape.K, draws.shape.N
    log(f"  deflated parity {draws.shape.name}: M={M} K={K} N={N} r={factors['L1'].shape[1]} "
        f"bias={bias_bits is not None}")
    ref = O.asp_linear(draws.x, factors, bias_bits=bias_bits, deflate=True)
    layer = gpu_layer(factors, bias_bits)
    x, xq, xs, t, y = run_gpu(layer, draws.x, deflate=True)
    assert (bits(t) == ref["t"]).all(), "t (bf16 of the exact sum)"
    assert (xq.cpu().numpy() == ref["xq"]).all(), "packed deflated activation bytes"
    assert (xs.cpu().numpy() == ref["sx"].T).all(), "deflated activation scales"
    if check_partials:
        P = Q.debug_group_partials(layer, xq)
        torch.cuda.synchronize()
        assert (P.cpu().numpy() == ref["P"]).all(), "int32 group partials"
    check_y(bits(y), ref["y"])
    return ref, (xq, xs, t, y)


@pytest.mark.parametrize("with_bias", [False, True])
def test_deflated_tiny_layer(with_bias):
    d = I.tiny(with_bias=with_bias)
    _deflated_parity(d, oracle_factors(d), d.bias)


DEFLATED_SHAPES = [
    # M, K, N, r, bias
    (1, 64, 16, 16, False),
    (15, 128, 48, 32, True),
    (17, 192, 144, 48, False),
    (129, 256, 272, 64, True),
    (200, 320, 400, 32, False),
    (130, 1024, 1040, 16, True),
    (33, 16448, 64, 32, False),      # K > 16384: 1/lambda read from global memory
    (20, 16448, 32, 64, True),
    # the largest K the entry points take
    (33, 65536, 64, 64, True),
    (130, 65536, 32, 16, False),
    (1 << 20, 64, 16, 16, False),    # the largest M
]


@pytest.mark.parametrize("M,K,N,r,bias", DEFLATED_SHAPES)
def test_deflated_edge_shapes(M, K, N, r, bias):
    d = I.custom(M=M, K=K, N=N, r=r, seed=M * 11 + K, n_outliers=max(1, K // 100), with_bias=bias)
    _deflated_parity(d, oracle_factors(d, r), d.bias)


def test_deflation_rounds_each_step():
    """x = 1, lambda = 1, K = 128, two branch directions of constant 2^-16:
    t_0 = t_1 = 128 * 2^-16 = 2^-9 and each step removes 2^-25, a tie that
    rounds back to 1; so x~_perp = 1 exactly and the scale is fl32(1/7).
    (Removing the summed correction would give 1 - 2^-24 and another scale.)"""
    M, K, N, r = 5, 128, 16, 16
    L1 = np.zeros((K, r))
    L1[:, :2] = 2.0 ** -16
    L1b = O.f64_to_bf16_bits(L1)
    L2b = np.zeros((r, N), dtype=np.uint16)
    xb = O.f64_to_bf16_bits(np.ones((M, K)))
    layer = Q.make_layer(torch.zeros((N, K), dtype=torch.float32, device="cuda:0"),
                         torch.ones(K, dtype=torch.float32, device="cuda:0"), bf16_dev(L1b), bf16_dev(L2b))
    xq, xs, t = Q.quantize_act_deflated(layer, bf16_dev(xb))
    torch.cuda.synchronize()
    tv = O.bf16_bits_to_f64(bits(t))
    assert (tv[:, :2] == 2.0 ** -9).all() and not tv[:, 2:].any()
    assert (xs.cpu().numpy() == np.float32(np.float32(1.0) / np.float32(7.0))).all()
    assert (O.unpack_codes(xq.cpu().numpy()) == 7).all()
    xq_o, sx_o, t_o, _, xp_o = O.quantize_activations_deflated(xb, np.ones(K, np.float32), L1b)
    assert (xp_o == 1.0).all()
    assert (xq.cpu().numpy() == xq_o).all() and (xs.cpu().numpy() == sx_o.T).all()


def test_deflation_on_coordinate_axes():
    """Protected directions = coordinate axes: on each protected channel the
    deflated activation is x~ - bf16(x~) (the bits bf16 drops), elsewhere x~."""
    d = I.custom(M=70, K=256, N=96, r=16, seed=41, n_outliers=2)
    rng = np.random.default_rng(41)
    axes = rng.choice(256, size=16, replace=False)
    V = np.zeros((256, 16))
    V[axes, np.arange(16)] = 1.0
    f = O.build_layer(d.x, d.w, V)
    ref, (xq, xs, t, y) = _deflated_parity(d, f)
    xt = O.smooth_activations(d.x, O.inverse_smoothing(f["lam"])).astype(np.float64)
    expect = xt.copy()
    expect[:, axes] = xt[:, axes] - O.round_to_bf16(xt[:, axes])
    codes, scales = O.quantize_groups(expect.astype(np.float32))
    assert (O.unpack_codes(xq.cpu().numpy()) == codes).all()
    assert (xs.cpu().numpy() == scales.T).all()


@pytest.mark.parametrize("which", ["video_dit_ffn_up", "video_dit_ffn_down"])
def test_deflated_full_size(which):
    """Full-size layer, launch configuration of the benchmark: every t element,
    code and scale is compared; y and the partials on sampled tokens."""
    draws = getattr(I, which)()
    M, K, N = draws.shape.M, draws.shape.K, draws.shape.N
    log(f"  deflated full size {draws.shape.name}: M={M} K={K} N={N}")
    f = oracle_factors(draws)
    _, sw = O.quantize_groups(f["R"])
    inv_lam = O.inverse_smoothing(f["lam"])
    layer = gpu_layer(f)
    wq = layer.wq.cpu().numpy()
    x, xq, xs, t, y = run_gpu(layer, draws.x, deflate=True)
    xq_ref, sx_ref, t_ref, _, _ = O.quantize_activations_deflated(draws.x, inv_lam, f["L1"])
    assert (bits(t) == t_ref).all(), "t"
    assert (xq.cpu().numpy() == xq_ref).all(), "packed deflated activation bytes"
    assert (xs.cpu().numpy() == sx_ref.T).all(), "deflated activation scales"
    check_sampled_rows(layer, xq, y, xq_ref, sx_ref, bits(t), wq, sw, f["L2"], sample_rows(M, seed=M + N + 1))
    # the deflated scales are smaller than the plain ones on the same tokens
    _, xs_plain, _ = Q.quantize_act(layer, x)
    ratio = float(xs.float().mean() / xs_plain.float().mean())
    log(f"    mean activation scale deflated / plain = {ratio:.3f}")
    assert ratio <= 1.0
    del x, xq, xs, t, y, layer, xs_plain
    torch.cuda.empty_cache()


@pytest.mark.parametrize("M,N", I.ACTION_EXPERT_SHAPES)
def test_deflated_action_expert_layers(M, N):
    d = I.action_expert(M, N)
    _deflated_parity(d, oracle_factors(d))
