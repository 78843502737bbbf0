"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bit-exact: weight codes/bytes/scales, 1/lambda, activation codes/bytes/scales
and the int32 group partials.  Floating point: t within the bf16 rounding
bound (see parity_helpers.check_t); y within relative Frobenius error 2e-3 of
the float64 oracle on the same codes.
"""

import numpy as np
import pytest
import torch

from oracle import qwam_oracle as O
from paper_2609_33269_amd import inputs as I
from paper_2609_33269_amd import qwam as Q

from parity_helpers import (bf16_dev, bits, check_t, check_y, f32_dev, gpu_layer, log, oracle_factors,
                            rel_fro, run_gpu, y_tolerance)

pytestmark = pytest.mark.gpu



@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    Q.lib()


def _full_parity(draws, factors, bias_bits=None, check_partials=True):
    """Run every entry point on the whole layer and compare everything."""
    M, K, N = draws.shape.M, draws.shape.K, draws.shape.N
    log(f"  parity {draws.shape.name}: M={M} K={K} N={N} r={factors['L1'].shape[1]} bias={bias_bits is not None}")
    ref = O.asp_linear(draws.x, factors, bias_bits=bias_bits)
    layer = gpu_layer(factors, bias_bits)
    x, xq, xs, t, y = run_gpu(layer, draws.x)
    assert (layer.wq.cpu().numpy() == ref["wq"]).all(), "packed weight bytes"
    assert (layer.ws.cpu().numpy() == ref["sw"].T).all(), "weight scales"
    assert (layer.inv_smooth.cpu().numpy() == ref["inv_lam"]).all(), "1/lambda"
    assert (xq.cpu().numpy() == ref["xq"]).all(), "packed activation bytes"
    assert (xs.cpu().numpy() == ref["sx"].T).all(), "activation scales"
    xt = O.smooth_activations(draws.x, ref["inv_lam"])
    check_t(bits(t), ref["t"], xt, factors["L1"])
    if check_partials:
        P = Q.debug_group_partials(layer, xq)
        torch.cuda.synchronize()
        assert (P.cpu().numpy() == ref["P"]).all(), "int32 group partials"
    return check_y(bits(y), ref["y"])


@pytest.mark.parametrize("with_bias", [False, True])
def test_tiny_layer_full_parity(with_bias):
    d = I.tiny(with_bias=with_bias)
    _full_parity(d, oracle_factors(d), d.bias)


EDGE_SHAPES = [
    # M, K, N, r, bias
    (1, 64, 16, 16, False),
    (15, 128, 48, 32, True),
    (17, 192, 144, 48, False),
    (129, 256, 272, 64, True),
    (200, 320, 400, 32, False),
    (130, 1024, 1040, 16, True),
    (257, 640, 256, 32, False),
    (33, 16448, 64, 32, False),      # K > 16384: 1/lambda read from global memory
]


@pytest.mark.parametrize("M,K,N,r,bias", EDGE_SHAPES)
def test_edge_shapes(M, K, N, r, bias):
    d = I.custom(M=M, K=K, N=N, r=r, seed=M * 7 + K, n_outliers=max(1, K // 100), with_bias=bias)
    _full_parity(d, oracle_factors(d, r), d.bias)


def test_zero_residual_reduces_to_branch():
    d = I.custom(M=33, K=256, N=128, r=16, seed=5, n_outliers=2)
    f = oracle_factors(d)
    f = dict(f, R=np.zeros_like(f["R"]))
    _full_parity(d, f)
    # y is bf16(t L2): compare against the product of the GPU's own t with L2 exactly
    layer = gpu_layer(f)
    _, _, _, t, y = run_gpu(layer, d.x)
    ty = O.bf16_bits_to_f64(bits(t)) @ O.bf16_bits_to_f64(f["L2"])
    yg = O.bf16_bits_to_f64(bits(y))
    assert np.all(np.abs(yg - ty) <= 0.5 * np.abs(ty) * 2.0 ** -7 + 1e-30 + np.abs(ty) * 2.0 ** -20)


def test_degenerate_activations():
    """Zero tokens, zero groups, tiny and subnormal values, on-grid values."""
    d = I.custom(M=40, K=256, N=64, r=16, seed=6, n_outliers=1)
    x = O.bf16_bits_to_f64(d.x).astype(np.float32)
    x[0, :] = 0.0                                  # an all-zero token
    x[1, 64:128] = 0.0                             # one all-zero group
    x[2, :64] = np.float32(1e-39)                  # subnormal group (scale 0 after smoothing)
    x[3, :] = np.float32(3e-38)                    # near the bottom of the normal range
    x[4, :] = np.tile(np.arange(-7, 9, dtype=np.float32), 16) * np.float32(0.25)   # on-grid
    x[5, :] = -x[5, :]
    xb = O.f64_to_bf16_bits(x.astype(np.float64))
    d.x = xb
    f = oracle_factors(d)
    f = dict(f, lam=np.ones_like(f["lam"]))        # unit smoothing keeps the constructed values
    _full_parity(d, f)
    layer = gpu_layer(f)
    _, xq, xs, _, _ = run_gpu(layer, xb)
    assert not xq[0].any().item() and not xs[:, 0].any().item()
    assert not xq[1, 32:64].any().item() and xs[1, 1].item() == 0.0


def _sample_rows(M, n, seed):
    rng = np.random.default_rng(seed)
    rows = set([0, M - 1])
    for tile in range(0, M, 128):                  # at least one row per M tile
        rows.add(int(min(M - 1, tile + rng.integers(0, 128))))
    extra = rng.choice(M, size=min(M, n), replace=False)
    rows.update(int(v) for v in extra)
    return np.array(sorted(rows))


def _large_parity(draws, n_rows=24):
    """Full-size layer in the benchmark's launch configuration: every code,
    scale and t element is checked; partials and y on sampled tokens."""
    M, K, N = draws.shape.M, draws.shape.K, draws.shape.N
    log(f"  large parity {draws.shape.name}: M={M} K={K} N={N} r={draws.shape.r}")
    f = oracle_factors(draws)
    wq, sw, inv_lam, qw = O.pack_weights(f["R"], f["lam"])
    layer = gpu_layer(f)
    x, xq, xs, t, y = run_gpu(layer, draws.x)
    assert (layer.wq.cpu().numpy() == wq).all(), "packed weight bytes"
    assert (layer.ws.cpu().numpy() == sw.T).all(), "weight scales"
    assert (layer.inv_smooth.cpu().numpy() == inv_lam).all()
    xq_ref, sx_ref, t_ref, qx, xt = O.quantize_activations(draws.x, inv_lam, f["L1"])
    assert (xq.cpu().numpy() == xq_ref).all(), "packed activation bytes"
    assert (xs.cpu().numpy() == sx_ref.T).all(), "activation scales"
    check_t(bits(t), t_ref, xt, f["L1"])
    rows = _sample_rows(M, n_rows, seed=M + N)
    y_ref, P_ref = O.asp_output_rows(xq_ref[rows], sx_ref[rows], t_ref[rows], wq, sw, f["L2"])
    yg = O.bf16_bits_to_f64(bits(y[torch.from_numpy(rows).cuda()]))
    err = rel_fro(yg, y_ref)
    row_err = max(rel_fro(yg[i], y_ref[i]) for i in range(len(rows)))
    log(f"    y rel Frobenius error on {len(rows)} sampled tokens {err:.3e} (worst token {row_err:.3e})")
    assert err <= y_tolerance(y_ref)
    P = Q.debug_group_partials(layer, xq[torch.from_numpy(rows).cuda()].contiguous())
    torch.cuda.synchronize()
    assert (P.cpu().numpy() == P_ref).all(), "int32 group partials of sampled tokens"
    del x, xq, xs, t, y, P, layer
    torch.cuda.empty_cache()


@pytest.mark.parametrize("which", ["video_dit_qkv", "video_dit_ffn_up", "video_dit_ffn_down"])
def test_video_dit_layers_full_size(which):
    _large_parity(getattr(I, which)())


@pytest.mark.parametrize("M,N", I.ACTION_EXPERT_SHAPES)
def test_action_expert_layers(M, N):
    d = I.action_expert(M, N)
    _full_parity(d, oracle_factors(d))


@pytest.mark.parametrize("block,which", [(0, 0), (13, 1), (29, 3)])
def test_denoise_step_sampled_layers(block, which):
    _large_parity(I.denoise_step_layer(block, which), n_rows=16)


def test_repeat_runs_bit_identical():
    d = I.custom(M=300, K=512, N=384, r=32, seed=9, n_outliers=5, with_bias=True)
    f = oracle_factors(d)
    layer = gpu_layer(f, d.bias)
    outs = []
    streams = [torch.cuda.Stream() for _ in range(2)]
    for i in range(6):
        s = streams[i % 2]
        with torch.cuda.stream(s):
            x = bf16_dev(d.x)
            xq, xs, t = Q.quantize_act(layer, x)
            y = Q.asp_linear(layer, xq, xs, t)
            P = Q.debug_group_partials(layer, xq)
        torch.cuda.synchronize()
        outs.append((xq.cpu().numpy(), xs.cpu().numpy(), bits(t), bits(y), P.cpu().numpy()))
    for o in outs[1:]:
        for a, b in zip(o, outs[0]):
            assert (a == b).all()
