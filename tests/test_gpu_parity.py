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

from parity_helpers import (bf16_dev, bits, check_weight_scales, check_sampled_rows, check_t, check_y, check_y_elements,
                            check_y_per_token, gpu_layer, log, oracle_factors, run_gpu, sample_rows, y_abs_terms)

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
    check_weight_scales(layer, ref["sw"])
    assert (layer.inv_smooth.cpu().numpy() == ref["inv_lam"]).all(), "1/lambda"
    assert (xq.cpu().numpy() == ref["xq"]).all(), "packed activation bytes"
    assert (xs.cpu().numpy() == ref["sx"].T).all(), "activation scales"
    xt = O.smooth_activations(draws.x, ref["inv_lam"])
    check_t(bits(t), ref["t"], xt, factors["L1"])
    if check_partials:
        P = Q.debug_group_partials(layer, xq)
        torch.cuda.synchronize()
        assert (P.cpu().numpy() == ref["P"]).all(), "int32 group partials"
    # token by token and element by element against the oracle's output for the
    # t the GEMM ran with (t itself is checked above): y_ref + (t_gpu - t_ref) L2
    tg = bits(t)
    y_t = ref["y"] + (O.bf16_bits_to_f64(tg) - O.bf16_bits_to_f64(ref["t"])) @ O.bf16_bits_to_f64(factors["L2"])
    at = y_abs_terms(ref["sx"], ref["sw"], ref["P"], tg, factors["L2"], bias_bits)
    check_y_per_token(bits(y), y_t, at, ref["P"].shape[2], factors["L1"].shape[1])
    check_y_elements(bits(y), y_t, at, ref["P"].shape[2], factors["L1"].shape[1])
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
    (97, 192, 176, 48, True),        # r = 48 on the large-tile GEMM, ragged N, bias
    (130, 1024, 1040, 16, True),
    (257, 640, 256, 32, False),
    (33, 16448, 64, 32, False),      # K > 16384: 1/lambda read from global memory
    # the largest sizes the entry points take
    (130, 65536, 64, 16, True),      # K = 65536, the large-tile GEMM
    (1, 64, 1 << 20, 16, False),     # N = 2^20, one token
    (1 << 20, 64, 16, 16, False),    # M = 2^20
    (65, 64, 1 << 20, 16, False),    # N = 2^20 on the large-tile GEMM
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


def _large_parity(draws, extra_rows=64):
    """Full-size layer in the benchmark's launch configuration: every code,
    scale and t element is checked; y (whole sample, every token, every
    element) and the partials on sampled tokens (more than 64, so the
    partials come from the large-tile GEMM)."""
    M, K, N = draws.shape.M, draws.shape.K, draws.shape.N
    log(f"  large parity {draws.shape.name}: M={M} K={K} N={N} r={draws.shape.r}")
    f = oracle_factors(draws)
    qw, sw = O.quantize_groups(f["R"])
    inv_lam = O.inverse_smoothing(f["lam"])
    layer = gpu_layer(f)
    x, xq, xs, t, y = run_gpu(layer, draws.x)
    wq = layer.wq.cpu().numpy()
    assert (O.unpack_codes(wq) == qw).all(), "weight codes"
    check_weight_scales(layer, sw)
    assert (layer.inv_smooth.cpu().numpy() == inv_lam).all()
    xq_ref, sx_ref, t_ref, qx, xt = O.quantize_activations(draws.x, inv_lam, f["L1"])
    assert (xq.cpu().numpy() == xq_ref).all(), "packed activation bytes"
    assert (xs.cpu().numpy() == sx_ref.T).all(), "activation scales"
    check_t(bits(t), t_ref, xt, f["L1"])
    # the packed weight bytes of a sample of rows (the full pack is checked on smaller layers)
    wrows = sample_rows(N, seed=N + 3, extra=32)
    assert (wq[wrows] == O.pack_codes(qw[wrows], O.quantize_groups_signed(f["R"][wrows])[2])).all(), \
        "packed weight bytes"
    rows = sample_rows(M, seed=M + N, extra=extra_rows)
    check_sampled_rows(layer, xq, y, xq_ref, sx_ref, bits(t), wq, sw, f["L2"], rows)
    del x, xq, xs, t, y, layer
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
    _large_parity(I.denoise_step_layer(block, which), extra_rows=32)


def test_repeat_runs_bit_identical():
    """Determinism / race proxy: 20 runs of every kernel of the layer (the
    large-tile GEMM, its debug partials, the few-token GEMM and the fused
    layer) on four streams, in varied launch orders and with the outputs of
    several runs in flight at once, give bit-identical codes, scales, t,
    partials and y."""
    d = I.custom(M=300, K=512, N=384, r=32, seed=9, n_outliers=5, with_bias=True)
    small = I.custom(M=48, K=1024, N=512, r=16, seed=10, n_outliers=4, with_bias=True)
    layer = gpu_layer(oracle_factors(d), d.bias)
    layer_s = gpu_layer(oracle_factors(small), small.bias)
    x, xsm = bf16_dev(d.x), bf16_dev(small.x)
    streams = [torch.cuda.Stream() for _ in range(4)]
    rng = np.random.default_rng(99)
    pending, outs = [], []
    for i in range(20):
        s = streams[int(rng.integers(0, 4))]
        s.wait_stream(torch.cuda.current_stream())
        order = rng.permutation(3)
        res = {}
        with torch.cuda.stream(s):
            for step in order:
                if step == 0:
                    xq, xs, t = Q.quantize_act(layer, x)
                    res["big"] = (xq, xs, t, Q.asp_linear(layer, xq, xs, t), Q.debug_group_partials(layer, xq))
                elif step == 1:
                    q2, s2, t2 = Q.quantize_act(layer_s, xsm)
                    res["small"] = (q2, s2, t2, Q.asp_linear(layer_s, q2, s2, t2))
                else:
                    res["fused"] = (Q.asp_layer(layer_s, xsm),)
        pending.append(res)
        if i % 5 == 4:                 # several runs in flight before each drain
            torch.cuda.synchronize()
            for r in pending:
                outs.append({k: [v.cpu().numpy() if v.dtype != torch.bfloat16 else bits(v) for v in vals]
                             for k, vals in r.items()})
            pending = []
    for o in outs[1:]:
        for k in o:
            for a, b in zip(o[k], outs[0][k]):
                assert (a == b).all(), k
