"""GPU parity of the fused few-token layer (qwam_asp_layer, M <= 64): the
activation step and the GEMM in one launch, in both of its forms (16-token
blocks with one, two or four weight blocks per workgroup; 32-token blocks).

Bit-exact: the codes, packed bytes and scales it reports (the activation
step's arithmetic is the activation kernel's).  t within its rounding bound
(parity_helpers.check_t; the fused kernel sums t in another float32 order).
y within the relative Frobenius tolerance of parity_helpers.check_y of the
float64 oracle, and bit-identical to the two-call path's y for every token
whose t both computed alike.
"""

import numpy as np
import pytest
import torch

from oracle import qwam_oracle as O
from paper_2609_33269_amd import inputs as I
from paper_2609_33269_amd import qwam as Q

from parity_helpers import bf16_dev, bits, check_t, check_y, gpu_layer, log, oracle_factors

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    Q.lib()


def _fused_parity(draws, factors, bias_bits=None):
    M, K, N = draws.shape.M, draws.shape.K, draws.shape.N
    r = factors["L1"].shape[1]
    log(f"  fused layer {draws.shape.name}: M={M} K={K} N={N} r={r} bias={bias_bits is not None}")
    ref = O.asp_linear(draws.x, factors, bias_bits=bias_bits)
    layer = gpu_layer(factors, bias_bits)
    x = bf16_dev(draws.x)
    xq = torch.empty((M, K // 2), dtype=torch.uint8, device="cuda:0")
    xs = torch.empty((K // 64, M), dtype=torch.float32, device="cuda:0")
    t = torch.empty((M, r), dtype=torch.bfloat16, device="cuda:0")
    y = Q.asp_layer(layer, x, act_out=(xq, xs, t))
    y_plain = Q.asp_layer(layer, x)
    xq2, xs2, t2 = Q.quantize_act(layer, x)
    y2 = Q.asp_linear(layer, xq2, xs2, t2)
    torch.cuda.synchronize()
    assert (xq.cpu().numpy() == ref["xq"]).all(), "packed activation bytes"
    assert (xs.cpu().numpy() == ref["sx"].T).all(), "activation scales"
    xt = O.smooth_activations(draws.x, ref["inv_lam"])
    check_t(bits(t), ref["t"], xt, factors["L1"])
    check_y(bits(y), ref["y"])
    assert (bits(y) == bits(y_plain)).all(), "optional outputs must not change y"
    same_t = (bits(t) == bits(t2)).all(axis=1)
    agree = (bits(y) == bits(y2)).all(axis=1)
    log(f"    tokens with identical t in both paths: {same_t.sum()}/{M}; identical y there: {agree[same_t].sum()}")
    # the fused kernel runs the two-call GEMM's arithmetic in the same order,
    # so every token with the same t has the same y, bit for bit
    assert agree[same_t].all(), f"tokens {np.flatnonzero(same_t & ~agree)[:8].tolist()} differ with equal t"


@pytest.mark.parametrize("M,N", I.ACTION_EXPERT_SHAPES)
def test_fused_action_expert_layers(M, N):
    d = I.action_expert(M, N)
    _fused_parity(d, oracle_factors(d))


@pytest.mark.parametrize("M,K,N,r,bias", [
    (1, 64, 16, 16, False),
    (7, 128, 48, 32, True),
    (33, 192, 144, 32, False),
    (64, 3072, 272, 32, True),
    (40, 16384, 64, 16, False),
    # M <= 16 runs the 16-token kernel: 65 spans (an odd count per wave), the
    # largest K
    (16, 4160, 80, 32, True),
    (3, 16384, 48, 16, False),
    # 16-token blocks with two or four weight blocks per workgroup (ragged
    # last token block and last column block), and the 32-token form once
    # more than 256 workgroups would be needed
    (48, 1024, 4160, 32, False),
    (32, 2048, 4096, 32, True),
    (64, 2048, 2304, 16, True),
    (64, 1024, 8192, 16, False),
    # N at the largest size the entry point takes
    (1, 64, 1 << 20, 16, False),
])
def test_fused_edge_shapes(M, K, N, r, bias):
    d = I.custom(M=M, K=K, N=N, r=r, seed=M * 23 + K, n_outliers=max(1, K // 100), with_bias=bias)
    _fused_parity(d, oracle_factors(d, r), d.bias)
