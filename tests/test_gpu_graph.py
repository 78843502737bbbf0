"""The entry points under HIP graph capture: one graph holds the layer calls
(both kernels; the deflated activation path; the rotated one with group 32;
the few-token fused layer, in its 16- and 32-token forms), others the AOG
accumulation and the eigensolve.  Each graph is replayed several times, with eager work and
synchronisations between the replays; every replay must give the eager calls'
outputs bit for bit, also after the captured input buffers have been
overwritten in place with new data.  The library records no memset and
allocates nothing, so a replay re-runs exactly the captured kernels.
"""

import numpy as np
import pytest
import torch

from paper_2609_33269_amd import inputs as I
from paper_2609_33269_amd import qwam as Q

from parity_helpers import bf16_dev, bits, f32_dev, gpu_layer, log, oracle_factors

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    Q.lib()


def _host(ts):
    return [bits(t) if t.dtype == torch.bfloat16 else t.cpu().numpy() for t in ts]


def _spoil(ts):
    """Eager work between replays: overwrite every output with a sentinel."""
    for t in ts:
        if t.dtype == torch.bfloat16:
            t.view(torch.int16).fill_(0x7FC1)          # a NaN no kernel writes
        elif t.dtype == torch.uint8:
            t.fill_(0xA5)
        else:
            t.fill_(-12345)


def _replays_match(graph, run_eager, outs, inputs, new_inputs, replays=3):
    """Eager reference, then `replays` replays against it; then the inputs are
    overwritten with `new_inputs` and a new eager reference is compared with
    one more replay."""
    _spoil(outs)
    run_eager()
    torch.cuda.synchronize()
    ref = _host(outs)
    for i in range(replays):
        _spoil(outs)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, (a, b) in enumerate(zip(_host(outs), ref)):
            assert (a == b).all(), f"replay {i}: output {k} differs from the eager call"
    for dst, src in zip(inputs, new_inputs):
        dst.copy_(src)
    _spoil(outs)
    run_eager()
    torch.cuda.synchronize()
    ref2 = _host(outs)
    assert any((a != b).any() for a, b in zip(ref2, ref)), "new inputs give new outputs"
    _spoil(outs)
    graph.replay()
    torch.cuda.synchronize()
    for k, (a, b) in enumerate(zip(_host(outs), ref2)):
        assert (a == b).all(), f"replay after new inputs: output {k} differs from the eager call"


def _acts(layer, M, dev):
    return (torch.empty((M, layer.K // 2), dtype=torch.uint8, device=dev),
            torch.empty((layer.K // layer.group, M), dtype=torch.float32, device=dev),
            torch.empty((M, layer.r), dtype=torch.bfloat16, device=dev))


def test_layer_calls_in_one_graph():
    dev = torch.device("cuda:0")
    big = I.custom(M=300, K=1024, N=384, r=32, seed=21, n_outliers=8, with_bias=True)
    rot = I.custom(M=130, K=2048, N=256, r=16, seed=22, n_outliers=10)
    few16 = I.custom(M=16, K=1024, N=512, r=16, seed=23, n_outliers=10, with_bias=True)
    few48 = I.custom(M=48, K=2048, N=4096, r=16, seed=24, n_outliers=20)
    layer = gpu_layer(oracle_factors(big), big.bias)
    layer_r = gpu_layer(dict(oracle_factors(rot, hadamard=True), group=32))
    layer_16 = gpu_layer(oracle_factors(few16), few16.bias)
    layer_48 = gpu_layer(oracle_factors(few48))
    x, xr, x16, x48 = bf16_dev(big.x), bf16_dev(rot.x), bf16_dev(few16.x), bf16_dev(few48.x)
    a1, a2, a3 = _acts(layer, big.shape.M, dev), _acts(layer, big.shape.M, dev), _acts(layer_r, rot.shape.M, dev)
    a16 = _acts(layer_16, 16, dev)
    y1 = torch.empty((big.shape.M, layer.N), dtype=torch.bfloat16, device=dev)
    y2, y3 = torch.empty_like(y1), torch.empty((rot.shape.M, layer_r.N), dtype=torch.bfloat16, device=dev)
    y16 = torch.empty((16, layer_16.N), dtype=torch.bfloat16, device=dev)
    y48 = torch.empty((48, layer_48.N), dtype=torch.bfloat16, device=dev)

    def run():
        Q.quantize_act(layer, x, out=a1)
        Q.asp_linear(layer, *a1, out=y1)
        Q.quantize_act_deflated(layer, x, out=a2)
        Q.asp_linear(layer, *a2, out=y2)
        Q.quantize_act(layer_r, xr, out=a3)
        Q.asp_linear(layer_r, *a3, out=y3)
        Q.asp_layer(layer_16, x16, out=y16, act_out=a16)
        Q.asp_layer(layer_48, x48, out=y48)

    log("  capture: quantize + linear (plain, deflated, rotated group 32), fused 16- and 48-token layers")
    run()                                                # first calls outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    outs = [*a1, y1, *a2, y2, *a3, y3, *a16, y16, y48]
    rng = np.random.default_rng(7)
    new = [bf16_dev(np.ascontiguousarray(v.x[rng.permutation(v.shape.M)])) for v in (big, rot, few16, few48)]
    _replays_match(g, run, outs, [x, xr, x16, x48], new)
    del g


def test_aog_calls_in_one_graph():
    """The accumulation adds to its captured accumulator on every replay: k
    replays equal k eager calls from the same start.  The eigensolve (with a
    caller-given workspace) reads the accumulator and overwrites V and the
    eigenvalues."""
    dev = torch.device("cuda:0")
    d, n, r = 1024, 512, 16
    rng = np.random.default_rng(31)
    col = np.exp(-np.arange(d) / (d / 8.0))
    gT = torch.from_numpy(rng.standard_normal((d, n)) * col[:, None]).to(torch.bfloat16).to(dev)
    A0 = torch.from_numpy(rng.standard_normal((d, 64))).to(dev)
    A0 = (A0 @ A0.T / 64 + 1e-3 * torch.eye(d, device=dev, dtype=torch.float64)).float()
    lam = f32_dev(np.exp(rng.uniform(-1.0, 1.0, d)))
    ws = torch.empty(Q.aog_protected_basis_workspace(d, r), dtype=torch.uint8, device=dev)
    A = A0.clone()

    log(f"  capture: aog accumulate d={d} n={n}")
    Q.aog_accumulate(gT, A0.clone())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        Q.aog_accumulate(gT, A)
    A_e = A0.clone()
    A.copy_(A0)
    for i in range(3):
        Q.aog_accumulate(gT, A_e)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(A, A_e), f"accumulation replay {i} differs from the eager call"
    del g

    log(f"  capture: eigensolve d={d} r={r} (Hadamard 64, smoothing)")
    Q.aog_protected_basis(A, r, iters=10, scale=1.0 / n, lam=lam, hadamard=64, workspace=ws)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        V, ev = Q.aog_protected_basis(A, r, iters=10, scale=1.0 / n, lam=lam, hadamard=64, workspace=ws)

    def eager():
        Ve, eve = Q.aog_protected_basis(A, r, iters=10, scale=1.0 / n, lam=lam, hadamard=64, workspace=ws)
        V.copy_(Ve)
        ev.copy_(eve)

    A_new = A0.clone()
    Q.aog_accumulate(gT, A_new)
    Q.aog_accumulate(gT, A_new)
    _replays_match(g, eager, [V, ev], [A], [A_new], replays=2)
    del g
