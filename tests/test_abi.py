"""The C ABI on the host: the library loads, exports every entry point that
include/qwam.h declares, and rejects bad arguments with the documented status
before any HIP call (no device memory is touched: the pointers below are
fake, never dereferenced)."""

import ctypes
import os
import re

import pytest
import torch

from paper_2609_33269_amd import qwam as Q

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("qwam.h", "qwam_probe.h")]

OK, INVALID, UNSUPPORTED, MISALIGNED, NO_DEVICE = 0, 1, 2, 3, 4
FAKE = 0x10000          # 16-byte aligned, never dereferenced


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(Q.LIB_PATH):
        from paper_2609_33269_amd import build
        build.build()
    return Q.lib()


def _declared_functions():
    names = set()
    for h in HEADERS:
        src = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(qwam_[a-z_]+)\s*\(", src))
    return sorted(names)


def test_exports_every_declared_symbol(lib):
    names = _declared_functions()
    assert set(names) == set(Q.SIGNATURES), "binding and header disagree"
    for n in names:
        assert hasattr(lib, n), n
    assert lib.qwam_abi_version() == 13
    assert lib.qwam_status_string(3) == b"QWAM_ERR_MISALIGNED"


def test_probe_argument_checks(lib):
    """The measurement probes reject bad arguments on the host."""
    assert lib.qwam_probe_mfma(99, 4, 4, FAKE, None) == INVALID
    assert lib.qwam_probe_mfma(0, 0, 4, FAKE, None) == INVALID
    assert lib.qwam_probe_mfma(0, 4, 4, None, None) == INVALID
    assert lib.qwam_probe_valu_fma(4, 0, FAKE, None) == INVALID
    assert lib.qwam_probe_copy(FAKE, FAKE, 24, 4, None) == INVALID
    assert lib.qwam_probe_copy(FAKE + 8, FAKE, 32, 4, None) == MISALIGNED
    assert lib.qwam_probe_copy(None, FAKE, 32, 4, None) == INVALID
    assert b"workgroups" in lib.qwam_probe_last_error() or b"bytes" in lib.qwam_probe_last_error() \
        or b"NULL" in lib.qwam_probe_last_error()


def _layer(K=256, N=256, r=16, group=64, hadamard=0, **ptrs):
    c = Q.QwamLayerC()
    c.K, c.N, c.r, c.group, c.hadamard = K, N, r, group, hadamard
    for f in ("wq", "ws", "wsp", "inv_smooth", "L1t", "L2t", "L1", "L1f"):
        setattr(c, f, ptrs.get(f, FAKE))
    c.bias = ptrs.get("bias", None)
    return c


def _act(lib, layer, M=64, x=FAKE, xq=FAKE, xs=FAKE, t=FAKE, deflated=False):
    fn = lib.qwam_quantize_act_deflated if deflated else lib.qwam_quantize_act
    return fn(ctypes.byref(layer), M, x, xq, xs, t, None)


def _lin(lib, layer, M=64, xq=FAKE, xs=FAKE, t=FAKE, y=FAKE):
    return lib.qwam_asp_linear(ctypes.byref(layer), M, xq, xs, t, y, None)


@pytest.mark.parametrize("K,N,group,status", [
    (256, 256, 16, INVALID), (256, 256, 128, INVALID), (96, 256, 32, INVALID), (100, 256, 64, INVALID), (0, 256, 64, INVALID), (256, 24, 64, INVALID),
    (256, 0, 64, INVALID), (-64, 256, 64, INVALID), (131072, 256, 64, UNSUPPORTED),
    (256, 1 << 21, 64, UNSUPPORTED)])
def test_pack_rejects_bad_shapes(lib, K, N, group, status):
    assert lib.qwam_pack_weights(K, N, group, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == status
    assert lib.qwam_last_error().startswith(b"qwam_pack_weights")


def test_pack_rejects_null_and_misaligned(lib):
    args = [FAKE] * 6
    for i in range(6):
        a = list(args); a[i] = None
        assert lib.qwam_pack_weights(256, 256, 64, *a, None) == INVALID
        a = list(args); a[i] = FAKE + 4
        assert lib.qwam_pack_weights(256, 256, 64, *a, None) == MISALIGNED


def test_layer_calls_reject_bad_arguments(lib):
    assert lib.qwam_quantize_act(None, 64, FAKE, FAKE, FAKE, FAKE, None) == INVALID
    for r in (0, 8, 24, 128):
        assert _act(lib, _layer(r=r)) == UNSUPPORTED
        assert _lin(lib, _layer(r=r)) == UNSUPPORTED
    for M, st in ((0, INVALID), (-3, INVALID), (1 << 21, UNSUPPORTED)):
        assert _act(lib, _layer(), M=M) == st
        assert _lin(lib, _layer(), M=M) == st
    assert _act(lib, _layer(group=128)) == INVALID
    assert _lin(lib, _layer(K=96)) == INVALID
    for f in ("inv_smooth", "L1t", "L1f"):
        assert _act(lib, _layer(**{f: None})) == INVALID
        assert _act(lib, _layer(**{f: FAKE + 2})) == MISALIGNED
    for f in ("wq", "ws", "wsp", "L2t"):
        assert _lin(lib, _layer(**{f: None})) == INVALID
        assert _lin(lib, _layer(**{f: FAKE + 8})) == MISALIGNED
    assert _lin(lib, _layer(bias=FAKE + 2)) == MISALIGNED
    for kw in ("x", "xq", "xs", "t"):
        assert _act(lib, _layer(), **{kw: None}) == INVALID
        assert _act(lib, _layer(), **{kw: FAKE + 1}) == MISALIGNED
    for kw in ("xq", "xs", "t", "y"):
        assert _lin(lib, _layer(), **{kw: None}) == INVALID
    msg = lib.qwam_last_error()
    assert msg.startswith(b"qwam_asp_linear") and b"y is NULL" in msg
    # the deflated activation call validates exactly like the plain one
    assert lib.qwam_quantize_act_deflated(None, 64, FAKE, FAKE, FAKE, FAKE, None) == INVALID
    for r in (0, 24):
        assert _act(lib, _layer(r=r), deflated=True) == UNSUPPORTED
    assert _act(lib, _layer(), M=0, deflated=True) == INVALID
    assert _act(lib, _layer(**{"L1t": FAKE + 2}), deflated=True) == MISALIGNED
    assert _act(lib, _layer(), t=None, deflated=True) == INVALID
    assert lib.qwam_last_error().startswith(b"qwam_quantize_act_deflated")
    # only the deflated call reads L1 ([K][r]): it must be set and aligned there
    assert _act(lib, _layer(L1=None), deflated=True) == INVALID
    assert b"L1 is NULL" in lib.qwam_last_error()
    assert _act(lib, _layer(L1=FAKE + 2), deflated=True) == MISALIGNED
    assert _act(lib, _layer(L1=None, hadamard=64), deflated=True) == INVALID
    assert _act(lib, _layer(L1=None)) in (OK, NO_DEVICE)
    # the rotation block: a power of two in [16, 1024] dividing K, or 0
    for B in (8, 2048, 96, 512):        # too small, too large, not a power of two, does not divide K = 256
        assert _act(lib, _layer(hadamard=B)) == INVALID
        assert _act(lib, _layer(hadamard=B), deflated=True) == INVALID
    assert b"hadamard" in lib.qwam_last_error()
    # partials: rank is not used, but shapes and pointers are checked
    assert lib.qwam_debug_group_partials(ctypes.byref(_layer(r=7)), 1, None, FAKE, None) == INVALID


def test_asp_layer_rejects_bad_arguments(lib):
    def call(layer, M=16, x=FAKE, y=FAKE, xq=None, xs=None, t=None):
        return lib.qwam_asp_layer(ctypes.byref(layer), M, x, y, xq, xs, t, None)
    assert call(_layer(), M=65) == UNSUPPORTED
    assert call(_layer(r=48)) == UNSUPPORTED
    assert call(_layer(group=32)) == UNSUPPORTED
    assert call(_layer(hadamard=256)) == UNSUPPORTED
    assert call(_layer(), M=0) == INVALID
    assert call(_layer(), x=None) == INVALID
    assert call(_layer(), y=FAKE + 2) == MISALIGNED
    assert call(_layer(), xq=FAKE) == INVALID          # xq without xs and t
    assert lib.qwam_last_error().startswith(b"qwam_asp_layer")


def test_aog_accumulate_rejects_bad_arguments(lib):
    for d, n, st in ((0, 64, INVALID), (24, 64, INVALID), (64, 0, INVALID), (64, 96, INVALID),
                     (32768, 64, UNSUPPORTED), (16384, 65536, UNSUPPORTED)):
        assert lib.qwam_aog_accumulate(d, n, FAKE, FAKE, None) == st, (d, n)
    assert lib.qwam_aog_accumulate(64, 64, None, FAKE, None) == INVALID
    assert lib.qwam_aog_accumulate(64, 64, FAKE, FAKE + 4, None) == MISALIGNED
    assert lib.qwam_last_error().startswith(b"qwam_aog_accumulate")


@pytest.mark.skipif(torch.cuda.device_count() > 0, reason="a GPU is visible: the no-device path cannot be forced")
def test_no_device_is_reported_before_any_launch(lib):
    assert lib.qwam_pack_weights(256, 256, 64, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == NO_DEVICE
    assert _act(lib, _layer()) == NO_DEVICE
    assert _act(lib, _layer(), deflated=True) == NO_DEVICE
    assert _lin(lib, _layer()) == NO_DEVICE
    assert lib.qwam_debug_group_partials(ctypes.byref(_layer()), 4, FAKE, FAKE, None) == NO_DEVICE
    assert lib.qwam_aog_accumulate(64, 64, FAKE, FAKE, None) == NO_DEVICE
    assert b"no HIP device" in lib.qwam_last_error()


def test_binding_rejects_host_tensors():
    layer = Q.PackedLayer(K=64, N=16, r=16, wq=torch.zeros(16, 32, dtype=torch.uint8),
                          ws=torch.zeros(1, 16), inv_smooth=torch.ones(64),
                          L1t=torch.zeros(16, 64, dtype=torch.bfloat16),
                          L2t=torch.zeros(16, 16, dtype=torch.bfloat16))
    with pytest.raises(ValueError, match="GPU tensor"):
        layer.c_struct()


def test_aog_protected_basis_argument_checks(lib):
    """Bad shapes, scale, rotation block, pointers and workspace size are
    rejected on the host with the documented status."""
    f = lib.qwam_aog_protected_basis
    need = lib.qwam_aog_protected_basis_workspace(4096, 32)
    assert need > 0 and lib.qwam_aog_protected_basis_workspace(100, 32) == -1
    assert lib.qwam_aog_protected_basis_workspace(4096, 49) == -1

    def call(d=4096, r=32, iters=8, A=FAKE, scale=1.0, lam=None, B=0, V=FAKE, ev=FAKE, ws=FAKE, wsb=None):
        return f(d, r, iters, A, scale, lam, B, V, ev, ws, need if wsb is None else wsb, None)

    assert call(d=4000) == INVALID
    assert call(d=64) == INVALID
    assert call(d=16384 + 64) == UNSUPPORTED
    assert call(r=0) == UNSUPPORTED and call(r=64) == UNSUPPORTED
    assert call(iters=-1) == INVALID
    assert call(scale=0.0) == INVALID and call(scale=float("nan")) == INVALID
    assert call(B=48) == INVALID and call(B=2048) == INVALID and call(B=8) == INVALID
    assert call(A=None) == INVALID and call(V=None) == INVALID and call(ev=None) == INVALID
    assert call(ws=None) == INVALID
    assert call(A=FAKE + 4) == MISALIGNED and call(lam=FAKE + 8) == MISALIGNED
    assert call(wsb=need - 1) == INVALID
    assert b"workspace" in lib.qwam_last_error()


@pytest.mark.parametrize("K,r", [(64, 16), (192, 32), (128, 48), (64, 64)])
def test_l1_fragment_order_matches_its_definition(K, r):
    """The binding's L1f layout against the header's definition, entry by entry:
    (g, b, h, l, e) = L1[64 g + 16 (l // 16) + 8 h + e][16 b + l % 16]."""
    L1 = torch.arange(K * r, dtype=torch.float32).reshape(K, r)
    F = Q.l1_fragment_order(L1)
    assert F.shape == (K // 64, r // 16, 2, 64, 8)
    for g in range(K // 64):
        for b in range(r // 16):
            for h in range(2):
                for l in range(64):
                    for e in range(8):
                        assert F[g, b, h, l, e] == L1[64 * g + 16 * (l // 16) + 8 * h + e, 16 * b + l % 16]
