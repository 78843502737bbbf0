"""Python binding of libqwam (ctypes): argument marshalling only.

Every step of the layer runs in the library's HIP kernels; this module checks
tensor devices, dtypes and shapes, allocates outputs with PyTorch and passes
raw device pointers plus the current HIP stream across the C ABI.  If the
library is not built, every call raises: there is no fallback.

Names follow the C ABI (include/qwam.h): pack_weights, quantize_act,
quantize_act_deflated, asp_linear, asp_layer, debug_group_partials,
aog_accumulate, aog_protected_basis; and the measurement probes of include/qwam_probe.h:
probe_mfma, probe_valu_fma, probe_copy, probe_empty.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

GROUP = 64
LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libqwam.so")

STATUS_NAMES = {0: "QWAM_OK", 1: "QWAM_ERR_INVALID_ARG", 2: "QWAM_ERR_UNSUPPORTED",
                3: "QWAM_ERR_MISALIGNED", 4: "QWAM_ERR_NO_DEVICE", 5: "QWAM_ERR_HIP"}

# every entry point the header declares, with (restype, argtypes)
_c_void_p, _i32 = ctypes.c_void_p, ctypes.c_int32


class QwamLayerC(ctypes.Structure):
    _fields_ = [("K", ctypes.c_int32), ("N", ctypes.c_int32), ("r", ctypes.c_int32),
                ("group", ctypes.c_int32), ("hadamard", ctypes.c_int32), ("wq", ctypes.c_void_p), ("ws", ctypes.c_void_p),
                ("inv_smooth", ctypes.c_void_p), ("L1t", ctypes.c_void_p),
                ("L2t", ctypes.c_void_p), ("bias", ctypes.c_void_p), ("L1", ctypes.c_void_p),
                ("wsp", ctypes.c_void_p), ("L1f", ctypes.c_void_p)]


_LP = ctypes.POINTER(QwamLayerC)
SIGNATURES = {
    "qwam_pack_weights": (ctypes.c_int, [_i32, _i32, _i32, _c_void_p, _c_void_p, _c_void_p,
                                         _c_void_p, _c_void_p, _c_void_p, _c_void_p]),
    "qwam_quantize_act": (ctypes.c_int, [_LP, _i32, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
                                         _c_void_p]),
    "qwam_quantize_act_deflated": (ctypes.c_int, [_LP, _i32, _c_void_p, _c_void_p, _c_void_p,
                                                  _c_void_p, _c_void_p]),
    "qwam_asp_linear": (ctypes.c_int, [_LP, _i32, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
                                       _c_void_p]),
    "qwam_debug_group_partials": (ctypes.c_int, [_LP, _i32, _c_void_p, _c_void_p, _c_void_p]),
    "qwam_asp_layer": (ctypes.c_int, [_LP, _i32, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
                                      _c_void_p]),
    "qwam_aog_accumulate": (ctypes.c_int, [_i32, _i32, _c_void_p, _c_void_p, _c_void_p]),
    "qwam_aog_protected_basis": (ctypes.c_int, [_i32, _i32, _i32, _c_void_p, ctypes.c_float, _c_void_p, _i32,
                                                _c_void_p, _c_void_p, _c_void_p, ctypes.c_int64, _c_void_p]),
    "qwam_aog_protected_basis_workspace": (ctypes.c_int64, [_i32, _i32]),
    "qwam_last_error": (ctypes.c_char_p, []),
    "qwam_probe_mfma": (ctypes.c_int, [_i32, _i32, _i32, _c_void_p, _c_void_p]),
    "qwam_probe_valu_fma": (ctypes.c_int, [_i32, _i32, _c_void_p, _c_void_p]),
    "qwam_probe_copy": (ctypes.c_int, [_c_void_p, _c_void_p, ctypes.c_int64, _i32, _c_void_p]),
    "qwam_probe_empty": (ctypes.c_int, [_c_void_p]),
    "qwam_probe_last_error": (ctypes.c_char_p, []),
    "qwam_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "qwam_abi_version": (ctypes.c_int32, []),
}

_lib = None


class QwamError(RuntimeError):
    def __init__(self, fn: str, status: int, message: str):
        super().__init__(f"{fn} -> {STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


def lib() -> ctypes.CDLL:
    """Load libqwam.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2609_33269_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(handle, name)
            f.restype = res
            f.argtypes = args
        _lib = handle
    return _lib


def _check(fn: str, status: int) -> None:
    if status != 0:
        raise QwamError(fn, status, lib().qwam_last_error().decode())


def _stream_ptr(stream) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return int(s.cuda_stream)


def _req(t: torch.Tensor, name: str, dtype: torch.dtype, shape) -> int:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor (got {t.device})")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)} (got {tuple(t.shape)})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


@dataclass
class PackedLayer:
    """Device tensors of one packed ASP layer (see include/qwam.h for layouts)."""
    K: int
    N: int
    r: int
    wq: torch.Tensor          # uint8 [N][K/2]
    ws: torch.Tensor          # float32 [K/64][N]
    inv_smooth: torch.Tensor  # float32 [K]
    L1t: torch.Tensor         # bf16 [r][K]
    L2t: torch.Tensor         # bf16 [N][r]
    bias: Optional[torch.Tensor] = None   # bf16 [N]
    hadamard: int = 0                     # block size of the rotation (Eq. 3), 0 = none
    group: int = GROUP                    # channels per scale: 64, or 32 (App. B.1)
    L1: Optional[torch.Tensor] = None     # bf16 [K][r] (the deflated activation path reads it)
    wsp: Optional[torch.Tensor] = None    # int32 [K/group][N]: ws as bf16 pieces hi | lo << 16 (asp_linear reads it)
    L1f: Optional[torch.Tensor] = None    # bf16 [K/64][r/16][2][64][8]: L1 in fragment order (the activation calls read it)

    def c_struct(self) -> QwamLayerC:
        G = self.K // self.group
        c = QwamLayerC()
        c.K, c.N, c.r, c.group, c.hadamard = self.K, self.N, self.r, self.group, self.hadamard
        c.wq = _req(self.wq, "wq", torch.uint8, (self.N, self.K // 2))
        c.ws = _req(self.ws, "ws", torch.float32, (G, self.N))
        c.inv_smooth = _req(self.inv_smooth, "inv_smooth", torch.float32, (self.K,))
        c.L1t = _req(self.L1t, "L1t", torch.bfloat16, (self.r, self.K))
        c.L2t = _req(self.L2t, "L2t", torch.bfloat16, (self.N, self.r))
        c.bias = None if self.bias is None else _req(self.bias, "bias", torch.bfloat16, (self.N,))
        c.L1 = None if self.L1 is None else _req(self.L1, "L1", torch.bfloat16, (self.K, self.r))
        c.wsp = None if self.wsp is None else _req(self.wsp, "wsp", torch.int32, (G, self.N))
        c.L1f = None if self.L1f is None else _req(self.L1f, "L1f", torch.bfloat16,
                                                   (self.K // 64, self.r // 16, 2, 64, 8))
        return c


def pack_weights(R: torch.Tensor, smooth: torch.Tensor, stream=None, group: int = GROUP):
    """qwam_pack_weights: R float32 [N][K], smooth float32 [K] ->
    (wq uint8 [N][K/2], ws float32 [K/group][N], wsp int32 [K/group][N] (the
    scales as bf16 pieces hi | lo << 16), inv_smooth float32 [K])."""
    N, K = R.shape
    dev = R.device
    wq = torch.empty((N, K // 2), dtype=torch.uint8, device=dev)
    ws = torch.empty((K // group, N), dtype=torch.float32, device=dev)
    wsp = torch.empty((K // group, N), dtype=torch.int32, device=dev)
    inv = torch.empty((K,), dtype=torch.float32, device=dev)
    st = lib().qwam_pack_weights(K, N, group, _req(R, "R", torch.float32, (N, K)),
                                 _req(smooth, "smooth", torch.float32, (K,)),
                                 wq.data_ptr(), ws.data_ptr(), wsp.data_ptr(), inv.data_ptr(), _stream_ptr(stream))
    _check("qwam_pack_weights", st)
    return wq, ws, wsp, inv


def l1_fragment_order(L1: torch.Tensor) -> torch.Tensor:
    """L1 bf16 [K][r] -> the activation kernels' fragment order
    [K/64][r/16][2][64][8]: entry (g, b, h, l, e) = L1[64 g + 16 (l // 16) + 8 h + e][16 b + l % 16]
    (a layout change only, like the transposes of L1 and L2)."""
    K, r = L1.shape
    v = L1.reshape(K // 64, 4, 2, 8, r // 16, 16)           # [g][c][h][e][b][j], l = 16 c + j
    return v.permute(0, 4, 2, 1, 5, 3).contiguous().reshape(K // 64, r // 16, 2, 64, 8)


def make_layer(R: torch.Tensor, smooth: torch.Tensor, L1: torch.Tensor, L2: torch.Tensor,
               bias: Optional[torch.Tensor] = None, stream=None, hadamard: int = 0,
               group: int = GROUP) -> PackedLayer:
    """Pack R and lambda and lay out the branch factors: L1 bf16 [K][r] and
    L2 bf16 [r][N] are stored transposed (L1t [r][K], L2t [N][r]), and L1 also
    as given (the deflated activation path reads its rows).  With
    `hadamard` = B, R, L1 and L2 must be those of the rotated layer (Eq. 3)."""
    N, K = R.shape
    r = L1.shape[1]
    wq, ws, wsp, inv = pack_weights(R, smooth, stream, group)
    return PackedLayer(K=K, N=N, r=r, wq=wq, ws=ws, wsp=wsp, inv_smooth=inv,
                       L1t=L1.t().contiguous(), L2t=L2.t().contiguous(), L1=L1.contiguous(),
                       L1f=l1_fragment_order(L1),
                       bias=None if bias is None else bias.contiguous(), hadamard=hadamard, group=group)


def quantize_act(layer: PackedLayer, x: torch.Tensor, stream=None, out=None):
    """qwam_quantize_act: x bf16 [M][K] -> (xq uint8 [M][K/2], xs float32 [K/64][M], t bf16 [M][r]).

    `out` may give the three output tensors (preallocated, e.g. for a benchmark loop)."""
    return _quantize(lib().qwam_quantize_act, "qwam_quantize_act", layer, x, stream, out)


def quantize_act_deflated(layer: PackedLayer, x: torch.Tensor, stream=None, out=None):
    """qwam_quantize_act_deflated: as quantize_act, but the codes are those of
    the deflated activation x~ - L1 t (Eq. 8 / Eq. 9)."""
    return _quantize(lib().qwam_quantize_act_deflated, "qwam_quantize_act_deflated", layer, x, stream, out)


def _quantize(fn, name: str, layer: PackedLayer, x: torch.Tensor, stream, out):
    M = x.shape[0]
    dev = x.device
    if out is None:
        xq = torch.empty((M, layer.K // 2), dtype=torch.uint8, device=dev)
        xs = torch.empty((layer.K // layer.group, M), dtype=torch.float32, device=dev)
        t = torch.empty((M, layer.r), dtype=torch.bfloat16, device=dev)
    else:
        xq, xs, t = out
    c = layer.c_struct()
    st = fn(ctypes.byref(c), M, _req(x, "x", torch.bfloat16, (M, layer.K)),
            _req(xq, "xq", torch.uint8, (M, layer.K // 2)),
            _req(xs, "xs", torch.float32, (layer.K // layer.group, M)),
            _req(t, "t", torch.bfloat16, (M, layer.r)), _stream_ptr(stream))
    _check(name, st)
    return xq, xs, t


def asp_linear(layer: PackedLayer, xq: torch.Tensor, xs: torch.Tensor, t: torch.Tensor,
               out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """qwam_asp_linear: -> y bf16 [M][N]."""
    M = xq.shape[0]
    G = layer.K // layer.group
    y = torch.empty((M, layer.N), dtype=torch.bfloat16, device=xq.device) if out is None else out
    c = layer.c_struct()
    st = lib().qwam_asp_linear(ctypes.byref(c), M, _req(xq, "xq", torch.uint8, (M, layer.K // 2)),
                               _req(xs, "xs", torch.float32, (G, M)),
                               _req(t, "t", torch.bfloat16, (M, layer.r)),
                               _req(y, "y", torch.bfloat16, (M, layer.N)), _stream_ptr(stream))
    _check("qwam_asp_linear", st)
    return y


def forward(layer: PackedLayer, x: torch.Tensor, stream=None, deflate: bool = False) -> torch.Tensor:
    """Both kernels of one layer call: quantize_act (or quantize_act_deflated)
    then asp_linear."""
    xq, xs, t = (quantize_act_deflated if deflate else quantize_act)(layer, x, stream)
    return asp_linear(layer, xq, xs, t, stream=stream)


def asp_layer(layer: PackedLayer, x: torch.Tensor, out=None, act_out=None, stream=None):
    """qwam_asp_layer: the whole layer for M <= 64 tokens in one launch.
    x bf16 [M][K] -> y bf16 [M][N].  `act_out` = (xq, xs, t) receives the
    activation step's outputs as well (optional)."""
    M = x.shape[0]
    y = torch.empty((M, layer.N), dtype=torch.bfloat16, device=x.device) if out is None else out
    c = layer.c_struct()
    if act_out is None:
        pq = ps = pt = None
    else:
        xq, xs, t = act_out
        pq = _req(xq, "xq", torch.uint8, (M, layer.K // 2))
        ps = _req(xs, "xs", torch.float32, (layer.K // layer.group, M))
        pt = _req(t, "t", torch.bfloat16, (M, layer.r))
    st = lib().qwam_asp_layer(ctypes.byref(c), M, _req(x, "x", torch.bfloat16, (M, layer.K)),
                              _req(y, "y", torch.bfloat16, (M, layer.N)), pq, ps, pt, _stream_ptr(stream))
    _check("qwam_asp_layer", st)
    return y


def debug_group_partials(layer: PackedLayer, xq: torch.Tensor, stream=None) -> torch.Tensor:
    """qwam_debug_group_partials: -> P int32 [M][N][K/group] (exact integer partials)."""
    M = xq.shape[0]
    G = layer.K // layer.group
    P = torch.empty((M, layer.N, G), dtype=torch.int32, device=xq.device)
    c = layer.c_struct()
    st = lib().qwam_debug_group_partials(ctypes.byref(c), M,
                                         _req(xq, "xq", torch.uint8, (M, layer.K // 2)),
                                         P.data_ptr(), _stream_ptr(stream))
    _check("qwam_debug_group_partials", st)
    return P


def aog_accumulate(gT: torch.Tensor, A: torch.Tensor, stream=None) -> torch.Tensor:
    """qwam_aog_accumulate: A float32 [d][d] += gT gT^T for a batch of probe
    VJPs gT bf16 [d][n] (row c = channel c).  Returns A (updated in place)."""
    d, n = gT.shape
    st = lib().qwam_aog_accumulate(d, n, _req(gT, "gT", torch.bfloat16, (d, n)),
                                   _req(A, "A", torch.float32, (d, d)), _stream_ptr(stream))
    _check("qwam_aog_accumulate", st)
    return A


def aog_protected_basis_workspace(d: int, r: int) -> int:
    """qwam_aog_protected_basis_workspace: bytes of workspace for (d, r)."""
    n = lib().qwam_aog_protected_basis_workspace(d, r)
    if n < 0:
        raise QwamError("qwam_aog_protected_basis_workspace", 2, lib().qwam_last_error().decode())
    return int(n)


def aog_protected_basis(A: torch.Tensor, r: int, iters: int = 20, scale: float = 1.0,
                        lam: Optional[torch.Tensor] = None, hadamard: int = 0,
                        workspace: Optional[torch.Tensor] = None, stream=None):
    """qwam_aog_protected_basis: top-r eigenvectors V float32 [d][r] and
    eigenvalues float32 [r] (descending) of scale * H diag(lam) A diag(lam) H.
    `workspace` (uint8, at least aog_protected_basis_workspace(d, r) bytes) is
    allocated here when not given."""
    d = A.shape[0]
    need = aog_protected_basis_workspace(d, r)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=A.device)
    if workspace.dtype != torch.uint8 or not workspace.is_contiguous() or not workspace.is_cuda:
        raise ValueError("workspace must be a contiguous uint8 GPU tensor")
    V = torch.empty((d, r), dtype=torch.float32, device=A.device)
    ev = torch.empty((r,), dtype=torch.float32, device=A.device)
    st = lib().qwam_aog_protected_basis(d, r, iters, _req(A, "A", torch.float32, (d, d)), float(scale),
                                        None if lam is None else _req(lam, "lam", torch.float32, (d,)),
                                        hadamard, V.data_ptr(), ev.data_ptr(), workspace.data_ptr(),
                                        workspace.numel(), _stream_ptr(stream))
    _check("qwam_aog_protected_basis", st)
    return V, ev


# ---------------------------------------------------------------------------
# measurement probes (include/qwam_probe.h): not part of the layer
# ---------------------------------------------------------------------------

PROBE_MFMA_KINDS = {"fp6": (0, 64, 1), "fp8": (1, 64, 1), "fp4": (2, 64, 1), "i8": (3, 32, 1),
                    "bf16": (4, 16, 1), "bf16_2b": (5, 4, 2)}   # name -> (kind, K, blocks per instruction)


def _probe_check(fn: str, status: int) -> None:
    if status != 0:
        raise QwamError(fn, status, lib().qwam_probe_last_error().decode())


def probe_mfma(kind: str, workgroups: int, iters: int, out: torch.Tensor, stream=None) -> float:
    """qwam_probe_mfma; returns the operations the launch performs."""
    code, k, blocks = PROBE_MFMA_KINDS[kind]
    _req(out, "out", torch.float32, (workgroups * 256,))
    _probe_check("qwam_probe_mfma", lib().qwam_probe_mfma(code, workgroups, iters, out.data_ptr(),
                                                          _stream_ptr(stream)))
    return float(workgroups) * 4 * 4 * iters * 2 * 32 * 32 * k * blocks


def probe_valu_fma(workgroups: int, iters: int, out: torch.Tensor, stream=None) -> float:
    """qwam_probe_valu_fma; returns the flops the launch performs."""
    _req(out, "out", torch.float32, (workgroups * 256,))
    _probe_check("qwam_probe_valu_fma", lib().qwam_probe_valu_fma(workgroups, iters, out.data_ptr(),
                                                                  _stream_ptr(stream)))
    return float(workgroups) * 256 * 256 * iters * 2


def probe_copy(src: torch.Tensor, dst: torch.Tensor, workgroups: int = 4096, stream=None) -> int:
    """qwam_probe_copy of all of src into dst (same size); returns the HBM bytes moved."""
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nbytes or not (src.is_cuda and dst.is_cuda):
        raise ValueError("probe_copy: src and dst must be GPU tensors of the same size")
    _probe_check("qwam_probe_copy", lib().qwam_probe_copy(src.data_ptr(), dst.data_ptr(), nbytes, workgroups,
                                                          _stream_ptr(stream)))
    return 2 * nbytes


def probe_empty(stream=None) -> None:
    """qwam_probe_empty: one empty launch."""
    _probe_check("qwam_probe_empty", lib().qwam_probe_empty(_stream_ptr(stream)))
