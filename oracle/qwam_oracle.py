"""CPU oracle for the Action-Subspace-Protected (ASP) linear layer.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with
the GPU library and never imports it.

It is a plain, slow, step-by-step restatement of what the paper
"Q-WAM: 4-Bit Quantization of World Action Models with Action-Subspace
Protection" computes for one quantized linear layer, written with numpy in
float64 / int64 (float32 where the method's rounding points are float32).
Library primitives used as single steps: matmul (float64; exact whenever every
operand and partial sum is an integer below 2**53), svd / eigh, frexp, rint.

Paper references used below
  Eq. 2   symmetric b-bit group quantizer (Sec. 3, "Post-Training Quantization")
  Eq. 3   smoothing + rotation pair, W~^T x~ = W^T x (Sec. 3)
  Eq. 7   eigen-decomposition of the (rotated) Gramian (Sec. 4.2)
  Eq. 8   split of x~ into V(V^T x~) + x~_perp (Sec. 4.2, "Splitting the layer")
  Eq. 9   ASP layer: (V^T W~)^T (V^T x~) + Q4(W~_perp)^T Q4(x~_perp) (Sec. 4.2)
  Prop. "Optimal protected subspace" (App. A.3, Ky Fan maximum principle)
  App. B.1 "Quantization settings and kernels": symmetric round-to-nearest,
      one scale per group of consecutive input channels, codes in [-8, 7],
      activation scale = group absmax / 7 per token, smoothing factor
      s_j = max|X_j|^a / max|W_:,j|^(1-a) with a = 0.5, divide the activation by
      s and multiply the weight by s; the fused kernels differ from the
      reference rule only in floating-point accumulation order.

Readings taken where the paper is silent (all are listed in the design notes):
  * group = 64 along K (the paper's 32 is the group-32 variant, `group`
    arguments below); scales are float32 in both; rounding is half-to-even;
    scale = fl32(absmax / 7), codes = clamp(rint(fl32(v * fl32(1/scale))), -8, 7);
    a group whose absmax is below 7 * 2**-126 gets scale 0 and all codes 0.
  * the activation is smoothed by multiplying with fl32(1/lambda) (the
    reciprocal is formed once, at weight-pack time).
  * the block Hadamard rotation of Eq. 3 is optional (App. B.1 applies it;
    the default path of this layer does not).  Block B = the largest power of
    two dividing K, at most 1024 (App. B.1); the weight side is rotated
    offline in float64; the activation side runs the fast Walsh-Hadamard
    transform in float32, one rounding per butterfly, stages on element bit
    0, 1, .., log2(B)-1 in that order, then multiplies by fl32(1/sqrt(B))
    (exact when B is a power of 4, e.g. 1024) (rotate_activations).
  * the 4-bit path quantizes either x~ itself (the default) or, in the
    deflated variant, x~_perp of Eq. 8 / Eq. 9; in exact arithmetic both give
    x~ W~_perp (Eq. 9 and R^T V = 0).  Deflation subtracts the bf16 branch's
    own rank-r part, t_j * L1[:, j], from x~ one direction at a time, j in
    ascending order, each step rounded to float32 (deflate_activations); each
    product of two bf16 values is exact in float32, so every step is one
    correctly rounded subtraction.
  * packing: 4 bits per code, sixteen codes per 8-byte block (pack_codes);
    the paper fixes the code range, not a byte layout.  Each code is stored as
    the sign and magnitude of the rounded scaled value (negative zero keeps
    its sign bit) in a 6-bit field with two zero bits, and the fields of a
    block are laid out so that those zero bits hold the block's last 32
    stream bits (format above pack_codes).  Needs |code| <= 7, which the
    quantizer guarantees.
  * the 16-bit branch is bf16: L1 = bf16(V), L2 = bf16(L1^T W~),
    R = fl32(W~ - L1 L2), t = bf16(sum_k bf16(x~_k) L1[k, j]) with an exact sum.
  * output reference y = sum_g sx sw P + t L2 (+ bias), float64, not rounded.

Layouts: x [M][K]; w, R [N][K] (row = output channel, i.e. the paper's W
transposed); codes [rows][K] int8; scales [rows][G] float32 (G = K / 64);
packed [rows][K/2] uint8; L1 [K][r]; L2 [r][N]; t [M][r]; P [M][N][G].
"""

from __future__ import annotations

import numpy as np

GROUP = 64
QMAX = 7          # 2**(4-1) - 1  (Eq. 2 with b = 4)
CODE_MIN, CODE_MAX = -8, 7
ALPHA = 0.5       # smoothing strength (App. B.1)
RIDGE = 1e-3      # the stand-in Gramian is A A^T / K + RIDGE * I

# ----------------------------------------------------------------------------
# bf16 helpers (round to nearest, ties to even)
# ----------------------------------------------------------------------------


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Value of bf16 bit patterns, as float64 (exact)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def round_to_bf16(v: np.ndarray) -> np.ndarray:
    """Round float32/float64 values to the nearest bf16 value, ties to even.

    Written from the definition: bf16 keeps 8 significant bits; the quantum of
    a normal value with exponent e (v = f * 2**e, 0.5 <= |f| < 1) is 2**(e-8);
    below 2**-126 the quantum is fixed at 2**-133.  Returns float64 values.
    """
    v = np.asarray(v, dtype=np.float64)
    _, e = np.frexp(v)
    e = np.maximum(e, -125)            # |v| < 2**-126  ->  subnormal quantum 2**-133
    q = np.ldexp(np.ones_like(v), e - 8)
    out = np.rint(v / q) * q           # v / q exact (power of two), rint ties to even
    return out


def f64_to_bf16_bits(v: np.ndarray) -> np.ndarray:
    """bf16 bit patterns of round_to_bf16(v)."""
    r = round_to_bf16(v).astype(np.float32)    # exact: r is representable in bf16
    return (r.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


# ----------------------------------------------------------------------------
# Offline construction of one ASP layer (Sec. 3, Sec. 4.2, App. B.1)
# ----------------------------------------------------------------------------


def smoothing_factors(x: np.ndarray, w: np.ndarray, alpha: float = ALPHA) -> np.ndarray:
    """Per-input-channel smoothing factor (App. B.1, Eq. 13).

    s_k = max_m |X[m, k]|**alpha / max_n |W[n, k]|**(1 - alpha), computed in
    float64 and stored as float32.  A channel whose activation or weight
    maximum is zero gets factor 1 (the formula is undefined there).
    x: float [M][K] activation values; w: float [N][K] weight values.
    """
    xmax = np.max(np.abs(np.asarray(x, dtype=np.float64)), axis=0)
    wmax = np.max(np.abs(np.asarray(w, dtype=np.float64)), axis=0)
    ok = (xmax > 0) & (wmax > 0)
    s = np.ones_like(xmax)
    s[ok] = xmax[ok] ** alpha / wmax[ok] ** (1.0 - alpha)
    return s.astype(np.float32)


def gramian(a: np.ndarray) -> np.ndarray:
    """The SPD stand-in for the layer's Gramian: G = A A^T / K + RIDGE * I."""
    a = np.asarray(a, dtype=np.float64)
    K = a.shape[0]
    return a @ a.T / K + RIDGE * np.eye(K)


def _fix_signs(V: np.ndarray) -> np.ndarray:
    """Eigenvectors are defined up to sign: make the largest-|entry| of each column positive."""
    V = V.copy()
    idx = np.argmax(np.abs(V), axis=0)
    sgn = np.sign(V[idx, np.arange(V.shape[1])])
    sgn[sgn == 0] = 1.0
    return V * sgn[None, :]


def protected_basis_eigh(G: np.ndarray, r: int):
    """Top-r eigenvectors of a symmetric PSD G (Eq. 7), by the definition.

    Returns (V [K][r] with orthonormal columns, eigenvalues of G sorted
    descending).  The span of V is the layer's action subspace (Sec. 4.2).
    """
    evals, evecs = np.linalg.eigh(np.asarray(G, dtype=np.float64))
    order = np.argsort(evals)[::-1]
    evals = evals[order]
    V = _fix_signs(evecs[:, order[:r]])
    return V, evals


def protected_basis_from_factor(a: np.ndarray, r: int) -> np.ndarray:
    """Top-r eigenvectors of G = A A^T / K + RIDGE * I without forming G.

    The eigenvectors of A A^T are the left singular vectors of A (eigenvalue
    sigma**2 / K + RIDGE, so the order is the singular-value order); the ridge
    shifts eigenvalues, not eigenvectors.  Requires r <= number of columns of A:
    the first 64 eigenvalues exceed the flat ridge part, so the top-r space is
    unique.
    """
    U, S, _ = np.linalg.svd(np.asarray(a, dtype=np.float64), full_matrices=False)
    assert r <= a.shape[1], "rank must not exceed the Gramian factor's width"
    return _fix_signs(U[:, :r])


def hadamard_block(K: int) -> int:
    """Block size of the rotation: the largest power of two dividing K, at most
    1024 (App. B.1)."""
    if K <= 0:
        raise ValueError("K must be positive")
    return min(K & -K, 1024)


def sylvester_hadamard(B: int) -> np.ndarray:
    """The +-1 Hadamard matrix of order B (a power of two) by Sylvester's
    doubling H_2n = [[H, H], [H, -H]]; symmetric, H H = B I."""
    H = np.ones((1, 1))
    while H.shape[0] < B:
        H = np.block([[H, H], [H, -H]])
    if H.shape[0] != B:
        raise ValueError("B must be a power of two")
    return H


def rotate_exact(v: np.ndarray, B: int) -> np.ndarray:
    """Row vectors times the orthonormal block Hadamard matrix diag(H_B, ..)/sqrt(B),
    float64 (Eq. 3's H; H is symmetric, so x H = (H x^T)^T)."""
    v = np.asarray(v, dtype=np.float64)
    rows, K = v.shape
    H = sylvester_hadamard(B) / np.sqrt(B)
    return (v.reshape(rows, K // B, B) @ H).reshape(rows, K)


def rotation_block(K: int, hadamard) -> int:
    """Block size of the rotation: 0 for none (False / 0), App. B.1's block for
    True, or the given power of two (which must divide K)."""
    if hadamard is True:
        return hadamard_block(K)
    B = int(hadamard)
    if B and (B & (B - 1) or K % B):
        raise ValueError("the rotation block must be a power of two dividing K")
    return B


def build_layer(x_bits: np.ndarray, w_bits: np.ndarray, V: np.ndarray, hadamard=False):
    """Deployed ASP factors of one layer from bf16 x [M][K], bf16 w [N][K] and
    a protected basis V [K][r] (float64, orthonormal columns).  `hadamard`:
    False, True (the block of App. B.1) or a block size B.

    Steps (Sec. 3 Eq. 3, Sec. 4.2 Eq. 9, App. B.1):
      lambda = smoothing factors (float32)
      W~[n, k] = lambda_k * W[n, k]                       (float64)
      with `hadamard`: W~ = W~ H (row n rotated blockwise, Eq. 3), and V is
      a basis of the rotated coordinates
      L1 = bf16(V)                                        [K][r]
      L2 = bf16(L1^T W~)     (the paper's V^T W~)         [r][N]
      R  = fl32(W~ - L1 L2)  (the paper's W~_perp, here built against the
                               rounded factors, so W~ = R + L1 L2 up to fl32)
    Returns a dict of numpy arrays: lam (f32 [K]), L1 (bf16 bits [K][r]),
    L2 (bf16 bits [r][N]), R (f32 [N][K]), and hadamard (the block size B, or
    0 without rotation).
    """
    x = bf16_bits_to_f64(x_bits)
    w = bf16_bits_to_f64(w_bits)
    lam = smoothing_factors(x, w)
    wt = w * lam.astype(np.float64)[None, :]                  # [N][K]
    B = rotation_block(wt.shape[1], hadamard)
    if B:
        wt = rotate_exact(wt, B)
    L1 = f64_to_bf16_bits(V)                                  # [K][r]
    L1f = bf16_bits_to_f64(L1)
    L2 = f64_to_bf16_bits(L1f.T @ wt.T)                       # [r][N]
    L2f = bf16_bits_to_f64(L2)
    R = (wt - (L1f @ L2f).T).astype(np.float32)               # [N][K]
    return {"lam": lam, "L1": L1, "L2": L2, "R": R, "hadamard": B}


def build_layer_exact(x: np.ndarray, w: np.ndarray, V: np.ndarray, hadamard: bool = False):
    """Exact-mode factors (float64 throughout, nothing rounded).

    lam (float64, by the formula), V, VtW = V^T W~ [r][N], R = (I - V V^T) W~
    stored [N][K] (Sec. 4.2: W~_perp); with `hadamard`, W~ is rotated (Eq. 3).
    """
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    xmax = np.max(np.abs(x), axis=0)
    wmax = np.max(np.abs(w), axis=0)
    ok = (xmax > 0) & (wmax > 0)
    lam = np.ones_like(xmax)
    lam[ok] = xmax[ok] ** ALPHA / wmax[ok] ** (1.0 - ALPHA)
    wt = w * lam[None, :]
    B = hadamard_block(wt.shape[1]) if hadamard else 0
    if B:
        wt = rotate_exact(wt, B)
    VtW = V.T @ wt.T                                          # [r][N]
    R = wt - (V @ VtW).T                                      # [N][K]
    return {"lam": lam, "V": V, "VtW": VtW, "R": R, "hadamard": B}


# ----------------------------------------------------------------------------
# The quantizer (Eq. 2) and packing
# ----------------------------------------------------------------------------


def quantize_groups(v: np.ndarray, group: int = GROUP, dtype=np.float32):
    """Symmetric 4-bit group quantizer of Eq. 2, one scale per `group`
    consecutive entries of each row.

    In precision `dtype` (float32 for the deployed layer):
      a = max |v| over the group                   (exact)
      a < 7 * 2**-126  ->  scale 0, codes 0        (guards 0 * inf)
      scale = fl(a / 7)
      inv   = fl(1 / scale)
      code  = clamp(rint(fl(v * inv)), -8, 7)      (rint: ties to even)
    Returns codes int8 [rows][K] and scales `dtype` [rows][K/group].
    """
    codes, scale, _ = quantize_groups_signed(v, group, dtype)
    return codes, scale


def quantize_groups_signed(v: np.ndarray, group: int = GROUP, dtype=np.float32):
    """quantize_groups, plus the IEEE sign of every rounded scaled value
    rint(x), x = fl(v * inv) (bool [rows][K]; rint keeps the sign of x, so
    rint(-0.3) = -0.0 counts as negative; with scale 0, inv is 0 and x = v * 0).
    The packed format stores each code as the sign and magnitude of rint(x),
    so a zero code keeps this sign."""
    v = np.asarray(v, dtype=dtype)
    rows, K = v.shape
    assert K % group == 0
    G = K // group
    vg = v.reshape(rows, G, group)
    a = np.max(np.abs(vg), axis=2)
    small = a < dtype(QMAX * 2.0 ** -126)
    scale = (a / dtype(QMAX)).astype(dtype)
    scale[small] = 0
    inv = np.zeros_like(scale)
    inv[~small] = dtype(1) / scale[~small]
    prod = (vg * inv[:, :, None]).astype(dtype)
    rounded = np.rint(prod)
    codes = np.clip(rounded, CODE_MIN, CODE_MAX).astype(np.int8)
    codes[small] = 0
    return codes.reshape(rows, K), scale, np.signbit(rounded).reshape(rows, K)


def dequantize_groups(codes: np.ndarray, scales: np.ndarray, group: int = GROUP) -> np.ndarray:
    """Q_b(X) = scale * code (Eq. 2), float64."""
    rows, K = codes.shape
    c = codes.astype(np.float64).reshape(rows, K // group, group)
    return (c * np.asarray(scales, dtype=np.float64)[:, :, None]).reshape(rows, K)


# Code blocks (the packed format of the codes; the paper fixes the code range,
# not a byte layout).  Sixteen codes c_0 .. c_15 of consecutive channels form
# one 8-byte block, two little-endian 32-bit words W0, W1.  Code j is written
# as the 6-bit field F_j: bit 5 the sign, bits 3-4 zero, bits 0-2 the
# magnitude |c_j|; F_j occupies bits 6j .. 6j+5 of a 96-bit stream.  Stream
# bits 0-31 go to the same positions of W0 and bits 32-63 to those of W1.
# Bits 64-95 (the third 32 bits, D2) go to the positions q = bit - 64 of W0
# or W1 that the first 64 stream bits leave empty: the zero bits 3-4 of the
# fields in W0 (mask ZERO_W0) or in W1 (mask ZERO_W1); a pin checks that these
# free positions are exactly the positions of D2's data bits.  Only data bits
# are stored; the zero bits are implied.


def _zero_bit_mask(word: int) -> int:
    """Positions, within 32-bit word `word` of the stream, of bits 3-4 of the
    fields that lie there."""
    m = 0
    for j in range(16):
        for b in (3, 4):
            p = 6 * j + b
            if 32 * word <= p < 32 * word + 32:
                m |= 1 << (p - 32 * word)
    return m


ZERO_W0 = _zero_bit_mask(0)
ZERO_W1 = _zero_bit_mask(1)


FIELD_DATA_BITS = (0, 1, 2, 5)    # magnitude bits 0-2 and the sign bit; bits 3-4 are zero


def _stream_bit_home(p: int):
    """(word, bit) where data bit p of the stream is stored."""
    if p < 64:
        return p // 32, p % 32
    q = p - 64
    if (ZERO_W0 >> q) & 1:
        return 0, q
    if (ZERO_W1 >> q) & 1:
        return 1, q
    raise AssertionError(f"stream bit {p} has no home")


def pack_codes(codes: np.ndarray, neg: np.ndarray = None) -> np.ndarray:
    """Packed code blocks, 4 bits per code (format above), built one field bit
    at a time.

    codes int [rows][K] (K a multiple of 16), every code in [-7, 7] (with the
    scale absmax / 7 of Eq. 2 the code -8 is never produced).  The sign bit of
    a field is `neg`: True where the rounded scaled value the code stands for
    is negative, negative zero included (quantize_groups_signed), so a zero
    code may carry sign bit 1.  Without `neg` the sign bit is set exactly for
    the negative codes.  Returns uint8 [rows][K/2].
    """
    c = np.asarray(codes, dtype=np.int64)
    rows, K = c.shape
    if K % 16:
        raise ValueError("the channel count must be a multiple of 16")
    if c.size and (c.min() < -7 or c.max() > 7):
        raise ValueError("packed codes must lie in [-7, 7]")
    if neg is None:
        neg = c < 0
    neg = np.asarray(neg, dtype=bool)
    if neg.shape != c.shape or (neg & (c > 0)).any() or (~neg & (c < 0)).any():
        raise ValueError("a sign bit contradicts its nonzero code")
    field = (np.abs(c) | (neg.astype(np.int64) << 5)).reshape(rows, K // 16, 16)
    words = np.zeros((rows, K // 16, 2), dtype=np.uint64)
    for j in range(16):                       # code j of every block
        for b in FIELD_DATA_BITS:             # data bit b of its field
            bit = ((field[:, :, j] >> b) & 1).astype(np.uint64)
            w, q = _stream_bit_home(6 * j + b)
            words[:, :, w] |= bit << np.uint64(q)
    return words.astype("<u4").view(np.uint8).reshape(rows, K // 2)


def code_fields(packed: np.ndarray) -> np.ndarray:
    """The 6-bit fields of packed blocks, read one stream bit at a time:
    uint8 [rows][K] (zero bits 3-4 of every field read back as 0)."""
    p = np.ascontiguousarray(np.asarray(packed, dtype=np.uint8))
    rows, nbytes = p.shape
    if nbytes % 8:
        raise ValueError("packed rows are whole 8-byte blocks")
    words = p.view("<u4").reshape(rows, nbytes // 8, 2).astype(np.uint64)
    field = np.zeros((rows, nbytes // 8, 16), dtype=np.uint64)
    for j in range(16):
        for b in FIELD_DATA_BITS:
            w, q = _stream_bit_home(6 * j + b)
            field[:, :, j] |= ((words[:, :, w] >> np.uint64(q)) & np.uint64(1)) << np.uint64(b)
    return field.reshape(rows, -1).astype(np.uint8)


def unpack_codes(packed: np.ndarray) -> np.ndarray:
    """Inverse of pack_codes: code = (-1)^sign * magnitude (a negative zero
    reads as 0).  int8 [rows][K]."""
    f = code_fields(packed).astype(np.int16)
    mag, neg = f & 7, (f >> 5) & 1
    return np.where(neg == 1, -mag, mag).astype(np.int8)


# ----------------------------------------------------------------------------
# The hot path, deployed mode
# ----------------------------------------------------------------------------


def inverse_smoothing(lam: np.ndarray) -> np.ndarray:
    """fl32(1 / lambda): the reciprocal formed once when the weights are packed."""
    lam = np.asarray(lam, dtype=np.float32)
    return (np.float32(1) / lam).astype(np.float32)


def pack_weights(R: np.ndarray, lam: np.ndarray, group: int = GROUP):
    """Offline weight pack (weights are quantized once, Sec. 3 / App. B.1).

    R: float32 [N][K] residual weight.  Returns (packed codes uint8 [N][K/2],
    scales float32 [N][G], inverse smoothing float32 [K], codes int8 [N][K]).
    """
    codes, scales, neg = quantize_groups_signed(np.asarray(R, dtype=np.float32), group)
    return pack_codes(codes, neg), scales, inverse_smoothing(lam), codes


def smooth_activations(x_bits: np.ndarray, inv_lam: np.ndarray) -> np.ndarray:
    """x~ = fl32(x * fl32(1/lambda)) per channel (Eq. 3 without rotation)."""
    x = bf16_bits_to_f64(x_bits).astype(np.float32)
    return (x * np.asarray(inv_lam, dtype=np.float32)[None, :]).astype(np.float32)


def fwht_f32(v: np.ndarray, B: int) -> np.ndarray:
    """Fast Walsh-Hadamard transform of every block of B consecutive channels
    of every row, in float32 (unnormalized: the result is v H_B blockwise).

    Stage s = 0, 1, .., log2(B)-1 pairs the elements whose indices differ in
    bit s only; the one with the bit clear becomes fl32(a + b), the other
    fl32(a - b) (a: bit clear, b: bit set).  One rounding per butterfly."""
    v = np.array(v, dtype=np.float32, copy=True)
    rows, K = v.shape
    if B & (B - 1) or K % B:
        raise ValueError("B must be a power of two dividing K")
    x = v.reshape(rows, K // B, B)
    h = 1
    while h < B:
        y = x.reshape(rows, K // B, B // (2 * h), 2, h)
        a, b = y[:, :, :, 0, :], y[:, :, :, 1, :]
        x = np.stack([(a + b).astype(np.float32), (a - b).astype(np.float32)], axis=3).reshape(rows, K // B, B)
        h *= 2
    return x.reshape(rows, K)


def hadamard_scale(B: int) -> np.float32:
    """fl32(1/sqrt(B)), the normalization of the rotation (exact for B = 4^k)."""
    return np.float32(1.0 / np.sqrt(np.float64(B)))


def rotate_activations(xt: np.ndarray, B: int) -> np.ndarray:
    """The online rotation of the smoothed activation (Eq. 3): the float32
    fast Walsh-Hadamard transform, then one float32 multiply by fl32(1/sqrt(B))."""
    return (fwht_f32(xt, B) * hadamard_scale(B)).astype(np.float32)


def down_projection(xt: np.ndarray, L1_bits: np.ndarray) -> np.ndarray:
    """t = bf16( sum_k bf16(x~_k) * L1[k, j] ), the sum taken exactly (float64).

    The paper's V^T x~ (Eq. 8 / Eq. 9) in the 16-bit branch.  Returns bf16 bits [M][r].
    Every product of two bf16 values is exact in float64; the float64 sum of at
    most 2**14 such terms is within ~1e-12 relative of the exact sum.
    """
    xb = round_to_bf16(xt)
    s = xb @ bf16_bits_to_f64(L1_bits)
    return f64_to_bf16_bits(s)


def transformed_activations(x_bits: np.ndarray, inv_lam: np.ndarray, hadamard: int = 0) -> np.ndarray:
    """x~ of Eq. 3: smoothed, and rotated when `hadamard` (the block size) is set."""
    xt = smooth_activations(x_bits, inv_lam)
    return rotate_activations(xt, hadamard) if hadamard else xt


def quantize_activations(x_bits: np.ndarray, inv_lam: np.ndarray, L1_bits: np.ndarray, hadamard: int = 0,
                         group: int = GROUP):
    """The activation side of one layer call: smoothing (and the rotation, if
    `hadamard` is the block size), per-token group quantization (Eq. 2,
    absmax/7 per token, App. B.1), code packing and the rank-r
    down-projection.  Returns (packed uint8 [M][K/2], scales f32 [M][G],
    t bf16 bits [M][r], codes int8 [M][K], x~ float32 [M][K])."""
    xt = transformed_activations(x_bits, inv_lam, hadamard)
    codes, scales, neg = quantize_groups_signed(xt, group)
    t = down_projection(xt, L1_bits)
    return pack_codes(codes, neg), scales, t, codes, xt


def deflate_activations(xt: np.ndarray, t_bits: np.ndarray, L1_bits: np.ndarray) -> np.ndarray:
    """x~_perp = x~ - V (V^T x~) (Eq. 8), deployed with the branch's factors.

    V^T x~ is the rounded t of the 16-bit branch and V is L1 = bf16(V), so the
    4-bit path loses exactly the part the branch adds back.  The r directions
    are removed one at a time, j = 0 .. r-1:
        cur <- fl32(cur - t[:, j] * L1[:, j]),   cur starting at x~,
    each product of two bf16 values being exact in float32 (16 significant
    bits).  xt float32 [M][K]; t bf16 bits [M][r]; L1 bf16 bits [K][r].
    Returns float32 [M][K].
    """
    cur = np.array(xt, dtype=np.float32, copy=True)
    t = bf16_bits_to_f64(t_bits)
    L1 = bf16_bits_to_f64(L1_bits)
    for j in range(t.shape[1]):
        prod64 = t[:, j:j + 1] * L1[None, :, j]            # exact in float64
        prod = prod64.astype(np.float32)
        if not np.array_equal(prod.astype(np.float64), prod64):
            raise ValueError("a branch product is not exact in float32 (underflow or overflow)")
        cur = (cur - prod).astype(np.float32)              # one float32 rounding per step
    return cur


def quantize_activations_deflated(x_bits: np.ndarray, inv_lam: np.ndarray, L1_bits: np.ndarray,
                                  hadamard: int = 0, group: int = GROUP):
    """The activation side with the paper's deflation (Eq. 8 / Eq. 9): t is
    computed from x~ as in quantize_activations, then x~_perp (deflate_activations)
    is quantized per token and group.  Returns (packed uint8 [M][K/2], scales
    f32 [M][G], t bf16 bits [M][r], codes int8 [M][K], x~_perp float32 [M][K])."""
    xt = transformed_activations(x_bits, inv_lam, hadamard)
    t = down_projection(xt, L1_bits)
    xp = deflate_activations(xt, t, L1_bits)
    codes, scales, neg = quantize_groups_signed(xp, group)
    return pack_codes(codes, neg), scales, t, codes, xp


def group_partials(qx: np.ndarray, qw: np.ndarray, group: int = GROUP) -> np.ndarray:
    """P[m, n, g] = sum_{k in group g} qx[m, k] * qw[n, k] (the integer GEMM of
    Sec. 3, one partial per group because each group has its own scales).

    qx int8 [M][K], qw int8 [N][K] -> int64 [M][N][G].  Each group's product is
    a float64 matmul of integer values |v| <= 8 over 64 terms: every partial sum
    is an integer of magnitude <= 4096, so the float64 result is exact.
    """
    M, K = qx.shape
    N = qw.shape[0]
    G = K // group
    P = np.empty((M, N, G), dtype=np.int64)
    for g in range(G):
        sl = slice(g * group, (g + 1) * group)
        P[:, :, g] = np.rint(qx[:, sl].astype(np.float64) @ qw[:, sl].astype(np.float64).T).astype(np.int64)
    return P


def asp_output(sx: np.ndarray, sw: np.ndarray, P: np.ndarray, t_bits: np.ndarray,
               L2_bits: np.ndarray, bias_bits=None) -> np.ndarray:
    """y = sum_g sx[m, g] sw[n, g] P[m, n, g] + t L2 (+ bias), float64, unrounded.

    The dequantized 4-bit product Q4(R)^T Q4(x~) (Eq. 2 per group) plus the
    16-bit branch (V^T W~)^T (V^T x~) of Eq. 9, plus the bias.
    sx [M][G], sw [N][G] float32; P [M][N][G]; t [M][r], L2 [r][N] bf16 bits.
    """
    sx64 = np.asarray(sx, dtype=np.float64)
    sw64 = np.asarray(sw, dtype=np.float64)
    y = np.einsum("mg,ng,mng->mn", sx64, sw64, P.astype(np.float64))
    y = y + bf16_bits_to_f64(t_bits) @ bf16_bits_to_f64(L2_bits)
    if bias_bits is not None:
        y = y + bf16_bits_to_f64(bias_bits)[None, :]
    return y


def asp_output_bruteforce(qx, sx, qw, sw, t_bits, L2_bits, bias_bits=None) -> np.ndarray:
    """Same output computed the other way: dequantize both operands, multiply
    (the group size follows from the scales' shape)."""
    group = qx.shape[1] // sx.shape[1]
    xd = dequantize_groups(qx, sx, group)
    wd = dequantize_groups(qw, sw, group)
    y = xd @ wd.T + bf16_bits_to_f64(t_bits) @ bf16_bits_to_f64(L2_bits)
    if bias_bits is not None:
        y = y + bf16_bits_to_f64(bias_bits)[None, :]
    return y


def asp_linear(x_bits, layer, bias_bits=None, rows=None, deflate=False):
    """Whole deployed layer for the tokens `rows` (all if None); with
    `deflate` the 4-bit path quantizes x~_perp (Eq. 9) instead of x~.

    layer: dict from build_layer (lam, L1, L2, R; optional hadamard, group).
    Returns a dict with every intermediate: wq, sw, inv_lam, qw, xq, sx, t, qx,
    P, y.
    """
    group = layer.get("group", GROUP)
    wq, sw, inv_lam, qw = pack_weights(layer["R"], layer["lam"], group)
    xb = x_bits if rows is None else x_bits[rows]
    quant = quantize_activations_deflated if deflate else quantize_activations
    xq, sx, t, qx, _ = quant(xb, inv_lam, layer["L1"], layer.get("hadamard", 0), group)
    P = group_partials(qx, qw, group)
    y = asp_output(sx, sw, P, t, layer["L2"], bias_bits)
    return {"wq": wq, "sw": sw, "inv_lam": inv_lam, "qw": qw, "xq": xq, "sx": sx,
            "t": t, "qx": qx, "P": P, "y": y}


def asp_output_rows(xq_rows, sx_rows, t_rows, wq, sw, L2_bits, bias_bits=None):
    """Reference output for a few tokens, straight from their packed codes and
    scales (no full [M][N][G] tensor): used to check sampled rows of large layers."""
    qx = unpack_codes(xq_rows)
    qw = unpack_codes(wq)
    P = group_partials(qx, qw, qx.shape[1] // sx_rows.shape[1])
    return asp_output(sx_rows, sw, P, t_rows, L2_bits, bias_bits), P


# ----------------------------------------------------------------------------
# Exact mode: same steps, float64 factors, nothing rounded outside the quantizer
# ----------------------------------------------------------------------------


def asp_linear_exact(x: np.ndarray, layer_exact, deflate=False, group: int = GROUP) -> np.ndarray:
    """y = Q4(x~) Q4(R)^T + (x~ V)(V^T W~), all float64 (Eq. 9 with the 4-bit
    path applied to x~, or with `deflate` to x~_perp = x~ - (x~ V) V^T; the
    quantizer itself run in float64)."""
    x = np.asarray(x, dtype=np.float64)
    xt = x / layer_exact["lam"][None, :]
    if layer_exact.get("hadamard", 0):
        xt = rotate_exact(xt, layer_exact["hadamard"])
    V = layer_exact["V"]
    x4 = xt - (xt @ V) @ V.T if deflate else xt
    qx, sx = quantize_groups(x4, group, dtype=np.float64)
    qw, sw = quantize_groups(layer_exact["R"], group, dtype=np.float64)
    y4 = dequantize_groups(qx, sx, group) @ dequantize_groups(qw, sw, group).T
    return y4 + (xt @ layer_exact["V"]) @ layer_exact["VtW"]


def bits_per_weight(K: int, N: int, r: int, group: int = GROUP, scale_bits: int = 32,
                    branch_bits: int = 16, smooth_bits: int = 32) -> float:
    """Effective bits per weight of one packed ASP layer: 4-bit codes, one scale
    per group, the two bf16 branch factors (r(K + N) values) and the per-channel
    smoothing reciprocal, divided by the K*N weights it replaces."""
    total = 4 * K * N + scale_bits * (K // group) * N + branch_bits * r * (K + N) + smooth_bits * K
    return total / (K * N)


# ----------------------------------------------------------------------------
# The Action Observability Gramian (AOG) estimate (Sec. 4.1, App. A probe
# estimator): accumulation of probe vector-Jacobian products, the rotated AOG
# of Sec. 4.2 and the action mass of Sec. 4.3
# ----------------------------------------------------------------------------


def aog_accumulate(A: np.ndarray, gT_bits: np.ndarray) -> np.ndarray:
    """A + sum_i g_i g_i^T over the n vectors g_i, float64.

    The procedure of the probe estimator adds g g^T to a d x d accumulator
    for every probe VJP g = J^T u.  gT_bits: bf16 bits [d][n] (column i is
    g_i); A: [d][d].  Products of two bf16 values are exact in float64."""
    g = bf16_bits_to_f64(gT_bits)
    return np.asarray(A, dtype=np.float64) + g @ g.T


def aog_estimate(A: np.ndarray, n_inputs: int, n_probes: int) -> np.ndarray:
    """G^ = A / (N P): the unbiased probe estimate of Eq. (AOG estimate)."""
    return np.asarray(A, dtype=np.float64) / float(n_inputs * n_probes)


def rotated_aog(G: np.ndarray, lam: np.ndarray, B: int = 0) -> np.ndarray:
    """The AOG in the quantizer's coordinates (Sec. 4.2): an error delta of
    x~ = H diag(lam)^-1 x moves x by diag(lam) H delta, so
    G~ = H diag(lam) G diag(lam) H (H the orthonormal block Hadamard matrix of
    block B, or the identity for B = 0).  float64."""
    lam = np.asarray(lam, dtype=np.float64)
    X = lam[:, None] * np.asarray(G, dtype=np.float64) * lam[None, :]
    if B:
        X = rotate_exact(X, B)            # X H (H symmetric)
        X = rotate_exact(X.T, B).T        # H (X H)
    return X


def action_mass(G_tilde_list) -> float:
    """mu_E = sum over the layers of an expert of tr G~ (Eq. action mass)."""
    return float(sum(np.trace(np.asarray(G, dtype=np.float64)) for G in G_tilde_list))
