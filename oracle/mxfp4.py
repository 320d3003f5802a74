"""MXFP4 quantize-dequantize operator Q(.) -- oracle (test infrastructure only).

The paper writes Q(.) for "the MXFP4 quantize-dequantize operator" (Sec. Method,
under Eq. 2) and takes the format from the OCP Microscaling specification it
cites in the introduction: blocks of 32 consecutive elements along the
reduction dimension share one E8M0 power-of-two scale, and each element is an
FP4 E2M1 number (1 sign, 2 exponent, 1 mantissa bit; magnitudes
0, 0.5, 1, 1.5, 2, 3, 4, 6).  The paper does not restate the conversion rule;
the reading used here (shared by every side of the build) is the OCP one:

* shared exponent  X = floor(log2(amax)) - emax_E2M1, with emax_E2M1 = 2 and
  amax the largest magnitude in the block;  E8M0 code = X + 127 clamped to
  [0, 254] (0xFF is the NaN code and is never produced); an all-zero block
  gets code 0.  Equivalently code = clamp(biased_exp_fp32(amax) - 2, 0, 254).
* every element is divided by 2**X (exact: a power of two) and rounded to the
  nearest E2M1 magnitude, ties to the even code (mantissa bit 0), saturating
  at 6; the sign bit is the sign bit of the input (so -0.0 and small negative
  values encode as 0x8, "negative zero").
* packing (a layout choice the paper leaves open): code nibble = s<<3 | e<<1 | m,
  i.e. the index of the magnitude in the list above plus 8 for negative; byte i
  of a packed row holds element 2i in bits 0-3 and element 2i+1 in bits 4-7;
  scales are one byte per block, row-major.

Inputs are float32 arrays (the precision in which every side takes the
rounding decisions); all arithmetic here is exact in float64.
"""
from __future__ import annotations

import numpy as np

BLOCK = 32                     # elements per shared scale (OCP MX block size)
EMAX_E2M1 = 2                  # exponent of the largest E2M1 normal (6 = 1.5 * 2**2)
E8M0_BIAS = 127
# E2M1 magnitudes in code order: code & 7 indexes this table, code & 8 is the sign.
E2M1_MAGNITUDES = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0], dtype=np.float64)

_ROW_CHUNK_ELEMS = 1 << 21     # bound the [.., 8] distance table to ~128 MB


def e8m0_to_float(code):
    """Value of an E8M0 scale code: 2**(code - 127).  0xFF (NaN) is rejected."""
    code = np.asarray(code, dtype=np.int64)
    if np.any(code == 255):
        raise ValueError("E8M0 code 0xFF is NaN and is never produced by Q(.)")
    return np.ldexp(1.0, code - E8M0_BIAS)


def e2m1_decode(codes):
    """float64 value of E2M1 nibbles (0..15)."""
    codes = np.asarray(codes, dtype=np.uint8)
    mag = E2M1_MAGNITUDES[codes & 7]
    return np.where(codes & 8, -mag, mag)


def shared_scale_code(amax):
    """E8M0 code of blocks with the given float64 max-magnitudes (>= 0).

    floor(log2(amax)) is taken exactly from frexp: amax = f * 2**e with
    f in [0.5, 1), so floor(log2(amax)) = e - 1.
    """
    amax = np.asarray(amax, dtype=np.float64)
    _, e = np.frexp(amax)
    x = (e.astype(np.int64) - 1) - EMAX_E2M1          # shared exponent X
    code = np.clip(x + E8M0_BIAS, 0, 254)
    return np.where(amax > 0, code, 0).astype(np.uint8)


def _round_to_e2m1_index(t):
    """Index (0..7) of the E2M1 magnitude nearest to |t|, ties to even index.

    Written as the definition: measure the distance to every magnitude, keep
    the nearest ones, and among two equally near ones take the even code
    (mantissa bit 0).  |t| above 6 is nearest to 6, which is the saturation.
    All distances are exact in float64 (|t| < 8 carries at most 24 bits).
    """
    d = np.abs(np.abs(t)[..., None] - E2M1_MAGNITUDES)
    nearest = d == d.min(axis=-1, keepdims=True)
    even = nearest & (np.arange(8) % 2 == 0)
    first_even = np.argmax(even, axis=-1)
    first_any = np.argmax(nearest, axis=-1)
    return np.where(even.any(axis=-1), first_even, first_any).astype(np.uint8)


def mx_quantize(v):
    """Q(.) on the last axis of a float32 array whose length is a multiple of 32.

    Returns (codes, scales): codes uint8 nibbles with the shape of ``v`` (one
    per element, unpacked), scales uint8 E8M0 codes of shape [..., K/32].
    """
    v = np.asarray(v)
    if v.dtype != np.float32:
        raise TypeError("Q(.) takes float32 input (the precision of its decisions)")
    if v.shape[-1] % BLOCK:
        raise ValueError("the quantized axis must be a multiple of 32")
    if not np.all(np.isfinite(v)):
        raise ValueError("Q(.) is defined here for finite inputs only")
    lead = v.shape[:-1]
    K = v.shape[-1]
    flat = v.reshape(int(np.prod(lead, dtype=np.int64)), K)
    codes = np.empty(flat.shape, dtype=np.uint8)
    scales = np.empty((flat.shape[0], K // BLOCK), dtype=np.uint8)
    rows_per_chunk = max(1, _ROW_CHUNK_ELEMS // max(K, 1))
    for r0 in range(0, flat.shape[0], rows_per_chunk):
        blk = flat[r0:r0 + rows_per_chunk].astype(np.float64)
        blk = blk.reshape(blk.shape[0], K // BLOCK, BLOCK)
        amax = np.abs(blk).max(axis=-1)
        sc = shared_scale_code(amax)
        t = np.ldexp(blk, E8M0_BIAS - sc.astype(np.int64)[..., None])   # v / 2**X, exact
        idx = _round_to_e2m1_index(t)
        sign = np.signbit(blk).astype(np.uint8) << 3
        codes[r0:r0 + rows_per_chunk] = (idx | sign).reshape(blk.shape[0], K)
        scales[r0:r0 + rows_per_chunk] = sc
    return codes.reshape(*lead, K), scales.reshape(*lead, K // BLOCK)


def mx_quantize_with_scales(v, scales):
    """Elements of float32 ``v`` rounded to E2M1 under given E8M0 block codes
    (the element rule of Q(.) with the shared exponent replaced): codes uint8."""
    v = np.asarray(v)
    if v.dtype != np.float32:
        raise TypeError("Q(.) takes float32 input (the precision of its decisions)")
    K = v.shape[-1]
    blk = v.astype(np.float64).reshape(*v.shape[:-1], K // BLOCK, BLOCK)
    sc = np.asarray(scales, dtype=np.int64)
    t = np.ldexp(blk, E8M0_BIAS - sc[..., None])     # v / 2**(code - 127), exact
    idx = _round_to_e2m1_index(t)
    sign = np.signbit(blk).astype(np.uint8) << 3
    return (idx | sign).reshape(v.shape)


SEARCH_OFFSETS = (0, -1, 1)   # candidate codes around the OCP code, in preference order


def block_squared_errors(v, codes, scales):
    """sum_i (v_i - deq_i)^2 per 32-block, float64, summed in element order."""
    K = v.shape[-1]
    d = (v.astype(np.float64) - mx_dequantize(codes, scales)).reshape(*v.shape[:-1], K // BLOCK, BLOCK)
    err = np.zeros(d.shape[:-1])
    for i in range(BLOCK):               # one element at a time: a fixed summation order
        err = err + d[..., i] * d[..., i]
    return err


def mx_quantize_searched(v):
    """Q(.) with a local E8M0 search per block (the weight-side block-scale
    search of Sec. Ablation Studies, whose rule the paper does not give; the
    reading here): among the codes c0, c0 - 1, c0 + 1 (c0 the OCP code,
    clamped to [0, 254]) keep the first with the smallest squared block error
    sum_i (v_i - deq_i)^2, so no block is worse than under Q(.)."""
    v = np.asarray(v)
    codes0, sc0 = mx_quantize(v)
    best_codes, best_sc = codes0, sc0.copy()
    best_err = block_squared_errors(v, codes0, sc0)
    for off in SEARCH_OFFSETS[1:]:
        sc = np.clip(sc0.astype(np.int64) + off, 0, 254).astype(np.uint8)
        codes = mx_quantize_with_scales(v, sc)
        err = block_squared_errors(v, codes, sc)
        better = err < best_err
        best_err = np.where(better, err, best_err)
        best_sc = np.where(better, sc, best_sc)
        better_el = np.repeat(better, BLOCK, axis=-1).reshape(v.shape)
        best_codes = np.where(better_el, codes, best_codes)
    return best_codes.astype(np.uint8), best_sc.astype(np.uint8)


def mx_dequantize(codes, scales):
    """deq(code, scale) = e2m1(code) * 2**(scale - 127), float64."""
    codes = np.asarray(codes, dtype=np.uint8)
    scales = np.asarray(scales, dtype=np.uint8)
    K = codes.shape[-1]
    if scales.shape[-1] * BLOCK != K:
        raise ValueError("one scale per 32 codes expected")
    vals = e2m1_decode(codes).reshape(*codes.shape[:-1], K // BLOCK, BLOCK)
    vals = vals * e8m0_to_float(scales)[..., None]
    return vals.reshape(codes.shape)


def qdq(v):
    """Q(v) as a float64 array: quantize then dequantize."""
    c, s = mx_quantize(v)
    return mx_dequantize(c, s)


def pack_codes(codes):
    """Pack nibbles two per byte: element 2i -> bits 0-3, element 2i+1 -> bits 4-7."""
    codes = np.asarray(codes, dtype=np.uint8)
    if codes.shape[-1] % 2:
        raise ValueError("even number of codes expected")
    if np.any(codes > 15):
        raise ValueError("codes are 4-bit")
    return (codes[..., 0::2] | (codes[..., 1::2] << 4)).astype(np.uint8)


def unpack_codes(packed):
    """Inverse of pack_codes."""
    packed = np.asarray(packed, dtype=np.uint8)
    out = np.empty(packed.shape[:-1] + (packed.shape[-1] * 2,), dtype=np.uint8)
    out[..., 0::2] = packed & 0x0F
    out[..., 1::2] = packed >> 4
    return out
