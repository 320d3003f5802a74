"""Pins of the oracle's MXFP4 operator Q(.) against what the format fixes.

Q(.) is the paper's "MXFP4 quantize-dequantize operator" (under Eq. 2), in the
OCP Microscaling format the paper cites (Sec. 1).  Pins: hand-derived blocks
(tests/golden/mxfp4_hand_blocks.txt), element rounding against Python's
round-half-even, the scale rule against the float32 exponent field, and the
format's invariants.
"""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import mxfp4 as mx
from tests.golden import load_hand_blocks

BLOCKS = load_hand_blocks()


@pytest.mark.parametrize("blk", BLOCKS, ids=[b["name"] for b in BLOCKS])
def test_hand_blocks(blk):
    codes, scales = mx.mx_quantize(blk["values"][None, :])
    assert int(scales[0, 0]) == blk["scale"]
    np.testing.assert_array_equal(codes[0], blk["codes"])
    np.testing.assert_array_equal(mx.pack_codes(codes)[0], blk["packed"])


def test_hand_blocks_all_in_one_row():
    """The same blocks side by side in one row give the same per-block result."""
    row = np.concatenate([b["values"] for b in BLOCKS])[None, :]
    codes, scales = mx.mx_quantize(row)
    np.testing.assert_array_equal(scales[0], [b["scale"] for b in BLOCKS])
    np.testing.assert_array_equal(codes[0], np.concatenate([b["codes"] for b in BLOCKS]))


def test_e8m0_decode():
    assert mx.e8m0_to_float(0x7F) == 1.0
    assert mx.e8m0_to_float(0x80) == 2.0
    assert mx.e8m0_to_float(0x00) == 2.0 ** -127
    assert mx.e8m0_to_float(0xFE) == 2.0 ** 127
    with pytest.raises(ValueError):
        mx.e8m0_to_float(0xFF)


def _e2m1_from_bits(code):
    """E2M1 from its bit fields (sign, 2-bit exponent with bias 1, 1-bit mantissa)."""
    s, e, m = (code >> 3) & 1, (code >> 1) & 3, code & 1
    mag = 0.5 * m if e == 0 else 2.0 ** (e - 1) * (1 + 0.5 * m)
    return -mag if s else mag


def test_e2m1_table_matches_bit_fields():
    for c in range(16):
        assert mx.e2m1_decode(np.uint8(c)) == _e2m1_from_bits(c)


def _rne_e2m1(t):
    """Nearest E2M1 magnitude by Python's round-half-even on the grid spacing of
    each binade: 0.5 below 2, 1 in [2, 4), 2 above 4 (saturating at 6)."""
    a = abs(t)
    if a < 2:
        q = round(2 * a) / 2
    elif a < 4:
        q = float(round(a))
    else:
        q = min(2.0 * round(a / 2), 6.0)
    return q


def _rne_cases(rng, n):
    ties = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 7.0])
    grid = mx.E2M1_MAGNITUDES
    near = np.concatenate([ties, grid, np.nextafter(ties, 0), np.nextafter(ties, 8)])
    vals = np.concatenate([near, rng.uniform(0, 7.99, n)]).astype(np.float32)
    sign = rng.choice([-1.0, 1.0], vals.shape[0]).astype(np.float32)
    return vals * sign


def test_element_rounding_matches_round_half_even():
    rng = np.random.default_rng(1)
    vals = _rne_cases(rng, 4000)
    # one element 7.99 fixes amax in [4, 8): scale code 127 and t = v exactly
    n = (vals.size + 30) // 31
    pad = np.zeros(n * 31, np.float32)
    pad[:vals.size] = vals
    blocks = np.concatenate([np.full((n, 1), 7.99, np.float32), pad.reshape(n, 31)], axis=1)
    codes, scales = mx.mx_quantize(blocks)
    assert np.all(scales == 127)
    got = mx.e2m1_decode(codes[:, 1:]).ravel()
    want = np.array([_rne_e2m1(float(v)) for v in pad])
    np.testing.assert_array_equal(np.abs(got), want)
    # sign bit follows the input's sign bit
    np.testing.assert_array_equal((codes[:, 1:].ravel() >> 3) & 1, np.signbit(pad).astype(np.uint8))


def _scale_from_exponent_field(amax_f32):
    bits = np.asarray(amax_f32, np.float32).view(np.uint32)
    bexp = (bits >> 23) & 0xFF
    return np.clip(bexp.astype(np.int64) - 2, 0, 254)


@settings(max_examples=300, deadline=None)
@given(st.lists(st.floats(allow_nan=False, allow_infinity=False, width=32),
                min_size=32, max_size=32))
def test_scale_rule_and_top_binade(vals):
    v = np.array(vals, np.float32)[None, :]
    codes, scales = mx.mx_quantize(v)
    amax = np.abs(v).max()
    want = 0 if amax == 0 else int(_scale_from_exponent_field(amax))
    assert int(scales[0, 0]) == want
    t_max = float(amax) * 2.0 ** (127 - want)
    if want > 0:
        assert 4.0 <= t_max < 8.0          # the largest element lands in E2M1's top binade
    # every element's dequantized value is a nearest grid point of t (within 6 * 2^X)
    deq = mx.mx_dequantize(codes, scales)[0]
    X = 2.0 ** (want - 127)
    for x, d in zip(v[0].astype(np.float64), deq):
        t = x / X
        assert abs(d / X) == _rne_e2m1(t)


def test_pack_roundtrip_and_order():
    rng = np.random.default_rng(2)
    codes = rng.integers(0, 16, (3, 64), dtype=np.uint8)
    packed = mx.pack_codes(codes)
    assert packed.shape == (3, 32)
    np.testing.assert_array_equal(packed[:, 0], codes[:, 0] + 16 * codes[:, 1])
    np.testing.assert_array_equal(mx.unpack_codes(packed), codes)


def test_idempotent_on_grid_and_odd_symmetry():
    rng = np.random.default_rng(3)
    v = (rng.standard_normal((16, 256)) * rng.uniform(0.01, 100, (16, 1))).astype(np.float32)
    q = mx.qdq(v)
    np.testing.assert_array_equal(mx.qdq(q.astype(np.float32)), q)   # Q(Q(v)) = Q(v)
    np.testing.assert_array_equal(mx.qdq(-v), -q)                      # Q(-v) = -Q(v)
    # error bound: half the widest grid spacing (2 * 2^X) when |t| <= 6, below
    # 2 * 2^X in the saturating range 6 < |t| < 8
    X = 2.0 ** (mx.mx_quantize(v)[1].astype(np.float64) - 127)[..., None]
    err = np.abs(q - v).reshape(16, 8, 32)
    t = np.abs(v.astype(np.float64)).reshape(16, 8, 32) / X
    assert np.all(err[t <= 6] <= np.broadcast_to(X, t.shape)[t <= 6])
    assert np.all(err < 2 * X)


def test_rejects_bad_input():
    with pytest.raises(ValueError):
        mx.mx_quantize(np.zeros((1, 33), np.float32))
    with pytest.raises(TypeError):
        mx.mx_quantize(np.zeros((1, 32), np.float64))
    with pytest.raises(ValueError):
        mx.mx_quantize(np.full((1, 32), np.inf, np.float32))


# ------------------------------------------- E8M0 block-scale search ---
_E2M1_GRID = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]


def _scalar_block_error(block, code):
    """Exact squared error of a block under one E8M0 code, by a scalar loop
    independent of the oracle: each element is rounded to the nearest E2M1
    magnitude of |v| / 2**(code - 127) (ties to the even grid index,
    saturating at 6) and compared with the exact rational value."""
    from fractions import Fraction
    scale = Fraction(2) ** (int(code) - 127)
    err = Fraction(0)
    for v in block:
        fv = Fraction(float(v))
        t = abs(fv) / scale
        dists = [abs(t - Fraction(g)) for g in _E2M1_GRID]
        dmin = min(dists)
        cands = [i for i, d in enumerate(dists) if d == dmin]
        idx = next((i for i in cands if i % 2 == 0), cands[0])
        q = Fraction(_E2M1_GRID[idx]) * scale * (-1 if fv < 0 else 1)
        err += (fv - q) ** 2
    return err


def test_searched_scale_hand_blocks():
    """7.5 alone: the OCP code (127) saturates it to 6 (error 1.5^2); code 128
    rounds 3.75 to 4 -> 8 (error 0.5^2).  4.0 with 31 x 0.3: code 126 gives 4 ->
    3 (error 1) but 0.3 -> 0.25 (31 x 0.05^2), better than 127's 31 x 0.2^2."""
    b1 = np.zeros(32, np.float32)
    b1[0] = 7.5
    b2 = np.full(32, 0.3, np.float32)
    b2[0] = 4.0
    v = np.stack([b1, b2])
    _, s0 = mx.mx_quantize(v)
    codes, sc = mx.mx_quantize_searched(v)
    assert list(s0.ravel()) == [127, 127]
    assert list(sc.ravel()) == [128, 126]
    deq = mx.mx_dequantize(codes, sc)
    assert deq[0, 0] == 8.0 and deq[1, 0] == 3.0 and deq[1, 1] == 0.25


@pytest.mark.parametrize("seed", range(6))
def test_searched_scale_is_the_exact_minimizer(seed):
    """Against exact rational errors of every candidate code: the chosen code
    is a minimizer among c0, c0 - 1, c0 + 1 (first in that order on exact ties)
    and never worse than the OCP code; codes are Q(.)'s element rule under
    the chosen scale."""
    rng = np.random.default_rng(seed)
    kinds = [rng.standard_normal(32), rng.standard_t(2, 32) * 3, rng.uniform(-7.9, 7.9, 32),
             np.concatenate([[rng.uniform(4, 8)], rng.uniform(-0.4, 0.4, 31)])]
    blocks = np.stack([(k * 2.0 ** rng.integers(-20, 20)).astype(np.float32) for k in kinds
                       for _ in range(3)])
    codes, sc = mx.mx_quantize_searched(blocks)
    _, s0 = mx.mx_quantize(blocks)
    for b in range(blocks.shape[0]):
        c0 = int(s0[b, 0])
        cands = [min(max(c0 + off, 0), 254) for off in (0, -1, 1)]
        errs = [_scalar_block_error(blocks[b], c) for c in cands]
        chosen = int(sc[b, 0])
        assert chosen in cands
        e_chosen = _scalar_block_error(blocks[b], chosen)
        assert e_chosen == min(errs), (b, cands, [float(e) for e in errs], chosen)
        assert e_chosen <= errs[0]
        np.testing.assert_array_equal(codes[b], mx.mx_quantize_with_scales(blocks[b:b + 1], sc[b:b + 1])[0])


def test_searched_scale_edge_blocks():
    zeros = np.zeros((1, 32), np.float32)
    codes, sc = mx.mx_quantize_searched(zeros)
    assert sc[0, 0] == 0 and not codes.any()
    big = np.full((1, 32), 3.0e38, np.float32)           # c0 = 252: c0 + 1 = 253 is still normal
    codes, sc = mx.mx_quantize_searched(big)
    assert int(sc[0, 0]) in (251, 252, 253)
    assert np.isfinite(mx.mx_dequantize(codes, sc)).all()
