"""Pins of the PRQuant oracle (Algorithm 1, Eq. 1-3) against closed forms,
invariants, special cases and brute force -- never against itself."""
import math

import numpy as np
import pytest

from oracle import mxfp4 as mx
from oracle import prquant as pq
from paper_2609_22106_amd import inputs


def _bf16(x):
    return inputs.f32_to_bf16_bits(np.asarray(x, np.float32))


def _small(N=64, K=256, M=8, T=32, n_out=4, seed=0, scale=30.0):
    return inputs.make_dense("small", N=N, K=K, M=M, T=T, k_tail=64, n_out=n_out,
                             out_scale=scale, seed=seed)


# ---------------------------------------------------------------- scaling ---
def test_scale_closed_forms():
    """s_j = a_j^alpha / b_j^(1-alpha) (SmoothQuant form) and a_j^alpha (paper's
    printed form) at alphas where the power has a closed form."""
    c = _small()
    a = np.maximum(np.abs(inputs.bf16_bits_to_f32(c.Xcal)).max(0).astype(np.float64), 1e-5)
    b = np.maximum(np.abs(inputs.bf16_bits_to_f32(c.W)).max(0).astype(np.float64), 1e-5)
    s, inv = pq.channel_scales(c.W, c.Xcal, 1.0, "smooth")
    np.testing.assert_array_equal(s, a.astype(np.float32))          # alpha = 1: s = a
    s, _ = pq.channel_scales(c.W, c.Xcal, 0.0, "smooth")
    np.testing.assert_array_equal(s, (1.0 / b).astype(np.float32))  # alpha = 0: s = 1/b
    s, _ = pq.channel_scales(c.W, c.Xcal, 0.5, "smooth")
    ref = np.array([math.sqrt(x) / math.sqrt(y) for x, y in zip(a, b)], np.float32)
    assert np.max(np.abs(s.view(np.int32) - ref.view(np.int32))) <= 1   # within 1 ulp
    s, _ = pq.channel_scales(c.W, c.Xcal, 0.5, "act_only")
    ref = np.array([math.sqrt(x) for x in a], np.float32)
    assert np.max(np.abs(s.view(np.int32) - ref.view(np.int32))) <= 1
    s, inv = pq.channel_scales(c.W, c.Xcal, 0.5, "none")
    assert np.all(s == 1) and np.all(inv == 1)


def test_inverse_scale_is_float32_reciprocal():
    c = _small()
    s, inv = pq.channel_scales(c.W, c.Xcal, 0.5)
    assert inv.dtype == np.float32
    prod = s.astype(np.float64) * inv.astype(np.float64)
    assert np.max(np.abs(prod - 1.0)) <= 2.0 ** -23          # |1/s - inv| <= ulp/2
    # correctly rounded: neither neighbour of inv is closer to 1/s
    exact = 1.0 / s.astype(np.float64)
    for nb in (np.nextafter(inv, np.float32(0)), np.nextafter(inv, np.float32(np.inf))):
        assert np.all(np.abs(inv - exact) <= np.abs(nb.astype(np.float64) - exact))


def test_zero_calibration_channel_is_clamped():
    c = _small()
    Xcal = c.Xcal.copy()
    Xcal[:, 5] = 0
    s, _ = pq.channel_scales(c.W, Xcal, 1.0, "smooth")
    assert s[5] == np.float32(1e-5)


# --------------------------------------------------- selection, permutation ---
def _brute_column_errors(W_s):
    """Column errors by scalar Python loops with an independent E2M1 rounding
    (Python round-half-even) and scale rule (float32 exponent field)."""
    N, K = W_s.shape
    err = [0.0] * K
    for n in range(N):
        for b0 in range(0, K, 32):
            blk = [float(x) for x in W_s[n, b0:b0 + 32]]
            amax = max(abs(x) for x in blk)
            if amax == 0:
                code = 0
            else:
                bexp = (int(np.float32(amax).view(np.uint32)) >> 23) & 0xFF
                code = min(max(bexp - 2, 0), 254)
            X = 2.0 ** (code - 127)
            for j, x in enumerate(blk):
                t = x / X
                a = abs(t)
                if a < 2:
                    q = round(2 * a) / 2
                elif a < 4:
                    q = float(round(a))
                else:
                    q = min(2.0 * round(a / 2), 6.0)
                q = math.copysign(q, t) * X
                err[b0 + j] += (x - q) ** 2
    return err


@pytest.mark.parametrize("N,K", [(4, 64), (8, 96), (8, 128)])
@pytest.mark.parametrize("tied", [False, True])
def test_topk_brute_force(N, K, tied):
    rng = np.random.default_rng(N * 1000 + K + tied)
    W = (0.02 * rng.standard_normal((N, K))).astype(np.float32)
    W[:, rng.choice(K, 3, replace=False)] *= 20
    if tied:                                    # identical columns -> identical errors
        W[:, 10] = W[:, 40]
        W[:, 41] = W[:, 40]
        W[:, 3] = W[:, 60]
    Wb = _bf16(W)
    Xcal = _bf16(rng.standard_normal((16, K)))
    art = pq.prepare(Wb, Xcal, 0.5, 32)
    W_s = (inputs.bf16_bits_to_f32(Wb) * art["scale"][None, :]).astype(np.float32)
    err = _brute_column_errors(W_s)
    np.testing.assert_allclose(art["col_err"], err, rtol=1e-12, atol=0)
    want = sorted(sorted(range(K), key=lambda j: (-err[j], j))[:32])
    np.testing.assert_array_equal(art["selected"], want)
    sel = set(want)
    assert min(err[j] for j in sel) >= max(err[j] for j in range(K) if j not in sel)


def test_permutation_invariants():
    c = _small()
    art = pq.prepare(c.W, c.Xcal, 0.5, 64)
    perm, K, k = art["perm"], 256, 64
    assert sorted(perm.tolist()) == list(range(K))            # bijection
    assert np.all(np.diff(perm[:K - k]) > 0)                   # head increasing
    assert np.all(np.diff(perm[K - k:]) > 0)                   # tail increasing
    np.testing.assert_array_equal(perm[K - k:], art["selected"])
    np.testing.assert_array_equal(art["W_tilde"], art["W_s"][:, perm])


# ------------------------------------------------------------- Eq. 1 and 2 ---
def test_eq1_identity_without_quantization():
    """(X D^-1 P)(W D P)^T = X W^T (Eq. 1), fp64, no quantization."""
    c = _small()
    art = pq.prepare(c.W, c.Xcal, 0.5, 64)
    Y = pq.unquantized_transform_product(c.X, c.W, art["scale"], art["perm"])
    ref = pq.reference_product(c.X, c.W)
    assert np.max(np.abs(Y - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_residual_reconstructs_tail_exactly():
    """Q(W~_tail) + R = W~_tail exactly (Eq. 2), and Q(W~_tail) equals the tail
    of Q(W~) because the tail starts on a block boundary."""
    c = _small()
    art = pq.prepare(c.W, c.Xcal, 0.5, 64)
    Wt = art["W_tilde"].astype(np.float64)
    q_tail_alone = mx.qdq(art["W_tilde"][:, -64:])
    q_full = mx.qdq(art["W_tilde"])[:, -64:]
    np.testing.assert_array_equal(q_tail_alone, q_full)
    np.testing.assert_array_equal(q_tail_alone + art["R"].astype(np.float64), Wt[:, -64:])


def test_compensation_never_increases_elementwise_weight_error():
    """|W~_tail - Q(W~_tail) - Q(R)| <= |R| element by element."""
    c = _small(N=128, K=512)
    art = pq.prepare(c.W, c.Xcal, 0.5, 64)
    R = art["R"].astype(np.float64)
    resid = R - mx.qdq(art["R"])
    assert np.all(np.abs(resid) <= np.abs(R))


def test_augmented_weight_layout():
    c = _small()
    art = pq.prepare(c.W, c.Xcal, 0.5, 64)
    codes = mx.unpack_codes(art["Wq"])
    assert art["Wq"].shape == (64, (256 + 64) // 2) and art["Wsc"].shape == (64, 10)
    c_t, s_t = mx.mx_quantize(art["W_tilde"])
    c_r, s_r = mx.mx_quantize(art["R"])
    np.testing.assert_array_equal(codes[:, :256], c_t)
    np.testing.assert_array_equal(codes[:, 256:], c_r)
    np.testing.assert_array_equal(art["Wsc"], np.concatenate([s_t, s_r], 1))


# ------------------------------------------------------------------ Eq. 3 ---
def test_tail_copy_equals_quantizing_the_concatenation():
    """Quantize Z~ once and append its quantized tail blocks with their scales
    == Q([Z~, Z~_tail]) (Sec. Kernel design), codes and scales bit for bit."""
    c = _small()
    art = pq.prepare(c.W, c.Xcal, 0.5, 64)
    Aq, Asc = pq.quant_act(c.X, art["inv_scale"], art["perm"], 64)
    Z = pq.transformed_activation(c.X, art["inv_scale"], art["perm"])
    cz, sz = mx.mx_quantize(Z)
    copied_codes = np.concatenate([cz, cz[:, -64:]], 1)
    copied_scales = np.concatenate([sz, sz[:, -2:]], 1)
    np.testing.assert_array_equal(Aq, mx.pack_codes(copied_codes))
    np.testing.assert_array_equal(Asc, copied_scales)


def test_transformed_activation_definition():
    c = _small()
    art = pq.prepare(c.W, c.Xcal, 0.5, 64)
    Z = pq.transformed_activation(c.X, art["inv_scale"], art["perm"])
    X = inputs.bf16_bits_to_f32(c.X)
    for p in (0, 17, 191, 192, 255):
        j = art["perm"][p]
        np.testing.assert_array_equal(Z[:, p], (X[:, j] * art["inv_scale"][j]).astype(np.float32))


def test_k0_no_scaling_is_plain_mxfp4():
    """k = 0 and s = 1 reduce every step to plain MXFP4 (the paper's MXFP4 baseline)."""
    c = _small()
    art = pq.prepare(c.W, c.Xcal, 0.5, 0, "none")
    np.testing.assert_array_equal(art["perm"], np.arange(256))
    cw, sw = mx.mx_quantize(inputs.bf16_bits_to_f32(c.W))
    np.testing.assert_array_equal(art["Wq"], mx.pack_codes(cw))
    np.testing.assert_array_equal(art["Wsc"], sw)
    Aq, Asc = pq.quant_act(c.X, art["inv_scale"], art["perm"], 0)
    cx, sx = mx.mx_quantize(inputs.bf16_bits_to_f32(c.X))
    np.testing.assert_array_equal(Aq, mx.pack_codes(cx))
    np.testing.assert_array_equal(Asc, sx)
    Y = pq.gemm(Aq, Asc, art["Wq"], art["Wsc"])
    plain = mx.mx_dequantize(cx, sx) @ mx.mx_dequantize(cw, sw).T
    np.testing.assert_array_equal(Y, plain)


def test_k0_with_scaling_is_mxfp4_of_scaled_operands():
    c = _small()
    art = pq.prepare(c.W, c.Xcal, 0.5, 0, "smooth")
    np.testing.assert_array_equal(art["perm"], np.arange(256))
    Aq, Asc = pq.quant_act(c.X, art["inv_scale"], art["perm"], 0)
    Xs = (inputs.bf16_bits_to_f32(c.X) * art["inv_scale"][None, :]).astype(np.float32)
    Ws = (inputs.bf16_bits_to_f32(c.W) * art["scale"][None, :]).astype(np.float32)
    Y = pq.gemm(Aq, Asc, art["Wq"], art["Wsc"])
    np.testing.assert_array_equal(Y, mx.qdq(Xs) @ mx.qdq(Ws).T)


def _decode_brute(packed, scales):
    """Independent decode: bit fields of each nibble, scale 2^(code-127)."""
    R, Kh = packed.shape
    out = np.zeros((R, 2 * Kh))
    for r in range(R):
        for i in range(2 * Kh):
            byte = int(packed[r, i // 2])
            nib = (byte >> (4 * (i % 2))) & 0xF
            s, e, m = nib >> 3, (nib >> 1) & 3, nib & 1
            mag = 0.5 * m if e == 0 else 2.0 ** (e - 1) * (1 + 0.5 * m)
            out[r, i] = (-mag if s else mag) * 2.0 ** (int(scales[r, i // 32]) - 127)
    return out


def test_gemm_brute_force():
    rng = np.random.default_rng(7)
    M, N, K = 3, 5, 96
    Aq = rng.integers(0, 256, (M, K // 2), dtype=np.uint8)
    Wq = rng.integers(0, 256, (N, K // 2), dtype=np.uint8)
    Asc = rng.integers(110, 140, (M, K // 32), dtype=np.uint8)
    Wsc = rng.integers(110, 140, (N, K // 32), dtype=np.uint8)
    A, W = _decode_brute(Aq, Asc), _decode_brute(Wq, Wsc)
    Y = pq.gemm(Aq, Asc, Wq, Wsc)
    for m in range(M):
        for n in range(N):
            terms = [A[m, i] * W[n, i] for i in range(K)]       # each product exact
            bound = K * 2.0 ** -53 * math.fsum(abs(t) for t in terms)  # fp64 summation bound
            assert abs(Y[m, n] - math.fsum(terms)) <= bound


def test_gemm_hand_values():
    """All-ones block times all-halves block: 32 * 0.5 = 16 (Eq. 3 on one block);
    scales 2^1 and 2^-1 cancel; a second block at scales 2^3, 2^-1 adds 64."""
    ones, halves = np.full((1, 16), 0x22, np.uint8), np.full((1, 16), 0x11, np.uint8)
    assert pq.gemm(ones, np.array([[127]], np.uint8), halves, np.array([[127]], np.uint8))[0, 0] == 16
    assert pq.gemm(ones, np.array([[128]], np.uint8), halves, np.array([[126]], np.uint8))[0, 0] == 16
    A = np.concatenate([ones, ones], 1)
    W = np.concatenate([halves, halves], 1)
    assert pq.gemm(A, np.array([[127, 130]], np.uint8), W, np.array([[127, 126]], np.uint8))[0, 0] == 80


# ------------------------------------------------- reconstruction error ---
def test_residual_compensation_lowers_error_tiny_case():
    """Residual compensation lowers y-NRMSE versus the same scaling without it
    and versus plain MXFP4 (the paper's ablation direction, Sec. Ablation)."""
    c = inputs.tiny_case()
    ref = pq.reference_product(c.X, c.W)
    y_prq, _ = pq.prquant_forward(c.X, c.W, c.Xcal, 0.5, 64)
    y_nores, _ = pq.prquant_forward(c.X, c.W, c.Xcal, 0.5, 0)
    y_plain, _ = pq.prquant_forward(c.X, c.W, c.Xcal, 0.5, 0, "none")
    e_prq, e_nores, e_plain = (pq.nrmse(y, ref) for y in (y_prq, y_nores, y_plain))
    assert e_prq < e_nores
    assert e_prq < e_plain


def test_e8m0_search_prepare_never_worse_per_block():
    """The E8M0-W export: same selection and permutation as plain, every
    32-block of Q(W~) and of Q(R_W) no worse than under plain Q(.) (exact
    squared errors), the residual still exact, and the compensated tail still
    no worse than the uncompensated one element by element."""
    c = inputs.tiny_case()
    plain = pq.prepare(c.W, c.Xcal, 0.5, 64)
    srch = pq.prepare(c.W, c.Xcal, 0.5, 64, scale_search=True)
    np.testing.assert_array_equal(plain["perm"], srch["perm"])
    K = plain["K"]
    Wt = srch["W_tilde"]
    codes_p, codes_s = plain["codes"], srch["codes"]
    sc_p, sc_s = plain["Wsc"], srch["Wsc"]
    e_p = mx.block_squared_errors(Wt, codes_p[:, :K], sc_p[:, :K // 32])
    e_s = mx.block_squared_errors(Wt, codes_s[:, :K], sc_s[:, :K // 32])
    assert np.all(e_s <= e_p) and np.any(e_s < e_p)
    R = srch["R"]
    deq_s = mx.mx_dequantize(codes_s, sc_s)
    np.testing.assert_array_equal(Wt[:, K - 64:].astype(np.float64) - deq_s[:, K - 64:K], R)
    comp = np.abs(Wt[:, K - 64:] - deq_s[:, K - 64:K] - deq_s[:, K:])
    assert np.all(comp <= np.abs(R))
    ref = pq.reference_product(c.X, c.W)
    y_s, _ = pq.prquant_forward(c.X, c.W, c.Xcal, 0.5, 64, scale_search=True)
    y_p, _ = pq.prquant_forward(c.X, c.W, c.Xcal, 0.5, 64)
    print(f"tiny y-NRMSE: PRQuant {pq.nrmse(y_p, ref):.5f}, E8M0-W {pq.nrmse(y_s, ref):.5f}")


def test_alpha_search_selects_the_smallest_error():
    """Algorithm 1's loop: each candidate's error equals the y-NRMSE of that
    alpha's export evaluated on the calibration rows, and the selection is the
    first minimizer; without scaling every alpha is the same export (equal
    errors: the first is kept)."""
    c = inputs.tiny_case()
    alphas = [0.0, 0.5, 1.0]
    best, errs = pq.search_alpha(c.W, c.Xcal, alphas, 64)
    ref = pq.reference_product(c.Xcal, c.W)
    for a, e in zip(alphas, errs):
        art = pq.prepare(c.W, c.Xcal, a, 64)
        Aq, Asc = pq.quant_act(c.Xcal, art["inv_scale"], art["perm"], 64)
        assert e == pq.nrmse(pq.gemm(Aq, Asc, art["Wq"], art["Wsc"]), ref)
    assert errs[best] == errs.min() and all(errs[i] > errs[best] for i in range(best))
    b2, e2 = pq.search_alpha(c.W, c.Xcal, [0.2, 0.7], 64, scale_mode="none")
    assert b2 == 0 and e2[0] == e2[1]


def test_no_perm_variant_reductions():
    """w/o Perm: when the selected channels already are the last k (the
    permutation is the identity) it is PRQuant itself; with k = 0 it is the
    scaled MXFP4 product; the compensated weight columns are never worse than
    the uncompensated ones element by element."""
    rng = np.random.default_rng(8)
    K, k = 128, 32
    W = 0.02 * rng.standard_normal((24, K))
    W[:, K - k:] *= 40                                  # the largest errors sit in the last k channels
    Wb = _bf16(W)
    Xc = _bf16(rng.standard_normal((16, K)))
    X = _bf16(rng.standard_normal((5, K)))
    art = pq.prepare(Wb, Xc, 0.5, k)
    np.testing.assert_array_equal(art["perm"], np.arange(K))
    y_np, _ = pq.no_perm_forward(X, Wb, Xc, 0.5, k)
    y_prq, _ = pq.prquant_forward(X, Wb, Xc, 0.5, k)
    np.testing.assert_array_equal(y_np, y_prq)
    y0, _ = pq.no_perm_forward(X, Wb, Xc, 0.5, 0)
    y00, _ = pq.prquant_forward(X, Wb, Xc, 0.5, 0)
    np.testing.assert_array_equal(y0, y00)
    c = inputs.tiny_case()
    a2 = pq.prepare_no_perm(c.W, c.Xcal, 0.5, 64)
    W_s = (pq.bf16_bits_to_f32(c.W) * a2["scale"][None, :]).astype(np.float32)
    deq = mx.mx_dequantize(a2["codes"], a2["Wsc"])
    S = a2["selected"]
    Kt = W_s.shape[1]
    comp = np.abs(W_s[:, S] - deq[:, S] - deq[:, Kt:])
    assert np.all(comp <= np.abs(W_s[:, S] - deq[:, S]))


def test_ablation_grid_directions_tiny():
    """The paper's ablation directions on the tiny workload: PRQuant beats
    plain MXFP4 and the same scaling without the residual; E8M0-W is no worse
    than PRQuant here.  (Whether scaling alone beats plain MXFP4 is reported,
    not asserted.)"""
    c = inputs.tiny_case()
    g = pq.ablation_grid(c.X, c.W, c.Xcal, 0.5, 64)
    print({k: round(v, 5) for k, v in g.items()})
    assert g["PRQuant"] < g["w/o Res"] and g["PRQuant"] < g["plain MXFP4"]
    assert g["E8M0-W"] <= g["PRQuant"]


def _pow2_inverse_scales(rng, C):
    return (2.0 ** rng.integers(-3, 4, C)).astype(np.float32)


def test_offline_copy_expanded_ffn_emits_the_augmented_activation():
    """Eq. 1 with exact arithmetic: with power-of-two inverse scales (exact in
    bf16) the expanded producer's FFN output is [Z~, Z~_tail] of the original
    FFN output, Z~[:, p] = Z[:, perm[p]] / s_{perm[p]}, bit for bit."""
    rng = np.random.default_rng(2)
    f = inputs.make_ffn("f", H=64, C=256, M=7, T=4, seed=2)
    k = 64
    perm = rng.permutation(f.C).astype(np.int32)
    inv = _pow2_inverse_scales(rng, f.C)
    up_aug, gate_aug = pq.expand_producer(f.W_up, f.W_gate, inv, perm, k)
    assert up_aug.shape == (f.C + k, f.H) and gate_aug.shape == (f.C + k, f.H)
    Z = pq.gated_ffn(f.X_hidden, f.W_up, f.W_gate)
    Zt = Z[:, perm] * inv[perm].astype(np.float64)
    want = np.concatenate([Zt, Zt[:, f.C - k:]], axis=1)
    got = pq.gated_ffn(f.X_hidden, up_aug, gate_aug)
    np.testing.assert_array_equal(got, want)


def test_offline_copy_quantizes_like_the_online_copy():
    """With power-of-two scales the plain quantizer over C + k on the expanded
    producer's (bf16) output gives the online copy's codes and scales."""
    rng = np.random.default_rng(3)
    f = inputs.make_ffn("f", H=64, C=256, M=9, T=4, seed=3)
    k = 64
    perm = rng.permutation(f.C).astype(np.int32)
    inv = _pow2_inverse_scales(rng, f.C)
    up_aug, gate_aug = pq.expand_producer(f.W_up, f.W_gate, inv, perm, k)
    z_aug = pq.bf16_round_bits(pq.gated_ffn(f.X_hidden, up_aug, gate_aug).astype(np.float32))
    off_q, off_s = pq.quant_act(z_aug, None, None, 0)
    z = pq.bf16_round_bits(pq.gated_ffn(f.X_hidden, f.W_up, f.W_gate).astype(np.float32))
    on_q, on_s = pq.quant_act(z, inv, perm, k)
    np.testing.assert_array_equal(off_s, on_s)
    np.testing.assert_array_equal(off_q, on_q)


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -9, -2.5e-40, 3.0e38],
                 np.float32)
    b = pq.bf16_round_bits(x)
    back = pq.bf16_bits_to_f32(b)
    assert back[0] == 1.0 and back[1] == 1.0              # tie -> even mantissa
    assert back[2] == np.float32(1.0 + 4 * 2.0 ** -8)     # tie -> even (up)
    assert back[3] == 1.0
    for v, r in zip(x, back):                               # nearest: |v - r| <= half an ulp
        ulp = np.spacing(np.float32(abs(r))) * 2 ** 16 if r != 0 else 2.0 ** -133
        assert abs(float(v) - float(r)) <= ulp / 2


def test_grouped_matches_per_expert():
    rng = np.random.default_rng(3)
    E, N, K, k = 4, 16, 64, 32
    counts = [3, 0, 5, 1]
    off = inputs.routed_offsets(counts)
    Mt = int(off[-1])
    X = _bf16(rng.standard_normal((Mt, K)))
    arts = [pq.prepare(_bf16(0.02 * rng.standard_normal((N, K))), _bf16(rng.standard_normal((8, K))),
                       0.5, k) for _ in range(E)]
    inv = np.stack([a["inv_scale"] for a in arts])
    perm = np.stack([a["perm"] for a in arts])
    Aq, Asc = pq.quant_act_grouped(X, inv, perm, off, k)
    Wq = np.stack([a["Wq"] for a in arts])
    Wsc = np.stack([a["Wsc"] for a in arts])
    Y = pq.grouped_gemm(Aq, Asc, off, Wq, Wsc)
    for e in range(E):
        r0, r1 = off[e], off[e + 1]
        if r1 > r0:
            a_e, s_e = pq.quant_act(X[r0:r1], inv[e], perm[e], k)
            np.testing.assert_array_equal(Aq[r0:r1], a_e)
            np.testing.assert_array_equal(Y[r0:r1], pq.gemm(a_e, s_e, Wq[e], Wsc[e]))


def test_prepare_rejects_misaligned():
    c = _small()
    with pytest.raises(ValueError):
        pq.prepare(c.W, c.Xcal, 0.5, 48)
    with pytest.raises(ValueError):
        pq.prepare(c.W, c.Xcal, 1.5, 64)
    with pytest.raises(ValueError):
        pq.prepare(c.W[:, :100], c.Xcal[:, :100], 0.5, 32)


# ---------------------------------------- normalized error, ablation table ---
def test_nrmse_hand_values():
    """||Y_hat - Y||_F / ||Y||_F (reading of the paper's normalized
    reconstruction error, Sec. 4.3) on hand-computed cases: the norm of the
    difference over the norm of the REFERENCE (not of the estimate), not
    squared, taken over every element of the matrix."""
    assert pq.nrmse([[3.0, 5.0]], [[3.0, 4.0]]) == 0.2          # 1 / 5
    assert pq.nrmse([[1.0, 2.0], [2.0, 7.0]], [[1.0, 2.0], [2.0, 4.0]]) == 0.6   # 3 / 5
    assert pq.nrmse([[0.0, 0.0]], [[3.0, 4.0]]) == 1.0          # the zero estimate
    assert pq.nrmse([[6.0, 8.0]], [[3.0, 4.0]]) == 1.0          # twice the reference
    assert pq.nrmse([[3.0, 4.0]], [[3.0, 4.0]]) == 0.0
    # a column vector and its transpose give the same Frobenius ratio
    assert pq.nrmse([[0.0], [1.0]], [[0.0], [2.0]]) == 0.5


def _eq3_direct(X_bf16, W_bf16, s, k, searched=False):
    """Eq. 3 assembled here from the MXFP4 primitives for given scales s:
    W~ = (W s)[:, P] with P the tail permutation of the k columns of largest
    MXFP4 error of W s (ties to the smaller index), R = W~_tail - deq Q(W~)_tail,
    A = Q([Z~, Z~_tail]) with Z~ = (X / s)[:, P], Y = deq(A) deq([Q(W~) | Q(R)])^T.
    `searched` quantizes W~ and R with the E8M0 block-scale search."""
    Xf = pq.bf16_bits_to_f32(X_bf16)
    Wf = pq.bf16_bits_to_f32(W_bf16)
    s = np.asarray(s, np.float32)
    inv = (np.float32(1.0) / s).astype(np.float32)
    K = Wf.shape[1]
    W_s = (Wf * s[None, :]).astype(np.float32)
    deq0 = mx.qdq(W_s)
    err = np.array([sum((float(W_s[n, j]) - float(deq0[n, j])) ** 2 for n in range(W_s.shape[0]))
                    for j in range(K)])
    order = sorted(range(K), key=lambda j: (-err[j], j))
    sel = sorted(order[:k])
    P = np.array([j for j in range(K) if j not in set(sel)] + sel, np.int64)
    Wt = W_s[:, P]
    quant = mx.mx_quantize_searched if searched else mx.mx_quantize
    cw, sw = quant(Wt)
    R = (Wt[:, K - k:].astype(np.float64) - mx.mx_dequantize(cw, sw)[:, K - k:]).astype(np.float32)
    cr, sr = quant(R) if k else (np.zeros((Wt.shape[0], 0), np.uint8),
                                 np.zeros((Wt.shape[0], 0), np.uint8))
    Zt = (Xf * inv[None, :]).astype(np.float32)[:, P]
    ca, sa = mx.mx_quantize(np.ascontiguousarray(np.concatenate([Zt, Zt[:, K - k:]], axis=1)))
    Wd = np.concatenate([mx.mx_dequantize(cw, sw), mx.mx_dequantize(cr, sr)], axis=1)
    return mx.mx_dequantize(ca, sa) @ Wd.T


def test_ablation_variants_match_their_definitions():
    """Each entry of the ablation grid (Sec. Ablation Studies) is the variant
    its name defines, assembled directly from the MXFP4 primitives:
      plain MXFP4: Q(X) Q(W)^T (no scaling, no tail);
      w/o Res:     Q(X / s) Q(W s)^T with the SmoothQuant scales (k = 0);
      w/o AWQ:     Eq. 3 with s = 1 and the k-column tail;
      PRQuant:     Eq. 3 with the SmoothQuant scales and the tail;
      E8M0-W:      PRQuant with the weight block scales searched;
    and the device grid's variant table is the oracle's."""
    from paper_2609_22106_amd import ablation
    assert ablation.VARIANTS == pq.ABLATION_VARIANTS
    rng = np.random.default_rng(31)
    N, K, k, alpha = 24, 128, 32, 0.5
    W = 0.02 * rng.standard_normal((N, K))
    W[:, rng.choice(K, 5, replace=False)] *= 15
    Wb = _bf16(W)
    out = rng.choice(K, 4, replace=False)
    Xc = rng.standard_normal((16, K))
    Xc[:, out] *= 30
    X = rng.standard_normal((6, K))
    X[:, out] *= 30
    Xcb, Xb = _bf16(Xc), _bf16(X)
    g = pq.ablation_grid(Xb, Wb, Xcb, alpha, k)
    ref = pq.bf16_bits_to_f32(Xb).astype(np.float64) @ pq.bf16_bits_to_f32(Wb).astype(np.float64).T
    s, _ = pq.channel_scales(Wb, Xcb, alpha, "smooth")
    plain = mx.qdq(pq.bf16_bits_to_f32(Xb)) @ mx.qdq(pq.bf16_bits_to_f32(Wb)).T
    want = {
        "plain MXFP4": plain,
        "w/o Res": _eq3_direct(Xb, Wb, s, 0),
        "w/o AWQ": _eq3_direct(Xb, Wb, np.ones(K, np.float32), k),
        "PRQuant": _eq3_direct(Xb, Wb, s, k),
        "E8M0-W": _eq3_direct(Xb, Wb, s, k, searched=True),
    }
    for name, y in want.items():
        e = float(np.linalg.norm(y - ref) / np.linalg.norm(ref))
        assert g[name] == pytest.approx(e, rel=1e-12, abs=0), name
    # the five values are distinct, so no two names can trade places unnoticed
    vals = [g[n] for n in want]
    assert len(set(vals)) == len(vals), g


# --------------------------------------------------------------------------- #
# Offline copy, producer side: SiLU(gate) * up quantized as it is formed
# --------------------------------------------------------------------------- #
def _ulps(got, want):
    got = np.asarray(got, np.float32)
    return np.abs(got.astype(np.float64) - want) / np.spacing(np.abs(got)).astype(np.float64)


def test_exp_f32_against_float64():
    """The fixed float32 exponential stays within 3 ulp of the float64 exp on
    a dense sweep of its finite range; e^0 = 1 exactly; past the clamp it is
    0 or inf."""
    x = np.linspace(-87.0, 88.0, 350001, dtype=np.float32)
    e = pq.exp_f32(x)
    assert np.all(np.isfinite(e)) and np.all(e > 0)
    assert _ulps(e, np.exp(x.astype(np.float64))).max() <= 3.0
    assert pq.exp_f32(np.float32(0.0)) == np.float32(1.0)
    assert pq.exp_f32(np.float32(1.0)) == np.float32(math.e)
    big = pq.exp_f32(np.array([89.0, 1e30, np.finfo(np.float32).max], np.float32))
    assert np.all(np.isinf(big)) and np.all(big > 0)
    assert np.all(pq.exp_f32(np.array([-104.0, -1e30, -np.finfo(np.float32).max], np.float32)) == 0)


def test_silu_f32_against_float64():
    """SiLU(g) = g / (1 + e^-g) within 5 ulp of its float64 value while 1 + e^-g
    is finite in float32 (g >= -85); SiLU(0) = 0; SiLU(g) = g exactly once e^-g
    is below half an ulp of 1 (g >= 17); -0 far left, where e^-g overflows
    float32 (the float64 value there is below 1e-35)."""
    g = np.linspace(-85.0, 100.0, 400001, dtype=np.float32)
    s = pq.silu_f32(g)
    ref = g.astype(np.float64) / (1.0 + np.exp(-g.astype(np.float64)))
    keep = np.abs(ref) > 0
    assert _ulps(s[keep], ref[keep]).max() <= 5.0
    assert pq.silu_f32(np.float32(0.0)) == 0.0
    big = np.array([17.0, 100.0, 3.0e38], np.float32)
    np.testing.assert_array_equal(pq.silu_f32(big), big)
    far = pq.silu_f32(np.array([-104.0, -1e20], np.float32))
    assert np.all(far == 0) and np.all(np.signbit(far))


def test_swiglu_quant_definition():
    """The gate gets the SiLU, the up output multiplies it (against the float64
    formula with the roles written out: a swap fails); where SiLU is exact
    (gate >= 17) the codes are those of Q(gate * up) formed directly; a zero
    gate gives zeros carrying the up output's sign and the all-zero scale."""
    rng = np.random.default_rng(41)
    M, K = 5, 96
    gate = rng.standard_normal((M, K)).astype(np.float32) * 3
    up = rng.standard_normal((M, K)).astype(np.float32) * 2
    gb, ub = pq.bf16_round_bits(gate), pq.bf16_round_bits(up)
    g64 = pq.bf16_bits_to_f32(gb).astype(np.float64)
    u64 = pq.bf16_bits_to_f32(ub).astype(np.float64)
    z = pq.swiglu_f32(gb, ub)
    want = u64 * g64 / (1.0 + np.exp(-g64))
    assert _ulps(z[np.abs(want) > 1e-30], want[np.abs(want) > 1e-30]).max() <= 5.0
    swapped = g64 * u64 / (1.0 + np.exp(-u64))
    assert np.max(np.abs(z - swapped)) > 1e-2
    # exact SiLU: gate >= 17
    gate_hi = pq.bf16_round_bits(17.0 + np.abs(rng.standard_normal((M, K))).astype(np.float32) * 40)
    Aq, Asc = pq.swiglu_quant(gate_hi, ub)
    direct = (pq.bf16_bits_to_f32(gate_hi) * pq.bf16_bits_to_f32(ub)).astype(np.float32)
    c, sc = mx.mx_quantize(direct)
    np.testing.assert_array_equal(Aq, mx.pack_codes(c))
    np.testing.assert_array_equal(Asc, sc)
    Aq0, Asc0 = pq.swiglu_quant(np.zeros((M, K), np.uint16), ub)   # 0 * up: signed zeros
    c0 = mx.unpack_codes(Aq0)
    assert not (c0 & 7).any() and not Asc0.any()
    np.testing.assert_array_equal(c0 >> 3, np.signbit(pq.bf16_bits_to_f32(ub)).astype(np.uint8))


def test_swiglu_quant_of_expanded_producers_is_the_augmented_activation():
    """Offline copy end to end on the oracle: the expanded producers' outputs
    (bf16) through SiLU(gate) * up give, column for column, the permuted and
    scaled gated activation with its last k channels repeated -- the
    [Z~, Z~_tail] layout of Eq. 3 -- so the quantized result has its tail
    blocks equal to the copied ones."""
    rng = np.random.default_rng(43)
    H, C, k, M = 64, 128, 32, 6
    Wup = pq.bf16_round_bits((rng.standard_normal((C, H)) * 0.1).astype(np.float32))
    Wg = pq.bf16_round_bits((rng.standard_normal((C, H)) * 0.1).astype(np.float32))
    X = pq.bf16_round_bits(rng.standard_normal((M, H)).astype(np.float32))
    inv = (np.float32(1.0) / rng.uniform(0.5, 2.0, C).astype(np.float32)).astype(np.float32)
    perm = rng.permutation(C)
    up_aug, gate_aug = pq.expand_producer(Wup, Wg, inv, perm, k)
    Xf = pq.bf16_bits_to_f32(X).astype(np.float64)
    up_out = pq.bf16_round_bits((Xf @ pq.bf16_bits_to_f32(up_aug).astype(np.float64).T).astype(np.float32))
    g_out = pq.bf16_round_bits((Xf @ pq.bf16_bits_to_f32(gate_aug).astype(np.float64).T).astype(np.float32))
    Aq, Asc = pq.swiglu_quant(g_out, up_out)
    assert Aq.shape == (M, (C + k) // 2) and Asc.shape == (M, (C + k) // 32)
    np.testing.assert_array_equal(Aq[:, (C + k) // 2 - k // 2:], Aq[:, C // 2 - k // 2:C // 2])
    np.testing.assert_array_equal(Asc[:, -(k // 32):], Asc[:, C // 32 - k // 32:C // 32])
