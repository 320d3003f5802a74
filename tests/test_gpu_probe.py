"""Single-instruction checks of the gfx950 semantics the kernels rely on:
the operand/scale/output lane layout of the block-scaled FP4 MFMA, and the
hardware FP32->FP4 conversion against the E2M1 rounding rule (all finite
float32 inputs).  In-bounds by construction (one wave; a fixed sweep)."""
import ctypes
import itertools

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


def _probe_lib():
    from paper_2609_22106_amd import build, prq  # noqa: F401  (prq loads torch first)
    lib = ctypes.CDLL(build.PROBE_LIB)
    lib.prq_probe_mfma16.argtypes = [ctypes.c_void_p] * 6
    lib.prq_probe_cvt_sweep.argtypes = [ctypes.c_void_p] * 2
    lib.prq_probe_cvt_pairs.argtypes = [ctypes.c_void_p] * 3 + [ctypes.c_int] + [ctypes.c_void_p] * 2
    return lib


E2M1 = np.array([0, .5, 1, 1.5, 2, 3, 4, 6, -0., -.5, -1, -1.5, -2, -3, -4, -6])


def _nibbles(lane_bytes, high_first):
    lo, hi = lane_bytes & 15, lane_bytes >> 4
    pair = (hi, lo) if high_first else (lo, hi)
    return np.stack(pair, axis=-1).reshape(lane_bytes.shape[0], 32)


def _operand(lane_bytes, lane_scales, layout, high_first):
    """16 x 128 matrix of values under a lane-layout hypothesis."""
    mat = np.zeros((16, 128))
    vals = E2M1[_nibbles(lane_bytes, high_first)]
    for l in range(64):
        r, g = l % 16, l // 16
        if layout == "contiguous32":
            ks = np.arange(32 * g, 32 * g + 32)
        else:  # two 16-element halves, 64 apart
            ks = np.concatenate([np.arange(16 * g, 16 * g + 16), np.arange(64 + 16 * g, 80 + 16 * g)])
        mat[r, ks] = vals[l] * 2.0 ** (int(lane_scales[l]) - 127)
    return mat


def test_block_scaled_fp4_mfma_layout():
    lib = _probe_lib()
    rng = np.random.default_rng(0)
    a = rng.integers(0, 256, (64, 16), dtype=np.uint8)
    b = rng.integers(0, 256, (64, 16), dtype=np.uint8)
    sa = rng.integers(124, 131, 64).astype(np.uint32)
    sb = rng.integers(124, 131, 64).astype(np.uint32)
    dev = [torch.from_numpy(x.copy()).cuda() for x in (a, b, sa.view(np.int32), sb.view(np.int32))]
    out = torch.zeros(64 * 4, dtype=torch.float32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    assert lib.prq_probe_mfma16(*[t.data_ptr() for t in dev], out.data_ptr(), s) == 0
    got = out.cpu().numpy().reshape(64, 4).astype(np.float64)
    matches = []
    for layout, high_first, transposed in itertools.product(("contiguous32", "split16"), (False, True),
                                                            (False, True)):
        A = _operand(a, sa, layout, high_first)
        B = _operand(b, sb, layout, high_first)
        C = A @ B.T
        pred = np.zeros((64, 4))
        for l in range(64):
            for q in range(4):
                i, j = 4 * (l // 16) + q, l % 16
                pred[l, q] = C[j, i] if transposed else C[i, j]
        if np.allclose(pred, got, rtol=1e-6, atol=1e-6 * np.abs(C).max()):
            matches.append((layout, high_first, transposed))
    print("matching layouts:", matches, flush=True)
    assert ("contiguous32", False, False) in matches, f"layout differs; matches={matches}\n{got[:4]}"


def test_block_scaled_fp4_mfma_32x32x64_layout():
    """The 32x32x64 form: lane l supplies row l % 32 and K elements
    [32 (l / 32), +32) of its operand (low nibble first), with that block's
    scale; it receives C[8 (j / 4) + 4 (l / 32) + j % 4][l % 32] in element j."""
    lib = _probe_lib()
    lib.prq_probe_mfma32.argtypes = [ctypes.c_void_p] * 6
    rng = np.random.default_rng(1)
    a = rng.integers(0, 256, (64, 16), dtype=np.uint8)
    b = rng.integers(0, 256, (64, 16), dtype=np.uint8)
    sa = rng.integers(124, 131, 64).astype(np.uint32)
    sb = rng.integers(124, 131, 64).astype(np.uint32)
    dev = [torch.from_numpy(x.copy()).cuda() for x in (a, b, sa.view(np.int32), sb.view(np.int32))]
    out = torch.zeros(64 * 16, dtype=torch.float32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    assert lib.prq_probe_mfma32(*[t.data_ptr() for t in dev], out.data_ptr(), s) == 0
    got = out.cpu().numpy().reshape(64, 16).astype(np.float64)

    def operand(lane_bytes, lane_scales):
        mat = np.zeros((32, 64))
        vals = E2M1[_nibbles(lane_bytes, False)]
        for l in range(64):
            r, g = l % 32, l // 32
            mat[r, 32 * g:32 * g + 32] = vals[l] * 2.0 ** (int(lane_scales[l]) - 127)
        return mat

    C = operand(a, sa) @ operand(b, sb).T
    hyps = {
        "8(j/4)+4(l/32)+j%4": lambda l, j: (8 * (j // 4) + 4 * (l // 32) + j % 4, l % 32),
        "16(l/32)+j": lambda l, j: (16 * (l // 32) + j, l % 32),
        "transposed": lambda l, j: (l % 32, 8 * (j // 4) + 4 * (l // 32) + j % 4),
    }
    matches = []
    for name, f in hyps.items():
        pred = np.array([[C[f(l, j)] for j in range(16)] for l in range(64)])
        if np.allclose(pred, got, rtol=1e-6, atol=1e-6 * np.abs(C).max()):
            matches.append(name)
    print("32x32x64 matching layouts:", matches, flush=True)
    assert matches == ["8(j/4)+4(l/32)+j%4"], f"layout differs; matches={matches}\n{got[:2]}"


def test_hw_fp4_convert_matches_rounding_rule():
    lib = _probe_lib()
    res = torch.zeros(17, dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    assert lib.prq_probe_cvt_sweep(res.data_ptr(), s) == 0
    r = res.cpu().numpy().view(np.uint32)
    first = [(hex(r[1 + 2 * k]), hex(r[2 + 2 * k])) for k in range(min(8, int(r[0])))]
    print("cvt mismatches:", int(r[0]), first, flush=True)
    # scale-operand semantics, reported for the record
    x = torch.tensor([3.0, 3.0, 0.75, 5.0], device="cuda")
    y = torch.tensor([1.0, 1.0, -0.1, 6.5], device="cuda")
    sc = torch.tensor([1.0, 2.0, 1.0, 1.0], device="cuda")
    o = torch.zeros(4, dtype=torch.uint8, device="cuda")
    assert lib.prq_probe_cvt_pairs(x.data_ptr(), y.data_ptr(), sc.data_ptr(), 4, o.data_ptr(), s) == 0
    print("cvt pairs (x=3,y=1,s=1), (x=3,y=1,s=2), (.75,-.1), (5,6.5):",
          [hex(v) for v in o.cpu().numpy()], flush=True)
    assert int(r[0]) == 0


def test_direct_global_to_lds_load_layout():
    """global_load_lds: lane l's 16 bytes land at LDS base + 16 l (one
    lane-ordered MFMA operand block per wave instruction); lane l's single byte
    lands in the dword slot at base + 4 l, upper bytes zero (how the tile GEMM
    stages its scale bytes)."""
    from paper_2609_22106_amd import build
    lib = ctypes.CDLL(build.PROBE_LIB)
    lib.prq_probe_lds_dma.argtypes = [ctypes.c_void_p] * 4
    rng = np.random.default_rng(5)
    g16 = rng.integers(1, 256, 1024, dtype=np.uint8)
    g1 = rng.integers(1, 256, 64, dtype=np.uint8)
    d16, d1 = torch.from_numpy(g16).cuda(), torch.from_numpy(g1).cuda()
    out = torch.zeros(8192, dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    assert lib.prq_probe_lds_dma(d16.data_ptr(), d1.data_ptr(), out.data_ptr(), s) == 0
    o = out.cpu().numpy()
    nz16 = np.flatnonzero(o[:4096])
    nz1 = np.flatnonzero(o[4096:])
    print("lds dma: 16-byte data at", nz16[:4], "...", nz16[-2:], "; bytes at", nz1[:8], flush=True)
    np.testing.assert_array_equal(o[:1024], g16)
    assert not o[1024:4096].any()
    slots = o[4096:4096 + 256].reshape(64, 4)
    np.testing.assert_array_equal(slots[:, 0], g1)
    assert not slots[:, 1:].any() and not o[4096 + 256:].any()


def test_fp4_convert_destination_byte_select():
    """Byte `sel` of the result holds the pair's codes (x low nibble, y high),
    the other three bytes of the old value are kept: the quantizers build a
    word of 8 codes with four converts and no masking."""
    lib = _probe_lib()
    lib.prq_probe_cvt_sel.argtypes = [ctypes.c_void_p] * 4
    rng = np.random.default_rng(4)
    x = rng.choice(E2M1, 64).astype(np.float32)
    y = rng.choice(E2M1, 64).astype(np.float32)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    out = torch.zeros(256, dtype=torch.int32, device="cuda")
    assert lib.prq_probe_cvt_sel(xd.data_ptr(), yd.data_ptr(), out.data_ptr(),
                                 torch.cuda.current_stream().cuda_stream) == 0
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint32).reshape(64, 4)
    code = {float(v): i for i, v in enumerate(E2M1[:8])}

    def c(v):
        return code[abs(float(v))] | (8 if np.signbit(v) else 0)
    old = 0x89ABCDEF
    for l in range(64):
        pair = c(x[l]) | (c(y[l]) << 4)
        for sel in range(4):
            want = (old & ~(0xFF << (8 * sel))) | (pair << (8 * sel))
            assert int(got[l, sel]) == want, (l, sel, hex(int(got[l, sel])), hex(want))



def _lds_pattern_expected(mode, iters):
    """The folded value of every thread of the LDS read-pattern kernel (the
    LDS word i holds i * 2654435761 mod 2^32), computed on the host."""
    words = (np.arange(4096, dtype=np.uint64) * 2654435761) & 0xFFFFFFFF
    halves = words.astype(np.uint32).view(np.uint16)   # little-endian 2-byte pieces
    out = np.zeros(256, dtype=np.uint64)
    for tid in range(256):
        lane, wave = tid & 63, tid >> 6
        acc = 0
        for it in range(iters):
            base = ((it + wave) & 15) * 1024
            if mode == 0:
                w = (base + 16 * lane) // 4
                acc ^= int(words[w] ^ words[w + 1] ^ words[w + 2] ^ words[w + 3])
            elif mode == 1:
                acc ^= int(words[(base + ((lane >> 4) & 1) * 256 + ((lane & 15) + 16 * (lane >> 5)) * 4) // 4])
            elif mode == 2:
                acc ^= int(words[(base + 4 * lane) // 4])
            elif mode == 4:
                odd = (lane >> 4) & 1
                acc ^= int(words[(base + odd * 256 + ((lane & 15) + 16 * ((lane >> 5) ^ odd)) * 4) // 4])
            else:
                acc = (acc + sum(int(halves[(base + 16 * lane + 2 * j) // 2]) for j in range(8))) & 0xFFFFFFFF
        out[tid] = acc
    return out.astype(np.uint32)


@pytest.mark.parametrize("mode", [0, 1, 2, 3, 4])
def test_lds_read_pattern_probe(mode):
    """The LDS read-pattern kernels (reference points for the bank-conflict
    counters: the tile GEMM's operand reads, its scale reads without and with
    the staging swap, one dword per bank, the quantizer's 2-byte gather) read
    what their patterns name."""
    from paper_2609_22106_amd import build
    lib = ctypes.CDLL(build.PROBE_LIB)
    lib.prq_probe_lds_pattern.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                          ctypes.c_void_p]
    blocks, iters = 3, 37
    out = torch.zeros(blocks * 256, dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    assert lib.prq_probe_lds_pattern(mode, blocks, iters, out.data_ptr(), s) == 0
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint32).reshape(blocks, 256)
    exp = _lds_pattern_expected(mode, iters)
    for b in range(blocks):
        np.testing.assert_array_equal(got[b], exp)
