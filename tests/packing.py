"""The packed operand layout of include/prq.h written out from its definition
(plain loops over rows, K steps and lanes; no GPU): used by the GPU tests to
build expected packed bytes from the oracle's row-major codes and scales."""
import numpy as np


def pack_rows(q, sc):
    """Row-major codes q [..., R, K_aug/2] and scales sc [..., R, K_aug/32] ->
    (codes [..., ceil(R/16), S, 64, 16], scales [..., ceil(R/16), ceil(S/4), 64, 4]),
    flattened.  Rows past R and K positions past K_aug: zero codes, scale 127."""
    q = np.asarray(q, dtype=np.uint8)
    sc = np.asarray(sc, dtype=np.uint8)
    lead = q.shape[:-2]
    R, Kh = q.shape[-2:]
    K_aug = 2 * Kh
    S = -(-K_aug // 128)
    Q = -(-S // 4)
    nb = K_aug // 32
    B = -(-R // 16)
    P = np.zeros(lead + (B, S, 64, 16), np.uint8)
    Ps = np.zeros(lead + (B, Q, 64, 4), np.uint8)
    for t in range(B):
        for lane in range(64):
            row = 16 * t + lane % 16
            for s in range(S):
                k0 = (128 * s + 32 * (lane // 16)) // 2
                if row < R and k0 < Kh:
                    P[..., t, s, lane, :] = q[..., row, k0:k0 + 16]
            for qq in range(Q):
                for j in range(4):
                    b = 4 * (4 * qq + j) + lane // 16
                    Ps[..., t, qq, lane, j] = sc[..., row, b] if (row < R and b < nb) else 127
    return P.ravel(), Ps.ravel()
