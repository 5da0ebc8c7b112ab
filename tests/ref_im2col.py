"""A second, separately written formulation of the convolution, used only to
pin the oracle: explicit im2col (the "explicit GEMM-based convolution" of the
paper's related work, Sec. 3) followed by a naive matrix product.

It builds the (IC*fltH*fltW) x (B*outH*outW) patch matrix with zero rows for
taps outside the input, then multiplies by the OC x (IC*fltH*fltW) filter
matrix.  Output sizes are counted by walking window positions, not by the
floor formula, so this file shares no formula with the oracle.
"""
import numpy as np


def _positions(size, pad, k, stride):
    # window start positions (in padded coordinates) that fit entirely
    out = []
    start = 0
    while start + k <= size + 2 * pad:
        out.append(start)
        start += stride
    return out


def im2col_conv_nchw(x, w, stride=(1, 1), pad=(0, 0), dtype=np.float64):
    """x[N,C,H,W], w[K,C,R,S] -> y[N,K,Ho,Wo] via im2col + naive GEMM."""
    N, C, H, W = x.shape
    K, C2, R, S = w.shape
    assert C == C2
    rows = _positions(H, pad[0], R, stride[0])
    cols = _positions(W, pad[1], S, stride[1])
    Ho, Wo = len(rows), len(cols)
    patches = np.zeros((C * R * S, N * Ho * Wo), dtype=dtype)
    for b in range(N):
        for i, top in enumerate(rows):
            for j, left in enumerate(cols):
                col = (b * Ho + i) * Wo + j
                for c in range(C):
                    for r in range(R):
                        for s in range(S):
                            yy = top + r - pad[0]
                            xx = left + s - pad[1]
                            if 0 <= yy < H and 0 <= xx < W:
                                patches[(c * R + r) * S + s, col] = x[b, c, yy, xx]
    fmat = w.reshape(K, C * R * S).astype(dtype)
    out = np.zeros((K, N * Ho * Wo), dtype=dtype)
    for k in range(K):                       # naive GEMM
        for q in range(C * R * S):
            f = fmat[k, q]
            if f != 0:
                out[k, :] += f * patches[q, :]
    return out.reshape(K, N, Ho, Wo).transpose(1, 0, 2, 3).copy()
