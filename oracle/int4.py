"""INT4 factor encoding (Section 4.3, "Quantization Compatibility") -- test
infrastructure, see oracle/__init__.py. Written in numpy, fp64.

Steps, in the paper's order:
  1. Balance the truncated-SVD factors by absorbing Sigma^(1/2) into both:
     L~ = U Sigma^(1/2), R~ = Sigma^(1/2) W^T. From the Eq. (2) pair
     (L = U_r, R = Sigma_r W_r^T) this is L~ = L diag(sqrt s), R~ = diag(1/sqrt s) R;
     a zero singular value gives a zero column of L~ and a zero row of R~.
  2. Symmetric INT4 per factor, along the paper's direction: column-wise for
     L~_K, R~_K and R~_V, row-wise for L~_V. Each line is cut into runs of at
     most 32 consecutive elements; every run has its own scale.
  3. Scale s = fp16 round-to-nearest-even of max|x| / 7 over the run; code =
     clamp(round-half-even(x / s), -7, 7) with the division in fp64; s = 0 gives
     all-zero codes. The dequantized value is code * s.

Reading taken where the paper is silent: the run length (32), the fp16 scale,
the symmetric range [-7, 7] and round-half-even.
"""
from __future__ import annotations

import numpy as np

GROUP = 32
QMAX = 7


def balance(L: np.ndarray, R: np.ndarray, sig: np.ndarray):
    """Step 1: (L diag(sqrt s), diag(1/sqrt s) R) for the first r singular values."""
    r = L.shape[1]
    s = np.asarray(sig[:r], dtype=np.float64)
    root = np.sqrt(np.maximum(s, 0.0))
    inv = np.where(root > 0.0, 1.0 / np.where(root > 0.0, root, 1.0), 0.0)
    Lt = np.asarray(L, dtype=np.float64) * root[None, :]
    Rt = np.asarray(R, dtype=np.float64) * inv[:, None]
    Lt[:, root == 0.0] = 0.0
    return Lt, Rt


def quantize_lines(x: np.ndarray, axis: int, group: int = GROUP):
    """Steps 2-3 along `axis` (0: each column is a line, 1: each row is a line).

    Returns (codes int8 with x's shape, scales float64 of shape
    (runs_per_line, n_lines)); scales are exact fp16 values."""
    x = np.asarray(x, dtype=np.float64)
    lines = x if axis == 0 else x.T            # lines are the columns of `lines`
    n, m = lines.shape
    runs = -(-n // group)
    codes = np.zeros((n, m), dtype=np.int8)
    scales = np.zeros((runs, m), dtype=np.float64)
    for g in range(runs):
        blk = lines[g * group:(g + 1) * group, :]
        amax = np.abs(blk).max(axis=0)
        s = (amax / QMAX).astype(np.float16).astype(np.float64)   # fp16 RNE
        scales[g] = s
        safe = np.where(s > 0.0, s, 1.0)
        c = np.clip(np.rint(blk / safe[None, :]), -QMAX, QMAX)
        c[:, s == 0.0] = 0
        codes[g * group:(g + 1) * group, :] = c.astype(np.int8)
    if axis == 1:
        codes = codes.T.copy()
    return codes, scales


def dequantize_lines(codes: np.ndarray, scales: np.ndarray, axis: int,
                     group: int = GROUP) -> np.ndarray:
    c = np.asarray(codes, dtype=np.float64)
    lines = c if axis == 0 else c.T
    n = lines.shape[0]
    out = np.empty_like(lines)
    for g in range(scales.shape[0]):
        out[g * group:(g + 1) * group, :] = lines[g * group:(g + 1) * group, :] * scales[g][None, :]
    return out if axis == 0 else out.T.copy()


# Direction of each factor (Section 4.3): 0 = column-wise, 1 = row-wise.
AXIS = {"L_K": 0, "R_K": 0, "L_V": 1, "R_V": 0}


def encode_page(which: str, L: np.ndarray, R: np.ndarray, sig: np.ndarray):
    """Balance and quantize one factor pair; which is "K" or "V".

    Returns dict with codes/scales for L and R and their dequantized values."""
    Lt, Rt = balance(L, R, sig)
    aL, aR = AXIS["L_" + which], AXIS["R_" + which]
    cL, sL = quantize_lines(Lt, aL)
    cR, sR = quantize_lines(Rt, aR)
    return {
        "L_bal": Lt, "R_bal": Rt,
        "L_codes": cL, "L_scales": sL, "R_codes": cR, "R_scales": sR,
        "L_deq": dequantize_lines(cL, sL, aL), "R_deq": dequantize_lines(cR, sR, aR),
    }
