"""Activation diagnostics behind the paper's Figs. 2-4 (oracle; test infrastructure only).

Sec. 4.2 explains the rollout accuracy loss by the activations' distribution:
  * Fig. 2: the share of zero values in an activation tensor before quantization (bf16) and
    after it (the "zero collapse" of Q(X) in layers with outliers);
  * Fig. 3: the share of quantization blocks (the format's block size along d) holding an
    outlier, which tracks that collapse;
  * Fig. 4: the error that S_2:4 causes on Q(X) and on Q(Delta X), as MSE and RMSE between a
    quantized tensor and its S_2:4-sparsified version (Sec. 4.3 uses it to motivate
    sparsifying the residual rather than the activation).

Readings of points the paper leaves open (also listed in the design notes):

  D1  a zero of Q(X) is an element whose dequantized value is 0 (magnitude code 0, either
      sign); a zero of X is a bf16 +0 or -0.
  D2  the paper does not define an outlier.  A block holds one when some |x| > T for a
      threshold T the caller chooses (for example a multiple of the tensor's RMS); the
      comparison is made on float32 values.
  D3  the S_2:4 error of a quantized tensor q is sum over elements of (q - S_2:4(q))^2, i.e.
      the sum of the squares of the pruned values, divided by m*d for the MSE; RMSE is its
      square root.  S_2:4 is the function of Sec. 4.3 (two largest |values| of every four,
      lower index on ties).
"""
from __future__ import annotations

import numpy as np

from . import formats as F
from . import resq as Q

# Order of the statistics (the library writes the same order).
FIELDS = ("elements", "zeros_x", "zeros_qx", "blocks", "outlier_blocks", "energy_qx",
          "sse24_qx", "energy_qr", "sse24_qr")


def diagnostics(fmt: str, x: np.ndarray, threshold: float) -> dict:
    """The Figs. 2-4 statistics of activations x (m x d, values of bf16 inputs as float32)."""
    x = np.asarray(x, dtype=np.float32)
    m, d = x.shape
    b = F.block_size(fmt)
    codes, scales = F.quantize(fmt, x)
    xhat = F.dequantize(fmt, codes, scales)
    r = Q.residual(x, xhat)
    rcodes, rscales = F.quantize(fmt, r)
    rhat = F.dequantize(fmt, rcodes, rscales)
    amax = np.abs(x).reshape(m, d // b, b).max(axis=-1)
    keep_x, keep_r = Q.keep_2_4(xhat), Q.keep_2_4(rhat)
    return {
        "elements": m * d,
        "zeros_x": int(np.count_nonzero(x == 0)),
        "zeros_qx": int(np.count_nonzero(xhat == 0)),
        "blocks": m * (d // b),
        "outlier_blocks": int(np.count_nonzero(amax > np.float32(threshold))),
        "energy_qx": float(np.sum(xhat.astype(np.float64) ** 2)),
        "sse24_qx": float(np.sum(np.where(keep_x, 0.0, xhat.astype(np.float64)) ** 2)),
        "energy_qr": float(np.sum(rhat.astype(np.float64) ** 2)),
        "sse24_qr": float(np.sum(np.where(keep_r, 0.0, rhat.astype(np.float64)) ** 2)),
    }


def mse_rmse(stats: dict, which: str = "qx"):
    """(MSE, RMSE) of S_2:4 on Q(X) (which="qx") or on Q(Delta X) (which="qr"), reading D3."""
    mse = stats["sse24_" + which] / stats["elements"]
    return mse, float(np.sqrt(mse))
