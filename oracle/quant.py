"""Block-scaled 8-bit weight quantisation, as the quantised workload stores its
matrices.  TEST INFRASTRUCTURE ONLY (nothing on the product path imports this).

The paper's applications run GGUF models whose sizes (Tab. "model_conf") put
them at about 8.5 bits per weight (Sec. "Experiment Setup"); the paper does not
spell the format out.  The reading taken here: each row of a matrix [out, in] is
cut into blocks of 32 consecutive weights along the input dimension, and a block
is stored as 32 signed 8-bit codes plus one half-precision scale (34 bytes per 32
weights = 8.5 bits per weight).  Every decision is made in float32:

  s   = max_i |w_i| / 127                 float32 division of float32 values
  d   = fp16(s)                            nearest half-precision value, ties to even
  q_i = clamp(rint(w_i / d), -127, 127)    float32 division, rint = ties to even;
                                           q_i = 0 for every i when d == 0
  w'_i = q_i * d                           the weight the quantised model computes with
                                           (exact in float32 and float64: <= 19 bits)

Weights must be finite and small enough that s is finite in half precision.
"""

from __future__ import annotations

import numpy as np

BLOCK = 32
QMAX = 127


def quantize_q8(w) -> tuple[np.ndarray, np.ndarray]:
    """Quantise a float32 matrix [rows, cols] (cols a multiple of 32).  Returns the
    int8 codes [rows, cols] and the float16 scales [rows, cols / 32]."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    rows, cols = w.shape
    if cols % BLOCK:
        raise ValueError("cols must be a multiple of 32")
    if not np.all(np.isfinite(w)):
        raise ValueError("non-finite weight")
    blocks = w.reshape(rows, cols // BLOCK, BLOCK)
    amax = np.max(np.abs(blocks), axis=2)                       # float32
    s = (amax / np.float32(QMAX)).astype(np.float32)           # float32 division
    d = s.astype(np.float16)                                    # ties to even
    if not np.all(np.isfinite(d)):
        raise ValueError("block scale overflows half precision")
    d32 = d.astype(np.float32)
    safe = np.where(d32 == 0, np.float32(1), d32)
    ratio = (blocks / safe[:, :, None]).astype(np.float32)      # float32 division
    q = np.clip(np.rint(ratio), -QMAX, QMAX)
    q = np.where(d32[:, :, None] == 0, 0, q).astype(np.int8)
    return q.reshape(rows, cols), d


def dequantize_q8(q: np.ndarray, d: np.ndarray) -> np.ndarray:
    """w' = q * d per block, as float64 (exact)."""
    rows, cols = q.shape
    scale = np.repeat(d.astype(np.float64), BLOCK, axis=1)
    return q.astype(np.float64) * scale


def quantize_q8_loops(w) -> tuple[np.ndarray, np.ndarray]:
    """The same rule written as scalar loops (for small inputs): each block's scale,
    then each code, with numpy float32 / float16 scalars doing the rounding."""
    w = np.asarray(w, dtype=np.float32)
    rows, cols = w.shape
    q = np.zeros((rows, cols), np.int8)
    d = np.zeros((rows, cols // BLOCK), np.float16)
    for r in range(rows):
        for b in range(cols // BLOCK):
            blk = [np.float32(v) for v in w[r, b * BLOCK:(b + 1) * BLOCK]]
            amax = np.float32(0)
            for v in blk:
                if abs(v) > amax:
                    amax = np.float32(abs(v))
            scale = np.float16(np.float32(amax / np.float32(QMAX)))
            d[r, b] = scale
            if np.float32(scale) == 0:
                continue
            for i, v in enumerate(blk):
                c = float(np.rint(np.float32(v / np.float32(scale))))
                q[r, b * BLOCK + i] = int(min(max(c, -QMAX), QMAX))
    return q, d


def q8_model_f64(weights: dict, threads: int = 16) -> dict:
    """Oracle weights of a block-scaled 8-bit model from its source tensors (bf16 bit
    patterns as uint16, or float32): every matrix quantised and dequantised to
    float64, every vector (norm gains) widened to float64."""
    from concurrent.futures import ThreadPoolExecutor

    def one(item):
        name, a = item
        a = np.asarray(a)
        f = (a.astype(np.uint32) << 16).view(np.float32) if a.dtype == np.uint16 else \
            a.astype(np.float32)
        if f.ndim == 2:
            q, d = quantize_q8(f)
            return name, dequantize_q8(q, d)
        return name, f.astype(np.float64)

    with ThreadPoolExecutor(max(1, threads)) as ex:
        return dict(ex.map(one, weights.items()))
