"""Error measures of the GPU parity tests (test infrastructure, numpy only).

row_errors backs the norm-wise relative error per parameter block with a
measure that a localized defect cannot hide in: the largest relative error
of a row (rows far below the block's typical norm measured against that
typical norm)."""

import numpy as np


def row_errors(a, b, rows):
    """Largest relative row error of a against the reference b, both cut
    into `rows` rows: |a_r - b_r| / max(|b_r|, rms), where rms is the
    root-mean-square row norm of b (the floor keeps rows far smaller than
    the rest, such as the W_s rows of classes no frame is labelled with,
    from dividing rounding noise by almost nothing).  A norm-wise relative
    error over a whole block moves by only about 1/sqrt(rows) when one row
    is wrong (a gate row of one unit, a frame, an edge tile of a product);
    this measure moves by about 1."""
    a = np.asarray(a, dtype=np.float64).reshape(rows, -1)
    b = np.asarray(b, dtype=np.float64).reshape(rows, -1)
    nb = np.linalg.norm(b, axis=1)
    rms = np.linalg.norm(b) / np.sqrt(rows)
    return float(np.max(np.linalg.norm(a - b, axis=1) / np.maximum(nb, max(rms, 1e-30))))


def block_row_errors(g_gpu, g_ref, dims, chunk=16, param_layout=None):
    """row_errors per parameter block: matrices by their rows, vectors in
    rows of `chunk` elements (zero-padded).  param_layout: the oracle's
    layout function (dims -> {block: (offset, shape)}, ...)."""
    blocks, _ = param_layout(dims)
    out = {}
    for key, (off, shape) in blocks.items():
        n = int(np.prod(shape))
        a, b = g_gpu[off:off + n], g_ref[off:off + n]
        if len(shape) >= 2:
            out[key] = row_errors(a, b, shape[0])
        else:
            pad = (-n) % chunk
            out[key] = row_errors(np.pad(a, (0, pad)), np.pad(b, (0, pad)), (n + pad) // chunk)
    return out
