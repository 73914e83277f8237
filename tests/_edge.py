"""Inputs built from the HIF4 quantizer's special cases (test data only).

Seven kinds of 64-element group, chosen to reach every branch of a group
quantizer: all zeros (base byte 0), a single non-zero element, exact ties of
the element rounding (base 1, step 1/4: 0.125, 0.375 and 0.625 sit halfway
between grid points), fp16 subnormals, large magnitudes, nested E2/E3 blocks
(one large element among small ones), and negative zeros among random
values."""
import numpy as np

KINDS = 7


def _group(kind, rng, large):
    x = rng.standard_normal(64).astype(np.float16)
    if kind == 0:
        x[:] = 0
    elif kind == 1:
        x[:] = 0
        x[rng.integers(64)] = -3.0
    elif kind == 2:
        x[:] = np.tile(np.array([1.75, 0.125, -0.375, 0.625], np.float16), 16)
    elif kind == 3:
        x[:] = (rng.integers(-40, 41, 64) * 2.0 ** -24).astype(np.float16)
    elif kind == 4:
        x[:] = (rng.standard_normal(64) * large).astype(np.float16)
    elif kind == 5:
        x[:] = (rng.standard_normal(64) * 0.01).astype(np.float16)
        x[3] = 1.0
        x[12:16] = 0.3
    else:
        x[::2] = np.float16(-0.0)
    return x


def edge_rows(x, seed, large=150.0):
    """Overwrites every 64-channel group of x [..., D] (fp16) in place with
    one of the special kinds, cycling through them."""
    rng = np.random.default_rng(seed)
    g = x.reshape(-1, 64)
    for i in range(g.shape[0]):
        g[i] = _group(i % KINDS, rng, large)
    return x


def edge_tokens(v, cu, seed, large=150.0):
    """Overwrites the 64-token groups of each (kv head, channel) column of
    v [T, H, D] (fp16), aligned to each sequence's first token (a partial last
    group takes the head of its pattern), in place."""
    rng = np.random.default_rng(seed)
    i = 0
    for b in range(len(cu) - 1):
        for t0 in range(cu[b], cu[b + 1], 64):
            n = min(64, cu[b + 1] - t0)
            for hh in range(v.shape[1]):
                for c in range(v.shape[2]):
                    v[t0:t0 + n, hh, c] = _group(i % KINDS, rng, large)[:n]
                    i += 1
    return v
