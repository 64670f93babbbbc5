"""Shared test helpers: seeded quantized inputs and device upload."""
import numpy as np

import qx_inputs as qi

TOL = 2e-3  # max |y - y_ref| / max |y_ref| per output vector, fp32 accumulate vs fp64 oracle


def random_quant(n, k, bits, group, kind, seed, scale_range=(2e-3, 2e-2)):
    """Uniformly random codes and tables (every code value and table entry exercised)."""
    rng = np.random.default_rng(seed)
    G = k // group
    codes = rng.integers(0, 2**bits, (n, k), dtype=np.uint8)
    if kind == 0:
        s = rng.uniform(*scale_range, (n, G)) * rng.choice([-1.0, 1.0], (n, G), p=[0.1, 0.9])
        z = rng.integers(0, 2**bits, (n, G)).astype(np.float16)
        return qi.QuantWeight(n, k, bits, group, kind, codes, scales=np.float16(s).view(np.uint16),
                              zeros=z.view(np.uint16))
    cb = np.sort(rng.standard_normal((n, G, 2**bits)) * scale_range[1], axis=-1).astype(np.float16)
    return qi.QuantWeight(n, k, bits, group, kind, codes, codebook=cb.view(np.uint16))


def realistic_quant(n, k, bits, group, kind, seed):
    w = qi.weights("t4" if kind == 0 else "laplace", 0.02 if kind == 0 else 0.008, seed, 0, n, k)
    return qi.quantize(w, bits, group, kind)


def activations(k, seed, m=None):
    v = qi.fill("normal", 1.0, seed, 99, 0, k if m is None else m * k)
    v = v.astype(np.float16)
    return v if m is None else v.reshape(m, k)


def to_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()
