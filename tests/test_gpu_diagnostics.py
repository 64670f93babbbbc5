"""Error diagnostics of the batch-1 GEMV on the benchmark workloads.

The parity metric is normwise: per output vector, max_i |y_i - yhat_i| / max_i
|yhat_i| <= 2e-3 (fp32 accumulation against the fp64 oracle). Next to it this
reports the elementwise relative error over the outputs that are not near zero,
max |y_i - yhat_i| / |yhat_i| over |yhat_i| >= 0.1 rms(yhat) (elementwise error is
ill-posed where yhat_i vanishes), for c1, c2, c3 and layer 0 of the decode step.
The uniform GEMV multiplies the exact levels s (q - z) (the zero point folded
once per group), while the oracle's W' rounds each level to binary16 first; the
two products differ by the sum of those roundings (2^-12 relative per weight,
random signs), which shows on outputs near zero. For uniform matrices the test
therefore also compares with the exact levels in fp64: against them the kernel
error is fp32 summation plus the fp16 output rounding. On c2 (3-bit uniform
groups with outlier activations) it also multiplies the dequantized W'
(qx_dequant, bit-exact with the oracle) in fp32 on the GPU, an exact per-weight
decode: its distance from the kernel is what the fold costs. The figures are
written to gpurun_out/diagnostics.json when that folder exists.
"""
import json
import os

import numpy as np
import pytest

import oracle
from qx_inputs import configs
from helpers import TOL, to_dev

pytestmark = pytest.mark.gpu


def elementwise_rel_err(y, ref) -> float:
    y, ref = np.asarray(y, np.float64), np.asarray(ref, np.float64)
    big = np.abs(ref) >= 0.1 * np.sqrt(np.mean(ref ** 2))
    return float(np.max(np.abs(y[big] - ref[big]) / np.abs(ref[big])))


def test_gemv_error_diagnostics(gpu):
    import torch
    qx = gpu
    cases = [(f"c{i}",) + getattr(configs, f"c{i}")() for i in (1, 2, 3)]
    for name in ("q", "o", "gate", "down"):
        spec = configs.c4_matrix(0, name)
        cases.append((f"c4 layer 0 {name}", spec, configs.c4_activation(0, configs.DECODER_X[name])))
    report = {}
    for label, spec, x in cases:
        print(f"diagnostics {label}", flush=True)
        q = spec.quantized()
        pw = qx.PackedWeight.from_quant(q)
        y = pw.gemv(to_dev(x)).cpu().numpy()
        w16 = oracle.dequant(q.codes, q.group, q.kind, q.scales, q.zeros, q.codebook)
        ref = oracle.gemv(w16, x)
        r = {"normwise": oracle.normwise_rel_err(y, ref), "elementwise_over_0.1rms": elementwise_rel_err(y, ref),
             "outputs_over_0.1rms": int(np.sum(np.abs(ref) >= 0.1 * np.sqrt(np.mean(ref ** 2)))), "n": spec.n}
        assert r["normwise"] <= TOL, (label, r)
        assert r["elementwise_over_0.1rms"] <= 1e-2, (label, r)
        if q.kind == 0:  # exact levels s (q - z) in fp64, not rounded to binary16
            j = np.arange(spec.k) // q.group
            s16 = q.scales.view(np.float16).astype(np.float64)[:, j]
            z16 = q.zeros.view(np.float16).astype(np.float64)[:, j]
            ref_levels = (s16 * (q.codes.astype(np.float64) - z16)) @ x.astype(np.float64)
            r["elementwise_vs_exact_levels"] = elementwise_rel_err(y, ref_levels)
            r["normwise_vs_exact_levels"] = oracle.normwise_rel_err(y, ref_levels)
            assert r["elementwise_vs_exact_levels"] <= TOL, (label, r)
        if label == "c2":
            W = pw.dequant(qx.QX_OUT_F16).float()
            y_exact = (W @ to_dev(x).float()).half().cpu().numpy()
            r["exact_decode_fp32_normwise"] = oracle.normwise_rel_err(y_exact, ref)
            r["exact_decode_fp32_elementwise"] = elementwise_rel_err(y_exact, ref)
            r["kernel_vs_exact_decode_normwise"] = oracle.normwise_rel_err(y, y_exact.astype(np.float64))
            assert r["kernel_vs_exact_decode_normwise"] <= 4 * 2.0 ** -11
        report[label] = r
        print(f"  {label}: " + ", ".join(f"{k} {v:.3e}" if isinstance(v, float) else f"{k} {v}"
                                        for k, v in r.items()), flush=True)
    out = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "gpurun_out")
    if os.path.isdir(out):
        with open(os.path.join(out, "diagnostics.json"), "w") as f:
            json.dump(report, f, indent=1)
