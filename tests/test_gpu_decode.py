"""Full-size decode step (32 layers, 224 GEMVs) in the launch configuration the
benchmark times: q|k|v and gate|up packed as single matrices, graph replay.

The oracle computes sampled rows of every GEMV one by one (fp64 on the fp16
dequantized rows); the normwise bound is taken over the sampled rows, which is
stricter than over the whole vector. Launching the 224 GEMVs one by one must
give the same outputs (bit-identical where the same kernel runs).
"""
import numpy as np
import pytest

import oracle
from qx_inputs import configs
from helpers import TOL

pytestmark = pytest.mark.gpu

SAMPLED_ROWS = 48


@pytest.fixture(scope="module")
def decode_steps(gpu):
    import torch
    import bench
    plan = configs.c4_plan(32)
    print("quantizing the 224 decoder matrices", flush=True)
    quant = bench.quantize_plan(plan)
    dev = torch.device("cuda:0")
    fused = bench.DecodeStep(gpu, dev, plan, quant, fused=True)
    single = bench.DecodeStep(gpu, dev, plan, quant, fused=False)
    stream = torch.cuda.Stream()
    print("replaying both launch plans", flush=True)
    bench.time_graph(fused.launch, stream, steps=2, warmup=1)
    bench.time_graph(single.launch, stream, steps=2, warmup=1)
    torch.cuda.synchronize()
    yield plan, quant, fused, single
    del fused, single
    torch.cuda.empty_cache()


def test_decode_step_sampled_rows_match_oracle(decode_steps):
    plan, quant, fused, _ = decode_steps
    rng = np.random.default_rng(0)
    worst = 0.0
    for i, (spec, (layer, t)) in enumerate(plan):
        q = quant[i]
        rows = np.sort(rng.choice(spec.n, SAMPLED_ROWS, replace=False))
        rows[0], rows[-1] = 0, spec.n - 1  # always include the first and the last row
        w16 = oracle.dequant(q.codes[rows], q.group, q.kind,
                             None if q.scales is None else q.scales[rows],
                             None if q.zeros is None else q.zeros[rows],
                             None if q.codebook is None else q.codebook[rows])
        ref = oracle.gemv(w16, configs.c4_activation(layer, t))
        y = fused.output(i).cpu().numpy()[rows]
        err = oracle.normwise_rel_err(y, ref)
        worst = max(worst, err)
        assert err <= TOL, (spec.name, err)
    print(f"worst sampled normwise rel err over 224 GEMVs: {worst:.3e}")


def test_fused_and_single_launch_plans_agree(decode_steps):
    """Launching the 224 GEMVs one by one gives the same rows as the fused plan: bit for
    bit where both plans run the same kernel on the row (o, gate, up, down), within the
    parity bound for q, k, v, whose 4096-row matrices take the two-lanes-per-chunk kernel
    alone but the one-lane-per-chunk kernel inside the 12288-row q|k|v (different
    summation order)."""
    plan, _, fused, single = decode_steps
    for i, (spec, _) in enumerate(plan):
        a = fused.output(i).cpu().numpy()
        b = single.output(i).cpu().numpy()
        if spec.name.split(".")[-1] in ("q", "k", "v"):
            assert oracle.normwise_rel_err(a, b.astype(np.float64)) <= TOL, spec.name
        else:
            assert np.array_equal(a.view(np.uint16), b.view(np.uint16)), spec.name


@pytest.mark.parametrize("m", [2, 4])
def test_batched_decode_step_sampled_rows_match_oracle(gpu, decode_steps, m):
    """The fused decode step for m sequences (qx_gemm per launch: the small-batch kernel
    or the matrix-core GEMM, as the library routes each shape), graph replay; sampled
    rows of the first two layers against the oracle for every sequence."""
    import torch
    import bench
    plan, quant, _, _ = decode_steps
    step = bench.DecodeStep(gpu, torch.device("cuda:0"), plan, quant, fused=True, batch=m)
    bench.time_graph(step.launch, torch.cuda.Stream(), steps=2, warmup=1)
    torch.cuda.synchronize()
    rng = np.random.default_rng(m)
    for i, (spec, (layer, t)) in enumerate(plan[:14]):
        q = quant[i]
        rows = np.sort(rng.choice(spec.n, SAMPLED_ROWS, replace=False))
        w16 = oracle.dequant(q.codes[rows], q.group, q.kind,
                             None if q.scales is None else q.scales[rows],
                             None if q.zeros is None else q.zeros[rows],
                             None if q.codebook is None else q.codebook[rows])
        X = configs.c4_batch_activations(layer, t, m)
        Y = step.output(i).cpu().numpy()
        for r in range(m):
            err = oracle.normwise_rel_err(Y[r][rows], oracle.gemv(w16, X[r]))
            assert err <= TOL, (spec.name, r, err)
    del step
    torch.cuda.empty_cache()
