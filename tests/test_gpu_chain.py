"""GEMV chains (qx_chain_*): the products of a decode step in one persistent launch.

Each chain feeds outputs of earlier products into later ones (the dependency the
grid-wide barrier must honour). The oracle runs the same chain on the CPU from the
same weights and first input: every product in fp64 on the fp16 dequantized rows,
its output rounded to fp16 before it is used as the next input, as the library
stores it. Chains exercise the three kernel variants: the decoder mix (3-bit
codebook + 4-bit uniform, groups of 128), one format alone, and every format.
"""
import numpy as np
import pytest

import oracle
from helpers import TOL, activations, realistic_quant, to_dev

pytestmark = pytest.mark.gpu

# (bits, group, kind, n, k, index of the product whose output is x; -1 = the chain input)
DECODER = [(3, 128, 1, 4096, 4096, -1),
           (4, 128, 0, 8448, 4096, 0),
           (4, 128, 0, 4096, 8448, 1),
           (3, 128, 1, 301, 4096, 2),
           (4, 128, 0, 777, 4096, 0),     # reads an output two products back
           (4, 128, 0, 4096, 4224, -1),   # 33 chunks, one per lane of a row
           (4, 128, 0, 300, 11264, -1)]   # 88 chunks: lanes 0-23 take two
SINGLE = [(3, 64, 0, 4224, 4096, -1),
          (3, 64, 0, 4096, 4224, 0),
          (3, 64, 0, 11008, 4096, 1),
          (3, 64, 0, 515, 11008, 2)]
MIXED = [(3, 64, 0, 4096, 4096, -1),
         (4, 32, 1, 5632, 4096, 0),
         (3, 32, 1, 4096, 5632, 1),
         (4, 64, 0, 64, 4096, 2),
         (3, 128, 0, 4096, 4096, -1)]


def _build(qx, spec, seed):
    import torch
    quants, packs, xs, ys = [], [], [], []
    x0_len = {s[4] for s in spec if s[5] < 0}
    inputs = {k: to_dev(activations(k, seed=seed + k)) for k in x0_len}
    for i, (bits, g, kind, n, k, src) in enumerate(spec):
        q = realistic_quant(n, k, bits, g, kind, seed=seed * 100 + i)
        quants.append(q)
        packs.append(qx.PackedWeight.from_quant(q))
        ys.append(torch.full((n,), float("nan"), dtype=torch.float16, device="cuda"))
    for i, (bits, g, kind, n, k, src) in enumerate(spec):
        xs.append(inputs[k] if src < 0 else ys[src])
        assert xs[-1].numel() == k
    ops = [(p.desc, p.data, x, y) for p, x, y in zip(packs, xs, ys)]
    return quants, packs, xs, ys, ops, inputs


def _oracle_chain(spec, quants, inputs):
    outs = []
    for i, (bits, g, kind, n, k, src) in enumerate(spec):
        q = quants[i]
        x = inputs[k].cpu().numpy() if src < 0 else outs[src]
        w16 = oracle.dequant(q.codes, q.group, q.kind, q.scales, q.zeros, q.codebook)
        outs.append(oracle.gemv(w16, x).astype(np.float16))
    return outs


@pytest.mark.parametrize("name,spec,plan", [("decoder", DECODER, 1), ("single", SINGLE, None),
                                            ("mixed", MIXED, 0)])
def test_chain_matches_oracle_chain(gpu, name, spec, plan):
    import torch
    qx = gpu
    print(f"chain {name}: {len(spec)} products", flush=True)
    quants, packs, xs, ys, ops, inputs = _build(qx, spec, seed=len(name))
    chain = qx.GemvChain(ops)
    if plan is not None:
        assert chain.plan == plan
    else:
        assert chain.plan >= 2  # a single-format kernel
    chain.run()
    assert chain.status() == qx.QX_OK
    got = [y.cpu().numpy() for y in ys]
    ref = _oracle_chain(spec, quants, inputs)
    for i, (g, r) in enumerate(zip(got, ref)):
        assert np.all(np.isfinite(g.astype(np.float32))), i
        err = oracle.normwise_rel_err(g, r.astype(np.float64))
        assert err <= 2 * TOL, (name, i, err)
    # a second run rearms the barrier and gives the same bits
    for y in ys:
        y.fill_(float("nan"))
    chain.run()
    torch.cuda.synchronize()
    assert chain.status() == qx.QX_OK
    for i, (g, y) in enumerate(zip(got, ys)):
        assert np.array_equal(g.view(np.uint16), y.cpu().numpy().view(np.uint16)), (name, i)


def test_chain_equals_gemv_bits_where_the_kernels_share_the_order(gpu):
    """K = 128*32 uniform products use the batch-1 GEMV's per-row order (one chunk per
    lane, DPP sums over 32 lanes): the chain gives qx_gemv's bits on the same inputs."""
    import torch
    qx = gpu
    spec = [(4, 128, 0, 11008, 4096, -1), (4, 128, 0, 4096, 4096, -1), (3, 64, 0, 513, 4096, -1)]
    quants, packs, xs, ys, ops, inputs = _build(qx, spec, seed=7)
    chain = qx.GemvChain(ops)
    chain.run()
    assert chain.status() == qx.QX_OK
    for p, x, y in zip(packs, xs, ys):
        ref = torch.empty_like(y)
        qx.qx_gemv(p.desc, p.data, x, ref)
        torch.cuda.synchronize()
        assert np.array_equal(ref.cpu().numpy().view(np.uint16), y.cpu().numpy().view(np.uint16))


def test_chain_gives_up_at_a_spin_limit_and_recovers(gpu):
    """A spin limit of one poll (forced from the host) makes the barrier give up: every
    block exits and the status says so; a fresh prepare makes the chain usable again."""
    import torch
    qx = gpu
    quants, packs, xs, ys, ops, inputs = _build(qx, DECODER[:3], seed=3)
    chain = qx.GemvChain(ops)
    chain.run()
    assert chain.status() == qx.QX_OK
    good = [y.cpu().numpy().copy() for y in ys]
    chain.run(spin_limit=1)
    assert chain.status() == qx.QX_E_TIMEOUT
    chain.plan = qx.qx_chain_prepare(ops, chain.workspace)
    for y in ys:
        y.fill_(float("nan"))
    chain.run()
    torch.cuda.synchronize()
    assert chain.status() == qx.QX_OK
    for g, y in zip(good, ys):
        assert np.array_equal(g.view(np.uint16), y.cpu().numpy().view(np.uint16))


def test_chain_count_or_plan_mismatch_is_refused_by_the_kernel(gpu):
    import torch
    qx = gpu
    quants, packs, xs, ys, ops, inputs = _build(qx, SINGLE[:2], seed=5)
    chain = qx.GemvChain(ops)
    qx.qx_chain_run(chain.workspace, 1, chain.plan)   # prepared for 2
    assert chain.status() == qx.QX_E_TIMEOUT
    chain.plan = qx.qx_chain_prepare(ops, chain.workspace)
    qx.qx_chain_run(chain.workspace, 2, 1 if chain.plan != 1 else 0)
    assert chain.status() == qx.QX_E_TIMEOUT
    chain.plan = qx.qx_chain_prepare(ops, chain.workspace)
    chain.run()
    torch.cuda.synchronize()
    assert chain.status() == qx.QX_OK
