"""Decode plans whose staged input fills the LDS (regression).

At batch 7 a column slab of the widest plan took exactly the compute unit's
160 KiB of dynamic LDS (161,392 bytes of staging divide evenly by 7 into
160-word slabs), and the stage kernels' own __shared__ words came on top, so
the launch asked for more LDS than a compute unit has.  The planner now
budgets the dynamic LDS below the unit's LDS by a reserve for those words,
and every stage, multi-layer and stream launch checks static + dynamic LDS
before it is made.  These cases run b=7 with rows of at least 160 words in
either product, through each entry point that plans such stages, against
the fp64 oracle."""
import numpy as np
import pytest
import torch

from paper_2609_06161_amd import af1, synth
from paper_2609_06161_amd.layer import (DeviceLayer, LayerStream, bf16_bits_to_f64, gemv_multi,
                                        to_device)

pytestmark = pytest.mark.gpu

TOL = 5e-3


def check(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    worst = 0.0
    for a, e in zip(got, ref):
        ne = np.linalg.norm(e)
        worst = max(worst, np.linalg.norm(a - e) / ne if ne > 0 else float(np.abs(a).max()))
    scale = np.sqrt(np.mean(ref ** 2, axis=1, keepdims=True))
    bad = ~(np.abs(got - ref) <= 2 ** -7 * np.abs(ref) + 1e-3 * scale)
    assert worst <= TOL and not bad.any(), (worst, np.argwhere(bad)[:5])


def oracle_y(oracle, lin, x):
    return oracle.forward(lin.m, lin.n, lin.r, lin.Bu, lin.Bv, lin.s_out, lin.s_mid, lin.s_in, x)


@pytest.mark.parametrize("m,n,r", [(2208, 7904, 160),    # first product: 247-word rows
                                   (1024, 512, 5152),    # second product: 161-word rows
                                   (544, 16384, 5120)])  # both
def test_gemv_b7_full_width_slabs(oracle, m, n, r):
    b = 7
    lin = synth.make_linear(7700 + m, m, n, r, b)
    print(f"lds limit gemv m={m} n={n} r={r} b={b}", flush=True)
    L = DeviceLayer.from_host(lin)
    y = torch.full((b, m), 0x7FC0, dtype=torch.int16, device="cuda")
    L.gemv(to_device(lin.x), y=y)
    torch.cuda.synchronize()
    check(bf16_bits_to_f64(y), oracle_y(oracle, lin, lin.x))


def test_gemv_noalloc_b7_full_width_slabs(oracle):
    m, n, r, b = 2208, 7904, 160, 7
    lin = synth.make_linear(7710, m, n, r, b)
    print(f"lds limit noalloc m={m} n={n} r={r} b={b}", flush=True)
    L = DeviceLayer.from_host(lin)
    y = torch.full((b, m), 0x7FC0, dtype=torch.int16, device="cuda")
    af1.af1_linear_gemv_noalloc(L.desc, to_device(lin.x), b, y)
    torch.cuda.synchronize()
    check(bf16_bits_to_f64(y), oracle_y(oracle, lin, lin.x))


def test_gemv_multi_b7_full_width_slabs(oracle):
    n, b = 11008, 7
    x = synth.make_activations(7720, b, n)
    lins = []
    for i, (m, r) in enumerate([(5472, 224), (2720, 64), (384, 384)]):
        lin = synth.make_linear(7721 + i, m, n, r, b)
        lin.x = x
        lins.append(lin)
    print(f"lds limit gemv_multi n={n} b={b}", flush=True)
    layers = [DeviceLayer.from_host(lin) for lin in lins]
    ys = gemv_multi(layers, to_device(x))
    torch.cuda.synchronize()
    for lin, y in zip(lins, ys):
        check(bf16_bits_to_f64(y), oracle_y(oracle, lin, x))


def test_stream_b7_full_width_rows(oracle):
    b = 7
    lin0 = synth.make_linear(7730, 1536, 9216, 320, b)     # 288-word rows in the first product
    lin1 = synth.make_linear(7731, 704, 1536, 5376, b)     # 168-word rows in the second
    print(f"lds limit stream b={b}", flush=True)
    L0, L1 = DeviceLayer.from_host(lin0), DeviceLayer.from_host(lin1)
    x0 = to_device(lin0.x)
    y0 = torch.full((b, 1536), 0x7FC0, dtype=torch.int16, device="cuda")
    y1 = torch.full((b, 704), 0x7FC0, dtype=torch.int16, device="cuda")
    S = LayerStream([(L0, x0, y0, False), (L1, y0, y1, True)], b)
    S.run()
    torch.cuda.synchronize()
    assert S.error_word() == 0
    check(bf16_bits_to_f64(y0), oracle_y(oracle, lin0, lin0.x))
    x1 = y0.detach().cpu().numpy().view(np.uint16)
    check(bf16_bits_to_f64(y1), oracle_y(oracle, lin1, x1))
