"""GPU test of af1_linear_gemv_noalloc, the decode entry point that
allocates nothing (its workspace is a library-owned device array): through
the C ABI, its output is bit-identical to af1_linear_gemv's on the same
inputs and within the oracle bar, on consecutive calls of different sizes
(the second smaller), including plans whose column slabs use the arrival
counters."""
import numpy as np
import pytest
import torch

from paper_2609_06161_amd import af1, synth
from paper_2609_06161_amd.layer import DeviceLayer, bf16_bits_to_f64, to_device

pytestmark = pytest.mark.gpu

TOL = 5e-3


def max_row_rel_l2(y, ref):
    worst = 0.0
    for a, e in zip(np.asarray(y, np.float64), np.asarray(ref, np.float64)):
        ne = np.linalg.norm(e)
        worst = max(worst, np.linalg.norm(a - e) / ne if ne > 0 else float(np.abs(a).max()))
    return worst


def both(lin):
    """(no-alloc output, workspace output) for one layer, NaN-prefilled."""
    L = DeviceLayer.from_host(lin)
    x = to_device(lin.x)
    b = lin.x.shape[0]
    print(f"noalloc m={lin.m} n={lin.n} r={lin.r} b={b}", flush=True)
    y0 = torch.full((b, lin.m), 0x7FC0, dtype=torch.int16, device="cuda")
    af1.af1_linear_gemv_noalloc(L.desc, x, b, y0)
    torch.cuda.synchronize()
    y1 = torch.full((b, lin.m), 0x7FC0, dtype=torch.int16, device="cuda")
    ws = torch.zeros(max(256, af1.af1_gemv_workspace_bytes(lin.m, lin.n, lin.r, b)),
                     dtype=torch.uint8, device="cuda")
    af1.af1_linear_gemv(L.desc, x, b, y1, ws, ws.numel())
    torch.cuda.synchronize()
    return y0, y1


@pytest.mark.parametrize("first,second", [
    ((14336, 4096, 3136, 16), (1024, 1024, 480, 1)),
    ((4096, 14336, 3136, 16), (4096, 4096, 2016, 8)),
    ((4096, 4096, 2016, 1), (96, 2080, 160, 3)),
])
def test_noalloc_matches_workspace_entry_point(oracle, first, second):
    for k, (m, n, r, b) in enumerate((first, second)):
        lin = synth.make_linear(8100 + 7 * k + b, m, n, r, b)
        assert af1.af1_gemv_workspace_bytes(m, n, r, b) <= af1.AF1_GEMV_SCRATCH_BYTES
        y0, y1 = both(lin)
        assert torch.equal(y0, y1), (m, n, r, b)
        ref = oracle.forward(m, n, r, lin.Bu, lin.Bv, lin.s_out, lin.s_mid, lin.s_in, lin.x)
        assert max_row_rel_l2(bf16_bits_to_f64(y0), ref) <= TOL


def test_noalloc_repeated_calls_of_a_counter_plan(oracle):
    """A batch whose stages hand partial sums between workgroups through the
    arrival counters, five calls in a row interleaved with a smaller layer:
    every call gives the same bits."""
    big = synth.make_linear(8200, 14336, 4096, 3136, 16)
    small = synth.make_linear(8201, 1024, 4096, 800, 2)
    Lb, Ls = DeviceLayer.from_host(big), DeviceLayer.from_host(small)
    xb, xs = to_device(big.x), to_device(small.x)
    ref_b = ref_s = None
    for i in range(5):
        yb = torch.full((16, 14336), 0x7FC0, dtype=torch.int16, device="cuda")
        ys = torch.full((2, 1024), 0x7FC0, dtype=torch.int16, device="cuda")
        af1.af1_linear_gemv_noalloc(Lb.desc, xb, 16, yb)
        af1.af1_linear_gemv_noalloc(Ls.desc, xs, 2, ys)
        torch.cuda.synchronize()
        if i == 0:
            ref_b, ref_s = yb.clone(), ys.clone()
            ob = oracle.forward(big.m, big.n, big.r, big.Bu, big.Bv, big.s_out, big.s_mid,
                                big.s_in, big.x)
            assert max_row_rel_l2(bf16_bits_to_f64(yb), ob) <= TOL
        assert torch.equal(yb, ref_b) and torch.equal(ys, ref_s), i


def test_noalloc_rejects_shapes_beyond_the_scratch():
    m, n, r, b = 28672, 8192, 6336, 16
    assert af1.af1_gemv_workspace_bytes(m, n, r, b) > af1.AF1_GEMV_SCRATCH_BYTES
    z = lambda *shape, dt=torch.int32: torch.zeros(shape, dtype=dt, device="cuda")
    arrays = (z(m, r // 32), z(r, n // 32), z(m, dt=torch.int16), z(r, dt=torch.int16),
              z(n, dt=torch.int16))
    desc = af1.make_layer(m, n, r, *arrays)
    x = torch.zeros((b, n), dtype=torch.int16, device="cuda")
    y = torch.zeros((b, m), dtype=torch.int16, device="cuda")
    st = af1.af1_linear_gemv_noalloc(desc, x, b, y, check=False)
    assert st == af1.AF1_ERR_WORKSPACE
