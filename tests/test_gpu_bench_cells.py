"""One GPU parity test per cell that bench.py publishes, at that cell's
shape, batch / token count and entry point, against the fp64 oracle.

The decode cells are parametrized from bench.py's own table, so a new cell
cannot appear without a test.  Where the oracle would take minutes (long
prefill calls) it checks a seeded sample of tokens, the first and last
included; every other cell is checked element-wise in full."""
import numpy as np
import pytest
import torch

import bench
from paper_2609_06161_amd import af1, synth
from paper_2609_06161_amd.layer import DeviceLayer, bf16_bits_to_f64, gemv_multi, to_device

pytestmark = pytest.mark.gpu

TOL = 5e-3


def max_row_rel_l2(y, ref):
    worst = 0.0
    for a, e in zip(np.asarray(y, np.float64), np.asarray(ref, np.float64)):
        ne = np.linalg.norm(e)
        worst = max(worst, np.linalg.norm(a - e) / ne if ne > 0 else float(np.abs(a).max()))
    return worst


def elementwise_ok(y, ref, rel=2 ** -7, abs_rms=1e-3):
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.sqrt(np.mean(ref ** 2, axis=1, keepdims=True))
    bad = ~(np.abs(y - ref) <= rel * np.abs(ref) + abs_rms * scale)
    return not bad.any(), np.argwhere(bad)[:5]


def oracle_y(oracle, lin, x):
    return oracle.forward(lin.m, lin.n, lin.r, lin.Bu, lin.Bv, lin.s_out, lin.s_mid, lin.s_in, x)


@pytest.mark.parametrize("name,b", bench.DECODE_TABLE + [("attn4096", 1)],
                         ids=[f"{n}_b{b}" for n, b in bench.DECODE_TABLE + [("attn4096", 1)]])
def test_decode_table_cell(oracle, name, b):
    """Every decode_table cell (and the headline 4096^2 b=1) through
    af1_linear_gemv itself, NaN-prefilled output, element-wise."""
    m, n, r = bench.shape_of(name)
    lin = synth.make_linear(2000 + b, m, n, r, b, outliers=(name != "sq1024"))
    print(f"decode cell {name} b={b}: {m}x{n} r={r}", flush=True)
    L = DeviceLayer.from_host(lin)
    y = torch.full((b, m), 0x7FC0, dtype=torch.int16, device="cuda")
    L.gemv(to_device(lin.x), y=y)
    torch.cuda.synchronize()
    got, ref = bf16_bits_to_f64(y), oracle_y(oracle, lin, lin.x)
    ok, where = elementwise_ok(got, ref)
    assert max_row_rel_l2(got, ref) <= TOL and ok, where


@pytest.mark.parametrize("name", ["attn4096", "sq8192"])
@pytest.mark.parametrize("T", [32, 128, 512])
def test_gemm_few_tokens_cell(oracle, name, T):
    """gemm.few_tokens: the chunked-prefill calls at 4096^2 and 8192^2 (split
    K or 64-token tiles).  All tokens at 4096^2 and for T <= 128 at 8192^2,
    a seeded sample of 48 tokens otherwise."""
    m, n, r = bench.shape_of(name)
    lin = synth.make_linear(57, m, n, r, T)
    print(f"few-token cell {name} T={T}", flush=True)
    L = DeviceLayer.from_host(lin)
    y = torch.full((T, m), 0x7FC0, dtype=torch.int16, device="cuda")
    L.gemm(to_device(lin.x), y=y)
    torch.cuda.synchronize()
    got = bf16_bits_to_f64(y)
    idx = np.arange(T)
    if name == "sq8192" and T > 128:
        idx = np.sort(np.random.default_rng(T).choice(np.arange(1, T - 1), 46, replace=False))
        idx = np.concatenate([[0], idx, [T - 1]])
    ref = oracle_y(oracle, lin, lin.x[idx])
    ok, where = elementwise_ok(got[idx], ref, rel=2 ** -6, abs_rms=6e-3)
    assert max_row_rel_l2(got[idx], ref) <= TOL and ok, where


def test_gemm_25bpw_2048_tokens_cell(oracle):
    """The 2.5-BPW GEMM cell (4096^2, the paper's rank rule: r = 5120) at
    2048 tokens: 16 sampled tokens, first and last included."""
    m, n, r = bench.paper_25bpw_shape()
    assert r == 5120
    T = 2048
    lin = synth.make_linear(56, m, n, r, T)
    L = DeviceLayer.from_host(lin)
    y = L.gemm(to_device(lin.x))
    torch.cuda.synchronize()
    idx = np.sort(np.random.default_rng(5).choice(np.arange(1, T - 1), 14, replace=False))
    idx = np.concatenate([[0], idx, [T - 1]])
    got = bf16_bits_to_f64(y)[idx]
    ref = oracle_y(oracle, lin, lin.x[idx])
    ok, where = elementwise_ok(got, ref, rel=2 ** -6, abs_rms=6e-3)
    assert max_row_rel_l2(got, ref) <= TOL and ok, where


@pytest.mark.parametrize("layer", [0, 31])
def test_stack_fused_projection_cells(oracle, layer):
    """decode_stack_8b's fused schedule: q/k/v and gate/up of one decoder
    layer (the stack's heterogeneous ranks) through af1_linear_gemv_multi,
    each output element-wise against the oracle."""
    entries = synth.draw_stack_ranks(77, 32, bench.STACK_LINEARS, af1.af1_storage_bits)
    ent = entries[7 * layer: 7 * layer + 7]
    for group in (ent[0:3], ent[4:6]):
        n = group[0][2]
        x = synth.make_activations(60 + n % 97, 1, n)
        lins = []
        for i, (name, m, nn, r0, r) in enumerate(group):
            lin = synth.make_linear(5000 + 7 * layer + i, m, nn, r, 1)
            lin.x = x
            lins.append(lin)
        layers = [DeviceLayer.from_host(lin) for lin in lins]
        ys = [torch.full((1, L.m), 0x7FC0, dtype=torch.int16, device="cuda") for L in layers]
        gemv_multi(layers, to_device(x), ys=ys)
        torch.cuda.synchronize()
        for lin, y in zip(lins, ys):
            ok, where = elementwise_ok(bf16_bits_to_f64(y), oracle_y(oracle, lin, x))
            assert ok, (layer, lin.m, lin.n, lin.r, where)


@pytest.mark.parametrize("dtype,code", [("f32", af1.AF1_SRC_F32), ("bf16", af1.AF1_SRC_BF16),
                                        ("i8", af1.AF1_SRC_I8)])
def test_pack_16384_cell(oracle, dtype, code):
    """pack_16384x16384: the full matrix packed on the device in the bench's
    launch; 65 sampled rows (the last included) bit-exact against the
    oracle's packing of the same rows."""
    rows = cols = 16384
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "i8": torch.int8}[dtype]
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    src = torch.randint(-100, 100, (rows, cols), device="cuda", generator=g).to(tdt)
    src[7, :32] = -0.0 if dtype != "i8" else 0     # signed zeros in one word
    dst = torch.empty(rows * cols // 32, dtype=torch.int32, device="cuda")
    af1.af1_pack(src, code, rows, cols, dst)
    torch.cuda.synchronize()
    pick = np.sort(np.random.default_rng(4).choice(rows - 1, 64, replace=False))
    pick = np.concatenate([pick, [rows - 1]])
    pick = np.union1d(pick, [7])
    host = src[torch.from_numpy(pick).cuda()].cpu()
    if dtype == "bf16":
        hsrc = host.view(torch.int16).numpy().view(np.uint16)
    else:
        hsrc = host.numpy()
    want = oracle.pack(np.ascontiguousarray(hsrc), bf16_bits=(dtype == "bf16"))
    got = dst.view(rows, cols // 32)[torch.from_numpy(pick).cuda()].cpu().numpy().view(np.uint32)
    assert np.array_equal(got, want)
