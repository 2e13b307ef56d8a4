"""GPU parity: the HIP path through the C ABI against the fp64 CPU oracle on
the same seeded inputs.

Bars: packing and unpacking bit-exact; forward outputs within relative L2
5e-3 per batch row / token (max over rows), with y == 0 exactly when the
oracle's row is exactly zero."""
import numpy as np
import pytest
import torch

from paper_2609_06161_amd import af1, synth
from paper_2609_06161_amd.layer import DeviceLayer, bf16_bits_to_f64, gemv_multi, to_device

pytestmark = pytest.mark.gpu

TOL = 5e-3


def max_row_rel_l2(y, ref):
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    worst = 0.0
    for a, e in zip(y, ref):
        ne = np.linalg.norm(e)
        if ne == 0.0:
            assert np.all(a == 0.0)
            continue
        worst = max(worst, np.linalg.norm(a - e) / ne)
    return worst


def oracle_y(oracle, lin, x=None):
    x = lin.x if x is None else x
    return oracle.forward(lin.m, lin.n, lin.r, lin.Bu, lin.Bv, lin.s_out, lin.s_mid, lin.s_in, x)


def gpu_gemv(lin, x=None):
    x = lin.x if x is None else x
    print(f"gemv m={lin.m} n={lin.n} r={lin.r} b={x.shape[0]}", flush=True)
    L = DeviceLayer.from_host(lin)
    y = L.gemv(to_device(x))
    torch.cuda.synchronize()
    return bf16_bits_to_f64(y)


def gpu_gemm(lin, x=None):
    x = lin.x if x is None else x
    print(f"gemm m={lin.m} n={lin.n} r={lin.r} T={x.shape[0]}", flush=True)
    L = DeviceLayer.from_host(lin)
    y = L.gemm(to_device(x))
    torch.cuda.synchronize()
    return bf16_bits_to_f64(y)


# --------------------------------------------------------------------------
# packing
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dtype,code", [("f32", 0), ("bf16", 1), ("f16", 2), ("i8", 3)])
@pytest.mark.parametrize("rows,cols", [(1, 32), (37, 96), (300, 4096)])
def test_pack_bit_exact(oracle, dtype, code, rows, cols):
    src = synth.random_sign_source(rows * 7 + cols, rows, cols, dtype)
    want = oracle.pack(src, bf16_bits=(dtype == "bf16"))
    host = src if dtype != "f16" else src.view(np.uint16)
    d_src = to_device(host)
    d_dst = torch.empty((rows, cols // 32), dtype=torch.int32, device="cuda")
    af1.af1_pack(d_src, code, rows, cols, d_dst)
    torch.cuda.synchronize()
    got = d_dst.cpu().numpy().view(np.uint32)
    assert np.array_equal(got, want)


def test_pack_zero_rows_is_noop():
    src = torch.zeros(32, dtype=torch.float32, device="cuda")
    d = torch.full((4,), 7, dtype=torch.int32, device="cuda")
    af1.af1_pack(src, 0, 0, 32, d)
    torch.cuda.synchronize()
    assert d.cpu().tolist() == [7, 7, 7, 7]


@pytest.mark.parametrize("rows,cols", [(1, 32), (45, 160), (2016, 4096)])
def test_unpack_bit_exact(oracle, rows, cols):
    words = synth.random_words(np.random.default_rng(rows), rows, cols)
    d_out = torch.empty((rows, cols), dtype=torch.int8, device="cuda")
    af1.af1_unpack(to_device(words), rows, cols, d_out)
    torch.cuda.synchronize()
    assert np.array_equal(d_out.cpu().numpy(), oracle.unpack(words, cols))


# --------------------------------------------------------------------------
# GEMV (decode)
# --------------------------------------------------------------------------

SMALL = [(32, 32, 32), (96, 2080, 160), (544, 4128, 96), (1056, 64, 2080)]


@pytest.mark.parametrize("m,n,r", SMALL)
@pytest.mark.parametrize("b", [1, 2, 3, 5, 8, 16])
def test_gemv_small_shapes(oracle, m, n, r, b):
    lin = synth.make_linear(1000 + m + n + r + b, m, n, r, b)
    assert max_row_rel_l2(gpu_gemv(lin), oracle_y(oracle, lin)) <= TOL


@pytest.mark.parametrize("name,b", [("sq1024", 1), ("attn4096", 1), ("attn4096", 8),
                                    ("kv1024x4096", 1), ("mlp_up14336x4096", 1),
                                    ("mlp_up14336x4096", 4), ("mlp_down4096x14336", 1),
                                    ("mlp_down4096x14336", 16)])
def test_gemv_named_shapes(oracle, name, b):
    m, n, r = synth.SHAPES[name]
    lin = synth.make_linear(7, m, n, r, b, outliers=(name != "sq1024"))
    err = max_row_rel_l2(gpu_gemv(lin), oracle_y(oracle, lin))
    print(f"{name} b={b} max row rel-L2 {err:.3e}")
    assert err <= TOL


def elementwise_ok(y, ref, rel=2 ** -7, abs_rms=1e-3):
    """Every element within bf16-level error of its reference, relative to
    the element and to its row's rms (abs_rms), so that a single wrong
    element fails: dropping one 32-column word of a 2016-term sum moves an
    element by about 0.13 rms."""
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.sqrt(np.mean(ref ** 2, axis=1, keepdims=True))
    bad = np.abs(y - ref) > rel * np.abs(ref) + abs_rms * scale
    return not bad.any(), np.argwhere(bad)[:5]


@pytest.mark.parametrize("m,n,r,b", [(4096, 4096, 2016, 1), (1056, 2080, 4064, 3),
                                     (96, 1056, 96, 1)])
def test_gemv_elementwise_including_last_rows(oracle, m, n, r, b):
    """Odd word counts (r/32 = 63, 127; n/32 = 65, 33): the last row's last
    word is read next to the end of its buffer."""
    lin = synth.make_linear(77 + r, m, n, r, b)
    ok, where = elementwise_ok(gpu_gemv(lin), oracle_y(oracle, lin))
    assert ok, where


@pytest.mark.parametrize("m,n,r,T", [(4096, 4096, 2016, 40), (1056, 2080, 4064, 33)])
def test_gemm_elementwise_including_last_rows(oracle, m, n, r, T):
    lin = synth.make_linear(91 + r, m, n, r, T)
    # the intermediate is rounded once to fp16 (2^-12 relative, summed over r
    # terms: about 2.4e-4 rms of absolute error, with rare 4-5 sigma tails)
    ok, where = elementwise_ok(gpu_gemm(lin), oracle_y(oracle, lin), rel=2 ** -6, abs_rms=6e-3)
    assert ok, where


def test_gemv_zero_input_gives_exact_zero():
    lin = synth.make_linear(3, 1024, 1024, 480, 2)
    y = gpu_gemv(lin, np.zeros_like(lin.x))
    assert np.all(y == 0.0)


def test_gemv_sign_gauge_bit_identical():
    lin = synth.make_linear(5, 4096, 4096, 2016, 2)
    y0 = gpu_gemv(lin)
    k = 1234
    lin.Bu = lin.Bu.copy()
    lin.Bv = lin.Bv.copy()
    lin.Bu[:, k // 32] ^= np.uint32(1 << (k % 32))
    lin.Bv[k, :] ^= np.uint32(0xFFFFFFFF)
    assert np.array_equal(gpu_gemv(lin), y0)


@pytest.mark.parametrize("m,n,r,b", [(544, 4128, 96, 5), (4096, 4096, 2016, 16),
                                     (1024, 4096, 800, 8)])
def test_gemv_column_slabs_reuse_workspace(oracle, m, n, r, b):
    """Shapes whose columns split over several workgroups: one zero-filled
    workspace serves repeated calls and a different shape afterwards (the
    arrival counters are left at zero by every call)."""
    lin = synth.make_linear(31 + b, m, n, r, b)
    L = DeviceLayer.from_host(lin)
    x = to_device(lin.x)
    ws = torch.zeros(1 << 24, dtype=torch.uint8, device="cuda")
    ref = oracle_y(oracle, lin)
    for _ in range(3):
        # NaN-filled output: a row the kernel failed to write cannot pass
        y = torch.full((b, m), 0x7FC0, dtype=torch.int16, device="cuda")
        L.gemv(x, y=y, ws=ws)
        torch.cuda.synchronize()
        assert max_row_rel_l2(bf16_bits_to_f64(y), ref) <= TOL
    small = synth.make_linear(5, 96, 2080, 160, 3)
    ys = torch.full((3, 96), 0x7FC0, dtype=torch.int16, device="cuda")
    DeviceLayer.from_host(small).gemv(to_device(small.x), y=ys, ws=ws)
    torch.cuda.synchronize()
    assert max_row_rel_l2(bf16_bits_to_f64(ys), oracle_y(oracle, small)) <= TOL


def test_gemv_workspace_shared_by_shapes_and_batches(oracle):
    """One zero-filled workspace, 3 x 20 calls alternating shapes whose
    stages use different column plans (a last-slab reduction at b=16, split
    partial sums at b=1, single slabs at 14336x4096): the arrival counters
    sit at fixed offsets and return to zero after every call, so every call
    gives the same bits as on a fresh workspace."""
    cases = []
    for name, b in (("attn4096", 16), ("attn4096", 1), ("mlp_up14336x4096", 2)):
        m, n, r = synth.SHAPES[name]
        lin = synth.make_linear(500 + b, m, n, r, b)
        L = DeviceLayer.from_host(lin)
        x = to_device(lin.x)
        ref = L.gemv(x)
        torch.cuda.synchronize()
        assert max_row_rel_l2(bf16_bits_to_f64(ref), oracle_y(oracle, lin)) <= TOL
        cases.append((L, x, b, ref))
    ws = torch.zeros(max(af1.af1_gemv_workspace_bytes(L.m, L.n, L.r, b) for L, _, b, _ in cases),
                     dtype=torch.uint8, device="cuda")
    for i in range(20):
        for L, x, b, ref in cases:
            y = torch.full((b, L.m), 0x7FC0, dtype=torch.int16, device="cuda")
            L.gemv(x, y=y, ws=ws)
            torch.cuda.synchronize()
            assert torch.equal(y, ref), (i, L.m, L.n, L.r, b)


@pytest.mark.parametrize("m,n,r,b", [(14368, 4096, 3136, 4), (4128, 14336, 3136, 8),
                                     (1056, 2080, 4064, 16), (14368, 4096, 3136, 16)])
def test_gemv_multi_tile_workgroups_ragged(oracle, m, n, r, b):
    """Batches whose plans give workgroups several 16-row tiles (2 to 8)
    sharing one staged input, with row counts that leave the last workgroup
    partly empty (m/16 = 898 and 258 tiles), every element checked, y
    prefilled with NaN."""
    lin = synth.make_linear(900 + b, m, n, r, b)
    print(f"multi-tile m={m} n={n} r={r} b={b}", flush=True)
    L = DeviceLayer.from_host(lin)
    y = torch.full((b, m), 0x7FC0, dtype=torch.int16, device="cuda")
    L.gemv(to_device(lin.x), y=y)
    torch.cuda.synchronize()
    ok, where = elementwise_ok(bf16_bits_to_f64(y), oracle_y(oracle, lin))
    assert ok, where


@pytest.mark.parametrize("m,n,r,b", [(1024, 1024, 1280, 1), (4096, 4096, 5120, 1),
                                     (4096, 4096, 5120, 8)])
def test_gemv_rank_above_dimensions(oracle, m, n, r, b):
    """The paper's 2.5-bit setting has r > min(m, n) (Table 1): the same
    kernels, with the second product the wider one."""
    lin = synth.make_linear(40 + b, m, n, r, b)
    assert max_row_rel_l2(gpu_gemv(lin), oracle_y(oracle, lin)) <= TOL


def test_gemm_rank_above_dimensions(oracle):
    lin = synth.make_linear(41, 4096, 4096, 5120, 96)
    assert max_row_rel_l2(gpu_gemm(lin), oracle_y(oracle, lin)) <= TOL


@pytest.mark.parametrize("layer", [0, 31])
def test_gemv_stack_linears_heterogeneous_ranks(oracle, layer):
    """The decoder-stack workload's ranks (drawn +-25% around the budget rank
    with the stack at <= 1.0 BPW): every linear of one layer at b=1, each
    checked element-wise."""
    linears = [("q", 4096, 4096, 2016), ("k", 1024, 4096, 800), ("v", 1024, 4096, 800),
               ("o", 4096, 4096, 2016), ("gate", 14336, 4096, 3136),
               ("up", 14336, 4096, 3136), ("down", 4096, 14336, 3136)]
    entries = synth.draw_stack_ranks(77, 32, linears, af1.af1_storage_bits)
    for i, (name, m, n, r0, r) in enumerate(entries[7 * layer: 7 * layer + 7]):
        lin = synth.make_linear(7000 + 7 * layer + i, m, n, r, 1)
        print(f"stack layer {layer} {name}: {m}x{n} r={r}", flush=True)
        ok, where = elementwise_ok(gpu_gemv(lin), oracle_y(oracle, lin))
        assert ok, (name, r, where)


def test_gemv_subnormal_scales(oracle):
    """fp16 subnormal scales (no flush to zero anywhere on the decode path):
    s_in, s_mid, s_out drawn from the subnormal range, x large enough that
    y stays normal in bf16."""
    m, n, r, b = 1024, 2048, 512, 3
    lin = synth.make_linear(13, m, n, r, b)
    rng = np.random.default_rng(5)
    for name, k in (("s_in", n), ("s_mid", r), ("s_out", m)):
        setattr(lin, name, rng.integers(1, 0x0400, size=k, dtype=np.uint16))
    lin.x = synth.f32_to_bf16_bits(rng.standard_normal((b, n)).astype(np.float32) * 1e4)
    ref = oracle_y(oracle, lin)
    assert np.all(np.abs(ref[np.abs(ref) > 0]) > 1e-30)
    assert max_row_rel_l2(gpu_gemv(lin), ref) <= TOL


def test_gemm_max_tokens(oracle):
    """The largest token count the entry point accepts (2^20) on a small
    layer: sampled tokens, the last one included, against the oracle."""
    m, n, r, T = 64, 96, 64, 1 << 20
    lin = synth.make_linear(17, m, n, r, T)
    y = gpu_gemm(lin)
    idx = np.sort(np.random.default_rng(1).choice(T, 64, replace=False))
    idx[-1] = T - 1
    assert max_row_rel_l2(y[idx], oracle_y(oracle, lin, lin.x[idx])) <= TOL


QKV = [(4096, 4096, 2016), (1024, 4096, 800), (1024, 4096, 800)]
GATE_UP = [(14336, 4096, 3136), (14336, 4096, 3136)]


@pytest.mark.parametrize("shapes,b", [(QKV, 1), (QKV, 4), (QKV, 8), (GATE_UP, 1),
                                      (GATE_UP, 16), (QKV[:1], 1),
                                      ([(96, 2080, 160), (544, 2080, 96), (1056, 2080, 4064),
                                        (32, 2080, 32)], 3)])
def test_gemv_multi_matches_oracle(oracle, shapes, b):
    """Several layers reading one x in one call (two launches for q/k/v and
    gate/up; at b=16 gate/up need last-slab reductions and run one after
    the other): every output element against the oracle, outputs prefilled
    with NaN."""
    x = synth.make_activations(33 + b, b, shapes[0][1])
    lins = [synth.make_linear(600 + i, m, n, r, b) for i, (m, n, r) in enumerate(shapes)]
    for lin in lins:
        lin.x = x
    print(f"multi {[s[:3] for s in shapes]} b={b}", flush=True)
    layers = [DeviceLayer.from_host(lin) for lin in lins]
    ys = [torch.full((b, L.m), 0x7FC0, dtype=torch.int16, device="cuda") for L in layers]
    gemv_multi(layers, to_device(x), ys=ys)
    torch.cuda.synchronize()
    for lin, y in zip(lins, ys):
        ok, where = elementwise_ok(bf16_bits_to_f64(y), oracle_y(oracle, lin))
        assert ok, (lin.m, lin.n, lin.r, where)


def test_gemv_multi_workspace_reuse_with_single_calls(oracle):
    """One workspace serving multi calls and single-layer calls in turn."""
    b = 2
    x = synth.make_activations(70, b, 4096)
    lins = [synth.make_linear(700 + i, m, n, r, b) for i, (m, n, r) in enumerate(QKV)]
    for lin in lins:
        lin.x = x
    layers = [DeviceLayer.from_host(lin) for lin in lins]
    xd = to_device(x)
    descs = [L.desc for L in layers]
    ws = torch.zeros(af1.af1_gemv_multi_workspace_bytes(descs, b), dtype=torch.uint8,
                     device="cuda")
    refs = [oracle_y(oracle, lin) for lin in lins]
    for _ in range(3):
        ys = gemv_multi(layers, xd, ws=ws)
        single = layers[1].gemv(xd, ws=ws)
        torch.cuda.synchronize()
        for y, ref in zip(ys, refs):
            assert max_row_rel_l2(bf16_bits_to_f64(y), ref) <= TOL
        assert max_row_rel_l2(bf16_bits_to_f64(single), refs[1]) <= TOL


def test_gemv_deterministic():
    lin = synth.make_linear(9, 4096, 4096, 2016, 4)
    assert np.array_equal(gpu_gemv(lin), gpu_gemv(lin))


def test_gemv_hadamard_identity(oracle):
    import scipy.linalg
    n = 1024
    H = scipy.linalg.hadamard(n)
    w = oracle.pack(np.where(H < 0, -1, 1).astype(np.int8))
    rng = np.random.default_rng(2)
    lin = synth.Linear(n, n, n, w, w, synth.lognormal_f16(rng, n),
                       np.full(n, 1.0 / n, np.float16).view(np.uint16),
                       synth.lognormal_f16(rng, n),
                       synth.activations_bf16(rng, 3, n), np.zeros(0))
    y = gpu_gemv(lin)
    f = lambda h: h.view(np.float16).astype(np.float64)
    expect = f(lin.s_out) * f(lin.s_in) * bf16_bits_to_f64(torch.from_numpy(lin.x.view(np.int16)))
    assert max_row_rel_l2(y, expect) <= TOL


def test_gemv_one_hot_columns(oracle):
    m, n, r = 64, 96, 64
    lin = synth.make_linear(17, m, n, r, 1)
    cols = [0, 31, 32, 63, 95]
    x = np.zeros((len(cols), n), np.uint16)
    x[np.arange(len(cols)), cols] = 0x3F80
    W = oracle.what_packed(m, n, r, lin.Bu, lin.Bv, lin.s_out, lin.s_mid, lin.s_in)
    assert max_row_rel_l2(gpu_gemv(lin, x), W[:, cols].T) <= TOL


# --------------------------------------------------------------------------
# GEMM (prefill)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("m,n,r,T", [(32, 32, 32, 1), (96, 2080, 160, 7), (544, 4128, 96, 130),
                                     (1056, 64, 2080, 257), (4096, 4096, 2016, 64)])
def test_gemm_small_shapes(oracle, m, n, r, T):
    lin = synth.make_linear(2000 + m + n + r + T, m, n, r, T)
    err = max_row_rel_l2(gpu_gemm(lin), oracle_y(oracle, lin))
    print(f"gemm {m}x{n} r={r} T={T} max row rel-L2 {err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("name", ["sq8192", "mlp_up28672x8192", "mlp_down8192x28672"])
def test_gemm_full_size_sampled_tokens(oracle, name):
    """2048 tokens at the 70B-shaped sizes; the oracle checks a seeded sample
    of 16 tokens, the last token included (it computes each token
    independently)."""
    m, n, r = synth.SHAPES[name]
    T = 2048
    lin = synth.make_linear(11, m, n, r, T)
    y = gpu_gemm(lin)
    idx = np.sort(np.random.default_rng(0).choice(T, 16, replace=False))
    idx[-1] = T - 1
    ref = oracle_y(oracle, lin, lin.x[idx])
    err = max_row_rel_l2(y[idx], ref)
    print(f"{name} T=2048 sampled max row rel-L2 {err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("m,n,r,T", [(4096, 4096, 2016, 17), (4096, 4096, 2016, 100),
                                     (4096, 14336, 3136, 33), (14336, 4096, 3136, 48),
                                     (1056, 2080, 4064, 3)])
def test_gemm_split_k_few_tokens(oracle, m, n, r, T):
    """Token counts whose tile grid leaves most compute units idle: the
    contractions split their K steps over several workgroups (partial last
    step included: 2016/32 = 63 and 4064/32 = 127 words) and a second launch
    adds the partials in split order.  Element-wise against the oracle, and
    bit-identical on a repeat."""
    lin = synth.make_linear(3000 + m + r + T, m, n, r, T)
    y = gpu_gemm(lin)
    ref = oracle_y(oracle, lin)
    assert max_row_rel_l2(y, ref) <= TOL
    ok, where = elementwise_ok(y, ref, rel=2 ** -6, abs_rms=6e-3)
    assert ok, where
    assert np.array_equal(y, gpu_gemm(lin))


def test_gemm_matches_gemv_rows(oracle):
    lin = synth.make_linear(23, 4096, 4096, 2016, 16)
    a = gpu_gemm(lin)
    b = gpu_gemv(lin)
    ref = oracle_y(oracle, lin)
    assert max_row_rel_l2(a, ref) <= TOL and max_row_rel_l2(b, ref) <= TOL
