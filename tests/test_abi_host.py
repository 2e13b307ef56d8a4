"""Host-only checks of the C ABI: the library loads, exports every entry
point the header declares, its host arithmetic agrees with the oracle, and
every argument error is returned before anything is enqueued (fake device
addresses are safe here because no call below passes validation)."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2609_06161_amd import af1, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "af1.h")

BASE = 0x7F00_0000_0000          # fake, 16-byte aligned "device" addresses
MB = 1 << 20


def declared_functions(header=HEADER):
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(af1_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 10
    L = af1.lib()
    for name in names:
        assert hasattr(L, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", af1.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (af1_\w+)", out))
    assert set(names) == exported


def test_version_and_status_strings():
    assert "gfx950" in af1.af1_version()
    for st in range(0, 9):
        assert af1.status_string(st)
    assert af1.status_string(99) == "unknown status"


def test_storage_bits_matches_oracle(oracle):
    rng = np.random.default_rng(0)
    for _ in range(200):
        m, n, r = (int(v) for v in rng.integers(1, 1 << 15, size=3))
        assert af1.af1_storage_bits(m, n, r) == oracle.storage_bits(m, n, r)
    assert af1.af1_storage_bits(-1, 2, 3) == -1


def test_budget_rank_matches_oracle(oracle):
    for name, (m, n, r) in synth.SHAPES.items():
        assert af1.af1_budget_rank(m, n) == r, name
    rng = np.random.default_rng(1)
    for _ in range(300):
        m, n = (int(v) for v in rng.integers(1, 40000, size=2))
        assert af1.af1_budget_rank(m, n) == oracle.budget_rank(m, n), (m, n)
    assert af1.af1_budget_rank(0, 5) == 0
    assert af1.af1_budget_rank(32, 32) == 0      # scales alone exceed the budget


def test_budget_rank_other_budgets(oracle):
    """Any budget: the rank's storage (oracle.storage_bits, pinned to the
    paper's count) fits floor(bpw m n) bits and one more multiple does not."""
    rng = np.random.default_rng(2)
    for _ in range(300):
        m, n = (int(v) for v in rng.integers(32, 40000, size=2))
        bpw = float(rng.choice([0.55, 1.0, 1.5, 2.0, 2.5, 3.3]))
        mult = int(rng.choice([1, 16, 32, 64]))
        r = af1.af1_budget_rank(m, n, bpw, mult)
        budget = int(np.floor(bpw * m * n))
        assert r % mult == 0
        if r > 0:
            assert oracle.storage_bits(m, n, r) <= budget, (m, n, bpw, mult)
        assert oracle.storage_bits(m, n, r + mult) > budget, (m, n, bpw, mult)
    assert af1.af1_budget_rank(4096, 4096, 2.5, 32) == 5088   # scales counted
    assert af1.af1_budget_rank(4096, 4096, 0.0, 32) == 0
    assert af1.af1_budget_rank(4096, 4096, 1.0, 0) == 0


def test_paper_rank_matches_oracle(oracle):
    """The paper's sign-bits-only rank rule (App. A.1.3) through the ABI."""
    assert af1.af1_paper_rank(4096, 4096, 2.5) == 5120
    rng = np.random.default_rng(3)
    for _ in range(200):
        m, n = (int(v) for v in rng.integers(1, 40000, size=2))
        bpw = float(rng.uniform(0.1, 4.0))
        assert af1.af1_paper_rank(m, n, bpw) == oracle.paper_rank(bpw, m, n), (m, n, bpw)
    assert af1.af1_paper_rank(0, 5, 1.0) == 0


# --------------------------------------------------------------------------
# argument validation (no launch happens on any of these paths)
# --------------------------------------------------------------------------

def fake_layer(m=4096, n=4096, r=2016, base=BASE):
    # Bu, Bv, s_out, s_mid, s_in laid out 64 MB apart
    return af1.make_layer(m, n, r, base, base + 64 * MB, base + 128 * MB,
                          base + 129 * MB, base + 130 * MB)


X = BASE + 200 * MB
Y = BASE + 300 * MB
WS = BASE + 400 * MB


def gemv(layer, x=X, b=1, y=Y, ws=WS, ws_bytes=1 << 30):
    return af1.af1_linear_gemv(layer, x, b, y, ws, ws_bytes, stream=0, check=False)


def gemm(layer, x=X, T=16, y=Y, ws=WS, ws_bytes=1 << 30):
    return af1.af1_linear_gemm(layer, x, T, y, ws, ws_bytes, stream=0, check=False)


@pytest.mark.parametrize("fn", [gemv, gemm])
def test_forward_validation(fn):
    assert fn(None) == af1.AF1_ERR_NULL
    for m, n, r in [(0, 4096, 32), (4096, 4096, 33), (4096, 4064 + 16, 32),
                    (af1.AF1_MAX_DIM + 32, 4096, 32), (-32, 64, 32)]:
        assert fn(fake_layer(m, n, r)) == af1.AF1_ERR_SHAPE, (m, n, r)
    L = fake_layer()
    L.Bv = None
    assert fn(L) == af1.AF1_ERR_NULL
    assert fn(fake_layer(), x=None) == af1.AF1_ERR_NULL
    assert fn(fake_layer(), y=None) == af1.AF1_ERR_NULL
    assert fn(fake_layer(), x=X + 8) == af1.AF1_ERR_ALIGN
    L = fake_layer()
    L.s_mid = BASE + 129 * MB + 2
    assert fn(L) == af1.AF1_ERR_ALIGN
    # output overlapping an input or the workspace
    assert fn(fake_layer(), y=X + 16) == af1.AF1_ERR_ALIAS
    assert fn(fake_layer(), y=BASE + 128 * MB) == af1.AF1_ERR_ALIAS
    assert fn(fake_layer(), y=WS) == af1.AF1_ERR_ALIAS
    assert fn(fake_layer(), ws=BASE + 64 * MB) == af1.AF1_ERR_ALIAS


def test_gemv_batch_and_workspace_validation():
    L = fake_layer()
    assert gemv(L, b=0) == af1.AF1_ERR_BATCH
    assert gemv(L, b=17) == af1.AF1_ERR_BATCH
    need = af1.af1_gemv_workspace_bytes(4096, 4096, 2016, 8)
    assert need > 0
    assert gemv(L, b=8, ws_bytes=need - 1) == af1.AF1_ERR_WORKSPACE
    assert gemv(L, b=8, ws=None, ws_bytes=0) == af1.AF1_ERR_WORKSPACE
    assert af1.af1_gemv_workspace_bytes(4096, 4096, 2016, 0) == 0
    assert af1.af1_gemv_workspace_bytes(4096, 4096, 2016, 17) == 0
    assert af1.af1_gemv_workspace_bytes(4096, 4096, 33, 1) == 0


def test_gemm_token_and_workspace_validation():
    L = fake_layer()
    assert gemm(L, T=0) == af1.AF1_ERR_BATCH
    assert gemm(L, T=(1 << 20) + 1) == af1.AF1_ERR_BATCH
    need = af1.af1_gemm_workspace_bytes(4096, 4096, 2016, 2048)
    assert need >= 2048 * 2016 * 2
    assert gemm(L, T=2048, ws_bytes=need - 1) == af1.AF1_ERR_WORKSPACE


def test_gemm_workspace_holds_split_partials_only_for_few_tokens():
    """The GEMM workspace is fp16(s_in .* x), Z, the per-token range-guard
    record (four floats a token and four more) and the first product's row
    sums of Z per 256-column tile (a row padded to a multiple of 4 floats),
    each part 256-byte aligned, plus fp32 partials when a contraction splits
    its K steps, which happens only when the tile grid leaves compute units
    idle (here no GPU is present and the library plans for 256 compute
    units)."""
    a = lambda v: (v + 255) // 256 * 256
    m = n = 4096
    r = 2016
    ld = ((r + 255) // 256 + 3) // 4 * 4
    base = lambda T: a(T * n * 2) + a(T * r * 2) + a((4 * T + 4) * 4) + a(T * ld * 4)
    assert af1.af1_gemm_workspace_bytes(m, n, r, 2048) == base(2048)
    few = af1.af1_gemm_workspace_bytes(m, n, r, 64)
    assert few > base(64)
    # the partials: some number of splits of the larger of the two outputs
    extra = few - base(64)
    assert extra % 256 == 0 and extra <= 64 * (64 * max(r, m) * 4)


def test_gemm_rejects_operands_beyond_32bit_offsets():
    """The GEMM kernels address operands with 32-bit byte offsets: T * max(n,
    r) * 2 must stay below 2^31 (a batch error), a sign matrix below 2 GiB (a
    shape error); both are reported before anything is launched."""
    L = fake_layer(4096, 32768, 2016)            # widest operand row: 64 KiB
    assert gemm(L, T=32768, ws_bytes=1 << 40) == af1.AF1_ERR_BATCH
    L = fake_layer(4096, 2048, 32768)            # Z rows are the widest here
    assert gemm(L, T=32768, ws_bytes=1 << 40) == af1.AF1_ERR_BATCH
    big = 1 << 20
    assert gemm(fake_layer(big, 4096, big), T=1) == af1.AF1_ERR_SHAPE
    assert gemm(fake_layer(4096, big, big), T=1) == af1.AF1_ERR_SHAPE


def test_gemv_multi_validation():
    M = af1.af1_linear_gemv_multi
    q = fake_layer(4096, 4096, 2016)
    k = fake_layer(1024, 4096, 800, base=BASE + 512 * MB)
    v = fake_layer(1024, 4096, 800, base=BASE + 1024 * MB)
    ys = [Y, Y + 16 * MB, Y + 32 * MB]
    call = lambda layers, ys, **kw: M(layers, kw.get("x", X), kw.get("b", 1), ys, WS,
                                      kw.get("ws_bytes", 1 << 30), stream=0, check=False)
    assert call([q, k, v], None) == af1.AF1_ERR_NULL
    assert call([q, k, v], [Y, None, Y + 32 * MB]) == af1.AF1_ERR_NULL
    assert call([q, k, fake_layer(1024, 2048, 800, base=BASE + 1024 * MB)], ys) == af1.AF1_ERR_SHAPE
    assert call([q, k, v, q, k], ys + [Y + 48 * MB, Y + 64 * MB]) == af1.AF1_ERR_SHAPE
    assert call([q, k, v], ys, b=17) == af1.AF1_ERR_BATCH
    assert call([q, k, v], ys, ws_bytes=1024) == af1.AF1_ERR_WORKSPACE
    # two outputs overlapping each other, and an output over another layer's signs
    assert call([q, k, v], [Y, Y + 4096, Y + 32 * MB]) == af1.AF1_ERR_ALIAS
    assert call([q, k, v], [Y, Y + 16 * MB, BASE + 512 * MB]) == af1.AF1_ERR_ALIAS
    need = af1.af1_gemv_multi_workspace_bytes([q, k, v], 1)
    assert need >= af1.af1_gemv_workspace_bytes(4096, 4096, 2016, 1)
    assert af1.af1_gemv_multi_workspace_bytes([q, k, v], 0) == 0
    assert af1.af1_gemv_multi_workspace_bytes([], 1) == 0


def test_pack_validation():
    P = af1.af1_pack
    assert P(None, 0, 4, 64, Y, stream=0, check=False) == af1.AF1_ERR_NULL
    assert P(X, 0, 4, 64, None, stream=0, check=False) == af1.AF1_ERR_NULL
    assert P(X, 7, 4, 64, Y, stream=0, check=False) == af1.AF1_ERR_DTYPE
    assert P(X, -1, 4, 64, Y, stream=0, check=False) == af1.AF1_ERR_DTYPE
    assert P(X, 0, 4, 48, Y, stream=0, check=False) == af1.AF1_ERR_SHAPE
    assert P(X, 0, 4, 0, Y, stream=0, check=False) == af1.AF1_ERR_SHAPE
    assert P(X, 0, -1, 64, Y, stream=0, check=False) == af1.AF1_ERR_SHAPE
    assert P(X + 4, 0, 4, 64, Y, stream=0, check=False) == af1.AF1_ERR_ALIGN
    assert P(X, 0, 4, 64, X + 512, stream=0, check=False) == af1.AF1_ERR_ALIAS
    U = af1.af1_unpack
    assert U(None, 4, 64, Y, stream=0, check=False) == af1.AF1_ERR_NULL
    assert U(X, 4, 40, Y, stream=0, check=False) == af1.AF1_ERR_SHAPE
    assert U(X, 4, 64, Y + 1, stream=0, check=False) == af1.AF1_ERR_ALIGN
    assert U(X, 4, 64, X + 16, stream=0, check=False) == af1.AF1_ERR_ALIAS


def test_binding_raises_on_error():
    with pytest.raises(af1.Af1Error) as ei:
        af1.af1_linear_gemv(None, X, 1, Y, WS, 1 << 20, stream=0)
    assert ei.value.status == af1.AF1_ERR_NULL


def test_transpose_validation():
    Tp = af1.af1_pack_transpose
    call = lambda src=X, rows=64, cols=96, dst=Y: Tp(src, rows, cols, dst, stream=0, check=False)
    assert call(src=None) == af1.AF1_ERR_NULL
    assert call(dst=None) == af1.AF1_ERR_NULL
    for rows, cols in [(48, 96), (64, 40), (-32, 64), (64, -32),
                       ((1 << 24) + 32, 32), (32, (1 << 24) + 32), (1 << 21, 1 << 20)]:
        assert call(rows=rows, cols=cols) == af1.AF1_ERR_SHAPE, (rows, cols)
    assert call(src=X + 4) == af1.AF1_ERR_ALIGN
    assert call(dst=Y + 8) == af1.AF1_ERR_ALIGN
    assert call(dst=X + 256) == af1.AF1_ERR_ALIAS   # 64 x 96 bits = 768 bytes


SAVED = BASE + 600 * MB
BUT = BASE + 700 * MB
BVT = BASE + 800 * MB
DY = BASE + 900 * MB
DX = BASE + 1000 * MB
G_OUT, G_MID, G_IN = BASE + 1100 * MB, BASE + 1101 * MB, BASE + 1102 * MB


def fwd_train(layer, x=X, T=16, y=Y, saved=SAVED, saved_bytes=1 << 30, ws=WS, ws_bytes=1 << 30):
    return af1.af1_linear_forward_train(layer, x, T, y, saved, saved_bytes, ws, ws_bytes,
                                        stream=0, check=False)


def bwd(layer, BuT=BUT, BvT=BVT, x=X, dy=DY, T=16, saved=SAVED, saved_bytes=1 << 30, dx=DX,
        g=(G_OUT, G_MID, G_IN), acc=0, ws=WS, ws_bytes=1 << 30):
    return af1.af1_linear_backward(layer, BuT, BvT, x, dy, T, saved, saved_bytes, dx, g[0], g[1],
                                   g[2], acc, ws, ws_bytes, stream=0, check=False)


def test_forward_train_validation():
    assert fwd_train(None) == af1.AF1_ERR_NULL
    assert fwd_train(fake_layer(4096, 4096, 33)) == af1.AF1_ERR_SHAPE
    assert fwd_train(fake_layer(), saved=None) == af1.AF1_ERR_NULL
    assert fwd_train(fake_layer(), saved=SAVED + 8) == af1.AF1_ERR_ALIGN
    assert fwd_train(fake_layer(), T=0) == af1.AF1_ERR_BATCH
    # T * max(m, n, r) * 2 < 2^31: m is the widest here
    assert fwd_train(fake_layer(65536, 1024, 512), T=16384, saved_bytes=1 << 40,
                     ws_bytes=1 << 40) == af1.AF1_ERR_BATCH
    need = af1.af1_train_saved_bytes(4096, 4096, 2016, 16)
    assert need >= 16 * 2016 * 2 + 16 * 4096 * 4
    assert fwd_train(fake_layer(), saved_bytes=need - 1) == af1.AF1_ERR_WORKSPACE
    wneed = af1.af1_train_workspace_bytes(4096, 4096, 2016, 16)
    assert wneed >= af1.af1_gemm_workspace_bytes(4096, 4096, 2016, 16)
    assert fwd_train(fake_layer(), ws_bytes=wneed - 1) == af1.AF1_ERR_WORKSPACE
    assert fwd_train(fake_layer(), saved=X) == af1.AF1_ERR_ALIAS
    assert fwd_train(fake_layer(), saved=Y) == af1.AF1_ERR_ALIAS
    assert fwd_train(fake_layer(), saved=WS + 1024) == af1.AF1_ERR_ALIAS
    assert fwd_train(fake_layer(), y=SAVED) == af1.AF1_ERR_ALIAS
    assert af1.af1_train_saved_bytes(4096, 4096, 2016, 0) == 0
    assert af1.af1_train_workspace_bytes(4096, 33, 2016, 1) == 0


def test_backward_validation():
    L = fake_layer()
    assert bwd(None) == af1.AF1_ERR_NULL
    assert bwd(fake_layer(4096, 48, 2016)) == af1.AF1_ERR_SHAPE
    for kw in ("BuT", "BvT", "x", "dy", "saved"):
        assert bwd(L, **{kw: None}) == af1.AF1_ERR_NULL, kw
    assert bwd(L, g=(None, G_MID, G_IN)) == af1.AF1_ERR_NULL
    assert bwd(L, g=(G_OUT, G_MID, None)) == af1.AF1_ERR_NULL
    Lnull = fake_layer()
    Lnull.Bu = None
    Lnull.Bv = None                  # the forward factors are not read: the
    assert bwd(Lnull, T=0) == af1.AF1_ERR_BATCH   # next check is reached
    Ls = fake_layer()
    Ls.s_mid = None
    assert bwd(Ls) == af1.AF1_ERR_NULL
    assert bwd(L, T=0) == af1.AF1_ERR_BATCH
    assert bwd(L, T=(1 << 20) + 1) == af1.AF1_ERR_BATCH
    assert bwd(L, dy=DY + 2) == af1.AF1_ERR_ALIGN
    assert bwd(L, g=(G_OUT + 4, G_MID, G_IN)) == af1.AF1_ERR_ALIGN
    need = af1.af1_train_saved_bytes(4096, 4096, 2016, 16)
    assert bwd(L, saved_bytes=need - 1) == af1.AF1_ERR_WORKSPACE
    assert bwd(L, ws=None, ws_bytes=0) == af1.AF1_ERR_WORKSPACE
    # outputs against inputs and against each other
    assert bwd(L, dx=DY) == af1.AF1_ERR_ALIAS
    assert bwd(L, dx=SAVED + 256) == af1.AF1_ERR_ALIAS
    assert bwd(L, g=(G_OUT, G_OUT + 1024, G_IN)) == af1.AF1_ERR_ALIAS
    assert bwd(L, g=(BASE + 128 * MB, G_MID, G_IN)) == af1.AF1_ERR_ALIAS
    assert bwd(L, ws=BUT) == af1.AF1_ERR_ALIAS
    assert bwd(L, dx=WS) == af1.AF1_ERR_ALIAS


# --------------------------------------------------------------------------
# NABF building blocks (libaf1_nabf.so, include/af1_nabf.h)
# --------------------------------------------------------------------------

from paper_2609_06161_amd import nabf  # noqa: E402

NABF_HEADER = os.path.join(ROOT, "include", "af1_nabf.h")


def test_nabf_library_exports_every_declared_symbol():
    names = declared_functions(NABF_HEADER)
    assert len(names) >= 8
    L = nabf.lib()
    for name in names:
        assert hasattr(L, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", nabf.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    assert set(names) == set(re.findall(r"\bT (af1_\w+)", out))


def test_nabf_workspace_query():
    a = nabf.af1_nabf_workspace_bytes(4096, 4096, 2016, 0)
    b = nabf.af1_nabf_workspace_bytes(4096, 4096, 2016, 4096)
    assert a >= 4 * (2 * 4096 * 2016 + 3 * 4096 * 2016 + 3 * 2016 * 2016) + 8 * 2 * 2016 * 2016
    assert b > a
    assert nabf.af1_nabf_workspace_bytes(4096, 4096, 33, 0) == 0
    assert nabf.af1_nabf_workspace_bytes(4096, 4096, 2016, -1) == 0
    assert nabf.af1_nabf_workspace_bytes(4096, 4096, nabf.AF1_NABF_MAX_DIM + 32, 0) == 0


W0, W1, W2, W3, W4, W5 = (BASE + k * 256 * MB for k in range(6))


def test_nabf_validation_before_any_launch():
    E = af1
    big = 1 << 40
    sv = lambda **kw: nabf.af1_svid(kw.get("Z", W0), kw.get("rows", 64), kw.get("cols", 96),
                                    kw.get("iters", 5), kw.get("bits", W1), kw.get("left", W2),
                                    kw.get("right", W3), kw.get("ws", W4), kw.get("wsb", big),
                                    stream=0, check=False)
    assert sv(Z=None) == E.AF1_ERR_NULL
    assert sv(rows=48) == E.AF1_ERR_SHAPE
    assert sv(iters=-1) == E.AF1_ERR_SHAPE
    assert sv(iters=nabf.AF1_NABF_MAX_POWER_ITERS + 1) == E.AF1_ERR_SHAPE
    assert sv(rows=65536, cols=65536) == E.AF1_ERR_SHAPE        # 2^32 elements
    assert sv(left=W2 + 4) == E.AF1_ERR_ALIGN
    assert sv(wsb=1024) == E.AF1_ERR_WORKSPACE
    pr = lambda **kw: nabf.af1_nullspace_projector(kw.get("C", W0), kw.get("r", 64),
                                                   kw.get("eta", 0.01), kw.get("P", W1), None,
                                                   kw.get("ws", W4), kw.get("wsb", big),
                                                   stream=0, check=False)
    assert pr(C=None) == E.AF1_ERR_NULL
    assert pr(eta=-0.5) == E.AF1_ERR_SHAPE
    assert pr(eta=float("nan")) == E.AF1_ERR_SHAPE
    assert pr(r=40) == E.AF1_ERR_SHAPE
    assert pr(P=W1 + 8) == E.AF1_ERR_ALIGN
    assert pr(ws=None, wsb=0) == E.AF1_ERR_WORKSPACE
    assert pr(P=W0) == E.AF1_ERR_ALIAS
    ad = lambda **kw: nabf.af1_admm_proxy(kw.get("side", 0), W0, 64, 96, 32, W1, W2, W3,
                                          kw.get("rho", 0.5), kw.get("out", W5), W4,
                                          kw.get("wsb", big), stream=0, check=False)
    assert ad(side=2) == E.AF1_ERR_SHAPE
    assert ad(rho=0.0) == E.AF1_ERR_SHAPE
    assert ad(rho=-1.0) == E.AF1_ERR_SHAPE
    assert ad(out=None) == E.AF1_ERR_NULL
    assert ad(out=W1) == E.AF1_ERR_ALIAS
    assert ad(wsb=100) == E.AF1_ERR_WORKSPACE
    sf = lambda **kw: nabf.af1_scale_fit(kw.get("side", 0), W0, W1, W2, W3, kw.get("rows", 64),
                                         kw.get("cols", 32), kw.get("P", W4), W5, W4 + MB,
                                         kw.get("wsb", big), stream=0, check=False)
    assert sf(side=-1) == E.AF1_ERR_SHAPE
    assert sf(P=None) == E.AF1_ERR_NULL
    assert sf(cols=33) == E.AF1_ERR_SHAPE
    assert sf(wsb=10) == E.AF1_ERR_WORKSPACE
    su = lambda **kw: nabf.af1_nabf_surrogate(W0, 64, 96, W1, W2, kw.get("T", 128),
                                              kw.get("Wp", W3), W4, W4 + MB, W5,
                                              kw.get("wsb", big), stream=0, check=False)
    assert su(T=0) == E.AF1_ERR_BATCH
    assert su(Wp=None) == E.AF1_ERR_NULL
    assert su(Wp=W0) == E.AF1_ERR_ALIAS
    assert su(wsb=16) == E.AF1_ERR_WORKSPACE


def test_nabf_iteration_validation():
    E = af1
    arrays = [BASE + k * 64 * MB for k in range(10)]
    S = nabf.make_state(64, 96, 32, *arrays)
    it = lambda S, **kw: nabf.af1_nabf_iteration(kw.get("Wp", BASE + 700 * MB), S,
                                                 kw.get("rho", 0.5), kw.get("eta", 0.01),
                                                 kw.get("iters", 10),
                                                 kw.get("ws", BASE + 800 * MB),
                                                 kw.get("wsb", 1 << 40), stream=0, check=False)
    assert it(None) == E.AF1_ERR_NULL
    assert it(S, Wp=None) == E.AF1_ERR_NULL
    bad = nabf.make_state(64, 96, 32, *arrays[:5], None, *arrays[6:])
    assert it(bad) == E.AF1_ERR_NULL
    assert it(nabf.make_state(64, 96, 48, *arrays)) == E.AF1_ERR_SHAPE
    assert it(S, rho=0.0) == E.AF1_ERR_SHAPE
    assert it(S, eta=2.0) == E.AF1_ERR_SHAPE
    assert it(S, iters=-3) == E.AF1_ERR_SHAPE
    assert it(nabf.make_state(64, 96, 32, *arrays[:9], arrays[9] + 4)) == E.AF1_ERR_ALIGN
    assert it(S, wsb=1000) == E.AF1_ERR_WORKSPACE
    # two arrays of the state overlapping, and the workspace over Wp
    assert it(nabf.make_state(64, 96, 32, arrays[0], arrays[0] + 1024, *arrays[2:])) == \
        E.AF1_ERR_ALIAS
    assert it(S, ws=BASE + 700 * MB) == E.AF1_ERR_ALIAS
    assert nabf.af1_nabf_export(None, None, None, W0, W1, W2, stream=0, check=False) == \
        E.AF1_ERR_NULL
    assert nabf.af1_nabf_export(S, None, None, W0, None, W2, stream=0, check=False) == \
        E.AF1_ERR_NULL


# --------------------------------------------------------------------------
# layer stream: planning and validation (host only; nothing is launched)
# --------------------------------------------------------------------------

def stream_entries(specs, base=BASE):
    """(m, n, r, x, y, wait) -> stream items over fake, disjoint layer arrays."""
    entries = []
    for i, (m, n, r, x, y, wait) in enumerate(specs):
        entries.append((fake_layer(m, n, r, base + 1024 * MB + i * 64 * MB), x, y, wait))
    return af1.stream_items(entries)


def test_stream_plan_sizes_and_validation():
    q = (4096, 4096, 2016, X, Y, False)
    o = (4096, 4096, 2016, Y, Y + 1 * MB, True)           # reads q's output, waits
    items = stream_entries([q, o])
    ws = af1.af1_stream_workspace_bytes(items, 1)
    plan = af1.af1_stream_plan_bytes(items, 1)
    assert ws >= 2 * 2016 * 4 and 0 < plan < 4096
    buf = np.zeros(plan, np.uint8)
    assert af1.af1_stream_plan(items, 1, WS, ws, buf, plan, check=False) == af1.AF1_OK
    assert af1.af1_stream_plan(items, 1, WS, ws - 1, buf, plan, check=False) == \
        af1.AF1_ERR_WORKSPACE
    assert af1.af1_stream_plan(items, 1, WS, ws, buf, plan - 1, check=False) == \
        af1.AF1_ERR_WORKSPACE
    assert af1.af1_stream_plan(items, 0, WS, ws, buf, plan, check=False) == af1.AF1_ERR_BATCH
    assert af1.af1_stream_plan(items, 17, WS, ws, buf, plan, check=False) == af1.AF1_ERR_BATCH
    assert af1.af1_stream_plan(items, 1, WS, ws, buf, plan, count=0, check=False) == \
        af1.AF1_ERR_SHAPE
    assert af1.af1_stream_plan(None, 1, WS, ws, buf, plan, count=1, check=False) == \
        af1.AF1_ERR_NULL
    # o reading q's output without waiting: rejected
    bad = stream_entries([q, (4096, 4096, 2016, Y, Y + 1 * MB, False)])
    assert af1.af1_stream_plan(bad, 1, WS, ws, buf, plan, check=False) == af1.AF1_ERR_ALIAS
    # two outputs on one buffer
    bad = stream_entries([q, (4096, 4096, 2016, X, Y, False)])
    assert af1.af1_stream_plan(bad, 1, WS, ws, buf, plan, check=False) == af1.AF1_ERR_ALIAS
    # the workspace over an input
    assert af1.af1_stream_plan(items, 1, X, ws, buf, plan, check=False) == af1.AF1_ERR_ALIAS
    # a misaligned item
    bad = stream_entries([(4096, 4096, 2016, X + 8, Y, False)])
    assert af1.af1_stream_plan(bad, 1, WS, ws, buf, plan, check=False) == af1.AF1_ERR_ALIGN


def test_stream_rejects_foreign_plans():
    junk = np.zeros(4096, np.uint8)
    assert af1.af1_linear_stream(junk, BASE, 0, check=False) == af1.AF1_ERR_PLAN
    assert af1.af1_linear_stream(None, BASE, 0, check=False) == af1.AF1_ERR_NULL
    assert af1.af1_linear_stream(junk, BASE + 8, 0, check=False) == af1.AF1_ERR_ALIGN


def test_stream_plan_of_the_8b_stack_is_small():
    """224 linears (the 32-layer stack): a plan of a few hundred kB at most
    and a workspace of a few MB."""
    entries = synth.draw_stack_ranks(77, 32, [("q", 4096, 4096, 2016), ("k", 1024, 4096, 800),
                                              ("v", 1024, 4096, 800), ("o", 4096, 4096, 2016),
                                              ("gate", 14336, 4096, 3136),
                                              ("up", 14336, 4096, 3136),
                                              ("down", 4096, 14336, 3136)],
                                     af1.af1_storage_bits)
    specs = []
    for i, (name, m, n, r0, r) in enumerate(entries):
        specs.append((m, n, r, X + (i % 7) * 256 * 1024, Y + i * 64 * 1024,
                      name in ("q", "o", "gate", "down")))
    items = af1.stream_items([(fake_layer(m, n, r, BASE + 2048 * MB + i * 32 * MB), x, y, w)
                              for i, (m, n, r, x, y, w) in enumerate(specs)])
    plan = af1.af1_stream_plan_bytes(items, 1)
    ws = af1.af1_stream_workspace_bytes(items, 1)
    assert 0 < plan < 512 * 1024 and 0 < ws < 16 * MB
