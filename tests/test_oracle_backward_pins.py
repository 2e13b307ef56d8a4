"""Pins for the oracle's scale-only reconstruction gradients and for the bit
transpose of the packed storage (Sec. 4.1, scale-only global reconstruction:
the sign matrices are frozen and only s_out, s_mid and s_in are trained).

The layer y = s_out .* (Bu (s_mid .* (Bv (s_in .* x)))) is linear in each of
s_out, s_mid, s_in and x separately.  So for L = sum(dy .* y):
  * a one-hot vector in place of one scale gives that gradient entry exactly
    (evaluated here through the entry-wise path sum of App. A.2.1, a route
    that shares no step with the oracle's factorised chain rule);
  * dx = dy W_hat with W_hat the brute-force matrix;
  * sum(s .* ds) = L for each scale vector, and sum(x .* dx) = L;
  * dx is the forward of the transposed layer (Bv^T, Bu^T, scales swapped)
    applied to dy.
A dropped scale, a wrong index or a transposed factor fails at least one."""
import numpy as np
import pytest

from paper_2609_06161_amd import synth


def _f16(h):
    return np.asarray(h, np.uint16).view(np.float16).astype(np.float64)


def _bf16(h):
    return (np.asarray(h, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _unpack_numpy(words, cols):
    """+-1 matrix from packed words with numpy.unpackbits (little bit order)."""
    by = np.ascontiguousarray(words, dtype="<u4").view(np.uint8)
    bits = np.unpackbits(by, axis=1, bitorder="little")[:, :cols]
    return np.where(bits == 1, -1, 1).astype(np.int8)


def _pack_numpy(S):
    bits = (np.asarray(S) < 0).astype(np.uint8)
    rows, cols = bits.shape
    by = np.packbits(bits, axis=1, bitorder="little")
    return np.ascontiguousarray(by).view("<u4").reshape(rows, cols // 32).astype(np.uint32)


# --------------------------------------------------------------------------
# bit transpose
# --------------------------------------------------------------------------

@pytest.mark.parametrize("rows,cols", [(32, 32), (64, 96), (160, 32), (96, 224)])
def test_transpose_matches_numpy(oracle, rows, cols):
    W = synth.random_words(np.random.default_rng(rows * 7 + cols), rows, cols)
    got = oracle.transpose_packed(W, cols)
    assert got.shape == (cols, rows // 32)
    assert np.array_equal(got, _pack_numpy(_unpack_numpy(W, cols).T))


def test_transpose_single_bit_moves_to_mirror_position(oracle):
    rows, cols = 64, 96
    for (i, j) in [(0, 0), (5, 70), (63, 95), (33, 1)]:
        W = np.zeros((rows, cols // 32), np.uint32)
        W[i, j // 32] = np.uint32(1 << (j % 32))
        T = oracle.transpose_packed(W, cols)
        expect = np.zeros((cols, rows // 32), np.uint32)
        expect[j, i // 32] = np.uint32(1 << (i % 32))
        assert np.array_equal(T, expect)


def test_transpose_twice_is_identity(oracle):
    W = synth.random_words(np.random.default_rng(3), 96, 160)
    assert np.array_equal(oracle.transpose_packed(oracle.transpose_packed(W, 160), 96), W)


def test_transpose_rejects_ragged(oracle):
    with pytest.raises(ValueError):
        oracle.transpose_packed(np.zeros((40, 1), np.uint32), 32)


# --------------------------------------------------------------------------
# gradients
# --------------------------------------------------------------------------

def _loss_dense(A, B, a, lam, b, X, DY, oracle):
    """L = sum(dy .* (x W_hat^T)) with W_hat from the path sum."""
    W = oracle.what_dense(A, B, a, lam, b)
    return float(np.sum(DY * (X @ W.T)))


def _case(seed, m, n, r, batch):
    L = synth.make_linear(seed, m, n, r, batch)
    dy = synth.make_output_grad(seed + 1000, batch, m, scale=1.0)
    return L, dy


@pytest.mark.parametrize("m,n,r,batch", [(32, 64, 32, 3), (64, 32, 96, 2)])
def test_gradients_are_one_hot_path_sums(oracle, m, n, r, batch):
    L, dy = _case(71 + m + r, m, n, r, batch)
    dx, ds_out, ds_mid, ds_in = oracle.backward(m, n, r, L.Bu, L.Bv, L.s_out, L.s_mid,
                                                L.s_in, L.x, dy)
    A = _unpack_numpy(L.Bu, r)
    B = _unpack_numpy(L.Bv, n)
    a, lam, b = _f16(L.s_out), _f16(L.s_mid), _f16(L.s_in)
    X, DY = _bf16(L.x), _bf16(dy)
    e = lambda size, k: np.eye(size)[k]
    ref_out = [_loss_dense(A, B, e(m, i), lam, b, X, DY, oracle) for i in range(m)]
    ref_mid = [_loss_dense(A, B, a, e(r, k), b, X, DY, oracle) for k in range(r)]
    ref_in = [_loss_dense(A, B, a, lam, e(n, j), X, DY, oracle) for j in range(n)]
    np.testing.assert_allclose(ds_out, ref_out, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(ds_mid, ref_mid, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(ds_in, ref_in, rtol=1e-11, atol=1e-11)
    W = oracle.what_dense(A, B, a, lam, b)
    np.testing.assert_allclose(dx, DY @ W, rtol=1e-11, atol=1e-11)


def test_gradients_match_numpy_matrix_chain_rule(oracle):
    """The same gradients from dense numpy matrices and explicit diagonal
    products (a library routine for every contraction)."""
    m, n, r, batch = 96, 64, 128, 4
    L, dy = _case(83, m, n, r, batch)
    dx, ds_out, ds_mid, ds_in = oracle.backward(m, n, r, L.Bu, L.Bv, L.s_out, L.s_mid,
                                                L.s_in, L.x, dy)
    A = _unpack_numpy(L.Bu, r).astype(float)
    B = _unpack_numpy(L.Bv, n).astype(float)
    a, lam, b = _f16(L.s_out), _f16(L.s_mid), _f16(L.s_in)
    X, DY = _bf16(L.x), _bf16(dy)
    V = (X * b) @ B.T                  # pre-scale intermediate, tokens x r
    Z = (V * lam) @ A.T                # pre-scale output, tokens x m
    DT = (DY * a) @ A                  # tokens x r
    DU = (DT * lam) @ B                # tokens x n
    np.testing.assert_allclose(ds_out, np.einsum("ti,ti->i", DY, Z), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(ds_mid, np.einsum("tk,tk->k", DT, V), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(ds_in, np.einsum("tj,tj->j", DU, X), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dx, DU * b, rtol=1e-11, atol=1e-11)


def test_homogeneity_identities(oracle):
    m, n, r, batch = 128, 96, 160, 5
    L, dy = _case(91, m, n, r, batch)
    dx, ds_out, ds_mid, ds_in = oracle.backward(m, n, r, L.Bu, L.Bv, L.s_out, L.s_mid,
                                                L.s_in, L.x, dy)
    y = oracle.forward(m, n, r, L.Bu, L.Bv, L.s_out, L.s_mid, L.s_in, L.x)
    loss = float(np.sum(_bf16(dy) * y))
    scale = float(np.sum(np.abs(_bf16(dy) * y)))
    for lhs in (np.dot(_f16(L.s_out), ds_out), np.dot(_f16(L.s_mid), ds_mid),
                np.dot(_f16(L.s_in), ds_in), float(np.sum(_bf16(L.x) * dx))):
        assert abs(lhs - loss) <= 1e-12 * scale


def test_dx_is_forward_of_transposed_layer(oracle):
    m, n, r, batch = 64, 128, 96, 3
    L, dy = _case(97, m, n, r, batch)
    dx, _, _, _ = oracle.backward(m, n, r, L.Bu, L.Bv, L.s_out, L.s_mid, L.s_in, L.x, dy)
    BuT = oracle.transpose_packed(L.Bu, r)   # r x m
    BvT = oracle.transpose_packed(L.Bv, n)   # n x r
    # the transposed layer maps m -> n: its "Bu" is Bv^T (n x r), its "Bv" is
    # Bu^T (r x m), its output scale s_in and its input scale s_out
    ref = oracle.forward(n, m, r, BvT, BuT, L.s_in, L.s_mid, L.s_out, dy)
    np.testing.assert_allclose(dx, ref, rtol=1e-12, atol=1e-12)


def test_zero_upstream_gradient_and_empty_batch(oracle):
    m, n, r = 32, 64, 32
    L, dy = _case(101, m, n, r, 2)
    dx, a, b_, c = oracle.backward(m, n, r, L.Bu, L.Bv, L.s_out, L.s_mid, L.s_in, L.x,
                                   np.zeros_like(dy))
    assert not dx.any() and not a.any() and not b_.any() and not c.any()
    e = np.zeros((0, n), np.uint16)
    dx, a, b_, c = oracle.backward(m, n, r, L.Bu, L.Bv, L.s_out, L.s_mid, L.s_in, e,
                                   np.zeros((0, m), np.uint16))
    assert dx.shape == (0, n) and not a.any() and not b_.any() and not c.any()


def test_gradient_of_zero_scale_is_not_zero(oracle):
    """A zero output scale blocks dx but still has a gradient (the quantity
    ds_out = sum dy .* z does not pass through s_out)."""
    m, n, r = 32, 32, 32
    L, dy = _case(107, m, n, r, 3)
    s_out = L.s_out.copy()
    s_out[:] = 0
    dx, ds_out, ds_mid, ds_in = oracle.backward(m, n, r, L.Bu, L.Bv, s_out, L.s_mid,
                                                L.s_in, L.x, dy)
    assert not dx.any() and not ds_mid.any() and not ds_in.any()
    _, ds_ref, _, _ = oracle.backward(m, n, r, L.Bu, L.Bv, L.s_out, L.s_mid, L.s_in, L.x, dy)
    np.testing.assert_array_equal(ds_out, ds_ref)
