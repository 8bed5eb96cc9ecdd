"""Pins for the oracle's layer functions: central finite differences in fp64,
torch CPU float64 as an independent library routine, and hand-built cases
with known answers (tie rules, padding counts, bf16 rounding)."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import layers as ly
from oracle import stage as ostage


def _dirs(shape, n, seed=0):
    rng = np.random.default_rng(seed)
    return [rng.standard_normal(shape) for _ in range(n)]


def _fd_vs_vjp(f, args, idx, cot, vjp_val, h=1e-6, n=10):
    x = args[idx]
    for e in _dirs(x.shape, n):
        a1 = list(args); a1[idx] = x + h * e
        a2 = list(args); a2[idx] = x - h * e
        fd = (np.sum(cot * f(*a1)) - np.sum(cot * f(*a2))) / (2 * h)
        an = np.sum(vjp_val * e)
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (fd, an)


@pytest.mark.parametrize("k,bias", [(3, True), (1, False), (5, False)])
def test_conv_vjp_finite_differences(k, bias):
    rng = np.random.default_rng(k)
    x = rng.standard_normal((2, 5, 6, 3))
    w = rng.standard_normal((4, k, k, 3))
    b = rng.standard_normal(4) if bias else None
    dy = rng.standard_normal((2, 5, 6, 4))
    dx, dw, db = ly.conv2d_vjp(x, w, dy, True, bias)
    _fd_vs_vjp(lambda x_: ly.conv2d(x_, w, b), [x], 0, dy, dx)
    _fd_vs_vjp(lambda w_: ly.conv2d(x, w_, b), [w], 0, dy, dw)
    if bias:
        _fd_vs_vjp(lambda b_: ly.conv2d(x, w, b_), [b], 0, dy, db)


@pytest.mark.parametrize("k", [1, 3, 5])
def test_conv_matches_torch(k):
    rng = np.random.default_rng(10 + k)
    x = rng.standard_normal((3, 7, 5, 6))
    w = rng.standard_normal((8, k, k, 6))
    b = rng.standard_normal(8)
    xt = torch.tensor(x.transpose(0, 3, 1, 2), requires_grad=True)
    wt = torch.tensor(w.transpose(0, 3, 1, 2), requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    yt = F.conv2d(xt, wt, bt, padding=k // 2)
    dy = rng.standard_normal(yt.shape)
    yt.backward(torch.tensor(dy))
    y = ly.conv2d(x, w, b)
    np.testing.assert_allclose(y, yt.detach().numpy().transpose(0, 2, 3, 1), rtol=1e-12, atol=1e-12)
    dx, dw, db = ly.conv2d_vjp(x, w, dy.transpose(0, 2, 3, 1), True, True)
    np.testing.assert_allclose(dx, xt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw, wt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_linear_vjp_and_torch():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((5, 7))
    w = rng.standard_normal((3, 7))
    b = rng.standard_normal(3)
    dy = rng.standard_normal((5, 3))
    dx, dw, db = ly.linear_vjp(x, w, dy, True, True)
    _fd_vs_vjp(lambda x_: ly.linear(x_, w, b), [x], 0, dy, dx)
    _fd_vs_vjp(lambda w_: ly.linear(x, w_, b), [w], 0, dy, dw)
    np.testing.assert_allclose(ly.linear(x, w, b), F.linear(torch.tensor(x), torch.tensor(w),
                                                            torch.tensor(b)).numpy(), rtol=1e-13)


def test_batchnorm_vjp_finite_differences_and_torch():
    rng = np.random.default_rng(4)
    z = rng.standard_normal((3, 4, 5, 6)) * 2 + 0.5
    g = rng.uniform(0.5, 1.5, 6)
    be = rng.standard_normal(6)
    dy = rng.standard_normal(z.shape)
    y, xhat, rstd = ly.batchnorm(z, g, be)
    dz, dg, db = ly.batchnorm_vjp(xhat, rstd, g, dy)
    _fd_vs_vjp(lambda z_: ly.batchnorm(z_, g, be)[0], [z], 0, dy, dz)
    _fd_vs_vjp(lambda g_: ly.batchnorm(z, g_, be)[0], [g], 0, dy, dg)
    _fd_vs_vjp(lambda b_: ly.batchnorm(z, g, b_)[0], [be], 0, dy, db)
    zt = torch.tensor(z.transpose(0, 3, 1, 2), requires_grad=True)
    gt = torch.tensor(g, requires_grad=True)
    bt = torch.tensor(be, requires_grad=True)
    yt = F.batch_norm(zt, None, None, gt, bt, training=True, eps=ly.BN_EPS)
    yt.backward(torch.tensor(dy.transpose(0, 3, 1, 2)))
    np.testing.assert_allclose(y, yt.detach().numpy().transpose(0, 2, 3, 1), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dz, zt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dg, gt.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_relu_vjp_away_from_kink_and_at_zero():
    x = np.array([-2.0, -1e-3, 0.0, 1e-3, 3.0])
    dy = np.ones(5)
    np.testing.assert_array_equal(ly.relu_vjp(x, dy), [0, 0, 0, 1, 1])  # ReLU'(0) = 0
    np.testing.assert_array_equal(ly.relu(x), [0, 0, 0, 1e-3, 3.0])


def test_maxpool_finite_differences_and_torch():
    rng = np.random.default_rng(5)
    x = rng.permutation(2 * 6 * 4 * 3).reshape(2, 6, 4, 3).astype(np.float64) / 7.0  # distinct
    y, idx = ly.maxpool2(x)
    dy = rng.standard_normal(y.shape)
    dx = ly.maxpool2_vjp(x.shape, idx, dy)
    _fd_vs_vjp(lambda x_: ly.maxpool2(x_)[0], [x], 0, dy, dx, h=1e-7)
    xt = torch.tensor(x.transpose(0, 3, 1, 2), requires_grad=True)
    yt = F.max_pool2d(xt, 2)
    yt.backward(torch.tensor(dy.transpose(0, 3, 1, 2)))
    np.testing.assert_array_equal(y, yt.detach().numpy().transpose(0, 2, 3, 1))
    np.testing.assert_array_equal(dx, xt.grad.numpy().transpose(0, 2, 3, 1))


def test_maxpool_tie_goes_to_first_in_row_major_order():
    x = np.zeros((1, 2, 2, 3))
    x[0, :, :, 0] = [[1.0, 1.0], [1.0, 1.0]]   # all tied -> (0, 0)
    x[0, :, :, 1] = [[0.0, 2.0], [2.0, 0.0]]   # tie between (0,1) and (1,0) -> (0,1)
    x[0, :, :, 2] = [[0.0, 0.0], [0.0, 5.0]]   # unique max at (1,1)
    y, idx = ly.maxpool2(x)
    assert idx[0, 0, 0].tolist() == [0, 1, 3]
    dx = ly.maxpool2_vjp(x.shape, idx, np.ones((1, 1, 1, 3)))
    assert dx[0, 0, 0].tolist() == [1, 0, 0] and dx[0, 0, 1].tolist() == [0, 1, 0]
    assert dx[0, 1, 0].tolist() == [0, 0, 0] and dx[0, 1, 1].tolist() == [0, 0, 1]


def test_avgpool_counts_padding_and_matches_torch():
    x = np.zeros((1, 4, 4, 1))
    x[0, 0, 0, 0] = 9.0
    y = ly.avgpool3(x)
    assert y[0, 0, 0, 0] == 1.0 and y[0, 1, 1, 0] == 1.0 and y[0, 2, 2, 0] == 0.0
    rng = np.random.default_rng(6)
    x = rng.standard_normal((2, 5, 7, 3))
    xt = torch.tensor(x.transpose(0, 3, 1, 2), requires_grad=True)
    yt = F.avg_pool2d(xt, 3, 1, 1, count_include_pad=True)
    dy = rng.standard_normal(yt.shape)
    yt.backward(torch.tensor(dy))
    np.testing.assert_allclose(ly.avgpool3(x), yt.detach().numpy().transpose(0, 2, 3, 1), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(ly.avgpool3_vjp(dy.transpose(0, 2, 3, 1)),
                               xt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-13, atol=1e-15)


def test_gap_vjp_finite_differences():
    rng = np.random.default_rng(7)
    x = rng.standard_normal((2, 3, 5, 4))
    dy = rng.standard_normal((2, 4))
    _fd_vs_vjp(ly.gap, [x], 0, dy, ly.gap_vjp(x.shape, dy))


def test_softmax_ce_finite_differences_and_torch():
    rng = np.random.default_rng(8)
    z = rng.standard_normal((6, 10)) * 3
    lab = rng.integers(0, 10, 6)
    N = 24
    loss, dz = ly.softmax_ce(z, lab, N)
    _fd_vs_vjp(lambda z_: np.array(ly.softmax_ce(z_, lab, N)[0]), [z], 0, np.array(1.0), dz)
    zt = torch.tensor(z, requires_grad=True)
    lt = F.cross_entropy(zt, torch.tensor(lab), reduction="sum") / N
    lt.backward()
    assert abs(loss - lt.item()) < 1e-14
    np.testing.assert_allclose(dz, zt.grad.numpy(), rtol=1e-12, atol=1e-16)
    # large logits do not overflow (max subtraction)
    big = np.array([[1000.0, 0.0]])
    l2, _ = ly.softmax_ce(big, np.array([1]), 1)
    assert abs(l2 - 1000.0) < 1e-9


def test_bf16_rounding_matches_torch_and_ties_to_even():
    one = 1.0
    # 1 + 2^-8 is halfway between bf16 neighbours 1 and 1 + 2^-7: ties to even -> 1
    assert ostage._round_bf16(np.array([one + 2 ** -8]))[0] == 1.0
    # 1 + 3*2^-8 is halfway between 1 + 2^-7 and 1 + 2^-6: even mantissa is 1 + 2^-6
    assert ostage._round_bf16(np.array([one + 3 * 2 ** -8]))[0] == 1.0 + 2 ** -6
    rng = np.random.default_rng(9)
    a = rng.standard_normal(100000) * 10.0 ** rng.uniform(-20, 20, 100000)
    want = torch.tensor(a, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(ostage._round_bf16(a), want)


@pytest.mark.parametrize("k,H,W", [(1, 8, 7), (3, 9, 8), (7, 12, 11)])
def test_strided_conv_matches_torch(k, H, W):
    """Stride 2 (ResNet-101's stem, first blocks and projections): values and
    every gradient against torch's float64 convolution, odd and even sizes."""
    rng = np.random.default_rng(20 + k)
    x = rng.standard_normal((2, H, W, 5))
    w = rng.standard_normal((6, k, k, 5))
    b = rng.standard_normal(6)
    xt = torch.tensor(x.transpose(0, 3, 1, 2), requires_grad=True)
    wt = torch.tensor(w.transpose(0, 3, 1, 2), requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    yt = F.conv2d(xt, wt, bt, stride=2, padding=k // 2)
    assert yt.shape[2:] == (ly.conv_out(H, k, 2), ly.conv_out(W, k, 2)) == ((H - 1) // 2 + 1, (W - 1) // 2 + 1)
    dy = rng.standard_normal(yt.shape)
    yt.backward(torch.tensor(dy))
    y = ly.conv2d(x, w, b, stride=2)
    np.testing.assert_allclose(y, yt.detach().numpy().transpose(0, 2, 3, 1), rtol=1e-12, atol=1e-12)
    dx, dw, db = ly.conv2d_vjp(x, w, dy.transpose(0, 2, 3, 1), True, True, stride=2)
    np.testing.assert_allclose(dx, xt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw, wt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_strided_conv_vjp_finite_differences():
    rng = np.random.default_rng(31)
    x = rng.standard_normal((1, 7, 6, 2))
    w = rng.standard_normal((3, 3, 3, 2))
    dy = rng.standard_normal((1, 4, 3, 3))
    dx, dw, _ = ly.conv2d_vjp(x, w, dy, True, False, stride=2)
    _fd_vs_vjp(lambda x_: ly.conv2d(x_, w, None, 2), [x], 0, dy, dx)
    _fd_vs_vjp(lambda w_: ly.conv2d(x, w_, None, 2), [w], 0, dy, dw)


@pytest.mark.parametrize("H,W", [(9, 8), (8, 7)])
def test_maxpool3s2_matches_torch(H, W):
    """3x3 window, stride 2, padding 1 (the ResNet stem's pool): overlapping
    windows, so an input can take the gradient of up to four outputs."""
    rng = np.random.default_rng(40 + H)
    x = rng.permutation(2 * H * W * 3).reshape(2, H, W, 3).astype(np.float64) / 11.0  # distinct
    y, idx = ly.maxpool3s2(x)
    assert y.shape[1:3] == ((H - 1) // 2 + 1, (W - 1) // 2 + 1)
    dy = rng.standard_normal(y.shape)
    dx = ly.maxpool3s2_vjp(x.shape, idx, dy)
    xt = torch.tensor(x.transpose(0, 3, 1, 2), requires_grad=True)
    yt = F.max_pool2d(xt, 3, stride=2, padding=1)
    yt.backward(torch.tensor(dy.transpose(0, 3, 1, 2)))
    np.testing.assert_array_equal(y, yt.detach().numpy().transpose(0, 2, 3, 1))
    np.testing.assert_allclose(dx, xt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-15, atol=1e-15)
    _fd_vs_vjp(lambda x_: ly.maxpool3s2(x_)[0], [x], 0, dy, dx, h=1e-7)


def test_maxpool3s2_ties_and_padding():
    # output (0, 0) sees rows/cols -1..1: the padding never wins, even over negatives
    # a 2x2 input has one output, whose window covers rows/cols -1..1
    x = -np.ones((1, 2, 2, 2))
    x[0, :, :, 1] = [[0.0, 2.0], [2.0, 0.0]]
    y, idx = ly.maxpool3s2(x)
    assert y.shape == (1, 1, 1, 2) and y[0, 0, 0].tolist() == [-1.0, 2.0]
    # window positions are row-major over rows -1..1, cols -1..1: (0, 0) is index 4,
    # (0, 1) index 5, (1, 0) index 7; channel 1 ties (0, 1) and (1, 0) -> (0, 1)
    assert idx[0, 0, 0].tolist() == [4, 5]
    dx = ly.maxpool3s2_vjp(x.shape, idx, np.ones(y.shape))
    assert dx[0, :, :, 0].tolist() == [[1.0, 0.0], [0.0, 0.0]]
    assert dx[0, :, :, 1].tolist() == [[0.0, 1.0], [0.0, 0.0]]
    # overlapping windows: on a 3x3 input the pixel (0, 1) is in the windows of
    # outputs (0, 0) and (0, 1), and takes both gradients when it is both maxima
    x3 = np.zeros((1, 3, 3, 1))
    x3[0, 0, 1, 0] = 5.0
    y3, idx3 = ly.maxpool3s2(x3)
    dx3 = ly.maxpool3s2_vjp(x3.shape, idx3, np.ones(y3.shape))
    assert dx3[0, 0, 1, 0] == 2.0 and dx3.sum() == 4.0


@pytest.mark.parametrize("R,S,stride,valid", [(1, 7, 1, False), (7, 1, 1, False), (1, 3, 1, False),
                                              (3, 1, 1, False), (3, 3, 1, True), (3, 3, 2, True),
                                              (5, 3, 2, True)])
def test_general_conv_matches_torch(R, S, stride, valid):
    """Inception-V3's convolutions: 1 x n / n x 1 kernels with "same" padding
    (R//2, S//2), and unpadded ("valid") ones, strided or not."""
    rng = np.random.default_rng(50 + R * 7 + S + stride)
    x = rng.standard_normal((2, 11, 10, 4))
    w = rng.standard_normal((5, R, S, 4))
    b = rng.standard_normal(5)
    xt = torch.tensor(x.transpose(0, 3, 1, 2), requires_grad=True)
    wt = torch.tensor(w.transpose(0, 3, 1, 2), requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    yt = F.conv2d(xt, wt, bt, stride=stride, padding=(0, 0) if valid else (R // 2, S // 2))
    assert yt.shape[2:] == (ly.conv_out(11, R, stride, valid), ly.conv_out(10, S, stride, valid))
    dy = rng.standard_normal(yt.shape)
    yt.backward(torch.tensor(dy))
    y = ly.conv2d(x, w, b, stride, valid)
    np.testing.assert_allclose(y, yt.detach().numpy().transpose(0, 2, 3, 1), rtol=1e-12, atol=1e-12)
    dx, dw, db = ly.conv2d_vjp(x, w, dy.transpose(0, 2, 3, 1), True, True, stride, valid)
    np.testing.assert_allclose(dx, xt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw, wt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("H,W", [(9, 8), (8, 7)])
def test_maxpool3s2_valid_matches_torch(H, W):
    """The unpadded 3x3 stride-2 pool of Inception-V3 (output floor((H - 3) / 2) + 1)."""
    rng = np.random.default_rng(60 + H)
    x = rng.permutation(2 * H * W * 3).reshape(2, H, W, 3).astype(np.float64) / 13.0
    y, idx = ly.maxpool3s2(x, valid=True)
    assert y.shape[1:3] == ((H - 3) // 2 + 1, (W - 3) // 2 + 1)
    dy = rng.standard_normal(y.shape)
    dx = ly.maxpool3s2_vjp(x.shape, idx, dy, valid=True)
    xt = torch.tensor(x.transpose(0, 3, 1, 2), requires_grad=True)
    yt = F.max_pool2d(xt, 3, stride=2)
    yt.backward(torch.tensor(dy.transpose(0, 3, 1, 2)))
    np.testing.assert_array_equal(y, yt.detach().numpy().transpose(0, 2, 3, 1))
    np.testing.assert_allclose(dx, xt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-15, atol=1e-15)
