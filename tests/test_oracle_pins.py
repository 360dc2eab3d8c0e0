"""Pins of the fp64 CPU oracle against facts fixed by the paper and by
mathematics, independent of the oracle's own loops:

* the relative index of eq. index_computation: a hand-worked 2x2 fixture and
  exact combinatorial properties (range, centre diagonal, antisymmetry, bin
  counts, translation);
* Theorem 3.1/3.2: inside one window WBMM is a depthwise cross-correlation with
  a (2w-1)x(2w-1) kernel and zero padding w-1 -> torch's conv2d in fp64;
* the operator as a sum over relative offsets (linearity in the table: each
  offset shifts every window by itself), in numpy, and its gradients through
  torch autograd;
* one-hot tables: the output is exactly a shifted copy of the input;
* the backward passes: exact finite differences on integer data (the operator
  is bilinear, so a step-1 central difference has no truncation error), the
  trilinear adjoint identity, and the reversed-table identity;
* invariants: linearity, window/channel independence, window-aligned roll,
  180-degree rotation with a reversed table, padding = pad-then-crop;
* the hierarchical reparameterisation: the fused inference matrix reproduces
  the training-mode sum of a w=2l and a w=l WBMM plus two identity shortcuts.

The last test builds planted-mistake variants of the oracle and checks that
each one fails at least one pin.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rng(seed=0):
    return np.random.default_rng(seed)


def rel_err(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = max(np.abs(b).max(), 1e-300)
    return float(np.abs(a - b).max() / den)


# ----------------------------------------------------------------- index map

def test_index_matches_hand_worked_2x2(olib):
    rows = [l.split() for l in open(os.path.join(GOLDEN, "index_w2.txt"))
            if l.strip() and not l.startswith("#")]
    want = np.array(rows, dtype=np.int32)
    assert np.array_equal(oracle.relative_index(2, lib=olib), want)


def test_table_sizes_printed_in_paper(olib):
    sizes = json.load(open(os.path.join(GOLDEN, "paper_sizes.json")))
    for w in (7, 14):
        I = oracle.relative_index(w, lib=olib)
        assert I.shape == (sizes["w%d" % w]["d"],) * 2
        assert int(I.max()) + 1 == sizes["w%d" % w]["table_len"]
        assert len(np.unique(I)) == sizes["w%d" % w]["table_len"]
    mib = 256 * 196 * 196 * 4 / 2 ** 20
    assert abs(mib - sizes["m_fp32_w14_c256_mib"]) < 0.05


@pytest.mark.parametrize("w", [1, 2, 3, 5, 7, 8, 13, 14, 16])
def test_index_properties(olib, w):
    I = oracle.relative_index(w, lib=olib).astype(np.int64)
    K = 2 * w - 1
    d = w * w
    assert I.min() == 0 and I.max() == K * K - 1
    centre = (w - 1) * K + (w - 1)
    assert np.all(np.diag(I) == centre)          # zero offset on the diagonal
    assert np.all(I + I.T == K * K - 1)          # swapping in/out negates the offset
    counts = np.bincount(I.ravel(), minlength=K * K)
    dh = np.arange(K) - (w - 1)
    want = np.outer(w - np.abs(dh), w - np.abs(dh)).ravel()
    assert np.array_equal(counts, want)          # (w-|dh|)(w-|dw|) pairs per offset
    assert counts.sum() == d * d
    # translation: shifting both positions by the same in-window step keeps I
    P = np.arange(d).reshape(w, w)
    if w > 1:
        a, b = P[:-1, :-1].ravel(), P[1:, 1:].ravel()
        assert np.array_equal(I[np.ix_(a, a)], I[np.ix_(b, b)])


def test_index_rectangular(olib):
    wh, ww = 3, 5
    I = oracle.relative_index((wh, ww), lib=olib)
    assert I.max() + 1 == (2 * wh - 1) * (2 * ww - 1)
    assert np.all(I + I.T == (2 * wh - 1) * (2 * ww - 1) - 1)


# ----------------------------------------------------- forward: equivalences

def conv_reference(x, t, wh, ww):
    """Per-window depthwise cross-correlation with torch conv2d (fp64): each
    window (zero-padded at the image border) is an independent image padded by
    (wh-1, ww-1); kernel K_c = T[c].view(2wh-1, 2ww-1)."""
    B, C, H, W = x.shape
    NH, NW = -(-H // wh), -(-W // ww)
    xp = np.zeros((B, C, NH * wh, NW * ww))
    xp[:, :, :H, :W] = x
    win = xp.reshape(B, C, NH, wh, NW, ww).transpose(0, 2, 4, 1, 3, 5)
    win = torch.from_numpy(np.ascontiguousarray(win)).reshape(B * NH * NW, C, wh, ww)
    k = torch.from_numpy(np.ascontiguousarray(t)).reshape(C, 1, 2 * wh - 1, 2 * ww - 1)
    out = torch.nn.functional.conv2d(win, k, padding=(wh - 1, ww - 1), groups=C)
    out = out.reshape(B, NH, NW, C, wh, ww).permute(0, 3, 1, 4, 2, 5).numpy()
    return out.reshape(B, C, NH * wh, NW * ww)[:, :, :H, :W]


def shift_sum_form(x, t, wh, ww, xp=np):
    """The operator as a sum over relative offsets (linearity in the table):
    for each offset (dh, dw) = input - output, every output position p of a
    window receives T[c, k(dh, dw)] * X[p + (dh, dw)] when p + (dh, dw) lies
    in the same (zero-padded) window.  Written as slices of the windowed
    array, one offset at a time; works on numpy arrays or, with xp=torch, on
    torch tensors (differentiable)."""
    B, C, H, W = x.shape
    NH, NW = -(-H // wh), -(-W // ww)
    K1w = 2 * ww - 1
    if xp is np:
        pad = np.zeros((B, C, NH * wh, NW * ww))
        pad[:, :, :H, :W] = x
        y = np.zeros_like(pad)
    else:
        pad = torch.nn.functional.pad(x, (0, NW * ww - W, 0, NH * wh - H))
        y = torch.zeros_like(pad)
    win = pad.reshape(B, C, NH, wh, NW, ww)
    yw = y.reshape(B, C, NH, wh, NW, ww)
    for dh in range(-(wh - 1), wh):
        for dw in range(-(ww - 1), ww):
            k = (dh + wh - 1) * K1w + (dw + ww - 1)
            # outputs ho with 0 <= ho + dh < wh, xo with 0 <= xo + dw < ww
            ho0, ho1 = max(0, -dh), min(wh, wh - dh)
            xo0, xo1 = max(0, -dw), min(ww, ww - dw)
            coef = t[:, k].reshape(1, C, 1, 1, 1, 1)
            src = win[:, :, :, ho0 + dh:ho1 + dh, :, xo0 + dw:xo1 + dw]
            if xp is np:
                yw[:, :, :, ho0:ho1, :, xo0:xo1] += coef * src
            else:
                upd = torch.zeros_like(yw)
                upd[:, :, :, ho0:ho1, :, xo0:xo1] = coef * src
                yw = yw + upd
    return yw.reshape(B, C, NH * wh, NW * ww)[:, :, :H, :W]


@pytest.mark.parametrize("shape,w", [
    ((2, 3, 7, 7), 7),        # single window: plain depthwise conv (Thm 3.1/3.2)
    ((1, 2, 14, 14), 14),
    ((2, 3, 14, 21), 7),      # several windows
    ((1, 2, 10, 13), 4),      # padding on both axes
    ((2, 2, 5, 9), (2, 3)),   # rectangular window with padding
])
def test_forward_equals_windowed_depthwise_conv(olib, shape, w):
    wh, ww = (w, w) if isinstance(w, int) else w
    r = rng(1)
    x = r.standard_normal(shape)
    t = r.standard_normal((shape[1], (2 * wh - 1) * (2 * ww - 1)))
    y = oracle.forward(x, t, w, lib=olib)
    assert rel_err(y, conv_reference(x, t, wh, ww)) < 1e-13
    assert rel_err(y, shift_sum_form(x, t, wh, ww)) < 1e-13


def test_single_window_is_plain_depthwise_conv(olib):
    """H = W = w: the window is the whole map, so WBMM is exactly a depthwise
    conv with a (2w-1)^2 kernel and 'same' zero padding (Theorem 3.1)."""
    r = rng(2)
    B, C, w = 3, 4, 7
    x = r.standard_normal((B, C, w, w))
    t = r.standard_normal((C, (2 * w - 1) ** 2))
    k = torch.from_numpy(t).reshape(C, 1, 2 * w - 1, 2 * w - 1)
    ref = torch.nn.functional.conv2d(torch.from_numpy(x), k, padding=w - 1, groups=C).numpy()
    assert rel_err(oracle.forward(x, t, w, lib=olib), ref) < 1e-13


@pytest.mark.parametrize("w", [3, 7])
def test_one_hot_table_is_exact_shift(olib, w):
    """T[c] = e_k with k <-> (dh, dw) = input - output: Y[p] = X[p + (dh, dw)]
    when that input lies in p's window and in the image, else exactly 0."""
    r = rng(3)
    B, C, H, W = 2, 3, 2 * w + 1, 2 * w
    x = r.standard_normal((B, C, H, W))
    K = 2 * w - 1
    offs = [(0, 0), (1, 0), (0, -1), (-(w - 1), w - 1)]
    t = np.zeros((C, K * K))
    for c in range(C):
        dh, dw = offs[c % len(offs)]
        t[c, (dh + w - 1) * K + (dw + w - 1)] = 1.0
    y = oracle.forward(x, t, w, lib=olib)
    want = np.zeros_like(x)
    for c in range(C):
        dh, dw = offs[c % len(offs)]
        for h in range(H):
            for xq in range(W):
                hi, xi = h + dh, xq + dw
                if (0 <= hi < H and 0 <= xi < W and hi // w == h // w and xi // w == xq // w):
                    want[:, c, h, xq] = x[:, c, hi, xi]
    assert np.array_equal(y, want)


# -------------------------------------------------------------- backward pins

def int_inputs(shape, K2, seed):
    r = rng(seed)
    x = r.integers(-3, 4, size=shape).astype(np.float64)
    t = r.integers(-3, 4, size=(shape[1], K2)).astype(np.float64)
    dy = r.integers(-3, 4, size=shape).astype(np.float64)
    return x, t, dy


@pytest.mark.parametrize("shape,w", [((2, 2, 6, 9), 3), ((1, 3, 7, 7), 7), ((1, 2, 5, 7), 4)])
def test_backward_exact_finite_differences(olib, shape, w):
    """L(X, T) = <dY, WBMM(X; T)> is bilinear, so the step-1 central
    difference in any single entry of X or T is exact; on small integers every
    sum is exact in fp64 and the comparison is bitwise."""
    x, t, dy = int_inputs(shape, (2 * w - 1) ** 2, 4)
    L = lambda xx, tt: float(np.sum(dy * oracle.forward(xx, tt, w, lib=olib)))
    dx = oracle.backward_input(dy, t, w, lib=olib)
    dt = oracle.backward_table(x, dy, w, lib=olib)
    r = rng(5)
    for idx in [tuple(r.integers(0, s) for s in x.shape) for _ in range(12)] + [(0, 0, shape[2] - 1, shape[3] - 1)]:
        e = np.zeros_like(x)
        e[idx] = 1.0
        assert (L(x + e, t) - L(x - e, t)) / 2 == dx[idx]
    for idx in [tuple(r.integers(0, s) for s in t.shape) for _ in range(12)] + [(0, 0), (0, t.shape[1] - 1)]:
        e = np.zeros_like(t)
        e[idx] = 1.0
        assert (L(x, t + e) - L(x, t - e)) / 2 == dt[idx]


@pytest.mark.parametrize("shape,w", [((2, 3, 14, 14), 7), ((1, 2, 28, 28), 14), ((2, 2, 9, 11), 4)])
def test_adjoint_identity(olib, shape, w):
    r = rng(6)
    x = r.standard_normal(shape)
    dy = r.standard_normal(shape)
    t = r.standard_normal((shape[1], (2 * w - 1) ** 2))
    a = np.sum(dy * oracle.forward(x, t, w, lib=olib))
    b = np.sum(x * oracle.backward_input(dy, t, w, lib=olib))
    c = np.sum(t * oracle.backward_table(x, dy, w, lib=olib))
    s = np.sqrt(np.sum(x * x) * np.sum(dy * dy) * np.sum(t * t))
    assert abs(a - b) / s < 1e-13 and abs(a - c) / s < 1e-13


def test_backward_input_is_forward_with_reversed_table(olib):
    """M^T is M built from the reversed table, since I[i,j] + I[j,i] = K^2-1."""
    r = rng(7)
    for shape, w in (((2, 3, 14, 14), 7), ((1, 2, 10, 13), 4)):
        dy = r.standard_normal(shape)
        t = r.standard_normal((shape[1], (2 * w - 1) ** 2))
        a = oracle.backward_input(dy, t, w, lib=olib)
        b = oracle.forward(dy, t[:, ::-1], w, lib=olib)
        assert rel_err(a, b) < 1e-14


def test_gradients_match_autograd_of_shift_sum_form(olib):
    """dX and dT of the shift-and-add form through torch autograd (fp64): an
    independent formulation of the operator differentiated by the library."""
    r = rng(8)
    B, C, H, W, w = 2, 3, 10, 12, 5
    x = r.standard_normal((B, C, H, W))
    dy = r.standard_normal((B, C, H, W))
    t = r.standard_normal((C, (2 * w - 1) ** 2))
    tt = torch.tensor(t, requires_grad=True)
    xx = torch.tensor(x, requires_grad=True)
    y = shift_sum_form(xx, tt, w, w, xp=torch)
    assert rel_err(y.detach().numpy(), oracle.forward(x, t, w, lib=olib)) < 1e-13
    (y * torch.from_numpy(dy)).sum().backward()
    assert rel_err(oracle.backward_table(x, dy, w, lib=olib), tt.grad.numpy()) < 1e-13
    assert rel_err(oracle.backward_input(dy, t, w, lib=olib), xx.grad.numpy()) < 1e-13


# ----------------------------------------------------------------- invariants

def test_linearity_and_independence(olib):
    r = rng(9)
    B, C, H, W, w = 2, 3, 14, 21, 7
    x1, x2 = r.standard_normal((2, B, C, H, W))
    t1, t2 = r.standard_normal((2, C, (2 * w - 1) ** 2))
    f = lambda x, t: oracle.forward(x, t, w, lib=olib)
    assert rel_err(f(2 * x1 - 3 * x2, t1), 2 * f(x1, t1) - 3 * f(x2, t1)) < 1e-13
    assert rel_err(f(x1, 2 * t1 - 3 * t2), 2 * f(x1, t1) - 3 * f(x1, t2)) < 1e-13
    y = f(x1, t1)
    # perturb one window of one (b, c): nothing else changes, bit for bit
    xp = x1.copy()
    xp[1, 2, 7:14, 14:21] += r.standard_normal((7, 7))
    yp = f(xp, t1)
    mask = np.zeros_like(y, dtype=bool)
    mask[1, 2, 7:14, 14:21] = True
    assert np.array_equal(yp[~mask], y[~mask]) and not np.array_equal(yp[mask], y[mask])


def test_window_aligned_roll_and_rotation(olib):
    r = rng(10)
    B, C, H, W, w = 1, 2, 14, 21, 7
    x = r.standard_normal((B, C, H, W))
    t = r.standard_normal((C, (2 * w - 1) ** 2))
    y = oracle.forward(x, t, w, lib=olib)
    yr = oracle.forward(np.roll(x, (w, 2 * w), axis=(2, 3)), t, w, lib=olib)
    assert np.array_equal(yr, np.roll(y, (w, 2 * w), axis=(2, 3)))
    # rotating the image by 180 degrees negates every offset: reverse the table
    yrot = oracle.forward(x[:, :, ::-1, ::-1], t[:, ::-1], w, lib=olib)
    assert rel_err(yrot, y[:, :, ::-1, ::-1]) < 1e-14


@pytest.mark.parametrize("shape,w", [((2, 2, 10, 13), 4), ((1, 3, 15, 8), 7), ((1, 1, 3, 2), 5)])
def test_padding_is_pad_then_crop(olib, shape, w):
    """Sec. 3.4.1: zero-pad H, W up to window multiples (bottom/right), run,
    crop.  The padded run only adds exact zeros, so results are equal."""
    r = rng(11)
    B, C, H, W = shape
    x, dy = r.standard_normal((2,) + shape)
    t = r.standard_normal((C, (2 * w - 1) ** 2))
    ph, pw = (w - H % w) % w, (w - W % w) % w
    pad = lambda a: np.pad(a, ((0, 0), (0, 0), (0, ph), (0, pw)))
    assert np.array_equal(oracle.forward(x, t, w, lib=olib), oracle.forward(pad(x), t, w, lib=olib)[:, :, :H, :W])
    assert np.array_equal(oracle.backward_input(dy, t, w, lib=olib),
                          oracle.backward_input(pad(dy), t, w, lib=olib)[:, :, :H, :W])
    assert np.array_equal(oracle.backward_table(x, dy, w, lib=olib),
                          oracle.backward_table(pad(x), pad(dy), w, lib=olib))


# ------------------------------------------------------ dense (cached M) form

@pytest.mark.parametrize("shape,w", [((2, 3, 9, 10), (3, 5)), ((1, 2, 7, 6), (4, 2)),
                                     ((2, 2, 8, 8), 4), ((1, 3, 5, 14), (2, 7))])
def test_dense_form_matches_table_form(olib, shape, w):
    """Alg. 1 with the matrix built once (M_c = R[c, I], the cached-matrix
    variant) equals the table form for square and rectangular windows, in all
    three passes; the matrix gradient folded onto the table by the index is
    the table gradient."""
    wh, ww = (w, w) if isinstance(w, int) else w
    r = rng(16)
    C = shape[1]
    x, dy = r.standard_normal(shape), r.standard_normal(shape)
    t = r.standard_normal((C, (2 * wh - 1) * (2 * ww - 1)))
    m = oracle.build_matrix(t, w, lib=olib)
    assert m.shape == (C, wh * ww, wh * ww)
    assert rel_err(oracle.dense_forward(x, m, w, lib=olib), oracle.forward(x, t, w, lib=olib)) < 1e-13
    assert rel_err(oracle.dense_backward_input(dy, m, w, lib=olib),
                   oracle.backward_input(dy, t, w, lib=olib)) < 1e-13
    dm = oracle.dense_backward_matrix(x, dy, w, lib=olib)
    assert rel_err(oracle.bin_matrix(dm, w, lib=olib), oracle.backward_table(x, dy, w, lib=olib)) < 1e-13


@pytest.mark.parametrize("w", [(3, 2), 3])
def test_dense_matrix_gradient_exact(olib, w):
    """dM pinned by exact finite differences of <dY, X_w M> in single entries
    of an arbitrary (non-Toeplitz) integer matrix, and the adjoint identity
    of the dense forward and input gradient."""
    wh, ww = (w, w) if isinstance(w, int) else w
    d = wh * ww
    r = rng(17)
    shape = (2, 2, 2 * wh + 1, 2 * ww + 1)
    x = r.integers(-3, 4, size=shape).astype(np.float64)
    dy = r.integers(-3, 4, size=shape).astype(np.float64)
    m = r.integers(-3, 4, size=(2, d, d)).astype(np.float64)
    loss = lambda mm: float(np.sum(dy * oracle.dense_forward(x, mm, w, lib=olib)))
    dm = oracle.dense_backward_matrix(x, dy, w, lib=olib)
    base = loss(m)
    for c, i, j in [(0, 0, 0), (1, d - 1, 0), (0, d // 2, d - 1), (1, 1, 2)]:
        e = np.zeros_like(m)
        e[c, i, j] = 1.0
        assert loss(m + e) - base == dm[c, i, j]
    assert float(np.sum(x * oracle.dense_backward_input(dy, m, w, lib=olib))) == base


# ------------------------------------------------------------- hierarchical

@pytest.mark.parametrize("shape,wl", [((2, 3, 28, 28), 7), ((1, 2, 20, 9), 3)])
def test_hierarchical_fused_equals_training_form(olib, shape, wl):
    """Training form: X_w M_g + X_w + X_sub M_l + X_sub; inference form:
    X_w M_fused with M_fused = M_g + diag_blocks(M_l) + 2 I."""
    r = rng(12)
    x = r.standard_normal(shape)
    C = shape[1]
    tg = r.standard_normal((C, (4 * wl - 1) ** 2))
    tl = r.standard_normal((C, (2 * wl - 1) ** 2))
    train = oracle.forward(x, tg, 2 * wl, lib=olib) + oracle.forward(x, tl, wl, lib=olib) + 2 * x
    assert rel_err(oracle.hier_forward(x, tg, tl, wl, lib=olib), train) < 1e-13
    z = oracle.hier_forward(x, 0 * tg, 0 * tl, wl, lib=olib)
    assert np.array_equal(z, 2 * x)


@pytest.mark.parametrize("shape,wl", [((2, 2, 12, 12), 3), ((1, 3, 10, 7), 2)])
def test_hierarchical_gradients(olib, shape, wl):
    """Gradients of the hierarchical form, pinned to its dense inference form
    (explicit M_fused, a separate code path): exact finite differences in
    both tables on integer data (the loss is bilinear), the adjoint identity
    for dX, and dX as the forward with both tables reversed."""
    r = rng(14)
    C = shape[1]
    x = r.integers(-3, 4, size=shape).astype(np.float64)
    dy = r.integers(-3, 4, size=shape).astype(np.float64)
    tg = r.integers(-3, 4, size=(C, (4 * wl - 1) ** 2)).astype(np.float64)
    tl = r.integers(-3, 4, size=(C, (2 * wl - 1) ** 2)).astype(np.float64)
    loss = lambda g, l: float(np.sum(dy * oracle.hier_forward(x, g, l, wl, lib=olib)))
    dtg, dtl = oracle.hier_backward_tables(x, dy, wl, lib=olib)
    base = loss(tg, tl)
    for c, k in [(0, 0), (C - 1, (4 * wl - 1) ** 2 // 2), (C // 2, 5)]:
        e = np.zeros_like(tg)
        e[c, k] = 1.0
        assert loss(tg + e, tl) - base == dtg[c, k]
    for c, k in [(0, 0), (C - 1, (2 * wl - 1) ** 2 // 2), (C // 2, 2)]:
        e = np.zeros_like(tl)
        e[c, k] = 1.0
        assert loss(tg, tl + e) - base == dtl[c, k]
    dx = oracle.hier_backward_input(dy, tg, tl, wl, lib=olib)
    assert float(np.sum(x * dx)) == base
    rev = oracle.hier_forward(dy, tg[:, ::-1].copy(), tl[:, ::-1].copy(), wl, lib=olib)
    assert np.array_equal(dx, rev)


# ------------------------------------------------ pins reject planted mistakes

def _pin_battery(lib):
    """Returns the list of pins that fail for the given oracle build."""
    failed = []
    r = rng(13)
    w = 4
    x = r.standard_normal((1, 2, 7, 10))
    t = r.standard_normal((2, (2 * w - 1) ** 2))
    dy = r.standard_normal(x.shape)
    if rel_err(oracle.forward(x, t, w, lib=lib), conv_reference(x, t, w, w)) > 1e-12:
        failed.append("conv")
    xi, ti, dyi = int_inputs((1, 2, 7, 10), (2 * w - 1) ** 2, 14)
    L = lambda xx, tt: float(np.sum(dyi * oracle.forward(xx, tt, w, lib=lib)))
    dt = oracle.backward_table(xi, dyi, w, lib=lib)
    dx = oracle.backward_input(dyi, ti, w, lib=lib)
    for k in range(ti.shape[1]):
        e = np.zeros_like(ti)
        e[0, k] = 1
        if (L(xi, ti + e) - L(xi, ti - e)) / 2 != dt[0, k]:
            failed.append("fd_t")
            break
    for h in range(7):
        for q in range(10):
            e = np.zeros_like(xi)
            e[0, 1, h, q] = 1
            if (L(xi + e, ti) - L(xi - e, ti)) / 2 != dx[0, 1, h, q]:
                failed.append("fd_x")
                break
        if failed and failed[-1] == "fd_x":
            break
    return failed


def test_pins_pass_on_real_oracle(olib):
    assert _pin_battery(olib) == []


@pytest.mark.parametrize("mutant", [1, 2, 3, 4])
def test_pins_reject_planted_mistakes(tmp_path, mutant):
    path = oracle.build(mutant=mutant, out_path=str(tmp_path / ("m%d.so" % mutant)),
                        openmp=False)
    lib = oracle.load(path)
    assert _pin_battery(lib) != []
