"""Pins of the CPU oracle against facts the definition fixes (CPU only).

Each test names the property it checks.  None re-types the oracle's loop:
they compare it with hand-worked values, closed forms, a library matmul,
exact identities on integer data, an independently written scatter-form
convolution, and torch's float64 CPU conv2d.
"""
import itertools
import os

import numpy as np
import pytest

import datagen
import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_conv_examples.txt")


def _read_golden():
    cases, cur = [], None
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        key, val = [t.strip() for t in line.split(":", 1)]
        if key == "case":
            cur = {"name": val}
            cases.append(cur)
            continue
        if "|" in val:
            shp, vals = val.split("|")
            shape = tuple(int(t) for t in shp.split())
            cur[key] = np.array([float(t) for t in vals.split()], dtype=np.float64).reshape(shape)
        elif key == "b":
            cur[key] = np.array([float(t) for t in val.split()], dtype=np.float32)
        elif key == "groups":
            cur[key] = int(val)
        else:
            cur[key] = tuple(int(t) for t in val.split())
    return cases


@pytest.mark.parametrize("case", _read_golden(), ids=lambda c: c["name"])
def test_hand_worked_examples(case):
    y, _ = oracle.conv2d(case["x"], case["w"], case.get("b"), case["stride"], case["pad"],
                         case["dil"], case["groups"])
    assert y.shape == case["y"].shape
    np.testing.assert_array_equal(y, case["y"])


# ---------------------------------------------------------------- P1 shape formula

def _brute_extent(size, pad, dil, ext, stride):
    # number of window starts ho >= 0 whose last tap ho*s + d*(R-1) stays inside the padded input
    count = 0
    ho = 0
    while ho * stride + dil * (ext - 1) <= size + 2 * pad - 1:
        count += 1
        ho += 1
    return count


def test_output_dims_match_enumeration():
    rng = np.random.default_rng(1)
    for _ in range(3000):
        h, w = rng.integers(1, 40, size=2)
        r, s = rng.integers(1, 9, size=2)
        st = tuple(int(v) for v in rng.integers(1, 5, size=2))
        pd = tuple(int(v) for v in rng.integers(0, 5, size=2))
        dl = tuple(int(v) for v in rng.integers(1, 4, size=2))
        eh = _brute_extent(h, pd[0], dl[0], r, st[0])
        ew = _brute_extent(w, pd[1], dl[1], s, st[1])
        if eh < 1 or ew < 1:
            with pytest.raises(oracle.OracleError) as ei:
                oracle.output_dims((1, 1, h, w), (1, 1, r, s), st, pd, dl)
            assert ei.value.code == -2
        else:
            assert oracle.output_dims((1, 1, h, w), (1, 1, r, s), st, pd, dl) == (eh, ew)


def test_output_dims_known_layers():
    assert oracle.output_dims((1, 3, 32, 32), (16, 3, 3, 3), (1, 1), (1, 1)) == (32, 32)
    assert oracle.output_dims((32, 64, 56, 56), (64, 64, 3, 3), (1, 1), (1, 1)) == (56, 56)
    assert oracle.output_dims((32, 256, 56, 56), (512, 256, 1, 1), (2, 2), (0, 0)) == (28, 28)
    assert oracle.output_dims((32, 3, 224, 224), (64, 3, 7, 7), (2, 2), (3, 3)) == (112, 112)


@pytest.mark.parametrize("bad", [
    dict(x=(0, 1, 4, 4)), dict(x=(1, 3, 4, 4), w=(2, 2, 1, 1), g=2),
    dict(stride=(0, 1)), dict(dil=(1, 0)), dict(pad=(-1, 0)), dict(g=0),
])
def test_invalid_params_rejected(bad):
    x = bad.get("x", (1, 2, 4, 4))
    w = bad.get("w", (2, 2 // max(bad.get("g", 1), 1) if bad.get("g", 1) else 2, 1, 1))
    with pytest.raises(oracle.OracleError) as ei:
        oracle.output_dims(x, w, bad.get("stride", (1, 1)), bad.get("pad", (0, 0)),
                           bad.get("dil", (1, 1)), bad.get("g", 1))
    assert ei.value.code == -1


# ---------------------------------------------------------------- P2 1x1 = matmul

@pytest.mark.parametrize("stride", [1, 2, 3])
def test_pointwise_equals_matmul(stride):
    n, c, h, w, k = 3, 13, 9, 7, 11
    x = datagen.draw(10, 0, (n, c, h, w))
    wt = datagen.draw(10, 1, (k, c, 1, 1))
    b = datagen.draw(10, 2, (k,))
    y, _ = oracle.conv2d(x, wt, b, (stride, stride))
    xs = x[:, :, ::stride, ::stride].astype(np.float64)
    ref = np.matmul(wt[:, :, 0, 0].astype(np.float64), xs.reshape(n, c, -1))
    ref = ref.reshape(n, k, xs.shape[2], xs.shape[3])
    ref += b.astype(np.float64)[None, :, None, None]
    np.testing.assert_allclose(y, ref, rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------- P3 delta filters

def _delta_cases():
    for r, s in [(1, 1), (3, 3), (5, 3), (2, 4), (7, 7)]:
        for st in [(1, 1), (2, 1), (3, 2)]:
            for dl in [(1, 1), (2, 3)]:
                for pd in [(0, 0), (1, 2), (3, 3)]:
                    yield r, s, st, dl, pd


def test_delta_filters_reproduce_input():
    n, c, h, w = 2, 3, 11, 13
    x = datagen.draw(11, 0, (n, c, h, w))
    rng = np.random.default_rng(2)
    checked = 0
    for r, s, st, dl, pd in _delta_cases():
        try:
            ho, wo = oracle.output_dims(x.shape, (c, c, r, s), st, pd, dl)
        except oracle.OracleError:
            continue
        r0, s0 = int(rng.integers(0, r)), int(rng.integers(0, s))
        wt = np.zeros((c, c, r, s), dtype=np.float32)
        for k in range(c):
            wt[k, k, r0, s0] = 1.0
        y, _ = oracle.conv2d(x, wt, None, st, pd, dl)
        ref = np.zeros((n, c, ho, wo))
        for i in range(ho):
            for j in range(wo):
                hi, wi = i * st[0] - pd[0] + r0 * dl[0], j * st[1] - pd[1] + s0 * dl[1]
                if 0 <= hi < h and 0 <= wi < w:
                    ref[:, :, i, j] = x[:, :, hi, wi]
        np.testing.assert_array_equal(y, ref)
        checked += 1
    assert checked > 60


def test_centre_delta_same_padding_is_identity():
    x = datagen.draw(12, 0, (2, 4, 9, 10))
    for r, d in [(3, 1), (5, 2), (7, 1)]:
        p = d * (r - 1) // 2
        wt = np.zeros((4, 4, r, r), dtype=np.float32)
        for k in range(4):
            wt[k, k, r // 2, r // 2] = 1.0
        y, _ = oracle.conv2d(x, wt, None, (1, 1), (p, p), (d, d))
        np.testing.assert_array_equal(y, x.astype(np.float64))
        y2, _ = oracle.conv2d(x, wt, None, (2, 2), (p, p), (d, d))
        np.testing.assert_array_equal(y2, x[:, :, ::2, ::2].astype(np.float64))


# ---------------------------------------------------------------- P4 linearity

def test_linearity_in_x_and_w_exact():
    shp = dict(stride=(2, 1), pad=(1, 2), dil=(1, 2), groups=1)
    x1 = datagen.draw(13, 0, (2, 4, 9, 8), "integer")
    x2 = datagen.draw(14, 0, (2, 4, 9, 8), "integer")
    w1 = datagen.draw(13, 1, (5, 4, 3, 2), "integer")
    w2 = datagen.draw(14, 1, (5, 4, 3, 2), "integer")
    a, b = 3.0, -2.0
    lhs, _ = oracle.conv2d(a * x1 + b * x2, w1, None, **shp)
    r1, _ = oracle.conv2d(x1, w1, None, **shp)
    r2, _ = oracle.conv2d(x2, w1, None, **shp)
    np.testing.assert_array_equal(lhs, a * r1 + b * r2)
    lhs, _ = oracle.conv2d(x1, a * w1 + b * w2, None, **shp)
    r3, _ = oracle.conv2d(x1, w2, None, **shp)
    np.testing.assert_array_equal(lhs, a * r1 + b * r3)


# ---------------------------------------------------------------- P5 groups

@pytest.mark.parametrize("groups", [2, 3, 6])
def test_groups_equal_independent_convs(groups):
    n, c, h, w, k = 2, 6, 10, 9, 12
    x = datagen.draw(15, 0, (n, c, h, w))
    wt = datagen.draw(15, 1, (k, c // groups, 3, 3))
    b = datagen.draw(15, 2, (k,))
    y, a = oracle.conv2d(x, wt, b, (2, 1), (1, 1), (1, 2), groups)
    cg, kg = c // groups, k // groups
    for g in range(groups):
        yg, ag = oracle.conv2d(x[:, g * cg:(g + 1) * cg], wt[g * kg:(g + 1) * kg],
                               b[g * kg:(g + 1) * kg], (2, 1), (1, 1), (1, 2), 1)
        np.testing.assert_array_equal(y[:, g * kg:(g + 1) * kg], yg)
        np.testing.assert_array_equal(a[:, g * kg:(g + 1) * kg], ag)


# ---------------------------------------------------------------- P6 constant data

def _taps_inside(o, stride, pad, dil, ext, size):
    return sum(1 for r in range(ext) if 0 <= o * stride - pad + r * dil < size)


@pytest.mark.parametrize("geom", [
    dict(r=3, s=3, st=(1, 1), pd=(1, 1), dl=(1, 1)),
    dict(r=7, s=7, st=(2, 2), pd=(3, 3), dl=(1, 1)),
    dict(r=5, s=3, st=(2, 3), pd=(4, 2), dl=(2, 1)),
])
def test_constant_data_closed_form(geom):
    n, c, h, w, k, groups = 2, 6, 12, 10, 4, 2
    a_val, beta = 0.75, -1.5
    x = np.full((n, c, h, w), a_val, dtype=np.float32)
    wt = np.full((k, c // groups, geom["r"], geom["s"]), beta, dtype=np.float32)
    b = np.arange(k, dtype=np.float32) - 1.0
    y, _ = oracle.conv2d(x, wt, b, geom["st"], geom["pd"], geom["dl"], groups)
    ho, wo = y.shape[2:]
    for i in range(ho):
        for j in range(wo):
            nr = _taps_inside(i, geom["st"][0], geom["pd"][0], geom["dl"][0], geom["r"], h)
            ns = _taps_inside(j, geom["st"][1], geom["pd"][1], geom["dl"][1], geom["s"], w)
            expect = b.astype(np.float64) + a_val * beta * (c // groups) * nr * ns
            np.testing.assert_array_equal(y[:, :, i, j], np.broadcast_to(expect, (n, k)))


# ---------------------------------------------------------------- P7 bias only

def test_zero_input_gives_bias():
    wt = datagen.draw(16, 1, (5, 3, 3, 3))
    b = datagen.draw(16, 2, (5,))
    y, a = oracle.conv2d(np.zeros((2, 3, 6, 7), np.float32), wt, b, (1, 1), (1, 1))
    np.testing.assert_array_equal(y, np.broadcast_to(b.astype(np.float64)[None, :, None, None],
                                                     y.shape))
    np.testing.assert_array_equal(a, np.abs(y))


# ---------------------------------------------------------------- P8 independent implementations

def _scatter_conv(x, w, b, st, pd, dl, groups):
    """Scatter form: every input pixel pushes its contribution to the outputs it feeds."""
    n, c, h, wd = x.shape
    k, cg, r, s = w.shape
    kg = k // groups
    ho = (h + 2 * pd[0] - dl[0] * (r - 1) - 1) // st[0] + 1
    wo = (wd + 2 * pd[1] - dl[1] * (s - 1) - 1) // st[1] + 1
    y = np.zeros((n, k, ho, wo))
    xd, wdd = x.astype(np.float64), w.astype(np.float64)
    for ci in range(c):
        g = ci // cg
        for hi in range(h):
            for wi in range(wd):
                for rr in range(r):
                    num_h = hi + pd[0] - rr * dl[0]
                    if num_h < 0 or num_h % st[0]:
                        continue
                    oh = num_h // st[0]
                    if oh >= ho:
                        continue
                    for ss in range(s):
                        num_w = wi + pd[1] - ss * dl[1]
                        if num_w < 0 or num_w % st[1]:
                            continue
                        ow = num_w // st[1]
                        if ow >= wo:
                            continue
                        for kk in range(g * kg, (g + 1) * kg):
                            y[:, kk, oh, ow] += xd[:, ci, hi, wi] * wdd[kk, ci - g * cg, rr, ss]
    if b is not None:
        y += b.astype(np.float64)[None, :, None, None]
    return y


TINY = [
    dict(x=(2, 4, 7, 9), w=(6, 2, 3, 2), st=(1, 2), pd=(1, 2), dl=(2, 1), g=2),
    dict(x=(1, 3, 8, 8), w=(5, 3, 3, 3), st=(2, 2), pd=(1, 1), dl=(1, 1), g=1),
    dict(x=(1, 4, 6, 11), w=(4, 1, 5, 3), st=(1, 3), pd=(2, 0), dl=(1, 2), g=4),
    dict(x=(3, 2, 5, 5), w=(3, 2, 1, 4), st=(3, 1), pd=(0, 3), dl=(1, 1), g=1),
    dict(x=(1, 6, 9, 7), w=(9, 2, 2, 3), st=(2, 1), pd=(3, 1), dl=(3, 2), g=3),
]


@pytest.mark.parametrize("t", TINY, ids=[str(i) for i in range(len(TINY))])
def test_tiny_against_scatter_and_torch(t):
    seed = 17 + TINY.index(t)
    x = datagen.draw(seed, 0, t["x"])
    w = datagen.draw(seed, 1, t["w"])
    b = datagen.draw(seed, 2, (t["w"][0],))
    y, a = oracle.conv2d(x, w, b, t["st"], t["pd"], t["dl"], t["g"])
    ys = _scatter_conv(x, w, b, t["st"], t["pd"], t["dl"], t["g"])
    np.testing.assert_allclose(y, ys, rtol=0, atol=1e-12)
    import torch
    yt = torch.nn.functional.conv2d(torch.from_numpy(x.astype(np.float64)),
                                    torch.from_numpy(w.astype(np.float64)),
                                    torch.from_numpy(b.astype(np.float64)), t["st"], t["pd"],
                                    t["dl"], t["g"]).numpy()
    np.testing.assert_allclose(y, yt, rtol=0, atol=1e-12)
    # A is the same sum over |x|, |w|, |b|
    ya, _ = oracle.conv2d(np.abs(x), np.abs(w), np.abs(b), t["st"], t["pd"], t["dl"], t["g"])
    np.testing.assert_array_equal(a, ya)


# ---------------------------------------------------------------- sampled mode, threads

def test_points_match_full_evaluation_and_threads():
    x = datagen.draw(30, 0, (2, 6, 13, 11))
    w = datagen.draw(30, 1, (8, 3, 3, 5))
    b = datagen.draw(30, 2, (8,))
    geom = dict(stride=(2, 1), pad=(1, 2), dil=(1, 1), groups=2)
    y1, a1 = oracle.conv2d(x, w, b, nthreads=1, **geom)
    y8, a8 = oracle.conv2d(x, w, b, nthreads=8, **geom)
    np.testing.assert_array_equal(y1, y8)
    np.testing.assert_array_equal(a1, a8)
    idx = np.array(list(itertools.product(range(2), range(8), range(y1.shape[2]),
                                          range(y1.shape[3]))), dtype=np.int64)
    yp, ap = oracle.conv2d_points(x, w, b, idx, **geom)
    np.testing.assert_array_equal(yp, y1.reshape(-1))
    np.testing.assert_array_equal(ap, a1.reshape(-1))
    with pytest.raises(oracle.OracleError):
        oracle.conv2d_points(x, w, b, np.array([[0, 8, 0, 0]]), **geom)


def test_normalised_error_readings():
    yref = np.array([1.0, -2.0, 0.0])
    a = np.array([2.0, 4.0, 0.0])
    lit, pt = oracle.normalised_errors(np.array([1.5, -2.0, 0.0]), yref, a)
    assert lit == pytest.approx(0.5 / 4.0) and pt == pytest.approx(0.25)
    _, pt = oracle.normalised_errors(np.array([1.0, -2.0, 1e-30]), yref, a)
    assert pt == float("inf")
