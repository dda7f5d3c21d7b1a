"""Pins for the channel-wise, label-weighted signal-product oracle (no GPU needed).

Each weight scales one irrep label.  The tests tie the oracle to the host
library's label index, to products of explicitly isolated labels (one-hot
weights against inputs zeroed by hand from the row layout), to the plain
product on repeated rows, and to rotation equivariance of every channel with
random weights (label (j, l) rotates by D^j)."""
import numpy as np
import pytest

import oracle.istp as oi
import paper_2602_21466_amd as lib
from test_istp_oracle import _complex
from test_oracle import _wigner_D


@pytest.mark.parametrize("spin", [0, 1])
def test_label_index_matches_library(spin):
    for L in (0, 1, 3, 6):
        lab = oi.labels(spin, L)
        assert lib.istp_num_labels(L, spin) == len(lab)
        for k, (j, l) in enumerate(lab):
            assert lib.istp_label_index(spin, j, l) == k
        cols = oi.column_labels(spin, L)
        size = oi.gaunt_size(L) if spin == 0 else oi.vector_size(L)
        assert len(cols) == size and sorted(set(cols)) == list(range(len(lab)))
    assert lib.istp_label_index(1, 0, 0) == -1 and lib.istp_label_index(0, 1, 2) == -1
    assert lib.istp_num_labels(-1, spin) == -1


@pytest.mark.parametrize("spin", [0, 1])
def test_one_hot_weights_isolate_labels(spin, rng):
    """w1, w2, wo one-hot on labels a, b, c: the output is label c of the product of label a of x1 alone
    with label b of x2 alone (inputs zeroed by hand from the row layout), zero elsewhere."""
    L, n, ch = 2, 2, 2
    fn = oi.gaunt_tp if spin == 0 else oi.vector_tp
    size = oi.gaunt_size if spin == 0 else oi.vector_size
    off = (lambda j, l: l * l) if spin == 0 else oi.vector_offset
    lin, lout = oi.labels(spin, L), oi.labels(spin, 2 * L)
    x1 = rng.standard_normal((n, ch, size(L)))
    x2 = rng.standard_normal((n, size(L)))
    for a, b in ((0, len(lin) - 1), (1, 1), (len(lin) - 1, len(lin) // 2)):
        z_iso = None
        for c in range(len(lout)):
            w1 = np.zeros((ch, len(lin))); w1[:, a] = 1
            w2 = np.zeros((ch, len(lin))); w2[:, b] = 1
            wo = np.zeros((ch, len(lout))); wo[:, c] = 1
            got = oi.channel_product(spin, L, x1, x2, w1, w2, wo)
            if z_iso is None:
                (ja, la), (jb, lb) = lin[a], lin[b]
                y1 = np.zeros_like(x1); o = off(ja, la); y1[..., o: o + 2 * ja + 1] = x1[..., o: o + 2 * ja + 1]
                y2 = np.zeros_like(x2); o = off(jb, lb); y2[..., o: o + 2 * jb + 1] = x2[..., o: o + 2 * jb + 1]
                z_iso = np.stack([fn(L, y1[:, k], y2) for k in range(ch)], axis=1)
            jc, lc = lout[c]
            o = off(jc, lc)
            np.testing.assert_allclose(got[..., o: o + 2 * jc + 1], z_iso[..., o: o + 2 * jc + 1], atol=1e-13)
            rest = np.delete(got, np.arange(o, o + 2 * jc + 1), axis=-1)
            assert np.abs(rest).max() == 0.0


def test_shared_input_and_unit_weights(rng):
    """Shared x2 = x2 repeated per channel; unit weights = no weights = the plain product per row."""
    L, n, ch = 3, 3, 4
    x1 = rng.standard_normal((n, ch, oi.vector_size(L)))
    x2 = rng.standard_normal((n, oi.vector_size(L)))
    ones = lambda Lx: np.ones((ch, len(oi.labels(1, Lx))))
    a = oi.channel_product(1, L, x1, x2, ones(L), ones(L), ones(2 * L))
    b = oi.channel_product(1, L, x1, np.repeat(x2[:, None], ch, axis=1))
    np.testing.assert_array_equal(a, b)
    np.testing.assert_allclose(b[2, 1], oi.vector_tp(L, x1[2, 1:2], x2[2:3])[0], atol=1e-14)


@pytest.mark.parametrize("spin", [0, 1])
def test_weighted_channels_are_equivariant(spin, rng):
    """Rotating both inputs (label (j, l) by D^j) rotates every channel's weighted output label by label."""
    from scipy.spatial.transform import Rotation
    L, n, ch = 2, 2, 3
    R = Rotation.random(random_state=int(rng.integers(1 << 30)))
    D = {j: _wigner_D(j, R, rng) for j in range(2 * L + 2)}
    size = oi.gaunt_size if spin == 0 else oi.vector_size
    off = (lambda j, l: l * l) if spin == 0 else oi.vector_offset

    def rot(x, Lx):
        y = np.array(x, dtype=complex)
        for j, l in oi.labels(spin, Lx):
            o = off(j, l)
            y[..., o: o + 2 * j + 1] = x[..., o: o + 2 * j + 1] @ D[j].T
        return y

    x1 = rng.standard_normal((n, ch, size(L)))
    x2 = rng.standard_normal((n, size(L)))
    w1 = rng.standard_normal((n, ch, len(oi.labels(spin, L))))
    w2 = rng.standard_normal((n, ch, len(oi.labels(spin, L))))
    wo = rng.standard_normal((n, ch, len(oi.labels(spin, 2 * L))))
    f = lambda L_, a, b: oi.channel_product(spin, L_, a, b, w1, w2, wo)
    z = f(L, x1, x2)
    zr = _complex(f, L, rot(x1, L), rot(x2, L))
    np.testing.assert_allclose(zr, rot(z, 2 * L), atol=1e-10)


@pytest.mark.parametrize("spin", [0, 1, 2])
def test_weighted_channel_gradients_euler(spin, rng):
    """Bilinearity of the weighted layer: <g, out> = <grad_x1, x1> = <grad_x2, x2>, per (pair, channel)."""
    L, n, ch = 2, 2, 3
    size = oi.spin_size(spin, L)
    x1 = rng.standard_normal((n, ch, size))
    x2 = rng.standard_normal((n, ch, size))
    g = rng.standard_normal((n, ch, oi.spin_size(spin, 2 * L)))
    w1 = rng.standard_normal((ch, len(oi.labels(spin, L))))
    w2 = rng.standard_normal((n, ch, len(oi.labels(spin, L))))
    wo = rng.standard_normal((ch, len(oi.labels(spin, 2 * L))))
    # w1 and wo per channel, w2 per pair: the layer takes one layout, so the per-channel rows are repeated
    out = oi.channel_product(spin, L, x1, x2, np.broadcast_to(w1, (n,) + w1.shape), w2,
                             np.broadcast_to(wo, (n,) + wo.shape))
    g1, g2 = oi.channel_product_vjp(spin, L, x1, x2, g, w1, w2, wo)
    want = (g * out).sum(-1)
    np.testing.assert_allclose((g1 * x1).sum(-1), want, rtol=1e-11)
    np.testing.assert_allclose((g2 * x2).sum(-1), want, rtol=1e-11)
