"""The algebra behind the token-reference layout of the fwd+bwd call, in fp64 on the CPU.

Without an entropy term the logit gradient of the masked clipped surrogate (Sec. 2.3.1, 2.3.2) is
dz_tj = g_t ([j = y_t] - p_tj), p = softmax(z).  The GPU path stores q_tj = exp(z_tj - r_t) against
the token's target logit r_t = z_{t,y_t}, replaces the target entry by expm1(logp_t) exp(lse_t - r_t)
and applies the row scale s_t = -g_t exp(r_t - lse_t), i.e. it relies on dz = diag(s) q.  A tile whose
maximum lies more than a span above r_t stores against c = m_tile - span instead, and the explicit
pass then forms dz_tj = -g_t exp(c - lse_t) q_tj away from the target.  The online log-softmax merges
per-tile partials (c_k, sum_j exp(z_j - c_k)) taken against any reference.  These tests check the
three statements against the plain definitions; they use no kernel and no oracle code.
"""
import numpy as np
import pytest

SPAN = 40.0   # the forward's clamp span, in nats
TILE = 256    # vocabulary entries per forward tile


def _instance(seed, T=24, V=1000, scale=1.3):
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((T, V)) * scale
    y = rng.integers(0, V, T)
    g = rng.standard_normal(T) * 1e-3
    g[::5] = 0.0                                 # clipped tokens
    return z, y, g


def _softmax_terms(z):
    m = z.max(axis=1, keepdims=True)
    lse = (m + np.log(np.exp(z - m).sum(axis=1, keepdims=True)))[:, 0]
    return lse, np.exp(z - lse[:, None])


def _dz_definition(z, y, g):
    _, p = _softmax_terms(z)
    onehot = np.zeros_like(z)
    onehot[np.arange(z.shape[0]), y] = 1.0
    return g[:, None] * (onehot - p)


@pytest.mark.parametrize("seed,scale", [(1, 1.3), (2, 4.0), (3, 0.05)])
def test_row_scaled_q_is_the_logit_gradient(seed, scale):
    z, y, g = _instance(seed, scale=scale)
    T = z.shape[0]
    lse, _ = _softmax_terms(z)
    r = z[np.arange(T), y]
    logp = r - lse
    q = np.exp(z - r[:, None])
    q[np.arange(T), y] = np.expm1(logp) * np.exp(lse - r)
    s = -g * np.exp(r - lse)
    np.testing.assert_allclose(s[:, None] * q, _dz_definition(z, y, g), rtol=1e-12, atol=1e-18)


def test_clamped_tile_references_give_the_same_gradient_through_the_explicit_pass():
    # one token per row whose target sits far below its largest logit, so that tiles clamp
    z, y, g = _instance(4, V=4 * TILE, scale=1.0)
    T, V = z.shape
    z[:, 3 * TILE + 7] += 80.0                   # a dominant entry in the last tile of every row
    lse, _ = _softmax_terms(z)
    r = z[np.arange(T), y]
    clamped = 0
    dz = np.empty_like(z)
    for k in range(V // TILE):
        sl = slice(k * TILE, (k + 1) * TILE)
        m = z[:, sl].max(axis=1)
        c = np.maximum(r, m - SPAN)
        clamped += int((r < m - SPAN).sum())
        q = np.exp(z[:, sl] - c[:, None])
        dz[:, sl] = -g[:, None] * np.exp(c - lse)[:, None] * q
    dz[np.arange(T), y] = -g * np.expm1(r - lse)  # the target entry from the exact log-prob
    assert clamped > 0
    np.testing.assert_allclose(dz, _dz_definition(z, y, g), rtol=1e-10, atol=1e-18)


def test_partials_against_any_reference_merge_to_the_log_partition():
    z, y, _ = _instance(5, V=5 * TILE, scale=3.0)
    T, V = z.shape
    lse, p = _softmax_terms(z)
    r = z[np.arange(T), y]
    refs, sums, ents = [], [], []
    for k in range(V // TILE):
        sl = slice(k * TILE, (k + 1) * TILE)
        c = np.maximum(r, z[:, sl].max(axis=1) - SPAN)
        e = np.exp(z[:, sl] - c[:, None])
        refs.append(c)
        sums.append(e.sum(axis=1))
        ents.append((e * (z[:, sl] - c[:, None])).sum(axis=1))
    C, S, U = np.array(refs), np.array(sums), np.array(ents)
    M = C.max(axis=0)
    w = np.exp(C - M)
    Stot = (w * S).sum(axis=0)
    Ttot = (w * (U + (C - M) * S)).sum(axis=0)
    np.testing.assert_allclose(M + np.log(Stot), lse, rtol=1e-13)
    H = -(p * np.log(p)).sum(axis=1)
    np.testing.assert_allclose(-(Ttot / Stot - np.log(Stot)), H, rtol=1e-11)
