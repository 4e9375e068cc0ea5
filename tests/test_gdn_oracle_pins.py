"""Pins for the gated-delta-rule oracle (CPU only).

The oracle's fused per-token update is checked against the paper's own form
of the recurrence with an explicit transition matrix (Sec. 2.1:
S_t = S_{t-1} F_t + v_t k_t^T with F_t = a_t (I - beta_t k_t k_t^T) and the
write scaled by beta_t, in the paper's Dv x Dk orientation), against two
closed forms (beta = 0 is pure decay; orthonormal keys with a = beta = 1
overwrite exactly), against central finite differences and a float64 torch
autograd route for every gradient, and against segment composition.
"""
import numpy as np
import pytest
import torch

from oracle import gdn


def rand(rng, B=2, L=23, H=2, Dk=6, Dv=5):
    q = rng.standard_normal((B, L, H, Dk))
    k = rng.standard_normal((B, L, H, Dk))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((B, L, H, Dv))
    g = -np.abs(rng.standard_normal((B, L, H))) * 0.3
    beta = rng.uniform(0.05, 1.0, (B, L, H))
    S_in = rng.standard_normal((B, H, Dk, Dv))
    dO = rng.standard_normal((B, L, H, Dv))
    dS = rng.standard_normal((B, H, Dk, Dv))
    return q, k, v, g, beta, S_in, dO, dS


def paper_form(q, k, v, g, beta, S_in):
    """S^p_t = S^p_{t-1} F_t + beta_t v_t k_t^T, y_t = S^p_t q_t, with S^p = S^T
    (Dv x Dk) and F_t = a_t (I - beta_t k_t k_t^T) built as a matrix.  Also
    returns the corrected values: the token's update beyond the decay,
    S^p_t - a_t S^p_{t-1}, is a rank-one matrix u_t k_t^T, so
    u_t = (S^p_t - a_t S^p_{t-1}) k_t / |k_t|^2."""
    B, L, H, Dk = q.shape
    Dv = v.shape[3]
    o = np.zeros((B, L, H, Dv))
    u = np.zeros((B, L, H, Dv))
    S_out = np.zeros((B, H, Dk, Dv))
    for b in range(B):
        for h in range(H):
            Sp = S_in[b, h].T.copy()
            for t in range(L):
                kt = k[b, t, h]
                a = np.exp(g[b, t, h])
                F = a * (np.eye(Dk) - beta[b, t, h] * np.outer(kt, kt))
                prev = Sp
                Sp = Sp @ F + beta[b, t, h] * np.outer(v[b, t, h], kt)
                o[b, t, h] = Sp @ q[b, t, h]
                u[b, t, h] = (Sp - a * prev) @ kt / (kt @ kt)
            S_out[b, h] = Sp.T
    return o, S_out, u


def test_matches_paper_matrix_form():
    rng = np.random.default_rng(0)
    q, k, v, g, beta, S_in, _, _ = rand(rng)
    o, S, u = gdn.forward(q, k, v, g, beta, S_in, with_u=True)
    ro, rS, ru = paper_form(q, k, v, g, beta, S_in)
    np.testing.assert_allclose(o, ro, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(S, rS, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(u, ru, rtol=1e-10, atol=1e-10)


def test_beta_zero_is_pure_decay():
    rng = np.random.default_rng(1)
    q, k, v, g, beta, S_in, _, _ = rand(rng)
    o, S = gdn.forward(q, k, v, g, np.zeros_like(beta), S_in)
    Bt = np.cumsum(g, axis=1)  # inclusive log-decay
    ref = np.exp(Bt)[..., None] * np.einsum("bhcj,blhc->blhj", S_in, q)
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(S, np.exp(Bt[:, -1])[..., None, None] * S_in, rtol=1e-12)


def test_orthonormal_keys_overwrite_exactly():
    """a = beta = 1 and orthonormal keys: each token removes the state's
    component along k_i and writes v_i there, so
    S_L = (I - sum k_i k_i^T) S_in + sum k_i v_i^T."""
    rng = np.random.default_rng(2)
    Dk, Dv, L = 8, 5, 6
    Q, _ = np.linalg.qr(rng.standard_normal((Dk, Dk)))
    k = Q[:, :L].T.reshape(1, L, 1, Dk)
    v = rng.standard_normal((1, L, 1, Dv))
    q = rng.standard_normal((1, L, 1, Dk))
    S_in = rng.standard_normal((1, 1, Dk, Dv))
    _, S, u = gdn.forward(q, k, v, np.zeros((1, L, 1)), np.ones((1, L, 1)), S_in, with_u=True)
    K = k[0, :, 0]
    ref = (np.eye(Dk) - K.T @ K) @ S_in[0, 0] + K.T @ v[0, :, 0]
    np.testing.assert_allclose(S[0, 0], ref, rtol=1e-12, atol=1e-12)
    # each corrected value replaces the state's old content along k_i: v_i - S_in^T k_i
    np.testing.assert_allclose(u[0, :, 0], v[0, :, 0] - K @ S_in[0, 0], rtol=1e-12, atol=1e-12)


def loss(q, k, v, g, beta, S_in, dO, dS):
    o, S = gdn.forward(q, k, v, g, beta, S_in)
    return float((o * dO).sum() + (S * dS).sum())


def test_gradients_finite_differences():
    rng = np.random.default_rng(3)
    args = list(rand(rng, B=1, L=9, H=1, Dk=4, Dv=3))
    q, k, v, g, beta, S_in, dO, dS = args
    grads = gdn.backward(q, k, v, g, beta, S_in, dO, dS)
    names = ["q", "k", "v", "g", "beta", "S_in"]
    h = 1e-6
    for ai, name in enumerate(names):
        x, gx = args[ai], grads[ai]
        for idx in [tuple(rng.integers(0, s) for s in x.shape) for _ in range(4)]:
            p, m = list(args), list(args)
            p[ai] = x.copy()
            m[ai] = x.copy()
            p[ai][idx] += h
            m[ai][idx] -= h
            fd = (loss(*p) - loss(*m)) / (2 * h)
            assert abs(fd - gx[idx]) <= 1e-6 * max(1.0, abs(fd)), (name, idx, fd, gx[idx])


def test_gradients_match_autograd_route():
    rng = np.random.default_rng(4)
    q, k, v, g, beta, S_in, dO, dS = rand(rng, B=1, L=17, H=2, Dk=5, Dv=4)
    T = [torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (q, k, v, g, beta, S_in)]
    tq, tk, tv, tg, tb, tS = T
    os_, S_fin = [], []
    for h in range(2):
        S = tS[0, h]
        outs = []
        for t in range(17):
            a = torch.exp(tg[0, t, h])
            P = a * S
            u = tb[0, t, h] * (tv[0, t, h] - P.T @ tk[0, t, h])
            S = P + torch.outer(tk[0, t, h], u)
            outs.append(S.T @ tq[0, t, h])
        os_.append(torch.stack(outs))
        S_fin.append(S)
    o = torch.stack(os_, dim=1).unsqueeze(0)
    S_out = torch.stack(S_fin).unsqueeze(0)
    L_ = (o * torch.tensor(dO)).sum() + (S_out * torch.tensor(dS)).sum()
    L_.backward()
    grads = gdn.backward(q, k, v, g, beta, S_in, dO, dS)
    for t, gr in zip(T, grads):
        np.testing.assert_allclose(gr, t.grad.numpy(), rtol=1e-10, atol=1e-10)


@pytest.mark.parametrize("cut", [1, 11])
def test_segment_composition(cut):
    rng = np.random.default_rng(5 + cut)
    q, k, v, g, beta, S_in, dO, dS = rand(rng)
    o, S = gdn.forward(q, k, v, g, beta, S_in)
    sl1, sl2 = slice(0, cut), slice(cut, None)
    o1, S1 = gdn.forward(q[:, sl1], k[:, sl1], v[:, sl1], g[:, sl1], beta[:, sl1], S_in)
    o2, S2 = gdn.forward(q[:, sl2], k[:, sl2], v[:, sl2], g[:, sl2], beta[:, sl2], S1)
    np.testing.assert_allclose(np.concatenate([o1, o2], 1), o, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(S2, S, rtol=1e-12, atol=1e-12)
    full = gdn.backward(q, k, v, g, beta, S_in, dO, dS)
    b2 = gdn.backward(q[:, sl2], k[:, sl2], v[:, sl2], g[:, sl2], beta[:, sl2], S1, dO[:, sl2], dS)
    b1 = gdn.backward(q[:, sl1], k[:, sl1], v[:, sl1], g[:, sl1], beta[:, sl1], S_in, dO[:, sl1], b2[5])
    for i in range(5):
        np.testing.assert_allclose(np.concatenate([b1[i], b2[i]], 1), full[i], rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(b1[5], full[5], rtol=1e-11, atol=1e-11)
