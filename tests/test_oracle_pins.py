"""Pins for the fp64 oracle (CPU only).

Each test checks the oracle against something other than itself: a hand-worked
example, the O(L^2) closed form of the recurrence, textbook causal linear
attention, closed forms of the boundary state and boundary gradient, central
finite differences, an independent autograd route, and the exact segment
composition that StateFlow's chunking relies on (paper Sec. 3.1 chaining
equations; Sec. 4.1 exactness).  A dropped term, a wrong sign, an off-by-one in
the decay or a transposed operand in the oracle fails at least one of them.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def rand_inputs(rng, B, L, H, Dk, Dv, vec=False, s_in=True, gscale=1.0):
    q = rng.standard_normal((B, L, H, Dk))
    k = rng.standard_normal((B, L, H, Dk))
    v = rng.standard_normal((B, L, H, Dv))
    gshape = (B, L, H, Dk) if vec else (B, L, H)
    g = -gscale * np.abs(rng.standard_normal(gshape)) - 0.01
    S_in = rng.standard_normal((B, H, Dk, Dv)) if s_in else None
    dO = rng.standard_normal((B, L, H, Dv))
    dS_out = rng.standard_normal((B, H, Dk, Dv))
    return q, k, v, g, S_in, dO, dS_out


# ---------------------------------------------------------------- closed forms
def brute_force_o(q, k, v, g, S_in):
    """o_t = sum_c q_t[c] e^{B_t[c]} S_in[c,:] + sum_{s<=t} (sum_c q_t[c] k_s[c]
    e^{B_t[c]-B_s[c]}) v_s with B the inclusive cumulative log-decay: the
    recurrence unrolled, one (t, s) pair at a time."""
    B, L, H, Dk = q.shape
    Dv = v.shape[3]
    vec = g.ndim == 4
    o = np.zeros((B, L, H, Dv))
    for b in range(B):
        for h in range(H):
            gg = g[b, :, h] if vec else np.repeat(g[b, :, h][:, None], Dk, axis=1)
            Bc = np.cumsum(gg, axis=0)  # [L, Dk]
            for t in range(L):
                acc = np.zeros(Dv)
                if S_in is not None:
                    acc += (q[b, t, h] * np.exp(Bc[t])) @ S_in[b, h]
                for s in range(t + 1):
                    w = np.sum(q[b, t, h] * k[b, s, h] * np.exp(Bc[t] - Bc[s]))
                    acc += w * v[b, s, h]
                o[b, t, h] = acc
    return o


def closed_form_S_out(k, v, g, S_in):
    """S_out = e^{B_L} o S_in + sum_s e^{B_L - B_s} o k_s v_s^T."""
    B, L, H, Dk = k.shape
    Dv = v.shape[3]
    vec = g.ndim == 4
    S = np.zeros((B, H, Dk, Dv))
    for b in range(B):
        for h in range(H):
            gg = g[b, :, h] if vec else np.repeat(g[b, :, h][:, None], Dk, axis=1)
            Bc = np.cumsum(gg, axis=0)
            tot = Bc[-1]
            acc = np.zeros((Dk, Dv))
            if S_in is not None:
                acc += np.exp(tot)[:, None] * S_in[b, h]
            for s in range(L):
                acc += np.exp(tot - Bc[s])[:, None] * np.outer(k[b, s, h], v[b, s, h])
            S[b, h] = acc
    return S


def closed_form_dS_in(q, g, dO, dS_out):
    """dS_in = e^{B_L} o dS_out + sum_t e^{B_t} o q_t dO_t^T."""
    B, L, H, Dk = q.shape
    Dv = dO.shape[3]
    vec = g.ndim == 4
    G = np.zeros((B, H, Dk, Dv))
    for b in range(B):
        for h in range(H):
            gg = g[b, :, h] if vec else np.repeat(g[b, :, h][:, None], Dk, axis=1)
            Bc = np.cumsum(gg, axis=0)
            acc = np.exp(Bc[-1])[:, None] * dS_out[b, h]
            for t in range(L):
                acc += np.exp(Bc[t])[:, None] * np.outer(q[b, t, h], dO[b, t, h])
            G[b, h] = acc
    return G


def loss(q, k, v, g, S_in, dO, dS_out):
    o, S_out, _ = oracle.forward(q, k, v, g, S_in)
    return float(np.sum(o * dO) + np.sum(S_out * dS_out))


# ----------------------------------------------------------------------- tests
def test_hand_worked_example():
    with open(os.path.join(HERE, "golden", "hand_example.json")) as f:
        ex = json.load(f)
    inp, exp = ex["inputs"], ex["expected"]
    q = np.array(inp["q"], float)[None, :, None, :]
    k = np.array(inp["k"], float)[None, :, None, :]
    v = np.array(inp["v"], float)[None, :, None, :]
    g = np.log(np.array(inp["a"], float))[None, :, None]
    S_in = np.array(inp["S_in"], float)[None, None]
    dO = np.array(inp["dO"], float)[None, :, None, :]
    dS_out = np.array(inp["dS_out"], float)[None, None]
    o, S_out, _ = oracle.forward(q, k, v, g, S_in)
    dq, dk, dv, dg, dS_in = oracle.backward(q, k, v, g, S_in, dO, dS_out)
    tol = dict(rtol=0, atol=1e-12)
    np.testing.assert_allclose(o[0, :, 0], exp["o"], **tol)
    np.testing.assert_allclose(S_out[0, 0], exp["S_out"], **tol)
    np.testing.assert_allclose(dq[0, :, 0], exp["dq"], **tol)
    np.testing.assert_allclose(dk[0, :, 0], exp["dk"], **tol)
    np.testing.assert_allclose(dv[0, :, 0], exp["dv"], **tol)
    np.testing.assert_allclose(dg[0, :, 0], exp["dg"], **tol)
    np.testing.assert_allclose(dS_in[0, 0], exp["dS_in"], **tol)


@pytest.mark.parametrize("vec", [False, True])
def test_forward_matches_bruteforce(vec):
    rng = np.random.default_rng(1)
    q, k, v, g, S_in, _, _ = rand_inputs(rng, 2, 37, 2, 5, 3, vec=vec)
    o, S_out, _ = oracle.forward(q, k, v, g, S_in)
    np.testing.assert_allclose(o, brute_force_o(q, k, v, g, S_in), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(S_out, closed_form_S_out(k, v, g, S_in), rtol=1e-11, atol=1e-11)


def test_zero_gate_is_causal_linear_attention():
    """g = 0, S_in = 0: o = tril(Q K^T) V, the textbook causal linear attention."""
    rng = np.random.default_rng(2)
    q, k, v, g, _, _, _ = rand_inputs(rng, 1, 50, 3, 6, 4, s_in=False)
    g = np.zeros_like(g)
    o, S_out, _ = oracle.forward(q, k, v, g, None)
    for h in range(3):
        Q, K, V = q[0, :, h], k[0, :, h], v[0, :, h]
        np.testing.assert_allclose(o[0, :, h], np.tril(Q @ K.T) @ V, rtol=1e-11, atol=1e-11)
        np.testing.assert_allclose(S_out[0, h], K.T @ V, rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("vec", [False, True])
def test_dS_in_closed_form(vec):
    rng = np.random.default_rng(3)
    q, k, v, g, S_in, dO, dS_out = rand_inputs(rng, 1, 29, 2, 4, 5, vec=vec)
    *_, dS_in = oracle.backward(q, k, v, g, S_in, dO, dS_out)
    np.testing.assert_allclose(dS_in, closed_form_dS_in(q, g, dO, dS_out), rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("vec", [False, True])
def test_gradients_finite_differences(vec):
    rng = np.random.default_rng(4)
    q, k, v, g, S_in, dO, dS_out = rand_inputs(rng, 1, 6, 1, 3, 2, vec=vec)
    grads = oracle.backward(q, k, v, g, S_in, dO, dS_out)
    args = [q, k, v, g, S_in]
    h = 1e-6
    for idx, (x, gx) in enumerate(zip(args, grads)):
        fd = np.zeros_like(x)
        for e in np.ndindex(x.shape):
            xp = x.copy(); xp[e] += h
            xm = x.copy(); xm[e] -= h
            ap = list(args); ap[idx] = xp
            am = list(args); am[idx] = xm
            fd[e] = (loss(*ap, dO, dS_out) - loss(*am, dO, dS_out)) / (2 * h)
        np.testing.assert_allclose(gx, fd, rtol=1e-6, atol=1e-7, err_msg=f"input {idx}")


@pytest.mark.parametrize("vec", [False, True])
def test_gradients_match_autograd_route(vec):
    """A separate token loop in torch float64, differentiated by autograd."""
    rng = np.random.default_rng(5)
    B, L, H, Dk, Dv = 2, 40, 2, 8, 6
    q, k, v, g, S_in, dO, dS_out = rand_inputs(rng, B, L, H, Dk, Dv, vec=vec)
    T = [torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (q, k, v, g, S_in)]
    tq, tk, tv, tg, tS = T
    total = 0.0
    S = tS.clone()
    for t in range(L):
        a = torch.exp(tg[:, t])  # [B,H] or [B,H,Dk]
        a = a[..., :, None] if vec else a[..., None, None]
        S = a * S + tk[:, t, :, :, None] * tv[:, t, :, None, :]
        o_t = torch.einsum("bhkv,bhk->bhv", S, tq[:, t])
        total = total + (o_t * torch.tensor(dO[:, t])).sum()
    total = total + (S * torch.tensor(dS_out)).sum()
    total.backward()
    ours = oracle.backward(q, k, v, g, S_in, dO, dS_out)
    for t_, mine in zip(T, ours):
        np.testing.assert_allclose(mine, t_.grad.numpy(), rtol=1e-10, atol=1e-10)


@pytest.mark.parametrize("vec", [False, True])
def test_segment_composition(vec):
    """Fwd(A) then Fwd(B) with S_in(B) = S_out(A) equals Fwd(AB); Bwd(B) then
    Bwd(A) with dS_out(A) = dS_in(B) equals Bwd(AB)  (Sec. 3.1 chaining)."""
    rng = np.random.default_rng(6)
    L = 45
    q, k, v, g, S_in, dO, dS_out = rand_inputs(rng, 2, L, 2, 4, 3, vec=vec)
    o_all, S_all, snaps = oracle.forward(q, k, v, g, S_in, snap_pos=[0, 1, 17, 44, 45])
    full = oracle.backward(q, k, v, g, S_in, dO, dS_out)
    for cuts in ([1], [17], [44], [1, 17, 44], [3, 4, 5, 30]):
        bounds = [0] + cuts + [L]
        S = S_in
        outs = []
        states = [S_in]
        for a, b in zip(bounds[:-1], bounds[1:]):
            sl = slice(a, b)
            o, S, _ = oracle.forward(q[:, sl], k[:, sl], v[:, sl], g[:, sl], S)
            outs.append(o)
            states.append(S)
        np.testing.assert_allclose(np.concatenate(outs, axis=1), o_all, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(S, S_all, rtol=1e-12, atol=1e-12)
        # backward, segments in reverse with dS chaining
        G = dS_out
        parts = [None] * (len(bounds) - 1)
        for i in reversed(range(len(bounds) - 1)):
            sl = slice(bounds[i], bounds[i + 1])
            dq, dk, dv, dg, G = oracle.backward(q[:, sl], k[:, sl], v[:, sl], g[:, sl], states[i],
                                                dO[:, sl], G)
            parts[i] = (dq, dk, dv, dg)
        for j in range(4):
            np.testing.assert_allclose(np.concatenate([p[j] for p in parts], axis=1), full[j],
                                       rtol=1e-11, atol=1e-11)
        np.testing.assert_allclose(G, full[4], rtol=1e-11, atol=1e-11)
    for p, pos in enumerate([0, 1, 17, 44, 45]):
        _, S_ref, _ = oracle.forward(q[:, :pos], k[:, :pos], v[:, :pos], g[:, :pos], S_in)
        np.testing.assert_allclose(snaps[p], S_ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("vec", [False, True])
def test_dg_cumulative_identity(vec):
    """dg_t = sum_{t'>=t} (q o dq - k o dk)_{t'} + <dS_out, S_out>: the gradient of
    the cumulative log-decay telescopes (independent of the oracle's
    a_t <G, S_{t-1}> route)."""
    rng = np.random.default_rng(7)
    q, k, v, g, S_in, dO, dS_out = rand_inputs(rng, 1, 33, 2, 5, 4, vec=vec)
    _, S_out, _ = oracle.forward(q, k, v, g, S_in)
    dq, dk, dv, dg, _ = oracle.backward(q, k, v, g, S_in, dO, dS_out)
    if vec:
        ell = q * dq - k * dk                                   # [B,L,H,Dk]
        tail = np.sum(dS_out * S_out, axis=3)                   # [B,H,Dk]
    else:
        ell = np.sum(q * dq - k * dk, axis=3)                   # [B,L,H]
        tail = np.sum(dS_out * S_out, axis=(2, 3))              # [B,H]
    suffix = np.flip(np.cumsum(np.flip(ell, axis=1), axis=1), axis=1)
    np.testing.assert_allclose(dg, suffix + tail[:, None], rtol=1e-10, atol=1e-10)


def test_single_token():
    rng = np.random.default_rng(8)
    q, k, v, g, S_in, _, _ = rand_inputs(rng, 1, 1, 1, 4, 3)
    o, S_out, _ = oracle.forward(q, k, v, g, S_in)
    S_ref = np.exp(g[0, 0, 0]) * S_in[0, 0] + np.outer(k[0, 0, 0], v[0, 0, 0])
    np.testing.assert_allclose(S_out[0, 0], S_ref, rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(o[0, 0, 0], S_ref.T @ q[0, 0, 0], rtol=1e-14, atol=1e-14)


def test_memoryless_gate():
    """a_t = 0 (g -> -inf): each token sees only itself, o_t = (q_t . k_t) v_t."""
    rng = np.random.default_rng(9)
    q, k, v, g, S_in, _, _ = rand_inputs(rng, 1, 20, 2, 4, 3)
    g = np.full_like(g, -1e4)
    o, _, _ = oracle.forward(q, k, v, g, S_in)
    ref = np.sum(q * k, axis=3, keepdims=True) * v
    np.testing.assert_allclose(o, ref, rtol=1e-13, atol=1e-13)


def test_linearity_in_v_and_state():
    rng = np.random.default_rng(10)
    q, k, v1, g, S1, _, _ = rand_inputs(rng, 1, 25, 2, 4, 3)
    v2 = rng.standard_normal(v1.shape)
    S2 = rng.standard_normal(S1.shape)
    o1, _, _ = oracle.forward(q, k, v1, g, S1)
    o2, _, _ = oracle.forward(q, k, v2, g, S2)
    o12, _, _ = oracle.forward(q, k, v1 + 2 * v2, g, S1 + 2 * S2)
    np.testing.assert_allclose(o12, o1 + 2 * o2, rtol=1e-12, atol=1e-12)


def test_empty_sequence():
    rng = np.random.default_rng(11)
    q, k, v, g, S_in, dO, dS_out = rand_inputs(rng, 1, 0, 2, 4, 3)
    _, S_out, _ = oracle.forward(q, k, v, g, S_in)
    np.testing.assert_array_equal(S_out, S_in)
    *_, dS_in = oracle.backward(q, k, v, g, S_in, dO, dS_out)
    np.testing.assert_array_equal(dS_in, dS_out)
