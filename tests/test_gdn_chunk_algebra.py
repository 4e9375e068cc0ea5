"""The chunk algebra behind the gated-delta-rule kernels, written out in fp64
numpy and checked against the token-level oracle (CPU only).

Per chunk of C tokens with state S entering it (b: chunk-local inclusive
log-decay, gamma = e^b):
  A = tril(beta_t e^{b_t - b_s} k_t.k_s, -1),  T = (I + A)^{-1}
  W = T diag(beta gamma) K,  Ubar = T diag(beta) V,  U = Ubar - W S
  O = diag(gamma) Q S + (Q K^T o Gamma) U,   S' = gamma_C S + (e^{b_C - b} o K)^T U
U is the V^new of the delta rule.  T is formed the way the kernels form it:
16 x 16 diagonal blocks by substitution, then T_ij = -T_ii sum_k A_ik T_kj
level by level.  A chunk's map is affine in S, so a run of chunks maps
S -> M S + N (the superchunk summary, Sec. 2.2's Pre for a matrix-valued
transition), and the state gradient goes back through M^T:
dS_start = M^T dS_end + E.  The backward per chunk is the one the per-chunk
gradient kernel evaluates.
"""
import numpy as np
import pytest

from oracle import gdn

C = 64  # the kernels' chunk


def rand(rng, L, Dk=8, Dv=6):
    q = rng.standard_normal((L, Dk))
    k = rng.standard_normal((L, Dk))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((L, Dv))
    g = np.log(1 / (1 + np.exp(-(rng.standard_normal(L) + 2.0))))
    beta = 1 / (1 + np.exp(-rng.standard_normal(L)))
    S0 = 0.3 * rng.standard_normal((Dk, Dv))
    return q, k, v, g, beta, S0


def tinv_blocked(A, blk=16):
    """(I + A)^{-1} for strictly lower A: diagonal blocks by substitution, then
    the off-diagonal blocks by level."""
    n = A.shape[0]
    nb = n // blk
    T = np.zeros_like(A)
    for i in range(nb):
        o = slice(i * blk, (i + 1) * blk)
        T[o, o] = np.linalg.solve(np.eye(blk) + A[o, o], np.eye(blk))
    for d in range(1, nb):
        for i in range(d, nb):
            j = i - d
            oi, oj = slice(i * blk, (i + 1) * blk), slice(j * blk, (j + 1) * blk)
            Y = sum(A[oi, k * blk:(k + 1) * blk] @ T[k * blk:(k + 1) * blk, oj] for k in range(j, i))
            T[oi, oj] = -T[oi, oi] @ Y
    return T


def chunk_parts(q, k, v, g, beta):
    b = np.cumsum(g)
    gam = np.exp(b)
    Gam = np.tril(np.exp(b[:, None] - b[None, :]))
    A = beta[:, None] * np.tril(np.exp(b[:, None] - b[None, :]) * (k @ k.T), -1)
    T = tinv_blocked(A)
    W = T @ ((beta * gam)[:, None] * k)
    Ub = T @ (beta[:, None] * v)
    P = (q @ k.T) * Gam
    se = np.exp(b[-1] - b)
    return dict(b=b, gam=gam, A=A, T=T, W=W, Ub=Ub, P=P, se=se)


def chunk_fwd(q, k, v, g, beta, S):
    c = chunk_parts(q, k, v, g, beta)
    U = c["Ub"] - c["W"] @ S
    O = c["gam"][:, None] * (q @ S) + c["P"] @ U
    Sn = c["gam"][-1] * S + (c["se"][:, None] * k).T @ U
    return O, Sn, U


def chunk_bwd(q, k, v, g, beta, S, dO, dSn):
    c = chunk_parts(q, k, v, g, beta)
    b, gam, A, T, W, Ub, P, se = (c[x] for x in ("b", "gam", "A", "T", "W", "Ub", "P", "se"))
    n = len(g)
    Ge = np.exp(b[:, None] - b[None, :])
    U = Ub - W @ S
    dU = se[:, None] * (k @ dSn) + P.T @ dO
    dS = gam[-1] * dSn + q.T @ (gam[:, None] * dO) - W.T @ dU
    dW = -dU @ S.T
    GW, GU = T.T @ dW, T.T @ dU
    dA = np.tril(-(GW @ W.T + GU @ Ub.T), -1)
    Ah = dA * beta[:, None] * Ge * np.tri(n, k=-1)
    dP = np.tril(dO @ U.T)
    dq = gam[:, None] * (dO @ S.T) + (dP * Ge) @ k
    dKt = U @ dSn.T
    dk = se[:, None] * dKt + (dP * Ge).T @ q + (beta * gam)[:, None] * GW + (Ah + Ah.T) @ k
    dv = beta[:, None] * GU
    KK = np.tril(Ge * (k @ k.T), -1)
    dbeta = gam * np.sum(GW * k, 1) + np.sum(GU * v, 1) + np.sum(dA * KK, 1)
    db = gam * np.sum(q * (dO @ S.T), 1)                       # through gamma in Q S
    E = dP * P
    db += E.sum(1) - E.sum(0)                                   # through Gamma
    db += beta * gam * np.sum(GW * k, 1)                        # through gamma in W
    EA = dA * A
    db += EA.sum(1) - EA.sum(0)                                 # through A
    r = se * np.sum(dKt * k, 1)                                 # through e^{b_C - b}
    db -= r
    db[-1] += r.sum() + gam[-1] * np.sum(dSn * S)               # through b_C
    dg = np.cumsum(db[::-1])[::-1]
    return dq, dk, dv, dg, dbeta, dS


def oracle(q, k, v, g, beta, S0, dO=None, dS=None):
    r = lambda x: x[None, :, None]
    o, S, u = gdn.forward(r(q), r(k), r(v), g[None, :, None], beta[None, :, None], S0[None, None], with_u=True)
    out = (o[0, :, 0], S[0, 0], u[0, :, 0])
    if dO is None:
        return out
    gr = gdn.backward(r(q), r(k), r(v), g[None, :, None], beta[None, :, None], S0[None, None], r(dO), dS[None, None])
    return out, [x[0, :, 0] for x in gr[:5]] + [gr[5][0, 0]]


def test_blocked_inverse():
    rng = np.random.default_rng(0)
    A = np.tril(rng.standard_normal((64, 64)) * 0.3, -1)
    np.testing.assert_allclose(tinv_blocked(A) @ (np.eye(64) + A), np.eye(64), atol=1e-10)


@pytest.mark.parametrize("L", [C, 5 * C])
def test_chunk_forward_and_v_new(L):
    rng = np.random.default_rng(L)
    q, k, v, g, beta, S0 = rand(rng, L)
    ro, rS, ru = oracle(q, k, v, g, beta, S0)
    S, outs, us = S0, [], []
    for c in range(L // C):
        sl = slice(c * C, (c + 1) * C)
        O, S, U = chunk_fwd(q[sl], k[sl], v[sl], g[sl], beta[sl], S)
        outs.append(O)
        us.append(U)
    np.testing.assert_allclose(np.concatenate(outs), ro, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(np.concatenate(us), ru, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(S, rS, rtol=1e-10, atol=1e-10)


def test_chunk_backward():
    rng = np.random.default_rng(7)
    L = 4 * C
    q, k, v, g, beta, S0 = rand(rng, L)
    dO = rng.standard_normal(v.shape)
    dSo = rng.standard_normal(S0.shape)
    _, ref = oracle(q, k, v, g, beta, S0, dO, dSo)
    states, S = [], S0
    for c in range(L // C):
        sl = slice(c * C, (c + 1) * C)
        states.append(S)
        _, S, _ = chunk_fwd(q[sl], k[sl], v[sl], g[sl], beta[sl], S)
    dS, parts = dSo, []
    for c in reversed(range(L // C)):
        sl = slice(c * C, (c + 1) * C)
        *gr, dS = chunk_bwd(q[sl], k[sl], v[sl], g[sl], beta[sl], states[c], dO[sl], dS)
        parts.insert(0, gr)
    for i, name in enumerate(("dq", "dk", "dv", "dg", "dbeta")):
        np.testing.assert_allclose(np.concatenate([p[i] for p in parts]), ref[i], rtol=1e-9, atol=1e-9,
                                   err_msg=name)
    np.testing.assert_allclose(dS, ref[5], rtol=1e-9, atol=1e-9)


def test_superchunk_affine_maps():
    """A run of chunks maps S to M S + N, with M the walk from the identity
    with Ubar = 0 and N the walk from zero; the state gradient goes back as
    dS_start = M^T dS_end + E, with E the backward walk from dS_end = 0."""
    rng = np.random.default_rng(11)
    L, Dk = 3 * C, 8
    q, k, v, g, beta, S0 = rand(rng, L, Dk=Dk)
    dO = rng.standard_normal(v.shape)
    dSend = rng.standard_normal(S0.shape)

    def walk(S, zero_ubar=False):
        for c in range(L // C):
            sl = slice(c * C, (c + 1) * C)
            p = chunk_parts(q[sl], k[sl], v[sl], g[sl], beta[sl])
            U = (0 if zero_ubar else p["Ub"]) - p["W"] @ S
            S = p["gam"][-1] * S + (p["se"][:, None] * k[sl]).T @ U
        return S

    M = walk(np.eye(Dk), zero_ubar=True)
    N = walk(np.zeros_like(S0))
    np.testing.assert_allclose(M @ S0 + N, walk(S0), rtol=1e-12, atol=1e-12)

    def back(dS, S_start, with_do=True):
        states, S = [], S_start
        for c in range(L // C):
            sl = slice(c * C, (c + 1) * C)
            states.append(S)
            _, S, _ = chunk_fwd(q[sl], k[sl], v[sl], g[sl], beta[sl], S)
        for c in reversed(range(L // C)):
            sl = slice(c * C, (c + 1) * C)
            dO_c = dO[sl] if with_do else np.zeros_like(dO[sl])
            dS = chunk_bwd(q[sl], k[sl], v[sl], g[sl], beta[sl], states[c], dO_c, dS)[5]
        return dS

    E = back(np.zeros_like(dSend), S0)
    np.testing.assert_allclose(M.T @ dSend + E, back(dSend, S0), rtol=1e-12, atol=1e-12)
    # the state gradient does not depend on the forward state (the map is affine)
    np.testing.assert_allclose(back(dSend, np.zeros_like(S0)), back(dSend, S0), rtol=1e-12, atol=1e-12)


def chunk_bwd_vblocks(q, k, v, g, beta, S, dO, dSn, vb=2):
    """The per-chunk gradients as the per-chunk kernel forms them: the value
    channels in blocks of vb columns, each block of S and dS' read once.
    Two identities remove the W and Ubar products of chunk_bwd:
      G_W = T^T (-dU S^T) = -G_U S^T,
      dA  = -(G_W W^T + G_U Ubar^T) = -G_U (Ubar - W S)^T = -G_U U^T.
    Per block b (columns J of v): U_J = Ubar_J - W S_J, dU_J = e o K dS'_J +
    P^T dO_J, G_U,J = T^T dU_J (so dv_J = beta o G_U,J); the v-contractions
    G_W, dO S^T, U dS'^T, dA and dP = dO U^T accumulate over the blocks."""
    c = chunk_parts(q, k, v, g, beta)
    b, gam, A, T, W, P, se = (c[x] for x in ("b", "gam", "A", "T", "W", "P", "se"))
    n, Dk = k.shape
    Dv = v.shape[1]
    Ge = np.exp(b[:, None] - b[None, :])
    KK = np.tril(Ge * (k @ k.T), -1)
    GW, dqS, dkS = np.zeros((n, Dk)), np.zeros((n, Dk)), np.zeros((n, Dk))
    dA, dP = np.zeros((n, n)), np.zeros((n, n))
    dv = np.zeros((n, Dv))
    rowU = np.zeros(n)  # sum_v G_U v (for dbeta)
    for j0 in range(0, Dv, vb):
        J = slice(j0, j0 + vb)
        UbJ = T @ (beta[:, None] * v[:, J])
        UJ = UbJ - W @ S[:, J]
        dUJ = se[:, None] * (k @ dSn[:, J]) + P.T @ dO[:, J]
        GUJ = T.T @ dUJ
        dv[:, J] = beta[:, None] * GUJ
        rowU += np.sum(GUJ * v[:, J], 1)
        GW -= GUJ @ S[:, J].T
        dqS += dO[:, J] @ S[:, J].T
        dkS += UJ @ dSn[:, J].T
        dA -= GUJ @ UJ.T
        dP += dO[:, J] @ UJ.T
    dA = np.tril(dA, -1)
    dP = np.tril(dP)
    Ah = dA * beta[:, None] * Ge
    dq = gam[:, None] * dqS + (dP * Ge) @ k
    dk = se[:, None] * dkS + (dP * Ge).T @ q + (beta * gam)[:, None] * GW + (Ah + Ah.T) @ k
    dbeta = gam * np.sum(GW * k, 1) + rowU + np.sum(dA * KK, 1)
    db = gam * np.sum(q * dqS, 1)
    E = dP * P
    db += E.sum(1) - E.sum(0)
    db += beta * gam * np.sum(GW * k, 1)
    EA = dA * A
    db += EA.sum(1) - EA.sum(0)
    r = se * np.sum(dkS * k, 1)
    db -= r
    db[-1] += r.sum() + gam[-1] * np.sum(dSn * S)
    dg = np.cumsum(db[::-1])[::-1]
    return dq, dk, dv, dg, dbeta


@pytest.mark.parametrize("vb", [1, 2, 6])
def test_chunk_backward_vblocks(vb):
    """The blocked form equals the direct per-chunk backward (fp64)."""
    rng = np.random.default_rng(13 + vb)
    q, k, v, g, beta, S = rand(rng, C)
    dO = rng.standard_normal(v.shape)
    dSn = rng.standard_normal(S.shape)
    ref = chunk_bwd(q, k, v, g, beta, S, dO, dSn)
    got = chunk_bwd_vblocks(q, k, v, g, beta, S, dO, dSn, vb=vb)
    for name, x, y in zip(("dq", "dk", "dv", "dg", "dbeta"), got, ref):
        np.testing.assert_allclose(x, y, rtol=1e-10, atol=1e-10, err_msg=name)
