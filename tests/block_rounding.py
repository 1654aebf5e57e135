"""The decoder block under the GPU path's bf16 storage policy, assembled from
the oracle's own pieces (the layer's dense products, sigma of a given Z and
the backward from a given Z; the block oracle's RMSNorm, its backward and the
rotation) with a rounding `R` applied wherever the path stores a bf16 tensor:
every activation and activation gradient between kernels (a, b, x1, x2, the
seven Z, H and layer outputs, att, m, dm and the gated product's gradients,
the layers' dZ and dX, dx1, dx0), and, inside the attention, the rotated
q and k and the probabilities and dS that enter its matrix products.  The
attention follows the kernels' order where it decides a rounding: the
forward's online softmax over 32-key blocks for groups of 32 queries, and
the softmax backward's D = rowsum(dO * O) from the stored O.  Parameter
gradients stay unrounded (fp32 outputs).

With R the identity every step is the block oracle's (the CPU test pins
that), so what separates this reference from the oracle is the storage
policy alone.  Test infrastructure: numpy in fp64, no code shared with the
GPU path."""
from __future__ import annotations

import numpy as np

import oracle
from oracle import block as OB


def _split(A, n):
    r = A.shape[0] // n
    return [A[i * r:(i + 1) * r] for i in range(n)]


def _layer_fwd(X, A, B, act, R):
    Z = R(oracle.dense_fwd(X, A))
    H = R(oracle.cola_up_from_z(Z, B, act)[0])
    return Z, H, R(oracle.dense_fwd(H, B))


def _layer_bwd(X, Z, H, A, B, dY, act, R):
    """(dZ, dX before its rounding, dA, dB)."""
    dZ = R(oracle.cola_bwd(X, Z, A, B, dY, act)[0])
    dX, dA = oracle.dense_bwd(X, A, dZ)
    return dZ, dX, dA, oracle.dense_bwd(H, B, dY)[1]


def _heads(c):
    hd = c.d // c.heads
    for s in range(c.n_seq):
        rows = slice(s * c.seq_len, (s + 1) * c.seq_len)
        for h in range(c.heads):
            yield rows, slice(h * hd, (h + 1) * hd), hd


def _attn_fwd(c, q, k, v, R):
    """Causal attention as the kernels order it: queries in groups of 32, keys
    in ascending blocks of 32, an online softmax in the exp2 domain whose
    reference maximum moves (rescaling l and the output) only when some query
    of the group sees a block maximum above it by more than 8, and the
    probabilities rounded as they enter the product with v.  With R the
    identity this is exactly softmax(S) v."""
    qr = R(OB.rope(q, c.n_seq, c.seq_len, c.heads, c.base))
    kr = R(OB.rope(k, c.n_seq, c.seq_len, c.heads, c.base))
    L = c.seq_len
    att = np.empty_like(q)
    probs = {}
    for rows, cols, hd in _heads(c):
        S = qr[rows, cols] @ kr[rows, cols].T
        S[np.triu(np.ones((L, L), dtype=bool), 1)] = -np.inf
        cl = np.log2(np.e) / np.sqrt(hd)                     # scores to the exp2 domain
        V = v[rows, cols]
        O = np.zeros((L, hd))
        lse = np.empty(L)
        for g0 in range(0, L, 32):
            qs = slice(g0, min(L, g0 + 32))
            m = np.full((qs.stop - g0, 1), -np.inf)
            l = np.zeros((qs.stop - g0, 1))
            o = np.zeros((qs.stop - g0, hd))
            for k0 in range(0, qs.stop, 32):
                ks = slice(k0, min(L, k0 + 32))
                sb = S[qs, ks] * cl
                mb = sb.max(axis=1, keepdims=True)
                if np.any(mb > m + 8.0):
                    mn = np.maximum(m, mb)
                    alpha = np.where(m == mn, 1.0, np.exp2(m - mn))
                    l, o, m = l * alpha, o * alpha, mn
                pb = np.exp2(sb - m)
                l = l + pb.sum(axis=1, keepdims=True)
                o = o + R(pb) @ V[ks]
            O[qs] = o / l
            lse[qs] = (m + np.log2(l))[:, 0]
        probs[rows.start, cols.start] = np.exp2(S * cl - lse[:, None])
        att[rows, cols] = O
    return R(att), probs, qr, kr


def _attn_bwd(c, v, att, probs, qr, kr, datt, R):
    dqr, dkr, dv = np.empty_like(qr), np.empty_like(kr), np.empty_like(v)
    for rows, cols, hd in _heads(c):
        P = probs[rows.start, cols.start]
        dO = datt[rows, cols]
        dv[rows, cols] = R(P).T @ dO
        dP = dO @ v[rows, cols].T
        D = np.sum(dO * att[rows, cols], axis=1, keepdims=True)
        dS = R(P * (dP - D))
        dqr[rows, cols] = dS @ kr[rows, cols] / np.sqrt(hd)
        dkr[rows, cols] = dS.T @ qr[rows, cols] / np.sqrt(hd)
    inv = lambda x: OB.rope(x, c.n_seq, c.seq_len, c.heads, c.base, inverse=True)
    return R(inv(dqr)), R(inv(dkr)), R(dv)


def rounded_block(c, w, x0, dx2, R, keep=None):
    """Forward and backward of the block (CoLA and CoLA-M give the same
    values) under the storage rounding R: (x2, dx0, parameter gradients).
    A dict passed as `keep` receives the forward's stored tensors by the
    names of the library's saved slots."""
    act = c.act
    Aq, Ak, Av = _split(w["A_qkv"], 3)
    Ag, Au = _split(w["A_gu"], 2)
    # forward
    a = R(OB.rmsnorm(x0, w["g1"], c.eps))
    fq, fk, fv = (_layer_fwd(a, A_, w[B_], act, R) for A_, B_ in ((Aq, "B_q"), (Ak, "B_k"), (Av, "B_v")))
    att, probs, qr, kr = _attn_fwd(c, fq[2], fk[2], fv[2], R)
    fo = _layer_fwd(att, w["A_o"], w["B_o"], act, R)
    x1 = R(x0 + fo[2])
    b = R(OB.rmsnorm(x1, w["g2"], c.eps))
    fg = _layer_fwd(b, Ag, w["B_g"], act, R)
    fu = _layer_fwd(b, Au, w["B_u"], act, R)
    m = R(fg[2] * fu[2])
    fd = _layer_fwd(m, w["A_d"], w["B_d"], act, R)
    x2 = R(x1 + fd[2])
    if keep is not None:
        keep.update(a=a, q=fq[2], k=fk[2], v=fv[2], att=att, x1=x1, b=b, gate=fg[2], up=fu[2], m=m,
                    Z_qkv=np.hstack([fq[0], fk[0], fv[0]]), H_qkv=np.hstack([fq[1], fk[1], fv[1]]),
                    Z_o=fo[0], H_o=fo[1], Z_gu=np.hstack([fg[0], fu[0]]), H_gu=np.hstack([fg[1], fu[1]]),
                    Z_down=fd[0], H_down=fd[1])
    # backward
    g = {}
    _, dm, g["A_d"], g["B_d"] = _layer_bwd(m, fd[0], fd[1], w["A_d"], w["B_d"], dx2, act, R)
    dm = R(dm)
    dgt, du = R(dm * fu[2]), R(dm * fg[2])
    dZg, dbg, dAg, g["B_g"] = _layer_bwd(b, fg[0], fg[1], Ag, w["B_g"], dgt, act, R)
    dZu, dbu, dAu, g["B_u"] = _layer_bwd(b, fu[0], fu[1], Au, w["B_u"], du, act, R)
    g["A_gu"] = np.concatenate([dAg, dAu])
    dx1_n, g["g2"] = OB.rmsnorm_bwd(x1, w["g2"], c.eps, R(dbg + dbu))
    dx1 = R(dx2 + dx1_n)
    _, datt, g["A_o"], g["B_o"] = _layer_bwd(att, fo[0], fo[1], w["A_o"], w["B_o"], dx1, act, R)
    dq, dk, dv = _attn_bwd(c, fv[2], att, probs, qr, kr, R(datt), R)
    das, dAs = [], []
    for (Z_, H_, _), A_, B_, dY_, name in ((fq, Aq, "B_q", dq, "B_q"), (fk, Ak, "B_k", dk, "B_k"),
                                           (fv, Av, "B_v", dv, "B_v")):
        _, da_p, dA_p, g[name] = _layer_bwd(a, Z_, H_, A_, w[B_], dY_, act, R)
        das.append(da_p)
        dAs.append(dA_p)
    g["A_qkv"] = np.concatenate(dAs)
    dx0_n, g["g1"] = OB.rmsnorm_bwd(x0, w["g1"], c.eps, R(das[0] + das[1] + das[2]))
    dx0 = R(dx1 + dx0_n)
    return x2, dx0, g
