"""Pins for the fp64 block oracle (oracle/block.py): RMSNorm, RoPE, causal
attention and the whole CoLA / CoLA-M decoder block, each checked against
something other than itself -- torch library routines (rms_norm,
scaled_dot_product_attention, autograd), closed forms, brute-force central
differences, and the memory and recompute counts of App. C.  CPU only."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import block as OB
from paper_2502_10940_amd import inputs as I


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def relerr(a, b):
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


# --------------------------------------------------------------------------
# RMSNorm
# --------------------------------------------------------------------------

def test_rmsnorm_against_torch_and_autograd():
    g0 = rng(1)
    x = g0.standard_normal((13, 24))
    g = 1 + 0.1 * g0.standard_normal(24)
    dy = g0.standard_normal((13, 24))
    eps = 1e-6
    tx = torch.tensor(x, requires_grad=True)
    tg = torch.tensor(g, requires_grad=True)
    ty = F.rms_norm(tx, (24,), weight=tg, eps=eps)
    ty.backward(torch.tensor(dy))
    assert relerr(OB.rmsnorm(x, g, eps), ty.detach().numpy()) < 1e-14
    dx, dg = OB.rmsnorm_bwd(x, g, eps, dy)
    assert relerr(dx, tx.grad.numpy()) < 1e-13
    assert relerr(dg, tg.grad.numpy()) < 1e-13


def test_rmsnorm_constant_row_closed_form():
    # x = c (every element): mean(x^2) = c^2, y = c g / sqrt(c^2 + eps)
    d, c, eps = 7, -2.5, 1e-3
    g = np.linspace(0.5, 1.5, d)
    y = OB.rmsnorm(np.full((1, d), c), g, eps)
    assert np.allclose(y[0], c * g / math.sqrt(c * c + eps), rtol=1e-15, atol=0)


def test_rmsnorm_backward_by_central_differences():
    g0 = rng(2)
    x = g0.standard_normal((3, 5))
    g = 1 + 0.1 * g0.standard_normal(5)
    dy = g0.standard_normal((3, 5))
    eps = 1e-2
    dx, dg = OB.rmsnorm_bwd(x, g, eps, dy)
    h = 1e-6
    for name, arr, grad in (("x", x, dx), ("g", g, dg)):
        fd = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            p = arr.copy(); p[idx] += h
            m = arr.copy(); m[idx] -= h
            lp = np.sum(dy * (OB.rmsnorm(p, g, eps) if name == "x" else OB.rmsnorm(x, p, eps)))
            lm = np.sum(dy * (OB.rmsnorm(m, g, eps) if name == "x" else OB.rmsnorm(x, m, eps)))
            fd[idx] = (lp - lm) / (2 * h)
        assert relerr(grad, fd) < 1e-8, name


# --------------------------------------------------------------------------
# RoPE
# --------------------------------------------------------------------------

def test_rope_complex_form_and_angles():
    # rotate-half pairing as complex numbers: z_i = x_i + i x_{i+hd/2} -> z_i e^{i pos theta_i}
    n_seq, L, heads, hd, base = 2, 6, 3, 8, 10000.0
    x = rng(3).standard_normal((n_seq * L, heads * hd))
    y = OB.rope(x, n_seq, L, heads, base)
    theta = base ** (-2.0 * np.arange(hd // 2) / hd)
    for t in range(n_seq * L):
        pos = t % L
        for h in range(heads):
            z = x[t, h * hd: h * hd + hd // 2] + 1j * x[t, h * hd + hd // 2:(h + 1) * hd]
            w = z * np.exp(1j * pos * theta)
            assert np.allclose(y[t, h * hd: h * hd + hd // 2], w.real, rtol=0, atol=1e-14)
            assert np.allclose(y[t, h * hd + hd // 2:(h + 1) * hd], w.imag, rtol=0, atol=1e-14)
    # position 0 is the identity; pair 0 turns by exactly pos radians
    assert np.array_equal(y[0], x[0])
    assert OB.rope_angles(L, hd, base)[1, 0] == 1.0


def test_rope_inverse_norms_and_relative_position():
    n_seq, L, heads, hd, base = 1, 9, 2, 6, 100.0
    x = rng(4).standard_normal((L, heads * hd))
    y = OB.rope(x, n_seq, L, heads, base)
    assert relerr(OB.rope(y, n_seq, L, heads, base, inverse=True), x) < 1e-15
    for h in range(heads):
        lo = slice(h * hd, h * hd + hd // 2)
        hi = slice(h * hd + hd // 2, (h + 1) * hd)
        assert np.allclose(x[:, lo] ** 2 + x[:, hi] ** 2, y[:, lo] ** 2 + y[:, hi] ** 2, rtol=1e-13)
    # <rope(q) at i, rope(k) at j> depends on i - j only
    q = rng(5).standard_normal(heads * hd)
    k = rng(6).standard_normal(heads * hd)
    Q = OB.rope(np.tile(q, (L, 1)), 1, L, heads, base)
    K = OB.rope(np.tile(k, (L, 1)), 1, L, heads, base)
    for shift in (1, 3):
        for i, j in ((2, 0), (4, 1), (5, 5)):
            assert Q[i] @ K[j] == pytest.approx(Q[i + shift] @ K[j + shift], rel=1e-12, abs=1e-12)


# --------------------------------------------------------------------------
# causal attention
# --------------------------------------------------------------------------

def _torch_attention(q, k, v, n_seq, L, heads, base):
    """torch's scaled_dot_product_attention (causal) on RoPE'd q, k; the RoPE
    here is the complex-number form."""
    T, d = q.shape
    hd = d // heads
    theta = torch.tensor(base, dtype=torch.float64) ** (-2.0 * torch.arange(hd // 2, dtype=torch.float64) / hd)
    ang = torch.arange(L, dtype=torch.float64)[:, None] * theta[None, :]
    rot = torch.polar(torch.ones_like(ang), ang)                       # e^{i angle} [L][hd/2]

    def rope_t(x):
        x = x.reshape(n_seq, L, heads, hd)
        z = torch.complex(x[..., : hd // 2], x[..., hd // 2:]) * rot[None, :, None, :]
        return torch.cat([z.real, z.imag], dim=-1)

    qh = rope_t(q).permute(0, 2, 1, 3)
    kh = rope_t(k).permute(0, 2, 1, 3)
    vh = v.reshape(n_seq, L, heads, hd).permute(0, 2, 1, 3)
    o = F.scaled_dot_product_attention(qh, kh, vh, is_causal=True)
    return o.permute(0, 2, 1, 3).reshape(T, d)


@pytest.mark.parametrize("shape", [(2, 7, 3, 4), (1, 16, 2, 8), (3, 5, 1, 6)])
def test_attention_against_torch_sdpa_and_autograd(shape):
    n_seq, L, heads, hd = shape
    T, d, base = n_seq * L, heads * hd, 10000.0
    g0 = rng(7)
    q, k, v, dO = (g0.standard_normal((T, d)) for _ in range(4))
    att, probs = OB.attention(q, k, v, n_seq, L, heads, base)
    tq, tk, tv = (torch.tensor(a, requires_grad=True) for a in (q, k, v))
    to = _torch_attention(tq, tk, tv, n_seq, L, heads, base)
    to.backward(torch.tensor(dO))
    assert relerr(att, to.detach().numpy()) < 1e-13
    dq, dk, dv = OB.attention_bwd(q, k, v, probs, dO, n_seq, L, heads, base)
    for ours, ref in ((dq, tq.grad), (dk, tk.grad), (dv, tv.grad)):
        assert relerr(ours, ref.numpy()) < 1e-12


def test_attention_causal_closed_forms():
    n_seq, L, heads, hd, base = 2, 6, 2, 4, 10000.0
    T, d = n_seq * L, heads * hd
    g0 = rng(8)
    k, v = g0.standard_normal((T, d)), g0.standard_normal((T, d))
    # the first token of a sequence sees only itself: att = v there
    att, _ = OB.attention(g0.standard_normal((T, d)), k, v, n_seq, L, heads, base)
    for s in range(n_seq):
        assert np.allclose(att[s * L], v[s * L], rtol=1e-15, atol=1e-15)
    # q = 0: every score is 0, so token i averages v over tokens 0..i of its sequence
    att0, _ = OB.attention(np.zeros((T, d)), k, v, n_seq, L, heads, base)
    for s in range(n_seq):
        for i in range(L):
            assert np.allclose(att0[s * L + i], v[s * L: s * L + i + 1].mean(axis=0), rtol=1e-14, atol=1e-15)


def test_attention_backward_by_central_differences():
    n_seq, L, heads, hd, base = 1, 4, 2, 2, 50.0
    T, d = n_seq * L, heads * hd
    g0 = rng(9)
    q, k, v, dO = (g0.standard_normal((T, d)) for _ in range(4))
    _, probs = OB.attention(q, k, v, n_seq, L, heads, base)
    grads = OB.attention_bwd(q, k, v, probs, dO, n_seq, L, heads, base)
    h = 1e-6
    for which, grad in enumerate(grads):
        fd = np.zeros_like(grad)
        for idx in np.ndindex(grad.shape):
            args_p = [q.copy(), k.copy(), v.copy()]
            args_m = [q.copy(), k.copy(), v.copy()]
            args_p[which][idx] += h
            args_m[which][idx] -= h
            lp = np.sum(dO * OB.attention(*args_p, n_seq, L, heads, base)[0])
            lm = np.sum(dO * OB.attention(*args_m, n_seq, L, heads, base)[0])
            fd[idx] = (lp - lm) / (2 * h)
        assert relerr(grad, fd) < 1e-8, which


# --------------------------------------------------------------------------
# the block
# --------------------------------------------------------------------------

def block_params(seed, c: OB.Cfg):
    ins = I.block_inputs(seed, c.n_seq, c.seq_len, c.d, c.ffn, c.r, "f32")
    return {k: v.f64 for k, v in ins.items()}


def _torch_block(p, c: OB.Cfg, act):
    """The block in torch ops (rms_norm, complex-form RoPE, scaled dot product
    attention, autograd); p: dict of fp64 tensors."""
    sig = {"silu": F.silu, "identity": lambda z: z, "gelu": lambda z: F.gelu(z, approximate="none")}[act]
    cola = lambda x, A, B: sig(x @ A.T) @ B.T
    r = c.r
    a = F.rms_norm(p["x0"], (c.d,), weight=p["g1"], eps=c.eps)
    A = p["A_qkv"]
    q = cola(a, A[:r], p["B_q"])
    k = cola(a, A[r:2 * r], p["B_k"])
    v = cola(a, A[2 * r:], p["B_v"])
    att = _torch_attention(q, k, v, c.n_seq, c.seq_len, c.heads, c.base)
    x1 = p["x0"] + cola(att, p["A_o"], p["B_o"])
    b = F.rms_norm(x1, (c.d,), weight=p["g2"], eps=c.eps)
    G = p["A_gu"]
    m = cola(b, G[:r], p["B_g"]) * cola(b, G[r:], p["B_u"])
    return x1 + cola(m, p["A_d"], p["B_d"])


PARAMS = ("g1", "g2", "A_qkv", "B_q", "B_k", "B_v", "A_o", "B_o", "A_gu", "B_g", "B_u", "A_d", "B_d")


@pytest.mark.parametrize("act", ["silu", "gelu"])
@pytest.mark.parametrize("recompute", [False, True])
def test_block_against_torch_autograd(act, recompute):
    c = OB.Cfg(n_seq=2, seq_len=9, d=16, ffn=40, heads=2, r=4, act=act)
    p = block_params(11, c)
    x2, saved = OB.block_forward(c, p, p["x0"], recompute)
    dx0, grads = OB.block_backward(c, p, p["x0"], saved, p["dx2"], recompute)
    tp = {k: torch.tensor(v, requires_grad=True) for k, v in p.items() if k != "dx2"}
    tx2 = _torch_block(tp, c, act)
    tx2.backward(torch.tensor(p["dx2"]))
    assert relerr(x2, tx2.detach().numpy()) < 1e-12
    assert relerr(dx0, tp["x0"].grad.numpy()) < 1e-12
    for k in PARAMS:
        assert relerr(grads[k], tp[k].grad.numpy()) < 1e-11, k


def test_block_identity_sigma_is_the_dense_block():
    # sigma = identity: every CoLA layer is the linear map with W = B A (Sec. 3.3),
    # so the block is the plain LLaMA block with those dense weights
    c = OB.Cfg(n_seq=2, seq_len=5, d=12, ffn=20, heads=3, r=3, act="identity")
    p = block_params(12, c)
    x2, _ = OB.block_forward(c, p, p["x0"])
    r = c.r
    W = {"q": p["B_q"] @ p["A_qkv"][:r], "k": p["B_k"] @ p["A_qkv"][r:2 * r], "v": p["B_v"] @ p["A_qkv"][2 * r:],
         "o": p["B_o"] @ p["A_o"], "g": p["B_g"] @ p["A_gu"][:r], "u": p["B_u"] @ p["A_gu"][r:],
         "d": p["B_d"] @ p["A_d"]}
    t = {k: torch.tensor(v) for k, v in p.items()}
    tw = {k: torch.tensor(v) for k, v in W.items()}
    a = F.rms_norm(t["x0"], (c.d,), weight=t["g1"], eps=c.eps)
    att = _torch_attention(a @ tw["q"].T, a @ tw["k"].T, a @ tw["v"].T, c.n_seq, c.seq_len, c.heads, c.base)
    x1 = t["x0"] + att @ tw["o"].T
    b = F.rms_norm(x1, (c.d,), weight=t["g2"], eps=c.eps)
    ref = x1 + ((b @ tw["g"].T) * (b @ tw["u"].T)) @ tw["d"].T
    assert relerr(x2, ref.numpy()) < 1e-12


def test_block_gradients_by_central_differences():
    c = OB.Cfg(n_seq=1, seq_len=3, d=4, ffn=6, heads=2, r=2, act="silu", eps=1e-2)
    p = block_params(13, c)
    dx2 = p["dx2"]
    x2, saved = OB.block_forward(c, p, p["x0"])
    dx0, grads = OB.block_backward(c, p, p["x0"], saved, dx2)
    grads = dict(grads, x0=dx0)

    def loss(pp):
        return float(np.sum(dx2 * OB.block_forward(c, pp, pp["x0"])[0]))

    h = 1e-6
    for name in ("x0",) + PARAMS:
        fd = np.zeros_like(p[name])
        for idx in np.ndindex(p[name].shape):
            pp = dict(p); pp[name] = p[name].copy(); pp[name][idx] += h
            pm = dict(p); pm[name] = p[name].copy(); pm[name][idx] -= h
            fd[idx] = (loss(pp) - loss(pm)) / (2 * h)
        assert relerr(grads[name], fd) < 1e-7, name


def test_block_cola_m_equals_cola():
    c = OB.Cfg(n_seq=2, seq_len=8, d=16, ffn=24, heads=4, r=4)
    p = block_params(14, c)
    x2a, sa = OB.block_forward(c, p, p["x0"], recompute=False)
    x2b, sb = OB.block_forward(c, p, p["x0"], recompute=True)
    assert np.array_equal(x2a, x2b)
    dxa, ga = OB.block_backward(c, p, p["x0"], sa, p["dx2"], recompute=False)
    dxb, gb = OB.block_backward(c, p, p["x0"], sb, p["dx2"], recompute=True)
    assert np.array_equal(dxa, dxb)
    for k in PARAMS:
        assert np.array_equal(ga[k], gb[k]), k


def test_cola_m_saved_memory_is_2nd_plus_7nr():
    # App. C: M_CoLA-M = 2nd + 7nr (block input and mid-block residual, and the
    # seven r-wide pre-activations)
    c = OB.Cfg(n_seq=3, seq_len=4, d=8, ffn=20, heads=2, r=3)
    p = block_params(15, c)
    _, saved = OB.block_forward(c, p, p["x0"], recompute=True)
    n = c.T
    assert set(saved) == {"x1", "Z"}
    assert OB.saved_elements(saved, True) == 2 * n * c.d + 7 * n * c.r
    # CoLA keeps the 14 nr of the low-rank activations (App. C) besides its n x d ones
    _, saved_c = OB.block_forward(c, p, p["x0"], recompute=False)
    low_rank = sum(z.size for z in saved_c["Z"].values()) + sum(h.size for h in saved_c["H"].values())
    assert low_rank == 14 * n * c.r


def test_cola_m_recompute_cost():
    # App. C: CoLA-M adds the re-computation of the up projections B h whose
    # outputs the backward reads (q, k, v, gate, up; sketched in Fig. "block")
    # and of the self-attention's scaled dot product, 4 n^2 d flops per
    # sequence (QK^T and PV over the whole n x n score matrix)
    c = OB.Cfg(n_seq=2, seq_len=6, d=8, ffn=20, heads=2, r=3)
    p = block_params(16, c)
    counts = {}
    for rc in (False, True):
        _, saved = OB.block_forward(c, p, p["x0"], rc)
        oracle.reset_macs()
        OB.reset_attn_macs()
        OB.block_backward(c, p, p["x0"], saved, p["dx2"], rc)
        counts[rc] = (oracle.macs(), OB.attn_macs())
    n, d, ffn, r = c.T, c.d, c.ffn, c.r
    assert 2 * (counts[True][0] - counts[False][0]) == 2 * n * r * (3 * d + 2 * ffn)
    assert 2 * (counts[True][1] - counts[False][1]) == c.n_seq * 4 * c.seq_len ** 2 * d
    # at d_ff = 2.5 d these B h products are 16 ndr, against the paper's 18.5 ndr
    # (half of its 37 ndr CoLA forward)
    assert 2 * r * (3 * d + 2 * 2.5 * d) == 16 * d * r
