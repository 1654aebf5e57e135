"""fp64 CPU oracle of a decoder block whose seven linear projections are CoLA
layers, in CoLA and in block-level CoLA-M -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module; the GPU product path never does, and it
shares no code with that path.

What it computes (arXiv 2502.10940):
  * the block of Fig. "block" (Sec. 3.2): a LLaMA-style pre-norm decoder
    block in which q, k, v, o, gate, up and down are CoLA layers
    h = B sigma(A x) (Eq. main-fwd), while the scaled dot product of
    self-attention, the residual connections and the element-wise product of
    the gated MLP stay as they are.  With only the low-rank sigma (the 1B/7B
    setting, App. ablation and App. C "remove original sigma") the MLP is
    down(gate(b) * up(b)).  Layer norms and rotary embeddings, which the
    figure omits, are LLaMA's: RMSNorm with a gain, and RoPE on q and k.
  * its backward by the chain rule (Sec. 3.4's rule for every GEMM),
  * CoLA-M at block level (Sec. 4.2, App. C): the forward keeps only the
    block input (the caller's), the mid-block residual x1 and the seven
    r-wide pre-activations Z (memory 2nd + 7nr); the backward recomputes the
    up projections B h whose outputs it needs (q, k, v, gate, up) and the
    self-attention, then runs the same backward.

Every array is fp64, token-major ([T][width], T = n_seq * seq_len, sequence s
in rows s*seq_len .. s*seq_len + seq_len - 1).  The CoLA layers are the C
oracle's (``oracle.cola_fwd`` / ``oracle.cola_bwd`` / ``oracle.cola_up_from_z``,
whose multiply-add counter they feed); the rest is plain numpy, one matrix
product (a library primitive) or elementwise expression per step of the
definition.  A separate counter records the attention's multiply-adds.

Readings (the paper is silent on these): RMSNorm y = x g / sqrt(mean(x^2) +
eps); RoPE with the rotate-half pairing (element i with i + hd/2 of each
head, angle pos * base^(-2i/hd), pos = index within the sequence); causal
attention with scale 1/sqrt(hd); parameters g1, g2 of the two norms.
"""
from __future__ import annotations

import numpy as np

import oracle

_attn_macs = 0


def reset_attn_macs():
    global _attn_macs
    _attn_macs = 0


def attn_macs():
    return _attn_macs


# --------------------------------------------------------------------------
# RMSNorm (LLaMA's layer norm)
# --------------------------------------------------------------------------

def rmsnorm(x, g, eps):
    """y[t] = x[t] * g / sqrt(mean_k x[t, k]^2 + eps)."""
    ms = np.mean(x * x, axis=1, keepdims=True)
    return x * g[None, :] / np.sqrt(ms + eps)


def rmsnorm_bwd(x, g, eps, dy):
    """Gradients of y = rmsnorm(x, g) for the upstream dy: (dx, dg).
    With s = 1/sqrt(mean(x^2) + eps) and u = dy * g:
    dx = s u - x s^3 (u . x) / d,   dg = sum_t dy[t] x[t] s[t]."""
    d = x.shape[1]
    s = 1.0 / np.sqrt(np.mean(x * x, axis=1, keepdims=True) + eps)
    u = dy * g[None, :]
    dx = s * u - x * (s ** 3) * np.sum(u * x, axis=1, keepdims=True) / d
    dg = np.sum(dy * x * s, axis=0)
    return dx, dg


# --------------------------------------------------------------------------
# rotary position embedding (rotate-half pairing)
# --------------------------------------------------------------------------

def rope_angles(seq_len, hd, base):
    """angle[pos][i] = pos * base^(-2i/hd), i < hd/2."""
    inv = base ** (-np.arange(0, hd // 2, dtype=np.float64) * 2.0 / hd)
    return np.arange(seq_len, dtype=np.float64)[:, None] * inv[None, :]


def rope(x, n_seq, seq_len, heads, base, inverse=False):
    """Rotate each head's pairs (i, i + hd/2) of every token by its angle
    (by minus the angle when inverse: the transpose, used by the backward)."""
    T, d = x.shape
    hd = d // heads
    ang = rope_angles(seq_len, hd, base)
    c = np.tile(np.cos(ang), (n_seq, 1))            # [T][hd/2]
    s = np.tile(np.sin(ang), (n_seq, 1))
    if inverse:
        s = -s
    y = np.empty_like(x)
    for h in range(heads):
        lo = x[:, h * hd: h * hd + hd // 2]
        hi = x[:, h * hd + hd // 2: (h + 1) * hd]
        y[:, h * hd: h * hd + hd // 2] = lo * c - hi * s
        y[:, h * hd + hd // 2: (h + 1) * hd] = hi * c + lo * s
    return y


# --------------------------------------------------------------------------
# causal scaled-dot-product attention per sequence and head
# --------------------------------------------------------------------------

def attention(q, k, v, n_seq, seq_len, heads, base):
    """att = softmax(rope(q) rope(k)^T / sqrt(hd), causal) v per sequence and
    head.  q, k, v are the projections' outputs (before RoPE).  Returns (att,
    probs) with probs[s][h] the [seq_len][seq_len] attention matrix."""
    global _attn_macs
    T, d = q.shape
    hd = d // heads
    qr = rope(q, n_seq, seq_len, heads, base)
    kr = rope(k, n_seq, seq_len, heads, base)
    att = np.empty_like(q)
    probs = np.empty((n_seq, heads, seq_len, seq_len))
    future = np.triu(np.ones((seq_len, seq_len), dtype=bool), 1)    # key after query
    for s in range(n_seq):
        rows = slice(s * seq_len, (s + 1) * seq_len)
        for h in range(heads):
            cols = slice(h * hd, (h + 1) * hd)
            S = qr[rows, cols] @ kr[rows, cols].T / np.sqrt(hd)
            S[future] = -np.inf
            S = S - S.max(axis=1, keepdims=True)
            P = np.exp(S)
            P /= P.sum(axis=1, keepdims=True)
            probs[s, h] = P
            att[rows, cols] = P @ v[rows, cols]
            _attn_macs += 2 * seq_len * seq_len * hd
    return att, probs


def attention_bwd(q, k, v, probs, datt, n_seq, seq_len, heads, base):
    """Gradients (dq, dk, dv) of attention() for the upstream datt, with respect
    to the projections' outputs (RoPE's transpose applied to dq, dk)."""
    global _attn_macs
    T, d = q.shape
    hd = d // heads
    qr = rope(q, n_seq, seq_len, heads, base)
    kr = rope(k, n_seq, seq_len, heads, base)
    dqr = np.empty_like(q)
    dkr = np.empty_like(k)
    dv = np.empty_like(v)
    for s in range(n_seq):
        rows = slice(s * seq_len, (s + 1) * seq_len)
        for h in range(heads):
            cols = slice(h * hd, (h + 1) * hd)
            P = probs[s, h]
            dO = datt[rows, cols]
            dv[rows, cols] = P.T @ dO
            dP = dO @ v[rows, cols].T
            dS = P * (dP - np.sum(dP * P, axis=1, keepdims=True))     # softmax backward
            dqr[rows, cols] = dS @ kr[rows, cols] / np.sqrt(hd)
            dkr[rows, cols] = dS.T @ qr[rows, cols] / np.sqrt(hd)
            _attn_macs += 4 * seq_len * seq_len * hd
    return (rope(dqr, n_seq, seq_len, heads, base, inverse=True),
            rope(dkr, n_seq, seq_len, heads, base, inverse=True), dv)


# --------------------------------------------------------------------------
# the block
# --------------------------------------------------------------------------

class Cfg:
    def __init__(self, n_seq, seq_len, d, ffn, heads, r, act="silu", eps=1e-6, base=10000.0):
        self.n_seq, self.seq_len, self.d, self.ffn = n_seq, seq_len, d, ffn
        self.heads, self.r, self.act, self.eps, self.base = heads, r, act, eps, base
        self.T = n_seq * seq_len


def _split(A_stacked, n):
    r = A_stacked.shape[0] // n
    return [A_stacked[i * r:(i + 1) * r] for i in range(n)]


def _attn(c, q, k, v):
    return attention(q, k, v, c.n_seq, c.seq_len, c.heads, c.base)


def block_forward(c: Cfg, w: dict, x0, recompute=False):
    """x2 and what the backward needs.  w holds the parameters by the names of
    ``inputs.block_shapes`` (fp64).  CoLA keeps every activation the backward
    reads; CoLA-M keeps x1 and the seven pre-activations only."""
    act = c.act
    Aq, Ak, Av = _split(w["A_qkv"], 3)
    Ag, Au = _split(w["A_gu"], 2)
    a = rmsnorm(x0, w["g1"], c.eps)
    Zq, Hq, q = oracle.cola_fwd(a, Aq, w["B_q"], act)
    Zk, Hk, k = oracle.cola_fwd(a, Ak, w["B_k"], act)
    Zv, Hv, v = oracle.cola_fwd(a, Av, w["B_v"], act)
    att, probs = _attn(c, q, k, v)
    Zo, Ho, o = oracle.cola_fwd(att, w["A_o"], w["B_o"], act)
    x1 = x0 + o
    b = rmsnorm(x1, w["g2"], c.eps)
    Zg, Hg, gt = oracle.cola_fwd(b, Ag, w["B_g"], act)
    Zu, Hu, u = oracle.cola_fwd(b, Au, w["B_u"], act)
    m = gt * u
    Zd, Hd, y = oracle.cola_fwd(m, w["A_d"], w["B_d"], act)
    x2 = x1 + y
    Z = {"q": Zq, "k": Zk, "v": Zv, "o": Zo, "gate": Zg, "up": Zu, "down": Zd}
    if recompute:
        saved = {"x1": x1, "Z": Z}
    else:
        saved = {"x1": x1, "Z": Z, "a": a, "q": q, "k": k, "v": v, "att": att, "probs": probs, "b": b,
                 "gate": gt, "up": u, "m": m,
                 "H": {"q": Hq, "k": Hk, "v": Hv, "o": Ho, "gate": Hg, "up": Hu, "down": Hd}}
    return x2, saved


def recompute_saved(c: Cfg, w: dict, x0, saved):
    """CoLA-M's recompute at the start of the backward: the norms, the up
    projections B sigma(Z) of q, k, v, gate and up, the gated product and the
    self-attention, from x0, x1 and the saved Z (o and down feed only the
    residual sums, so their outputs are not needed)."""
    act = c.act
    Z = saved["Z"]
    out = dict(saved)
    out["a"] = rmsnorm(x0, w["g1"], c.eps)
    _, out["q"] = oracle.cola_up_from_z(Z["q"], w["B_q"], act)
    _, out["k"] = oracle.cola_up_from_z(Z["k"], w["B_k"], act)
    _, out["v"] = oracle.cola_up_from_z(Z["v"], w["B_v"], act)
    out["att"], out["probs"] = _attn(c, out["q"], out["k"], out["v"])
    out["b"] = rmsnorm(saved["x1"], w["g2"], c.eps)
    _, out["gate"] = oracle.cola_up_from_z(Z["gate"], w["B_g"], act)
    _, out["up"] = oracle.cola_up_from_z(Z["up"], w["B_u"], act)
    out["m"] = out["gate"] * out["up"]
    return out


def block_backward(c: Cfg, w: dict, x0, saved, dx2, recompute=False):
    """dx0 and the parameter gradients (names of ``inputs.block_shapes``)."""
    act = c.act
    s = recompute_saved(c, w, x0, saved) if recompute else saved
    Z = s["Z"]
    Aq, Ak, Av = _split(w["A_qkv"], 3)
    Ag, Au = _split(w["A_gu"], 2)
    g = {}
    # x2 = x1 + down(m): the residual passes dx2 through
    _, dm, dAd, g["B_d"] = oracle.cola_bwd(s["m"], Z["down"], w["A_d"], w["B_d"], dx2, act)
    g["A_d"] = dAd
    dgt = dm * s["up"]
    du = dm * s["gate"]
    _, db_g, dAg, g["B_g"] = oracle.cola_bwd(s["b"], Z["gate"], Ag, w["B_g"], dgt, act)
    _, db_u, dAu, g["B_u"] = oracle.cola_bwd(s["b"], Z["up"], Au, w["B_u"], du, act)
    g["A_gu"] = np.concatenate([dAg, dAu])
    dx1_n, g["g2"] = rmsnorm_bwd(s["x1"], w["g2"], c.eps, db_g + db_u)
    dx1 = dx2 + dx1_n
    # x1 = x0 + o(att)
    _, datt, g["A_o"], g["B_o"] = oracle.cola_bwd(s["att"], Z["o"], w["A_o"], w["B_o"], dx1, act)
    dq, dk, dv = attention_bwd(s["q"], s["k"], s["v"], s["probs"], datt, c.n_seq, c.seq_len, c.heads, c.base)
    _, da_q, dAq, g["B_q"] = oracle.cola_bwd(s["a"], Z["q"], Aq, w["B_q"], dq, act)
    _, da_k, dAk, g["B_k"] = oracle.cola_bwd(s["a"], Z["k"], Ak, w["B_k"], dk, act)
    _, da_v, dAv, g["B_v"] = oracle.cola_bwd(s["a"], Z["v"], Av, w["B_v"], dv, act)
    g["A_qkv"] = np.concatenate([dAq, dAk, dAv])
    dx0_n, g["g1"] = rmsnorm_bwd(x0, w["g1"], c.eps, da_q + da_k + da_v)
    dx0 = dx1 + dx0_n
    return dx0, g


def saved_elements(saved, recompute):
    """Elements the forward keeps for the backward, counted as the paper's
    memory analysis does (App. C): the block input, which the caller keeps
    for the backward, counts as one n x d; CoLA's attention matrix is
    excluded (a kernel that recomputes it from q and k does not keep it)."""
    T, d = saved["x1"].shape
    n = T * d                                          # the block input x0
    n += saved["x1"].size + sum(z.size for z in saved["Z"].values())
    if not recompute:
        n += sum(saved[k].size for k in ("a", "q", "k", "v", "att", "b", "gate", "up", "m"))
        n += sum(h.size for h in saved["H"].values())
    return n
