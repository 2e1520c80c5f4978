"""fp64 CPU oracle of the block-int4 quantised-linear hot path.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
the benchmark's CPU-baseline leg may import this module.  It shares no code
with the HIP library and never runs on its outputs.

What it computes, and where the method defines it:
  * the paper runs every weight tensor as a quantised linear operator on
    whichever backend holds it (Sec. 4.1-4.2) and uses INT4 weights for most
    models (Sec. 5.1, "Models") without fixing the layout.  The reading used
    here: one signed code q in [-8, 7] per weight, stored offset-binary
    (u = q + 8) two per byte with the even input index in the low nibble,
    rows = output features, and one fp16 scale per 32 consecutive inputs;
  * the dense feed-forward block is SwiGLU; MoE layers route each token to
    its top-8 experts and combine their outputs with the softmax weights
    renormalised over the selected experts; only routed experts are touched
    (Sec. 4.2.2, the transfer of MoE experts waits until routing is known;
    Sec. 4.4.1, only activated experts count in a decode round);
  * prefill processes a whole chunk of tokens, decode one token per sequence
    (Sec. 2.2; chunked prefill in Sec. 5.1);
  * where a tensor lives (HBM or pinned host memory, Sec. 4.2.1) does not
    change any value, so nothing here looks at placement.

Arithmetic is fp64 throughout, with inputs taken exactly from their fp16
values and no intermediate rounding.  Each function that produces a
floating-point result also returns ``zeta``: the first-order magnitude that
bounds the error a faithful low-precision implementation may make, per unit
of relative error.  For one linear layer it is exactly |W| . |x|, the
magnitude named in the elementwise acceptance bound |y - y_ref| <= eps * zeta;
composite stages propagate it through each step (derivative bounds plus the
step's own rounding).

Pins (tests marked ``not gpu``): exhaustive nibble table and pack/unpack
identity; dequant round trip; exact rational brute force on tiny shapes;
linearity, scaling and permutation invariants; SiLU closed forms; softmax
renormalisation identities and dense brute-force MoE; bucketing invariants;
RMSNorm closed forms; the GQA stub against literal single-key attention.
"""
from __future__ import annotations

import numpy as np

GROUP = 32


# ----------------------------------------------------------------------------- format

def unpack_codes(codes: np.ndarray) -> np.ndarray:
    """Signed int4 codes q[N][K] from packed bytes codes[N][K/2].

    Byte j of a row holds inputs 2j (low nibble) and 2j+1 (high nibble), each
    as u = q + 8.
    """
    codes = np.asarray(codes, dtype=np.uint8)
    n, kb = codes.shape
    q = np.empty((n, 2 * kb), dtype=np.int8)
    q[:, 0::2] = (codes & 0x0F).astype(np.int8) - 8
    q[:, 1::2] = (codes >> 4).astype(np.int8) - 8
    return q


def dequant(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """w[n, k] = s[n, k // 32] * q[n, k] in fp64 (exact: an fp16 scale times a
    4-bit integer needs at most 15 significant bits)."""
    q = unpack_codes(codes).astype(np.float64)
    s = np.asarray(scales, dtype=np.float16).astype(np.float64)
    assert q.shape[1] == s.shape[1] * GROUP, "one scale per 32 inputs"
    return q * np.repeat(s, GROUP, axis=1)


# ----------------------------------------------------------------------------- linear

def linear_w(x: np.ndarray, w: np.ndarray, x_zeta: np.ndarray | None = None):
    """y = x . W^T for dequantised W[N][K]; returns (y, zeta) with
    zeta = |W| . (|x| + x_zeta)."""
    xd = np.asarray(x, dtype=np.float64)
    y = xd @ w.T
    mag = np.abs(xd) if x_zeta is None else np.abs(xd) + x_zeta
    return y, mag @ np.abs(w).T


def linear(x: np.ndarray, codes: np.ndarray, scales: np.ndarray, x_zeta: np.ndarray | None = None):
    """Quantised linear y[m, n] = sum_k x[m, k] * s[n, k//32] * q[n, k] (fp64, unrounded)."""
    return linear_w(x, dequant(codes, scales), x_zeta)


def linear_rows(x: np.ndarray, codes_rows: np.ndarray, scales_rows: np.ndarray):
    """The same linear restricted to a subset of output rows (for sampled checks
    of full-size tensors): codes_rows / scales_rows hold only those rows."""
    return linear(x, codes_rows, scales_rows)


# ----------------------------------------------------------------------------- SwiGLU FFN

SILU_DERIV_MAX = 1.1  # max |d silu / dz| is about 1.0998 (near z = 2.4)


def silu(z: np.ndarray) -> np.ndarray:
    """silu(z) = z / (1 + exp(-z))."""
    z = np.asarray(z, dtype=np.float64)
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def swiglu(g: np.ndarray, u: np.ndarray, g_zeta: np.ndarray, u_zeta: np.ndarray):
    """h = silu(g) * u with its propagated magnitude."""
    sg = silu(g)
    h = sg * u
    zeta = SILU_DERIV_MAX * g_zeta * np.abs(u) + np.abs(sg) * u_zeta + np.abs(h)
    return h, zeta


def swiglu_ffn(x: np.ndarray, gate, up, down, x_zeta: np.ndarray | None = None):
    """y = (silu(x W_gate) * (x W_up)) W_down; each weight is a (codes, scales) pair.

    Returns (y, zeta, h) where h is the exact intermediate activation.
    """
    g, zg = linear(x, *gate, x_zeta)
    u, zu = linear(x, *up, x_zeta)
    h, zh = swiglu(g, u, zg, zu)
    y, zy = linear(h, *down, zh)
    return y, zy, h


# ----------------------------------------------------------------------------- routing

def router_logits(x: np.ndarray, w_r: np.ndarray, bias: np.ndarray | None = None):
    """l[t, e] = sum_k x[t, k] * W_r[k, e] + b[e]; W_r is fp16 [H][E], not quantised."""
    xd = np.asarray(x, dtype=np.float64)
    wd = np.asarray(w_r, dtype=np.float16).astype(np.float64)
    logits = xd @ wd
    zeta = np.abs(xd) @ np.abs(wd)
    if bias is not None:
        b = np.asarray(bias, dtype=np.float64)
        logits = logits + b[None, :]
        zeta = zeta + np.abs(b)[None, :]
    return logits, zeta


def topk_route(logits: np.ndarray, k: int):
    """Top-k routing of each token.

    Experts are ranked by (logit descending, expert id ascending); the first k
    form the selection, listed in that rank order (so slot 0 has the largest
    weight).  Weights p are the softmax over the k selected logits, which
    equals the softmax over all experts renormalised over the selection.
    Returns idx int32[T][k] and p float64[T][k].
    """
    logits = np.asarray(logits, dtype=np.float64)
    t, e = logits.shape
    ids = np.arange(e)
    idx = np.empty((t, k), dtype=np.int32)
    p = np.empty((t, k), dtype=np.float64)
    for i in range(t):
        order = np.lexsort((ids, -logits[i]))  # last key is primary
        sel = order[:k]
        z = logits[i, sel] - logits[i, sel[0]]
        ez = np.exp(z)
        idx[i] = sel
        p[i] = ez / ez.sum()
    return idx, p


def softmax_weight_zeta(p: np.ndarray, sel_logit_zeta: np.ndarray) -> np.ndarray:
    """Magnitude of the error of p given logit errors: dp_j = p_j (dl_j - sum_i p_i dl_i)."""
    mean = (p * sel_logit_zeta).sum(axis=1, keepdims=True)
    return p * (sel_logit_zeta + mean) + p


# ----------------------------------------------------------------------------- bucketing

def bucket(idx: np.ndarray, n_experts: int):
    """Token-to-expert bucketing of the T*k routed pairs.

    Pair id of (token t, slot j) is k*t + j.  counts[e] = number of pairs routed
    to e; offsets = exclusive prefix sum (offsets[E] = T*k); perm lists pair ids
    ordered by (expert ascending, token ascending) -- unique, as a token selects
    an expert at most once; inv_perm[perm[i]] = i.
    """
    idx = np.asarray(idx, dtype=np.int64)
    t, k = idx.shape
    flat = idx.reshape(-1)
    counts = np.bincount(flat, minlength=n_experts).astype(np.int32)
    offsets = np.zeros(n_experts + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(counts)
    perm = np.argsort(flat, kind="stable").astype(np.int32)  # pair ids rise with token
    inv_perm = np.empty_like(perm)
    inv_perm[perm] = np.arange(t * k, dtype=np.int32)
    return counts, offsets, perm, inv_perm


# ----------------------------------------------------------------------------- MoE

def moe_ffn(x: np.ndarray, w_r: np.ndarray, bias, experts, k: int, x_zeta=None, route=None):
    """Routed MoE layer y[t] = sum_j p[t, j] * FFN_{idx[t, j]}(x[t]).

    experts[e] = (gate, up, down), each a (codes, scales) pair; only experts
    some token selected are evaluated.  Returns (y, zeta, aux) with aux holding
    logits, idx, p and per-pair expert outputs out[T][k][H].

    route = (idx, p) evaluates the layer on a given selection and given
    weights instead of the top-k of the fp64 logits: when two experts' logits
    are within rounding of each other, either selection is a correct routing,
    and the output is then defined by the selection actually made.  The
    weights' own error is then not part of zeta.
    """
    xd = np.asarray(x, dtype=np.float64)
    t, hdim = xd.shape
    logits, zl = router_logits(xd, w_r, bias)
    if x_zeta is not None:
        zl = zl + x_zeta @ np.abs(np.asarray(w_r, np.float16).astype(np.float64))
    if route is None:
        idx, p = topk_route(logits, k)
    else:
        idx = np.asarray(route[0], dtype=np.int32).reshape(t, k)
        p = np.asarray(route[1], dtype=np.float64).reshape(t, k)
    out = np.zeros((t, k, hdim))
    zout = np.zeros((t, k, hdim))
    for e in np.unique(idx):
        tok, slot = np.nonzero(idx == e)
        xz = None if x_zeta is None else x_zeta[tok]
        ye, zye, _ = swiglu_ffn(xd[tok], *experts[int(e)], x_zeta=xz)
        out[tok, slot] = ye
        zout[tok, slot] = zye
    y = np.einsum("tj,tjh->th", p, out)
    zsel = np.take_along_axis(zl, idx.astype(np.int64), axis=1)
    zp = softmax_weight_zeta(p, zsel) if route is None else np.zeros_like(p)
    zeta = np.einsum("tj,tjh->th", p, zout) + np.einsum("tj,tjh->th", zp, np.abs(out)) + np.abs(y)
    return y, zeta, {"logits": logits, "logit_zeta": zl, "idx": idx, "p": p, "out": out}


# ----------------------------------------------------------------------------- glue of a decoder layer

def rmsnorm(v: np.ndarray, eps: float = 1e-6, v_zeta: np.ndarray | None = None):
    """n = v / sqrt(mean(v^2) + eps) per row (unit gain)."""
    v = np.asarray(v, dtype=np.float64)
    kdim = v.shape[-1]
    r = np.sqrt((v * v).mean(axis=-1, keepdims=True) + eps)
    n = v / r
    zeta = np.abs(n)
    if v_zeta is not None:
        cross = (np.abs(v) * v_zeta).sum(axis=-1, keepdims=True)
        zeta = zeta + v_zeta / r + np.abs(v) * cross / (kdim * r ** 3)
    return n, zeta


def gqa_stub(v: np.ndarray, n_heads: int, n_kv: int, head_dim: int) -> np.ndarray:
    """Attention output at context length 1: query head i reads KV head i // (n_heads / n_kv)."""
    g = n_heads // n_kv
    v = np.asarray(v)
    m = v.shape[0]
    vh = v.reshape(m, n_kv, head_dim)
    return np.repeat(vh, g, axis=1).reshape(m, n_heads * head_dim)


def attention_single_key(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_heads: int, n_kv: int, head_dim: int):
    """Literal scaled-dot-product grouped-query attention of each token over a
    context of exactly one key (its own); the GQA stub must equal it."""
    m = q.shape[0]
    g = n_heads // n_kv
    out = np.zeros((m, n_heads * head_dim))
    for t in range(m):
        for i in range(n_heads):
            qi = q[t, i * head_dim:(i + 1) * head_dim]
            j = i // g
            kj = k[t, j * head_dim:(j + 1) * head_dim]
            vj = v[t, j * head_dim:(j + 1) * head_dim]
            scores = np.array([qi @ kj / np.sqrt(head_dim)])
            w = np.exp(scores - scores.max())
            w = w / w.sum()
            out[t, i * head_dim:(i + 1) * head_dim] = w[0] * vj
    return out


def decoder_layer(h: np.ndarray, W: dict, n_heads: int, n_kv: int, head_dim: int,
                  eps: float = 1e-6, h_zeta: np.ndarray | None = None, ffn=None):
    """Pre-norm decoder layer with a context-length-1 attention stub.

      a = rms(h); q, k, v = a Wq, a Wk, a Wv; h1 = h + gqa(v) Wo;
      b = rms(h1); h2 = h1 + FFN(b)

    W maps role names to (codes, scales).  ``ffn(b, b_zeta) -> (y, zeta)``
    replaces the dense SwiGLU FFN (an MoE layer, for instance).  Returns
    (h2, zeta, aux) with aux holding the q and k projections.
    """
    hd = np.asarray(h, dtype=np.float64)
    a, za = rmsnorm(hd, eps, h_zeta)
    q, _ = linear(a, *W["q"], za)
    kk, _ = linear(a, *W["k"], za)
    v, zv = linear(a, *W["v"], za)
    o_in = gqa_stub(v, n_heads, n_kv, head_dim)
    zo_in = gqa_stub(zv, n_heads, n_kv, head_dim)
    o, zo = linear(o_in, *W["o"], zo_in)
    h1 = hd + o
    zh1 = zo + np.abs(h1) + (0 if h_zeta is None else h_zeta)
    b, zb = rmsnorm(h1, eps, zh1)
    if ffn is None:
        f, zf, _ = swiglu_ffn(b, W["gate"], W["up"], W["down"], zb)
    else:
        f, zf = ffn(b, zb)
    h2 = h1 + f
    zh2 = zh1 + zf + np.abs(h2)
    return h2, zh2, {"q": q, "k": kk, "v": v}
