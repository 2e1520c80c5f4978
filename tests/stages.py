"""Teacher-forced checks of the stages inside a decoder-layer call: each stage
is compared with the oracle evaluated on the GPU's own fp16 input to that
stage (its attention output, its residual stream after attention, its SwiGLU
activation), with the magnitude zeta = |W| . |x| of that one stage."""
import numpy as np

import oracle
from tests.parity import check, tight_eps

# Per-token norm gate of a SwiGLU activation: silu(g) * u moves by about
# |g| * (1 - sigmoid(g)) * (relative error of g) where g is negative, so a
# token whose gate values are mostly negative sees the error of its gate
# products amplified many times in relative terms.  With fp16-rounded weights
# (the MFMA path) and nothing else inexact, one routed token of the
# 235B-shaped layer already reaches 1.2e-2 this way.  The elementwise gate,
# with its SiLU-derivative term, stays the tight one for this stage.
SWIGLU_ROW_L2 = 2e-2
# Whole composite stages (a layer, an MoE FFN) free-running from the oracle's
# own intermediates: per-token relative L2 at the required 1e-2 bound; the
# stages inside are gated teacher-forced.
COMPOSITE_ROW_L2 = 1e-2


def _np(t):
    return t.detach().cpu().numpy() if hasattr(t, "detach") else np.asarray(t)


def rows_of(n, limit, seed_perm):
    """All rows when there are at most `limit`, else a seeded sample."""
    return np.arange(n) if n <= limit else np.sort(seed_perm[:limit])


def attention_stages(W, n_heads, n_kv, head_dim, h_in, q_out, k_out, attn, h_attn, name, eps=1e-6, cols=None):
    """q, k and the attention output from rms(h_in); h_attn = h_in + attn Wo.
    cols: output columns to check (all when None) of q, attn and h_attn."""
    M, H = h_in.shape
    mfma = M > 16
    x = h_in.astype(np.float64)
    a, _ = oracle.rmsnorm(x, eps)
    t_in = tight_eps(H, mfma, norm=True)
    Hq = n_heads * head_dim
    cq = np.arange(Hq) if cols is None else cols[cols < Hq]
    qr, zq = oracle.linear(a, W["q"][0][cq], W["q"][1][cq])
    check(_np(q_out)[:, cq], qr, zq, name=f"{name} q", tight=t_in)
    kr, zk = oracle.linear(a, *W["k"])
    check(_np(k_out), kr, zk, name=f"{name} k", tight=t_in)
    vr, zv = oracle.linear(a, *W["v"])
    ar = oracle.gqa_stub(vr, n_heads, n_kv, head_dim)
    za = oracle.gqa_stub(zv, n_heads, n_kv, head_dim)
    check(_np(attn)[:, cq], ar[:, cq], za[:, cq], name=f"{name} attention output", tight=t_in)
    # O projection plus residual, on the GPU's own attention output
    co = np.arange(H) if cols is None else cols[cols < H]
    o_in = _np(attn).astype(np.float64)
    orr, zo = oracle.linear(o_in, W["o"][0][co], W["o"][1][co])
    check(_np(h_attn)[:, co], x[:, co] + orr, zo + np.abs(x[:, co]), name=f"{name} O + residual",
          tight=tight_eps(Hq, mfma))


def ffn_stages(W, h_attn, act, h_out, name, eps=1e-6, cols=None, sum32=None):
    """act = silu(rms(h_attn) Wg) * (rms(h_attn) Wu) and h_out = h_attn + act Wd
    (or sum32 = that sum in fp32 when the layer renormalises its output)."""
    M, H = h_attn.shape
    mfma = M > 16
    x = _np(h_attn).astype(np.float64)
    b, _ = oracle.rmsnorm(x, eps)
    I = W["gate"][0].shape[0]
    ci = np.arange(I) if cols is None else cols[cols < I]
    g, zg = oracle.linear(b, W["gate"][0][ci], W["gate"][1][ci])
    u, zu = oracle.linear(b, W["up"][0][ci], W["up"][1][ci])
    hr, zh = oracle.swiglu(g, u, zg, zu)
    check(_np(act)[:, ci], hr, zh, name=f"{name} SwiGLU activation", tight=tight_eps(H, mfma, norm=True),
          rel_l2=SWIGLU_ROW_L2)
    ch = np.arange(H) if cols is None else cols[cols < H]
    dr, zd = oracle.linear(_np(act).astype(np.float64), W["down"][0][ch], W["down"][1][ch])
    want = x[:, ch] + dr
    zeta = zd + np.abs(x[:, ch])
    if sum32 is None:
        check(_np(h_out)[:, ch], want, zeta, name=f"{name} down + residual", tight=tight_eps(I, mfma))
    else:
        # fp32 residual sum (no fp16 rounding of its own)
        check(_np(sum32)[:, ch], want, zeta, name=f"{name} down + residual (fp32)",
              tight=tight_eps(I, mfma) - 2.0 ** -11 + 2.0 ** -22)
        s32 = _np(sum32).astype(np.float64)
        n, zn = oracle.rmsnorm(s32, eps)
        check(_np(h_out), n, zn + 2.0 ** -14, name=f"{name} output renormalisation", tight=2.0 ** -10)


def moe_routing(logits_gpu, idx, p, logits_ref, E, k, name):
    """The GPU's selection is k distinct experts per token, a valid top-k of
    the oracle logits within the GPU's own logit error, the oracle's exact
    selection wherever no near-tie allows another, and its weights sum to 1."""
    idx = np.asarray(idx)
    assert idx.min() >= 0 and idx.max() < E, f"{name}: expert id out of range"
    assert all(len(set(r)) == k for r in idx.tolist()), f"{name}: a token selected an expert twice"
    delta = np.abs(logits_gpu - logits_ref).max(axis=1)
    srt = -np.sort(-logits_ref, axis=1)
    kth = srt[:, k - 1]
    chosen = np.take_along_axis(logits_ref, idx.astype(np.int64), axis=1)
    assert np.all(chosen >= (kth - 2 * delta)[:, None] - 1e-12), f"{name}: a selection is not a valid top-k"
    decided = srt[:, k - 1] - srt[:, k] > 2 * delta + 1e-12
    ref_idx, _ = oracle.topk_route(logits_ref, k)
    for t in np.nonzero(decided)[0]:
        assert set(idx[t]) == set(ref_idx[t]), f"{name}: token {t} routed to other experts"
    assert np.all(np.abs(np.asarray(p, np.float64).sum(axis=1) - 1) <= 1e-6), f"{name}: weights do not sum to 1"
    # the slot order is rank order of the GPU's own logits (ties to the lower id)
    own = np.take_along_axis(logits_gpu, idx.astype(np.int64), axis=1)
    for t in range(idx.shape[0]):
        key = list(zip((-own[t]).tolist(), idx[t].tolist()))
        assert key == sorted(key), f"{name}: token {t} slots not in rank order"
    return decided


def moe_stages(experts, x, idx, p, expert_h, expert_out, y, name, res=None, mfma=False, norm=False,
               pairs=None, cols_i=None, cols_h=None):
    """Teacher-forced stages of the routed experts for pairs k*t + j:
    expert_h = silu(x_t Wg_e) * (x_t Wu_e) on the stage's input x (fp64 rows,
    already normalised when the layer normalises); expert_out = expert_h Wd_e
    on the GPU's own expert_h; y_t = res_t + sum_j p_tj expert_out_tj on the
    GPU's own weights and expert outputs.  pairs / cols_*: samples (all when
    None)."""
    idx = np.asarray(idx)
    T, k = idx.shape
    I = expert_h.shape[1]
    H = expert_out.shape[1]
    pairs = np.arange(T * k) if pairs is None else np.asarray(pairs)
    ci = np.arange(I) if cols_i is None else np.asarray(cols_i)
    ch = np.arange(H) if cols_h is None else np.asarray(cols_h)
    eh = np.asarray(expert_h, np.float64)
    eo = np.asarray(expert_out, np.float64)
    pe = idx.reshape(-1)[pairs]
    for e in np.unique(pe):
        sel = pairs[pe == e]
        tok = sel // k
        (gc, gs), (uc, us), (dc, ds) = experts[int(e)]
        g, zg = oracle.linear(x[tok], gc[ci], gs[ci])
        u, zu = oracle.linear(x[tok], uc[ci], us[ci])
        hr, zh = oracle.swiglu(g, u, zg, zu)
        check(eh[sel][:, ci], hr, zh, name=f"{name} expert {int(e)} SwiGLU activation",
              tight=tight_eps(x.shape[1], mfma, norm), rel_l2=SWIGLU_ROW_L2)
        dr, zd = oracle.linear(eh[sel], dc[ch], ds[ch])
        check(eo[sel][:, ch], dr, zd, name=f"{name} expert {int(e)} down", tight=tight_eps(I, mfma))
    # combine: fp32 sum of k products in slot order plus the residual, one rounding
    pw = np.asarray(p, np.float64)
    terms = pw[:, :, None] * eo.reshape(T, k, H)
    want = terms.sum(axis=1)
    zeta = np.abs(terms).sum(axis=1)
    if res is not None:
        r = np.asarray(res, np.float64)
        want = want + r
        zeta = zeta + np.abs(r)
    check(y, want, zeta, name=f"{name} combine", tight=2.0 ** -11 + (k + 2) * 2.0 ** -23)
