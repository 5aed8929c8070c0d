"""Plain CPU oracle of the action-guided sparse denoising step.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import this module.  The product path never
calls it, and it shares no code with the HIP path: it consumes the same seeded
arrays from ``workload`` and nothing else.

Everything is written in the paper's order and notation (Sparse-WAM, Sec. 3.1,
Sec. 4, App. A) as slow, obviously correct numpy:

* float64 arithmetic throughout;
* explicit rounding to the storage precision (float32, or bf16 with
  round-to-nearest-even) exactly where the GPU path stores a tensor, so both
  sides see the same quantisation points;
* fp32 values wherever an integer decision (a top-k, a count) is taken, so both
  sides take the decision on identical bits.

Readings of points the paper leaves open (token order, masks, tie-breaking,
budgets, the synthetic DiT block, the mass-threshold variant) are listed in the
design notes and restated at each function.

Pins: every function here is checked in ``tests/test_oracle_*.py`` against
closed forms, invariants stated by the paper, values it prints and brute force.
The synthetic DiT block has no counterpart in the paper; it is pinned against a
composition of textbook library routines.  End-to-end step values beyond those
pins are "parity unpinned" (the paper prints no per-step numbers).
"""
from __future__ import annotations

import math
from fractions import Fraction
from dataclasses import dataclass

import numpy as np

LN_EPS = 1e-6


# ---------------------------------------------------------------------------
# storage precision
# ---------------------------------------------------------------------------
def round_f32(x) -> np.ndarray:
    """Round to float32 (the precision of every fp32 store), returned as float64."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_bf16(x) -> np.ndarray:
    """Round to bf16 with ties to even, via float32 (how the GPU stores bf16)."""
    x32 = np.ascontiguousarray(np.asarray(x, dtype=np.float64).astype(np.float32))
    bits = x32.view(np.uint32).astype(np.uint64)
    lsb = (bits >> np.uint64(16)) & np.uint64(1)
    bits = (bits + np.uint64(0x7FFF) + lsb) & np.uint64(0xFFFF0000)
    return bits.astype(np.uint32).view(np.float32).astype(np.float64)


def storage_round(dtype: str):
    """Rounding applied at every stored activation for a configuration dtype."""
    if dtype == "bf16":
        return round_bf16
    if dtype == "f32":
        return round_f32
    if dtype == "f64":          # no storage rounding (used by library-routine pins)
        return lambda x: np.asarray(x, dtype=np.float64)
    raise ValueError(dtype)


# ---------------------------------------------------------------------------
# the synthetic DiT block (adaLN-modulated pre-LN transformer block)
# ---------------------------------------------------------------------------
def silu(t):
    t = np.asarray(t, dtype=np.float64)
    return t / (1.0 + np.exp(-t))


def gelu_tanh(u):
    """0.5 u (1 + tanh(sqrt(2/pi) (u + 0.044715 u^3)))."""
    u = np.asarray(u, dtype=np.float64)
    return 0.5 * u * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (u + 0.044715 * u ** 3)))


def layer_norm(x):
    """Per-row normalisation, biased variance, eps 1e-6, no affine."""
    x = np.asarray(x, dtype=np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + LN_EPS)


def modulation(w_ada, b_ada, temb):
    """adaLN vector m = W_ada SiLU(t_emb) + b_ada, split into six d-vectors.

    Order: (shift1, scale1, gate1, shift2, scale2, gate2).  Stored as float32.
    """
    m = np.asarray(w_ada, np.float64) @ silu(temb) + np.asarray(b_ada, np.float64)
    m = round_f32(m)
    return np.split(m, 6)


def attention(q, k, v, cu_seqlens, n_heads):
    """Full bidirectional softmax attention inside each sequence.

    q, k, v: [T][N_h * hd].  Keys visible to a query are all tokens of its own
    sequence (no mask, no positional term).  Returns the output [T][N_h * hd]
    and the natural-log normaliser lambda [T][N_h] of every query row.
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    T, D = q.shape
    hd = D // n_heads
    o = np.zeros((T, D))
    lse = np.zeros((T, n_heads))
    for b in range(len(cu_seqlens) - 1):
        s0, s1 = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
        if s1 == s0:
            continue
        for h in range(n_heads):
            cols = slice(h * hd, (h + 1) * hd)
            logits = q[s0:s1, cols] @ k[s0:s1, cols].T / math.sqrt(hd)
            mx = logits.max(axis=1, keepdims=True)
            lam = mx[:, 0] + np.log(np.exp(logits - mx).sum(axis=1))
            p = np.exp(logits - lam[:, None])
            o[s0:s1, cols] = p @ v[s0:s1, cols]
            lse[s0:s1, h] = lam
    return o, lse


ROPE_BASE = 10000.0


def rope_angles(positions, hd=64, base=ROPE_BASE):
    """Rotary angles pos * base^(-2i/hd) for pairs i = 0..hd/2-1, [T][hd/2]."""
    pos = np.asarray(positions, np.float64)
    inv = base ** (-2.0 * np.arange(hd // 2, dtype=np.float64) / hd)
    return pos[:, None] * inv[None, :]


def apply_rope(x, positions, n_heads):
    """Rotary position embedding (RoFormer convention): in every head, the pair
    (x_2i, x_2i+1) is rotated by the angle of its row's position."""
    x = np.asarray(x, np.float64)
    T, D = x.shape
    hd = D // n_heads
    ang = rope_angles(positions, hd)
    c, s = np.cos(ang), np.sin(ang)
    y = x.reshape(T, n_heads, hd // 2, 2)
    a, b = y[..., 0], y[..., 1]
    out = np.stack([a * c[:, None, :] - b * s[:, None, :], a * s[:, None, :] + b * c[:, None, :]], axis=-1)
    return out.reshape(T, D)


def qk_rms_norm(x, n_heads, eps=LN_EPS):
    """RMS normalisation of every head vector, unit gain."""
    x = np.asarray(x, np.float64)
    T, D = x.shape
    y = x.reshape(T, n_heads, D // n_heads)
    return (y / np.sqrt((y * y).mean(axis=2, keepdims=True) + eps)).reshape(T, D)


def qk_post(qkv, n_heads, positions, rope, qk_norm, st):
    """Optional backbone variants on the stored q and k (v untouched): QK-norm,
    then RoPE at the rows' original positions; re-stored."""
    if not (rope or qk_norm):
        return qkv
    qkv = np.array(qkv, np.float64, copy=True)
    d = qkv.shape[1] // 3
    for sl in (slice(0, d), slice(d, 2 * d)):
        t = qkv[:, sl]
        if qk_norm:
            t = qk_rms_norm(t, n_heads)
        if rope:
            t = apply_rope(t, positions, n_heads)
        qkv[:, sl] = st(t)
    return qkv


@dataclass
class BlockTrace:
    """Intermediate tensors of one block (as stored), for scoring and tests."""
    qkv: np.ndarray   # [T][3d]
    lse: np.ndarray   # [T][N_h] float32 values
    x_mid: np.ndarray  # residual stream after the attention half


def block(x, w, temb, cu_seqlens, n_heads, dtype, positions=None, rope=False, qk_norm=False):
    """One DiT block on rows ``x`` [T][d] grouped into sequences by cu_seqlens.

    h  = LN(x) (1 + scale1) + shift1
    qkv = h W_qkv^T + b_qkv, heads of 64
    o  = softmax(q k^T / sqrt(hd)) v  inside each sequence
    x1 = x + gate1 * (o W_o^T + b_o)
    h2 = LN(x1) (1 + scale2) + shift2
    y  = x1 + gate2 * (GELU_tanh(h2 W_1^T + b_1) W_2^T + b_2)

    Every tensor the GPU stores (h, qkv, o, x1, h2, the GELU output, y) is
    rounded to the storage precision; math in between is float64.  With the
    backbone variants, q and k are QK-normed and/or rotated at ``positions``
    (the rows' original indices in their full sequences) and stored again.
    """
    st = storage_round(dtype)
    x = np.asarray(x, np.float64)
    d = x.shape[1]
    sh1, sc1, g1, sh2, sc2, g2 = modulation(w["w_ada"], w["b_ada"], temb)
    W = {k: np.asarray(v, np.float64) for k, v in w.items()}
    h = st(layer_norm(x) * (1.0 + sc1) + sh1)
    qkv = st(h @ W["w_qkv"].T + W["b_qkv"])
    qkv = qk_post(qkv, n_heads, positions, rope, qk_norm, st)
    q, k, v = qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]
    o, lse = attention(q, k, v, cu_seqlens, n_heads)
    o = st(o)
    x1 = st(x + g1 * (o @ W["w_o"].T + W["b_o"]))
    h2 = st(layer_norm(x1) * (1.0 + sc2) + sh2)
    u = st(gelu_tanh(h2 @ W["w_1"].T + W["b_1"]))
    y = st(x1 + g2 * (u @ W["w_2"].T + W["b_2"]))
    return y, BlockTrace(qkv=qkv, lse=round_f32(lse), x_mid=x1)


def block_rows(x, w, temb, cu_seqlens, rows, n_heads, dtype, positions=None, rope=False,
               qk_norm=False):
    """The block output of selected rows only (same arithmetic as ``block``).

    Keys and values need every row of the sampled rows' sequences; queries,
    the attention output, the projections and the MLP are formed for the
    sampled rows alone, so large workloads can be checked one row at a time.
    Returns ([len(rows)][d] outputs, [len(rows)][N_h] normalisers).
    """
    st = storage_round(dtype)
    x = np.asarray(x, np.float64)
    d = x.shape[1]
    hd = d // n_heads
    rows = np.asarray(rows, np.int64)
    sh1, sc1, g1, sh2, sc2, g2 = modulation(w["w_ada"], w["b_ada"], temb)
    W = {k: np.asarray(v, np.float64) for k, v in w.items()}
    cu = np.asarray(cu_seqlens, np.int64)
    out = np.zeros((len(rows), d))
    lam = np.zeros((len(rows), n_heads))
    for b in range(len(cu) - 1):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        sel = np.nonzero((rows >= s0) & (rows < s1))[0]
        if len(sel) == 0:
            continue
        h = st(layer_norm(x[s0:s1]) * (1.0 + sc1) + sh1)
        kv = st(h @ W["w_qkv"][d:].T + W["b_qkv"][d:])
        r = rows[sel]
        q = st(h[r - s0] @ W["w_qkv"][:d].T + W["b_qkv"][:d])
        if rope or qk_norm:
            pos = np.asarray(positions)
            zq = np.zeros((len(r), d))
            q = qk_post(np.concatenate([q, zq, zq], axis=1), n_heads, pos[r], rope, qk_norm, st)[:, :d]
            zk = np.zeros((s1 - s0, d))
            kv = np.concatenate([zk, kv], axis=1)
            kv = qk_post(kv, n_heads, pos[s0:s1], rope, qk_norm, st)[:, d:]
        k, v = kv[:, :d], kv[:, d:]
        o = np.zeros((len(r), d))
        for hh in range(n_heads):
            cols = slice(hh * hd, (hh + 1) * hd)
            logits = q[:, cols] @ k[:, cols].T / math.sqrt(hd)
            mx = logits.max(axis=1, keepdims=True)
            lm = mx[:, 0] + np.log(np.exp(logits - mx).sum(axis=1))
            o[:, cols] = np.exp(logits - lm[:, None]) @ v[:, cols]
            lam[sel, hh] = lm
        o = st(o)
        x1 = st(x[r] + g1 * (o @ W["w_o"].T + W["b_o"]))
        h2 = st(layer_norm(x1) * (1.0 + sc2) + sh2)
        u = st(gelu_tanh(h2 @ W["w_1"].T + W["b_1"]))
        out[sel] = st(x1 + g2 * (u @ W["w_2"].T + W["b_2"]))
    return out, round_f32(lam)


# ---------------------------------------------------------------------------
# action-to-future scoring (Sec. 4.1 frame-aligned score; App. A.1, A.2)
# ---------------------------------------------------------------------------
def frame_groups(n_act: int, n_frames: int):
    """Consecutive query groups I_f of size H/F (App. A.1, action-frame groups)."""
    if n_act % n_frames:
        raise ValueError("H must be divisible by F")
    g = n_act // n_frames
    return [list(range(f * g, (f + 1) * g)) for f in range(n_frames)]


def alpha_weights(g: int) -> np.ndarray:
    """Centre-weighted query weights of one group (App. B.2).

    Queries in the central half (|i - (g-1)/2| < g/4) weigh twice the outer
    quarters; weights are normalised to sum to one.
    """
    c = (g - 1) / 2.0
    w = np.array([2.0 if abs(i - c) < g / 4.0 else 1.0 for i in range(g)])
    return w / w.sum()


def score(q_act, k_fut, lse_act, n_frames, n_s, n_heads, alpha=None):
    """Spatial score S(f, j) of one layer from reused normalisers (App. A.2).

    S(f,j) = (1/N_h) sum_{i in I_f} sum_h alpha_{f,i} exp(x_h(i,f,j) - lambda_h(i))
    with x_h the scaled query-key logit.  q_act [H][N_h*hd], k_fut
    [F*N_s][N_h*hd], lse_act [H][N_h].  Returns float32 values [F][N_s].
    """
    q = np.asarray(q_act, np.float64)
    k = np.asarray(k_fut, np.float64)
    lam = np.asarray(lse_act, np.float64)
    H, D = q.shape
    hd = D // n_heads
    groups = frame_groups(H, n_frames)
    if alpha is None:
        alpha = np.stack([alpha_weights(len(I)) for I in groups])
    S = np.zeros((n_frames, n_s))
    for f, I in enumerate(groups):
        kf = k[f * n_s:(f + 1) * n_s]
        for a, i in enumerate(I):
            for h in range(n_heads):
                cols = slice(h * hd, (h + 1) * hd)
                x = kf[:, cols] @ q[i, cols] / math.sqrt(hd)
                S[f] += alpha[f, a] * np.exp(x - lam[i, h])
    return round_f32(S / n_heads)


def lse_all_keys(q_act, k_all, n_heads):
    """lambda_h(i) over every visible key (the full sequence), float32 values."""
    q = np.asarray(q_act, np.float64)
    k = np.asarray(k_all, np.float64)
    H, D = q.shape
    hd = D // n_heads
    out = np.zeros((H, n_heads))
    for h in range(n_heads):
        cols = slice(h * hd, (h + 1) * hd)
        x = q[:, cols] @ k[:, cols].T / math.sqrt(hd)
        mx = x.max(axis=1, keepdims=True)
        out[:, h] = mx[:, 0] + np.log(np.exp(x - mx).sum(axis=1))
    return round_f32(out)


# ---------------------------------------------------------------------------
# layer quality, core score and anchor key (Sec. 4.1; App. A.1)
# ---------------------------------------------------------------------------
def layer_quality(S_all):
    """R_l, E_l, Q_l = R_l (1 - E_l) per layer from S_all [L][F][N_s].

    R_l = (1/F) sum_{f,j} S; Sbar = S / sum_j S (0 where a frame sums to 0);
    E_l = -sum Sbar log Sbar / (F log N_s) with 0 log 0 = 0.
    Returns float64 arrays (R, E, Q).
    """
    S_all = np.asarray(S_all, np.float64)
    L, F, N_s = S_all.shape
    R = np.zeros(L)
    E = np.zeros(L)
    for l in range(L):
        tot = S_all[l].sum(axis=1)
        R[l] = tot.sum() / F
        ent = 0.0
        for f in range(F):
            if tot[f] == 0.0:
                continue
            p = S_all[l, f] / tot[f]
            nz = p > 0
            ent -= float((p[nz] * np.log(p[nz])).sum())
        E[l] = ent / (F * math.log(N_s))
    Q = R * (1.0 - E)
    return R, E, Q


def topk(scores, candidates, k):
    """Indices of the k best candidates, returned in ascending index order.

    Order: score descending, then index ascending (lowest index wins a tie).
    ``scores`` is indexed by position; comparison is on the given values.
    """
    cand = np.asarray(sorted(int(c) for c in candidates), dtype=np.int64)
    if k > len(cand):
        raise ValueError("k exceeds the candidate count")
    s = np.asarray(scores)[cand]
    order = np.lexsort((cand, -s.astype(np.float64)))
    return np.sort(cand[order[:k]])


def core_layers(Q, k_layer):
    """L_core: the min(K_layer, L) layers of largest fp32 Q, lowest index on ties."""
    Q32 = np.asarray(Q, np.float64).astype(np.float32)
    k = min(k_layer, len(Q32))
    return topk(Q32, range(len(Q32)), k)


def weighted_mean(S_all, Q, layers):
    """sum_{l in layers} Q_l S_l / sum Q_l (float64); unweighted mean if sum Q = 0."""
    S_all = np.asarray(S_all, np.float64)
    Q = np.asarray(Q, np.float64)
    layers = list(layers)
    den = float(sum(Q[l] for l in layers))
    if den == 0.0:
        return sum(S_all[l] for l in layers) / len(layers)
    return sum(Q[l] * S_all[l] for l in layers) / den


def anchor_key(V_all, cv_penalty=1.0):
    """A_j = mu_j / (1 + c CV_j), CV_j = Std_f / mu_j (population std); 0 if mu_j = 0."""
    V_all = np.asarray(V_all, np.float64)
    F = V_all.shape[0]
    mu = V_all.sum(axis=0) / F
    sd = np.sqrt(((V_all - mu) ** 2).sum(axis=0) / F)
    A = np.zeros_like(mu)
    nz = mu != 0.0
    cv = sd[nz] / mu[nz]
    A[nz] = mu[nz] / (1.0 + cv_penalty * cv)
    return A


@dataclass
class Reduced:
    R: np.ndarray
    E: np.ndarray
    Q: np.ndarray        # float32 values
    L_core: np.ndarray
    V: np.ndarray        # [F][N_s] float32 values
    V_all: np.ndarray    # [F][N_s] float64
    A: np.ndarray        # [N_s] float32 values


def score_reduce(S_all, k_layer=6, cv_penalty=1.0):
    """Layer quality -> L_core -> core score V and anchor key A (Sec. 4.1, App. A.1)."""
    R, E, Q = layer_quality(S_all)
    Lc = core_layers(Q, k_layer)
    V = round_f32(weighted_mean(S_all, Q, Lc))
    V_all = weighted_mean(S_all, Q, range(len(Q)))
    A = round_f32(anchor_key(V_all, cv_penalty))
    return Reduced(R=R, E=E, Q=round_f32(Q), L_core=Lc, V=V, V_all=V_all, A=A)


# ---------------------------------------------------------------------------
# selection (Sec. 4.1 pool / core / anchors; App. A.1 anchor availability)
# ---------------------------------------------------------------------------
MASS_SCALE_BITS = 40


def threshold_fraction(theta: float) -> Fraction:
    """Mass threshold as an exact fraction with denominator dividing 1000.

    The threshold is a float32 configuration value; 1000 times it is formed
    exactly (Fraction arithmetic) and rounded to the nearest integer (a float32
    value is a dyadic rational, so 1000 theta is never halfway between
    integers).  A numerator of 0 (theta below 0.0005) is allowed."""
    exact = Fraction(float(np.float32(theta))) * 1000
    num = math.floor(exact + Fraction(1, 2))
    return Fraction(num, 1000)


def mass_code(val) -> int:
    """Integer code of one fp32 score for the mass rule: floor(V 2^40) of the
    exact fp32 value, 0 for V <= 0 and 2^40 for V >= 1."""
    val = float(np.float32(val))
    if not val > 0.0:
        return 0
    if val >= 1.0:
        return 1 << MASS_SCALE_BITS
    return math.floor(Fraction(val) * (1 << MASS_SCALE_BITS))


def mass_count(v_row, pool, theta):
    """Per-frame core count from a score-mass threshold (ragged extension).

    q_j = mass_code(V(f,j)), T = sum over all positions, and candidates of the
    pool are walked in top-k order; k is the smallest count >= 1 whose prefix
    reaches theta * T, capped at the pool size.
    """
    frac = threshold_fraction(theta)
    v32 = np.asarray(v_row, dtype=np.float32)
    q = [mass_code(val) for val in v32]
    T = sum(q)
    ranked = sorted((int(j) for j in pool), key=lambda j: (-float(v32[j]), j))
    run = 0
    for k, j in enumerate(ranked, start=1):
        run += q[j]
        if frac.denominator * run >= frac.numerator * T:
            return k
    return len(ranked)


@dataclass
class Selection:
    pool: np.ndarray          # P
    core: list                # C_f per frame
    unused: np.ndarray        # E
    anchors: np.ndarray       # S
    retained: list            # R_f = C_f u S, ascending, per frame


def select(V, A, k_core, k_anchor, mass_threshold=0.0):
    """Pool P, per-frame cores C_f, shared anchors S and retained sets R_f.

    P   = TopK_j(max_f V(f,j), N_s - K_s)
    C_f = TopK_{j in P}(V(f,j), K_c)   (K_c from the mass rule if threshold > 0)
    E   = J minus the union of the C_f
    S   = TopK_{j in E}(A_j, K_s)
    R_f = C_f u S in ascending order.
    Inputs are fp32 values; comparisons are on them.
    """
    V = np.asarray(V, np.float32)
    A = np.asarray(A, np.float32)
    F, N_s = V.shape
    if not (0 <= k_anchor <= N_s) or (mass_threshold <= 0 and k_core + k_anchor > N_s):
        raise ValueError("budgets exceed the frame size")
    J = np.arange(N_s)
    m = V.max(axis=0)
    P = topk(m, J, N_s - k_anchor)
    core = []
    for f in range(F):
        kc = mass_count(V[f], P, mass_threshold) if mass_threshold > 0 else k_core
        core.append(topk(V[f], P, kc))
    used = np.zeros(N_s, bool)
    for c in core:
        used[c] = True
    E = J[~used]
    S = topk(A, E, k_anchor)
    retained = [np.union1d(c, S) for c in core]
    return Selection(pool=P, core=core, unused=E, anchors=S, retained=retained)


# ---------------------------------------------------------------------------
# random-selection baseline (the component ablation compares against tokens
# chosen at random at the same per-frame budget)
# ---------------------------------------------------------------------------
PHILOX_M = (0xD2E7470EE14C6C93, 0xCA5A826395121157)   # Philox4x64 round multipliers
PHILOX_W = (0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B)   # Philox4x64 key increments
_M32 = np.uint64(0xFFFFFFFF)


def _mulhilo64(a, b):
    """(high, low) 64-bit halves of the 128-bit product of uint64 arrays."""
    a = np.asarray(a, np.uint64)
    b = np.uint64(b)
    a0, a1 = a & _M32, a >> np.uint64(32)
    b0, b1 = b & _M32, b >> np.uint64(32)
    p00, p01, p10, p11 = a0 * b0, a0 * b1, a1 * b0, a1 * b1
    mid = (p00 >> np.uint64(32)) + (p01 & _M32) + (p10 & _M32)
    hi = p11 + (p01 >> np.uint64(32)) + (p10 >> np.uint64(32)) + (mid >> np.uint64(32))
    return hi, a * b


def philox4x64_10(counter, key):
    """Philox4x64 with 10 rounds (the counter-based generator of Salmon et al.,
    SC 2011): each round multiplies words 0 and 2 by the round constants,
    crosses the halves with words 1 and 3 and the key, and bumps the key by
    the Weyl increments.  counter: [n][4] uint64, key: 2 ints -> [n][4]."""
    x = [np.asarray(c, np.uint64).copy() for c in np.asarray(counter, np.uint64).T]
    k0, k1 = int(key[0]) & ((1 << 64) - 1), int(key[1]) & ((1 << 64) - 1)
    with np.errstate(over="ignore"):
        for _ in range(10):
            hi0, lo0 = _mulhilo64(x[0], PHILOX_M[0])
            hi1, lo1 = _mulhilo64(x[2], PHILOX_M[1])
            x = [hi1 ^ x[1] ^ np.uint64(k0), lo1, hi0 ^ x[3] ^ np.uint64(k1), lo0]
            k0 = (k0 + PHILOX_W[0]) & ((1 << 64) - 1)
            k1 = (k1 + PHILOX_W[1]) & ((1 << 64) - 1)
    return np.stack(x, axis=1)


def random_keys(seed, n_seqs, F, N_s):
    """Uniform keys in [0, 1) on the float32 grid for every (sequence, frame,
    position): word 0 of Philox4x64-10 at counter (index, 0, 0, 0), key
    (seed, 0), top 24 bits scaled by 2^-24.  [n_seqs][F][N_s] float32."""
    n = n_seqs * F * N_s
    ctr = np.zeros((n, 4), np.uint64)
    ctr[:, 0] = np.arange(n, dtype=np.uint64)
    w = philox4x64_10(ctr, (seed, 0))[:, 0]
    u = (w >> np.uint64(40)).astype(np.float64) * 2.0 ** -24
    return u.astype(np.float32).reshape(n_seqs, F, N_s)


def random_selection(keys, k_ret):
    """Per frame the k_ret positions of largest key (ties to the lower index): a uniformly random subset of the frame, independent across
    frames; expressed as the selection with V = keys, K_c = k_ret, K_s = 0."""
    keys = np.asarray(keys, np.float32)
    return select(keys, np.zeros(keys.shape[1], np.float32), k_ret, 0)


# ---------------------------------------------------------------------------
# packing metadata, pack and scatter (Sec. 4.2 compact execution)
# ---------------------------------------------------------------------------
def keep_mask(cfg, retained_per_seq):
    """Keep flags over the concatenated full sequences: context and action rows
    always kept, future (f, j) kept iff j in R_f of its sequence."""
    out = []
    for b in range(cfg.batch):
        m = np.zeros(cfg.l_full, bool)
        m[:cfg.n_ctx] = True
        m[cfg.n_ctx + cfg.n_fut:] = True
        for f, Rf in enumerate(retained_per_seq[b]):
            m[cfg.n_ctx + f * cfg.n_s + np.asarray(Rf, np.int64)] = True
        out.append(m)
    return np.concatenate(out)


@dataclass
class PackMap:
    pack_pos: np.ndarray    # [B*L_full] int32, -1 where pruned
    gather: np.ndarray      # [T_pack] int32 original row of each packed row
    cu_seqlens: np.ndarray  # [B+1] int32 packed sequence offsets


def pack_map(mask, batch):
    """Exclusive prefix sum of the keep flags in original order."""
    mask = np.asarray(mask, bool)
    pos = np.cumsum(mask) - 1
    pack_pos = np.where(mask, pos, -1).astype(np.int32)
    gather = np.nonzero(mask)[0].astype(np.int32)
    per = mask.reshape(batch, -1).sum(axis=1)
    cu = np.concatenate([[0], np.cumsum(per)]).astype(np.int32)
    return PackMap(pack_pos=pack_pos, gather=gather, cu_seqlens=cu)


def pack(x_full, pm: PackMap):
    return np.asarray(x_full, dtype=np.float64)[pm.gather]


def unpack(y_packed, x_full, pm: PackMap):
    """Pruned rows keep x_full unchanged; retained rows take the packed output."""
    y = np.array(x_full, dtype=np.float64, copy=True)
    y[pm.gather] = y_packed
    return y


# ---------------------------------------------------------------------------
# steps and the schedule (Sec. 4.2)
# ---------------------------------------------------------------------------
def dense_cu(cfg):
    return (np.arange(cfg.batch + 1) * cfg.l_full).astype(np.int32)


@dataclass
class RefreshResult:
    y: np.ndarray
    S_all: np.ndarray      # [B_s][L][F][N_s] float32 values (B_s = scored sequences)
    reduced: list          # per scored sequence Reduced
    selection: list        # per scored sequence Selection
    packmap: PackMap


def dense_positions(cfg):
    """Original index of every full-layout row inside its sequence."""
    return np.tile(np.arange(cfg.l_full), cfg.batch)


def run_blocks(x, model, temb, cu, cfg, trace_cb=None, positions=None):
    y = np.asarray(x, np.float64)
    rope, qkn = bool(getattr(cfg, "rope", 0)), bool(getattr(cfg, "qk_norm", 0))
    if positions is None:
        positions = dense_positions(cfg)
    for l, w in enumerate(model):
        y, tr = block(y, w, temb, cu, cfg.n_heads, cfg.dtype, positions, rope, qkn)
        if trace_cb is not None:
            trace_cb(l, tr)
    return y


def dense_step(x_full, model, temb, cfg):
    """The ordinary dense step over every token (no scoring)."""
    return run_blocks(x_full, model, temb, dense_cu(cfg), cfg)


def n_scored(cfg):
    """Sequences whose attention is scored: with guidance pairs only the
    conditional half [0, B/2) (the selection statistics come from the dense
    conditional forward, Sec. 4.2 / App. B.2); otherwise every sequence."""
    return cfg.batch // 2 if getattr(cfg, "cfg_pairs", 0) else cfg.batch


def layer_scores(cfg, tr: BlockTrace):
    """S_l for every scored sequence from one block's stored q, k and lambda."""
    d = cfg.d_model
    out = []
    for b in range(n_scored(cfg)):
        base = b * cfg.l_full
        act = slice(base + cfg.n_ctx + cfg.n_fut, base + cfg.l_full)
        fut = slice(base + cfg.n_ctx, base + cfg.n_ctx + cfg.n_fut)
        out.append(score(tr.qkv[act, :d], tr.qkv[fut, d:2 * d], tr.lse[act],
                         cfg.n_frames, cfg.n_s, cfg.n_heads))
    return out


def selection_from_scores(cfg, S_all):
    """Reduce and select every scored sequence; with guidance pairs the
    unconditional partner b + B/2 keeps the positions selected for b."""
    reduced, sel = [], []
    P = n_scored(cfg)
    for b in range(P):
        r = score_reduce(S_all[b], cfg.k_layer, cfg.cv_penalty)
        reduced.append(r)
        sel.append(select(r.V, r.A, cfg.k_core, cfg.k_anchor, cfg.mass_threshold))
    retained = [sel[b % P].retained for b in range(cfg.batch)]
    pm = pack_map(keep_mask(cfg, retained), cfg.batch)
    return reduced, sel, pm


def refresh_step(x_full, model, temb, cfg):
    """Full step: dense forward, per-layer scores, reduce, select, pack map."""
    S_all = np.zeros((n_scored(cfg), len(model), cfg.n_frames, cfg.n_s))

    def cb(l, tr):
        for b, S in enumerate(layer_scores(cfg, tr)):
            S_all[b, l] = S

    y = run_blocks(x_full, model, temb, dense_cu(cfg), cfg, cb)
    reduced, sel, pm = selection_from_scores(cfg, S_all)
    return RefreshResult(y=y, S_all=S_all, reduced=reduced, selection=sel, packmap=pm)


def sparse_step(x_full, model, temb, cfg, pm: PackMap):
    """Blocks on the packed sequence only; pruned rows carry x_full unchanged."""
    xp = pack(x_full, pm)
    # packed rows keep the positions of their original rows (Sec. 4.2)
    yp = run_blocks(xp, model, temb, pm.cu_seqlens, cfg, positions=pm.gather % cfg.l_full)
    return unpack(yp, x_full, pm)


def is_refresh(tau, reuse_R):
    return tau % reuse_R == 0


def run_schedule(cfg, model, x_of_tau, temb_of_tau, n_steps=None, refresh_at=None):
    """Open-loop schedule: refresh at tau mod R == 0 (or at the steps listed in
    ``refresh_at``, e.g. {0} for the paper's default of one full step per
    action chunk; App. C.2 compares such schedules), sparse otherwise.

    Returns per-step outputs and the refresh results (keyed by tau)."""
    n = cfg.n_steps if n_steps is None else n_steps
    ys, refreshes, cur = [], {}, None
    for tau in range(n):
        x = x_of_tau(tau)
        t = temb_of_tau(tau)
        full = is_refresh(tau, cfg.reuse_R) if refresh_at is None else tau in refresh_at
        if full:
            r = refresh_step(x, model, t, cfg)
            refreshes[tau] = r
            cur = r.packmap
            ys.append(r.y)
        else:
            ys.append(sparse_step(x, model, t, cfg, cur))
    return ys, refreshes


# ---------------------------------------------------------------------------
# diagnostics (App. C: cross-step and cross-frame attention overlap)
# ---------------------------------------------------------------------------
def overlap(P, Q):
    """Overlap(P, Q) = sum_i min(P_i, Q_i) of two spatial distributions, each
    non-negative map first normalised to unit mass (a map of zero mass counts
    as all zeros, overlap 0)."""
    P = np.asarray(P, np.float64).ravel()
    Q = np.asarray(Q, np.float64).ravel()
    sp, sq = P.sum(), Q.sum()
    if sp <= 0 or sq <= 0:
        return 0.0
    return float(np.minimum(P / sp, Q / sq).sum())
