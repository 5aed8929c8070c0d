"""Shared test plumbing: device copies of workload arrays and error metrics."""
import numpy as np
import torch

import workload as W


def act_dtype(cfg):
    return torch.bfloat16 if cfg.dtype == "bf16" else torch.float32


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to("cuda:0", dtype=dtype) if dtype is not None else t.to("cuda:0")


def host(t):
    return t.detach().float().cpu().double().numpy() if t.dtype == torch.bfloat16 else \
        t.detach().cpu().numpy().astype(np.float64) if t.is_floating_point() else t.detach().cpu().numpy()


def maxrel(a, b):
    """||a - b||_inf / ||b||_inf."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.abs(b).max()
    return float(np.abs(a - b).max() / (den if den > 0 else 1.0))


def rowwise_maxrel(a, b):
    """max over rows (last axis) of ||a_r - b_r||_inf / ||b_r||_inf."""
    a = np.asarray(a, np.float64).reshape(-1, np.shape(a)[-1])
    b = np.asarray(b, np.float64).reshape(-1, np.shape(b)[-1])
    den = np.abs(b).max(axis=1)
    den[den == 0] = 1.0
    return float((np.abs(a - b).max(axis=1) / den).max())


def device_blocks(cfg, blocks):
    dt = act_dtype(cfg)
    return [{k: dev(v, dt) for k, v in b.items()} for b in blocks]


def model_for(cfg, n_blocks=None):
    from paper_2609_38984_amd import swam
    n = cfg.n_blocks if n_blocks is None else n_blocks
    blocks = [W.block_weights(cfg, l) for l in range(n)]
    dblocks = device_blocks(cfg, blocks)
    return blocks, dblocks, swam.Model(dblocks, act_dtype(cfg))


def lse_from_qkv(qkv, cu, rows, n_heads):
    """lambda[r][h] = log sum_j exp(q_h(r) . k_h(j) / 8) over every key j of the
    sequence that holds row r, in float64 from a QKV buffer [rows][3][N_h][64]
    (the normaliser the attention kernel exports, recomputed from the very q
    and k it read)."""
    qkv = np.asarray(qkv, np.float64)
    d = n_heads * 64
    cu = np.asarray(cu, np.int64)
    out = np.empty((len(rows), n_heads))
    for i, r in enumerate(rows):
        b = int(np.searchsorted(cu, r, side="right") - 1)
        k = qkv[cu[b]:cu[b + 1], d:2 * d].reshape(-1, n_heads, 64)
        q = qkv[r, :d].reshape(n_heads, 64)
        x = np.einsum("he,jhe->hj", q, k) / 8.0
        m = x.max(axis=1, keepdims=True)
        out[i] = (m[:, 0] + np.log(np.exp(x - m).sum(axis=1)))
    return out
