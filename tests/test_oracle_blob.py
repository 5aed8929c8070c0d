"""The selection finds the planted action-relevant region.

Every future frame of the synthetic workloads carries a Gaussian blob of
tokens shifted along the token-space direction that raises the action
queries' logits.  The method keeps, per frame, the tokens the frame's action
queries attend to most (Sec. 4.1 core selection), so the blob's centre must be
one of each frame's core tokens after a refresh.  Checked on the oracle's
refresh of the 8-block d = 1024 workload (1,312 tokens, 4 frames of 16 x 16).

At the 1-block d = 128 workload the same 0.5-amplitude shift does not stand
out of the per-head logit noise of two 64-wide heads (the centres rank 29th
and 35th of 64 by V), so that workload is not pinned this way.
"""
import numpy as np

import oracle as O
import workload as W


def blob_centres(inp, cfg, b, tau):
    """Frame-local index of every blob centre of sequence b at step tau, per frame."""
    out = [[] for _ in range(cfg.n_frames)]
    for bl in inp.blobs[b]:
        for f in range(cfg.n_frames):
            r = int((bl.centers[f, 0] + tau * bl.dirs[f, 0]) % cfg.frame_h)
            c = int((bl.centers[f, 1] + tau * bl.dirs[f, 1]) % cfg.frame_w)
            out[f].append(r * cfg.frame_w + c)
    return out


def test_refresh_cores_cover_the_planted_blob_centres():
    cfg = W.preset(2)
    blocks = [W.block_weights(cfg, l) for l in range(cfg.n_blocks)]
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    r = O.refresh_step(inp.x(0), blocks, inp.temb(0), cfg)
    sel = r.selection[0]
    V = r.reduced[0].V
    for f, centres in enumerate(blob_centres(inp, cfg, 0, 0)):
        core = set(int(j) for j in sel.core[f])
        for j in centres:
            rank = int((V[f] > V[f, j]).sum())
            assert j in core, f"frame {f}: blob centre {j} ranks {rank} of {cfg.n_s}"
            assert j in set(int(i) for i in sel.retained[f])
        # the blob lifts its neighbourhood too: the centre ranks in the top tenth
        assert all(int((V[f] > V[f, j]).sum()) < cfg.n_s // 10 for j in centres)
