"""Shared plumbing of the GPU parity tests (seeded inputs, model handles, oracle runs)."""
import numpy as np
import torch

import synth
from oracle import network as N, sampler as S


def dev():
    return torch.device("cuda:0")


def oracle_net(cfg, tensors):
    specs = synth.weight_specs(cfg)
    return N.Network(N.Weights(cfg, [s[0] for s in specs], tensors))


def gpu_model(cfg, tensors, max_batch, max_seq):
    import paper_2609_37924_amd as tadm
    m = tadm.load_model(cfg, [t.to(dev()) for t in tensors], max_batch=max_batch, max_seq=max_seq,
                        stream=torch.cuda.current_stream().cuda_stream)
    return m


def rows_close(got, ref, rtol, atol, what, tail=0.0, max_err=None, scale_atol=False):
    """Elementwise |got - ref| <= atol + rtol |ref|.

    ``tail``: fraction of elements allowed beyond the bound (bf16 rounding noise),
    provided every element stays within ``max_err``.  ``scale_atol``: atol is taken
    relative to the rms of ``ref`` (for tensors whose scale is far from 1).
    """
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    err = np.abs(got - ref)
    rms_ref = np.sqrt((ref ** 2).mean())
    a = atol * rms_ref if scale_atol else atol
    bad = err > a + rtol * np.abs(ref)
    print(f"[parity] {what}: max|err| {err.max():.3g} rms err {np.sqrt((err ** 2).mean()):.3g} "
          f"rms ref {rms_ref:.3g} outside {int(bad.sum())}/{bad.size}")
    if tail and bad.mean() <= tail and (max_err is None or err.max() <= max_err):
        return
    if bad.any():
        idx = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {int(bad.sum())}/{bad.size} outside rtol={rtol} atol={atol}; "
                             f"first at {tuple(idx)}: got {got[tuple(idx)]} ref {ref[tuple(idx)]}; "
                             f"max err {err.max():.3g}")


def oracle_step(net, canvas_row, pos, cache, off):
    """Oracle stale step on one row: (c, h~, final hidden of canvas rows, logits fp32)."""
    c = net.shared(canvas_row, pos)
    ht = net.fuse(c, cache)
    xf = net.denoise(ht, pos)
    return c, ht, xf[off:], net.head(xf[off:]).astype(np.float32)


def oracle_sample_rows(logits, canvas, mask_id, n, pos0, off, step_id, seed, inv_temp):
    """Oracle reverse step for every row: (next canvas, choice, conf) as arrays."""
    B = canvas.shape[0]
    nxt = canvas.copy()
    choice = np.full((B, canvas.shape[1] - off), -1, dtype=np.int64)
    conf = np.full((B, canvas.shape[1] - off), -np.inf, dtype=np.float32)
    for b in range(B):
        nx, ch, cf = S.reverse_step(logits[b], canvas[b, off:], mask_id, n, pos0 + off, b, step_id,
                                    seed, np.float32(inv_temp))
        nxt[b, off:] = nx
        choice[b] = ch
        conf[b] = cf
    return nxt, choice, conf
