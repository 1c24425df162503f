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


def oracle_sample_rows(logits, canvas, mask_id, n, pos0, off, step_id, seed, inv_temp, top_p=1.0):
    """Oracle reverse step for every row: (next canvas, choice, conf) as arrays."""
    B = canvas.shape[0]
    nxt = canvas.copy()
    choice = np.full((B, canvas.shape[1] - off), -1, dtype=np.int64)
    conf = np.full((B, canvas.shape[1] - off), -np.inf, dtype=np.float32)
    for b in range(B):
        nx, ch, cf = S.reverse_step(logits[b], canvas[b, off:], mask_id, n, pos0 + off, b, step_id,
                                    seed, np.float32(inv_temp), top_p)
        nxt[b, off:] = nx
        choice[b] = ch
        conf[b] = cf
    return nxt, choice, conf


def unnormalised_attention(orig):
    """An equally valid bf16 attention for the oracle: the probabilities enter the PV
    product as exp(s - max) rounded to bf16 and the row sum is divided out afterwards
    (the oracle itself normalises before rounding).  Two such evaluations bound how
    close any bf16 implementation can be expected to come to the oracle."""
    def attn(q, k, v, op=lambda x: x):
        H, Hkv, dh = q.shape[1], k.shape[1], q.shape[2]
        q, k, v = op(q), op(k), op(v)
        out = np.empty((q.shape[0], H, v.shape[2]))
        for h in range(H):
            kh = (h * Hkv) // H
            s = q[:, h, :] @ k[:, kh, :].T / np.sqrt(dh)
            e = np.exp(s - s.max(axis=-1, keepdims=True))
            out[:, h, :] = (op(e) @ v[:, kh, :]) / e.sum(axis=-1, keepdims=True)
        return out
    return attn


def within_noise_floor(got, ref, alt, what, rtol=2e-2, atol=2e-2):
    """got vs ref, judged against the spread between two valid bf16 oracle evaluations
    (ref, alt): rms error at most twice the oracle's own (plus 1e-3 of the tensor's
    rms), every element within twice the oracle's own largest deviation (and 4e-2),
    and the share of elements beyond the elementwise bar at most three times the
    oracle's own share (at least 1e-5).  atol is scaled by the tensor's rms when that
    exceeds 1."""
    got, ref, alt = (np.asarray(x, dtype=np.float64) for x in (got, ref, alt))
    rms_ref = np.sqrt((ref ** 2).mean())
    a = atol * max(1.0, rms_ref)
    err, spread = np.abs(got - ref), np.abs(alt - ref)
    bar = a + rtol * np.abs(ref)
    e_rms, s_rms = np.sqrt((err ** 2).mean()), np.sqrt((spread ** 2).mean())
    out, s_out = (err > bar).mean(), (spread > bar).mean()
    print(f"[parity] {what}: rms err {e_rms:.3g} (oracle spread {s_rms:.3g}), max {err.max():.3g} "
          f"(spread {spread.max():.3g}), beyond bar {out:.2e} (spread {s_out:.2e}), rms ref {rms_ref:.3g}")
    # the additive 1e-3 rms covers float32 summation order where the two oracle
    # evaluations happen to agree (e.g. identical rows); it is far below bf16 noise
    assert e_rms <= 2 * s_rms + 1e-3 * rms_ref, f"{what}: rms error {e_rms:.3g} above twice the bf16 floor {s_rms:.3g}"
    assert err.max() <= max(4e-2 * max(1.0, rms_ref), 2 * spread.max()), f"{what}: max error {err.max():.3g}"
    assert out <= max(1e-5, 3 * s_out), f"{what}: {out:.2e} of elements beyond the bar (floor {s_out:.2e})"
