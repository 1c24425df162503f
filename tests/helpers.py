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


def rows_close(got, ref, rtol, atol, what, stats=None):
    """Elementwise |got - ref| <= atol + rtol |ref| for every element.

    Prints the tap's figures (max and rms error, rms of the reference, elements outside
    the bound) and, when ``stats`` is a list, appends them to it as well.
    """
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    err = np.abs(got - ref)
    rms_ref = np.sqrt((ref ** 2).mean())
    bad = err > atol + rtol * np.abs(ref)
    rec = dict(what=what, max_err=float(err.max()), rms_err=float(np.sqrt((err ** 2).mean())),
               rms_ref=float(rms_ref), outside=int(bad.sum()), size=int(bad.size))
    print(f"[parity] {what}: max|err| {rec['max_err']:.3g} rms err {rec['rms_err']:.3g} "
          f"rms ref {rms_ref:.3g} outside {rec['outside']}/{rec['size']}", flush=True)
    if stats is not None:
        stats.append(rec)
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


def gpu_generated_weights(cfg, perturb=True, keep=None):
    """The seeded weights of ``cfg`` generated on the GPU (fast at full size): device
    tensors for the model, and float64 host arrays for the oracle (same values) of the
    tensors whose name ``keep`` accepts (all when ``keep`` is None), as a dict."""
    dev_t, host = [], {}
    for i, spec in enumerate(synth.weight_specs(cfg)):
        t = synth.make_tensor(cfg, i, spec, device=dev(), perturb=perturb)
        dev_t.append(t)
        if keep is None or keep(spec[0]):
            host[spec[0]] = t.to(torch.float64).cpu().numpy()
    return dev_t, host
