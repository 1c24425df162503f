"""The allocation-free sampler entry point (tadm_sample_noalloc) against tadm_sample.

Through the C ABI: two calls in a row on one model, the second with a smaller input,
in each step mode it supports (confidence-ranked with one count or per-row counts,
nucleus, remasking), with and without caller buffers for the tokens and
confidences; results equal tadm_sample's bit for bit.  Sizes beyond the fixed scratch
and the entropy mode are rejected before any device work.
"""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

tadm = pytest.importorskip("paper_2609_37924_amd")

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def _case(V, B, L, off, seed):
    g = torch.Generator().manual_seed(seed)
    canvas = torch.randint(0, V, (B, L), generator=g, dtype=torch.int32)
    canvas[:, off:][torch.rand(B, L - off, generator=g) < 0.6] = V
    logits = synth.make_logits(B * (L - off), V, seed=seed, std=2.0).view(B, L - off, V)
    return logits.cuda(), canvas.cuda()


def _args(mode, B, n_rows_keep):
    if mode == "ranked":
        return tadm.step_args(5, 16, 7, 11, 0xABCDEF, 1.0)
    if mode == "rows":
        n = torch.arange(1, B + 1, dtype=torch.int32, device="cuda") * 3
        n_rows_keep.append(n)
        return tadm.step_args(5, 16, 0, 12, 0xABCDEF, 1.0, n_unmask_rows=n)
    if mode == "nucleus":
        return tadm.step_args(5, 16, 7, 13, 0xABCDEF, float(np.float32(1 / 0.9)), top_p=0.9)
    if mode == "remask":
        return tadm.step_args(5, 16, 0, 14, 0xABCDEF, 1.0, remask=(0.3, 0.04))
    raise ValueError(mode)


@pytest.mark.parametrize("mode", ["ranked", "rows", "nucleus", "remask"])
def test_noalloc_sampler_equals_sample(mode):
    V = 32768
    m = tadm.tadm_model_create(tadm.make_config(synth.get_config("tiny", vocab=V), max_batch=4, max_seq=512))
    tadm.tadm_set_stream(m, torch.cuda.current_stream().cuda_stream)
    keep = []
    try:
        # the second call is smaller than the first: nothing of the first may leak into it
        for call, (B, L, off) in enumerate(((4, 300, 12), (2, 40, 5))):
            print(f"[no-alloc] mode={mode} call={call} B={B} L={L} off={off} V={V}", flush=True)
            logits, canvas = _case(V, B, L, off, 100 * call + len(mode))
            args = _args(mode, B, keep)
            ref_next = torch.empty_like(canvas)
            ref_choice = torch.empty(B, L - off, dtype=torch.int32, device="cuda")
            ref_conf = torch.empty(B, L - off, dtype=torch.float32, device="cuda")
            tadm.tadm_sample(m, logits, canvas, B, L, off, 9, args, ref_next, ref_choice, ref_conf)
            got_next = torch.empty_like(canvas)
            got_choice = torch.empty_like(ref_choice)
            got_conf = torch.empty_like(ref_conf)
            tadm.tadm_sample_noalloc(m, logits, canvas, B, L, off, 9, args, got_next, got_choice, got_conf)
            got_next2 = torch.full_like(canvas, -7)
            tadm.tadm_sample_noalloc(m, logits, canvas, B, L, off, 9, args, got_next2)  # tokens in the scratch
            torch.cuda.synchronize()
            assert torch.equal(got_next, ref_next)
            assert torch.equal(got_next2, ref_next)
            assert torch.equal(got_choice, ref_choice)
            assert torch.equal(got_conf.view(torch.int32), ref_conf.view(torch.int32))
            masked = canvas[:, off:] == V
            assert masked.any() and (ref_choice[masked] >= 0).all()
    finally:
        tadm.tadm_model_destroy(m)


def test_noalloc_sampler_rejects_what_it_cannot_hold():
    V = 64
    m = tadm.tadm_model_create(tadm.make_config(synth.get_config("tiny", vocab=V), max_batch=17, max_seq=4096))
    try:
        B, L = 17, 4000  # 68000 positions > TADM_NOALLOC_MAX_POSITIONS
        assert B * L > tadm.NOALLOC_MAX_POSITIONS
        dummy_f = torch.zeros(1, device="cuda")
        dummy_i = torch.zeros(1, dtype=torch.int32, device="cuda")
        args = tadm.step_args(1, 1, 1, 0, 0, 1.0)
        with pytest.raises(tadm.TadmError) as e:
            tadm.tadm_sample_noalloc(m, dummy_f, dummy_i, B, L, 0, 0, args, dummy_i)
        assert e.value.status == tadm.TADM_ERR_INVALID
        ent = tadm.step_args(1, 1, 0, 0, 0, 1.0, entropy_eta=0.1)
        with pytest.raises(tadm.TadmError) as e:
            tadm.tadm_sample_noalloc(m, dummy_f, dummy_i, 1, 8, 0, 0, ent, dummy_i)
        assert e.value.status == tadm.TADM_ERR_UNSUPPORTED
    finally:
        tadm.tadm_model_destroy(m)
