"""GPU parity of the pretraining objective (T-ANELBO with gamma = 0) against the oracle."""
import numpy as np
import pytest
import torch

import synth
from helpers import dev, gpu_model, oracle_net
from oracle import train

tadm = pytest.importorskip("paper_2609_37924_amd")
pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,overrides,B,L,rtol", [
    ("tiny", {}, 3, 24, 1e-4),
    ("tiny", dict(n_kv_heads=2), 4, 40, 1e-4),
    ("small", dict(vocab=4096, n_anchor=2, n_denoise=1), 2, 64, 2e-2),
])
def test_train_loss_matches_oracle(name, overrides, B, L, rtol):
    """Corrupted pair bit-exact, masked counts exact, per-row loss within the bar (fp32:
    1e-4 relative; bf16: 2e-2), for the library's own training times plus a fresh-anchor
    row, a fully stale row and a row with nothing masked."""
    cfg = synth.get_config(name, **overrides)
    V = cfg["vocab"]
    tensors = synth.make_weights(cfg, perturb=name == "tiny")
    x = torch.randint(0, V, (B, L), generator=torch.Generator().manual_seed(B * L), dtype=torch.int32)
    t, ts, _, _, _ = tadm.tadm_stale_times(B, 17, 3, 1e-3)
    t[0], ts[0] = np.float32(0.6), np.float32(0.6)            # fresh anchor
    t[1], ts[1] = np.float32(0.3), np.float32(1.0)            # anchor on an all-mask canvas
    if B > 3:
        t[3], ts[3] = np.float32(1e-7), np.float32(0.2)       # nothing masked in z_t
    m = gpu_model(cfg, tensors, B, L)
    try:
        loss = torch.empty(B, device=dev())
        n = torch.empty(B, dtype=torch.int32, device=dev())
        zt = torch.empty(B, L, dtype=torch.int32, device=dev())
        zs = torch.empty(B, L, dtype=torch.int32, device=dev())
        tadm.tadm_train_loss(m, x.to(dev()), B, L, torch.from_numpy(t).to(dev()), torch.from_numpy(ts).to(dev()),
                             1e-3, 99, 4, loss, n, zt, zs)
        torch.cuda.synchronize()
        got = loss.cpu().numpy().astype(np.float64)
    finally:
        tadm.tadm_model_destroy(m)
    net = oracle_net(cfg, tensors)
    ref, rzt, rzs, rn = train.train_loss(net, x.numpy(), t, ts, 1e-3, 99, 4)
    np.testing.assert_array_equal(zt.cpu().numpy(), rzt)
    np.testing.assert_array_equal(zs.cpu().numpy(), rzs)
    np.testing.assert_array_equal(n.cpu().numpy(), rn)
    print(f"[parity] {name} losses got {got} ref {ref}")
    assert np.all(np.abs(got - ref) <= rtol * np.abs(ref) + 1e-6), (got, ref)
    if B > 3:
        assert got[3] == 0.0
