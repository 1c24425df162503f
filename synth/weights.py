"""Fixed tensor order and seeded random-init weights.

Matrices are stored ``[out_features, in_features]`` (row n holds the weights that
produce output feature n), vectors as ``[n]``.  The order below is the order the
C ABI expects (``tadm_weight_info`` reports the same list).

Global tensors come first, then the fusion module, then the transformer layers in
network order: shared layers, anchor layers, denoiser layers.
"""
import torch

from .configs import n_layers

STD = 0.02


def _layer_specs(cfg, li):
    d, H, Hkv, dh, F = (cfg["d_model"], cfg["n_heads"], cfg["n_kv_heads"],
                        cfg["head_dim"], cfg["d_ffn"])
    p = f"layer{li}."
    specs = [
        (p + "attn_norm", (d,), "ones"),
        (p + "wq", (H * dh, d), "normal"),
        (p + "wk", (Hkv * dh, d), "normal"),
        (p + "wv", (Hkv * dh, d), "normal"),
        (p + "wo", (d, H * dh), "normal"),
        (p + "ffn_norm", (d,), "ones"),
    ]
    if cfg["ffn_kind"] == "gelu":
        specs += [(p + "w_up", (F, d), "normal"), (p + "w_down", (d, F), "normal")]
    else:
        specs += [(p + "w_gate", (F, d), "normal"), (p + "w_up", (F, d), "normal"),
                  (p + "w_down", (d, F), "normal")]
    return specs


def _fusion_specs(cfg):
    d = cfg["d_model"]
    if cfg["fusion_kind"] == "gated_mlp":
        return [
            ("fusion.ln_s_w", (d,), "ones"), ("fusion.ln_s_b", (d,), "zeros"),
            ("fusion.ln_a_w", (d,), "ones"), ("fusion.ln_a_b", (d,), "zeros"),
            ("fusion.w1", (4 * d, 2 * d), "normal"), ("fusion.b1", (4 * d,), "zeros"),
            ("fusion.wg", (d, 2 * d), "normal"), ("fusion.bg", (d,), "zeros"),
            ("fusion.w2", (d, 4 * d), "normal"), ("fusion.b2", (d,), "zeros"),
            ("fusion.ln_o_w", (d,), "ones"), ("fusion.ln_o_b", (d,), "zeros"),
        ]
    r = cfg["fusion_rank"]
    return [
        ("fusion.w_c", (r, d), "normal"), ("fusion.w_h", (r, d), "normal"),
        ("fusion.w_q", (r, 2 * r), "normal"), ("fusion.w_k", (r, 2 * r), "normal"),
        ("fusion.w_v", (r, 2 * r), "normal"), ("fusion.w_o", (r, r), "normal"),
        ("fusion.w_f1", (2 * r, r), "normal"), ("fusion.w_f2", (r, 2 * r), "normal"),
        ("fusion.w_g1", (r, 4 * r), "normal"), ("fusion.w_g2", (1, r), "normal"),
        ("fusion.b_g", (1,), "gate_bias"), ("fusion.w_up", (d, r), "normal"),
    ]


def weight_specs(cfg):
    """List of (name, shape, init) in ABI order."""
    d, V = cfg["d_model"], cfg["vocab"]
    specs = [("embed", (V + 1, d), "normal"), ("final_norm", (d,), "ones"),
             ("w_out", (V, d), "normal")]
    specs += _fusion_specs(cfg)
    for li in range(n_layers(cfg)):
        specs += _layer_specs(cfg, li)
    return specs


def tensor_seed(seed, index):
    """Per-tensor generator seed, so any tensor can be regenerated on its own."""
    return (int(seed) * 1000003 + 7919 * int(index) + 12345) & 0x7FFFFFFFFFFFFFFF


def torch_dtype(cfg):
    return torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32


def make_tensor(cfg, index, spec, seed=None, device="cpu", perturb=False):
    name, shape, init = spec
    seed = cfg["weight_seed"] if seed is None else seed
    g = torch.Generator(device=device)
    g.manual_seed(tensor_seed(seed, index))
    dt = torch_dtype(cfg)
    if init == "normal":
        t = torch.randn(shape, generator=g, device=device, dtype=torch.float32) * STD
    elif init in ("ones", "zeros", "gate_bias"):
        base = {"ones": 1.0, "zeros": 0.0, "gate_bias": -3.0}[init]
        t = torch.full(shape, base, device=device, dtype=torch.float32)
        if perturb:
            t = t + 0.1 * torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    else:
        raise ValueError(init)
    return t.to(dt)


def make_weights(cfg, seed=None, device="cpu", perturb=False):
    """All weights of ``cfg`` as a list of tensors in ABI order (model dtype)."""
    return [make_tensor(cfg, i, s, seed=seed, device=device, perturb=perturb)
            for i, s in enumerate(weight_specs(cfg))]


def weights_dict(cfg, tensors):
    return {s[0]: t for s, t in zip(weight_specs(cfg), tensors)}
