"""Model and workload shapes for the five synthetic TADM workloads.

Each entry names a model (vocabulary, widths, layer split, fusion kind) and the
generation workload run on it (batch, prompt, generated length, block length,
reverse steps T and the refresh intervals K that are measured).

Layer split: ``n_shared`` layers form the shared network S (embedding only when 0),
``n_anchor`` the anchor network A, ``n_denoise`` the denoiser D (Sec. 3.1).
The mask token id is ``vocab`` (one past the last real token): the embedding has
``vocab + 1`` rows and the output head ``vocab`` columns (zero-masking, App. B.1.1).
"""

MASK_OFFSET = 0  # mask id == vocab + MASK_OFFSET


def mask_id(cfg):
    return cfg["vocab"] + MASK_OFFSET


CONFIGS = {
    # Tiny fp32 masked-diffusion LM: the case the oracle finishes in well under a second.
    "tiny": dict(
        dtype="f32", vocab=256, d_model=64, n_heads=4, n_kv_heads=4, head_dim=16,
        d_ffn=256, ffn_kind="gelu", n_shared=0, n_anchor=2, n_denoise=1,
        fusion_kind="gated_mlp", fusion_rank=0,
        batch=1, prompt_len=8, gen_len=24, block_len=24, T=16, Ks=(4, 1),
        temperature=1.0, weight_seed=0, input_seed=1, sampler_seed=2),
    # Small TADM-shaped model, d=768 with 12 anchor + 2 denoiser layers.
    "small": dict(
        dtype="bf16", vocab=32768, d_model=768, n_heads=12, n_kv_heads=12, head_dim=64,
        d_ffn=2048, ffn_kind="swiglu", n_shared=0, n_anchor=12, n_denoise=2,
        fusion_kind="gated_mlp", fusion_rank=0,
        batch=8, prompt_len=128, gen_len=256, block_len=256, T=64, Ks=(1, 2, 4, 8),
        temperature=1.0, weight_seed=0, input_seed=1, sampler_seed=2),
    # Block-diffusion shape: prompt + 8 blocks of 64, GQA with 4 KV heads.
    "block": dict(
        dtype="bf16", vocab=128256, d_model=2048, n_heads=16, n_kv_heads=4, head_dim=128,
        d_ffn=8192, ffn_kind="swiglu", n_shared=0, n_anchor=20, n_denoise=4,
        fusion_kind="gated_mlp", fusion_rank=0,
        batch=16, prompt_len=512, gen_len=512, block_len=64, T=32, Ks=(4, 1),
        temperature=1.0, weight_seed=0, input_seed=1, sampler_seed=2),
    # 1B-parameter-class pretraining-style TADM, 1024-token fully masked canvases.
    "1b": dict(
        dtype="bf16", vocab=50304, d_model=2048, n_heads=16, n_kv_heads=16, head_dim=128,
        d_ffn=8192, ffn_kind="gelu", n_shared=0, n_anchor=18, n_denoise=6,
        fusion_kind="gated_mlp", fusion_rank=0,
        batch=32, prompt_len=0, gen_len=1024, block_len=1024, T=128, Ks=(1, 4, 8),
        temperature=1.0, weight_seed=0, input_seed=1, sampler_seed=2),
    # 26B-parameter-class post-trained shape with paired-attention fusion.
    "26b": dict(
        dtype="bf16", vocab=262144, d_model=4608, n_heads=32, n_kv_heads=16, head_dim=128,
        d_ffn=36864, ffn_kind="geglu", n_shared=0, n_anchor=40, n_denoise=6,
        fusion_kind="paired", fusion_rank=256,
        batch=4, prompt_len=1024, gen_len=1024, block_len=256, T=64, Ks=(4, 8, 1),
        temperature=1.0, weight_seed=0, input_seed=1, sampler_seed=2),
}

# Fixed numerical constants of the model definition (the readings are listed in the
# design notes): RMSNorm epsilon for transformer layers and paired-attention scales,
# LayerNorm epsilon for the gated-MLP fusion, RoPE base.
RMS_EPS = 1e-6
LN_EPS = 1e-5
ROPE_THETA = 10000.0
PAIRED_HEADS = 4


def get_config(name, **overrides):
    cfg = dict(CONFIGS[name])
    cfg["name"] = name
    cfg.update(overrides)
    cfg.setdefault("rms_eps", RMS_EPS)
    cfg.setdefault("ln_eps", LN_EPS)
    cfg.setdefault("rope_theta", ROPE_THETA)
    cfg.setdefault("paired_heads", PAIRED_HEADS)
    return cfg


def n_layers(cfg):
    return cfg["n_shared"] + cfg["n_anchor"] + cfg["n_denoise"]
