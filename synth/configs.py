"""The synthetic layer workloads and their generator recipes.

Shapes follow the backbones the paper evaluates (Sec. IV-A and App. A-B):
DeiT/ViT patch tokens (197 per image) and BERT sequences of at most 128
tokens with dynamic padding. Expert counts, block counts and thresholds are
per workload. ``n_experts`` is K, the number of residual experts; every
layer also holds the shared expert, stored as expert 0, so the weights hold
K + 1 upcycled experts (Sec. III-A).

Layer fields mirror the C structure ``unif_moe_config``:
  mass_threshold  t: the cumulative target is min(1 - alpha, t) in "coupled"
                  mode (t = 1 is Eq. beta / expert-count exactly), t in
                  "fixed" mode; unused in "topk" mode.
  max_shared      cap applied to the shared block count after Eq. block-count.
  alpha_mode      "adaptive" (Eq. alpha) or "fixed" (the ablation's constant
                  alpha, Table mechanism-ablation).
  mass_mode       "coupled", "fixed" or "topk" (top-k residual activation).
  select_mode     "prototype" (Eq. shared-indices) or "prefix" (ablation).
  max_pairs       capacity of the forward's workspace in (token, expert)
                  pairs; 0 sizes it for the worst case N (K+1).
"""
import copy

_LAYER_DEFAULTS = dict(
    tau=None, mass_threshold=1.0, max_shared=None, alpha_mode="adaptive",
    alpha_fixed=0.0, mass_mode="coupled", fixed_k=1, select_mode="prototype",
    max_pairs=0,
)

CONFIGS = {
    # 256 tokens x d=64, E=4 experts from one d_ff=256 FFN, B=4 blocks of 64.
    "tiny_f32": dict(
        index=1, seed=0, n_tokens=256, d_model=64, n_experts=4, n_blocks=4,
        block_width=64, dtype="f32", mass_threshold=0.6, max_shared=4,
        tokens="normal", router="default"),
    # ViT-S/16: 64 images x 197 tokens, d=384, d_ff=1536, K=8, B=8 (M=192).
    "vit_s16": dict(
        index=2, seed=1, n_tokens=64 * 197, d_model=384, n_experts=8,
        n_blocks=8, block_width=192, dtype="bf16", mass_threshold=0.6,
        tokens="normal_ln", router="default"),
    # BERT-base: 32 x 128 slots with valid lengths U{16..128}, d=768,
    # d_ff=3072, K=8, B=16 (M=192); residual router rows scaled so that the
    # mean residual expert count is about 2.
    "bert_base_padded": dict(
        index=3, seed=2, n_tokens=32 * 128, d_model=768, n_experts=8,
        n_blocks=16, block_width=192, dtype="bf16", mass_threshold=0.5,
        tokens="normal_ln", padding=dict(n_seq=32, seq_len=128, lo=16, hi=128),
        router="scaled_residual"),
    # ViT-B/16: 256 images x 197 tokens, d=768, d_ff=3072, K=16, B=16.
    "vit_b16": dict(
        index=4, seed=3, n_tokens=256 * 197, d_model=768, n_experts=16,
        n_blocks=16, block_width=192, dtype="bf16", mass_threshold=0.6,
        max_shared=16, tokens="normal_ln", router="default"),
    # Skewed load: 131072 tokens, d=1024, d_ff=4096, K=32, B=32 (M=128);
    # Zipf(1.2) top-1 popularity and bimodal shared demand.
    "zipf_stress": dict(
        index=5, seed=4, n_tokens=131072, d_model=1024, n_experts=32,
        n_blocks=32, block_width=128, dtype="bf16", mass_threshold=0.8,
        tokens="bimodal", router="zipf_bimodal"),
    # The paper's own operating points (Sec. IV-A and the architecture
    # details of the appendix), with the cumulative target exactly Eq. beta
    # (t = 1). Vision: DeiT-S/16 (d=384, H=1536) with K=6 residual experts
    # and B=8 blocks, evaluation batch 64 x 197 tokens. Language: BERT-large
    # (d=1024, H=4096) with K=16, B=16, evaluation batch 32 x 128 slots with
    # dynamic padding (valid lengths U{16..128}).
    "paper_vision": dict(
        index=6, seed=5, n_tokens=64 * 197, d_model=384, n_experts=6,
        n_blocks=8, block_width=192, dtype="bf16", mass_threshold=1.0,
        tokens="normal_ln", router="default"),
    "paper_language": dict(
        index=7, seed=6, n_tokens=32 * 128, d_model=1024, n_experts=16,
        n_blocks=16, block_width=256, dtype="bf16", mass_threshold=1.0,
        tokens="normal_ln", padding=dict(n_seq=32, seq_len=128, lo=16, hi=128),
        router="default"),
}

for _c in CONFIGS.values():
    for _k, _v in _LAYER_DEFAULTS.items():
        _c.setdefault(_k, _v)
    if _c["max_shared"] is None:
        _c["max_shared"] = _c["n_blocks"]
    _c.setdefault("padding", None)
    _c.setdefault("sigma_base", 0.02)   # base FFN weights ~ N(0, 0.02^2)
    _c.setdefault("sigma_pert", 0.002)  # per-expert perturbation ~ N(0, 0.002^2)

LAYER_KEYS = ("n_tokens", "d_model", "n_experts", "n_blocks", "block_width",
              "dtype", "tau", "mass_threshold", "max_shared", "alpha_mode",
              "alpha_fixed", "mass_mode", "fixed_k", "select_mode", "max_pairs")


def config_names():
    return sorted(CONFIGS, key=lambda n: CONFIGS[n]["index"])


def get_config(name, **overrides):
    """Full recipe of a named workload, with optional field overrides."""
    if name not in CONFIGS:
        raise KeyError(f"unknown workload {name!r}; known: {config_names()}")
    cfg = copy.deepcopy(CONFIGS[name])
    cfg["name"] = name
    for k, v in overrides.items():
        if k not in cfg and k not in _LAYER_DEFAULTS:
            raise KeyError(f"unknown config field {k!r}")
        cfg[k] = v
    return cfg


def layer_config(cfg):
    """Just the layer fields (what the C structure carries)."""
    return {k: cfg[k] for k in LAYER_KEYS}
