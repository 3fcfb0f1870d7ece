"""Synthetic workload descriptions: model shapes, batch shapes, seeds, SLQ settings.

Plain numbers only.  They stand in for the paper's pretrained checkpoints and
datasets (wikitext-2, the Pile): random N(0, 0.02) weights and uniform or
Zipf(1.1) tokens of the paper's sequence lengths (1024 in section 5.1, 2048 in
section 7.1).
"""

SEED_PARAMS = 1
SEED_TOKENS = 2
SEED_PROBE = 3      # SLQ probe j uses seed SEED_PROBE + j
SEED_GAUSS = 4      # Exp I direction

WORKLOADS = {
    # tiny GPT-2-like LM, fp32
    "tiny-gpt2-fp32": dict(
        family="gpt2", n_layers=2, d_model=64, n_heads=4, n_kv_heads=4, d_ff=256,
        vocab=256, max_seq=64, rope_base=10000.0, dtype="f32",
        batch=8, seq=64, token_dist="uniform",
        probes=1, m=20, reorth="full", window=0, basis="f32", eps=[1e-3]),
    # small GPT-2-like LM, fp32, eps sweep
    "small-gpt2-fp32": dict(
        family="gpt2", n_layers=6, d_model=512, n_heads=8, n_kv_heads=8, d_ff=2048,
        vocab=8192, max_seq=512, rope_base=10000.0, dtype="f32",
        batch=16, seq=512, token_dist="zipf",
        probes=4, m=80, reorth="full", window=0, basis="f32", eps=[1e-4, 1e-3, 1e-2]),
    # GPT-2-medium-shaped LM, bf16 weights
    "gpt2-medium-bf16": dict(
        family="gpt2", n_layers=24, d_model=1024, n_heads=16, n_kv_heads=16, d_ff=4096,
        vocab=32000, max_seq=1024, rope_base=10000.0, dtype="bf16",
        batch=8, seq=1024, token_dist="zipf",
        probes=4, m=100, reorth="full", window=0, basis="bf16", eps=[1e-3]),
    # Llama-style 1.3B LM, bf16
    "llama-1.3b-bf16": dict(
        family="llama", n_layers=24, d_model=2048, n_heads=16, n_kv_heads=16, d_ff=5632,
        vocab=32000, max_seq=2048, rope_base=10000.0, dtype="bf16",
        batch=4, seq=2048, token_dist="zipf",
        probes=8, m=40, reorth="full", window=0, basis="bf16", eps=[1e-3]),
    # Llama-3-8B-shaped LM, bf16, GQA
    "llama3-8b-bf16": dict(
        family="llama", n_layers=32, d_model=4096, n_heads=32, n_kv_heads=8, d_ff=14336,
        vocab=128256, max_seq=2048, rope_base=500000.0, dtype="bf16",
        batch=1, seq=2048, token_dist="zipf",
        probes=2, m=30, reorth="window", window=8, basis="bf16", eps=[1e-3], recompute=True),
}

MODEL_KEYS = ("family", "n_layers", "d_model", "n_heads", "n_kv_heads", "d_ff",
              "vocab", "max_seq", "rope_base")


def model_fields(name_or_dict):
    w = WORKLOADS[name_or_dict] if isinstance(name_or_dict, str) else name_or_dict
    return {k: w[k] for k in MODEL_KEYS}
