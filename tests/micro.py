"""Micro model shapes for exhaustive CPU checks (brute force is cheap)."""
from paper_2607_04749_amd.workloads import GPT, LLAMA, LAYERS_ONLY, ModelShape, Parallel

# layers divisible by 1, 2, 4; every TP-split dim divisible by 1, 2, 4
MICRO_GPT = ModelShape(GPT, 4, 16, 4, 4, 32, 16, 8, 1)
MICRO_GPT_UNTIED = ModelShape(GPT, 4, 16, 4, 4, 32, 16, 0, 0)
MICRO_LLAMA_GQA = ModelShape(LLAMA, 4, 16, 8, 4, 32, 16, 0, 0)
MICRO_LLAMA_TIED = ModelShape(LLAMA, 4, 16, 4, 4, 32, 16, 0, 1)
# ragged: shard boxes that are not multiples of 8 elements (3-wide heads)
RAGGED_LLAMA = ModelShape(LLAMA, 4, 12, 4, 4, 20, 12, 0, 0)
RAGGED_GPT = ModelShape(GPT, 2, 12, 4, 4, 20, 12, 6, 1)

MICRO_MODELS = {
    "gpt": MICRO_GPT,
    "gpt_untied": MICRO_GPT_UNTIED,
    "llama_gqa": MICRO_LLAMA_GQA,
    "llama_tied": MICRO_LLAMA_TIED,
    "ragged_llama": RAGGED_LLAMA,
    "ragged_gpt": RAGGED_GPT,
}

CFGS = [Parallel(tp, pp) for tp in (1, 2, 4) for pp in (1, 2, 4)]


def cfg_pairs(model):
    out = []
    for a in CFGS:
        for b in CFGS:
            if model.num_layers % a.pp or model.num_layers % b.pp:
                continue
            out.append((a, b))
    return out


def layers_only(num_layers, arch=GPT, hidden=8):
    return ModelShape(arch, num_layers, hidden, 2, 2, 16, 8, 0, 0, LAYERS_ONLY)
