"""Small helpers shared by the oracle tests: custom tiny workloads and weight sets."""
import numpy as np

import sd2_inputs as si
from sd2_inputs.configs import Dims, Workload

# Grouped-query shapes (H/Hkv = 4 and 2) at a size the float64 oracle runs in milliseconds.
GQA = Workload(
    name="gqa-tiny", verifier=Dims(3, 256, 8, 2, 512, 512, 5e5), drafter=Dims(2, 256, 4, 2, 768, 512, 5e5),
    dtype="bf16", k=3, batch=2, prompt=(5, 9), new_tokens=24, temperature=1.0, seed=7)

# Vocabulary of 8 for exact enumeration of one round's output law.
LAW = Workload(
    name="law-v8", verifier=Dims(2, 16, 2, 1, 32, 8, 1e4), drafter=Dims(1, 16, 2, 2, 32, 8, 1e4),
    dtype="f32", k=2, batch=1, prompt=(4, 4), new_tokens=64, temperature=1.0, seed=3)


def scaled_weights(wl, model, scale):
    """Model weights drawn from the shared generator with a custom standard deviation."""
    dm = wl.verifier if model == si.VERIFIER else wl.drafter
    w = {
        "embed": si.normal((dm.vocab, dm.d_model), wl.dtype, wl.seed, si.tensor_id(model, 0, "embed"), scale),
        "layers": [],
        "final_norm": si.ones((dm.d_model,), wl.dtype),
        "lm_head": si.normal((dm.vocab, dm.d_model), wl.dtype, wl.seed, si.tensor_id(model, 0, "lm_head"), scale),
    }
    shapes = si.layer_shapes(dm)
    for l in range(dm.n_layers):
        row = []
        for n in si.LAYER_TENSORS:
            if n.endswith("_norm"):
                row.append(si.ones(shapes[n], wl.dtype))
            else:
                row.append(si.normal(shapes[n], wl.dtype, wl.seed, si.tensor_id(model, l, n), scale))
        w["layers"].append(row)
    return w


def weights(wl):
    return si.model_weights(wl, 0), si.model_weights(wl, 1), si.steer_weights(wl)


def zeros_like_ws(wl):
    ws = si.steer_weights(wl)
    return np.zeros_like(ws)


def to_f64(a, dtype):
    return si.bf16_to_f32(a).astype(np.float64) if dtype == "bf16" else a.astype(np.float64)

# Shapes the persistent-launch path takes (every projection K a multiple of 512), small enough
# for the float64 oracle: one layer each, then two layers with head dim 128, two sequences.
MK1 = Workload(
    name="mk-one-layer", verifier=Dims(1, 512, 8, 2, 1024, 2048, 5e5), drafter=Dims(1, 512, 8, 2, 1024, 2048, 5e5),
    dtype="bf16", k=3, batch=1, prompt=(6, 6), new_tokens=8, temperature=1.0, seed=11)
MK2 = Workload(
    name="mk-two-layers", verifier=Dims(2, 1024, 8, 2, 2048, 4096, 5e5), drafter=Dims(2, 512, 8, 4, 1536, 4096, 5e5),
    dtype="bf16", k=4, batch=2, prompt=(5, 13), new_tokens=12, temperature=1.0, seed=12)
# Split-K projections on the persistent path: drafter down projection K = 14336 (4 ranges of 3584
# columns, 7 waves per unit), verifier K = 8192 (2 ranges, 8 waves per unit); 6 verifier rows.
MK3 = Workload(
    name="mk-split-k", verifier=Dims(1, 512, 4, 2, 8192, 8192, 5e5), drafter=Dims(1, 512, 4, 2, 14336, 8192, 5e5),
    dtype="bf16", k=5, batch=1, prompt=(7, 7), new_tokens=7, temperature=1.0, seed=13)
# Contexts over several 64-position attention spans on the persistent path, ragged: prompts of
# 232, 273 and 63 tokens (the last crosses a span boundary while generating).
MK4 = Workload(
    name="mk-long-ragged", verifier=Dims(1, 512, 8, 2, 1024, 2048, 5e5), drafter=Dims(1, 512, 8, 2, 1024, 2048, 5e5),
    dtype="bf16", k=3, batch=3, prompt=(40, 300), new_tokens=24, temperature=1.0, seed=15)
# More attention units than workgroups on the persistent path: verifier with 8 KV heads, 3 groups of
# 8 query vectors (6 rows x 4 query heads per KV head) and a 730-token prompt (12 live spans of 64
# positions): 8 x 3 x 12 = 288 units on 256 workgroups, so some workgroups take a second unit.
MK5 = Workload(
    name="mk-many-attention-units", verifier=Dims(1, 2048, 32, 8, 1024, 2048, 5e5),
    drafter=Dims(1, 1024, 16, 8, 1024, 2048, 5e5),
    dtype="bf16", k=5, batch=1, prompt=(730, 730), new_tokens=8, temperature=1.0, seed=17)
# Head dim 128 at long contexts (the verify pass's attention at the 8B verifier's head shape):
# 16 query / 4 KV heads, prompts of 629 and 1114 tokens.  Persistent path: 10 and 18 live spans of
# 64 positions, so the last-arriver fold runs its second batch of 16 (span partials of 12 rows
# x 16 heads x 19 spans are 1.9 MB, above the size the O projection merges itself); per-operation
# path: 5 and 9 spans of 128 merged by the last span workgroup.
MK6 = Workload(
    name="mk-hd128-long", verifier=Dims(1, 2048, 16, 4, 2048, 4096, 5e5),
    drafter=Dims(1, 1024, 16, 8, 1024, 4096, 5e5),
    dtype="bf16", k=5, batch=2, prompt=(512, 1160), new_tokens=24, temperature=1.0, seed=21)
# The batched workload's structure at a depth the float64 oracle affords: 16 sequences with
# prompts drawn from [256, 2048] (257 ... 1992 tokens), k = 7, T = 0.7, head dim 128 verifier and
# head dim 64 drafter; 128 verify rows per round, so the per-operation path runs it.
RAG16 = Workload(
    name="ragged-16-long", verifier=Dims(1, 1024, 8, 2, 2048, 4096, 5e5),
    drafter=Dims(1, 512, 8, 2, 1024, 4096, 5e5),
    dtype="bf16", k=7, batch=16, prompt=(256, 2048), new_tokens=16, temperature=0.7, seed=42)
RAG16_SHORTEST, RAG16_LONGEST = 1, 8
# The 70B shape's verify attention at long contexts: 8 query heads per KV head (k_pattn's two
# passes of 4 heads), 9 rows per sequence (k = 8), head dim 128, prompts of 731 and 1026 tokens:
# flash attention over several key spans merged by the last span to arrive.  18
# verify rows, so the per-operation path runs it.
G8LONG = Workload(
    name="g8-hd128-long", verifier=Dims(1, 2048, 16, 2, 4096, 4096, 5e5),
    drafter=Dims(1, 1024, 8, 2, 2048, 4096, 5e5),
    dtype="bf16", k=8, batch=2, prompt=(600, 1100), new_tokens=18, temperature=1.0, seed=37)


def scaled_set(wl, scale):
    """Verifier, drafter and W_s all drawn with standard deviation `scale`: wider logit gaps, so
    that fewer greedy decisions are near-ties."""
    ws = si.normal((wl.drafter.d_model, wl.verifier.d_model), wl.dtype, wl.seed, si.tensor_id(2, 0, "w_s"), scale)
    return scaled_weights(wl, 0, scale), scaled_weights(wl, 1, scale), ws
