"""Seeded synthetic inputs (weights, prompts) shared by the oracle and the GPU path.

Only value generation lives here: the C generator in ``gen.c`` (Philox4x32-10 +
Box-Muller, see its header) and the tensor-id scheme below.  Weights are
N(0, 0.02) for every matrix (embeddings, projections, LM heads and the steering
projection W_s); RMSNorm gains are 1.  bf16 tensors are returned as numpy
``uint16`` arrays holding the bf16 bit patterns, f32 tensors as ``float32``.
"""
import ctypes
import os
import subprocess

import numpy as np

from .configs import Dims, Workload, PRESETS, BY_NAME, TINY, SMALL, LLAMA8B, LLAMA8B_BATCHED, LLAMA70B  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "libsd2gen.so")
_lib = None

WEIGHT_STD = 0.02
LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")
_MATRIX_IDS = {"wq": 0, "wk": 1, "wv": 2, "wo": 3, "w_gate": 4, "w_up": 5, "w_down": 6}
VERIFIER, DRAFTER = 0, 1


def build(force: bool = False) -> str:
    """Compile gen.c into libsd2gen.so next to it."""
    if force or not os.path.exists(_SO):
        cmd = ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-o", _SO + ".tmp",
               os.path.join(_HERE, "gen.c"), "-lm"]
        subprocess.check_call(cmd)
        os.replace(_SO + ".tmp", _SO)
    return _SO


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_SO)
        u64, u32, i32 = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int32
        lib.gen_normal_bf16.argtypes = [ctypes.c_void_p, u64, u64, u32, ctypes.c_double]
        lib.gen_normal_f32.argtypes = [ctypes.c_void_p, u64, u64, u32, ctypes.c_double]
        lib.gen_prompt.argtypes = [ctypes.c_void_p, u64, u64, u32, i32]
        lib.gen_prompt_lens.argtypes = [ctypes.c_void_p, u64, u64, i32, i32]
        lib.gen_philox_block.argtypes = [ctypes.c_void_p, u64, ctypes.c_void_p]
        lib.gen_uniform_int.argtypes = [ctypes.c_void_p, u64, u64, u32, u32, i32, i32]
        _lib = lib
    return _lib


def tensor_id(model: int, layer: int, name: str) -> int:
    """Generator stream of one tensor: model 0 = verifier, 1 = drafter, 2 = steering."""
    if name == "embed":
        return ((model + 1) << 20) | 0
    if name == "lm_head":
        return ((model + 1) << 20) | 1
    if name == "w_s":
        return 3 << 20
    return ((model + 1) << 20) | ((layer + 1) << 4) | _MATRIX_IDS[name]


def normal(shape, dtype: str, seed: int, tid: int, scale: float = WEIGHT_STD) -> np.ndarray:
    lib = _load()
    n = int(np.prod(shape))
    if dtype == "bf16":
        out = np.empty(shape, dtype=np.uint16)
        lib.gen_normal_bf16(out.ctypes.data, n, seed, tid, scale)
    elif dtype == "f32":
        out = np.empty(shape, dtype=np.float32)
        lib.gen_normal_f32(out.ctypes.data, n, seed, tid, scale)
    else:
        raise ValueError(dtype)
    return out


def ones(shape, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return np.full(shape, 0x3F80, dtype=np.uint16)
    return np.ones(shape, dtype=np.float32)


def layer_shapes(dm: Dims):
    hd = dm.head_dim
    return {
        "attn_norm": (dm.d_model,),
        "wq": (dm.n_heads * hd, dm.d_model),
        "wk": (dm.n_kv_heads * hd, dm.d_model),
        "wv": (dm.n_kv_heads * hd, dm.d_model),
        "wo": (dm.d_model, dm.n_heads * hd),
        "ffn_norm": (dm.d_model,),
        "w_gate": (dm.d_ff, dm.d_model),
        "w_up": (dm.d_ff, dm.d_model),
        "w_down": (dm.d_model, dm.d_ff),
    }


def layer_tensor(wl: Workload, model: int, layer: int, name: str) -> np.ndarray:
    dm = wl.verifier if model == VERIFIER else wl.drafter
    shp = layer_shapes(dm)[name]
    if name.endswith("_norm"):
        return ones(shp, wl.dtype)
    return normal(shp, wl.dtype, wl.seed, tensor_id(model, layer, name))


def model_weights(wl: Workload, model: int) -> dict:
    """All weights of one model as host arrays: embed, layers[l][9], final_norm, lm_head."""
    dm = wl.verifier if model == VERIFIER else wl.drafter
    return {
        "embed": normal((dm.vocab, dm.d_model), wl.dtype, wl.seed, tensor_id(model, 0, "embed")),
        "layers": [[layer_tensor(wl, model, l, n) for n in LAYER_TENSORS] for l in range(dm.n_layers)],
        "final_norm": ones((dm.d_model,), wl.dtype),
        "lm_head": normal((dm.vocab, dm.d_model), wl.dtype, wl.seed, tensor_id(model, 0, "lm_head")),
    }


def iter_model_tensors(wl: Workload, model: int):
    """Yield (key, array) one tensor at a time, so a caller can stream large models."""
    dm = wl.verifier if model == VERIFIER else wl.drafter
    yield ("embed",), normal((dm.vocab, dm.d_model), wl.dtype, wl.seed, tensor_id(model, 0, "embed"))
    for l in range(dm.n_layers):
        for n in LAYER_TENSORS:
            yield ("layers", l, n), layer_tensor(wl, model, l, n)
    yield ("final_norm",), ones((dm.d_model,), wl.dtype)
    yield ("lm_head",), normal((dm.vocab, dm.d_model), wl.dtype, wl.seed, tensor_id(model, 0, "lm_head"))


def steer_weights(wl: Workload) -> np.ndarray:
    """W_s, shape [d_drafter][d_verifier]."""
    return normal((wl.drafter.d_model, wl.verifier.d_model), wl.dtype, wl.seed, tensor_id(2, 0, "w_s"))


def mlp_steer_weights(wl: Workload, hml: str = "normal", ln: str = "normal", ln_eps: float = 1e-5,
                      form: int = 1, rank: int = 256, cond_scale: float = WEIGHT_STD) -> dict:
    """Weights of the MLP steering forms: W_s [L_D*F_D][d_V] (form 1: one d_ff block per drafter
    layer) or [d_D][d_V] (form 2: one bias after every MLP); form 3 (the conditional bias, a
    two-layer MLP per drafter layer of hidden width `rank`): W_s = V^g [L_D*rank][d_V] plus
    w_cf = V^f [L_D*rank][d_D] and w_cu = U [L_D*F_D][rank], drawn with std `cond_scale`;
    W_hml [d_V][3 d_V] ("normal" draws, or "identity" for [I I I], which maps [h; m; l] to
    h + m + l), LayerNorm gain and shift [d_V] ("normal": 1 + N(0, 0.02) and N(0, 0.02); "unit":
    ones and zeros)."""
    dV, dD = wl.verifier.d_model, wl.drafter
    rows = dD.n_layers * dD.d_ff if form == 1 else (dD.n_layers * rank if form == 3 else dD.d_model)
    purpose = {1: 1, 2: 5, 3: 6}[form]
    w_s = normal((rows, dV), wl.dtype, wl.seed, (3 << 20) | purpose, cond_scale if form == 3 else WEIGHT_STD)
    if hml == "identity":
        eye = np.eye(dV, dtype=np.float32)
        w = np.concatenate([eye, eye, eye], axis=1)
        w_hml = ((w.view(np.uint32) >> 16).astype(np.uint16) if wl.dtype == "bf16" else w)
    else:
        w_hml = normal((dV, 3 * dV), wl.dtype, wl.seed, (3 << 20) | 2)
    if ln == "unit":
        gain, shift = ones((dV,), wl.dtype), (np.zeros((dV,), np.uint16) if wl.dtype == "bf16" else np.zeros((dV,), np.float32))
    else:
        d = normal((dV,), "f32", wl.seed, (3 << 20) | 3)
        g32 = (1.0 + d).astype(np.float32)
        gain = ((g32.view(np.uint32) + 0x7FFF + ((g32.view(np.uint32) >> 16) & 1)) >> 16).astype(np.uint16) \
            if wl.dtype == "bf16" else g32
        shift = normal((dV,), wl.dtype, wl.seed, (3 << 20) | 4)
    out = {"w_s": np.ascontiguousarray(w_s), "w_hml": np.ascontiguousarray(w_hml),
           "ln_gain": np.ascontiguousarray(gain), "ln_bias": np.ascontiguousarray(shift), "ln_eps": ln_eps,
           "form": form}
    if form == 3:
        out["w_cf"] = np.ascontiguousarray(normal((dD.n_layers * rank, dD.d_model), wl.dtype, wl.seed,
                                                  (3 << 20) | 7, cond_scale))
        out["w_cu"] = np.ascontiguousarray(normal((dD.n_layers * dD.d_ff, rank), wl.dtype, wl.seed,
                                                  (3 << 20) | 8, cond_scale))
        out["rank"] = rank
    return out


def prompt_lens(wl: Workload) -> np.ndarray:
    lo, hi = wl.prompt
    if lo == hi:
        return np.full((wl.batch,), lo, dtype=np.int32)
    out = np.empty((wl.batch,), dtype=np.int32)
    _load().gen_prompt_lens(out.ctypes.data, wl.batch, wl.seed, lo, hi)
    return out


def prompts(wl: Workload):
    """(tokens int32 [B][max_prompt] zero-padded, lens int32 [B])."""
    lens = prompt_lens(wl)
    toks = np.zeros((wl.batch, wl.max_prompt), dtype=np.int32)
    lib = _load()
    for b in range(wl.batch):
        row = np.empty((int(lens[b]),), dtype=np.int32)
        lib.gen_prompt(row.ctypes.data, int(lens[b]), wl.seed, b, wl.verifier.vocab)
        toks[b, : lens[b]] = row
    return toks, lens


def bf16_to_f32(a: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float32."""
    return (a.astype(np.uint32) << 16).view(np.float32)


# generator purposes of the training-objective inputs (beyond weights 0x10, prompts 0x11, lengths 0x12)
PURPOSE_TRAIN_TOKENS, PURPOSE_TRAIN_OFFSETS = 0x13, 0x14


def loss_inputs(wl: Workload, n: int, stream: int = 0):
    """Inputs of the training-objective forward: a token sequence of length n, uniform over the
    vocabulary (standing in for the verifier's own samples, which the paper trains on), and the
    offset delta_tau of every target, uniform in [1, k] (entry 0 unused).  Both int32 [n]."""
    lib = _load()
    toks = np.empty((n,), dtype=np.int32)
    lib.gen_uniform_int(toks.ctypes.data, n, wl.seed, PURPOSE_TRAIN_TOKENS, stream, 0, wl.verifier.vocab - 1)
    deltas = np.empty((n,), dtype=np.int32)
    lib.gen_uniform_int(deltas.ctypes.data, n, wl.seed, PURPOSE_TRAIN_OFFSETS, stream, 1, wl.k)
    return toks, deltas
