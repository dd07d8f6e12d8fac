"""GPU rounds with the paper's MLP steering (eq. (2)) and its bias-after-MLP ablation vs the CPU
oracle, through the C ABI.

Every round compares logits, the per-layer up-projection biases W_s LayerNorm(W_hml [h; m; l])
of every sequence (tolerance of the dtype), emitted tokens, counts and cache lengths (exact),
and the library's own decisions wherever the oracle's margin pins them."""
import numpy as np
import pytest

import sd2_inputs as si
from sd2_inputs.configs import Dims, Workload

pytestmark = pytest.mark.gpu

# Persistent-launch shapes (K multiples of 512, head dims 128 / 64) with a 4-layer verifier: taps
# after blocks 2, 2 and 3; W_hml has K = 3072 and W_s 2 x 1536 rows.
MLP_MK = Workload(
    name="mlp-steer-persistent", verifier=Dims(4, 1024, 8, 2, 2048, 4096, 5e5),
    drafter=Dims(2, 512, 8, 4, 1536, 4096, 5e5),
    dtype="bf16", k=4, batch=2, prompt=(5, 13), new_tokens=12, temperature=1.0, seed=23)
# Head dim 32 (per-operation path) with an 8-layer verifier: taps after blocks 6, 4 and 3, all
# distinct.  (bf16 models have d_model % 256 == 0, so both steering projections take the MFMA
# kernel; the f32 case below takes the vector kernel.)
MLP_SMALL = Workload(
    name="mlp-steer-small", verifier=Dims(8, 256, 8, 2, 512, 512, 5e5), drafter=Dims(2, 256, 4, 2, 768, 512, 5e5),
    dtype="bf16", k=3, batch=2, prompt=(1, 9), new_tokens=16, temperature=1.0, seed=21)


def _run(wl, hml="normal", ln="normal", zero_ws=False, mlp=None, form=1, **kw):
    from gpu_harness import parity_run
    if mlp is None:
        mlp = si.mlp_steer_weights(wl, hml=hml, ln=ln, form=form)
    if zero_ws:
        mlp["w_s"] = np.zeros_like(mlp["w_s"])
    st = parity_run(wl, mlp=mlp, **kw)
    assert st.pinned > 0
    return st


def test_mlp_steering_persistent_path():
    _run(MLP_MK, expect_path=1)


def test_mlp_steering_separate_kernels():
    _run(MLP_MK, separate_kernels=True, expect_path=0)


def test_mlp_steering_persistent_greedy_identity_hml():
    """Greedy, with the paper's initialisation of W_hml ([I I I]) and a unit LayerNorm."""
    _run(MLP_MK.with_(temperature=0.0, new_tokens=16), hml="identity", ln="unit", expect_path=1)


def test_mlp_steering_eight_layer_verifier():
    """Three distinct tap blocks; ragged prompts (2 and 9 tokens)."""
    _run(MLP_SMALL, expect_path=0)


def test_mlp_steering_one_token_prompt():
    """A one-token prompt: nothing is prefilled and the first round runs without a bias."""
    _run(MLP_SMALL.with_(prompt=(1, 1), batch=1), expect_path=0)


def test_mlp_steering_f32():
    """f32 weights: the steering projections run on the vector kernel."""
    _run(si.TINY.with_(new_tokens=16), expect_path=0)


def test_mlp_steering_zero_ws_persistent():
    """W_s = 0 (the paper's initialisation): every bias is zero and the drafter is unsteered."""
    _run(MLP_MK, zero_ws=True, expect_path=1)


def test_bias_after_mlp_persistent_path():
    """The ablation with one bias W_s g after every drafter MLP (added in the down projection's
    residual epilogue)."""
    _run(MLP_MK, form=2, expect_path=1)


def test_bias_after_mlp_separate_kernels():
    _run(MLP_MK, form=2, separate_kernels=True, expect_path=0)


def test_bias_after_mlp_f32():
    _run(si.TINY.with_(new_tokens=16), form=2, expect_path=0)


@pytest.fixture(scope="module")
def host_8b_mlp():
    """Host weights of the 8B-shaped verifier / 1B-shaped drafter and of the MLP steering
    (W_hml 4096 x 12288, W_s 16 * 8192 x 4096), generated once."""
    wl = si.LLAMA8B
    return si.model_weights(wl, 0), si.model_weights(wl, 1), si.mlp_steer_weights(wl)


def test_mlp_steering_8b_shapes_short_prompt(host_8b_mlp):
    """The shapes bench.py --steering mlp times (taps after verifier blocks 30, 16 and 3; a bias
    of 8192 features in each of the 16 drafter layers) on the persistent launches, T=1, k=5;
    a 16-token prompt keeps the float64 oracle within seconds."""
    wl = si.LLAMA8B.with_(prompt=(16, 16), new_tokens=10)
    wv, wd, mlp = host_8b_mlp
    _run(wl, wv=wv, wd=wd, mlp=mlp, expect_path=1)


def _cond(wl, rank, scale=0.1, **kw):
    """The "Cond. bias in MLP" ablation: per drafter layer and row, U_l SiLU(V_l^f f + V_l^g g)
    added to the up projection (one kernel per operation); compared where the biases are
    otherwise: the per-round g parts V_l^g g [L_D][R]."""
    mlp = si.mlp_steer_weights(wl, form=3, rank=rank, cond_scale=scale)
    return _run(wl, mlp=mlp, expect_path=0, **kw)


def test_cond_bias_bf16_mfma_projections():
    # R = 256: both bias projections (V^f with K = 512, U with K = 256) on the MFMA kernel
    _cond(MLP_MK, 256)


def test_cond_bias_small_rank_ragged():
    # R = 64: U takes the vector kernel (K = 64); two sequences with 2- and 9-token prompts
    _cond(MLP_SMALL, 64)


def test_cond_bias_one_token_prompt():
    _cond(MLP_SMALL.with_(prompt=(1, 1), batch=1), 64)


def test_cond_bias_f32():
    _cond(si.TINY.with_(new_tokens=16), 32)
