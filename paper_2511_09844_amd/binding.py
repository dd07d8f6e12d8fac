"""ctypes binding of include/sd2.h.  Argument marshalling only: no computation here.

PyTorch provides the device buffers (weights, workspace, token buffers) and the
HIP stream; the library never allocates device memory itself.
"""
import ctypes
import os

import numpy as np
import torch

from .build import SO

P = ctypes.c_void_p

SD2_OK = 0
STATUS = {0: "ok", -1: "invalid argument", -2: "capacity", -3: "state", -4: "hip error", -5: "unsupported"}
DBG_LOGITS_V, DBG_LOGITS_D, DBG_STEER, DBG_OWN_DRAFTS, DBG_OWN_N, DBG_OWN_Y, DBG_STATE, DBG_HIST, DBG_HIDDEN_V, DBG_PATH, \
    DBG_TRACE, DBG_UBIAS, DBG_NONFINITE = range(1, 14)

EXPORTS = ["sd2_workspace_bytes", "sd2_create", "sd2_create_noalloc", "sd2_create_mlp", "sd2_train_loss",
           "sd2_train_loss_scratch_bytes", "sd2_prefill", "sd2_round", "sd2_round_forced", "sd2_destroy",
           "sd2_status_string", "sd2_last_error", "sd2_debug_read", "sd2_profile", "sd2_profile_read"]
PROF_GEMV, PROF_ATTN, PROF_SAMPLER, PROF_OTHER, PROF_PROGRAM = 1, 2, 3, 4, 5


class Dims(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("d_ff", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("rope_theta", ctypes.c_float), ("rms_eps", ctypes.c_float)]


class Weights(ctypes.Structure):
    _fields_ = [("embed", P), ("layers", ctypes.POINTER(P)), ("final_norm", P), ("lm_head", P)]


class Config(ctypes.Structure):
    _fields_ = [("verifier", Dims), ("drafter", Dims), ("dtype", ctypes.c_int32), ("k", ctypes.c_int32),
                ("max_batch", ctypes.c_int32), ("max_seq_len", ctypes.c_int32), ("max_new_tokens", ctypes.c_int32),
                ("temperature", ctypes.c_float), ("seed", ctypes.c_uint64), ("steering", ctypes.c_int32),
                ("cond_rank", ctypes.c_int32)]


STEER_INPUT, STEER_MLP, STEER_MLP_OUT, STEER_NONE, STEER_MLP_COND = 0, 1, 2, 3, 4


class MlpSteering(ctypes.Structure):
    _fields_ = [("w_s", P), ("w_hml", P), ("ln_gain", P), ("ln_bias", P), ("ln_eps", ctypes.c_float),
                ("w_cf", P), ("w_cu", P)]


_lib = None


def load():
    """Load libsd2.so (built in-tree); raises if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(SO):
            raise RuntimeError(f"{SO} is not built; run paper_2511_09844_amd.build() first")
        lib = ctypes.CDLL(SO)
        lib.sd2_workspace_bytes.argtypes = [ctypes.POINTER(Config)]
        lib.sd2_workspace_bytes.restype = ctypes.c_size_t
        lib.sd2_create.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(Weights), ctypes.POINTER(Weights), P, P,
                                   ctypes.c_size_t, P, ctypes.POINTER(P)]
        lib.sd2_create.restype = ctypes.c_int32
        lib.sd2_create_noalloc.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(Weights), ctypes.POINTER(Weights),
                                           P, P, ctypes.POINTER(P)]
        lib.sd2_create_noalloc.restype = ctypes.c_int32
        lib.sd2_train_loss_scratch_bytes.argtypes = [ctypes.POINTER(Config), ctypes.c_int32, ctypes.c_int32]
        lib.sd2_train_loss_scratch_bytes.restype = ctypes.c_size_t
        lib.sd2_train_loss.argtypes = [P, P, P, ctypes.c_int32, ctypes.c_int32, P, P, P, ctypes.c_size_t]
        lib.sd2_train_loss.restype = ctypes.c_int32
        lib.sd2_create_mlp.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(Weights), ctypes.POINTER(Weights),
                                       ctypes.POINTER(MlpSteering), P, ctypes.c_size_t, P, ctypes.POINTER(P)]
        lib.sd2_create_mlp.restype = ctypes.c_int32
        lib.sd2_prefill.argtypes = [P, ctypes.c_int32, P, P, ctypes.c_int32]
        lib.sd2_prefill.restype = ctypes.c_int32
        lib.sd2_round.argtypes = [P, P, P]
        lib.sd2_round.restype = ctypes.c_int32
        lib.sd2_round_forced.argtypes = [P, P, P, P]
        lib.sd2_round_forced.restype = ctypes.c_int32
        lib.sd2_destroy.argtypes = [P]
        lib.sd2_destroy.restype = ctypes.c_int32
        lib.sd2_status_string.argtypes = [ctypes.c_int32]
        lib.sd2_status_string.restype = ctypes.c_char_p
        lib.sd2_last_error.argtypes = [P]
        lib.sd2_last_error.restype = ctypes.c_char_p
        lib.sd2_debug_read.argtypes = [P, ctypes.c_int32, P, ctypes.c_size_t]
        lib.sd2_debug_read.restype = ctypes.c_int32
        lib.sd2_profile.argtypes = [P, ctypes.c_int32]
        lib.sd2_profile.restype = ctypes.c_int32
        lib.sd2_profile_read.argtypes = [P, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32),
                                         ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
        lib.sd2_profile_read.restype = ctypes.c_int32
        _lib = lib
    return _lib


def dims_of(dm) -> Dims:
    return Dims(dm.n_layers, dm.d_model, dm.n_heads, dm.n_kv_heads, dm.d_ff, dm.vocab, dm.rope_theta, dm.rms_eps)


def config_of(wl, max_batch=None, max_seq_len=None, max_new_tokens=None, temperature=None, k=None, seed=None,
              steering=STEER_INPUT, cond_rank=0):
    return Config(dims_of(wl.verifier), dims_of(wl.drafter), 1 if wl.dtype == "bf16" else 0,
                  wl.k if k is None else k,
                  wl.batch if max_batch is None else max_batch,
                  wl.max_seq_len if max_seq_len is None else max_seq_len,
                  wl.new_tokens if max_new_tokens is None else max_new_tokens,
                  wl.temperature if temperature is None else temperature,
                  wl.seed if seed is None else seed, steering, cond_rank)


class Sd2Error(RuntimeError):
    pass


def check(rc, h=None, what=""):
    if rc != SD2_OK:
        lib = load()
        msg = lib.sd2_status_string(rc).decode()
        if h is not None:
            msg += " / " + lib.sd2_last_error(h).decode()
        raise Sd2Error(f"{what}: {msg} ({rc})")


def to_device(arr: np.ndarray, device="cuda") -> torch.Tensor:
    """Host array (float32, or uint16 bf16 bit patterns) -> device tensor with the same bytes."""
    if arr.dtype == np.uint16:
        return torch.from_numpy(arr.view(np.int16)).to(device)
    return torch.from_numpy(arr).to(device)


class DeviceModel:
    """Device copies of one model's weights, uploaded tensor by tensor."""

    def __init__(self, tensors, device="cuda"):
        # tensors: iterable of (key, numpy array) in the order of sd2_inputs.iter_model_tensors
        self.t = {}
        self.layers = {}
        for key, arr in tensors:
            dev = to_device(arr, device)
            if key[0] == "layers":
                self.layers.setdefault(key[1], []).append(dev)
            else:
                self.t[key[0]] = dev
        n = len(self.layers)
        ptrs = [x.data_ptr() for l in range(n) for x in self.layers[l]]
        self._arr = (P * len(ptrs))(*ptrs)
        self.w = Weights(self.t["embed"].data_ptr(), self._arr, self.t["final_norm"].data_ptr(),
                         self.t["lm_head"].data_ptr())


class Engine:
    """One libsd2 handle.  `stream` is a torch.cuda.Stream (default: the current stream).

    With `mlp` (a dict of device tensors w_s, w_hml, ln_gain, ln_bias and a float ln_eps) the
    handle is created by sd2_create_mlp (cfg.steering STEER_MLP or STEER_MLP_OUT) and `w_steer` is
    unused; with cfg.steering STEER_NONE (the unsteered drafter) `w_steer` may be None."""

    def __init__(self, cfg: Config, verifier: DeviceModel, drafter: DeviceModel, w_steer: torch.Tensor,
                 stream=None, device="cuda", mlp=None, noalloc=False):
        lib = load()
        self.lib = lib
        self.cfg = cfg
        self.models = (verifier, drafter)
        self.w_steer = w_steer
        self.mlp = mlp
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        nbytes = lib.sd2_workspace_bytes(ctypes.byref(cfg))
        if nbytes == 0:
            raise Sd2Error("invalid configuration")
        self.h = P()
        self.workspace = None
        ws_ptr = w_steer.data_ptr() if w_steer is not None else None
        if noalloc:
            # the library's static workspace (sd2_create_noalloc): nothing is allocated here
            assert mlp is None
            rc = lib.sd2_create_noalloc(ctypes.byref(cfg), ctypes.byref(verifier.w), ctypes.byref(drafter.w),
                                        ws_ptr, self.stream.cuda_stream, ctypes.byref(self.h))
            check(rc, None, "sd2_create_noalloc")
        else:
            self.workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
            base = self.workspace.data_ptr()
            off = (-base) % 256
            if mlp is None:
                rc = lib.sd2_create(ctypes.byref(cfg), ctypes.byref(verifier.w), ctypes.byref(drafter.w), ws_ptr,
                                    base + off, nbytes, self.stream.cuda_stream, ctypes.byref(self.h))
                check(rc, None, "sd2_create")
            else:
                ms = MlpSteering(mlp["w_s"].data_ptr(), mlp["w_hml"].data_ptr(), mlp["ln_gain"].data_ptr(),
                                 mlp["ln_bias"].data_ptr(), float(mlp["ln_eps"]),
                                 mlp["w_cf"].data_ptr() if "w_cf" in mlp else None,
                                 mlp["w_cu"].data_ptr() if "w_cu" in mlp else None)
                rc = lib.sd2_create_mlp(ctypes.byref(cfg), ctypes.byref(verifier.w), ctypes.byref(drafter.w),
                                        ctypes.byref(ms), base + off, nbytes, self.stream.cuda_stream,
                                        ctypes.byref(self.h))
                check(rc, None, "sd2_create_mlp")
        self.batch = 0
        k = cfg.k
        self.out_tokens = torch.zeros((cfg.max_batch, k + 1), dtype=torch.int32, device=device)
        self.out_counts = torch.zeros((cfg.max_batch,), dtype=torch.int32, device=device)

    def close(self):
        if self.h:
            self.lib.sd2_destroy(self.h)
            self.h = P()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def prefill(self, tokens: torch.Tensor, lens: torch.Tensor, max_prompt: int):
        assert tokens.dtype == torch.int32 and lens.dtype == torch.int32 and tokens.is_contiguous()
        assert tokens.shape[1] == max_prompt
        self.batch = tokens.shape[0]
        self._prompt = (tokens, lens)
        check(self.lib.sd2_prefill(self.h, self.batch, tokens.data_ptr(), lens.data_ptr(), max_prompt), self.h,
              "sd2_prefill")

    def round(self, forced: torch.Tensor = None):
        """Enqueue one round; returns the (device) out_tokens / out_counts views."""
        if forced is None:
            rc = self.lib.sd2_round(self.h, self.out_tokens.data_ptr(), self.out_counts.data_ptr())
        else:
            assert forced.dtype == torch.int32 and forced.is_contiguous()
            assert forced.shape == (self.batch, self.cfg.k + 2)
            self._forced = forced
            rc = self.lib.sd2_round_forced(self.h, forced.data_ptr(), self.out_tokens.data_ptr(),
                                           self.out_counts.data_ptr())
        check(rc, self.h, "sd2_round")
        return self.out_tokens[: self.batch], self.out_counts[: self.batch]

    def train_loss(self, tokens: torch.Tensor, deltas: torch.Tensor, rows_per_chunk: int = 512):
        """Training-objective forward (sd2_train_loss) over one device token sequence and its
        offsets: returns (mean KL over targets 1..n-1, per-target KL as numpy [n]).  The handle's
        generation state is lost (prefill again before a round)."""
        assert tokens.dtype == torch.int32 and deltas.dtype == torch.int32
        assert tokens.is_contiguous() and deltas.is_contiguous() and tokens.numel() == deltas.numel()
        n = tokens.numel()
        nbytes = self.lib.sd2_train_loss_scratch_bytes(ctypes.byref(self.cfg), n, rows_per_chunk)
        if nbytes == 0:
            raise Sd2Error("train_loss: unsupported configuration or sizes")
        scratch = torch.empty(nbytes + 256, dtype=torch.uint8, device=tokens.device)
        off = (-scratch.data_ptr()) % 256
        kl = torch.empty(n, dtype=torch.float32, device=tokens.device)
        loss = torch.empty(1, dtype=torch.float32, device=tokens.device)
        check(self.lib.sd2_train_loss(self.h, tokens.data_ptr(), deltas.data_ptr(), n, rows_per_chunk, kl.data_ptr(),
                                      loss.data_ptr(), scratch.data_ptr() + off, nbytes), self.h, "sd2_train_loss")
        self.batch = 0
        torch.cuda.synchronize()
        return float(loss.item()), kl.cpu().numpy()

    def debug(self, what: int) -> np.ndarray:
        B, k = self.batch, self.cfg.k
        V, dV, dD = self.cfg.verifier.vocab, self.cfg.verifier.d_model, self.cfg.drafter.d_model
        shapes = {
            DBG_LOGITS_V: ((B, k + 1, V), np.float32), DBG_LOGITS_D: ((B, k, V), np.float32),
            DBG_STEER: ((B, dD), np.float32), DBG_OWN_DRAFTS: ((B, k), np.int32), DBG_OWN_N: ((B,), np.int32),
            DBG_OWN_Y: ((B,), np.int32), DBG_STATE: ((B, 5), np.int32),
            DBG_HIST: ((B, self.cfg.max_seq_len), np.int32), DBG_HIDDEN_V: ((B, k + 1, dV), np.float32),
            DBG_PATH: ((2,), np.int32), DBG_TRACE: ((33, 1024), np.int64), DBG_NONFINITE: ((1,), np.int32),
            DBG_UBIAS: (((B, self.cfg.drafter.n_layers, self.cfg.drafter.d_ff) if self.cfg.steering == STEER_MLP
                         else (B, self.cfg.drafter.n_layers, self.cfg.cond_rank)
                         if self.cfg.steering == STEER_MLP_COND else (B, self.cfg.drafter.d_model)), np.float32),
        }
        shp, dt = shapes[what]
        out = np.zeros(shp, dtype=dt)
        check(self.lib.sd2_debug_read(self.h, what, out.ctypes.data, out.nbytes), self.h, "sd2_debug_read")
        return out

    def profile(self, enable: bool):
        check(self.lib.sd2_profile(self.h, 1 if enable else 0), self.h, "sd2_profile")

    def profile_read(self, cls: int):
        """(launches, total ms, algorithmic bytes) of kernel class cls in the last profiled round."""
        n, ms, by = ctypes.c_int32(), ctypes.c_double(), ctypes.c_double()
        check(self.lib.sd2_profile_read(self.h, cls, ctypes.byref(n), ctypes.byref(ms), ctypes.byref(by)),
              self.h, "sd2_profile_read")
        return n.value, ms.value, by.value

    def state(self):
        s = self.debug(DBG_STATE)
        return [dict(zip(("t", "len_v", "len_d", "produced", "done"), map(int, row))) for row in s]
