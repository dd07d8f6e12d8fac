"""CPU oracle of one SD^2 speculative round (ctypes binding over oracle.c).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's CPU
baseline leg may use this package; the GPU library never does.  See the
header of ``oracle.c`` for what is computed and which passages of the paper
each step follows.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liboracle.so")
_lib = None
MAX_K = 64


def build(force: bool = False) -> str:
    """Compile oracle.c (plain C, OpenMP over output rows) into liboracle.so."""
    if force or not os.path.exists(_SO):
        cmd = ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-o", _SO + ".tmp",
               os.path.join(_HERE, "oracle.c"), "-lm"]
        subprocess.check_call(cmd)
        os.replace(_SO + ".tmp", _SO)
    return _SO


class RoundLog(ctypes.Structure):
    _fields_ = [
        ("active", ctypes.c_int32),
        ("t_start", ctypes.c_int32),
        ("n", ctypes.c_int32),
        ("y", ctypes.c_int32),
        ("count", ctypes.c_int32),
        ("used_fallback", ctypes.c_int32),
        ("final_margin", ctypes.c_float),
        ("drafts", ctypes.c_int32 * MAX_K),
        ("draft_margin", ctypes.c_float * MAX_K),
        ("accept_margin", ctypes.c_float * MAX_K),
        ("lse_v", ctypes.c_float * (MAX_K + 1)),
        ("lse_d", ctypes.c_float * MAX_K),
    ]


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_SO)
        P = ctypes.c_void_p
        i32, u32, u64, f32 = ctypes.c_int32, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_float
        lib.oracle_create.restype = P
        lib.oracle_create.argtypes = [P, P, P, P, ctypes.c_int, P, P, P, ctypes.c_int, ctypes.c_int,
                                      ctypes.c_int, ctypes.c_int, f32, u64, ctypes.c_int, P, P, P,
                                      ctypes.c_double, P, P, ctypes.c_int]
        lib.oracle_destroy.argtypes = [P]
        lib.oracle_prefill_one.argtypes = [P, ctypes.c_int, P, ctypes.c_int]
        lib.oracle_prefill_one.restype = ctypes.c_int
        lib.oracle_round_one.argtypes = [P, ctypes.c_int, P, ctypes.POINTER(RoundLog), P, P, P]
        lib.oracle_round_one.restype = ctypes.c_int
        lib.oracle_get_state.argtypes = [P, ctypes.c_int, P, P, P, P, P]
        lib.oracle_get_steer.argtypes = [P, ctypes.c_int, P]
        lib.oracle_set_steer.argtypes = [P, ctypes.c_int, P]
        lib.oracle_get_hist.argtypes = [P, ctypes.c_int, P, ctypes.c_int]
        lib.oracle_round_log_size.restype = ctypes.c_int
        lib.oracle_forward.argtypes = [P, ctypes.c_int, P, ctypes.c_int, P, P, P]
        lib.oracle_steer.argtypes = [P, P, P]
        lib.oracle_get_ubias.argtypes = [P, ctypes.c_int, P]
        lib.oracle_forward_mlp.argtypes = [P, ctypes.c_int, P, ctypes.c_int, P, P, P, P, P]
        lib.oracle_mlp_steer.argtypes = [P, P, P]
        lib.oracle_forward_cond.argtypes = [P, ctypes.c_int, P, ctypes.c_int, P, P, P]
        lib.oracle_train_loss.argtypes = [P, P, ctypes.c_int, P, P, P]
        lib.oracle_train_loss.restype = ctypes.c_double
        lib.oracle_philox.argtypes = [P, u32, u32, P]
        lib.oracle_uniform.argtypes = [u32]
        lib.oracle_uniform.restype = f32
        lib.oracle_gumbel.argtypes = [u32]
        lib.oracle_gumbel.restype = f32
        lib.oracle_set_seed.argtypes = [P, u64]
        lib.oracle_pick.argtypes = [P, ctypes.c_int, f32, u64, ctypes.c_int, ctypes.c_int, ctypes.c_int, P]
        lib.oracle_pick.restype = ctypes.c_int
        lib.oracle_accept_final.argtypes = [ctypes.c_int, ctypes.c_int, f32, u64, ctypes.c_int, ctypes.c_int,
                                            P, P, P, ctypes.POINTER(RoundLog)]
        assert lib.oracle_round_log_size() == ctypes.sizeof(RoundLog)
        _lib = lib
    return _lib


def philox(ctr, key):
    """Philox4x32-10 block for counter (4 words) and key (2 words)."""
    lib = _load()
    c = np.asarray(ctr, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib.oracle_philox(c.ctypes.data, int(key[0]), int(key[1]), out.ctypes.data)
    return out


def uniform(word: int) -> float:
    return _load().oracle_uniform(int(word))


def gumbel(word: int) -> float:
    return _load().oracle_gumbel(int(word))


def pick(q, T, seed, j, t, b):
    """Draft pick from one logit row: (token, margin)."""
    q = np.ascontiguousarray(q, dtype=np.float32)
    m = np.zeros(1, dtype=np.float32)
    x = _load().oracle_pick(q.ctypes.data, len(q), float(T), int(seed), int(j), int(t), int(b), m.ctypes.data)
    return int(x), float(m[0])


def accept_final(drafts, plog, qlog, T, seed, t, b):
    """Verification decisions for one block given logit tables: returns a RoundLog (n, y, margins)."""
    drafts = np.ascontiguousarray(drafts, dtype=np.int32)
    plog = np.ascontiguousarray(plog, dtype=np.float32)
    qlog = np.ascontiguousarray(qlog, dtype=np.float32)
    k = len(drafts)
    assert plog.shape[0] == k + 1 and qlog.shape[0] == k and plog.shape[1] == qlog.shape[1]
    log = RoundLog()
    _load().oracle_accept_final(k, plog.shape[1], float(T), int(seed), int(t), int(b), drafts.ctypes.data,
                                plog.ctypes.data, qlog.ctypes.data, ctypes.byref(log))
    return log


def _dims(dm):
    return (np.array([dm.n_layers, dm.d_model, dm.n_heads, dm.n_kv_heads, dm.d_ff, dm.vocab], dtype=np.int32),
            np.array([dm.rope_theta, dm.rms_eps], dtype=np.float64))


def _ptrs(w):
    arrs = [w["embed"]] + [t for layer in w["layers"] for t in layer] + [w["final_norm"], w["lm_head"]]
    for a in arrs:
        assert a.flags["C_CONTIGUOUS"]
    return (ctypes.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs]), arrs


class Oracle:
    """One oracle engine: a verifier, a drafter, W_s and per-sequence state.

    ``wv`` / ``wd`` are dicts as returned by ``sd2_inputs.model_weights`` and
    ``ws`` is W_s [d_D][d_V]; arrays must stay alive (they are referenced).
    ``mlp`` selects the MLP steering of eq. (2) instead: a dict as returned by
    ``sd2_inputs.mlp_steer_weights`` (w_s [L_D*F_D][d_V], w_hml [d_V][3 d_V],
    ln_gain, ln_bias, ln_eps; form 2, the bias after every MLP: w_s [d_D][d_V];
    form 3, the conditional bias: w_s = V^g [L_D*R][d_V], w_cf = V^f [L_D*R][d_D],
    w_cu = U [L_D*F_D][R], rank R); ``ws`` is then ignored.
    """

    def __init__(self, wl, wv, wd, ws, max_batch=None, cap=None, temperature=None, k=None, max_new=None,
                 mlp=None):
        lib = _load()
        self.wl = wl
        self.k = wl.k if k is None else k
        self.max_batch = wl.batch if max_batch is None else max_batch
        self.max_new = wl.new_tokens if max_new is None else max_new
        self.cap = wl.max_seq_len if cap is None else cap
        self.temperature = wl.temperature if temperature is None else temperature
        assert self.k <= MAX_K
        self._dv, self._rv = _dims(wl.verifier)
        self._dd, self._rd = _dims(wl.drafter)
        self._pv, self._keep_v = _ptrs(wv)
        self._pd, self._keep_d = _ptrs(wd)
        self.mlp = mlp
        if mlp is None:
            self._ws = ws
            form, extra = 0, (None, None, None, 0.0)
        else:
            self._ws = mlp["w_s"]
            for key in ("w_s", "w_hml", "ln_gain", "ln_bias"):
                assert mlp[key].flags["C_CONTIGUOUS"]
            form = int(mlp.get("form", 1))
            extra = (mlp["w_hml"].ctypes.data, mlp["ln_gain"].ctypes.data, mlp["ln_bias"].ctypes.data,
                     float(mlp["ln_eps"]))
            if form == 3:
                for key in ("w_cf", "w_cu"):
                    assert mlp[key].flags["C_CONTIGUOUS"]
                extra += (mlp["w_cf"].ctypes.data, mlp["w_cu"].ctypes.data, int(mlp["rank"]))
        if len(extra) == 4:
            extra += (None, None, 0)
        self.h = lib.oracle_create(self._dv.ctypes.data, self._rv.ctypes.data, self._dd.ctypes.data,
                                   self._rd.ctypes.data, 1 if wl.dtype == "bf16" else 0, self._pv, self._pd,
                                   self._ws.ctypes.data, self.k, self.max_batch, self.cap, self.max_new,
                                   float(self.temperature), int(wl.seed), form, *extra)
        if not self.h:
            raise ValueError("oracle_create rejected the steering arguments")
        self.lib = lib

    def close(self):
        if self.h:
            self.lib.oracle_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def prefill_one(self, b, prompt):
        p = np.ascontiguousarray(prompt, dtype=np.int32)
        rc = self.lib.oracle_prefill_one(self.h, b, p.ctypes.data, len(p))
        if rc != 0:
            raise ValueError("oracle_prefill_one failed")

    def prefill(self, tokens, lens, seqs=None):
        for b in (range(len(lens)) if seqs is None else seqs):
            self.prefill_one(b, tokens[b, : lens[b]])

    def round_one(self, b, dump=False):
        """Run one round for sequence b; returns (emitted tokens, RoundLog, dumps dict)."""
        V, dV = self.wl.verifier.vocab, self.wl.verifier.d_model
        out = np.zeros(self.k + 1, dtype=np.int32)
        log = RoundLog()
        dumps = {}
        pv = pd = ph = None
        if dump:
            dumps["logits_v"] = np.zeros((self.k + 1, V), dtype=np.float32)
            dumps["logits_d"] = np.zeros((self.k, V), dtype=np.float32)
            dumps["hf_v"] = np.zeros((self.k + 1, dV), dtype=np.float64)
            pv, pd, ph = (dumps["logits_v"].ctypes.data, dumps["logits_d"].ctypes.data, dumps["hf_v"].ctypes.data)
        rc = self.lib.oracle_round_one(self.h, b, out.ctypes.data, ctypes.byref(log), pv, pd, ph)
        if rc != 0:
            raise RuntimeError("oracle_round_one failed")
        return out[: log.count].copy(), log, dumps

    def set_seed(self, seed):
        self.lib.oracle_set_seed(self.h, int(seed))

    def state(self, b):
        vals = [np.zeros(1, dtype=np.int32) for _ in range(5)]
        self.lib.oracle_get_state(self.h, b, *[v.ctypes.data for v in vals])
        return dict(zip(("t", "len_v", "len_d", "produced", "done"), [int(v[0]) for v in vals]))

    def steer_vec(self, b):
        out = np.zeros(self.wl.drafter.d_model, dtype=np.float64)
        self.lib.oracle_get_steer(self.h, b, out.ctypes.data)
        return out

    def set_steer_vec(self, b, s):
        s = np.ascontiguousarray(s, dtype=np.float64)
        self.lib.oracle_set_steer(self.h, b, s.ctypes.data)

    def hist(self, b, n):
        out = np.zeros(n, dtype=np.int32)
        self.lib.oracle_get_hist(self.h, b, out.ctypes.data, n)
        return out

    def forward(self, which, toks, add=None):
        """Whole-sequence forward from an empty cache: returns (hF [n][d], logits [n][V]) in float64."""
        dm = self.wl.verifier if which == 0 else self.wl.drafter
        toks = np.ascontiguousarray(toks, dtype=np.int32)
        n = len(toks)
        hF = np.zeros((n, dm.d_model), dtype=np.float64)
        lg = np.zeros((n, dm.vocab), dtype=np.float64)
        a = None
        if add is not None:
            add = np.ascontiguousarray(add, dtype=np.float64)
            assert add.shape == (n, dm.d_model)
            a = add.ctypes.data
        self.lib.oracle_forward(self.h, which, toks.ctypes.data, n, a, hF.ctypes.data, lg.ctypes.data)
        return hF, lg

    def steer(self, h):
        h = np.ascontiguousarray(h, dtype=np.float64)
        s = np.zeros(self.wl.drafter.d_model, dtype=np.float64)
        self.lib.oracle_steer(self.h, h.ctypes.data, s.ctypes.data)
        return s

    def _bias_shape(self):
        dm = self.wl.drafter
        form = int(self.mlp.get("form", 1))
        if form == 3:
            return (dm.n_layers, int(self.mlp["rank"]))
        return (dm.n_layers, dm.d_ff) if form == 1 else (dm.d_model,)

    def ubias(self, b):
        """MLP steering: the biases of sequence b for its next round: per-layer up-projection
        biases [L_D][F_D] (form 1), the bias after every MLP [d_D] (form 2), or the g parts
        V_l^g g of the conditional biases [L_D][R] (form 3)."""
        out = np.zeros(self._bias_shape(), dtype=np.float64)
        self.lib.oracle_get_ubias(self.h, b, out.ctypes.data)
        return out

    def forward_mlp(self, which, toks, ubias=None, taps=False, obias=None):
        """Whole-sequence forward with optional up-projection biases [L][F] and a bias after every
        MLP [d] on every row; returns (hF [n][d], logits [n][V], taps [n][3][d] or None) in float64."""
        dm = self.wl.verifier if which == 0 else self.wl.drafter
        toks = np.ascontiguousarray(toks, dtype=np.int32)
        n = len(toks)
        hF = np.zeros((n, dm.d_model), dtype=np.float64)
        lg = np.zeros((n, dm.vocab), dtype=np.float64)
        tp = np.zeros((n, 3, dm.d_model), dtype=np.float64) if taps else None
        ub = None
        if ubias is not None:
            ubias = np.ascontiguousarray(ubias, dtype=np.float64)
            assert ubias.shape == (dm.n_layers, dm.d_ff)
            ub = ubias.ctypes.data
        ob = None
        if obias is not None:
            obias = np.ascontiguousarray(obias, dtype=np.float64)
            assert obias.shape == (dm.d_model,)
            ob = obias.ctypes.data
        self.lib.oracle_forward_mlp(self.h, which, toks.ctypes.data, n, ub, ob, tp.ctypes.data if taps else None,
                                    hF.ctypes.data, lg.ctypes.data)
        return hF, lg, tp

    def mlp_steer(self, z):
        """ub = W_s LayerNorm(W_hml z) for z = [h; m; l] (3 d_V); returns [L_D][F_D] (form 2: [d_D])."""
        z = np.ascontiguousarray(z, dtype=np.float64).reshape(-1)
        ub = np.zeros(self._bias_shape(), dtype=np.float64)
        self.lib.oracle_mlp_steer(self.h, z.ctypes.data, ub.ctypes.data)
        return ub

    def forward_cond(self, which, toks, c=None):
        """Whole-sequence forward with the conditional MLP bias of form 3 on every row, for the g
        whose parts V_l^g g are c [L][R] (None: no bias); returns (hF [n][d], logits [n][V])."""
        dm = self.wl.verifier if which == 0 else self.wl.drafter
        toks = np.ascontiguousarray(toks, dtype=np.int32)
        n = len(toks)
        hF = np.zeros((n, dm.d_model), dtype=np.float64)
        lg = np.zeros((n, dm.vocab), dtype=np.float64)
        cp = None
        if c is not None:
            c = np.ascontiguousarray(c, dtype=np.float64)
            assert c.shape == (dm.n_layers, int(self.mlp["rank"]))
            cp = c.ctypes.data
        self.lib.oracle_forward_cond(self.h, which, toks.ctypes.data, n, cp, hF.ctypes.data, lg.ctypes.data)
        return hF, lg

    def train_loss(self, toks, deltas, spread=False):
        """Training-objective forward (input-form steering): per-target KL divergences [n] (entry 0
        is 0) and their mean over targets 1..n-1, for tokens x_0..x_{n-1} and offsets deltas[tau];
        with spread=True also E_pV|d - KL| per target (d = log p_V - log p_D)."""
        toks = np.ascontiguousarray(toks, dtype=np.int32)
        deltas = np.ascontiguousarray(deltas, dtype=np.int32)
        assert len(deltas) == len(toks)
        kl = np.zeros(len(toks), dtype=np.float64)
        sp = np.zeros(len(toks), dtype=np.float64)
        mean = self.lib.oracle_train_loss(self.h, toks.ctypes.data, len(toks), deltas.ctypes.data, kl.ctypes.data,
                                          sp.ctypes.data if spread else None)
        return (float(mean), kl, sp) if spread else (float(mean), kl)
