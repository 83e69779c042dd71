"""Plain CPU reference ("oracle") of the BART sweep of arXiv 2410.23244.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product path
(``paper_2410_23244_amd``) never imports it, and this package never imports the
product: the two share no code.  The arithmetic lives in ``bart_oracle.c``
(scalar C, fp64 accumulation, one observation at a time); this module only
marshals numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bart_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain -O2, no fast-math, no contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-Wall", "-ffp-contract=off",
                               "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class Config(C.Structure):
    _fields_ = [("n", C.c_int32), ("p", C.c_int32), ("m", C.c_int32), ("D", C.c_int32),
                ("idx_bytes", C.c_int32), ("fix_sigma2", C.c_int32),
                ("chain", C.c_int32), ("pad", C.c_int32), ("alpha", C.c_double), ("beta", C.c_double), ("mu_mu", C.c_double),
                ("sigma_mu", C.c_double), ("nu", C.c_double), ("lam", C.c_double),
                ("p_grow", C.c_double), ("probit", C.c_int32), ("pad2", C.c_int32),
                ("probit_offset", C.c_double)]


class _State(C.Structure):
    _fields_ = [("axis", C.c_void_p), ("cut", C.c_void_p), ("leaf", C.c_void_p),
                ("idx", C.c_void_p), ("resid", C.c_void_p), ("sigma2", C.c_double),
                ("sweep", C.c_int64), ("next", C.c_int32), ("latent", C.c_void_p),
                ("ybin", C.c_void_p)]


TRACE_DTYPE = np.dtype([
    ("kind", "<i4"), ("tree", "<i4"), ("sweep", "<i8"), ("move", "<i4"), ("eta", "<i4"),
    ("axis", "<i4"), ("cut", "<i4"), ("n_grow_cand", "<i4"), ("n_prune_cand", "<i4"),
    ("accept", "<i4"), ("n_leaves", "<i4"), ("log_r", "<f8"), ("ln_u", "<f8"),
    ("log_r_scale", "<f8"), ("ssr", "<f8"), ("sigma2", "<f8"), ("pad", "<i4", (10,)),
    ("count", "<i4", (256,)), ("sum", "<f8", (256,)), ("leaf_new", "<f4", (256,))])
assert TRACE_DTYPE.itemsize == 4224

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = C.CDLL(_LIB)
        vp, i32, i64, u64, f64 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64, C.c_double
        P = C.POINTER
        L.oc_philox4x64_10.argtypes = [vp, vp, vp]
        L.oc_normal.argtypes = [u64, u64, u64, u64]
        L.oc_normal.restype = f64
        L.oc_norm_cdf.argtypes = [f64]
        L.oc_norm_cdf.restype = f64
        L.oc_norm_ppf.argtypes = [f64]
        L.oc_norm_ppf.restype = f64
        L.oc_latent_draw.argtypes = [f64, i32, f64]
        L.oc_latent_draw.restype = f64
        L.oc_gamma_draw.argtypes = [u64, u64, f64]
        L.oc_gamma_draw.restype = f64
        L.oc_sigma2_draw.argtypes = [u64, u64, f64, f64, i64, f64]
        L.oc_sigma2_draw.restype = f64
        L.oc_tree_info.argtypes = [P(Config), vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.oc_log_prior.argtypes = [P(Config), vp, vp, vp]
        L.oc_log_prior.restype = f64
        L.oc_propose.argtypes = [P(Config), vp, vp, vp, vp, vp]
        L.oc_llr.argtypes = [f64] * 7
        L.oc_llr.restype = f64
        L.oc_leaf_posterior.argtypes = [f64] * 5 + [P(f64), P(f64)]
        L.oc_log_ratio.argtypes = [P(Config), vp, vp, i64, vp, vp, vp, vp, vp, f64, i32, i32,
                                   i32, i32, P(f64)]
        L.oc_log_ratio.restype = f64
        L.oc_route.argtypes = [i32, vp, vp, vp, i64, i64]
        L.oc_route.restype = i32
        L.oc_step.argtypes = [P(Config), vp, vp, i64, P(_State), u64, i32, vp, vp]
        L.oc_step.restype = C.c_int
        L.oc_run.argtypes = [P(Config), vp, vp, i64, P(_State), u64, i64, vp]
        L.oc_run.restype = C.c_int
        L.oc_predict.argtypes = [P(Config), vp, vp, vp, vp, i64, i64, f64, vp]
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data


def make_config(n, p, m, D, idx_bytes=1, alpha=0.95, beta=2.0, mu_mu=0.0, sigma_mu=1.0,
                nu=3.0, lam=1.0, p_grow=0.5, fix_sigma2=False, chain=0, probit=False,
                probit_offset=0.0) -> Config:
    """chain selects the random stream: counter word 3 offset by chain * 2^32.
    probit: binary y, latent normals, sigma^2 held at its initial value 1."""
    return Config(int(n), int(p), int(m), int(D), int(idx_bytes), int(bool(fix_sigma2)),
                  int(chain), 0, float(alpha), float(beta), float(mu_mu), float(sigma_mu), float(nu),
                  float(lam), float(p_grow), int(bool(probit)), 0, float(probit_offset))


def philox(counter, key) -> np.ndarray:
    ctr = np.ascontiguousarray(counter, dtype=np.uint64)
    k = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.zeros(4, dtype=np.uint64)
    lib().oc_philox4x64_10(_ptr(ctr), _ptr(k), _ptr(out))
    return out


def norm_cdf(x) -> float:
    return lib().oc_norm_cdf(float(x))


def norm_ppf(p) -> float:
    return lib().oc_norm_ppf(float(p))


def latent_draw(f, y, u) -> float:
    return lib().oc_latent_draw(float(f), int(y), float(u))


def normal(seed, s, j, slot) -> float:
    return lib().oc_normal(seed, s, j, slot)


def gamma_draw(seed, s, shape) -> float:
    return lib().oc_gamma_draw(seed, s, shape)


def sigma2_draw(seed, s, nu, lam, n, ssr) -> float:
    return lib().oc_sigma2_draw(seed, s, nu, lam, n, ssr)


def llr(sigma2, mu_mu, sigma_mu, nL, SL, nR, SR) -> float:
    return lib().oc_llr(sigma2, mu_mu, sigma_mu, nL, SL, nR, SR)


def leaf_posterior(n, S, sigma2, mu_mu, sigma_mu):
    mean, prec = C.c_double(), C.c_double()
    lib().oc_leaf_posterior(n, S, sigma2, mu_mu, sigma_mu, C.byref(mean), C.byref(prec))
    return mean.value, prec.value


def tree_info(cfg: Config, n_cuts, axis, cut) -> dict:
    H = 1 << (cfg.D - 1)
    n_cuts = np.ascontiguousarray(n_cuts, dtype=np.int32)
    axis = np.ascontiguousarray(axis, dtype=np.uint16)
    cut = np.ascontiguousarray(cut, dtype=np.uint8)
    is_leaf = np.zeros(2 * H, np.int32)
    p_adj = np.zeros(2 * H, np.int32)
    p_split = np.zeros(2 * H, np.float64)
    G = np.zeros(2 * H, np.int32)
    P = np.zeros(2 * H, np.int32)
    nG = np.zeros(1, np.int32)
    nP = np.zeros(1, np.int32)
    lib().oc_tree_info(C.byref(cfg), _ptr(n_cuts), _ptr(axis), _ptr(cut), _ptr(is_leaf),
                       _ptr(p_adj), _ptr(p_split), _ptr(G), _ptr(nG), _ptr(P), _ptr(nP))
    return dict(is_leaf=is_leaf, p_adj=p_adj, p_split=p_split, grow=G[: nG[0]].copy(),
                prune=P[: nP[0]].copy())


def log_prior(cfg: Config, n_cuts, axis, cut) -> float:
    n_cuts = np.ascontiguousarray(n_cuts, dtype=np.int32)
    axis = np.ascontiguousarray(axis, dtype=np.uint16)
    cut = np.ascontiguousarray(cut, dtype=np.uint8)
    return lib().oc_log_prior(C.byref(cfg), _ptr(n_cuts), _ptr(axis), _ptr(cut))


def propose(cfg: Config, n_cuts, axis, cut, words):
    n_cuts = np.ascontiguousarray(n_cuts, dtype=np.int32)
    axis = np.ascontiguousarray(axis, dtype=np.uint16)
    cut = np.ascontiguousarray(cut, dtype=np.uint8)
    w = np.ascontiguousarray(words, dtype=np.uint64)
    out = np.zeros(6, np.int32)
    lib().oc_propose(C.byref(cfg), _ptr(n_cuts), _ptr(axis), _ptr(cut), _ptr(w), _ptr(out))
    return tuple(int(v) for v in out)


def log_ratio(cfg: Config, n_cuts, X, axis, cut, leaf, idx_row, resid, sigma2, move, eta, a,
              s):
    """log r of the move on one tree given the data; returns (log r, sum |terms|)."""
    n_cuts = np.ascontiguousarray(n_cuts, dtype=np.int32)
    X = np.ascontiguousarray(X, dtype=np.uint8)
    axis = np.ascontiguousarray(axis, dtype=np.uint16)
    cut = np.ascontiguousarray(cut, dtype=np.uint8)
    leaf = np.ascontiguousarray(leaf, dtype=np.float32)
    idx_row = np.ascontiguousarray(idx_row, dtype=np.uint8 if cfg.idx_bytes == 1 else np.uint16)
    resid = np.ascontiguousarray(resid, dtype=np.float32)
    scale = C.c_double()
    v = lib().oc_log_ratio(C.byref(cfg), _ptr(n_cuts), _ptr(X), X.shape[1], _ptr(axis),
                           _ptr(cut), _ptr(leaf), _ptr(idx_row), _ptr(resid), sigma2, move,
                           eta, a, s, C.byref(scale))
    return v, scale.value


def route(D, axis, cut, X, i) -> int:
    axis = np.ascontiguousarray(axis, dtype=np.uint16)
    cut = np.ascontiguousarray(cut, dtype=np.uint8)
    X = np.ascontiguousarray(X, dtype=np.uint8)
    return lib().oc_route(D, _ptr(axis), _ptr(cut), _ptr(X), X.shape[1], i)


class Chain:
    """One BART chain on the CPU.  State arrays are numpy and may be loaded
    from (or compared with) a device snapshot: axis u16 [m][H], cut u8 [m][H],
    leaf f32 [m][2H], idx u8|u16 [m][n], resid f32 [n], sigma2, sweep, next."""

    def __init__(self, cfg: Config, X: np.ndarray, n_cuts, y_c: np.ndarray, sigma2: float):
        self.cfg = cfg
        self.X = np.ascontiguousarray(X, dtype=np.uint8)
        assert self.X.shape[0] == cfg.p and self.X.shape[1] >= cfg.n
        self.n_cuts = np.ascontiguousarray(n_cuts, dtype=np.int32)
        H = 1 << (cfg.D - 1)
        m, n = cfg.m, cfg.n
        self.axis = np.zeros((m, H), np.uint16)
        self.cut = np.zeros((m, H), np.uint8)
        self.leaf = np.zeros((m, 2 * H), np.float32)
        self.idx = np.ones((m, n), np.uint8 if cfg.idx_bytes == 1 else np.uint16)
        self.resid = np.ascontiguousarray(y_c[:n], dtype=np.float32).copy()
        self.sigma2 = float(sigma2)
        self.sweep = 0
        self.next = 0
        self.latent = self.ybin = None
        if cfg.probit:
            # binary y = [y_c > 0]; latents start at +-1 on their side of 0,
            # residuals at z - offset (the trees are all zero); sigma^2 = 1
            self.ybin = (np.asarray(y_c[:n]) > 0).astype(np.uint8)
            self.latent = np.where(self.ybin == 1, 1.0, -1.0).astype(np.float32)
            self.resid = (self.latent.astype(np.float64) - cfg.probit_offset).astype(np.float32)
            self.sigma2 = 1.0

    def load(self, axis, cut, leaf, idx, resid, sigma2, sweep, next_step=0, latent=None):
        if latent is not None:
            self.latent[...] = latent
        self.axis[...] = axis
        self.cut[...] = cut
        self.leaf[...] = leaf
        self.idx[...] = idx
        self.resid[...] = resid
        self.sigma2 = float(sigma2)
        self.sweep = int(sweep)
        self.next = int(next_step)

    def _state(self) -> _State:
        return _State(_ptr(self.axis), _ptr(self.cut), _ptr(self.leaf), _ptr(self.idx),
                      _ptr(self.resid), self.sigma2, self.sweep, self.next,
                      None if self.latent is None else _ptr(self.latent),
                      None if self.ybin is None else _ptr(self.ybin))

    def _pull(self, st: _State):
        self.sigma2 = st.sigma2
        self.sweep = st.sweep
        self.next = st.next

    def step(self, seed: int, force: int = -1, trace: bool = True, adopt=None):
        """One step: tree step `next` of the current sweep, or the sigma^2 step.
        force (0/1) and adopt (256 leaf values) are lockstep hooks: the state
        continues from that decision / those draws; the trace still reports
        the oracle's own."""
        st = self._state()
        tr = np.zeros(1, TRACE_DTYPE) if trace else None
        ad = None if adopt is None else np.ascontiguousarray(adopt, dtype=np.float32)
        rc = lib().oc_step(C.byref(self.cfg), _ptr(self.n_cuts), _ptr(self.X), self.X.shape[1],
                           C.byref(st), seed, force, None if ad is None else _ptr(ad),
                           _ptr(tr) if trace else None)
        if rc:
            raise RuntimeError(f"oracle step failed ({rc})")
        self._pull(st)
        return tr[0] if trace else None

    def run(self, seed: int, n_steps: int, trace: bool = False):
        st = self._state()
        tr = np.zeros(n_steps, TRACE_DTYPE) if trace else None
        rc = lib().oc_run(C.byref(self.cfg), _ptr(self.n_cuts), _ptr(self.X), self.X.shape[1],
                          C.byref(st), seed, n_steps, _ptr(tr) if trace else None)
        if rc:
            raise RuntimeError(f"oracle run failed ({rc})")
        self._pull(st)
        return tr

    def sweeps(self, seed: int, k: int):
        """k whole sweeps (the chain must sit at a sweep boundary)."""
        assert self.next == 0
        self.run(seed, k * (self.cfg.m + 1))

    def predict(self, Xt: np.ndarray, offset: float = 0.0) -> np.ndarray:
        Xt = np.ascontiguousarray(Xt, dtype=np.uint8)
        out = np.zeros(Xt.shape[1], np.float32)
        lib().oc_predict(C.byref(self.cfg), _ptr(self.axis), _ptr(self.cut), _ptr(self.leaf),
                         _ptr(Xt), Xt.shape[1], Xt.shape[1], offset, _ptr(out))
        return out


def config_for(inp, fix_sigma2=False, chain=0) -> Config:
    """Oracle configuration of a generated workload (an ``Inputs`` object of the
    seeded input generators: shapes in n, p, m, D, idx_bytes, hyperparameters
    in ``hyper``).  The oracle always keeps an index cache: u8 when the device
    runs without one."""
    h = inp.hyper
    probit = bool(getattr(inp, "probit", False))
    return make_config(n=inp.n, p=inp.p, m=inp.m, D=inp.D, idx_bytes=inp.idx_bytes or 1,
                       alpha=h.alpha, beta=h.beta, mu_mu=h.mu_mu, sigma_mu=h.sigma_mu,
                       nu=h.nu, lam=h.lam, p_grow=h.p_grow, fix_sigma2=fix_sigma2,
                       chain=chain, probit=probit,
                       probit_offset=inp.offset if probit else 0.0)


def chain_from_state(inp, st: dict, chain: int = 0) -> Chain:
    """An oracle chain of workload inp (random stream `chain`) loaded with a
    state snapshot: a dict with axis, cut, leaf, idx, resid, sigma2, sweep,
    next (and latent for probit), in the layouts of ``Chain``."""
    ch = Chain(config_for(inp, chain=chain), inp.X_b, inp.n_cuts, inp.y_c, st["sigma2"])
    ch.load(st["axis"], st["cut"], st["leaf"], st["idx"], st["resid"], st["sigma2"],
            st["sweep"], st["next"], latent=st.get("latent"))
    return ch
