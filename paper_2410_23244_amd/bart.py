"""Thin Python binding of libbart (include/bart.h): argument marshalling only.

Every step of the sweep runs in the HIP kernels of libbart.so; PyTorch only
provides device memory and the stream.  The functions below carry the C names
(``bart_init``, ``bart_step`` ...); :class:`Bart` bundles them with the device
buffers a chain needs.  There is no CPU fallback: if the library is missing
or no GPU is visible, the calls raise.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libbart.so")

BART_OK, BART_EINVAL, BART_ENOSPACE, BART_EHIP, BART_ESTATE, BART_ENOTSUP, BART_EDEVICE = (
    0, -1, -2, -3, -4, -5, -6)


class BartError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libbart error {code}: {msg}")
        self.code = code


BART_LAUNCH_COOPERATIVE = 0
BART_LAUNCH_ORDINARY = 1
BART_RESID_AUTO, BART_RESID_REGISTERS, BART_RESID_STREAMED = 0, 1, 2
BART_GRID_UNIFORM, BART_GRID_QUANTILE = 0, 1


class Config(C.Structure):
    _fields_ = [("n", C.c_int32), ("p", C.c_int32), ("ntree", C.c_int32),
                ("max_depth", C.c_int32), ("idx_bytes", C.c_int32), ("grid", C.c_int32),
                ("launch", C.c_int32), ("residency", C.c_int32), ("nchain", C.c_int32),
                ("probit", C.c_int32), ("x_stride", C.c_int64),
                ("alpha", C.c_double), ("beta", C.c_double),
                ("mu_mu", C.c_double), ("sigma_mu", C.c_double), ("nu", C.c_double),
                ("lam", C.c_double), ("sigma2_init", C.c_double), ("p_grow", C.c_double),
                ("probit_offset", C.c_double)]


class State(C.Structure):
    _fields_ = [("axis", C.c_void_p), ("cut", C.c_void_p), ("leaf", C.c_void_p),
                ("idx", C.c_void_p), ("resid", C.c_void_p), ("sigma2", C.c_double),
                ("sweep", C.c_int64), ("next", C.c_int32), ("chain", C.c_int32),
                ("latent", C.c_void_p), ("count", C.c_void_p)]


class LaunchInfo(C.Structure):
    _fields_ = [("grid", C.c_int32), ("block", C.c_int32), ("chunks_per_thread", C.c_int32),
                ("lds_bytes", C.c_int32), ("obs_per_thread", C.c_int32),
                ("max_leaves", C.c_int32), ("launch", C.c_int32), ("residency", C.c_int32),
                ("nchain", C.c_int32), ("rank_stash", C.c_int32),
                ("stash_chunks", C.c_int32), ("lds_resid_chunks", C.c_int32)]


# bart_trace, 4224 bytes (include/bart.h)
TRACE_DTYPE = np.dtype([
    ("kind", "<i4"), ("tree", "<i4"), ("sweep", "<i8"), ("move", "<i4"), ("eta", "<i4"),
    ("axis", "<i4"), ("cut", "<i4"), ("n_grow_cand", "<i4"), ("n_prune_cand", "<i4"),
    ("accept", "<i4"), ("n_leaves", "<i4"), ("log_r", "<f8"), ("ln_u", "<f8"),
    ("log_r_scale", "<f8"), ("ssr", "<f8"), ("sigma2", "<f8"), ("pad", "<i4", (10,)),
    ("count", "<i4", (256,)), ("sum", "<f8", (256,)), ("leaf_new", "<f4", (256,))])
assert TRACE_DTYPE.itemsize == 4224

_lib = None


def lib():
    """Load libbart.so (built in-tree by paper_2410_23244_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        vp, P = C.c_void_p, C.POINTER
        L.bart_workspace_bytes.argtypes = [P(Config)]
        L.bart_workspace_bytes.restype = C.c_size_t
        L.bart_init.argtypes = [P(Config), vp, vp, vp, vp, C.c_size_t, vp, P(vp)]
        L.bart_step.argtypes = [vp, C.c_int32, C.c_uint64]
        L.bart_step_static.argtypes = [vp, C.c_int32, C.c_uint64]
        L.bart_predict.argtypes = [vp, vp, C.c_int64, C.c_int64, C.c_double, vp]
        L.bart_predict_accumulate.argtypes = [vp, vp, C.c_int64, C.c_int64, C.c_double, vp, vp]
        L.bart_posterior_summary.argtypes = [vp, vp, vp, C.c_int64, C.c_int64, vp, vp]
        L.bart_cutpoints.argtypes = [vp, C.c_int64, C.c_int32, C.c_int64, C.c_int32, C.c_int32,
                                     vp, vp]
        L.bart_bin.argtypes = [vp, C.c_int64, C.c_int32, C.c_int64, vp, vp, C.c_int32, vp,
                               C.c_int64]
        L.bart_default_hyper.argtypes = [vp, C.c_int64, C.c_int32, vp, vp, P(Config)]
        L.bart_get_state.argtypes = [vp, P(State)]
        L.bart_set_state.argtypes = [vp, P(State)]
        L.bart_debug_steps.argtypes = [vp, C.c_int32, C.c_uint64, vp]
        L.bart_debug_stall.argtypes = [vp, C.c_int32, C.c_uint64, C.c_int32, C.c_uint32]
        L.bart_status.argtypes = [vp, P(C.c_uint32)]
        L.bart_launch_info.argtypes = [vp, P(LaunchInfo)]
        L.bart_move_stats.argtypes = [vp, C.c_int32, vp]
        L.bart_destroy.argtypes = [vp]
        L.bart_destroy.restype = None
        L.bart_last_error.restype = C.c_char_p
        for f in ["bart_init", "bart_step", "bart_step_static", "bart_predict", "bart_get_state", "bart_set_state",
                  "bart_debug_steps", "bart_debug_stall", "bart_status", "bart_launch_info",
                  "bart_predict_accumulate", "bart_posterior_summary", "bart_cutpoints", "bart_bin", "bart_default_hyper",
                  "bart_move_stats"]:
            getattr(L, f).restype = C.c_int
        _lib = L
    return _lib


def _check(rc: int) -> None:
    if rc != BART_OK:
        raise BartError(rc, lib().bart_last_error().decode())


# ---------------------------------------------------------------- C names

def bart_workspace_bytes(cfg: Config) -> int:
    return int(lib().bart_workspace_bytes(C.byref(cfg)))


def bart_init(cfg: Config, X_b_ptr: int, y_c_ptr: int, n_cuts: np.ndarray, ws_ptr: int,
              ws_bytes: int, stream: int) -> int:
    nc = np.ascontiguousarray(n_cuts, dtype=np.int32)
    h = C.c_void_p()
    _check(lib().bart_init(C.byref(cfg), X_b_ptr, y_c_ptr, nc.ctypes.data, ws_ptr, ws_bytes,
                           stream, C.byref(h)))
    return h.value


def bart_step(h: int, k_sweeps: int, seed: int) -> None:
    _check(lib().bart_step(h, int(k_sweeps), int(seed)))


def bart_step_static(h: int, k_sweeps: int, seed: int) -> None:
    _check(lib().bart_step_static(h, int(k_sweeps), int(seed)))


def bart_predict(h: int, xt_ptr: int, xt_stride: int, n_t: int, offset: float,
                 out_ptr: int) -> None:
    _check(lib().bart_predict(h, xt_ptr, int(xt_stride), int(n_t), float(offset), out_ptr))


def bart_predict_accumulate(h: int, xt_ptr: int, xt_stride: int, n_t: int, offset: float,
                            sum_ptr: int, sumsq_ptr: int) -> None:
    _check(lib().bart_predict_accumulate(h, xt_ptr, int(xt_stride), int(n_t), float(offset),
                                         sum_ptr, sumsq_ptr))


def bart_posterior_summary(h: int, sum_ptr: int, sumsq_ptr: int, n_t: int, n_keep: int,
                           mean_ptr: int, sd_ptr: int) -> None:
    _check(lib().bart_posterior_summary(h, sum_ptr, sumsq_ptr, int(n_t), int(n_keep), mean_ptr,
                                        sd_ptr))


def bart_cutpoints(X: np.ndarray, K: int, grid: int) -> tuple[np.ndarray, np.ndarray]:
    """Host splitting grid of X (f32 [p][n]): cuts f64 [p][K], n_cuts i32 [p]."""
    X = np.ascontiguousarray(X, dtype=np.float32)
    p, n = X.shape
    cuts = np.empty((p, K), np.float64)
    nc = np.empty(p, np.int32)
    _check(lib().bart_cutpoints(X.ctypes.data, n, p, n, int(K), int(grid), cuts.ctypes.data,
                                nc.ctypes.data))
    return cuts, nc


def bart_bin(X: np.ndarray, cuts: np.ndarray, n_cuts: np.ndarray) -> np.ndarray:
    """Host binning of X (f32 [p][n]) on a grid from bart_cutpoints: u8 [p][n]."""
    X = np.ascontiguousarray(X, dtype=np.float32)
    cuts = np.ascontiguousarray(cuts, dtype=np.float64)
    nc = np.ascontiguousarray(n_cuts, dtype=np.int32)
    p, n = X.shape
    out = np.empty((p, n), np.uint8)
    _check(lib().bart_bin(X.ctypes.data, n, p, n, cuts.ctypes.data, nc.ctypes.data,
                          cuts.shape[1], out.ctypes.data, n))
    return out


def bart_default_hyper(y: np.ndarray, ntree: int) -> tuple[float, np.ndarray, Config]:
    """offset, y_c (f32) and a Config holding the default hyperparameters."""
    y = np.ascontiguousarray(y, dtype=np.float64)
    yc = np.empty(y.size, np.float32)
    off = C.c_double(0.0)
    cfg = Config()
    _check(lib().bart_default_hyper(y.ctypes.data, y.size, int(ntree), C.byref(off),
                                    yc.ctypes.data, C.byref(cfg)))
    return off.value, yc, cfg


def bart_get_state(h: int, st: State) -> None:
    _check(lib().bart_get_state(h, C.byref(st)))


def bart_set_state(h: int, st: State) -> None:
    _check(lib().bart_set_state(h, C.byref(st)))


def bart_debug_steps(h: int, n_steps: int, seed: int, trace_ptr: int) -> None:
    _check(lib().bart_debug_steps(h, int(n_steps), int(seed), trace_ptr))


def bart_debug_stall(h: int, n_steps: int, seed: int, wg: int, spin_limit: int) -> None:
    _check(lib().bart_debug_stall(h, int(n_steps), int(seed), int(wg), int(spin_limit)))


def bart_status(h: int) -> int:
    bits = C.c_uint32(0)
    rc = lib().bart_status(h, C.byref(bits))
    if rc not in (BART_OK, BART_EDEVICE):
        _check(rc)
    return int(bits.value)


def bart_launch_info(h: int) -> LaunchInfo:
    info = LaunchInfo()
    _check(lib().bart_launch_info(h, C.byref(info)))
    return info


def bart_move_stats(h: int, chain: int = 0) -> dict:
    out = np.zeros(6, np.uint64)
    _check(lib().bart_move_stats(h, int(chain), out.ctypes.data))
    keys = ["grow_proposed", "prune_proposed", "grow_accepted", "prune_accepted", "tree_steps",
            "leaves"]
    return {k: int(v) for k, v in zip(keys, out)}


def bart_destroy(h: int) -> None:
    lib().bart_destroy(h)


# ---------------------------------------------------------------- chain object

def x_stride_for(n: int) -> int:
    return (n + 255) // 256 * 256


class Bart:
    """nchain BART chains of one model on the current HIP device.

    X_b: uint8 [p][n] (numpy or torch); y_c: float32 [n]; n_cuts: int [p].
    The binned predictors are copied once to the device with a row stride that
    is a multiple of 256; the workspace is one torch uint8 tensor.  With one
    chain, traces and predictions are [n_steps] and [n_t]; with several they
    gain a leading chain axis."""

    def __init__(self, X_b, y_c, n_cuts, *, ntree: int, max_depth: int = 6,
                 idx_bytes: int = 1, alpha: float = 0.95, beta: float = 2.0,
                 mu_mu: float = 0.0, sigma_mu: float = 1.0, nu: float = 3.0,
                 lam: float = 1.0, sigma2_init: float = 1.0, p_grow: float = 0.5,
                 grid: int = 0, launch: int = 0, residency: int = 0, nchain: int = 1,
                 probit: bool = False, probit_offset: float = 0.0, device: str = "cuda"):
        import torch

        if not torch.cuda.is_available():
            raise RuntimeError("libbart needs a HIP device; none is visible")
        self.torch = torch
        self.device = torch.device(device)
        Xn = X_b.cpu().numpy() if hasattr(X_b, "cpu") else np.asarray(X_b)
        p, n = Xn.shape
        self.n, self.p, self.m, self.D, self.idx_bytes = n, p, ntree, max_depth, idx_bytes
        self.H = 1 << (max_depth - 1)
        self.x_stride = x_stride_for(n)
        Xd = torch.zeros((p, self.x_stride), dtype=torch.uint8, device=self.device)
        Xd[:, :n] = torch.from_numpy(np.ascontiguousarray(Xn, dtype=np.uint8)).to(self.device)
        self.X = Xd
        yn = y_c.cpu().numpy() if hasattr(y_c, "cpu") else np.asarray(y_c)
        self.y = torch.from_numpy(np.ascontiguousarray(yn, dtype=np.float32)).to(self.device)
        self.n_cuts = np.ascontiguousarray(n_cuts, dtype=np.int32)
        self.nchain = nchain
        self.probit = bool(probit)
        self.cfg = Config(n, p, ntree, max_depth, idx_bytes, grid, launch, residency, nchain,
                          int(self.probit), self.x_stride, alpha, beta, mu_mu, sigma_mu, nu, lam,
                          sigma2_init, p_grow, probit_offset)
        nbytes = bart_workspace_bytes(self.cfg)
        if nbytes == 0:
            raise BartError(BART_EINVAL, "invalid configuration")
        self.ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        base = self.ws.data_ptr()
        self.ws_ptr = (base + 255) // 256 * 256
        self.ws_bytes = nbytes
        self.stream = torch.cuda.current_stream(self.device)
        self.h = bart_init(self.cfg, self.X.data_ptr(), self.y.data_ptr(), self.n_cuts,
                           self.ws_ptr, nbytes, self.stream.cuda_stream)

    # -- running
    def step(self, k_sweeps: int, seed: int) -> None:
        bart_step(self.h, k_sweeps, seed)

    def step_static(self, k_sweeps: int, seed: int) -> None:
        bart_step_static(self.h, k_sweeps, seed)

    def debug_steps(self, n_steps: int, seed: int) -> np.ndarray:
        torch = self.torch
        C_ = self.nchain
        buf = torch.zeros(C_ * n_steps * TRACE_DTYPE.itemsize, dtype=torch.uint8,
                          device=self.device)
        bart_debug_steps(self.h, n_steps, seed, buf.data_ptr())
        self.stream.synchronize()
        tr = buf.cpu().numpy().view(TRACE_DTYPE)
        return tr if C_ == 1 else tr.reshape(C_, n_steps)

    def debug_stall(self, n_steps: int, seed: int, wg: int, spin_limit: int) -> None:
        """One launch with workgroup wg left out and every cross-workgroup wait
        bounded by spin_limit poll rounds (the timeout path); see bart.h."""
        bart_debug_stall(self.h, n_steps, seed, wg, spin_limit)
        self.stream.synchronize()

    def predict(self, Xt, offset: float = 0.0):
        torch = self.torch
        Xn = Xt.cpu().numpy() if hasattr(Xt, "cpu") else np.asarray(Xt)
        p, nt = Xn.shape
        assert p == self.p
        stride = x_stride_for(nt)
        Xd = torch.zeros((p, stride), dtype=torch.uint8, device=self.device)
        Xd[:, :nt] = torch.from_numpy(np.ascontiguousarray(Xn, dtype=np.uint8)).to(self.device)
        out = torch.empty((self.nchain, nt), dtype=torch.float32, device=self.device)
        bart_predict(self.h, Xd.data_ptr(), stride, nt, offset, out.data_ptr())
        self.stream.synchronize()
        return out[0] if self.nchain == 1 else out

    def upload_x(self, Xt):
        """Binned points (u8 [p][n_t]) on the device with a 256-multiple stride."""
        torch = self.torch
        Xn = Xt.cpu().numpy() if hasattr(Xt, "cpu") else np.asarray(Xt)
        p, nt = Xn.shape
        assert p == self.p
        stride = x_stride_for(nt)
        Xd = torch.zeros((p, stride), dtype=torch.uint8, device=self.device)
        Xd[:, :nt] = torch.from_numpy(np.ascontiguousarray(Xn, dtype=np.uint8)).to(self.device)
        return Xd, nt

    def predict_accumulate(self, Xd, nt: int, offset: float, acc_sum, acc_sumsq) -> None:
        """acc_sum/acc_sumsq: float64 device tensors [nchain][nt]; Xd from upload_x."""
        bart_predict_accumulate(self.h, Xd.data_ptr(), Xd.shape[1], nt, offset,
                                acc_sum.data_ptr(), acc_sumsq.data_ptr())

    def posterior_summary(self, acc_sum, acc_sumsq, nt: int, n_keep: int):
        """Pooled posterior mean and sd (float64 device tensors [nt]) from the
        accumulators of predict_accumulate over n_keep kept sweeps."""
        mean = self.torch.empty(nt, dtype=self.torch.float64, device=self.device)
        sd = self.torch.empty_like(mean)
        bart_posterior_summary(self.h, acc_sum.data_ptr(), acc_sumsq.data_ptr(), nt, n_keep,
                               mean.data_ptr(), sd.data_ptr())
        return mean, sd

    def status(self) -> int:
        return bart_status(self.h)

    def launch_info(self) -> LaunchInfo:
        return bart_launch_info(self.h)

    def move_stats(self, chain: int = 0) -> dict:
        return bart_move_stats(self.h, chain)

    # -- state
    def get_state(self, chain: int = 0) -> dict:
        torch = self.torch
        m, H, n = self.m, self.H, self.n
        it = torch.int16 if self.idx_bytes == 2 else torch.uint8  # 0: no cache, u8 leaves
        bufs = dict(axis=torch.empty((m, H), dtype=torch.int16, device=self.device),
                    cut=torch.empty((m, H), dtype=torch.uint8, device=self.device),
                    leaf=torch.empty((m, 2 * H), dtype=torch.float32, device=self.device),
                    idx=torch.empty((m, n), dtype=it, device=self.device),
                    resid=torch.empty(n, dtype=torch.float32, device=self.device))
        if self.probit:
            bufs["latent"] = torch.empty(n, dtype=torch.float32, device=self.device)
        bufs["count"] = torch.empty((m, 2 * H), dtype=torch.int32, device=self.device)
        st = State(bufs["axis"].data_ptr(), bufs["cut"].data_ptr(), bufs["leaf"].data_ptr(),
                   bufs["idx"].data_ptr(), bufs["resid"].data_ptr(), 0.0, 0, 0, int(chain),
                   bufs["latent"].data_ptr() if self.probit else None,
                   bufs["count"].data_ptr())
        bart_get_state(self.h, st)
        out = {k: v.cpu().numpy() for k, v in bufs.items()}
        out["axis"] = out["axis"].view(np.uint16)
        if self.idx_bytes == 2:
            out["idx"] = out["idx"].view(np.uint16)
        out.update(sigma2=st.sigma2, sweep=st.sweep, next=st.next)
        return out

    def sigma2(self, chain: int = 0) -> float:
        """Current sigma^2 of a chain (no array copies)."""
        st = State(None, None, None, None, None, 0.0, 0, 0, int(chain), None, None)
        bart_get_state(self.h, st)
        return st.sigma2

    def set_state(self, s: dict, chain: int = 0) -> None:
        torch = self.torch
        dev = {}
        keys = ["axis", "cut", "leaf", "idx", "resid"] + (["latent"] if self.probit else [])
        for k in keys:
            a = np.ascontiguousarray(s[k])
            if a.dtype == np.uint16:
                a = a.view(np.int16)
            dev[k] = torch.from_numpy(a).to(self.device)
        st = State(dev["axis"].data_ptr(), dev["cut"].data_ptr(), dev["leaf"].data_ptr(),
                   dev["idx"].data_ptr(), dev["resid"].data_ptr(), float(s["sigma2"]),
                   int(s["sweep"]), int(s.get("next", 0)), int(chain),
                   dev["latent"].data_ptr() if self.probit else None, None)
        bart_set_state(self.h, st)
        self.stream.synchronize()

    def close(self) -> None:
        if getattr(self, "h", None):
            bart_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def from_inputs(inp, grid: int = 0, launch: int = 0, residency: int = 0, nchain: int = 1) -> Bart:
    """Chains for a generated workload (paper_2410_23244_amd.inputs.Inputs);
    a probit workload gives probit chains with its offset."""
    h = inp.hyper
    return Bart(inp.X_b, inp.y_c, inp.n_cuts, ntree=inp.m, max_depth=inp.D,
                idx_bytes=inp.idx_bytes, alpha=h.alpha, beta=h.beta, mu_mu=h.mu_mu,
                sigma_mu=h.sigma_mu, nu=h.nu, lam=h.lam, sigma2_init=h.sigma2_init,
                p_grow=h.p_grow, grid=grid, launch=launch, residency=residency, nchain=nchain,
                probit=getattr(inp, "probit", False),
                probit_offset=inp.offset if getattr(inp, "probit", False) else 0.0)


class Regressor:
    """BART regression with the defaults of sec. 2.1: bins X on the host
    (bart_cutpoints, bart_bin), sets the hyperparameters from y
    (bart_default_hyper), runs nchain chains on the device and accumulates the
    posterior mean and sd of f at the test points over the kept sweeps
    (bart_predict_accumulate).  X is f32 [n][p] (one row per observation)."""

    def __init__(self, ntree: int = 200, max_depth: int = 6, K: int = 255,
                 grid: int = BART_GRID_QUANTILE, nchain: int = 1, seed: int = 0):
        self.ntree, self.max_depth, self.K, self.grid = ntree, max_depth, K, grid
        self.nchain, self.seed = nchain, seed

    def fit(self, X, y, X_test, n_burn: int = 100, n_keep: int = 1000):
        import torch

        Xt = np.ascontiguousarray(np.asarray(X, dtype=np.float32).T)
        Xs = np.ascontiguousarray(np.asarray(X_test, dtype=np.float32).T)
        self.cuts, self.n_cuts = bart_cutpoints(Xt, self.K, self.grid)
        Xb = bart_bin(Xt, self.cuts, self.n_cuts)
        Xsb = bart_bin(Xs, self.cuts, self.n_cuts)
        self.offset, yc, hc = bart_default_hyper(np.asarray(y, dtype=np.float64), self.ntree)
        self.chain = Bart(Xb, yc, self.n_cuts, ntree=self.ntree, max_depth=self.max_depth,
                          alpha=hc.alpha, beta=hc.beta, mu_mu=hc.mu_mu, sigma_mu=hc.sigma_mu,
                          nu=hc.nu, lam=hc.lam, sigma2_init=hc.sigma2_init, p_grow=hc.p_grow,
                          nchain=self.nchain)
        g = self.chain
        Xd, nt = g.upload_x(Xsb)
        s = torch.zeros((self.nchain, nt), dtype=torch.float64, device=g.device)
        s2 = torch.zeros_like(s)
        g.step(n_burn, self.seed)
        sig = np.empty((n_keep, self.nchain))
        for k in range(n_keep):
            g.step(1, self.seed)
            g.predict_accumulate(Xd, nt, self.offset, s, s2)
            for c in range(self.nchain):
                sig[k, c] = g.sigma2(c)
        if g.status():
            raise BartError(BART_EDEVICE, "device error during sampling")
        mean, sd = g.posterior_summary(s, s2, nt, n_keep)
        self.mean = mean.cpu().numpy()               # posterior mean over all chains
        self.sd = sd.cpu().numpy()
        self.sums = (s.cpu().numpy(), s2.cpu().numpy())  # [nchain][n_test] each
        self.n_keep = n_keep
        self.sigma2_trace = sig
        return self
