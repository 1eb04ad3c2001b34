"""ctypes binding of the CPU oracle (``oracle/soma_oracle.c``).

TEST INFRASTRUCTURE ONLY: the test suite, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg are the only callers.  The product package
never imports this module, and this module imports nothing from the product.

The oracle is a plain fp64 implementation of the SOMA SPSA step (paper
Section 4, Eq. main-spsa; Appendix E, Eq. localspsa; Appendix C for the
recurrent body), written from the paper without blocking or fusion.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

from .plateau import Plateau  # noqa: F401  (the lr / eps schedule, plain Python)

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "soma_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

CFLAGS = ["-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
          "-shared", "-fPIC"]


def build(force: bool = False) -> str:
    """Compile the oracle with the system C compiler (always when force)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cc = os.environ.get("CC", "gcc")
        subprocess.check_call([cc, *CFLAGS, "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class OracleCfg(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_experts", "n_layers", "embed", "hidden", "batch", "seq_len", "n_pairs", "loss_mode",
        "probe", "accum", "arch")] + [("tied_head", ctypes.c_void_p), ("head_stride", ctypes.c_int64),
                                      ("perturb_mask", ctypes.c_uint32)]


def _load():
    global _lib
    with _lock:
        if _lib is None:
            lib = ctypes.CDLL(build())
            P = ctypes.POINTER
            u32p, f32p, f64p = P(ctypes.c_uint32), P(ctypes.c_float), P(ctypes.c_double)
            u8p, u64p, i64p = P(ctypes.c_uint8), P(ctypes.c_uint64), P(ctypes.c_int64)
            cfgp = P(OracleCfg)
            sig = {
                "oracle_param_count": (ctypes.c_int64, [cfgp]),
                "oracle_philox4x32_10": (None, [u32p, u32p, u32p]),
                "oracle_series_constants": (None, [f32p]),
                "oracle_ln_u24": (ctypes.c_float, [ctypes.c_uint32]),
                "oracle_sincos_2pi_u24": (None, [ctypes.c_uint32, f32p, f32p]),
                "oracle_ln_u24_array": (None, [u32p, ctypes.c_int64, f32p]),
                "oracle_sincos_2pi_u24_array": (None, [u32p, ctypes.c_int64, f32p, f32p]),
                "oracle_box_muller": (None, [ctypes.c_uint32, ctypes.c_uint32, f32p, f32p]),
                "oracle_box_muller_array": (None, [u32p, u32p, ctypes.c_int64, f32p, f32p]),
                "oracle_gaussian": (None, [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint32,
                                           ctypes.c_uint64, ctypes.c_uint64, f32p]),
                "oracle_probe": (ctypes.c_int, [ctypes.c_int, ctypes.c_uint64, ctypes.c_uint64,
                                                ctypes.c_uint32, ctypes.c_uint64, ctypes.c_uint64,
                                                f32p]),
                "oracle_forward_loss_f64": (ctypes.c_double, [cfgp, f64p, u8p]),
                "oracle_forward_loss": (ctypes.c_double, [cfgp, f32p, u8p]),
                "oracle_perturb": (None, [cfgp, f32p, ctypes.c_uint64, ctypes.c_uint64,
                                          ctypes.c_uint32, ctypes.c_float, f32p]),
                "oracle_perturbed_loss": (ctypes.c_double, [cfgp, f32p, ctypes.c_uint64,
                                                            ctypes.c_uint64, ctypes.c_uint32,
                                                            ctypes.c_int, ctypes.c_float, u8p]),
                "oracle_apply_update": (None, [cfgp, f32p, ctypes.c_uint64, ctypes.c_uint64,
                                               ctypes.c_float, f64p, i64p, ctypes.c_int64,
                                               f32p, f64p]),
                "oracle_apply_adam": (None, [cfgp, f32p, f32p, f32p, ctypes.c_int64, ctypes.c_uint64,
                                             ctypes.c_uint64, ctypes.c_float, f64p, ctypes.c_double,
                                             ctypes.c_double, ctypes.c_double, ctypes.c_double, i64p,
                                             ctypes.c_int64, f32p, f32p, f32p, f64p]),
                "oracle_spsa_step": (ctypes.c_int, [cfgp, f32p, u64p, ctypes.c_uint64,
                                                    ctypes.c_float, ctypes.c_float, u8p, f32p,
                                                    f64p, f32p, f64p]),
                "oracle_spsa_step_rates": (ctypes.c_int, [cfgp, f32p, u64p, ctypes.c_uint64, f32p, f32p,
                                                          u8p, f32p, f64p, f32p, f64p]),
                "oracle_eval_loss": (ctypes.c_int, [cfgp, f32p, u8p, f64p]),
                "oracle_num_threads": (ctypes.c_int, []),
                "oracle_head_delta": (ctypes.c_double, [cfgp, f32p, u8p, f64p]),
            }
            for name, (res, args) in sig.items():
                fn = getattr(lib, name)
                fn.restype = res
                fn.argtypes = args
            _lib = lib
    return _lib


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


VOCAB = 256
PROBE_GAUSSIAN, PROBE_SPARSE_RADEMACHER, PROBE_RADEMACHER = 0, 1, 2


ARCH_LSTM, ARCH_PAPER_BODY, ARCH_WIDE = 0, 1, 2
# perturb_mask bits: the parameter groups that are perturbed and updated
# (0 = all of them).
PERTURB_EMBEDDING, PERTURB_LSTM, PERTURB_HEAD = 1, 2, 4


def make_cfg(n_experts, n_layers, embed, hidden, batch, seq_len, n_pairs, loss_mode=0,
             probe=PROBE_GAUSSIAN, accum=1, arch=ARCH_LSTM, tied_head=None, perturb_mask=0):
    """tied_head (arch 1, 2): the tied matrix E, [V][w] (shared by all
    experts) or [N][V][w] (one per expert), w = hidden for arch 1 and
    w = embed for arch 2; the configuration keeps it alive.
    perturb_mask: PERTURB_* bits of the perturbed and updated groups (0: all)."""
    cfg = OracleCfg(n_experts, n_layers, embed, hidden, batch, seq_len, n_pairs, loss_mode, probe, accum,
                    arch, None, 0, perturb_mask)
    if tied_head is not None:
        h = np.ascontiguousarray(tied_head, dtype=np.float32)
        cfg._head_ref = h
        cfg.tied_head = h.ctypes.data
        cfg.head_stride = 0 if h.ndim == 2 else VOCAB * (embed if arch == ARCH_WIDE else hidden)
    return cfg


def cfg_from(shape) -> OracleCfg:
    """Build the oracle's configuration from any object with the shape fields."""
    return make_cfg(shape.n_experts, shape.n_layers, shape.embed, shape.hidden, shape.batch,
                    shape.seq_len, shape.n_pairs, getattr(shape, "loss_mode", 0),
                    getattr(shape, "probe", PROBE_GAUSSIAN), getattr(shape, "accum", 1),
                    getattr(shape, "arch", ARCH_LSTM), getattr(shape, "tied_head", None),
                    getattr(shape, "perturb_mask", 0))


def head_delta(cfg: OracleCfg, theta_e, bytes_e):
    """(mean CE, dE [V][w] fp64): the decoder-path derivative of the
    unperturbed loss with respect to the tied matrix (arch 1 or 2; one
    expert, cfg.tied_head pointing at its E)."""
    t = np.ascontiguousarray(theta_e, dtype=np.float32)
    b = np.ascontiguousarray(bytes_e, dtype=np.uint8)
    g = np.empty((VOCAB, cfg.embed if cfg.arch == ARCH_WIDE else cfg.hidden), dtype=np.float64)
    loss = _load().oracle_head_delta(ctypes.byref(cfg), _ptr(t, ctypes.c_float), _ptr(b, ctypes.c_uint8),
                                     _ptr(g, ctypes.c_double))
    return float(loss), g


def param_count(cfg: OracleCfg) -> int:
    return int(_load().oracle_param_count(ctypes.byref(cfg)))


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def philox(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    _load().oracle_philox4x32_10(_ptr(c, ctypes.c_uint32), _ptr(k, ctypes.c_uint32),
                                 _ptr(out, ctypes.c_uint32))
    return out


def series_constants() -> np.ndarray:
    out = np.zeros(13, dtype=np.float32)
    _load().oracle_series_constants(_ptr(out, ctypes.c_float))
    return out


def ln_u24(m: int) -> np.float32:
    return np.float32(_load().oracle_ln_u24(int(m)))


def sincos_2pi_u24(i: int):
    c, s = ctypes.c_float(), ctypes.c_float()
    _load().oracle_sincos_2pi_u24(int(i), ctypes.byref(c), ctypes.byref(s))
    return np.float32(c.value), np.float32(s.value)


def ln_u24_array(m: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(m, dtype=np.uint32)
    out = np.empty(a.size, dtype=np.float32)
    _load().oracle_ln_u24_array(_ptr(a, ctypes.c_uint32), a.size, _ptr(out, ctypes.c_float))
    return out


def sincos_2pi_u24_array(i: np.ndarray):
    a = np.ascontiguousarray(i, dtype=np.uint32)
    c = np.empty(a.size, dtype=np.float32)
    s = np.empty(a.size, dtype=np.float32)
    _load().oracle_sincos_2pi_u24_array(_ptr(a, ctypes.c_uint32), a.size, _ptr(c, ctypes.c_float),
                                        _ptr(s, ctypes.c_float))
    return c, s


def box_muller(wa: int, wb: int):
    a, b = ctypes.c_float(), ctypes.c_float()
    _load().oracle_box_muller(int(wa), int(wb), ctypes.byref(a), ctypes.byref(b))
    return np.float32(a.value), np.float32(b.value)


def box_muller_array(wa: np.ndarray, wb: np.ndarray):
    a = np.ascontiguousarray(wa, dtype=np.uint32)
    b = np.ascontiguousarray(wb, dtype=np.uint32)
    za = np.empty(a.size, dtype=np.float32)
    zb = np.empty(a.size, dtype=np.float32)
    _load().oracle_box_muller_array(_ptr(a, ctypes.c_uint32), _ptr(b, ctypes.c_uint32), a.size,
                                    _ptr(za, ctypes.c_float), _ptr(zb, ctypes.c_float))
    return za, zb


def gaussian(seed: int, step: int, pair: int, k0: int, count: int) -> np.ndarray:
    out = np.empty(int(count), dtype=np.float32)
    _load().oracle_gaussian(int(seed), int(step), int(pair), int(k0), int(count),
                            _ptr(out, ctypes.c_float))
    return out


def probe(law: int, seed: int, step: int, pair: int, k0: int, count: int) -> np.ndarray:
    """Probe values z_pair[k0 .. k0+count) under law 0 (Gaussian), 1 (sparse
    Rademacher) or 2 (dense Rademacher)."""
    out = np.empty(int(count), dtype=np.float32)
    rc = _load().oracle_probe(int(law), int(seed), int(step), int(pair), int(k0), int(count),
                              _ptr(out, ctypes.c_float))
    if rc != 0:
        raise ValueError(f"unknown probe law {law}")
    return out


def forward_loss_f64(cfg: OracleCfg, w64: np.ndarray, bytes_e: np.ndarray) -> float:
    w = np.ascontiguousarray(w64, dtype=np.float64)
    b = np.ascontiguousarray(bytes_e, dtype=np.uint8)
    return float(_load().oracle_forward_loss_f64(ctypes.byref(cfg), _ptr(w, ctypes.c_double),
                                                  _ptr(b, ctypes.c_uint8)))


def forward_loss(cfg: OracleCfg, w32: np.ndarray, bytes_e: np.ndarray) -> float:
    w = np.ascontiguousarray(w32, dtype=np.float32)
    b = np.ascontiguousarray(bytes_e, dtype=np.uint8)
    return float(_load().oracle_forward_loss(ctypes.byref(cfg), _ptr(w, ctypes.c_float),
                                              _ptr(b, ctypes.c_uint8)))


def perturb(cfg: OracleCfg, theta_e: np.ndarray, seed: int, step: int, pair: int,
            sign_eps: float) -> np.ndarray:
    t = np.ascontiguousarray(theta_e, dtype=np.float32)
    out = np.empty_like(t)
    _load().oracle_perturb(ctypes.byref(cfg), _ptr(t, ctypes.c_float), int(seed), int(step),
                           int(pair), float(sign_eps), _ptr(out, ctypes.c_float))
    return out


def perturbed_loss(cfg: OracleCfg, theta_e: np.ndarray, seed: int, step: int, pair: int,
                   sign: int, eps: float, bytes_e: np.ndarray) -> float:
    t = np.ascontiguousarray(theta_e, dtype=np.float32)
    b = np.ascontiguousarray(bytes_e, dtype=np.uint8)
    return float(_load().oracle_perturbed_loss(ctypes.byref(cfg), _ptr(t, ctypes.c_float),
                                                int(seed), int(step), int(pair), int(sign),
                                                float(eps), _ptr(b, ctypes.c_uint8)))


def apply_update(cfg: OracleCfg, theta_e: np.ndarray, seed: int, step: int, lr: float,
                 coef: np.ndarray, ks=None, want_ghat: bool = False):
    """theta'[k] (and optionally g_hat[k]) for the given coefficients."""
    t = np.ascontiguousarray(theta_e, dtype=np.float32)
    cf = np.ascontiguousarray(coef, dtype=np.float64)
    if ks is None:
        n, ksp, nk = t.size, None, 0
    else:
        ka = np.ascontiguousarray(ks, dtype=np.int64)
        n, ksp, nk = ka.size, _ptr(ka, ctypes.c_int64), ka.size
    out = np.empty(n, dtype=np.float32)
    gh = np.empty(n, dtype=np.float64) if want_ghat else None
    _load().oracle_apply_update(ctypes.byref(cfg), _ptr(t, ctypes.c_float), int(seed), int(step),
                                float(lr), _ptr(cf, ctypes.c_double), ksp, nk,
                                _ptr(out, ctypes.c_float),
                                _ptr(gh, ctypes.c_double) if want_ghat else None)
    return (out, gh) if want_ghat else out


ADAM_DEFAULTS = dict(beta1=0.9, beta2=0.999, delta=1e-8, weight_decay=1e-4)


def apply_adam(cfg: OracleCfg, theta_e, m_e, v_e, t: int, seed: int, step: int, lr: float, coef,
               beta1=0.9, beta2=0.999, delta=1e-8, weight_decay=1e-4, ks=None, want_ghat=False):
    """The paper's Adam-style update of one expert (update number t >= 1)
    from the coefficients coef[j]; returns (theta', m', v'[, g_hat])."""
    th = np.ascontiguousarray(theta_e, dtype=np.float32)
    m = np.ascontiguousarray(m_e, dtype=np.float32)
    v = np.ascontiguousarray(v_e, dtype=np.float32)
    cf = np.ascontiguousarray(coef, dtype=np.float64)
    if ks is None:
        n, kp = th.size, None
    else:
        kk = np.ascontiguousarray(ks, dtype=np.int64)
        n, kp = kk.size, _ptr(kk, ctypes.c_int64)
    to = np.empty(n, np.float32)
    mo = np.empty(n, np.float32)
    vo = np.empty(n, np.float32)
    gh = np.empty(n, np.float64) if want_ghat else None
    _load().oracle_apply_adam(ctypes.byref(cfg), _ptr(th, ctypes.c_float), _ptr(m, ctypes.c_float),
                              _ptr(v, ctypes.c_float), int(t), int(seed), int(step), float(lr),
                              _ptr(cf, ctypes.c_double), float(beta1), float(beta2), float(delta),
                              float(weight_decay), kp, n, _ptr(to, ctypes.c_float),
                              _ptr(mo, ctypes.c_float), _ptr(vo, ctypes.c_float),
                              _ptr(gh, ctypes.c_double) if want_ghat else None)
    return (to, mo, vo, gh) if want_ghat else (to, mo, vo)


def spsa_step(cfg: OracleCfg, theta: np.ndarray, seeds, step: int, eps, lr,
              bytes_all: np.ndarray, want_ghat: bool = False):
    """Full oracle step.  bytes_all is [N][B][T], or [A][N][B][T] with A =
    cfg.accum accumulation batches.  eps and lr are scalars, or [N] arrays
    (one radius and learning rate per expert).  Returns dict(losses [N,D,2]
    f32, coef [N,D] f64, theta [N,d] f32, ghat [N,d] f64 or None), D = A P
    directions."""
    A = max(1, cfg.accum)
    N, P = cfg.n_experts, cfg.n_pairs * A
    d = param_count(cfg)
    t = np.ascontiguousarray(theta, dtype=np.float32).reshape(N, d)
    sd = np.ascontiguousarray(seeds, dtype=np.uint64).reshape(N)
    b = np.ascontiguousarray(bytes_all, dtype=np.uint8).reshape(A, N, cfg.batch, cfg.seq_len)
    losses = np.empty((N, P, 2), dtype=np.float32)
    coef = np.empty((N, P), dtype=np.float64)
    out = np.empty_like(t)
    gh = np.empty((N, d), dtype=np.float64) if want_ghat else None
    if np.ndim(eps) == 0 and np.ndim(lr) == 0:
        rc = _load().oracle_spsa_step(ctypes.byref(cfg), _ptr(t, ctypes.c_float),
                                      _ptr(sd, ctypes.c_uint64), int(step), float(eps), float(lr),
                                      _ptr(b, ctypes.c_uint8), _ptr(losses, ctypes.c_float),
                                      _ptr(coef, ctypes.c_double), _ptr(out, ctypes.c_float),
                                      _ptr(gh, ctypes.c_double) if want_ghat else None)
    else:
        ev = np.ascontiguousarray(np.broadcast_to(np.asarray(eps, np.float32), (N,)))
        lv = np.ascontiguousarray(np.broadcast_to(np.asarray(lr, np.float32), (N,)))
        rc = _load().oracle_spsa_step_rates(ctypes.byref(cfg), _ptr(t, ctypes.c_float),
                                            _ptr(sd, ctypes.c_uint64), int(step), _ptr(ev, ctypes.c_float),
                                            _ptr(lv, ctypes.c_float), _ptr(b, ctypes.c_uint8),
                                            _ptr(losses, ctypes.c_float), _ptr(coef, ctypes.c_double),
                                            _ptr(out, ctypes.c_float),
                                            _ptr(gh, ctypes.c_double) if want_ghat else None)
    if rc != 0:
        raise ValueError("oracle_spsa_step rejected the configuration")
    return {"losses": losses, "coef": coef, "theta": out, "ghat": gh}


def eval_loss(cfg: OracleCfg, theta: np.ndarray, bytes_all: np.ndarray) -> np.ndarray:
    N = cfg.n_experts
    d = param_count(cfg)
    t = np.ascontiguousarray(theta, dtype=np.float32).reshape(N, d)
    b = np.ascontiguousarray(bytes_all, dtype=np.uint8).reshape(N, cfg.batch, cfg.seq_len)
    out = np.empty(N, dtype=np.float64)
    _load().oracle_eval_loss(ctypes.byref(cfg), _ptr(t, ctypes.c_float), _ptr(b, ctypes.c_uint8),
                             _ptr(out, ctypes.c_double))
    return out
