"""Thin Python binding of ``libsoma.so`` (include/soma.h): argument marshalling only.

Every step of the SPSA hot path runs in the HIP library.  torch supplies
device memory and the stream; nothing here computes.  If the library is not
built (``python -m paper_2609_37899_amd.build``), every call raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libsoma.so")

SOMA_OK, SOMA_EINVAL, SOMA_ESHAPE, SOMA_EDEVICE, SOMA_EWORKSPACE = 0, -1, -2, -3, -4
LOSS_INDEPENDENT, LOSS_SUMMED = 0, 1
PROBE_GAUSSIAN, PROBE_SPARSE_RADEMACHER, PROBE_RADEMACHER = 0, 1, 2
FLAG_PER_STEP_RECURRENCE = 1
FLAG_TILED_WEIGHTS = 2
FLAG_STAGED_RECURRENCE = 4
FLAG_FP32_SEQUENCE = 8
ARCH_LSTM, ARCH_BODY, ARCH_WIDE = 0, 1, 2
PERTURB_EMBEDDING, PERTURB_LSTM, PERTURB_HEAD, PERTURB_ALL = 1, 2, 4, 7

EXPORTS = ("soma_param_count", "soma_workspace_size", "soma_create", "soma_destroy",
           "soma_spsa_step", "soma_spsa_step_adam", "soma_eval_loss", "soma_coefficients",
           "soma_apply_update", "soma_apply_adam", "soma_spsa_step_adam_sched", "soma_schedule_init",
           "soma_schedule_observe", "soma_estimator_moments", "soma_set_tied_head", "soma_head_delta",
           "soma_gaussian", "soma_probe", "soma_philox", "soma_box_muller", "soma_set_phase_timing",
           "soma_get_phase_times", "soma_set_spin_limit", "soma_spsa_step_noalloc",
           "soma_last_error")


class SomaError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"soma error {code}: {msg}")
        self.code = code


class PhaseTimes(ctypes.Structure):
    _fields_ = [("fold_ms", ctypes.c_float), ("proj_ms", ctypes.c_float),
                ("rec_ms", ctypes.c_float), ("head_ms", ctypes.c_float),
                ("reduce_ms", ctypes.c_float), ("update_ms", ctypes.c_float),
                ("rec_launches", ctypes.c_int32), ("proj_launches", ctypes.c_int32),
                ("xchg_launches", ctypes.c_int32)]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


class Adam(ctypes.Structure):
    """soma_adam; the defaults are the paper's (Appendix E)."""
    _fields_ = [("beta1", ctypes.c_float), ("beta2", ctypes.c_float), ("delta", ctypes.c_float),
                ("weight_decay", ctypes.c_float)]

    def __init__(self, beta1=0.9, beta2=0.999, delta=1e-8, weight_decay=1e-4):
        super().__init__(beta1, beta2, delta, weight_decay)


class Plateau(ctypes.Structure):
    """soma_plateau; the defaults are the paper's schedule."""
    _fields_ = [("factor", ctypes.c_float), ("patience", ctypes.c_int32), ("threshold", ctypes.c_float),
                ("floor", ctypes.c_float)]

    def __init__(self, factor=0.5, patience=1000, threshold=1e-8, floor=1e-5):
        super().__init__(factor, patience, threshold, floor)


SCHEDULE_ENTRY_BYTES = 16   # soma_schedule_entry: lr, eps, best (fp32), since (int32)


class Config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_experts", "n_layers", "embed", "hidden", "batch", "seq_len", "n_pairs", "loss_mode",
        "pair_chunk", "flags", "probe", "accum", "arch")] + [("perturb_mask", ctypes.c_uint32)]


_lib = None


def load():
    """Load libsoma.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_37899_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        vp, cp = ctypes.c_void_p, ctypes.POINTER(Config)
        u64, u32, f32, i64p = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_float, ctypes.POINTER(ctypes.c_int64)
        sig = {
            "soma_param_count": (ctypes.c_int, [cp, i64p]),
            "soma_workspace_size": (ctypes.c_int, [cp, ctypes.POINTER(ctypes.c_size_t)]),
            "soma_create": (ctypes.c_int, [cp, vp, ctypes.c_size_t, ctypes.POINTER(vp)]),
            "soma_destroy": (None, [vp]),
            "soma_spsa_step": (ctypes.c_int, [vp, vp, vp, u64, f32, f32, vp, vp, vp]),
            "soma_spsa_step_noalloc": (ctypes.c_int, [cp, vp, vp, u64, f32, f32, vp, vp, vp]),
            "soma_spsa_step_adam": (ctypes.c_int, [vp, vp, vp, vp, ctypes.c_int64, ctypes.POINTER(Adam),
                                                   vp, u64, f32, f32, vp, vp, vp]),
            "soma_apply_adam": (ctypes.c_int, [vp, vp, vp, vp, ctypes.c_int64, ctypes.POINTER(Adam), vp,
                                               u64, f32, vp, vp]),
            "soma_spsa_step_adam_sched": (ctypes.c_int, [vp, vp, vp, vp, ctypes.c_int64, ctypes.POINTER(Adam),
                                                         vp, u64, vp, vp, vp, vp]),
            "soma_schedule_init": (ctypes.c_int, [vp, ctypes.c_int32, f32, f32, vp]),
            "soma_estimator_moments": (ctypes.c_int, [vp, vp, u64, vp, ctypes.c_int32, vp, vp]),
            "soma_schedule_observe": (ctypes.c_int, [vp, ctypes.c_int32, vp, ctypes.c_int32,
                                                     ctypes.POINTER(Plateau), vp]),
            "soma_eval_loss": (ctypes.c_int, [vp, vp, vp, vp, vp]),
            "soma_set_tied_head": (ctypes.c_int, [vp, vp, ctypes.c_int64]),
            "soma_head_delta": (ctypes.c_int, [vp, vp, vp, f32, vp, vp, vp]),
            "soma_coefficients": (ctypes.c_int, [vp, vp, vp]),
            "soma_apply_update": (ctypes.c_int, [vp, vp, vp, u64, f32, vp, vp]),
            "soma_gaussian": (ctypes.c_int, [u64, u64, u32, u64, u64, vp, vp]),
            "soma_probe": (ctypes.c_int, [ctypes.c_int, u64, u64, u32, u64, u64, vp, vp]),
            "soma_philox": (ctypes.c_int, [vp, vp, vp, u64, vp]),
            "soma_box_muller": (ctypes.c_int, [vp, vp, vp, vp, u64, vp]),
            "soma_set_phase_timing": (ctypes.c_int, [vp, ctypes.c_int]),
            "soma_set_spin_limit": (ctypes.c_int, [vp, ctypes.c_uint32]),
            "soma_get_phase_times": (ctypes.c_int, [vp, ctypes.POINTER(PhaseTimes)]),
            "soma_last_error": (ctypes.c_char_p, []),
        }
        for name, (res, args) in sig.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def _check(rc: int):
    if rc != SOMA_OK:
        raise SomaError(rc, load().soma_last_error().decode())


def _stream(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dptr(t, dtype=None, name="tensor"):
    import torch
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{name} must be a device tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


@dataclass
class Shape:
    n_experts: int
    n_layers: int
    embed: int
    hidden: int
    batch: int
    seq_len: int
    n_pairs: int
    loss_mode: int = LOSS_INDEPENDENT
    pair_chunk: int = 0
    flags: int = 0
    probe: int = PROBE_GAUSSIAN
    accum: int = 1
    arch: int = ARCH_LSTM
    perturb_mask: int = 0        # PERTURB_* bits of the perturbed groups; 0 = all

    def cfg(self) -> Config:
        return Config(self.n_experts, self.n_layers, self.embed, self.hidden, self.batch,
                      self.seq_len, self.n_pairs, self.loss_mode, self.pair_chunk, self.flags,
                      self.probe, self.accum, self.arch, self.perturb_mask)

    @property
    def directions(self) -> int:
        """Directions per update, n_pairs per accumulation batch."""
        return self.n_pairs * max(1, self.accum)


def param_count(shape: Shape) -> int:
    out = ctypes.c_int64()
    _check(load().soma_param_count(ctypes.byref(shape.cfg()), ctypes.byref(out)))
    return out.value


def workspace_size(shape: Shape) -> int:
    out = ctypes.c_size_t()
    _check(load().soma_workspace_size(ctypes.byref(shape.cfg()), ctypes.byref(out)))
    return out.value


class Context:
    """A shape bound to a device workspace (a torch uint8 tensor)."""

    def __init__(self, shape: Shape, device="cuda"):
        import torch
        self.shape = shape
        self._cfg = shape.cfg()
        nbytes = workspace_size(shape)
        self.workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        h = ctypes.c_void_p()
        _check(load().soma_create(ctypes.byref(self._cfg), ctypes.c_void_p(self.workspace.data_ptr()),
                                  nbytes, ctypes.byref(h)))
        self._h = h
        self.d = param_count(shape)

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            load().soma_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def spsa_step(self, theta, seeds, step: int, eps: float, lr: float, bytes_, losses,
                  stream=None):
        import torch
        _check(load().soma_spsa_step(self._h, _dptr(theta, torch.float32, "theta"),
                                     _dptr(seeds, torch.int64, "seeds"), int(step), float(eps),
                                     float(lr), _dptr(bytes_, torch.uint8, "bytes"),
                                     _dptr(losses, torch.float32, "losses"), _stream(stream)))

    def spsa_step_adam(self, theta, m, v, t: int, adam, seeds, step: int, eps: float, lr: float, bytes_,
                       losses, stream=None):
        import torch
        _check(load().soma_spsa_step_adam(self._h, _dptr(theta, torch.float32, "theta"),
                                          _dptr(m, torch.float32, "m"), _dptr(v, torch.float32, "v"),
                                          int(t), ctypes.byref(adam), _dptr(seeds, torch.int64, "seeds"),
                                          int(step), float(eps), float(lr),
                                          _dptr(bytes_, torch.uint8, "bytes"),
                                          _dptr(losses, torch.float32, "losses"), _stream(stream)))

    def spsa_step_adam_sched(self, theta, m, v, t: int, adam, seeds, step: int, sched, bytes_, losses,
                             stream=None):
        import torch
        _check(load().soma_spsa_step_adam_sched(self._h, _dptr(theta, torch.float32, "theta"),
                                                _dptr(m, torch.float32, "m"), _dptr(v, torch.float32, "v"),
                                                int(t), ctypes.byref(adam), _dptr(seeds, torch.int64, "seeds"),
                                                int(step), _dptr(sched, None, "schedule"),
                                                _dptr(bytes_, torch.uint8, "bytes"),
                                                _dptr(losses, torch.float32, "losses"), _stream(stream)))

    def estimator_moments(self, seeds, step: int, coef, group: int, out, stream=None):
        import torch
        _check(load().soma_estimator_moments(self._h, _dptr(seeds, torch.int64, "seeds"), int(step),
                                             _dptr(coef, torch.float32, "coef"), int(group),
                                             _dptr(out, torch.float64, "out"), _stream(stream)))

    def apply_adam(self, theta, m, v, t: int, adam, seeds, step: int, lr: float, coef, stream=None):
        import torch
        _check(load().soma_apply_adam(self._h, _dptr(theta, torch.float32, "theta"),
                                      _dptr(m, torch.float32, "m"), _dptr(v, torch.float32, "v"), int(t),
                                      ctypes.byref(adam), _dptr(seeds, torch.int64, "seeds"), int(step),
                                      float(lr), _dptr(coef, torch.float32, "coef"), _stream(stream)))

    def set_phase_timing(self, enable: bool = True):
        _check(load().soma_set_phase_timing(self._h, 1 if enable else 0))

    def set_spin_limit(self, polls: int):
        """Polls per group barrier of the persistent recurrence (0: default)."""
        _check(load().soma_set_spin_limit(self._h, int(polls)))

    def phase_times(self) -> dict:
        out = PhaseTimes()
        _check(load().soma_get_phase_times(self._h, ctypes.byref(out)))
        return out.as_dict()

    def eval_loss(self, theta, bytes_, loss, stream=None):
        import torch
        _check(load().soma_eval_loss(self._h, _dptr(theta, torch.float32, "theta"),
                                     _dptr(bytes_, torch.uint8, "bytes"),
                                     _dptr(loss, torch.float32, "loss"), _stream(stream)))

    def set_tied_head(self, E, per_expert: bool = False):
        """The tied matrix of a body context: E [V][w] shared by every expert,
        or [N][V][w] one per expert (per_expert=True); w = d, or d_E for the
        wide body.  The context reads the tensor's memory on every later
        call: keep it alive."""
        import torch
        stride = E.shape[-2] * E.shape[-1] if per_expert else 0
        _check(load().soma_set_tied_head(self._h, _dptr(E, torch.float32, "E"), stride))
        self._head = E

    def head_delta(self, theta, bytes_, lr: float = 0.0, grad=None, loss=None, stream=None):
        """The decoder-path delta rule: grad [N][V][d] and loss [N] (either may
        be None); with lr != 0 the tied matrix is also moved by -lr grad."""
        import torch
        g = _dptr(grad, torch.float32, "grad") if grad is not None else None
        lo = _dptr(loss, torch.float32, "loss") if loss is not None else None
        _check(load().soma_head_delta(self._h, _dptr(theta, torch.float32, "theta"),
                                      _dptr(bytes_, torch.uint8, "bytes"), float(lr), g, lo, _stream(stream)))

    def coefficients(self, coef, stream=None):
        import torch
        _check(load().soma_coefficients(self._h, _dptr(coef, torch.float32, "coef"), _stream(stream)))

    def apply_update(self, theta, seeds, step: int, lr: float, coef, stream=None):
        import torch
        _check(load().soma_apply_update(self._h, _dptr(theta, torch.float32, "theta"),
                                        _dptr(seeds, torch.int64, "seeds"), int(step), float(lr),
                                        _dptr(coef, torch.float32, "coef"), _stream(stream)))


def spsa_step_noalloc(shape: Shape, theta, seeds, step: int, eps: float, lr: float, bytes_, losses, stream=None):
    """soma_spsa_step without a context or workspace: the library's static
    per-device scratch (small shapes only; calls on one GPU must not overlap)."""
    import torch
    cfg = shape.cfg()
    _check(load().soma_spsa_step_noalloc(ctypes.byref(cfg), _dptr(theta, torch.float32, "theta"),
                                         _dptr(seeds, torch.int64, "seeds"), int(step), float(eps), float(lr),
                                         _dptr(bytes_, torch.uint8, "bytes"), _dptr(losses, torch.float32, "losses"),
                                         _stream(stream)))


def gaussian(seed: int, step: int, pair: int, k0: int, out, stream=None):
    import torch
    _check(load().soma_gaussian(int(seed) & (2**64 - 1), int(step), int(pair), int(k0), out.numel(),
                                _dptr(out, torch.float32, "out"), _stream(stream)))


def probe(law: int, seed: int, step: int, pair: int, k0: int, out, stream=None):
    import torch
    _check(load().soma_probe(int(law), int(seed) & (2**64 - 1), int(step), int(pair), int(k0), out.numel(),
                             _dptr(out, torch.float32, "out"), _stream(stream)))


def schedule_tensor(n: int, device="cuda"):
    """Device memory for n soma_schedule_entry records (int32 view, 4 words each)."""
    import torch
    return torch.empty((n, SCHEDULE_ENTRY_BYTES // 4), dtype=torch.int32, device=device)


def schedule_init(sched, lr0: float, eps0: float, stream=None):
    _check(load().soma_schedule_init(_dptr(sched, None, "schedule"), sched.shape[0], float(lr0), float(eps0),
                                     _stream(stream)))


def schedule_observe(sched, val_loss, updates: int, rule, stream=None):
    import torch
    _check(load().soma_schedule_observe(_dptr(sched, None, "schedule"), sched.shape[0],
                                        _dptr(val_loss, torch.float32, "val_loss"), int(updates),
                                        ctypes.byref(rule), _stream(stream)))


def schedule_fields(sched):
    """(lr, eps, best, since) numpy arrays of a schedule tensor (copies to the host)."""
    import numpy as np
    a = sched.cpu().numpy()
    f = a.view(np.float32)
    return f[:, 0].copy(), f[:, 1].copy(), f[:, 2].copy(), a[:, 3].copy()


def philox(ctr, key, out, stream=None):
    import torch
    n = ctr.shape[0]
    _check(load().soma_philox(_dptr(ctr, torch.int32, "ctr"), _dptr(key, torch.int32, "key"),
                              _dptr(out, torch.int32, "out"), n, _stream(stream)))


def box_muller(wa, wb, za, zb, stream=None):
    import torch
    _check(load().soma_box_muller(_dptr(wa, torch.int32, "wa"), _dptr(wb, torch.int32, "wb"),
                                  _dptr(za, torch.float32, "za"), _dptr(zb, torch.float32, "zb"),
                                  wa.numel(), _stream(stream)))


def group_covariance_trace(moments, directions: int, group: int):
    """tr Cov of the group means of `group` consecutive single-direction
    estimates, from soma_estimator_moments' two sums (per expert)."""
    import numpy as np
    m = np.asarray(moments, dtype=np.float64).reshape(-1, 2)
    G = directions // group
    return (m[:, 0] - m[:, 1] / G) / (group * group * (G - 1))


def seeds_tensor(seeds, device="cuda"):
    """uint64 seeds as the int64 device tensor the library reads bit for bit."""
    import numpy as np
    import torch
    a = np.ascontiguousarray(seeds, dtype=np.uint64).view(np.int64)
    return torch.from_numpy(a.copy()).to(device)
