"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function include/soma.h declares, and rejects bad arguments with the
documented codes before enqueuing anything."""
import ctypes
import os
import re

import pytest

from paper_2609_37899_amd import soma, workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "soma.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(soma_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(soma.LIB_PATH):
        from paper_2609_37899_amd import build
        build.build()
    return soma.load()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert set(names) == set(soma.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def shape_of(w, **kw):
    s = soma.Shape(w.n_experts, w.n_layers, w.embed, w.hidden, w.batch, w.seq_len, w.n_pairs,
                   w.loss_mode, probe=w.probe, arch=w.arch)
    for k, v in kw.items():
        setattr(s, k, v)
    return s


def test_param_counts_match_layout(lib):
    for w in workloads.ALL.values():
        assert soma.param_count(shape_of(w)) == w.params_per_expert


def test_workspace_size_and_auto_chunk(lib):
    s = shape_of(workloads.SOMA_N2)
    ws = soma.workspace_size(s)
    assert 0 < ws < 24 * 2**30
    s1 = shape_of(workloads.SOMA_N2, pair_chunk=1)
    assert soma.workspace_size(s1) < ws
    # The automatic chunk keeps the workspace within 64 GiB: the monolith's
    # 128 directions fit in one chunk, its 512 do not.
    mono = workloads.MONOLITH
    assert soma.workspace_size(shape_of(mono)) == soma.workspace_size(shape_of(mono, pair_chunk=mono.n_pairs))
    big = shape_of(mono.with_(n_pairs=512))
    assert soma.workspace_size(big) <= 64 * 2**30
    assert soma.workspace_size(big) < soma.workspace_size(shape_of(mono.with_(n_pairs=512), pair_chunk=512))


@pytest.mark.parametrize("field,value,code", [
    ("embed", 24, soma.SOMA_ESHAPE), ("hidden", 0, soma.SOMA_ESHAPE), ("seq_len", 1, soma.SOMA_ESHAPE),
    ("n_pairs", 0, soma.SOMA_ESHAPE), ("loss_mode", 2, soma.SOMA_EINVAL),
    ("pair_chunk", 99, soma.SOMA_ESHAPE), ("flags", 16, soma.SOMA_EINVAL), ("probe", 3, soma.SOMA_EINVAL),
    ("probe", -1, soma.SOMA_EINVAL), ("accum", -1, soma.SOMA_ESHAPE), ("perturb_mask", 8, soma.SOMA_EINVAL)])
def test_invalid_shapes_are_rejected(lib, field, value, code):
    s = shape_of(workloads.TINY)
    cfg = s.cfg()
    setattr(cfg, field, value)
    out = ctypes.c_size_t()
    assert lib.soma_workspace_size(ctypes.byref(cfg), ctypes.byref(out)) == code
    assert lib.soma_last_error()


def test_perturb_mask_is_checked(lib):
    """Any combination of the three groups is accepted for the stacked LSTM
    (0 meaning all); the body's parameters are one group, which a mask must
    include."""
    out = ctypes.c_size_t()
    for mask in range(8):
        cfg = shape_of(workloads.TINY, perturb_mask=mask).cfg()
        assert lib.soma_workspace_size(ctypes.byref(cfg), ctypes.byref(out)) == soma.SOMA_OK
    body = workloads.PAPER_BODY_N8
    for mask, code in ((0, soma.SOMA_OK), (soma.PERTURB_LSTM, soma.SOMA_OK), (soma.PERTURB_ALL, soma.SOMA_OK),
                       (soma.PERTURB_EMBEDDING | soma.PERTURB_HEAD, soma.SOMA_EINVAL)):
        cfg = shape_of(body, perturb_mask=mask).cfg()
        assert lib.soma_workspace_size(ctypes.byref(cfg), ctypes.byref(out)) == code


def test_create_checks_workspace(lib):
    cfg = shape_of(workloads.TINY).cfg()
    need = soma.workspace_size(shape_of(workloads.TINY))
    h = ctypes.c_void_p()
    assert lib.soma_create(ctypes.byref(cfg), None, need, ctypes.byref(h)) == soma.SOMA_EWORKSPACE
    assert lib.soma_create(ctypes.byref(cfg), ctypes.c_void_p(0x1000 + 8), need, ctypes.byref(h)) == soma.SOMA_EWORKSPACE
    assert lib.soma_create(ctypes.byref(cfg), ctypes.c_void_p(0x100000), need - 1, ctypes.byref(h)) == soma.SOMA_EWORKSPACE


def test_step_rejects_bad_scalars_before_enqueueing(lib):
    # A context over a fake (never dereferenced) workspace address: every call
    # below fails validation on the host, so no device work is issued.
    cfg = shape_of(workloads.TINY).cfg()
    need = soma.workspace_size(shape_of(workloads.TINY))
    h = ctypes.c_void_p()
    assert lib.soma_create(ctypes.byref(cfg), ctypes.c_void_p(0x100000), need, ctypes.byref(h)) == 0
    p = ctypes.c_void_p(0x200000)
    try:
        for eps in (0.0, -1e-3, float("nan"), float("inf")):
            assert lib.soma_spsa_step(h, p, p, 0, eps, 1e-2, p, p, None) == soma.SOMA_EINVAL
        assert lib.soma_spsa_step(h, p, p, 0, 1e-3, float("nan"), p, p, None) == soma.SOMA_EINVAL
        assert lib.soma_spsa_step(h, None, p, 0, 1e-3, 1e-2, p, p, None) == soma.SOMA_EINVAL
        assert lib.soma_spsa_step(h, ctypes.c_void_p(0x200004), p, 0, 1e-3, 1e-2, p, p, None) == soma.SOMA_EINVAL
        assert lib.soma_coefficients(h, p, None) == soma.SOMA_EINVAL   # no step ran yet
        assert lib.soma_gaussian(0, 0, 0, 2**40, 1, p, None) == soma.SOMA_EINVAL
        assert lib.soma_gaussian(0, 0, 0, 0, 1, None, None) == soma.SOMA_EINVAL
        assert lib.soma_probe(3, 0, 0, 0, 0, 1, p, None) == soma.SOMA_EINVAL
        assert lib.soma_probe(1, 0, 0, 0, 2**40, 1, p, None) == soma.SOMA_EINVAL
        good = soma.Adam()
        assert lib.soma_apply_adam(h, p, p, p, 0, ctypes.byref(good), p, 0, 1e-3, p, None) == soma.SOMA_EINVAL
        for bad in (soma.Adam(beta1=1.0), soma.Adam(beta2=-0.1), soma.Adam(delta=0.0),
                    soma.Adam(weight_decay=float("nan"))):
            assert lib.soma_apply_adam(h, p, p, p, 1, ctypes.byref(bad), p, 0, 1e-3, p, None) == soma.SOMA_EINVAL
            assert lib.soma_spsa_step_adam(h, p, p, p, 1, ctypes.byref(bad), p, 0, 1e-3, 1e-3, p, p,
                                           None) == soma.SOMA_EINVAL
        assert lib.soma_apply_adam(h, p, None, p, 1, ctypes.byref(good), p, 0, 1e-3, p, None) == soma.SOMA_EINVAL
        assert lib.soma_apply_adam(h, p, p, ctypes.c_void_p(0x200008), 1, ctypes.byref(good), p, 0, 1e-3, p,
                                   None) == soma.SOMA_EINVAL
        assert lib.soma_apply_adam(h, p, p, p, 1, None, p, 0, 1e-3, p, None) == soma.SOMA_EINVAL
    finally:
        lib.soma_destroy(h)


@pytest.mark.parametrize("field,value,code", [
    ("embed", 16, soma.SOMA_ESHAPE), ("hidden", 3, soma.SOMA_ESHAPE), ("hidden", 513, soma.SOMA_ESHAPE),
    ("batch", 65, soma.SOMA_ESHAPE), ("flags", 1, soma.SOMA_EINVAL),
    ("perturb_mask", soma.PERTURB_EMBEDDING | soma.PERTURB_HEAD, soma.SOMA_EINVAL)])
def test_wide_body_limits(lib, field, value, code):
    """The wide controls' body: head width 32, 4 <= d_t <= 512 at any width in
    between (odd widths included), batch <= 64, no execution flags, the body
    one group."""
    w = workloads.WIDE_N2
    out = ctypes.c_size_t()
    for dt in (4, 13, 181, 361, 509, 512):
        cfg = shape_of(w.with_(hidden=dt)).cfg()
        assert lib.soma_workspace_size(ctypes.byref(cfg), ctypes.byref(out)) == soma.SOMA_OK, dt
    cfg = shape_of(w).cfg()
    setattr(cfg, field, value)
    assert lib.soma_workspace_size(ctypes.byref(cfg), ctypes.byref(out)) == code
    assert lib.soma_last_error()


def test_wide_body_parameter_counts_and_chunks(lib):
    """16 D d_t^2 + (2D + 1) d_t + 2 d_E d_t per expert at the table's widths,
    and a workspace that the automatic chunking keeps within 64 GiB in equal
    chunks (the N = 2 control: two chunks of 16 directions)."""
    w = workloads.WIDE_N2
    for dt, body in ((509, 8_325_713), (361, 4_195_181), (181, 1_060_841)):
        assert soma.param_count(shape_of(w.with_(hidden=dt))) == body
    ws = soma.workspace_size(shape_of(w))
    assert ws <= 64 * 2**30
    assert ws == soma.workspace_size(shape_of(w, pair_chunk=16))
