"""Host-only checks of the transformer C ABI (include/erase_tf.h): the library
exports every declared entry point, counts parameters like the input
generator, and rejects bad configurations and arguments before any HIP call
(no GPU needed)."""
import ctypes
import os
import re

import pytest

from paper_2608_18469_amd import erase, erase_tf, synth_tf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    with open(os.path.join(ROOT, "include", "erase_tf.h")) as f:
        text = re.sub(r"/\*.*?\*/", "", f.read(), flags=re.S)
    return sorted(set(re.findall(r"\b(erase_tf_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_tf_symbol():
    L = erase_tf.lib()
    names = _declared()
    assert len(names) >= 12
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(erase_tf.SIGNATURES), set(names) ^ set(erase_tf.SIGNATURES)


@pytest.mark.parametrize("name", ["tf_tiny", "tf_small", "tf_c5"])
def test_param_count_matches_generator(name):
    cfg = synth_tf.tf_config(name)
    for b in range(cfg["layers"]):
        assert erase_tf.param_count(cfg, b) == synth_tf.param_count(cfg, b)


def test_pack_unpack_roundtrip():
    import numpy as np
    cfg = synth_tf.tf_config("tf_tiny")
    params, _ = synth_tf.make_workload(cfg)
    for b in range(cfg["layers"]):
        flat = synth_tf.pack_block(cfg, b, params[b])
        back = synth_tf.unpack_block(cfg, b, flat)
        for k in params[b]:
            assert np.array_equal(back[k], params[b][k])


def test_workspace_grows_with_batch():
    a = erase_tf.workspace_bytes(synth_tf.tf_config("tf_small"))
    b = erase_tf.workspace_bytes(synth_tf.tf_config("tf_small", batch=4))
    assert 0 < a < b


@pytest.mark.parametrize("mut,code", [
    (dict(d=96, heads=1), erase.ERR_SHAPE),            # d != 64 * heads
    (dict(d=128, heads=1), erase.ERR_SHAPE),
    (dict(vocab=100), erase.ERR_SHAPE),                # not a multiple of 64
    (dict(layers=0), erase.ERR_SHAPE),
    (dict(layers=65), erase.ERR_SHAPE),
    (dict(seq=0), erase.ERR_SHAPE),
    (dict(batch=1 << 14, seq=1 << 11), erase.ERR_SHAPE),   # B*T > 2^24
    (dict(d=64 * 65, heads=65), erase.ERR_SHAPE),      # d > 4096
    (dict(adam=dict(lr=-1.0, beta1=0.9, beta2=0.999, eps=1e-8)), erase.ERR_INVALID_ARG),
    (dict(adam=dict(lr=1e-3, beta1=1.0, beta2=0.999, eps=1e-8)), erase.ERR_INVALID_ARG),
    (dict(lam=float("nan")), erase.ERR_INVALID_ARG),
])
def test_validation_errors(mut, code):
    cfg = synth_tf.tf_config("tf_small", **mut)
    n = ctypes.c_size_t(0)
    nc = erase_tf.native_config(cfg)
    assert erase_tf.lib().erase_tf_workspace_bytes(ctypes.byref(nc), ctypes.byref(n)) == code


def test_init_rejects_bad_arguments_before_any_hip_call():
    L = erase_tf.lib()
    cfg = synth_tf.tf_config("tf_tiny")
    nc = erase_tf.native_config(cfg)
    need = erase_tf.workspace_bytes(cfg)
    bufs = (erase.BlockBuffers * cfg["layers"])()
    for b in range(cfg["layers"]):
        bufs[b] = erase.BlockBuffers(0x1000, 0x2000, 0x3000, None)
    ctx = ctypes.c_void_p()
    s1, s2 = ctypes.c_void_p(0x10), ctypes.c_void_p(0x20)
    ws = ctypes.c_void_p(0x100000)
    init = L.erase_tf_init
    assert init(ctypes.byref(nc), None, ws, need, s1, s2, ctypes.byref(ctx)) == erase.ERR_INVALID_ARG
    assert init(ctypes.byref(nc), bufs, ws, need, None, s2, ctypes.byref(ctx)) == erase.ERR_INVALID_ARG
    assert init(ctypes.byref(nc), bufs, ws, need, s1, s1, ctypes.byref(ctx)) == erase.ERR_INVALID_ARG
    assert init(ctypes.byref(nc), bufs, ctypes.c_void_p(0x100010), need, s1, s2, ctypes.byref(ctx)) == \
        erase.ERR_WORKSPACE
    assert init(ctypes.byref(nc), bufs, ws, need - 1, s1, s2, ctypes.byref(ctx)) == erase.ERR_WORKSPACE
    bad = (erase.BlockBuffers * cfg["layers"])()
    for b in range(cfg["layers"]):
        bad[b] = erase.BlockBuffers(0x1002, 0x2000, 0x3000, None)
    assert init(ctypes.byref(nc), bad, ws, need, s1, s2, ctypes.byref(ctx)) == erase.ERR_INVALID_ARG
    assert ctx.value is None
    assert L.erase_tf_destroy(None) == erase.OK
    assert L.erase_tf_step(None, None, 0, None) == erase.ERR_INVALID_ARG
    assert L.erase_tf_sync(None) == erase.ERR_INVALID_ARG


def test_flop_count_of_c5():
    f = synth_tf.flops_per_step(synth_tf.tf_config("tf_c5"))
    # heads: 3 GEMMs of 2 * 16384 * 512 * 32768 per layer, 8 layers
    assert f["total"] > 8 * 3 * 2 * 16384 * 512 * 32768
    assert f["total"] < 2.0e13
