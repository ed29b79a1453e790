"""The C-ABI library loads on a machine without a GPU, exports every symbol
include/dex.h declares, and rejects bad arguments before touching a device."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2606_29223_amd import dexlib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "dex.h")).read()
    return sorted(set(re.findall(r"\b(dex_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(dexlib.LIB_PATH):
        pytest.skip("libdex.so not built")
    return dexlib.load()


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(names) == sorted(dexlib.EXPORTED)


def _model(**kw):
    m = dexlib.DexModel()
    m.n_layers, m.d_model, m.n_heads, m.n_kv_heads, m.head_dim, m.d_ffn, m.vocab = 4, 128, 4, 4, 32, 344, 512
    m.rope_theta, m.rms_eps, m.residual_scale, m.weight_dtype = 1e4, 1e-5, 0.3, dexlib.DEX_F32
    fake = ctypes.c_void_p(0x1000)
    m.embed = m.final_norm = m.lm_head = 0x1000
    arr = (ctypes.c_void_p * (4 * 9))(*([0x1000] * 36))
    m.layers = ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p))
    for k, v in kw.items():
        setattr(m, k, v)
    return m, arr, fake


def _config(X, W=0, B=1, ctxlen=64):
    c = dexlib.DexConfig()
    x = np.array(X, dtype=np.int32)
    c.explored = x.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    c.n_explored, c.width_cap, c.decs, c.batch, c.max_context, c.hip_stream = len(X), W, 1, B, ctxlen, None
    return c, x


@pytest.mark.parametrize("X,W,B,msg", [
    ([1, 2, 3], 0, 1, "last explored depth"),
    ([2, 1, 4], 0, 1, "strictly increasing"),
    ([0, 4], 0, 1, "strictly increasing"),
    ([1, 2, 3, 4], 0, 64, "DEX_MAX_ROWS"),
    ([4], -1, 1, "width_cap"),
])
def test_create_rejects_bad_explored_sets(lib, X, W, B, msg):
    m, _a, _f = _model()
    c, _x = _config(X, W, B)
    ctx = ctypes.c_void_p()
    st = lib.dex_create(ctypes.byref(m), ctypes.byref(c), ctypes.byref(ctx))
    assert st == dexlib.DEX_E_INVAL
    assert msg in lib.dex_last_error(None).decode()
    assert not ctx.value


def test_create_rejects_bad_dims(lib):
    for kw in (dict(d_model=100), dict(head_dim=24), dict(n_kv_heads=3), dict(weight_dtype=7),
               dict(head_dim=16), dict(head_dim=48), dict(head_dim=80), dict(head_dim=96), dict(head_dim=112)):
        m, _a, _f = _model(**kw)
        c, _x = _config([4])
        ctx = ctypes.c_void_p()
        assert lib.dex_create(ctypes.byref(m), ctypes.byref(c), ctypes.byref(ctx)) == dexlib.DEX_E_INVAL


@pytest.mark.parametrize("tau", [-0.5, float("nan"), float("inf")])
def test_create_rejects_bad_temperature(lib, tau):
    m, _a, _f = _model()
    c, _x = _config([4])
    c.temperature = tau
    ctx = ctypes.c_void_p()
    assert lib.dex_create(ctypes.byref(m), ctypes.byref(c), ctypes.byref(ctx)) == dexlib.DEX_E_INVAL
    assert "temperature" in lib.dex_last_error(None).decode()


def test_null_and_state_errors(lib):
    assert lib.dex_step(None, None, None) == dexlib.DEX_E_INVAL
    assert lib.dex_prefill(None, None, 0, None) == dexlib.DEX_E_INVAL
    lib.dex_destroy(None)
    assert lib.dex_debug_copy(None, None, 16, None) == dexlib.DEX_E_INVAL
    assert lib.dex_debug_gemm(1, None, 16, 16, None, 1, None, None) == dexlib.DEX_E_INVAL
    assert lib.dex_debug_gumbel(1, 0, 0, 16, None, None) == dexlib.DEX_E_INVAL


def test_debug_attention_rejects_bad_tables(lib):
    """Every malformed table is refused on the host, before any device call
    (the base arguments below are valid and are never passed unchanged)."""
    fake = 0x1000

    def call(dtype=1, hd=128, H=32, Hkv=8, B=1, E=100, seq=(0,), pos=(10,), nc=(10,), coff=(0,), chain=(50,),
             q=fake):
        arr = lambda v: (ctypes.c_int32 * len(v))(*v)
        return lib.dex_debug_attention(dtype, hd, H, Hkv, B, E, fake, fake, q, len(seq), arr(seq), arr(pos),
                                       arr(nc), arr(coff), arr(chain), len(chain), fake, None)

    bad = [dict(seq=(1,)), dict(nc=(12,)), dict(pos=(90,)), dict(chain=(100,)), dict(chain=(-1,)),
           dict(coff=(1,)), dict(hd=48), dict(H=72), dict(H=30), dict(pos=(100,), nc=(100,)), dict(q=None),
           dict(dtype=2), dict(B=0), dict(nc=(-1,))]
    for kw in bad:
        assert call(**kw) == dexlib.DEX_E_INVAL, kw



def test_attention_noalloc_rejects_before_any_device_call(lib):
    """The no-allocation attention refuses bad tables (DEX_E_INVAL) and sizes
    beyond its fixed scratch (DEX_E_CAPACITY) on the host."""
    fake = 0x1000
    arr = lambda v: (ctypes.c_int32 * len(v))(*v)

    def call(n_rows=1, pos=10, nc=10, chain=(50,), E=100, H=32, Hkv=8, hd=128):
        seq = [0] * n_rows
        return lib.dex_debug_attention_noalloc(1, hd, H, Hkv, 1, E, fake, fake, fake, n_rows, arr(seq),
                                               arr([pos] * n_rows), arr([nc] * n_rows), arr([0] * n_rows),
                                               arr(chain), len(chain), fake, None)

    assert call(nc=12) == dexlib.DEX_E_INVAL
    assert call(hd=48) == dexlib.DEX_E_INVAL
    assert call(n_rows=257, E=300) == dexlib.DEX_E_CAPACITY
    assert "256 rows" in lib.dex_last_error(None).decode()
    assert call(chain=tuple([50] * 16385), E=20000) == dexlib.DEX_E_CAPACITY
    # 8 rows x 32 heads x 516 splits x 130 floats x 4 B = 68.7 MB of partials (> 63.75 MiB)
    assert call(n_rows=8, pos=33000, nc=33000, chain=(33010,), E=33100) == dexlib.DEX_E_CAPACITY
    assert "scratch" in lib.dex_last_error(None).decode()
