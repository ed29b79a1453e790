"""GPU: dex_debug_attention_noalloc (row tables and split partials in the
library's fixed scratch array, no device allocation) gives the same output
bits as dex_debug_attention (which allocates them) on two calls in a row,
the second with fewer rows and a shorter context, so nothing the first call
left in the shared scratch leaks into the second."""
import ctypes

import numpy as np
import pytest

from tests.gpu_common import torch_cuda
from tests.test_gpu_attention import Case

pytestmark = pytest.mark.gpu


def _call(torch, c, noalloc):
    from paper_2606_29223_amd import dexlib
    lib = dexlib.load()
    kdt = torch.int16 if c.dtype == 1 else torch.float32
    kk = c.k.view(np.int16) if c.dtype == 1 else c.k
    vv = c.v.view(np.int16) if c.dtype == 1 else c.v
    kd, vd = torch.from_numpy(kk).cuda(), torch.from_numpy(vv).cuda()
    q = torch.from_numpy(np.ascontiguousarray(c.q)).cuda()
    out = torch.full((c.R, c.H * c.hd), -1, dtype=kdt, device="cuda")
    P = ctypes.POINTER(ctypes.c_int32)
    keep = []

    def tab(a):
        a = np.ascontiguousarray(a, dtype=np.int32)
        keep.append(a)
        return a.ctypes.data_as(P)

    fn = lib.dex_debug_attention_noalloc if noalloc else lib.dex_debug_attention
    torch.cuda.synchronize()
    st = fn(c.dtype, c.hd, c.H, c.Hkv, c.B, c.E, kd.data_ptr(), vd.data_ptr(), q.data_ptr(), c.R, tab(c.seq),
            tab(c.pos), tab(c.nc), tab(c.coff), tab(c.chain), len(c.chain), out.data_ptr(),
            torch.cuda.current_stream().cuda_stream)
    assert st == dexlib.DEX_OK, (st, lib.dex_last_error(None))
    return out.cpu().numpy()


@pytest.mark.parametrize("dtype,hd,H,Hkv", [(1, 128, 32, 8), (1, 64, 12, 12), (0, 32, 4, 4)])
def test_noalloc_attention_equals_allocating_entry(dtype, hd, H, Hkv):
    torch = torch_cuda()
    big = Case(dtype, hd, H, Hkv, [(4100, [1, 2, 3]), (700, [1, 2, 3, 4, 5]), (190, [0, 1, 9])], seed=41)
    small = Case(dtype, hd, H, Hkv, [(300, [2]), (64, [1])], seed=42)
    for c in (big, small):                       # second call: fewer rows, shorter context
        got = _call(torch, c, noalloc=True)
        ref = _call(torch, c, noalloc=False)
        assert np.array_equal(got, ref)
        assert not np.array_equal(got, np.full_like(got, -1))
