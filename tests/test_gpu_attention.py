"""GPU: the decode attention (K4) and its split combine through the C ABI
(dex_debug_attention), on synthetic caches and row tables shaped like the
lattice's: rows of one sequence share a committed prefix [0, nc) and read
positions nc..pos from their own chain of slot entries.

Parity with a float64 softmax attention over the same cache values (bf16 or
fp32), for the matrix-core kernel (bf16, head_dim 64 and 128) and the VALU
kernels (fp32; bf16 head_dim 32):
  * chains of 1..9 positions, crossing a 64-key split boundary;
  * groups of more than 16 (row, query head) pairs, so the matrix-core
    kernel runs several pair tiles, and groups split at 64 pairs;
  * rows with no chain positions (nc = pos + 1, as in the prompt prefill);
  * long contexts (more than 128 splits);
and the properties the lossless decoding rests on: a row's output bits do
not depend on the other rows of the launch or on how they are grouped, and
repeated launches are bit-identical."""
import numpy as np
import pytest

from synth import gen
from tests.gpu_common import torch_cuda

pytestmark = pytest.mark.gpu

BF16_RTOL = 1e-2   # q, P and the output are rounded to bf16 (2^-9 each)
F32_RTOL = 1e-5


class Case:
    """Caches [B][Hkv][E][hd] and row tables.  `seqs` lists, per sequence,
    (nc, chain lengths of its rows); chain entries live past every committed
    region, at slot entries E0 + k."""

    def __init__(self, dtype, hd, H, Hkv, seqs, seed):
        self.dtype, self.hd, self.H, self.Hkv = dtype, hd, H, Hkv
        self.B = len(seqs)
        top = max(nc for nc, _ in seqs)
        self.E0 = top + 8
        n_slots = sum(sum(ch) for _, ch in seqs) + 16
        self.E = self.E0 + n_slots
        n = self.B * Hkv * self.E * hd
        bf = dtype == 1
        self.k = gen.uniform(gen.mix64(seed), n, 1.0, bf16=bf)
        self.v = gen.uniform(gen.mix64(seed + 1), n, 1.0, bf16=bf)
        rows_seq, rows_pos, rows_nc, coff, chain = [], [], [], [], []
        slot = self.E0
        for s, (nc, lens) in enumerate(seqs):
            for ln in lens:
                # ln chain positions nc .. nc + ln - 1 (0: all committed)
                rows_seq.append(s)
                rows_nc.append(nc)
                if ln == 0:
                    rows_pos.append(nc - 1)
                    coff.append(0)
                    continue
                rows_pos.append(nc + ln - 1)
                coff.append(len(chain))
                for _ in range(ln):
                    chain.append(slot)
                    slot += 1
        assert slot <= self.E
        self.seq = np.array(rows_seq, np.int32)
        self.pos = np.array(rows_pos, np.int32)
        self.nc = np.array(rows_nc, np.int32)
        self.coff = np.array(coff, np.int32)
        self.chain = np.array(chain if chain else [0], np.int32)
        self.R = len(rows_seq)
        self.q = gen.uniform(gen.mix64(seed + 2), self.R * H * hd, 1.0).reshape(self.R, H * hd)

    def values(self, bits):
        a = gen.bf16_bits_to_f32(bits) if self.dtype == 1 else bits
        return a.astype(np.float64).reshape(self.B, self.Hkv, self.E, self.hd)

    def reference(self, rows=None):
        """float64 attention of the listed rows: [len(rows)][H*hd]."""
        K, V = self.values(self.k), self.values(self.v)
        G = self.H // self.Hkv
        q = self.q.astype(np.float64)
        if self.dtype == 1 and self.hd in (64, 128):
            q = gen.bf16_bits_to_f32(gen.f32_to_bf16_bits(self.q)).astype(np.float64)
        out = []
        for r in (range(self.R) if rows is None else rows):
            s, pos, nc = self.seq[r], self.pos[r], self.nc[r]
            ent = np.arange(pos + 1)
            if nc <= pos:
                ent[nc:] = self.chain[self.coff[r]:self.coff[r] + pos + 1 - nc]
            o = np.empty(self.H * self.hd)
            for h in range(self.H):
                kk, vv = K[s, h // G, ent], V[s, h // G, ent]
                sc = kk @ q[r, h * self.hd:(h + 1) * self.hd] / np.sqrt(self.hd)
                p = np.exp(sc - sc.max())
                o[h * self.hd:(h + 1) * self.hd] = (p @ vv) / p.sum()
            out.append(o)
        return np.array(out)


def _run(torch, c, rows=None):
    """dex_debug_attention over the listed rows (default: all), returned as
    float64 [n][H*hd] plus the raw output bits."""
    import ctypes

    from paper_2606_29223_amd import dexlib
    lib = dexlib.load()
    rows = list(range(c.R)) if rows is None else list(rows)
    kdt = torch.int16 if c.dtype == 1 else torch.float32
    if not hasattr(c, "_dev"):
        kk = c.k.view(np.int16) if c.dtype == 1 else c.k
        vv = c.v.view(np.int16) if c.dtype == 1 else c.v
        c._dev = (torch.from_numpy(kk).cuda(), torch.from_numpy(vv).cuda())
    kd, vd = c._dev
    q = torch.from_numpy(np.ascontiguousarray(c.q[rows])).cuda()
    out = torch.zeros((len(rows), c.H * c.hd), dtype=kdt, device="cuda")
    P = ctypes.POINTER(ctypes.c_int32)

    def tab(a):
        a = np.ascontiguousarray(a, dtype=np.int32)
        return a, a.ctypes.data_as(P)

    seq, pseq = tab(c.seq[rows])
    pos, ppos = tab(c.pos[rows])
    nc, pnc = tab(c.nc[rows])
    coff, pcoff = tab(c.coff[rows])
    chain, pchain = tab(c.chain)
    st = lib.dex_debug_attention(c.dtype, c.hd, c.H, c.Hkv, c.B, c.E, kd.data_ptr(), vd.data_ptr(),
                                 q.data_ptr(), len(rows), pseq, ppos, pnc, pcoff, pchain, len(chain),
                                 out.data_ptr(), torch.cuda.current_stream().cuda_stream)
    assert st == dexlib.DEX_OK, st
    raw = out.cpu().numpy()
    if c.dtype == 1:
        vals = gen.bf16_bits_to_f32(raw.view(np.uint16)).astype(np.float64)
    else:
        vals = raw.astype(np.float64)
    return vals, raw


def _check(c, got, ref, rtol):
    for r in range(got.shape[0]):
        for h in range(c.H):
            sl = slice(h * c.hd, (h + 1) * c.hd)
            err = np.abs(got[r, sl] - ref[r, sl]).max() / np.abs(ref[r, sl]).max()
            assert err <= rtol, (r, h, err)


LATTICE = [(700, [1, 2, 3, 4, 5]), (190, [1, 3, 6, 9, 2]), (64, [1, 2]), (1000, [0, 1, 4])]
WIDE = [(513, [1] * 10 + [2] * 10), (130, [0, 0, 0, 1, 2, 3])]


@pytest.mark.parametrize("dtype,hd,H,Hkv", [(1, 128, 32, 8), (1, 64, 12, 12), (1, 64, 16, 2),
                                            (0, 32, 4, 4), (0, 128, 8, 2), (1, 32, 4, 4)])
@pytest.mark.parametrize("layout", ["lattice", "wide"])
def test_attention_matches_float64(dtype, hd, H, Hkv, layout):
    torch = torch_cuda()
    c = Case(dtype, hd, H, Hkv, LATTICE if layout == "lattice" else WIDE, seed=11 + hd + H)
    got, _ = _run(torch, c)
    _check(c, got, c.reference(), BF16_RTOL if dtype == 1 else F32_RTOL)


def test_attention_long_context():
    """More than 128 splits per row (the 8 x 8192 workload's shape), with
    one to three rows per sequence."""
    torch = torch_cuda()
    c = Case(1, 128, 32, 8, [(9001, [1]), (8300, [1, 2, 3]), (4097, [2, 5])], seed=5)
    got, _ = _run(torch, c)
    _check(c, got, c.reference(), BF16_RTOL)


@pytest.mark.parametrize("dtype,hd,H,Hkv", [(1, 128, 32, 8), (1, 64, 12, 12), (0, 32, 4, 4)])
def test_attention_rows_do_not_depend_on_the_launch(dtype, hd, H, Hkv):
    """A row's bits are the same alone, inside its full launch, in a launch
    with a different row subset (other groups and tile fills), and on a
    repeated launch."""
    torch = torch_cuda()
    c = Case(dtype, hd, H, Hkv, LATTICE + WIDE, seed=23)
    _, full = _run(torch, c)
    _, again = _run(torch, c)
    assert np.array_equal(full, again)
    rng = np.random.default_rng(3)
    for r in rng.choice(c.R, size=6, replace=False):
        _, alone = _run(torch, c, [int(r)])
        assert np.array_equal(alone[0], full[r]), r
    sub = sorted(int(x) for x in rng.choice(c.R, size=c.R // 2, replace=False))
    _, part = _run(torch, c, sub)
    for i, r in enumerate(sub):
        assert np.array_equal(part[i], full[r]), r


@pytest.mark.parametrize("dtype,hd,H,Hkv", [(1, 128, 32, 8), (1, 64, 12, 12), (0, 32, 4, 4)])
def test_short_rows_same_bits_beside_a_long_row(dtype, hd, H, Hkv):
    """Short rows (at most 64 splits) get the same bits alone and in a launch
    that also holds a 71-split row (more split items, the long row setting
    the launch's split count)."""
    torch = torch_cuda()
    c = Case(dtype, hd, H, Hkv, LATTICE + [(4500, [1, 2])], seed=29)
    short = [r for r in range(c.R) if c.pos[r] // 64 + 1 <= 64]
    assert len(short) < c.R
    _, mixed = _run(torch, c)
    _, alone = _run(torch, c, short)
    for i, r in enumerate(short):
        assert np.array_equal(alone[i], mixed[r]), r
    got, _ = _run(torch, c)
    _check(c, got, c.reference(), BF16_RTOL if dtype == 1 else F32_RTOL)
