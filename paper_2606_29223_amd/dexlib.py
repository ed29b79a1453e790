"""ctypes binding of libdex.so (include/dex.h), same names as the C ABI.

Argument marshalling only: every step of the decode path runs in the HIP
library.  PyTorch provides device memory and the stream.  If the library is
not built this module raises on first use -- there is no fallback.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdex.so")

DEX_OK, DEX_E_INVAL, DEX_E_NOMEM, DEX_E_HIP, DEX_E_STATE, DEX_E_CAPACITY = 0, -1, -2, -3, -4, -5
DEX_F32, DEX_BF16 = 0, 1
DEX_MAX_BATCH, DEX_MAX_EXPLORED, DEX_MAX_ROWS = 64, 32, 256
LAYER_PARAMS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")
ADAPTER_PARTS = ("norm", "w1", "b1", "w2", "b2", "alpha")

EXPORTED = (
    "dex_create", "dex_prefill", "dex_step", "dex_destroy", "dex_last_error",
    "dex_debug_set_logits_tap", "dex_debug_lattice", "dex_debug_last_collapse",
    "dex_debug_kv_layout", "dex_debug_slot_entry", "dex_debug_set_kernel_timing",
    "dex_debug_kernel_times", "dex_debug_time_kernel", "dex_debug_gemm", "dex_debug_attention",
    "dex_debug_gumbel", "dex_debug_copy", "dex_debug_plan", "dex_debug_attention_noalloc",
    "dex_debug_set_round_timing", "dex_debug_round_times",
)


class DexModel(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("d_ffn", ctypes.c_int32),
        ("vocab", ctypes.c_int32),
        ("rope_theta", ctypes.c_float), ("rms_eps", ctypes.c_float), ("residual_scale", ctypes.c_float),
        ("weight_dtype", ctypes.c_int32),
        ("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p), ("lm_head", ctypes.c_void_p),
        ("layers", ctypes.POINTER(ctypes.c_void_p)),
    ]


class DexConfig(ctypes.Structure):
    _fields_ = [
        ("explored", ctypes.POINTER(ctypes.c_int32)), ("n_explored", ctypes.c_int32),
        ("width_cap", ctypes.c_int32), ("decs", ctypes.c_int32), ("batch", ctypes.c_int32),
        ("max_context", ctypes.c_int32), ("hip_stream", ctypes.c_void_p),
        ("stage_streams", ctypes.c_int32), ("temperature", ctypes.c_float),
        ("sample_seed", ctypes.c_uint64), ("adapter_dim", ctypes.c_int32),
        ("adapters", ctypes.POINTER(ctypes.c_void_p)), ("stage_grouping", ctypes.c_int32),
    ]


class DexStepInfo(ctypes.Structure):
    _fields_ = [
        ("n_rows", ctypes.c_int32),
        ("rows_per_stage", ctypes.c_int32 * DEX_MAX_EXPLORED),
        ("layers_streamed", ctypes.c_int32),
        ("row_layers", ctypes.c_int32),
        ("q", ctypes.c_int32 * DEX_MAX_BATCH),
        ("kstar", ctypes.c_int32 * DEX_MAX_BATCH),
        ("row_seq", ctypes.c_int32 * DEX_MAX_ROWS),
        ("row_slot", ctypes.c_int32 * DEX_MAX_ROWS),
        ("row_stage", ctypes.c_int32 * DEX_MAX_ROWS),
        ("row_pos", ctypes.c_int32 * DEX_MAX_ROWS),
        ("row_token", ctypes.c_int32 * DEX_MAX_ROWS),
        ("rounds_total", ctypes.c_int64),
        ("attn_bytes", ctypes.c_double),
    ]


_lib = None


def load(path: str | None = None):
    """Load libdex.so (raises if it is missing: there is no other path)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"libdex.so not built ({p}); run __graft_entry__.build()")
    lib = ctypes.CDLL(p)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    P = ctypes.POINTER
    lib.dex_create.argtypes = [P(DexModel), P(DexConfig), P(vp)]
    lib.dex_prefill.argtypes = [vp, P(i32), i32, P(i32)]
    lib.dex_step.argtypes = [vp, P(i32), P(DexStepInfo)]
    lib.dex_destroy.argtypes = [vp]
    lib.dex_destroy.restype = None
    lib.dex_last_error.argtypes = [vp]
    lib.dex_last_error.restype = ctypes.c_char_p
    lib.dex_debug_set_logits_tap.argtypes = [vp, vp, i32]
    lib.dex_debug_lattice.argtypes = [vp, i32, P(i32), i32, P(i32)]
    lib.dex_debug_last_collapse.argtypes = [vp, i32, P(i32), i32, P(i32), P(i32), P(i32)]
    lib.dex_debug_kv_layout.argtypes = [vp, P(vp), P(vp), P(i64)]
    lib.dex_debug_slot_entry.argtypes = [vp, i32, i32, P(i32)]
    lib.dex_debug_set_kernel_timing.argtypes = [vp, i32]
    lib.dex_debug_kernel_times.argtypes = [vp, i32, P(ctypes.c_double), P(i64), P(ctypes.c_double)]
    lib.dex_debug_time_kernel.argtypes = [vp, i32, i32, i32, P(ctypes.c_double), P(ctypes.c_double)]
    lib.dex_debug_gemm.argtypes = [i32, vp, i32, i32, vp, i32, vp, vp]
    lib.dex_debug_copy.argtypes = [vp, vp, i64, vp]
    lib.dex_debug_attention.argtypes = [i32, i32, i32, i32, i32, i32, vp, vp, vp, i32, P(i32), P(i32), P(i32),
                                        P(i32), P(i32), i32, vp, vp]
    lib.dex_debug_attention_noalloc.argtypes = list(lib.dex_debug_attention.argtypes)
    lib.dex_debug_gumbel.argtypes = [ctypes.c_uint64, i32, i32, i32, vp, vp]
    lib.dex_debug_set_round_timing.argtypes = [vp, i32]
    lib.dex_debug_round_times.argtypes = [vp, i32, P(ctypes.c_double), P(i64)]
    lib.dex_debug_plan.argtypes = [i32, i32, i32, i32, P(i32), i32, P(i32), i32, P(i32)]
    for name in EXPORTED:
        if name not in ("dex_destroy", "dex_last_error"):
            getattr(lib, name).restype = ctypes.c_int32
    if path is None:
        _lib = lib
    return lib


class DexError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"dex status {status}: {msg}")
        self.status = status


def _check(lib, ctx, st):
    if st != DEX_OK:
        m = lib.dex_last_error(ctx)
        raise DexError(st, m.decode() if m else "")


def _i32p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


# --------------------------------------------------------------- C-ABI names

def dex_create(model: DexModel, config: DexConfig) -> ctypes.c_void_p:
    lib = load()
    ctx = ctypes.c_void_p()
    _check(lib, None, lib.dex_create(ctypes.byref(model), ctypes.byref(config), ctypes.byref(ctx)))
    return ctx


def dex_prefill(ctx, prompts: np.ndarray) -> np.ndarray:
    lib = load()
    prompts = np.ascontiguousarray(prompts, dtype=np.int32)
    first = np.empty(prompts.shape[0], dtype=np.int32)
    _check(lib, ctx, lib.dex_prefill(ctx, _i32p(prompts), prompts.shape[1], _i32p(first)))
    return first


def dex_step(ctx, batch: int, info: DexStepInfo | None = None) -> np.ndarray:
    lib = load()
    out = np.empty(batch, dtype=np.int32)
    _check(lib, ctx, lib.dex_step(ctx, _i32p(out), ctypes.byref(info) if info is not None else None))
    return out


def dex_destroy(ctx) -> None:
    load().dex_destroy(ctx)


def dex_debug_plan(n_explored: int, width_cap: int, decs: int, max_context: int, slots) -> list:
    """Planner tap (host only): slots = [(parent, fork_stage, c, pos, u), ...]
    in canonical order; returns [(kind, slot, f)] in priority order."""
    lib = load()
    n = len(slots)
    rec = np.full((n, 4 + n_explored), -1, dtype=np.int32)
    for i, (par, f, c, pos, u) in enumerate(slots):
        rec[i, :4] = (par, f, c, pos)
        rec[i, 4:4 + len(u)] = u
    cap = 4 * n * n_explored + 1
    out = np.empty((cap, 3), dtype=np.int32)
    cnt = ctypes.c_int32()
    _check(lib, None, lib.dex_debug_plan(n_explored, width_cap, decs, max_context, _i32p(rec), n, _i32p(out), cap,
                                         ctypes.byref(cnt)))
    return [tuple(int(v) for v in out[j]) for j in range(cnt.value)]


# ---------------------------------------------------------------- convenience

def device_weights(cfg: dict, weights: dict, device="cuda"):
    """Copy generated weights to device tensors (PyTorch allocates; nothing is
    computed here).  bf16 arrays arrive as uint16 bit patterns."""
    import torch
    out = {}
    for name, arr in weights.items():
        if arr.dtype == np.uint16:
            t = torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(device)
        else:
            t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(device)
        out[name] = t
    return out


class Decoder:
    """One library context over device-resident weights."""

    def __init__(self, cfg: dict, dev_weights: dict, explored=None, width_cap=None, decs=None,
                 batch=None, max_context=None, stream=None, stage_streams=0, temperature=0.0, seed=0,
                 adapters=None, stage_grouping=0):
        import torch
        self.lib = load()
        self.cfg = cfg
        self.w = dev_weights                    # keeps the tensors alive
        L = cfg["n_layers"]
        self.explored = list(cfg["explored"] if explored is None else explored)
        self.batch = int(cfg["batch"] if batch is None else batch)
        self.N = len(self.explored)
        m = DexModel()
        m.n_layers, m.d_model, m.n_heads = L, cfg["d_model"], cfg["n_heads"]
        m.n_kv_heads, m.head_dim, m.d_ffn, m.vocab = (cfg["n_kv_heads"], cfg["head_dim"], cfg["d_ffn"],
                                                      cfg["vocab"])
        m.rope_theta, m.rms_eps, m.residual_scale = cfg["rope_theta"], cfg["rms_eps"], cfg["residual_scale"]
        m.weight_dtype = DEX_BF16 if cfg["dtype"] == "bf16" else DEX_F32
        m.embed = dev_weights["embed"].data_ptr()
        m.final_norm = dev_weights["final_norm"].data_ptr()
        m.lm_head = dev_weights["lm_head"].data_ptr()
        self._layers = (ctypes.c_void_p * (L * 9))(*[
            dev_weights[f"layers.{l}.{p}"].data_ptr() for l in range(L) for p in LAYER_PARAMS])
        m.layers = ctypes.cast(self._layers, ctypes.POINTER(ctypes.c_void_p))
        self._x = np.array(self.explored, dtype=np.int32)
        c = DexConfig()
        c.explored = _i32p(self._x)
        c.n_explored = self.N
        c.width_cap = int(cfg["width_cap"] if width_cap is None else width_cap)
        c.decs = int(cfg.get("decs", 1) if decs is None else decs)
        c.batch = self.batch
        c.max_context = int(max_context if max_context is not None else cfg["prompt_len"] + cfg["gen_len"])
        # a dedicated stream (default priority, non-blocking): launches on the
        # legacy null stream would also order against every other stream
        self.stream = stream if stream is not None else torch.cuda.Stream()
        c.hip_stream = self.stream.cuda_stream
        c.stage_streams = int(stage_streams)
        c.stage_grouping = int(stage_grouping)
        c.temperature = float(temperature)
        c.sample_seed = int(seed) & ((1 << 64) - 1)
        # inducing adapters: device tensors "adapters.{k}.{part}" for the
        # non-final explored depths k (see ADAPTER_PARTS)
        self.adapters = adapters
        if adapters is not None:
            n_ad = self.N - 1
            ptrs = [adapters[f"adapters.{k}.{p}"].data_ptr() for k in range(n_ad) for p in ADAPTER_PARTS]
            self._adp = (ctypes.c_void_p * max(len(ptrs), 1))(*ptrs)
            c.adapters = ctypes.cast(self._adp, ctypes.POINTER(ctypes.c_void_p))
            c.adapter_dim = int(adapters["adapters.0.w1"].shape[0]) if n_ad > 0 else 0
        torch.cuda.synchronize()                # weights uploaded on other streams are complete
        self.model_struct, self.config_struct = m, c
        self.max_context = c.max_context
        self.ctx = dex_create(m, c)
        self.info = DexStepInfo()

    def prefill(self, prompts) -> np.ndarray:
        return dex_prefill(self.ctx, np.asarray(prompts, dtype=np.int32).reshape(self.batch, -1))

    def step(self) -> np.ndarray:
        return dex_step(self.ctx, self.batch, self.info)

    def generate(self, prompts, n_tokens: int):
        """Prefill, then dex_step until every sequence holds n_tokens
        generated tokens (y_0 counts) or max_context stops it.  Returns
        (tokens: list per sequence, stats: rounds, rows and layers streamed,
        matched depth k* per commit)."""
        first = self.prefill(prompts)
        toks = [[int(first[b])] for b in range(self.batch)]
        stats = {"rounds": 0, "rows": 0, "layers_streamed": 0, "row_layers": 0, "kstar": []}
        while min(len(t) for t in toks) < n_tokens:
            try:
                c = self.step()
            except DexError as e:
                if e.status == DEX_E_CAPACITY:
                    break
                raise
            inf = self.info
            stats["rounds"] += 1
            stats["rows"] += inf.n_rows
            stats["layers_streamed"] += inf.layers_streamed
            stats["row_layers"] += inf.row_layers
            for b in range(self.batch):
                if c[b] >= 0 and len(toks[b]) < n_tokens:
                    toks[b].append(int(c[b]))
                    stats["kstar"].append(int(inf.kstar[b]))
        return toks, stats

    def set_logits_tap(self, tensor):
        st = self.lib.dex_debug_set_logits_tap(self.ctx, tensor.data_ptr() if tensor is not None else None,
                                                tensor.shape[0] if tensor is not None else 0)
        _check(self.lib, self.ctx, st)

    def lattice(self, seq: int = 0):
        cap = 4096
        buf = np.empty(cap * (5 + self.N), dtype=np.int32)
        n = ctypes.c_int32()
        _check(self.lib, self.ctx, self.lib.dex_debug_lattice(self.ctx, seq, _i32p(buf), cap, ctypes.byref(n)))
        return buf[: n.value * (5 + self.N)].reshape(n.value, 5 + self.N)

    def last_collapse(self, seq: int = 0):
        buf = np.empty(4096, dtype=np.int32)
        n, fresh, cpos = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        _check(self.lib, self.ctx, self.lib.dex_debug_last_collapse(
            self.ctx, seq, _i32p(buf), 4096, ctypes.byref(n), ctypes.byref(fresh), ctypes.byref(cpos)))
        return list(buf[: n.value]), fresh.value, cpos.value

    def kv_layout(self):
        k, v, e = ctypes.c_void_p(), ctypes.c_void_p(), ctypes.c_int64()
        _check(self.lib, self.ctx, self.lib.dex_debug_kv_layout(self.ctx, ctypes.byref(k), ctypes.byref(v),
                                                                ctypes.byref(e)))
        return k.value, v.value, e.value

    def slot_entry(self, seq: int, slot: int) -> int:
        e = ctypes.c_int32()
        _check(self.lib, self.ctx, self.lib.dex_debug_slot_entry(self.ctx, seq, slot, ctypes.byref(e)))
        return e.value

    def set_timing(self, on: bool):
        _check(self.lib, self.ctx, self.lib.dex_debug_set_kernel_timing(self.ctx, int(on)))

    def kernel_times(self):
        ms = (ctypes.c_double * 8)()
        n = (ctypes.c_int64 * 8)()
        b = (ctypes.c_double * 8)()
        _check(self.lib, self.ctx, self.lib.dex_debug_kernel_times(self.ctx, 8, ms, n, b))
        return list(ms), list(n), list(b)

    def set_round_timing(self, on: bool):
        _check(self.lib, self.ctx, self.lib.dex_debug_set_round_timing(self.ctx, int(on)))

    def round_times(self):
        """(per-phase milliseconds summed over the timed rounds, rounds); see
        ROUND_PHASES."""
        ms = (ctypes.c_double * 7)()
        n = ctypes.c_int64()
        _check(self.lib, self.ctx, self.lib.dex_debug_round_times(self.ctx, 7, ms, ctypes.byref(n)))
        return list(ms), n.value

    def time_kernel(self, cls: int, M: int, reps: int = 64):
        """(mean microseconds, algorithmic bytes) of one decode GEMM launch."""
        us, b = ctypes.c_double(), ctypes.c_double()
        _check(self.lib, self.ctx, self.lib.dex_debug_time_kernel(self.ctx, cls, M, reps, ctypes.byref(us),
                                                                  ctypes.byref(b)))
        return us.value, b.value

    def close(self):
        if self.ctx:
            dex_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


ROUND_PHASES = ("upload", "sweep", "exit", "copy", "commit_collapse", "gap_before_round", "host_plan")
KERNEL_CLASSES = ("qkv", "attention", "attn_combine", "o_proj", "gate_up", "down", "lm_head", "other")
