"""ctypes binding of libdcl (``include/dcl.h``): same names, argument marshalling only.

Device buffers are torch tensors on ``cuda`` (ROCm); their ``data_ptr()`` and the current
stream's handle are passed through unchanged. Every step of the computation runs in the
library's HIP kernels.

Before a call, every tensor argument is checked against what the call will read or write
through it: on the device, contiguous, of the element type the C declaration states (int32
ids and positions, float32 statistics and residuals, 16-bit bfloat16 patterns), and holding at
least the elements the sizes imply. A failed check raises ``DclError`` (DCL_E_ARG) before the
library is called. Plain integers are taken as raw device addresses and passed unchecked.
"""
import ctypes
import os
from typing import Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
DCL_DTYPE_F32, DCL_DTYPE_BF16 = 0, 1
DCL_SCORE_ALL_UNCOMMITTED = 0x1
DCL_SCORE_SUPPRESS_MASK = 0x2
DCL_SEL_NO_PROGRESS_GUARD = 0x1
DCL_SEL_SCORE_ALL = 0x2
DCL_SEL_NONCONTIGUOUS = 0x4
DCL_SEL_CONTIGUOUS_DRAFTS = 0x8
DCL_SEL_MARGIN = 0x10
STATUS = {0: "DCL_OK", 1: "DCL_E_ARG", 2: "DCL_E_UNSUPPORTED", 3: "DCL_E_WORKSPACE", 4: "DCL_E_HIP",
          5: "DCL_E_STATE"}


class DclError(RuntimeError):
    def __init__(self, status, where, detail):
        super().__init__(f"{where}: {STATUS.get(status, status)}: {detail}")
        self.status = status


class DclConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("n_layers", "d_model", "n_heads", "n_kv_heads", "head_dim",
                                              "d_ffn", "vocab", "mask_id")] + \
               [("rms_eps", ctypes.c_float), ("rope_base", ctypes.c_float), ("qkv_bias", ctypes.c_int32),
                ("rope_enabled", ctypes.c_int32), ("max_positions", ctypes.c_int32)]


class DclRowStats(ctypes.Structure):
    _fields_ = [("top1", ctypes.c_void_p), ("top2", ctypes.c_void_p), ("conf", ctypes.c_void_p),
                ("p2", ctypes.c_void_p), ("lse", ctypes.c_void_p), ("entropy", ctypes.c_void_p)]


PROF_CLASSES = ("embed", "rmsnorm", "gemm_qkv_rope", "attention", "gemm_o_residual", "gemm_gate_up_swiglu",
                "gemm_down_residual", "compact_rows", "gemm_lm_head_top2", "merge_partials", "select")


class DclProfile(ctypes.Structure):
    _fields_ = [("launches", ctypes.c_int64 * len(PROF_CLASSES)), ("ms", ctypes.c_double * len(PROF_CLASSES))]


class DclLayerTaps(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("u", "q", "k", "v", "o", "r_mid", "u2", "a", "r_out")]


class DclKV(ctypes.Structure):
    _fields_ = [("k", ctypes.POINTER(ctypes.c_void_p)), ("v", ctypes.POINTER(ctypes.c_void_p)),
                ("prefix_len", ctypes.c_int32), ("capacity", ctypes.c_int32)]


def library_path() -> str:
    return os.path.join(HERE, "libdcl.so")


_lib = None


def load_library():
    """Load libdcl.so; raises if it has not been built (no fallback exists)."""
    global _lib
    if _lib is not None:
        return _lib
    path = library_path()
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -c 'import __graft_entry__ as g; g.build()'`")
    lib = ctypes.CDLL(path)
    vp, i32, u32, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32, ctypes.c_float, ctypes.c_size_t
    sig = {
        "dcl_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "dcl_last_error": (ctypes.c_char_p, []),
        "dcl_model_create": (ctypes.c_int, [ctypes.POINTER(DclConfig), ctypes.POINTER(vp)]),
        "dcl_model_destroy": (None, [vp]),
        "dcl_weights_bytes": (sz, [ctypes.POINTER(DclConfig)]),
        "dcl_load_weights": (ctypes.c_int, [vp, vp, sz, ctypes.POINTER(vp), i32, i32, vp]),
        "dcl_workspace_bytes": (sz, [vp, i32, i32, i32]),
        "dcl_denoise_step": (ctypes.c_int, [vp, vp, i32, i32, vp, i32, ctypes.POINTER(DclKV), u32, DclRowStats,
                                            vp, sz, vp]),
        "dcl_denoise_step_noalloc": (ctypes.c_int, [vp, vp, i32, i32, vp, i32, ctypes.POINTER(DclKV), u32,
                                                    DclRowStats, vp]),
        "dcl_select_contiguous": (ctypes.c_int, [vp, i32, i32, vp, i32, i32, i32, i32, f32, f32, i32, DclRowStats,
                                                 vp, vp, u32, vp]),
        "dcl_generate": (ctypes.c_int, [vp, vp, i32, i32, vp, i32, ctypes.POINTER(DclKV), u32, i32, i32, i32, f32, f32,
                                        u32, i32, i32, DclRowStats, vp, vp, vp, vp, sz, ctypes.POINTER(i32), vp]),
        "dcl_score_workspace_bytes": (sz, [vp, i32]),
        "dcl_kv_append": (ctypes.c_int, [vp, vp, i32, i32, ctypes.POINTER(DclKV), vp, sz, vp]),
        "dcl_profile_enable": (ctypes.c_int, [i32]),
        "dcl_profile_read": (ctypes.c_int, [ctypes.POINTER(DclProfile)]),
        "dcl_score_hidden": (ctypes.c_int, [vp, vp, i32, DclRowStats, vp, sz, vp]),
        "dcl_debug_logits": (ctypes.c_int, [vp, vp, i32, i32, ctypes.POINTER(DclKV), vp, i32, vp, vp, vp, sz, vp]),
        "dcl_debug_layer": (ctypes.c_int, [vp, i32, i32, ctypes.POINTER(DclKV), i32, vp, DclLayerTaps, vp, sz, vp]),
        "dcl_debug_gemm_plan": (ctypes.c_int, [i32, i32, i32, i32, i32, ctypes.POINTER(i32)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status, where):
    if status != 0:
        raise DclError(status, where, dcl_last_error())


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


_I32 = ("int32",)
_F32 = ("float32",)
_B16 = ("int16", "bfloat16", "uint16")       # bfloat16 bit patterns
_ANY = None


def _arg(x, name, where, kinds, numel=None, nbytes=None):
    """Device address of tensor argument ``x`` after checking it against the call: device memory,
    contiguous, element type among ``kinds`` (torch dtype names; None = any), at least ``numel``
    elements and ``nbytes`` bytes. None stays None; an int is a raw address and is not checked."""
    if x is None or isinstance(x, int):
        return x
    bad = None
    if not getattr(x, "is_cuda", False):
        bad = "must be a device (cuda) tensor"
    elif not x.is_contiguous():
        bad = "must be contiguous"
    elif kinds is not None and str(x.dtype).replace("torch.", "") not in kinds:
        bad = f"has dtype {x.dtype}, expected {' or '.join(kinds)}"
    elif numel is not None and x.numel() < numel:
        bad = f"holds {x.numel()} elements, the call needs {numel}"
    elif nbytes is not None and x.numel() * x.element_size() < nbytes:
        bad = f"holds {x.numel() * x.element_size()} bytes, the call needs {nbytes}"
    if bad:
        raise DclError(1, where, f"{name} {bad}")
    return x.data_ptr()


# Geometry of every handle this binding created (sizes for the argument checks).
_geometry = {}


def _cfg_of(model):
    return _geometry.get(model)


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


# ---------------------------------------------------------------- one function per C entry point

def dcl_status_string(status: int) -> str:
    return load_library().dcl_status_string(status).decode()


def dcl_last_error() -> str:
    return load_library().dcl_last_error().decode()


def dcl_model_create(cfg: DclConfig) -> int:
    h = ctypes.c_void_p()
    _check(load_library().dcl_model_create(ctypes.byref(cfg), ctypes.byref(h)), "dcl_model_create")
    _geometry[h.value] = DclConfig.from_buffer_copy(cfg)
    return h.value


def dcl_model_destroy(model: int) -> None:
    _geometry.pop(model, None)
    load_library().dcl_model_destroy(model)


def dcl_weights_bytes(cfg: DclConfig) -> int:
    return load_library().dcl_weights_bytes(ctypes.byref(cfg))


def dcl_load_weights(model: int, dev_buf, nbytes: int, src_ptrs: Sequence[Optional[int]], src_dtype: int,
                     stream=None) -> None:
    arr = (ctypes.c_void_p * len(src_ptrs))(*src_ptrs)
    buf = _arg(dev_buf, "dev_buf", "dcl_load_weights", _ANY, nbytes=nbytes)
    _check(load_library().dcl_load_weights(model, buf, nbytes, arr, len(src_ptrs), src_dtype,
                                           _stream(stream)), "dcl_load_weights")


def dcl_workspace_bytes(model: int, B: int, S: int, kv_prefix: int = 0) -> int:
    return load_library().dcl_workspace_bytes(model, B, S, kv_prefix)


def _stats(st, n=None, where="") -> DclRowStats:
    """st: dict of device arrays (each >= n elements); "entropy" is optional (not written when absent)."""
    kinds = {"top1": _I32, "top2": _I32, "conf": _F32, "p2": _F32, "lse": _F32, "entropy": _F32}
    return DclRowStats(*(_arg(st.get(k), f"stats[{k!r}]", where, kinds[k], n) for k in kinds))


def _kv(kv, model=None, B=None, where=""):
    """kv: None or (per-layer K tensors, per-layer V tensors, prefix_len[, capacity])."""
    if kv is None:
        return None, None
    ks, vs, P = kv[:3]
    cap = kv[3] if len(kv) > 3 else 0
    g = _cfg_of(model)
    need = None
    if g is not None and B is not None:
        if len(ks) != g.n_layers or len(vs) != g.n_layers:
            raise DclError(1, where, f"kv holds {len(ks)}/{len(vs)} layers, the model has {g.n_layers}")
        need = B * g.n_kv_heads * (cap or P) * g.head_dim
    ka = (ctypes.c_void_p * len(ks))(*[_arg(t, f"kv K[{i}]", where, _B16, need) for i, t in enumerate(ks)])
    va = (ctypes.c_void_p * len(vs))(*[_arg(t, f"kv V[{i}]", where, _B16, need) for i, t in enumerate(vs)])
    s = DclKV(ctypes.cast(ka, ctypes.POINTER(ctypes.c_void_p)), ctypes.cast(va, ctypes.POINTER(ctypes.c_void_p)), P,
              cap)
    return ctypes.byref(s), (s, ka, va)


def _state(tokens, p, B, S, where):
    n = B * S if B > 0 and S > 0 else None
    return (_arg(tokens, "tokens", where, _I32, n), _arg(p, "p", where, _I32, B if B > 0 else None))


def dcl_denoise_step(model: int, tokens, B: int, S: int, p, gen_end: int, kv, flags: int, stats, ws, ws_bytes: int,
                     stream=None) -> None:
    w = "dcl_denoise_step"
    kvp, keep = _kv(kv, model, B, w)
    tp, pp = _state(tokens, p, B, S, w)
    _check(load_library().dcl_denoise_step(model, tp, B, S, pp, gen_end, kvp, flags, _stats(stats, B * S, w),
                                           _arg(ws, "ws", w, _ANY, nbytes=ws_bytes), ws_bytes, _stream(stream)), w)
    del keep


DCL_NOALLOC_SCRATCH_BYTES = 96 << 20


def dcl_denoise_step_noalloc(model: int, tokens, B: int, S: int, p, gen_end: int, kv, flags: int, stats,
                             stream=None) -> None:
    w = "dcl_denoise_step_noalloc"
    kvp, keep = _kv(kv, model, B, w)
    tp, pp = _state(tokens, p, B, S, w)
    _check(load_library().dcl_denoise_step_noalloc(model, tp, B, S, pp, gen_end, kvp, flags,
                                                   _stats(stats, B * S, w), _stream(stream)), w)
    del keep


def dcl_select_contiguous(tokens, B: int, S: int, p, gen_end: int, L: int, tau_commit: float, tau_draft: float,
                          mask_id: int, stats, k_raw=None, k_eff=None, flags: int = 0, stream=None,
                          block_origin: int = 0, block_len: int = 0) -> None:
    """block_origin / block_len: semi-autoregressive blocks (block_len 0 = none), as in include/dcl.h."""
    w = "dcl_select_contiguous"
    tp, pp = _state(tokens, p, B, S, w)
    _check(load_library().dcl_select_contiguous(tp, B, S, pp, gen_end, L, block_origin, block_len, tau_commit,
                                                tau_draft, mask_id,
                                                _stats(stats, B * S, w), _arg(k_raw, "k_raw", w, _I32, B),
                                                _arg(k_eff, "k_eff", w, _I32, B), flags, _stream(stream)), w)


def dcl_generate(model: int, tokens, B: int, S: int, p, gen_end: int, kv, score_flags: int, L: int,
                 tau_commit: float, tau_draft: float, select_flags: int, max_steps: int, check_every: int, stats,
                 k_raw, k_eff, k_hist, ws, ws_bytes: int, stream=None, block_origin: int = 0,
                 block_len: int = 0) -> int:
    """Returns the number of iterations run. block_origin / block_len: semi-autoregressive blocks."""
    w = "dcl_generate"
    kvp, keep = _kv(kv, model, B, w)
    tp, pp = _state(tokens, p, B, S, w)
    steps = ctypes.c_int32(0)
    _check(load_library().dcl_generate(model, tp, B, S, pp, gen_end, kvp, score_flags, L, block_origin, block_len,
                                       tau_commit,
                                       tau_draft, select_flags, max_steps, check_every, _stats(stats, B * S, w),
                                       _arg(k_raw, "k_raw", w, _I32, B), _arg(k_eff, "k_eff", w, _I32, B),
                                       _arg(k_hist, "k_hist", w, _I32, L + 1 if L >= 0 else None),
                                       _arg(ws, "ws", w, _ANY, nbytes=ws_bytes), ws_bytes, ctypes.byref(steps),
                                       _stream(stream)), w)
    del keep
    return steps.value


def dcl_kv_append(model: int, tokens, B: int, S: int, kv, ws, ws_bytes: int, stream=None) -> None:
    w = "dcl_kv_append"
    kvp, keep = _kv(kv, model, B, w)
    _check(load_library().dcl_kv_append(model, _arg(tokens, "tokens", w, _I32, B * S), B, S, kvp,
                                        _arg(ws, "ws", w, _ANY, nbytes=ws_bytes), ws_bytes, _stream(stream)), w)
    del keep


def dcl_profile_enable(on: bool) -> None:
    _check(load_library().dcl_profile_enable(1 if on else 0), "dcl_profile_enable")


def dcl_profile_read() -> dict:
    """{class name: (launches, total ms)} since the last enable."""
    pr = DclProfile()
    _check(load_library().dcl_profile_read(ctypes.byref(pr)), "dcl_profile_read")
    return {n: (int(pr.launches[i]), float(pr.ms[i])) for i, n in enumerate(PROF_CLASSES)}


def dcl_score_workspace_bytes(model: int, n: int) -> int:
    return load_library().dcl_score_workspace_bytes(model, n)


def dcl_score_hidden(model: int, hidden, n: int, stats, ws, ws_bytes: int, stream=None) -> None:
    w = "dcl_score_hidden"
    g = _cfg_of(model)
    _check(load_library().dcl_score_hidden(model, _arg(hidden, "hidden", w, _B16, n * g.d_model if g else None), n,
                                           _stats(stats, n, w), _arg(ws, "ws", w, _ANY, nbytes=ws_bytes), ws_bytes,
                                           _stream(stream)), w)


def dcl_debug_logits(model: int, tokens, B: int, S: int, kv, rows, n_rows: int, out, hidden_out, ws, ws_bytes: int,
                     stream=None) -> None:
    w = "dcl_debug_logits"
    g = _cfg_of(model)
    kvp, keep = _kv(kv, model, B, w)
    _check(load_library().dcl_debug_logits(
        model, _arg(tokens, "tokens", w, _I32, B * S), B, S, kvp, _arg(rows, "rows", w, _I32, n_rows), n_rows,
        _arg(out, "out", w, _F32, n_rows * g.vocab if g else None),
        _arg(hidden_out, "hidden_out", w, _B16, n_rows * g.d_model if g else None),
        _arg(ws, "ws", w, _ANY, nbytes=ws_bytes), ws_bytes, _stream(stream)), w)
    del keep


def dcl_debug_layer(model: int, B: int, S: int, kv, layer: int, r_in, taps: dict, ws, ws_bytes: int,
                    stream=None) -> None:
    """taps: dict name -> device tensor (names of DclLayerTaps; absent = not copied out)."""
    w = "dcl_debug_layer"
    g = _cfg_of(model)
    koff = (kv[2] % 8) if kv is not None else 0      # carried cached keys in front of the fresh ones
    T, Sp = B * S, (koff + S + 7) // 8 * 8
    size = {}
    if g is not None:
        hd, kd = g.n_heads * g.head_dim, g.n_kv_heads * g.head_dim
        size = {"u": (_B16, T * g.d_model), "q": (_B16, T * hd), "k": (_B16, B * (koff + S) * kd),
                "v": (_B16, B * kd * Sp),
                "o": (_B16, T * hd), "r_mid": (_F32, T * g.d_model), "u2": (_B16, T * g.d_model),
                "a": (_B16, T * g.d_ffn), "r_out": (_F32, T * g.d_model)}
    unknown = set(taps) - {f for f, _ in DclLayerTaps._fields_}
    if unknown:
        raise DclError(1, w, f"unknown taps {sorted(unknown)}")
    ct = DclLayerTaps(*(_arg(taps.get(f), f"taps[{f!r}]", w, *size.get(f, (_ANY, None)))
                        for f, _ in DclLayerTaps._fields_))
    kvp, keep = _kv(kv, model, B, w)
    _check(load_library().dcl_debug_layer(model, B, S, kvp, layer,
                                          _arg(r_in, "r_in", w, _F32, T * g.d_model if g else None), ct,
                                          _arg(ws, "ws", w, _ANY, nbytes=ws_bytes), ws_bytes, _stream(stream)), w)
    del keep


def dcl_debug_gemm_plan(Nw: int, T: int, K: int, lm_head: bool = False, max_split: int = 4) -> dict:
    """The tile plan of a GEMM shape (host only): configuration, K-split slices and tile geometry."""
    info = (ctypes.c_int32 * 8)()
    _check(load_library().dcl_debug_gemm_plan(Nw, T, K, 1 if lm_head else 0, max_split, info), "dcl_debug_gemm_plan")
    keys = ("cfg", "nsplit", "bw", "bt", "kd", "stages", "ww", "wt")
    return dict(zip(keys, list(info)))


# ---------------------------------------------------------------- convenience owner of device buffers

def config_from_geometry(g, max_positions: int = 4096, rope_enabled: bool = True) -> DclConfig:
    """DclConfig from any object with the geometry fields (e.g. ``synth.Geometry``)."""
    return DclConfig(g.n_layers, g.d_model, g.n_heads, g.n_kv_heads, g.head_dim, g.d_ffn, g.vocab, g.mask_id,
                     g.rms_eps, g.rope_base, int(g.qkv_bias), int(rope_enabled), max_positions)


class Runner:
    """Owns a model handle plus torch-allocated weight buffer, workspace and statistics buffers."""

    def __init__(self, geom, tensors, max_positions: int = 4096, rope_enabled: bool = True, stream=None):
        """tensors: sequence of numpy arrays / torch tensors (or None for absent biases) in the load order of
        ``include/dcl.h``; float32 or bfloat16 bit patterns (uint16 / int16 / torch.bfloat16)."""
        import numpy as np
        import torch
        self.torch = torch
        self.geom = geom
        self.cfg = config_from_geometry(geom, max_positions, rope_enabled)
        self.model = dcl_model_create(self.cfg)
        nbytes = dcl_weights_bytes(self.cfg)
        self.wbuf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        dtype = None
        keep, ptrs = [], []
        for t in tensors:
            if t is None:
                ptrs.append(None)
                continue
            if isinstance(t, np.ndarray):
                t = torch.from_numpy(np.ascontiguousarray(t))
            t = t.contiguous()
            dt = DCL_DTYPE_F32 if t.dtype == torch.float32 else DCL_DTYPE_BF16
            if dtype is None:
                dtype = dt
            elif dt != dtype and t.dim() > 1:
                raise ValueError("all weight matrices must share one dtype")
            if dt != dtype:  # vectors follow the matrices' dtype
                t = t.float() if dtype == DCL_DTYPE_F32 else t.view(torch.int16)
            keep.append(t)
            ptrs.append(t.data_ptr())
        dcl_load_weights(self.model, self.wbuf, nbytes, ptrs, dtype, stream)
        del keep
        self.ws = None
        self.ws_key = None

    def workspace(self, B, S, P=0):
        need = dcl_workspace_bytes(self.model, B, S, P)
        if self.ws is None or self.ws.numel() < need:
            self.ws = self.torch.empty(need, dtype=self.torch.uint8, device="cuda")
        return self.ws, need

    def new_stats(self, B, S):
        t = self.torch
        return {"top1": t.empty((B, S), dtype=t.int32, device="cuda"),
                "top2": t.empty((B, S), dtype=t.int32, device="cuda"),
                "conf": t.empty((B, S), dtype=t.float32, device="cuda"),
                "p2": t.empty((B, S), dtype=t.float32, device="cuda"),
                "lse": t.empty((B, S), dtype=t.float32, device="cuda"),
                "entropy": t.empty((B, S), dtype=t.float32, device="cuda")}

    def step(self, tokens, p, gen_end, stats=None, kv=None, flags=0, stream=None):
        B, S = tokens.shape
        ws, n = self.workspace(B, S, 0 if kv is None else kv[2])
        if stats is None:
            stats = self.new_stats(B, S)
        dcl_denoise_step(self.model, tokens, B, S, p, gen_end, kv, flags, stats, ws, n, stream)
        return stats

    def logits(self, tokens, rows, kv=None, stream=None, with_hidden=False):
        """float32 logits [n_rows, V] (and, with_hidden, bf16-bit hidden states [n_rows, d] as int16)."""
        B, S = tokens.shape
        ws, n = self.workspace(B, S, 0 if kv is None else kv[2])
        out = self.torch.empty((rows.numel(), self.geom.vocab), dtype=self.torch.float32, device="cuda")
        hid = self.torch.empty((rows.numel(), self.geom.d_model), dtype=self.torch.int16, device="cuda") \
            if with_hidden else None
        dcl_debug_logits(self.model, tokens, B, S, kv, rows, rows.numel(), out, hid, ws, n, stream)
        return (out, hid) if with_hidden else out

    def kv_append(self, tokens, kv, stream=None):
        """Write the keys/values of tokens [B, S] at positions kv[2] + i into the cache kv (see dcl_kv_append)."""
        B, S = tokens.shape
        ws, n = self.workspace(B, S, kv[2])
        dcl_kv_append(self.model, tokens, B, S, kv, ws, n, stream)

    def score_hidden(self, hidden, stream=None):
        """Statistics of given bf16 hidden rows (int16 bit patterns or torch.bfloat16, [n, d])."""
        n = hidden.shape[0]
        need = dcl_score_workspace_bytes(self.model, n)
        ws = self.torch.empty(need, dtype=self.torch.uint8, device="cuda")
        st = self.new_stats(1, n)
        dcl_score_hidden(self.model, hidden, n, st, ws, need, stream)
        return {k: v.view(n) for k, v in st.items()}

    def close(self):
        if self.model:
            dcl_model_destroy(self.model)
            self.model = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
