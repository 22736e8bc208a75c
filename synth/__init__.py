"""Seeded synthetic inputs shared by the oracle and the HIP path.

This module only *produces inputs*: model geometries, random-init weights,
prompts, decode states (token ids, pointer p) and the prefix KV cache. It holds
none of the decoding method's arithmetic, imports neither ``oracle`` nor the
HIP package, and both sides consume exactly the arrays it returns.

Workloads (stand-ins for the paper's LLaDA / Dream runs on GSM8K, MATH, MBPP,
HumanEval, IFEval, none of which is reproduced): random-init weights with the
geometry of the paper's base models (Section 4 setup), uniform random prompt
ids, generation lengths 64 / 256 / 512 / 1024 as in the paper's runs, decode
windows of one 32-token block.

Random numbers:
* matrices, biases and the KV cache: Philox4x32-10 + Box-Muller
  (``philox_normal.c``), key = config seed, stream = tensor index, scaled by
  the init std and rounded to bfloat16 (round-to-nearest-even); the tiny
  config keeps float32 weights (the HIP library rounds them at load);
* prompt and draft ids: numpy ``default_rng([seed, 10000 + b])`` /
  ``default_rng([seed, 20000 + b])``, uniform in [0, vocab - 2).
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
from typing import Dict, Iterator, List, Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "philox_normal.c")
_LIB = os.path.join(_HERE, "_philox_normal.so")


def build(force: bool = False) -> str:
    """Compile the generator (gcc, no GPU needed). Returns the .so path."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-pthread", "-ffp-contract=off",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        for name, ptr in (("synth_normal_f32", ctypes.c_void_p), ("synth_normal_bf16", ctypes.c_void_p)):
            fn = getattr(lib, name)
            fn.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_double, ptr, ctypes.c_int64, ctypes.c_int]
            fn.restype = None
        _lib = lib
    return _lib


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def normal_f32(seed: int, stream: int, scale: float, shape) -> np.ndarray:
    """N(0, scale^2) float32 array from the Philox stream (seed, stream)."""
    out = np.empty(shape, dtype=np.float32)
    _load().synth_normal_f32(seed, stream, scale, out.ctypes.data, out.size, _threads())
    return out


def normal_bf16(seed: int, stream: int, scale: float, shape) -> np.ndarray:
    """N(0, scale^2) rounded to bfloat16; returned as the uint16 bit patterns."""
    out = np.empty(shape, dtype=np.uint16)
    _load().synth_normal_bf16(seed, stream, scale, out.ctypes.data, out.size, _threads())
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns to float32 (exact)."""
    return (bits.astype(np.uint32) << 16).view(np.float32)


# ----------------------------------------------------------------------------------------------
# Geometries and workloads
# ----------------------------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Geometry:
    """Bidirectional LLaMA-style mask predictor (RMSNorm, RoPE, SwiGLU)."""
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    mask_id: int
    rms_eps: float
    rope_base: float
    qkv_bias: bool
    weight_dtype: str          # "f32" (tiny config) or "bf16"
    init_std: float
    lm_scale: float            # LM-head multiplier that spreads the top-1 confidences
    seed: int


@dataclasses.dataclass(frozen=True)
class Workload:
    """One denoising-iteration input: geometry, batch, the decode state, selection params."""
    key: str
    geom: Geometry
    batch: int
    prompt_len: int            # N
    gen_len: int               # M (total of the generation region visible in `tokens`)
    window: int                # L, maximum decoding-window size
    p: int                     # first uncommitted position (index into tokens)
    draft: Tuple[int, int]     # half-open region holding draft placeholders ((0,0) = none)
    tau_commit: float
    tau_draft: float
    kv_prefix: int = 0         # cached prefix length (0 = full forward)
    kv_seed: int = 0
    description: str = ""

    @property
    def seq(self) -> int:       # S, tokens per sequence passed to one step
        return self.prompt_len + self.gen_len if self.kv_prefix == 0 else self.gen_len

    @property
    def gen_end(self) -> int:   # end of the generation region, index into tokens
        return self.seq


TINY = Geometry("tiny-2L-d256", n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64,
                d_ffn=688, vocab=4096, mask_id=4095, rms_eps=1e-5, rope_base=1e4, qkv_bias=False,
                weight_dtype="f32", init_std=0.02, lm_scale=40.0, seed=0)
# LLaDA-8B geometry. RoPE base 5e5 and eps 1e-5 are the public LLaDA-8B values (not stated in the paper).
LLADA8B = Geometry("llada-8b", n_layers=32, d_model=4096, n_heads=32, n_kv_heads=32, head_dim=128,
                   d_ffn=12288, vocab=126464, mask_id=126463, rms_eps=1e-5, rope_base=5e5,
                   qkv_bias=False, weight_dtype="bf16", init_std=0.02, lm_scale=12.0, seed=1)
# Dream-7B (Qwen2.5-7B geometry): GQA 28/4, q/k/v biases, RoPE base 1e6, eps 1e-6.
DREAM7B = Geometry("dream-7b", n_layers=28, d_model=3584, n_heads=28, n_kv_heads=4, head_dim=128,
                   d_ffn=18944, vocab=152064, mask_id=152063, rms_eps=1e-6, rope_base=1e6,
                   qkv_bias=True, weight_dtype="bf16", init_std=0.02, lm_scale=13.0, seed=2)

WORKLOADS: Dict[str, Workload] = {
    "c1": Workload("c1", TINY, batch=1, prompt_len=32, gen_len=64, window=16, p=32, draft=(48, 64),
                   tau_commit=0.7, tau_draft=0.98,
                   description="tiny mask predictor, 32 prompt + 64 generation, block 16, drafts in [48,64)"),
    "c2": Workload("c2", LLADA8B, batch=1, prompt_len=128, gen_len=256, window=32, p=128, draft=(0, 0),
                   tau_commit=0.7, tau_draft=0.98,
                   description="LLaDA-8B shape, B1, 128 prompt + 256 generation, first step of a block"),
    "c3": Workload("c3", LLADA8B, batch=1, prompt_len=256, gen_len=1024, window=32, p=256,
                   draft=(288, 352), tau_commit=0.7, tau_draft=0.98,
                   description="LLaDA-8B shape, B1, 256 prompt + 1024 generation, 64 draft positions"),
    "c4": Workload("c4", DREAM7B, batch=4, prompt_len=256, gen_len=512, window=32, p=256, draft=(0, 0),
                   tau_commit=0.75, tau_draft=0.98,
                   description="Dream-7B shape (GQA 28/4), B4, 256 prompt + 512 generation"),
    # Test-only variant of c1: with N(0, 0.02) init every masked row of c1 gets nearly the same hidden
    # state (confidences within ~0.002 of each other), so windows are always accepted whole. A larger
    # init std sharpens attention enough that confidences spread over about [0.3, 1].
    "c1s": Workload("c1s", dataclasses.replace(TINY, name="tiny-spread", init_std=0.08, lm_scale=10.0),
                    batch=2, prompt_len=32, gen_len=64, window=16, p=32, draft=(48, 64),
                    tau_commit=0.7, tau_draft=0.98,
                    description="tiny mask predictor with spread confidences, B2"),
    "c5": Workload("c5", LLADA8B, batch=8, prompt_len=0, gen_len=64, window=32, p=0, draft=(32, 64),
                   tau_commit=0.7, tau_draft=0.98, kv_prefix=1216, kv_seed=3,
                   description="LLaDA-8B shape, B8, 64 query tokens after a 1216-token cached prefix"),
}


def scaled(w: Workload, **geom_overrides) -> Workload:
    """Same workload recipe on a smaller geometry (for parity tests at oracle-friendly sizes)."""
    g = dataclasses.replace(w.geom, **geom_overrides)
    return dataclasses.replace(w, geom=g)


# ----------------------------------------------------------------------------------------------
# Weights: fixed tensor order, shared by the oracle and the HIP library's loader
# ----------------------------------------------------------------------------------------------

PER_LAYER = ("wq", "wk", "wv", "bq", "bk", "bv", "wo", "wg", "wu", "wd", "g1", "g2")


def tensor_specs(g: Geometry) -> List[Tuple[str, Tuple[int, ...], str]]:
    """(name, shape, kind) in load order. kind: 'mat' (random), 'bias' (random or absent), 'gain' (ones)."""
    d, H, Hkv, dh, F, V = g.d_model, g.n_heads, g.n_kv_heads, g.head_dim, g.d_ffn, g.vocab
    specs = [("embed", (V, d), "mat")]
    for l in range(g.n_layers):
        specs += [
            (f"l{l}.wq", (H * dh, d), "mat"), (f"l{l}.wk", (Hkv * dh, d), "mat"),
            (f"l{l}.wv", (Hkv * dh, d), "mat"),
            (f"l{l}.bq", (H * dh,), "bias"), (f"l{l}.bk", (Hkv * dh,), "bias"),
            (f"l{l}.bv", (Hkv * dh,), "bias"),
            (f"l{l}.wo", (d, H * dh), "mat"), (f"l{l}.wg", (F, d), "mat"), (f"l{l}.wu", (F, d), "mat"),
            (f"l{l}.wd", (d, F), "mat"), (f"l{l}.g1", (d,), "gain"), (f"l{l}.g2", (d,), "gain"),
        ]
    specs += [("gf", (d,), "gain"), ("lm_head", (V, d), "mat")]
    return specs


def make_tensor(g: Geometry, idx: int, name: str, shape, kind: str) -> Optional[np.ndarray]:
    """Generate tensor number ``idx``: float32 for f32 geometries, bf16 bits (uint16) otherwise.

    Biases are None when the geometry has none; gains are ones.
    """
    if kind == "bias" and not g.qkv_bias:
        return None
    if kind == "gain":
        return np.ones(shape, np.float32) if g.weight_dtype == "f32" else np.full(shape, 0x3F80, np.uint16)
    std = g.init_std * (g.lm_scale if name == "lm_head" else 1.0)
    if g.weight_dtype == "f32":
        return normal_f32(g.seed, idx, std, shape)
    return normal_bf16(g.seed, idx, std, shape)


def iter_weights(g: Geometry) -> Iterator[Tuple[str, Optional[np.ndarray]]]:
    for idx, (name, shape, kind) in enumerate(tensor_specs(g)):
        yield name, make_tensor(g, idx, name, shape, kind)


def make_weights(g: Geometry) -> Dict[str, Optional[np.ndarray]]:
    """All weights in host memory (the 8B geometries take ~16 GB as bf16)."""
    return dict(iter_weights(g))


def weights_as_f32(w: Dict[str, Optional[np.ndarray]]) -> Dict[str, Optional[np.ndarray]]:
    """View of the weights as float32 values (bf16 bits widened exactly)."""
    return {k: (None if v is None else (bf16_bits_to_f32(v) if v.dtype == np.uint16 else v))
            for k, v in w.items()}


# ----------------------------------------------------------------------------------------------
# Decode state and KV cache
# ----------------------------------------------------------------------------------------------

def prompts(w: Workload) -> np.ndarray:
    """[B, N] int32 prompt ids, independent seeded stream per batch row."""
    V = w.geom.vocab
    out = np.empty((w.batch, w.prompt_len), np.int32)
    for b in range(w.batch):
        out[b] = np.random.default_rng([w.geom.seed, 10000 + b]).integers(0, V - 2, w.prompt_len)
    return out


def random_drafts(w: Workload) -> np.ndarray:
    """[B, n_draft] int32 stand-ins for earlier top-1 predictions (random weights carry no meaning)."""
    V = w.geom.vocab
    n = w.draft[1] - w.draft[0]
    out = np.empty((w.batch, n), np.int32)
    for b in range(w.batch):
        out[b] = np.random.default_rng([w.geom.seed, 20000 + b]).integers(0, V - 2, n)
    return out


_STORED = os.path.join(os.path.dirname(_HERE), "tests", "golden")


def stored_drafts(w: Workload) -> Optional[np.ndarray]:
    """[B, n_draft] draft ids stored for this workload (``{key}_drafts.json``, written from earlier
    predictions by the golden-value script), or None when there are none for its geometry and region."""
    import json
    path = os.path.join(_STORED, f"{w.key}_drafts.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    d = np.asarray(rec["drafts"], np.int32)
    if rec.get("geometry") != w.geom.name or list(rec.get("draft_region", [])) != list(w.draft) or \
            d.shape != (w.batch, w.draft[1] - w.draft[0]):
        return None
    return d


def initial_state(w: Workload, drafts: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
    """(tokens [B,S] int32, p [B] int32): prompt, then mask ids; draft region filled if given.

    With ``drafts=None`` and a non-empty draft region, the stored drafts of the workload (earlier
    predictions, ``stored_drafts``) are used when there are some, the seeded random stand-ins otherwise.
    """
    B, S, mask = w.batch, w.seq, w.geom.mask_id
    tok = np.full((B, S), mask, np.int32)
    if w.kv_prefix == 0:
        tok[:, : w.prompt_len] = prompts(w)
    lo, hi = w.draft
    if hi > lo:
        if drafts is None:
            drafts = stored_drafts(w)
        tok[:, lo:hi] = random_drafts(w) if drafts is None else drafts
    p = np.full((B,), w.p, np.int32)
    return tok, p


def kv_cache_layer(w: Workload, layer: int) -> Tuple[np.ndarray, np.ndarray]:
    """Cached prefix K and V for one layer, bf16 bits.

    K: [B, Hkv, P, dh] (post-RoPE keys), V: [B, Hkv, dh, P] (stored key-contiguous).
    Values are N(0,1) activations from stream (kv_seed, 2*layer) / (kv_seed, 2*layer+1).
    """
    g, P = w.geom, w.kv_prefix
    k = normal_bf16(w.kv_seed, 2 * layer, 1.0, (w.batch, g.n_kv_heads, P, g.head_dim))
    v = normal_bf16(w.kv_seed, 2 * layer + 1, 1.0, (w.batch, g.n_kv_heads, g.head_dim, P))
    return k, v
