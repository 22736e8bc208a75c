"""CPU-only checks of the C ABI: the library loads, exports every symbol include/dcl.h declares,
and rejects bad arguments on the host before touching a device."""
import ctypes
import os
import re

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def dcl():
    from paper_2607_20467_amd import build
    if build.is_stale():
        build.build()
    import paper_2607_20467_amd as m
    m.load_library()
    return m


def test_exports_every_declared_symbol(dcl):
    header = open(os.path.join(ROOT, "include", "dcl.h")).read()
    declared = set(re.findall(r"\b(dcl_[a-z_]+)\s*\(", header))
    assert {"dcl_denoise_step", "dcl_select_contiguous", "dcl_load_weights"} <= declared
    lib = ctypes.CDLL(dcl.library_path())
    for name in sorted(declared):
        assert hasattr(lib, name), name


def test_status_strings(dcl):
    assert dcl.dcl_status_string(0) == "ok"
    assert "argument" in dcl.dcl_status_string(1)
    assert dcl.dcl_status_string(99) == "unknown status"


def _cfg(dcl, **kw):
    c = dcl.config_from_geometry(synth.LLADA8B)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 96, 2), ("n_kv_heads", 5, 2), ("d_model", 4100, 2), ("d_model", 8208, 2), ("d_ffn", 8, 2), ("vocab", 1, 1),
    ("mask_id", 126464, 1), ("mask_id", -1, 1), ("rms_eps", 0.0, 1), ("rope_base", 1.0, 1),
    ("max_positions", 0, 1), ("n_layers", 0, 1), ("qkv_bias", 2, 1),
    ("vocab", 524288, 2), ("d_ffn", 262144, 2)])   # a weight matrix of 2^31 elements (LM head, gate||up)
def test_model_create_rejects(dcl, field, value, status):
    with pytest.raises(dcl.DclError) as e:
        dcl.dcl_model_create(_cfg(dcl, **{field: value}))
    assert e.value.status == status
    assert dcl.dcl_last_error()
    assert dcl.dcl_weights_bytes(_cfg(dcl, **{field: value})) == 0


def test_model_create_accepts_weight_matrices_just_below_2_31(dcl):
    m = dcl.dcl_model_create(_cfg(dcl, vocab=524287, d_ffn=262128))
    dcl.dcl_model_destroy(m)


def test_sizes(dcl):
    cfg = _cfg(dcl)
    wb = dcl.dcl_weights_bytes(cfg)
    params = synth.LLADA8B.vocab * 4096 * 2 + 32 * (4 * 4096 * 4096 + 3 * 4096 * 12288)
    assert params * 2 <= wb <= params * 2 + 64 * 2 ** 20        # bf16 matrices + small vectors / tables
    m = dcl.dcl_model_create(cfg)
    try:
        a = dcl.dcl_workspace_bytes(m, 1, 384, 0)
        assert a > 0 and dcl.dcl_workspace_bytes(m, 4, 768, 0) > a
        assert dcl.dcl_workspace_bytes(m, 0, 384, 0) == 0
        assert dcl.dcl_workspace_bytes(m, 1, 0, 0) == 0
    finally:
        dcl.dcl_model_destroy(m)


def test_step_and_select_argument_checks_without_gpu(dcl):
    """Every failure below is detected on the host; no HIP call is made (there is no GPU here)."""
    lib = dcl.load_library()
    m = dcl.dcl_model_create(_cfg(dcl))
    try:
        st = dcl.binding.DclRowStats(1, 1, 1, 1, 1)
        # weights not loaded
        r = lib.dcl_denoise_step(m, 8, 1, 384, 8, 384, None, 0, st, 256, 1 << 40, None)
        assert r == 5 and "not loaded" in dcl.dcl_last_error()
        steps = ctypes.c_int32(-1)
        r = lib.dcl_generate(m, 8, 1, 384, 8, 384, None, 0, 32, 0, 0, 0.7, 0.98, 0, 10, 1, st, None, None, None, 256,
                             1 << 40, ctypes.byref(steps), None)
        assert r == 5 and "not loaded" in dcl.dcl_last_error()
        # load: misaligned / too small / wrong count
        arr = (ctypes.c_void_p * 3)(1, 2, 3)
        assert lib.dcl_load_weights(m, 3, 1 << 40, arr, 3, 1, None) == 1
        assert lib.dcl_load_weights(m, 256, 16, arr, 3, 1, None) == 3
        assert lib.dcl_load_weights(m, 256, 1 << 40, arr, 3, 1, None) == 1
        assert "n_src" in dcl.dcl_last_error()
        assert lib.dcl_load_weights(m, 256, 1 << 40, arr, 3, 7, None) == 1
    finally:
        dcl.dcl_model_destroy(m)
    sel = lib.dcl_select_contiguous
    st = dcl.binding.DclRowStats(1, 1, 1, 1, 1)
    assert sel(None, 1, 8, 8, 8, 4, 0, 0, 0.7, 0.98, 3, st, None, None, 0, None) == 1
    assert sel(8, 1, 8, 8, 9, 4, 0, 0, 0.7, 0.98, 3, st, None, None, 0, None) == 1      # gen_end > S
    assert sel(8, 1, 8, 8, 8, 0, 0, 0, 0.7, 0.98, 3, st, None, None, 0, None) == 1      # L = 0
    assert sel(8, 1, 8, 8, 8, 4, 0, 0, 1.5, 0.98, 3, st, None, None, 0, None) == 1      # tau_commit > 1
    assert sel(8, 1, 8, 8, 8, 4, 0, 0, 0.7, -0.1, 3, st, None, None, 0, None) == 1      # tau_draft < 0
    assert sel(8, 1, 8, 8, 8, 4, 0, 0, 0.7, 0.98, 3, st, None, None, 64, None) == 1     # unknown flag
    assert "flags" in dcl.dcl_last_error()
    assert sel(8, 1, 8, 8, 8, 4, 0, 0, 0.7, 0.98, 3, st, None, None, 4 | 2, None) == 1  # non-contiguous + score-all
    assert sel(8, 1, 8, 8, 8, 4, 0, 0, 0.7, 0.98, 3, st, None, None, 4 | 8, None) == 1  # non-contiguous + chain drafts
    assert "NONCONTIGUOUS" in dcl.dcl_last_error()
    assert sel(8, 1, 8, 8, 8, 4, 0, -1, 0.7, 0.98, 3, st, None, None, 0, None) == 1   # block_len < 0
    assert sel(8, 1, 8, 8, 8, 4, 9, 4, 0.7, 0.98, 3, st, None, None, 0, None) == 1    # block origin > S
    assert "block" in dcl.dcl_last_error()
    bad = dcl.binding.DclRowStats(0, 1, 0, 1, 1)
    assert sel(8, 1, 8, 8, 8, 4, 0, 0, 0.7, 0.98, 3, bad, None, None, 0, None) == 1


def test_product_has_no_oracle_dependency():
    """The product package never imports the oracle (test infrastructure) or falls back to the CPU."""
    pkg = os.path.join(ROOT, "paper_2607_20467_amd")
    for fn in os.listdir(pkg):
        if fn.endswith(".py"):
            src = open(os.path.join(pkg, fn)).read()
            assert not re.search(r"^\s*(import|from)\s+oracle", src, re.M), fn


def test_binding_flag_constants_match_header():
    """Every #define DCL_* flag of include/dcl.h has the same value in the Python binding."""
    import paper_2607_20467_amd.binding as b
    hdr = open(os.path.join(ROOT, "include", "dcl.h")).read()
    defs = dict(re.findall(r"#define\s+(DCL_\w+)\s+(0x[0-9a-fA-F]+)u", hdr))
    assert {"DCL_SCORE_ALL_UNCOMMITTED", "DCL_SCORE_SUPPRESS_MASK", "DCL_SEL_NONCONTIGUOUS",
            "DCL_SEL_CONTIGUOUS_DRAFTS"} <= set(defs)
    for name, val in defs.items():
        assert getattr(b, name) == int(val, 16), name


def test_step_size_limits_rejected_on_the_host(dcl):
    """The 32-bit offset limits of dcl_denoise_step are checked before the weights-loaded state and before
    any HIP call: one 4096-token sequence more than the largest accepted batch of the small model (q/k/v^T
    would reach 2^31 elements), B*S above 2^22, and FFN activations of 2^31 elements."""
    import dataclasses
    lib = dcl.load_library()
    st = dcl.binding.DclRowStats(256, 256, 256, 256, 256)

    def step(cfg, B, S):
        m = dcl.dcl_model_create(cfg)
        try:
            r = lib.dcl_denoise_step(m, 256, B, S, 256, S, None, 0, st, 256, 1 << 40, None)
            return r, dcl.dcl_last_error()
        finally:
            dcl.dcl_model_destroy(m)

    tiny = dcl.config_from_geometry(synth.TINY, max_positions=4096)
    g = synth.TINY
    qkv_rows = (g.n_heads + 2 * g.n_kv_heads) * g.head_dim
    assert 681 * (4096 + 8) * qkv_rows < 2 ** 31 <= 682 * (4096 + 8) * qkv_rows
    r, msg = step(tiny, 682, 4096)
    assert r == 2 and "q/k/v" in msg
    r, msg = step(tiny, 681, 4096)
    assert r == 5 and "not loaded" in msg            # within the limits: only the state check remains
    r, msg = step(tiny, 1025, 4096)
    assert r == 1 and "too large" in msg
    wide = dcl.config_from_geometry(dataclasses.replace(g, n_layers=1, d_model=64, n_heads=1, n_kv_heads=1,
                                                        head_dim=64, d_ffn=65536, vocab=256, mask_id=255),
                                    max_positions=4096)
    r, msg = step(wide, 8, 4096)
    assert r == 2 and "activation" in msg


def test_binding_rejects_host_tensors_before_calling_the_library(dcl):
    """The binding checks tensor arguments (device, dtype, size) and raises before the C call."""
    import torch
    tok = torch.zeros((1, 8), dtype=torch.int32)
    with pytest.raises(dcl.DclError) as e:
        dcl.dcl_select_contiguous(tok, 1, 8, 256, 8, 4, 0.7, 0.98, 3, {"top1": 256, "conf": 256})
    assert e.value.status == 1 and "device" in str(e.value)


def test_noalloc_step_rejects_sizes_beyond_its_scratch_on_the_host(dcl):
    """dcl_denoise_step_noalloc refuses a step whose workspace exceeds the static scratch before the
    weights-loaded state and before any HIP call."""
    lib = dcl.load_library()
    m = dcl.dcl_model_create(dcl.config_from_geometry(synth.LLADA8B, max_positions=4096))
    try:
        st = dcl.binding.DclRowStats(256, 256, 256, 256, 256)
        assert dcl.dcl_workspace_bytes(m, 1, 384, 0) <= dcl.DCL_NOALLOC_SCRATCH_BYTES
        assert dcl.dcl_workspace_bytes(m, 1, 1280, 0) > dcl.DCL_NOALLOC_SCRATCH_BYTES
        r = lib.dcl_denoise_step_noalloc(m, 256, 1, 1280, 256, 1280, None, 0, st, None)
        assert r == 3 and "static scratch" in dcl.dcl_last_error()
        r = lib.dcl_denoise_step_noalloc(m, 256, 1, 384, 256, 384, None, 0, st, None)
        assert r == 5 and "not loaded" in dcl.dcl_last_error()
    finally:
        dcl.dcl_model_destroy(m)


@pytest.mark.parametrize("nw,t,k,lm", [(24576, 384, 4096, False), (4096, 384, 12288, False), (126464, 384, 4096, True),
                                       (800, 111, 208, False), (208, 111, 400, False), (1000, 60, 208, True),
                                       (4608, 3072, 3584, False), (12288, 1280, 4160, False)])
def test_gemm_plans_fit_their_depth(dcl, nw, t, k, lm):
    """The reported plan is the one that runs: its stage depth divides K (the tuned kernels carry no K-tail
    handling), except for the single tail-aware configuration 0 that serves every other K; an LM-head plan
    is one of the two vocabulary-tile layouts the fused epilogue is written for."""
    plan = dcl.dcl_debug_gemm_plan(nw, t, k, lm_head=lm)
    assert k % plan["kd"] == 0 or plan["cfg"] == 0, plan
    if lm:
        assert plan["bw"] // plan["ww"] == 128 or (plan["bw"] == 128 and plan["ww"] == 2), plan
