"""Host-side checks of the C ABI that need no GPU: the library loads, exports exactly the
symbols the headers declare, sizes workspaces, and rejects bad arguments with the documented
status codes before touching the device."""
import ctypes
import os
import re

import pytest

from paper_2608_21836_amd import binding as B
from synth import CONFIGS, TEST_CONFIGS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for h in ("ll.h", "ll_ops.h", "ll_mamba.h", "ll_mamba2.h", "ll_rglru.h"):
        text = open(os.path.join(ROOT, "include", h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(ll_\w+)\s*\(", text))
    return names


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        pytest.skip("libll.so not built")
    return B.load_library()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert names == {s[0] for s in B.SIGNATURES}
    for n in names:
        assert hasattr(lib, n), n
    # the binding's signatures resolve against the shared object
    for n, _, _ in B.SIGNATURES:
        ctypes.cast(getattr(lib, n), ctypes.c_void_p)


def cfg_for(name, **over):
    c = {**CONFIGS, **TEST_CONFIGS}[name]
    lens = c.prompt_list or ([c.prompt_len] * c.batch if c.prompt_len else [c.prompt_range[1]] * c.batch)
    cfg = B.make_config(c, c.batch, sum(lens), max(lens) + c.n_decode)
    for k, v in over.items():
        setattr(cfg, k, v)
    return cfg


def status_of(lib, cfg):
    n = ctypes.c_size_t(0)
    return lib.ll_workspace_size(ctypes.byref(cfg), ctypes.byref(n)), n.value


@pytest.mark.parametrize("name", sorted(CONFIGS) + sorted(TEST_CONFIGS))
def test_workspace_size_of_every_workload(lib, name):
    st, n = status_of(lib, cfg_for(name))
    assert st == B.LL_OK, lib.ll_last_error()
    c = {**CONFIGS, **TEST_CONFIGS}[name]
    eb = 2 if c.dtype == "bf16" else 4
    weights = (2 * c.vocab * c.d_model + c.n_layers * c.linear_params_per_layer()) * eb
    assert n > weights


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 96, B.LL_ERR_UNSUPPORTED),
    ("n_kv_heads", 5, B.LL_ERR_UNSUPPORTED),
    ("d_model", 200, B.LL_ERR_UNSUPPORTED),
    ("ffn_dim", 1000, B.LL_ERR_UNSUPPORTED),
    ("vocab", 1000, B.LL_ERR_UNSUPPORTED),
    ("dtype", 7, B.LL_ERR_UNSUPPORTED),
    ("max_batch", 257, B.LL_ERR_UNSUPPORTED),
    ("n_layers", 0, B.LL_ERR_INVALID_ARGUMENT),
    ("max_ctx", 0, B.LL_ERR_INVALID_ARGUMENT),
    ("rope_theta", -1.0, B.LL_ERR_INVALID_ARGUMENT),
    ("rms_eps", float("nan"), B.LL_ERR_INVALID_ARGUMENT),
    ("kv_page", 100, B.LL_ERR_UNSUPPORTED),       # pages hold a multiple of 256 positions
    ("kv_page", -256, B.LL_ERR_INVALID_ARGUMENT),
    ("kv_pages", 4, B.LL_ERR_INVALID_ARGUMENT),   # a pool size without a page size
])
def test_config_validation(lib, field, value, status):
    st, _ = status_of(lib, cfg_for("tiny-f32", **{field: value}))
    assert st == status
    assert lib.ll_last_error()


def test_paged_workspace_holds_the_pool_not_every_context():
    full = cfg_for("8b-gqa")
    st0, contiguous = status_of(lib := B.load_library(), full)
    paged = cfg_for("8b-gqa", kv_page=256)
    st1, same_pool = status_of(lib, paged)
    small = cfg_for("8b-gqa", kv_page=256, kv_pages=300)
    st2, small_pool = status_of(lib, small)
    assert st0 == st1 == st2 == B.LL_OK
    # the default pool covers max_batch full contexts (within page rounding); a smaller pool
    # saves exactly its missing pages (K and V, every layer)
    assert abs(same_pool - contiguous) < 0.05 * contiguous
    c = {**CONFIGS, **TEST_CONFIGS}["8b-gqa"]
    page_bytes = 2 * c.n_layers * c.n_kv_heads * 256 * c.head_dim * 2
    default_pages = full.max_batch * ((full.max_ctx + 255) // 256)
    assert abs((same_pool - small_pool) - (default_pages - 300) * page_bytes) < 4096


def test_group_of_sixteen_rejected(lib):
    st, _ = status_of(lib, cfg_for("tiny-f32", n_heads=16, n_kv_heads=1))
    assert st == B.LL_ERR_UNSUPPORTED


def test_null_arguments(lib):
    cfg = cfg_for("tiny-f32")
    assert lib.ll_workspace_size(None, ctypes.byref(ctypes.c_size_t())) == B.LL_ERR_INVALID_ARGUMENT
    assert lib.ll_workspace_size(ctypes.byref(cfg), None) == B.LL_ERR_INVALID_ARGUMENT
    h = ctypes.c_void_p()
    assert lib.ll_model_load(ctypes.byref(cfg), None, None, 0, None, ctypes.byref(h)) == \
        B.LL_ERR_INVALID_ARGUMENT
    assert lib.ll_prefill(None, 1, None, None, None, None) == B.LL_ERR_INVALID_ARGUMENT
    assert lib.ll_decode_step(None, None, None, None) == B.LL_ERR_INVALID_ARGUMENT
    assert lib.ll_kv_reset(None) == B.LL_ERR_INVALID_ARGUMENT
    lib.ll_model_free(None)


def _fake_weights(n_layers, ptr=0x1000):
    arr = (ctypes.c_void_p * n_layers)(*([ptr] * n_layers))
    p = ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p))
    return B.LLWeights(ptr, ptr, ptr, p, p, p, p, p, p, p, p, p), arr


def test_load_rejects_workspace_problems_before_any_device_call(lib):
    cfg = cfg_for("tiny-f32")
    w, keep = _fake_weights(cfg.n_layers)
    h = ctypes.c_void_p()
    _, need = status_of(lib, cfg)
    # NULL workspace
    assert lib.ll_model_load(ctypes.byref(cfg), ctypes.byref(w), None, need, None,
                             ctypes.byref(h)) == B.LL_ERR_WORKSPACE
    # misaligned
    assert lib.ll_model_load(ctypes.byref(cfg), ctypes.byref(w), 0x10010, need, None,
                             ctypes.byref(h)) == B.LL_ERR_WORKSPACE
    # too small
    assert lib.ll_model_load(ctypes.byref(cfg), ctypes.byref(w), 0x10000, need - 1, None,
                             ctypes.byref(h)) == B.LL_ERR_WORKSPACE
    assert "needs" in lib.ll_last_error().decode()
    # a NULL per-layer pointer
    arr = (ctypes.c_void_p * cfg.n_layers)(0x1000, None)
    w.wo = ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p))
    assert lib.ll_model_load(ctypes.byref(cfg), ctypes.byref(w), 0x10000, need, None,
                             ctypes.byref(h)) == B.LL_ERR_INVALID_ARGUMENT
    assert not h.value


def test_op_argument_validation(lib):
    # sizes are checked before any launch
    assert lib.ll_op_gemm(0, 1, 4, 100, 64, 1, 1, 1, 0, None) == B.LL_ERR_UNSUPPORTED
    assert lib.ll_op_gemm(1, 1, 4, 64, 60, 1, 1, 1, 0, None) == B.LL_ERR_UNSUPPORTED
    assert lib.ll_op_gemm(2, 1, 4, 64, 64, 1, 1, 1, 0, None) == B.LL_ERR_INVALID_ARGUMENT
    assert lib.ll_op_gemm(1, 1, 4, 64, 64, None, 1, 1, 0, None) == B.LL_ERR_INVALID_ARGUMENT
    assert lib.ll_op_rmsnorm(1, 4, 6, 1, 1, 1e-5, 1, None) == B.LL_ERR_INVALID_ARGUMENT
    assert lib.ll_op_repack(1, 20, 64, 1, 1, None) == B.LL_ERR_UNSUPPORTED
    lens = (ctypes.c_int32 * 2)(5, 0)
    assert lib.ll_op_attn_prefill(1, 2, lens, None, 8, 2, 64, 16, 1, 1, 1, 1, 0x10000, 4096,
                                  None) == B.LL_ERR_INVALID_ARGUMENT
    # cached keys + new tokens beyond max_ctx
    lens = (ctypes.c_int32 * 1)(5)
    cached = (ctypes.c_int32 * 1)(12)
    assert lib.ll_op_attn_prefill(1, 1, lens, cached, 8, 2, 64, 16, 1, 1, 1, 1, 0x10000, 4096,
                                  None) == B.LL_ERR_INVALID_ARGUMENT
    assert lib.ll_op_attn_decode(1, 1, 8, 3, 64, 16, 1, 1, 1, 1, 1, 0x10000, 1 << 20, None) == \
        B.LL_ERR_UNSUPPORTED
    assert lib.ll_op_attn_decode(1, 1, 8, 2, 64, 16, 1, 1, 1, 1, 1, 0x10000, 8, None) == \
        B.LL_ERR_WORKSPACE
    assert lib.ll_op_lmhead_argmax(1, 2, 100, 64, 1, 1, None, 1, 0x10000, 1 << 20, None) == \
        B.LL_ERR_UNSUPPORTED
    assert lib.ll_op_attn_decode_scratch(0, 8, 2, 64, 16) == 0


def test_option_calls_reject_a_null_model(lib):
    v = ctypes.c_int32(0)
    assert lib.ll_set_option(None, 0, 1) == B.LL_ERR_INVALID_ARGUMENT
    assert lib.ll_get_option(None, 0, ctypes.byref(v)) == B.LL_ERR_INVALID_ARGUMENT
    assert set(B.OPTIONS.values()) == set(range(len(B.OPTIONS)))


# ------------------------------------------------------------------------------------------
# State-space families (ll_mamba.h, ll_mamba2.h, ll_rglru.h): host-side checks only
# ------------------------------------------------------------------------------------------
def _ssm_families():
    from synth import mamba as SM
    from synth import mamba2 as S2
    from synth import rglru as SR
    out = []
    for prefix, make, cfgs in (("ll_mamba_", B.make_mamba_config, {**SM.MAMBA_CONFIGS, **SM.MAMBA_TEST_CONFIGS}),
                               ("ll_mamba2_", B.make_mamba2_config, {**S2.MAMBA2_CONFIGS, **S2.MAMBA2_TEST_CONFIGS}),
                               ("ll_rg_", B.make_rg_config, {**SR.RG_CONFIGS, **SR.RG_TEST_CONFIGS})):
        for name, c in cfgs.items():
            out.append((prefix, make, c))
    return out


def _ssm_status(lib, prefix, cfg):
    n = ctypes.c_size_t(0)
    return getattr(lib, prefix + "workspace_size")(ctypes.byref(cfg), ctypes.byref(n)), n.value


@pytest.mark.parametrize("prefix,make,c", _ssm_families(), ids=lambda v: getattr(v, "name", str(v)))
def test_ssm_workspace_size_of_every_workload(lib, prefix, make, c):
    lens = c.prompt_list or ([c.prompt_len] * c.batch if c.prompt_len else [c.prompt_range[1]] * c.batch)
    st, n = _ssm_status(lib, prefix, make(c, c.batch, sum(lens)))
    assert st == B.LL_OK, lib.ll_last_error()
    eb = 2 if c.dtype == "bf16" else 4
    assert n > (2 * c.vocab * c.d_model + c.n_layers * c.linear_params_per_layer()) * eb


def _rg_cfg(**over):
    from synth import rglru as SR
    cfg = B.make_rg_config(SR.RG_TEST_CONFIGS["t-rg-f32"], 2, 256)
    for k, v in over.items():
        setattr(cfg, k, v)
    return cfg


@pytest.mark.parametrize("field,value,status", [
    ("n_heads", 3, B.LL_ERR_UNSUPPORTED),          # blocks of 256 / 3 columns
    ("lru_width", 320, B.LL_ERR_UNSUPPORTED),      # blocks of 80
    ("mlp_width", 100, B.LL_ERR_UNSUPPORTED),
    ("d_model", 200, B.LL_ERR_UNSUPPORTED),
    ("d_conv", 5, B.LL_ERR_UNSUPPORTED),
    ("vocab", 1000, B.LL_ERR_UNSUPPORTED),
    ("max_batch", 257, B.LL_ERR_UNSUPPORTED),
    ("logit_cap", 0.0, B.LL_ERR_INVALID_ARGUMENT),
    ("embed_scale", float("inf"), B.LL_ERR_INVALID_ARGUMENT),
    ("rms_eps", float("nan"), B.LL_ERR_INVALID_ARGUMENT),
    ("n_layers", 0, B.LL_ERR_INVALID_ARGUMENT),
])
def test_rg_config_validation(lib, field, value, status):
    st, _ = _ssm_status(lib, "ll_rg_", _rg_cfg(**{field: value}))
    assert st == status
    assert lib.ll_last_error()


def test_rg_null_arguments_and_workspace_checks(lib):
    cfg = _rg_cfg()
    assert lib.ll_rg_workspace_size(None, ctypes.byref(ctypes.c_size_t())) == B.LL_ERR_INVALID_ARGUMENT
    h = ctypes.c_void_p()
    assert lib.ll_rg_load(ctypes.byref(cfg), None, None, 0, None, ctypes.byref(h)) == \
        B.LL_ERR_INVALID_ARGUMENT
    nl = cfg.n_layers
    arr = (ctypes.c_void_p * nl)(*([0x1000] * nl))
    p = ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p))
    w = B.LLRGWeights(0x1000, 0x1000, **{f: p for f in B.RG_LAYER_FIELDS})
    # misaligned workspace, then one too small: rejected before any device call
    assert lib.ll_rg_load(ctypes.byref(cfg), ctypes.byref(w), 0x1001, 1 << 40, None,
                          ctypes.byref(h)) != B.LL_OK
    assert lib.ll_rg_load(ctypes.byref(cfg), ctypes.byref(w), 0x100000, 16, None,
                          ctypes.byref(h)) == B.LL_ERR_WORKSPACE
    w.mlp_down_b = None
    assert lib.ll_rg_load(ctypes.byref(cfg), ctypes.byref(w), 0x100000, 1 << 40, None,
                          ctypes.byref(h)) == B.LL_ERR_INVALID_ARGUMENT
    assert lib.ll_rg_prefill(None, 1, None, None, None, None) == B.LL_ERR_INVALID_ARGUMENT
    assert lib.ll_rg_decode_step(None, None, None, None) == B.LL_ERR_INVALID_ARGUMENT
    assert lib.ll_rg_reset(None) == B.LL_ERR_INVALID_ARGUMENT
    assert lib.ll_rg_set_option(None, 0, 1) == B.LL_ERR_INVALID_ARGUMENT
    assert lib.ll_rg_kernel_class_name(B.LL_RGK_COUNT) == b""
    assert lib.ll_rg_kernel_class_name(5) == b"gates"
    lib.ll_rg_free(None)
