"""ctypes binding of libll.so: argument marshalling only.

Every step of the forward pass runs in the library's HIP kernels; PyTorch provides device
memory (weights, workspace, tokens, logits) and the stream.  There is no fallback: if the
library is missing, loading raises.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_float, c_int32, c_int64, c_size_t, c_uint64, c_void_p
from typing import Dict, List, Optional, Sequence, Tuple

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libll.so")

LL_OK, LL_ERR_INVALID_ARGUMENT, LL_ERR_UNSUPPORTED, LL_ERR_CAPACITY, LL_ERR_STATE, \
    LL_ERR_WORKSPACE, LL_ERR_HIP = range(7)
STATUS_NAMES = ["LL_OK", "LL_ERR_INVALID_ARGUMENT", "LL_ERR_UNSUPPORTED", "LL_ERR_CAPACITY",
                "LL_ERR_STATE", "LL_ERR_WORKSPACE", "LL_ERR_HIP"]
LL_F32, LL_BF16, LL_F16 = 0, 1, 2
LL_MAX_BATCH = 256
LL_K_COUNT = 11
# ll_option ids (include/ll.h)
OPTIONS = {"decode_graph": 0, "prefill_splitk": 1, "decode_splitk": 2, "prefill_tile": 3,
           "attn_decode_chunk": 4, "decode_fused": 5}
DECODER_OPTIONS = ("decode_graph", "prefill_splitk", "decode_splitk", "prefill_tile",
                   "attn_decode_chunk", "decode_fused")
MAMBA_OPTIONS = ("decode_graph", "prefill_splitk", "decode_splitk", "prefill_tile", "decode_fused")
MAMBA2_OPTIONS = ("decode_graph", "prefill_splitk", "decode_splitk", "prefill_tile")
RG_OPTIONS = MAMBA2_OPTIONS
PHASES = ("prefill", "decode")


class LLConfig(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("d_model", c_int32), ("n_heads", c_int32),
                ("n_kv_heads", c_int32), ("head_dim", c_int32), ("ffn_dim", c_int32),
                ("vocab", c_int32), ("rms_eps", c_float), ("rope_theta", c_double),
                ("dtype", c_int32), ("max_batch", c_int32), ("max_prefill_tokens", c_int32),
                ("max_ctx", c_int32), ("kv_page", c_int32), ("kv_pages", c_int32),
                ("f16_compute", c_int32)]


class LLWeights(ctypes.Structure):
    _fields_ = [("tok_embed", c_void_p), ("final_norm", c_void_p), ("lm_head", c_void_p),
                ("attn_norm", POINTER(c_void_p)), ("wq", POINTER(c_void_p)),
                ("wk", POINTER(c_void_p)), ("wv", POINTER(c_void_p)), ("wo", POINTER(c_void_p)),
                ("mlp_norm", POINTER(c_void_p)), ("w_gate", POINTER(c_void_p)),
                ("w_up", POINTER(c_void_p)), ("w_down", POINTER(c_void_p))]


class LLMambaConfig(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("d_model", c_int32), ("d_inner", c_int32),
                ("d_state", c_int32), ("d_conv", c_int32), ("dt_rank", c_int32),
                ("vocab", c_int32), ("rms_eps", c_float), ("dtype", c_int32),
                ("max_batch", c_int32), ("max_prefill_tokens", c_int32)]


MAMBA_LAYER_FIELDS = ("norm", "in_proj", "conv_w", "conv_b", "x_proj", "dt_w", "dt_b", "A_log",
                      "D", "out_proj")
# tensors kept in fp32 whatever the workload dtype
MAMBA_F32_FIELDS = ("conv_w", "conv_b", "dt_w", "dt_b", "A_log", "D")


class LLMambaWeights(ctypes.Structure):
    _fields_ = [("embed", c_void_p), ("final_norm", c_void_p)] + \
        [(f, POINTER(c_void_p)) for f in MAMBA_LAYER_FIELDS]


LL_MK_COUNT = 12


class LLMamba2Config(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("d_model", c_int32), ("d_inner", c_int32),
                ("d_state", c_int32), ("head_dim", c_int32), ("n_groups", c_int32),
                ("d_conv", c_int32), ("vocab", c_int32), ("rms_eps", c_float),
                ("dtype", c_int32), ("max_batch", c_int32), ("max_prefill_tokens", c_int32)]


MAMBA2_LAYER_FIELDS = ("norm", "in_proj", "conv_w", "conv_b", "dt_b", "A_log", "D", "gnorm",
                       "out_proj")
MAMBA2_F32_FIELDS = ("conv_w", "conv_b", "dt_b", "A_log", "D")


class LLMamba2Weights(ctypes.Structure):
    _fields_ = [("embed", c_void_p), ("final_norm", c_void_p)] + \
        [(f, POINTER(c_void_p)) for f in MAMBA2_LAYER_FIELDS]


LL_M2K_COUNT = 12


class LLRGConfig(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("d_model", c_int32), ("lru_width", c_int32),
                ("n_heads", c_int32), ("mlp_width", c_int32), ("d_conv", c_int32),
                ("vocab", c_int32), ("rms_eps", c_float), ("embed_scale", c_float),
                ("logit_cap", c_float), ("dtype", c_int32), ("max_batch", c_int32),
                ("max_prefill_tokens", c_int32)]


RG_LAYER_FIELDS = ("norm_t", "linear_y", "linear_y_b", "linear_x", "linear_x_b", "conv_w",
                   "conv_b", "gate_a", "gate_a_b", "gate_x", "gate_x_b", "lambda", "linear_out",
                   "linear_out_b", "norm_c", "mlp_gate", "mlp_gate_b", "mlp_up", "mlp_up_b",
                   "mlp_down", "mlp_down_b")
RG_F32_FIELDS = ("linear_y_b", "linear_x_b", "conv_w", "conv_b", "gate_a_b", "gate_x_b",
                 "lambda", "linear_out_b", "mlp_gate_b", "mlp_up_b", "mlp_down_b")


class LLRGWeights(ctypes.Structure):
    _fields_ = [("embed", c_void_p), ("final_norm", c_void_p)] + \
        [(f, POINTER(c_void_p)) for f in RG_LAYER_FIELDS]


LL_RGK_COUNT = 14

# (name, restype, argtypes) of every exported symbol; include/ll.h, include/ll_ops.h and
# include/ll_mamba.h declare the same set.
SIGNATURES = [
    ("ll_workspace_size", c_int32, [POINTER(LLConfig), POINTER(c_size_t)]),
    ("ll_model_load", c_int32, [POINTER(LLConfig), POINTER(LLWeights), c_void_p, c_size_t,
                                c_void_p, POINTER(c_void_p)]),
    ("ll_prefill", c_int32, [c_void_p, c_int32, POINTER(c_int32), c_void_p, c_void_p, c_void_p]),
    ("ll_decode_step", c_int32, [c_void_p, c_void_p, c_void_p, c_void_p]),
    ("ll_kv_reset", c_int32, [c_void_p]),
    ("ll_seq_lengths", c_int32, [c_void_p, POINTER(c_int32), c_int32, POINTER(c_int32)]),
    ("ll_workspace_regions", c_int32, [c_void_p, c_int32, POINTER(c_uint64), POINTER(c_uint64),
                                       POINTER(c_char_p), POINTER(c_int32)]),
    ("ll_kv_pages", c_int32, [c_void_p, POINTER(c_int32), POINTER(c_int32)]),
    ("ll_op_mfma_loop", c_int32, [c_int32, c_int32, c_void_p, c_void_p]),
    ("ll_op_read_stream", c_int32, [c_void_p, c_int64, c_int32, c_void_p, c_void_p]),
    ("ll_set_decode_graph", c_int32, [c_void_p, c_int32]),
    ("ll_set_option", c_int32, [c_void_p, c_int32, c_int32]),
    ("ll_get_option", c_int32, [c_void_p, c_int32, POINTER(c_int32)]),
    ("ll_device_flags", c_int32, [c_void_p, POINTER(c_int32)]),
    ("ll_set_kernel_timing", c_int32, [c_void_p, c_int32]),
    ("ll_kernel_timing_read", c_int32, [c_void_p, POINTER(c_int32), POINTER(c_double)]),
    ("ll_kernel_class_name", c_char_p, [c_int32]),
    ("ll_model_free", None, [c_void_p]),
    ("ll_last_error", c_char_p, []),
    ("ll_op_rmsnorm", c_int32, [c_int32, c_int32, c_int32, c_void_p, c_void_p, c_float,
                                c_void_p, c_void_p]),
    ("ll_op_repack", c_int32, [c_int32, c_int32, c_int32, c_void_p, c_void_p, c_void_p]),
    ("ll_op_gemm", c_int32, [c_int32, c_int32, c_int32, c_int32, c_int32, c_void_p, c_void_p,
                             c_void_p, c_int32, c_void_p]),
    ("ll_op_gemm_swiglu", c_int32, [c_int32, c_int32, c_int32, c_int32, c_void_p, c_void_p,
                                    c_void_p, c_void_p]),
    ("ll_op_gemm_splitk", c_int32, [c_int32, c_int32, c_int32, c_int32, c_void_p, c_void_p,
                                    c_void_p, c_int32, c_void_p, c_size_t, c_void_p]),
    ("ll_op_gemm_splitk_scratch", c_size_t, [c_int32, c_int32, c_int32, c_int32]),
    ("ll_op_gemm_prefill_splitk", c_int32, [c_int32, c_int32, c_int32, c_int32, c_void_p,
                                            c_void_p, c_void_p, c_int32, c_void_p, c_size_t,
                                            c_void_p]),
    ("ll_op_gemm_prefill_splitk_scratch", c_size_t, [c_int32, c_int32, c_int32, c_int32]),
    ("ll_op_attn_prefill", c_int32, [c_int32, c_int32, POINTER(c_int32), POINTER(c_int32),
                                     c_int32, c_int32, c_int32, c_int32, c_void_p, c_void_p,
                                     c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    ("ll_op_attn_prefill_scratch", c_size_t, [c_int32, c_int32, POINTER(c_int32),
                                              POINTER(c_int32), c_int32, c_int32, c_int32,
                                              c_int32]),
    ("ll_op_attn_decode", c_int32, [c_int32, c_int32, c_int32, c_int32, c_int32, c_int32,
                                    c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                    c_size_t, c_void_p]),
    ("ll_op_attn_decode_scratch", c_size_t, [c_int32, c_int32, c_int32, c_int32, c_int32]),
    ("ll_op_lmhead_argmax", c_int32, [c_int32, c_int32, c_int32, c_int32, c_void_p, c_void_p,
                                      c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    ("ll_op_lmhead_argmax_noalloc", c_int32, [c_int32, c_int32, c_int32, c_int32, c_void_p,
                                              c_void_p, c_void_p, c_void_p, c_void_p]),
    ("ll_mamba_workspace_size", c_int32, [POINTER(LLMambaConfig), POINTER(c_size_t)]),
    ("ll_mamba_load", c_int32, [POINTER(LLMambaConfig), POINTER(LLMambaWeights), c_void_p,
                                c_size_t, c_void_p, POINTER(c_void_p)]),
    ("ll_mamba_prefill", c_int32, [c_void_p, c_int32, POINTER(c_int32), c_void_p, c_void_p,
                                   c_void_p]),
    ("ll_mamba_decode_step", c_int32, [c_void_p, c_void_p, c_void_p, c_void_p]),
    ("ll_mamba_reset", c_int32, [c_void_p]),
    ("ll_mamba_seq_lengths", c_int32, [c_void_p, POINTER(c_int32), c_int32, POINTER(c_int32)]),
    ("ll_mamba_set_option", c_int32, [c_void_p, c_int32, c_int32]),
    ("ll_mamba_get_option", c_int32, [c_void_p, c_int32, POINTER(c_int32)]),
    ("ll_mamba_device_flags", c_int32, [c_void_p, POINTER(c_int32)]),
    ("ll_mamba_set_kernel_timing", c_int32, [c_void_p, c_int32]),
    ("ll_mamba_kernel_timing_read", c_int32, [c_void_p, POINTER(c_int32), POINTER(c_double)]),
    ("ll_mamba_kernel_class_name", c_char_p, [c_int32]),
    ("ll_mamba_free", None, [c_void_p]),
    ("ll_mamba2_workspace_size", c_int32, [POINTER(LLMamba2Config), POINTER(c_size_t)]),
    ("ll_mamba2_load", c_int32, [POINTER(LLMamba2Config), POINTER(LLMamba2Weights), c_void_p,
                                 c_size_t, c_void_p, POINTER(c_void_p)]),
    ("ll_mamba2_prefill", c_int32, [c_void_p, c_int32, POINTER(c_int32), c_void_p, c_void_p,
                                    c_void_p]),
    ("ll_mamba2_decode_step", c_int32, [c_void_p, c_void_p, c_void_p, c_void_p]),
    ("ll_mamba2_reset", c_int32, [c_void_p]),
    ("ll_mamba2_seq_lengths", c_int32, [c_void_p, POINTER(c_int32), c_int32, POINTER(c_int32)]),
    ("ll_mamba2_set_option", c_int32, [c_void_p, c_int32, c_int32]),
    ("ll_mamba2_get_option", c_int32, [c_void_p, c_int32, POINTER(c_int32)]),
    ("ll_mamba2_device_flags", c_int32, [c_void_p, POINTER(c_int32)]),
    ("ll_mamba2_set_kernel_timing", c_int32, [c_void_p, c_int32]),
    ("ll_mamba2_kernel_timing_read", c_int32, [c_void_p, POINTER(c_int32), POINTER(c_double)]),
    ("ll_mamba2_kernel_class_name", c_char_p, [c_int32]),
    ("ll_mamba2_free", None, [c_void_p]),
    ("ll_rg_workspace_size", c_int32, [POINTER(LLRGConfig), POINTER(c_size_t)]),
    ("ll_rg_load", c_int32, [POINTER(LLRGConfig), POINTER(LLRGWeights), c_void_p, c_size_t,
                             c_void_p, POINTER(c_void_p)]),
    ("ll_rg_prefill", c_int32, [c_void_p, c_int32, POINTER(c_int32), c_void_p, c_void_p,
                                c_void_p]),
    ("ll_rg_decode_step", c_int32, [c_void_p, c_void_p, c_void_p, c_void_p]),
    ("ll_rg_reset", c_int32, [c_void_p]),
    ("ll_rg_seq_lengths", c_int32, [c_void_p, POINTER(c_int32), c_int32, POINTER(c_int32)]),
    ("ll_rg_set_option", c_int32, [c_void_p, c_int32, c_int32]),
    ("ll_rg_get_option", c_int32, [c_void_p, c_int32, POINTER(c_int32)]),
    ("ll_rg_device_flags", c_int32, [c_void_p, POINTER(c_int32)]),
    ("ll_rg_set_kernel_timing", c_int32, [c_void_p, c_int32]),
    ("ll_rg_kernel_timing_read", c_int32, [c_void_p, POINTER(c_int32), POINTER(c_double)]),
    ("ll_rg_kernel_class_name", c_char_p, [c_int32]),
    ("ll_rg_free", None, [c_void_p]),
]

_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libll.so (built by paper_2608_21836_amd.build); raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} not found: build it with `python -m paper_2608_21836_amd.build`")
    lib = ctypes.CDLL(path)
    for name, res, args in SIGNATURES:
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


class LLError(RuntimeError):
    def __init__(self, status: int, where: str, message: str):
        self.status = status
        self.message = message
        super().__init__(f"{where}: {STATUS_NAMES[status] if 0 <= status < 7 else status}: {message}")


def _check(status: int, where: str) -> None:
    if status != LL_OK:
        msg = load_library().ll_last_error()
        raise LLError(status, where, msg.decode() if msg else "")


def make_config(cfg, max_batch: int, max_prefill_tokens: int, max_ctx: int, kv_page: int = 0,
                kv_pages: int = 0, f16_compute: Optional[bool] = None) -> LLConfig:
    """LLConfig from a synth.configs.ModelConfig-like object (kv_page > 0: paged cache).
    f16_compute (bf16 weights only): fp16 operands, the default for bf16 weights."""
    bf16 = cfg.dtype == "bf16"
    f16 = bf16 if f16_compute is None else bool(f16_compute)
    return LLConfig(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim,
                    cfg.ffn_dim, cfg.vocab, float(cfg.rms_eps), float(cfg.rope_theta),
                    LL_BF16 if bf16 else LL_F32, max_batch, max_prefill_tokens,
                    max_ctx, kv_page, kv_pages, 1 if f16 else 0)


def workspace_size(cfg: LLConfig) -> int:
    n = c_size_t(0)
    _check(load_library().ll_workspace_size(ctypes.byref(cfg), ctypes.byref(n)), "ll_workspace_size")
    return n.value


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream_handle(stream) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


class Model:
    """One loaded model: workspace (a torch uint8 tensor), handle and stream.

    ``weights`` maps synth.gen tensor names to CUDA tensors of the config's dtype.
    """

    def __init__(self, cfg, weights: Dict[str, "object"], max_batch: int,
                 max_prefill_tokens: int, max_ctx: int, stream=None, kv_page: int = 0,
                 kv_pages: int = 0, guard_bytes: int = 0, f16_compute: Optional[bool] = None):
        """guard_bytes (a multiple of 256): extra bytes allocated before and after the
        workspace (self.guarded), for checks that nothing is written outside it."""
        import torch
        self.lib = load_library()
        self.mcfg = cfg
        self.cfg = make_config(cfg, max_batch, max_prefill_tokens, max_ctx, kv_page, kv_pages,
                               f16_compute)
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        nbytes = workspace_size(self.cfg)
        if guard_bytes % 256:
            raise ValueError("guard_bytes must be a multiple of 256")
        self.guarded = torch.empty(nbytes + 2 * guard_bytes, dtype=torch.uint8, device="cuda")
        self.workspace = self.guarded[guard_bytes:guard_bytes + nbytes]
        nl = cfg.n_layers

        def arr(key):
            a = (c_void_p * nl)(*[weights[f"layers.{i}.{key}"].data_ptr() for i in range(nl)])
            return ctypes.cast(a, POINTER(c_void_p)), a

        keep = []
        fields = {}
        for key in ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down"):
            p, a = arr(key)
            keep.append(a)
            fields[key] = p
        w = LLWeights(weights["embed"].data_ptr(), weights["final_norm"].data_ptr(),
                      weights["lm_head"].data_ptr(), **fields)
        handle = c_void_p()
        _check(self.lib.ll_model_load(ctypes.byref(self.cfg), ctypes.byref(w),
                                      self.workspace.data_ptr(), nbytes,
                                      self.stream.cuda_stream, ctypes.byref(handle)),
               "ll_model_load")
        self.handle = handle
        self.batch = 0

    def close(self) -> None:
        if getattr(self, "handle", None):
            self.lib.ll_model_free(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def prefill(self, seq_lens: Sequence[int], tokens, next_tokens=None, logits=None):
        """tokens: int32 CUDA tensor of sum(seq_lens) ids.  Returns (next_tokens, logits)."""
        import torch
        b = len(seq_lens)
        lens = (c_int32 * b)(*[int(x) for x in seq_lens])
        if next_tokens is None:
            next_tokens = torch.empty(b, dtype=torch.int32, device="cuda")
        _check(self.lib.ll_prefill(self.handle, b, lens, tokens.data_ptr(), next_tokens.data_ptr(),
                                   _ptr(logits)), "ll_prefill")
        self.batch = b
        return next_tokens, logits

    def decode_step(self, in_tokens, next_tokens=None, logits=None):
        import torch
        if next_tokens is None:
            next_tokens = torch.empty(self.batch, dtype=torch.int32, device="cuda")
        _check(self.lib.ll_decode_step(self.handle, in_tokens.data_ptr(), next_tokens.data_ptr(),
                                       _ptr(logits)), "ll_decode_step")
        return next_tokens, logits

    def kv_reset(self) -> None:
        _check(self.lib.ll_kv_reset(self.handle), "ll_kv_reset")
        self.batch = 0

    def set_decode_graph(self, enable: bool) -> None:
        _check(self.lib.ll_set_decode_graph(self.handle, 1 if enable else 0), "ll_set_decode_graph")

    def set_option(self, name: str, value: int) -> None:
        _check(self.lib.ll_set_option(self.handle, OPTIONS[name], int(value)), "ll_set_option")

    def get_option(self, name: str) -> int:
        v = c_int32(0)
        _check(self.lib.ll_get_option(self.handle, OPTIONS[name], ctypes.byref(v)), "ll_get_option")
        return v.value

    def options(self) -> Dict[str, int]:
        return {k: self.get_option(k) for k in DECODER_OPTIONS}

    def regions(self) -> List[Tuple[str, int, int]]:
        """[(name, byte offset in the workspace, bytes)] of the workspace layout."""
        n = c_int32(0)
        _check(self.lib.ll_workspace_regions(self.handle, 0, None, None, None, ctypes.byref(n)),
               "ll_workspace_regions")
        cap = n.value
        off, nb, names = (c_uint64 * cap)(), (c_uint64 * cap)(), (c_char_p * cap)()
        _check(self.lib.ll_workspace_regions(self.handle, cap, off, nb, names, ctypes.byref(n)),
               "ll_workspace_regions")
        return [(names[i].decode(), int(off[i]), int(nb[i])) for i in range(cap)]

    def seq_lengths(self) -> List[int]:
        out = (c_int32 * LL_MAX_BATCH)()
        n = c_int32(0)
        _check(self.lib.ll_seq_lengths(self.handle, out, LL_MAX_BATCH, ctypes.byref(n)), "ll_seq_lengths")
        return list(out[:n.value])

    def kv_pages(self) -> Tuple[int, int]:
        """(pages held by the current sequences, pages in the pool); (0, 0) when contiguous."""
        used, total = c_int32(0), c_int32(0)
        _check(self.lib.ll_kv_pages(self.handle, ctypes.byref(used), ctypes.byref(total)),
               "ll_kv_pages")
        return used.value, total.value

    def set_kernel_timing(self, enable: bool) -> None:
        _check(self.lib.ll_set_kernel_timing(self.handle, 1 if enable else 0), "ll_set_kernel_timing")

    def kernel_timing(self) -> Dict[Tuple[str, str], Tuple[int, float]]:
        """{(phase, kernel class): (launches, summed kernel ms)} since the last read."""
        counts = (c_int32 * (2 * LL_K_COUNT))()
        ms = (c_double * (2 * LL_K_COUNT))()
        _check(self.lib.ll_kernel_timing_read(self.handle, counts, ms), "ll_kernel_timing_read")
        out = {}
        for p in range(2):
            for c in range(LL_K_COUNT):
                i = p * LL_K_COUNT + c
                if counts[i]:
                    name = self.lib.ll_kernel_class_name(c).decode()
                    out[(PHASES[p], name)] = (counts[i], ms[i])
        return out

    def device_flags(self) -> int:
        f = c_int32(0)
        _check(self.lib.ll_device_flags(self.handle, ctypes.byref(f)), "ll_device_flags")
        return f.value


def make_mamba_config(cfg, max_batch: int, max_prefill_tokens: int) -> LLMambaConfig:
    """LLMambaConfig from a synth.mamba.MambaConfig-like object."""
    return LLMambaConfig(cfg.n_layers, cfg.d_model, cfg.d_inner, cfg.d_state, cfg.d_conv,
                         cfg.dt_rank, cfg.vocab, float(cfg.rms_eps),
                         LL_BF16 if cfg.dtype == "bf16" else LL_F32, max_batch, max_prefill_tokens)


def mamba_workspace_size(cfg: LLMambaConfig) -> int:
    n = c_size_t(0)
    _check(load_library().ll_mamba_workspace_size(ctypes.byref(cfg), ctypes.byref(n)),
           "ll_mamba_workspace_size")
    return n.value


def make_mamba2_config(cfg, max_batch: int, max_prefill_tokens: int) -> LLMamba2Config:
    """LLMamba2Config from a synth.mamba2.Mamba2Config-like object."""
    return LLMamba2Config(cfg.n_layers, cfg.d_model, cfg.d_inner, cfg.d_state, cfg.head_dim,
                          cfg.n_groups, cfg.d_conv, cfg.vocab, float(cfg.rms_eps),
                          LL_BF16 if cfg.dtype == "bf16" else LL_F32, max_batch,
                          max_prefill_tokens)


def make_rg_config(cfg, max_batch: int, max_prefill_tokens: int) -> LLRGConfig:
    """LLRGConfig from a synth.rglru.RGConfig-like object."""
    return LLRGConfig(cfg.n_layers, cfg.d_model, cfg.lru_width, cfg.n_heads, cfg.mlp_width,
                      cfg.d_conv, cfg.vocab, float(cfg.rms_eps), float(cfg.embed_scale),
                      float(cfg.logit_cap), LL_BF16 if cfg.dtype == "bf16" else LL_F32,
                      max_batch, max_prefill_tokens)


# per state-space family: (entry-point prefix, config maker, weight struct, per-layer fields,
# fp32 fields, kernel class count, option names)
_FAMILIES = {
    "mamba": ("ll_mamba_", make_mamba_config, "LLMambaWeights", "MAMBA_LAYER_FIELDS",
              "MAMBA_F32_FIELDS", "LL_MK_COUNT", "MAMBA_OPTIONS"),
    "mamba2": ("ll_mamba2_", make_mamba2_config, "LLMamba2Weights", "MAMBA2_LAYER_FIELDS",
               "MAMBA2_F32_FIELDS", "LL_M2K_COUNT", "MAMBA2_OPTIONS"),
    "rglru": ("ll_rg_", make_rg_config, "LLRGWeights", "RG_LAYER_FIELDS", "RG_F32_FIELDS",
              "LL_RGK_COUNT", "RG_OPTIONS"),
}


class MambaModel:
    """One loaded state-space model of family cfg.family ("mamba", "mamba2" or "rglru"):
    workspace (a torch uint8 tensor), handle and stream.  The families differ only in the C
    entry points' prefix (ll_mamba_* / ll_mamba2_* / ll_rg_*), the config and weight structs,
    the kernel classes and the options that apply.

    ``weights`` maps synth.mamba / synth.mamba2 / synth.rglru tensor names to CUDA tensors
    (upload_mamba_weights)."""

    def __init__(self, cfg, weights: Dict[str, "object"], max_batch: int,
                 max_prefill_tokens: int, stream=None):
        import torch
        self.lib = load_library()
        self.mcfg = cfg
        self.family = getattr(cfg, "family", "mamba")
        self.v2 = self.family == "mamba2"
        prefix, make_cfg, wstruct, lfields, _, ncls, opts = _FAMILIES[self.family]
        g = globals()
        self.prefix = prefix
        self.n_classes = g[ncls]
        self.option_names = g[opts]
        self.cfg = make_cfg(cfg, max_batch, max_prefill_tokens)
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        n = c_size_t(0)
        _check(self._fn("workspace_size")(ctypes.byref(self.cfg), ctypes.byref(n)),
               self.prefix + "workspace_size")
        nbytes = n.value
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        nl = cfg.n_layers
        keep, fields = [], {}
        for key in g[lfields]:
            a = (c_void_p * nl)(*[weights[f"layers.{i}.{key}"].data_ptr() for i in range(nl)])
            keep.append(a)
            fields[key] = ctypes.cast(a, POINTER(c_void_p))
        W = g[wstruct]
        w = W(weights["embed"].data_ptr(), weights["final_norm"].data_ptr(), **fields)
        handle = c_void_p()
        _check(self._fn("load")(ctypes.byref(self.cfg), ctypes.byref(w), self.workspace.data_ptr(),
                                nbytes, self.stream.cuda_stream, ctypes.byref(handle)),
               self.prefix + "load")
        self.handle = handle
        self.batch = 0

    def _fn(self, name):
        return getattr(self.lib, self.prefix + name)

    def close(self) -> None:
        if getattr(self, "handle", None):
            self._fn("free")(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def prefill(self, seq_lens: Sequence[int], tokens, next_tokens=None, logits=None):
        import torch
        b = len(seq_lens)
        lens = (c_int32 * b)(*[int(x) for x in seq_lens])
        if next_tokens is None:
            next_tokens = torch.empty(b, dtype=torch.int32, device="cuda")
        _check(self._fn("prefill")(self.handle, b, lens, tokens.data_ptr(),
                                   next_tokens.data_ptr(), _ptr(logits)), self.prefix + "prefill")
        self.batch = b
        return next_tokens, logits

    def decode_step(self, in_tokens, next_tokens=None, logits=None):
        import torch
        if next_tokens is None:
            next_tokens = torch.empty(self.batch, dtype=torch.int32, device="cuda")
        _check(self._fn("decode_step")(self.handle, in_tokens.data_ptr(),
                                       next_tokens.data_ptr(), _ptr(logits)),
               self.prefix + "decode_step")
        return next_tokens, logits

    def reset(self) -> None:
        _check(self._fn("reset")(self.handle), self.prefix + "reset")
        self.batch = 0

    kv_reset = reset  # same call name as the decoder's (forget every held sequence)

    def set_option(self, name: str, value: int) -> None:
        _check(self._fn("set_option")(self.handle, OPTIONS[name], int(value)),
               self.prefix + "set_option")

    def get_option(self, name: str) -> int:
        v = c_int32(0)
        _check(self._fn("get_option")(self.handle, OPTIONS[name], ctypes.byref(v)),
               self.prefix + "get_option")
        return v.value

    def options(self) -> Dict[str, int]:
        return {k: self.get_option(k) for k in self.option_names}

    def regions(self) -> List[Tuple[str, int, int]]:
        """[(name, byte offset in the workspace, bytes)] of the workspace layout."""
        n = c_int32(0)
        _check(self.lib.ll_workspace_regions(self.handle, 0, None, None, None, ctypes.byref(n)),
               "ll_workspace_regions")
        cap = n.value
        off, nb, names = (c_uint64 * cap)(), (c_uint64 * cap)(), (c_char_p * cap)()
        _check(self.lib.ll_workspace_regions(self.handle, cap, off, nb, names, ctypes.byref(n)),
               "ll_workspace_regions")
        return [(names[i].decode(), int(off[i]), int(nb[i])) for i in range(cap)]

    def seq_lengths(self) -> List[int]:
        out = (c_int32 * LL_MAX_BATCH)()
        n = c_int32(0)
        _check(self._fn("seq_lengths")(self.handle, out, LL_MAX_BATCH, ctypes.byref(n)),
               self.prefix + "seq_lengths")
        return list(out[:n.value])

    def set_kernel_timing(self, enable: bool) -> None:
        _check(self._fn("set_kernel_timing")(self.handle, 1 if enable else 0),
               self.prefix + "set_kernel_timing")

    def kernel_timing(self) -> Dict[Tuple[str, str], Tuple[int, float]]:
        """{(phase, kernel class): (launches, summed kernel ms)} since the last read."""
        nc = self.n_classes
        counts = (c_int32 * (2 * nc))()
        ms = (c_double * (2 * nc))()
        _check(self._fn("kernel_timing_read")(self.handle, counts, ms),
               self.prefix + "kernel_timing_read")
        out = {}
        for p in range(2):
            for c in range(nc):
                i = p * nc + c
                if counts[i]:
                    name = self._fn("kernel_class_name")(c).decode()
                    out[(PHASES[p], name)] = (counts[i], ms[i])
        return out

    def device_flags(self) -> int:
        f = c_int32(0)
        _check(self._fn("device_flags")(self.handle, ctypes.byref(f)), self.prefix + "device_flags")
        return f.value


# ------------------------------------------------------------------------------------------
# Weights: numpy (synth.gen) -> CUDA tensors of the workload dtype
# ------------------------------------------------------------------------------------------

def to_device(arr, dtype: str):
    """fp32 numpy array (bf16-exact for bf16 workloads) -> CUDA tensor of the storage type."""
    import numpy as np
    import torch
    if dtype == "bf16":
        bits = (np.ascontiguousarray(arr, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)
        return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()
    if dtype == "f16":
        return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float16)).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).cuda()


def upload_weights(cfg, weights) -> Dict[str, "object"]:
    return {k: to_device(v, cfg.dtype) for k, v in weights.items()}


def upload_mamba_weights(cfg, weights) -> Dict[str, "object"]:
    """Mamba / Mamba2 / RG-LRU tensors: the small per-channel / per-head ones (conv, dt,
    A_log, D; biases and lambda) in fp32, the rest in the workload dtype."""
    f32 = globals()[_FAMILIES[getattr(cfg, "family", "mamba")][4]]
    out = {}
    for k, v in weights.items():
        out[k] = to_device(v, "f32" if k.rsplit(".", 1)[-1] in f32 else cfg.dtype)
    return out


# ------------------------------------------------------------------------------------------
# Per-kernel entry points (isolated qualification)
# ------------------------------------------------------------------------------------------

def _dt(t) -> int:
    import torch
    return {torch.bfloat16: LL_BF16, torch.float16: LL_F16}.get(t.dtype, LL_F32)


def op_mfma_loop(blocks: int, iters: int, out=None, stream=None):
    """Calibration MFMA loop (ll_op_mfma_loop); returns the fp32 output tensor."""
    import torch
    if out is None:
        out = torch.empty(4 * blocks, dtype=torch.float32, device="cuda")
    _check(load_library().ll_op_mfma_loop(blocks, iters, out.data_ptr(), _stream_handle(stream)),
           "ll_op_mfma_loop")
    return out


def op_read_stream(src, blocks: int, out=None, stream=None):
    """Calibration read stream over an fp32 device tensor (ll_op_read_stream); returns the
    per-block sums."""
    import torch
    if out is None:
        out = torch.empty(blocks, dtype=torch.float32, device="cuda")
    _check(load_library().ll_op_read_stream(src.data_ptr(), src.numel(), blocks, out.data_ptr(),
                                            _stream_handle(stream)), "ll_op_read_stream")
    return out


def op_rmsnorm(x, gain, eps: float, stream=None):
    import torch
    y = torch.empty(x.shape, dtype=gain.dtype, device="cuda")
    _check(load_library().ll_op_rmsnorm(_dt(gain), x.shape[0], x.shape[1], x.data_ptr(),
                                        gain.data_ptr(), eps, y.data_ptr(), _stream_handle(stream)),
           "ll_op_rmsnorm")
    return y


def op_repack(w, stream=None):
    import torch
    wt = torch.empty(w.numel() * w.element_size(), dtype=torch.uint8, device="cuda")
    _check(load_library().ll_op_repack(_dt(w), w.shape[0], w.shape[1], w.data_ptr(), wt.data_ptr(),
                                       _stream_handle(stream)), "ll_op_repack")
    return wt


def op_gemm(path: int, a, wt, n: int, c=None, accumulate: bool = False, stream=None):
    import torch
    m, k = a.shape
    if c is None:
        c = torch.empty(m, n, dtype=torch.float32, device="cuda")
    _check(load_library().ll_op_gemm(path, _dt(a), m, n, k, a.data_ptr(), wt.data_ptr(),
                                     c.data_ptr(), 1 if accumulate else 0, _stream_handle(stream)),
           "ll_op_gemm")
    return c


def op_gemm_splitk(a, wt, n: int, c=None, accumulate: bool = False, stream=None):
    """Split-K decode GEMM (more than 16 rows); scratch is allocated here."""
    import torch
    m, k = a.shape
    lib = load_library()
    nbytes = lib.ll_op_gemm_splitk_scratch(_dt(a), m, n, k)
    if c is None:
        c = torch.empty(m, n, dtype=torch.float32, device="cuda")
    scratch = torch.empty(max(nbytes, 1), dtype=torch.uint8, device="cuda")
    _check(lib.ll_op_gemm_splitk(_dt(a), m, n, k, a.data_ptr(), wt.data_ptr(), c.data_ptr(),
                                 1 if accumulate else 0, scratch.data_ptr(), nbytes,
                                 _stream_handle(stream)), "ll_op_gemm_splitk")
    return c


def op_gemm_prefill_splitk(a, wt, n: int, c=None, accumulate: bool = False, stream=None):
    """Split-K prefill GEMM (short prompts); scratch is allocated here."""
    import torch
    m, k = a.shape
    lib = load_library()
    nbytes = lib.ll_op_gemm_prefill_splitk_scratch(_dt(a), m, n, k)
    if c is None:
        c = torch.empty(m, n, dtype=torch.float32, device="cuda")
    scratch = torch.empty(max(nbytes, 1), dtype=torch.uint8, device="cuda")
    _check(lib.ll_op_gemm_prefill_splitk(_dt(a), m, n, k, a.data_ptr(), wt.data_ptr(),
                                         c.data_ptr(), 1 if accumulate else 0,
                                         scratch.data_ptr(), nbytes, _stream_handle(stream)),
           "ll_op_gemm_prefill_splitk")
    return c


def op_attn_prefill(seq_lens, q, kcache, vcache, n_heads, n_kv_heads, head_dim, max_ctx,
                    stream=None, cached=None):
    """cached[b]: keys already in the cache before sequence b's queries (default 0)."""
    import torch
    b = len(seq_lens)
    lens = (c_int32 * b)(*[int(x) for x in seq_lens])
    starts = (c_int32 * b)(*[int(x) for x in cached]) if cached is not None else None
    o = torch.empty_like(q)
    nbytes = load_library().ll_op_attn_prefill_scratch(_dt(q), b, lens, starts, n_heads,
                                                       n_kv_heads, head_dim, max_ctx)
    if nbytes == 0:
        raise LLError(1, "ll_op_attn_prefill_scratch", "invalid arguments")
    scratch = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    _check(load_library().ll_op_attn_prefill(_dt(q), b, lens, starts, n_heads, n_kv_heads,
                                             head_dim, max_ctx, q.data_ptr(), kcache.data_ptr(),
                                             vcache.data_ptr(), o.data_ptr(), scratch.data_ptr(),
                                             nbytes, _stream_handle(stream)), "ll_op_attn_prefill")
    return o


def op_attn_decode(q, kcache, vcache, ctx_lens, n_heads, n_kv_heads, head_dim, max_ctx,
                   stream=None):
    import torch
    lib = load_library()
    b = q.shape[0]
    nbytes = lib.ll_op_attn_decode_scratch(b, n_heads, n_kv_heads, head_dim, max_ctx)
    scratch = torch.empty(max(nbytes, 256), dtype=torch.uint8, device="cuda")
    o = torch.empty_like(q)
    _check(lib.ll_op_attn_decode(_dt(q), b, n_heads, n_kv_heads, head_dim, max_ctx, q.data_ptr(),
                                 kcache.data_ptr(), vcache.data_ptr(), ctx_lens.data_ptr(),
                                 o.data_ptr(), scratch.data_ptr(), nbytes, _stream_handle(stream)),
           "ll_op_attn_decode")
    return o


def op_gemm_swiglu(a, wt, n: int, act=None, stream=None):
    """ll_op_gemm_swiglu: act [M, n/2] (a's dtype) from the prefill GEMM with the SwiGLU
    epilogue; wt repacked from gate/up rows interleaved in blocks of 16."""
    import torch
    m, k = a.shape
    if act is None:
        act = torch.empty(m, n // 2, dtype=a.dtype, device="cuda")
    _check(load_library().ll_op_gemm_swiglu(_dt(a), m, n, k, a.data_ptr(), wt.data_ptr(),
                                            act.data_ptr(), _stream_handle(stream)),
           "ll_op_gemm_swiglu")
    return act


def op_lmhead_argmax(h, wt, vocab: int, want_logits: bool = True, stream=None):
    import torch
    rows, k = h.shape
    logits = torch.empty(rows, vocab, dtype=torch.float32, device="cuda") if want_logits else None
    nxt = torch.empty(rows, dtype=torch.int32, device="cuda")
    nbytes = 8 * rows * (vocab // 32)
    scratch = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    _check(load_library().ll_op_lmhead_argmax(_dt(h), rows, vocab, k, h.data_ptr(), wt.data_ptr(),
                                              _ptr(logits), nxt.data_ptr(), scratch.data_ptr(),
                                              nbytes, _stream_handle(stream)), "ll_op_lmhead_argmax")
    return nxt, logits


def op_lmhead_argmax_noalloc(h, wt, vocab: int, logits=None, nxt=None, stream=None):
    """ll_op_lmhead_argmax_noalloc: the LM head with fused argmax, partials in the library's
    static device array (nothing allocated by the library).  logits / nxt: caller tensors
    (logits nullable)."""
    rows, k = h.shape
    _check(load_library().ll_op_lmhead_argmax_noalloc(_dt(h), rows, vocab, k, h.data_ptr(),
                                                      wt.data_ptr(), _ptr(logits),
                                                      nxt.data_ptr(), _stream_handle(stream)),
           "ll_op_lmhead_argmax_noalloc")
    return nxt, logits
