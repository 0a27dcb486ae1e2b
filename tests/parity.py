"""Shared helpers for the GPU parity tests: running a workload through the C ABI and judging
it against the oracle.

Acceptance rules:
  * fp32 workloads: every compared logit within 1e-4 of the oracle, and the greedy token equal
    to the oracle's wherever the oracle's top-2 margin is >= 1e-3.
  * bf16 workloads: per compared row (sequence x step) max |gpu - oracle| <= 2e-2 * (oracle
    row max - row min).  Greedy-token disagreements at margin >= 1e-3 ("literal" mismatches)
    are counted and reported with their margins.  Each must be explained by precision: the
    two competing logits (the oracle's choice and the GPU's) carry errors no larger than
    ERR_OUTLIER times the row's root-mean-square logit error, i.e. the flip comes from the
    same rounding noise that moves every logit of the row, not from an error that singles out
    the top of the row.  (A flip needs e_gpu - e_oracle >= margin, so this also bounds the
    margin of an accepted flip by 2 * ERR_OUTLIER * rms.)
Rows compared: the prefill logits at each sequence's last prompt position and every
teacher-forced decode step (both sides consume the oracle's tokens).
"""
from __future__ import annotations

import dataclasses
import sys
from typing import List

import numpy as np

from synth import gen


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


ERR_OUTLIER = 4.0


@dataclasses.dataclass
class ParityReport:
    name: str
    rows: int
    max_abs_err: float
    worst_rel_row_err: float
    literal_mismatches: int
    unexplained_mismatches: int
    details: List[str]

    def ok(self, dtype: str, quant: float = 0.0) -> bool:
        """quant: relative error of stored reference logits (per unit of row range), taken off
        the bf16 bar so that a stored reference never loosens it."""
        if dtype == "f32":
            return self.max_abs_err <= 1e-4 and self.literal_mismatches == 0
        return self.worst_rel_row_err <= 2e-2 - quant and self.unexplained_mismatches == 0


def judge(name: str, dtype: str, ref_logits: np.ndarray, gpu_logits: np.ndarray,
          gpu_tokens: np.ndarray, ref_margin=None, ref_tokens=None) -> ParityReport:
    """ref/gpu logits [steps, B, V]; gpu_tokens [steps, B] (the library's fused argmax).
    ref_margin / ref_tokens: the oracle's fp64 top-2 margins and greedy tokens, when the
    reference logits are a stored (rounded) copy; computed from ref_logits otherwise."""
    ref = ref_logits.astype(np.float64)
    gpu = gpu_logits.astype(np.float64)
    err = np.abs(gpu - ref)
    row_err = err.max(axis=-1)
    row_range = ref.max(axis=-1) - ref.min(axis=-1)
    if ref_margin is None:
        part = np.partition(ref, -2, axis=-1)
        margin = part[..., -1] - part[..., -2]
    else:
        margin = np.asarray(ref_margin, dtype=np.float64)
    ref_tok = np.argmax(ref, axis=-1) if ref_tokens is None else np.asarray(ref_tokens)
    # the library's fused argmax must agree bitwise with an argmax over its own logits
    own = np.argmax(gpu_logits, axis=-1)
    assert np.array_equal(own, gpu_tokens), f"{name}: fused argmax disagrees with its logits"
    mism = (gpu_tokens != ref_tok) & (margin >= 1e-3)
    row_rms = np.sqrt(np.mean((gpu - ref) ** 2, axis=-1))
    details, unexplained = [], 0
    for s, b in zip(*np.nonzero(mism)):
        i, j = ref_tok[s, b], gpu_tokens[s, b]
        e_i, e_j = gpu[s, b, i] - ref[s, b, i], gpu[s, b, j] - ref[s, b, j]
        explained = max(abs(e_i), abs(e_j)) <= ERR_OUTLIER * row_rms[s, b]
        unexplained += int(not explained)
        details.append(f"step {s} seq {b}: oracle {i} gpu {j} margin {margin[s, b]:.3e} "
                       f"errors {e_i:+.3e} / {e_j:+.3e} row rms err {row_rms[s, b]:.3e} "
                       f"{'precision-explained' if explained else 'UNEXPLAINED'}")
    return ParityReport(name, int(np.prod(row_err.shape)), float(err.max()),
                        float((row_err / row_range).max()), int(mism.sum()), unexplained, details)


def run_gpu_teacher_forced(cfg, weights, lens, packed, ref_tokens, n_decode, use_graph=True,
                           options=None, paging=None, f16_compute=None):
    """Prefill + n_decode teacher-forced steps through the C ABI, with the given ll_option
    values (name -> value) set after loading.

    Returns (logits [n_decode + 1, B, V] fp32, tokens [n_decode + 1, B])."""
    import torch
    from paper_2608_21836_amd.binding import Model, upload_weights
    B = len(lens)
    dev_w = upload_weights(cfg, weights)
    model = Model(cfg, dev_w, max_batch=B, max_prefill_tokens=int(sum(lens)),
                  max_ctx=int(max(lens)) + n_decode, f16_compute=f16_compute, **(paging or {}))
    del dev_w
    model.set_decode_graph(use_graph)
    for name, value in (options or {}).items():
        model.set_option(name, value)
    toks = torch.from_numpy(np.asarray(packed, dtype=np.int32)).cuda()
    logits = torch.empty(B, cfg.vocab, dtype=torch.float32, device="cuda")
    nxt = torch.empty(B, dtype=torch.int32, device="cuda")
    out_l, out_t = [], []
    model.prefill(lens, toks, nxt, logits)
    torch.cuda.synchronize()
    out_l.append(logits.cpu().numpy().copy())
    out_t.append(nxt.cpu().numpy().copy())
    inp = torch.empty(B, dtype=torch.int32, device="cuda")
    for k in range(1, n_decode + 1):
        inp.copy_(torch.from_numpy(np.asarray(ref_tokens[k - 1], dtype=np.int32)))
        model.decode_step(inp, nxt, logits)
        torch.cuda.synchronize()
        out_l.append(logits.cpu().numpy().copy())
        out_t.append(nxt.cpu().numpy().copy())
    assert model.seq_lengths() == [int(x) + n_decode for x in lens]
    assert model.device_flags() == 0
    model.close()
    return np.stack(out_l), np.stack(out_t)


def chunk_prompts(prompts, n_chunks):
    """Each prompt cut into n_chunks consecutive pieces of near-equal length (each >= 1)."""
    out = []
    for i in range(n_chunks):
        out.append([np.array_split(np.asarray(p), n_chunks)[i] for p in prompts])
    return out


def oracle_chunked_run(model, chunks, n_decode):
    """Oracle: prefill of the first chunks, extend by the others, then n_decode teacher-forced
    greedy steps.  Returns (logits [n_chunks + n_decode, B, V], tokens)."""
    from oracle import argmax_lowest
    logits = [model.prefill(chunks[0])] + [model.extend(c) for c in chunks[1:]]
    toks = [argmax_lowest(lg) for lg in logits]
    for _ in range(n_decode):
        logits.append(model.decode(toks[-1]))
        toks.append(argmax_lowest(logits[-1]))
    return np.stack(logits), np.stack(toks)


def run_gpu_chunked(cfg, weights, chunks, ref_tokens, n_decode, options=None, paging=None):
    """The same through the C ABI: one ll_prefill per chunk (the later ones on the populated
    cache), then decode steps fed the oracle's tokens."""
    import torch
    from paper_2608_21836_amd.binding import Model, upload_weights
    B = len(chunks[0])
    total = [sum(len(c[b]) for c in chunks) for b in range(B)]
    dev_w = upload_weights(cfg, weights)
    model = Model(cfg, dev_w, max_batch=B, max_prefill_tokens=max(sum(len(x) for x in c) for c in chunks),
                  max_ctx=max(total) + n_decode, **(paging or {}))
    del dev_w
    for name, value in (options or {}).items():
        model.set_option(name, value)
    logits = torch.empty(B, cfg.vocab, dtype=torch.float32, device="cuda")
    nxt = torch.empty(B, dtype=torch.int32, device="cuda")
    out_l, out_t = [], []
    for c in chunks:
        toks = torch.from_numpy(np.concatenate(c).astype(np.int32)).cuda()
        model.prefill([len(x) for x in c], toks, nxt, logits)
        torch.cuda.synchronize()
        out_l.append(logits.cpu().numpy().copy())
        out_t.append(nxt.cpu().numpy().copy())
    n_chunks = len(chunks)
    inp = torch.empty(B, dtype=torch.int32, device="cuda")
    for k in range(n_decode):
        inp.copy_(torch.from_numpy(np.asarray(ref_tokens[n_chunks - 1 + k], dtype=np.int32)))
        model.decode_step(inp, nxt, logits)
        torch.cuda.synchronize()
        out_l.append(logits.cpu().numpy().copy())
        out_t.append(nxt.cpu().numpy().copy())
    assert model.seq_lengths() == [t + n_decode for t in total]
    assert model.device_flags() == 0
    model.close()
    return np.stack(out_l), np.stack(out_t)


def device_tensor(arr, dtype):
    from paper_2608_21836_amd.binding import to_device
    return to_device(arr, dtype)


def rounded(arr, dtype):
    """The values a tensor of `dtype` holds (fp32 numpy)."""
    a = np.asarray(arr, dtype=np.float32)
    if dtype == "f16":
        return a.astype(np.float16).astype(np.float32)
    return gen.round_to_bf16(a) if dtype == "bf16" else a


def run_gpu_mamba(cfg, weights, chunks, ref_tokens, n_decode, use_graph=True, options=None):
    """A Mamba workload through the C ABI: one ll_mamba_prefill per prompt chunk (the later
    ones continue the held state), then n_decode decode steps fed the oracle's tokens
    (ref_tokens[len(chunks) - 1 + k] at step k).  Returns (logits [n_chunks + n_decode, B, V],
    tokens)."""
    import torch
    from paper_2608_21836_amd.binding import MambaModel, upload_mamba_weights
    B = len(chunks[0])
    dev_w = upload_mamba_weights(cfg, weights)
    model = MambaModel(cfg, dev_w, max_batch=B,
                       max_prefill_tokens=max(sum(len(x) for x in c) for c in chunks))
    del dev_w
    model.set_option("decode_graph", 1 if use_graph else 0)
    for name, value in (options or {}).items():
        model.set_option(name, value)
    logits = torch.empty(B, cfg.vocab, dtype=torch.float32, device="cuda")
    nxt = torch.empty(B, dtype=torch.int32, device="cuda")
    out_l, out_t = [], []
    for c in chunks:
        toks = torch.from_numpy(np.concatenate(c).astype(np.int32)).cuda()
        model.prefill([len(x) for x in c], toks, nxt, logits)
        torch.cuda.synchronize()
        out_l.append(logits.cpu().numpy().copy())
        out_t.append(nxt.cpu().numpy().copy())
    inp = torch.empty(B, dtype=torch.int32, device="cuda")
    for k in range(n_decode):
        inp.copy_(torch.from_numpy(np.asarray(ref_tokens[len(chunks) - 1 + k], dtype=np.int32)))
        model.decode_step(inp, nxt, logits)
        torch.cuda.synchronize()
        out_l.append(logits.cpu().numpy().copy())
        out_t.append(nxt.cpu().numpy().copy())
    total = [sum(len(c[b]) for c in chunks) for b in range(B)]
    assert model.seq_lengths() == [t + n_decode for t in total]
    assert model.device_flags() == 0
    model.close()
    return np.stack(out_l), np.stack(out_t)
