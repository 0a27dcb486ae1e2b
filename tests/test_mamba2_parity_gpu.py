"""Acceptance of the Mamba2 model: whole workloads through ll_mamba2_load / ll_mamba2_prefill /
ll_mamba2_decode_step, teacher-forced, against the fp64 oracle on the same seeded inputs
(acceptance rules in parity.py).  Covers ragged batches with one-token prompts, two B/C
groups, state sizes 32, 64, 128 and 256, prompts long enough for the chunked scan, six sequences,
fp32 and bf16, prefill continued on held state, graph and direct decode, split-K switches and
the full mamba2-130m workload."""
import numpy as np
import pytest

from oracle import argmax_lowest, split_prompts
from oracle.mamba2 import OracleMamba2, teacher_forced_run_mamba2
from parity import chunk_prompts, judge, log, run_gpu_mamba
from synth import gen
from synth import mamba2 as S2

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21836_amd.binding import load_library
    load_library()


def _report(name, dtype, ref_l, gl, gt):
    rep = judge(name, dtype, ref_l, gl, gt)
    log(f"mamba2 parity {name}: rows={rep.rows} max_abs={rep.max_abs_err:.3e} "
        f"worst_row_rel={rep.worst_rel_row_err:.3e} literal_mismatch={rep.literal_mismatches} "
        f"unexplained={rep.unexplained_mismatches}")
    for d in rep.details:
        log("  " + d)
    return rep


# (workload, graph replay, decode steps (None: the workload's), options)
CASES = [("t-mamba2", True, None, {}), ("t-mamba2", False, None, {}),
         ("t-mamba2-f32", True, None, {}), ("t-mamba2-f32", False, None, {"prefill_splitk": 0}),
         ("t-mamba2-long", True, None, {}),
         ("t-mamba2-long", False, None, {"decode_splitk": 0, "prefill_tile": 3}),
         ("t-mamba2-n32", True, None, {}), ("t-mamba2-n256", False, None, {}),
         ("t-mamba2-f32", True, None, {"decode_splitk": 2}),
         ("mamba2-130m", True, 16, {})]


@pytest.mark.parametrize("name,graph,n_decode,options", CASES,
                         ids=[f"{c[0]}-{'graph' if c[1] else 'direct'}"
                              + "".join(f"-{k}{v}" for k, v in c[3].items()) for c in CASES])
def test_mamba2_workload_parity(name, graph, n_decode, options):
    cfg = S2.get_mamba2_config(name)
    nd = n_decode if n_decode is not None else cfg.n_decode
    log(f"mamba2 parity {name}: oracle ...")
    w = S2.weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    ref_l, ref_t = teacher_forced_run_mamba2(OracleMamba2(cfg, w), lens, packed, nd)
    log(f"mamba2 parity {name}: gpu ...")
    gl, gt = run_gpu_mamba(cfg, w, [split_prompts(lens, packed)], ref_t, nd, use_graph=graph,
                           options=options)
    rep = _report(name, cfg.dtype, ref_l, gl, gt)
    assert rep.ok(cfg.dtype), rep


@pytest.mark.parametrize("name,n_chunks", [("t-mamba2", 3), ("t-mamba2-f32", 2),
                                           ("t-mamba2-long", 2)])
def test_mamba2_chunked_prefill_parity(name, n_chunks):
    cfg = S2.get_mamba2_config(name)
    if name == "t-mamba2":
        cfg = cfg.replace(prompt_list=(37, 4, 70))
    if name == "t-mamba2-long":
        cfg = cfg.replace(prompt_range=(8, 700))
    w = S2.weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    chunks = chunk_prompts(split_prompts(lens, packed), n_chunks)
    nd = 3
    om = OracleMamba2(cfg, w)
    ref_l = [om.prefill(chunks[0])] + [om.extend(c) for c in chunks[1:]]
    ref_t = [argmax_lowest(x) for x in ref_l]
    for _ in range(nd):
        ref_l.append(om.decode(ref_t[-1]))
        ref_t.append(argmax_lowest(ref_l[-1]))
    ref_l, ref_t = np.stack(ref_l), np.stack(ref_t)
    gl, gt = run_gpu_mamba(cfg, w, chunks, ref_t, nd)
    rep = _report(f"{name}-chunked", cfg.dtype, ref_l, gl, gt)
    assert rep.ok(cfg.dtype), rep


# The matrix-form prefill scan of 16-bit models at the shapes the other cases leave out:
# head dim 32 with state 256 and with state 128 (multi-chunk prompts, ragged last chunks).
@pytest.mark.parametrize("name", ["t-mamba2-n256", "t-mamba2-f32"])
def test_mamba2_matrix_scan_bf16(name):
    base = S2.get_mamba2_config(name)
    cfg = base.replace(name=f"{name}-bf16", dtype="bf16", head_dim=32, prompt_list=(40, 300))
    log(f"mamba2 parity {cfg.name}: oracle ...")
    w = S2.weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    ref_l, ref_t = teacher_forced_run_mamba2(OracleMamba2(cfg, w), lens, packed, cfg.n_decode)
    gl, gt = run_gpu_mamba(cfg, w, [split_prompts(lens, packed)], ref_t, cfg.n_decode,
                           use_graph=True, options={})
    rep = _report(cfg.name, cfg.dtype, ref_l, gl, gt)
    assert rep.ok(cfg.dtype), rep
