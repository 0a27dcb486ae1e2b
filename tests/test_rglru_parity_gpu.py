"""Acceptance of the RG-LRU (Griffin recurrent block) model: whole workloads through ll_rg_load /
ll_rg_prefill / ll_rg_decode_step, teacher-forced, against the fp64 oracle on the same seeded
inputs (acceptance rules in parity.py).  Covers ragged batches with one-token prompts, gate
blocks of 64 (groups narrower than the 256-column GEMM tiles) and 256, prompts long enough
for the chunked scan, twenty sequences (decode GEMMs above 16 rows), fp32 and bf16, random
norm offsets, prefill continued on held state, graph and direct decode, split-K and tile
switches, and the rglru-2b layer shapes at full width (two of the blocks)."""
import numpy as np
import pytest

from oracle import argmax_lowest, split_prompts
from oracle.rglru import OracleRG, teacher_forced_run_rg
from parity import chunk_prompts, judge, log, run_gpu_mamba
from synth import gen
from synth import rglru as SR

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
    log(f"rglru parity {name}: rows={rep.rows} max_abs={rep.max_abs_err:.3e} "
        f"worst_row_rel={rep.worst_rel_row_err:.3e} literal_mismatch={rep.literal_mismatches} "
        f"unexplained={rep.unexplained_mismatches}")
    for d in rep.details:
        log("  " + d)
    return rep


def _config(name):
    if name == "rglru-2b-l2":
        # the rglru-2b shapes (d 2560, 10 blocks of 256, MLP 7680, vocab 256000), two blocks
        return SR.RG_CONFIGS["rglru-2b"].replace(name=name, n_layers=2, prompt_len=256,
                                                 n_decode=4)
    return SR.get_rg_config(name)


# (workload, graph replay, options)
CASES = [("t-rg", True, {}), ("t-rg", False, {}),
         ("t-rg-f32", True, {}), ("t-rg-f32", False, {"prefill_splitk": 0}),
         ("t-rg-long", True, {}), ("t-rg-long", False, {"decode_splitk": 0, "prefill_tile": 3}),
         ("t-rg-k2", True, {}), ("t-rg-k2", False, {}),
         ("t-rg-f32", True, {"decode_splitk": 2}), ("t-rg", True, {"decode_splitk": 2}),
         ("rglru-2b-l2", True, {})]


@pytest.mark.parametrize("name,graph,options", CASES,
                         ids=[f"{c[0]}-{'graph' if c[1] else 'direct'}"
                              + "".join(f"-{k}{v}" for k, v in c[2].items()) for c in CASES])
def test_rglru_workload_parity(name, graph, options):
    cfg = _config(name)
    log(f"rglru parity {name}: oracle ...")
    w = SR.weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    ref_l, ref_t = teacher_forced_run_rg(OracleRG(cfg, w), lens, packed, cfg.n_decode)
    log(f"rglru parity {name}: gpu ...")
    gl, gt = run_gpu_mamba(cfg, w, [split_prompts(lens, packed)], ref_t, cfg.n_decode,
                           use_graph=graph, options=options)
    rep = _report(name, cfg.dtype, ref_l, gl, gt)
    assert rep.ok(cfg.dtype), rep


@pytest.mark.parametrize("name,n_chunks", [("t-rg", 3), ("t-rg-f32", 2), ("t-rg-long", 2)])
def test_rglru_chunked_prefill_parity(name, n_chunks):
    cfg = SR.get_rg_config(name)
    if name == "t-rg":
        cfg = cfg.replace(prompt_list=(37, 4, 70))
    if name == "t-rg-long":
        cfg = cfg.replace(prompt_range=(8, 400))
    w = SR.weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    chunks = chunk_prompts(split_prompts(lens, packed), n_chunks)
    nd = 3
    om = OracleRG(cfg, w)
    ref_l = [om.prefill(chunks[0])] + [om.extend(c) for c in chunks[1:]]
    ref_t = [argmax_lowest(x) for x in ref_l]
    for _ in range(nd):
        ref_l.append(om.decode(ref_t[-1]))
        ref_t.append(argmax_lowest(ref_l[-1]))
    ref_l, ref_t = np.stack(ref_l), np.stack(ref_t)
    gl, gt = run_gpu_mamba(cfg, w, chunks, ref_t, nd)
    rep = _report(f"{name}-chunked", cfg.dtype, ref_l, gl, gt)
    assert rep.ok(cfg.dtype), rep


def test_rglru_reset_and_state_errors():
    import torch
    from paper_2608_21836_amd.binding import LLError, MambaModel, upload_mamba_weights
    cfg = SR.RG_TEST_CONFIGS["t-rg-f32"]
    w = SR.weights(cfg)
    m = MambaModel(cfg, upload_mamba_weights(cfg, w), max_batch=2, max_prefill_tokens=128)
    toks = torch.zeros(4, dtype=torch.int32, device="cuda")
    with pytest.raises(LLError):
        m.decode_step(toks[:2])            # decode before prefill
    m.prefill([2, 2], toks)
    with pytest.raises(LLError):
        m.prefill([4], toks)               # different batch on held state
    with pytest.raises(LLError):
        m.prefill([100, 100], torch.zeros(200, dtype=torch.int32, device="cuda"))  # capacity
    with pytest.raises(LLError):
        m.set_option("decode_fused", 1)    # not an option of this model
    m.reset()
    nxt, _ = m.prefill([4], toks)
    torch.cuda.synchronize()
    assert m.seq_lengths() == [4]
    assert m.device_flags() == 0
    m.close()


@pytest.mark.parametrize("family,name", [("mamba", "t-mamba"), ("mamba2", "t-mamba2"),
                                         ("rglru", "t-rg")])
def test_graph_replay_equals_direct_launches_bitwise(family, name):
    """Decode steps replayed from a captured HIP graph give the same bits as the same kernels
    launched one by one (state-space families; the Mamba step with fp32 atomics is excluded)."""
    from synth import mamba as SM
    from synth import mamba2 as S2
    mod = {"mamba": SM, "mamba2": S2, "rglru": SR}[family]
    get = {"mamba": SM.get_mamba_config, "mamba2": S2.get_mamba2_config,
           "rglru": SR.get_rg_config}[family]
    cfg = get(name)
    w = mod.weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    prompts = split_prompts(lens, packed)
    ref_t = np.zeros((cfg.n_decode + 1, len(prompts)), dtype=np.int64)   # fixed inputs
    opts = {"decode_fused": 1} if family == "mamba" else {}
    gl, gt = run_gpu_mamba(cfg, w, [prompts], ref_t, cfg.n_decode, use_graph=True, options=opts)
    dl, dt = run_gpu_mamba(cfg, w, [prompts], ref_t, cfg.n_decode, use_graph=False, options=opts)
    assert np.array_equal(gl, dl) and np.array_equal(gt, dt)
