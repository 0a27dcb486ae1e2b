"""Acceptance of the selective state-space (Mamba) model: whole workloads through
ll_mamba_load / ll_mamba_prefill / ll_mamba_decode_step, teacher-forced, against the fp64
oracle on the same seeded inputs (acceptance rules in parity.py).  Covers ragged batches with
one-token prompts, prompts long enough for the chunked (three-pass) scan, fp32 and bf16,
prefill continued on held state (chunks shorter than the convolution window too), graph and
direct decode, and the full mamba-130m workload."""
import numpy as np
import pytest

from oracle import argmax_lowest, split_prompts
from oracle.mamba import OracleMamba, teacher_forced_run_mamba
from parity import chunk_prompts, judge, log, run_gpu_mamba
from synth import gen
from synth import mamba as SM

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
    log(f"mamba parity {name}: rows={rep.rows} max_abs={rep.max_abs_err:.3e} "
        f"worst_row_rel={rep.worst_rel_row_err:.3e} literal_mismatch={rep.literal_mismatches} "
        f"unexplained={rep.unexplained_mismatches}")
    for d in rep.details:
        log("  " + d)
    return rep


# (workload, graph replay, decode steps (None: the workload's), options)
CASES = [("t-mamba", True, None, {}), ("t-mamba", False, None, {"decode_fused": 0}),
         ("t-mamba-f32", True, None, {}), ("t-mamba-f32", False, None, {"decode_fused": 0}),
         ("t-mamba-long", True, None, {}), ("t-mamba-b20", True, None, {}),
         ("t-mamba-b20", False, None, {"decode_splitk": 0, "prefill_splitk": 0}),
         ("t-mamba", True, None, {"decode_fused": 2}), ("t-mamba-f32", True, None, {"decode_fused": 2}),
         ("t-mamba-wide", True, None, {}), ("t-mamba-wide", True, None, {"decode_fused": 2}),
         ("t-mamba-r160", True, None, {}),
         ("t-mamba-k2", True, None, {}), ("t-mamba-k2", False, None, {"decode_fused": 0}),
         ("t-mamba-f32", True, None, {"decode_fused": 0, "decode_splitk": 2}),
         ("mamba-130m", True, 16, {}), ("mamba-130m", True, 16, {"decode_fused": 0}),
         ("mamba-130m", True, 16, {"decode_fused": 2})]


def _config(name):
    if name == "t-mamba-long":   # sequences of several hundred tokens, several scan chunks
        return SM.MAMBA_TEST_CONFIGS["t-mamba"].replace(name=name, seed=33,
                                                        prompt_list=(300, 17, 513), n_decode=4)
    return SM.get_mamba_config(name)


@pytest.mark.parametrize("name,graph,n_decode,options", CASES,
                         ids=[f"{c[0]}-{'graph' if c[1] else 'direct'}"
                              + "".join(f"-{k}{v}" for k, v in c[3].items()) for c in CASES])
def test_mamba_workload_parity(name, graph, n_decode, options):
    cfg = _config(name)
    nd = n_decode if n_decode is not None else cfg.n_decode
    log(f"mamba parity {name}: oracle ...")
    w = SM.weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    ref_l, ref_t = teacher_forced_run_mamba(OracleMamba(cfg, w), lens, packed, nd)
    log(f"mamba parity {name}: gpu ...")
    gl, gt = run_gpu_mamba(cfg, w, [split_prompts(lens, packed)], ref_t, nd, use_graph=graph,
                           options=options)
    rep = _report(name, cfg.dtype, ref_l, gl, gt)
    assert rep.ok(cfg.dtype), rep


@pytest.mark.parametrize("name,n_chunks", [("t-mamba", 3), ("t-mamba-f32", 2),
                                           ("t-mamba-long", 3)])
def test_mamba_chunked_prefill_parity(name, n_chunks):
    """Prompts cut into consecutive pieces, each a further ll_mamba_prefill on the held state
    (the 1-token prompt of t-mamba gives pieces of length 0 -> it is lengthened to 4)."""
    cfg = _config(name)
    if name == "t-mamba":
        cfg = cfg.replace(prompt_list=(37, 4, 70))
    w = SM.weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    chunks = chunk_prompts(split_prompts(lens, packed), n_chunks)
    nd = 3
    log(f"mamba chunked {name}: oracle ...")
    om = OracleMamba(cfg, w)
    ref_l = [om.prefill(chunks[0])] + [om.extend(c) for c in chunks[1:]]
    ref_t = [argmax_lowest(x) for x in ref_l]
    for _ in range(nd):
        ref_l.append(om.decode(ref_t[-1]))
        ref_t.append(argmax_lowest(ref_l[-1]))
    ref_l, ref_t = np.stack(ref_l), np.stack(ref_t)
    log(f"mamba chunked {name}: gpu ...")
    gl, gt = run_gpu_mamba(cfg, w, chunks, ref_t, nd)
    rep = _report(f"{name}-chunked", cfg.dtype, ref_l, gl, gt)
    assert rep.ok(cfg.dtype), rep


def test_mamba_reset_and_state_errors():
    import torch
    from paper_2608_21836_amd.binding import LLError, MambaModel, upload_mamba_weights
    cfg = SM.MAMBA_TEST_CONFIGS["t-mamba-f32"]
    w = SM.weights(cfg)
    m = MambaModel(cfg, upload_mamba_weights(cfg, w), max_batch=2, max_prefill_tokens=128)
    toks = torch.zeros(4, dtype=torch.int32, device="cuda")
    with pytest.raises(LLError):
        m.decode_step(toks[:2])            # decode before prefill
    m.prefill([2, 2], toks)
    with pytest.raises(LLError):
        m.prefill([4], toks)               # different batch on held state
    with pytest.raises(LLError):
        m.prefill([100, 100], torch.zeros(200, dtype=torch.int32, device="cuda"))  # capacity
    m.reset()
    nxt, _ = m.prefill([4], toks)
    torch.cuda.synchronize()
    assert m.seq_lengths() == [4]
    assert m.device_flags() == 0
    m.close()
