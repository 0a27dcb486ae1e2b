"""Every implementation variant (ll_option value) computes the same model: whole workloads
with a non-default option, teacher-forced, judged against the fp64 oracle like the default
path (acceptance rules in parity.py).  These are the candidates the tuner may admit, so each
must pass the in-model check on its own."""
import pytest

from oracle import OracleModel, teacher_forced_run
from parity import judge, log, run_gpu_teacher_forced
from synth import gen, get_config

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21836_amd.binding import load_library
    load_library()


CASES = [
    ("t-gqa-hd64", {"prefill_splitk": 0}),
    ("t-gqa-hd64", {"prefill_tile": 1}),
    ("t-gqa-hd64", {"prefill_tile": 2}),
    ("t-gqa-hd64", {"prefill_tile": 3}),
    ("t-gqa-hd64", {"attn_decode_chunk": 256}),
    ("t-gqa-hd128", {"prefill_tile": 1, "attn_decode_chunk": 128}),
    ("t-f32-ragged", {"prefill_tile": 2, "prefill_splitk": 0}),
    ("t-b32-hd128", {"decode_splitk": 0}),
    ("t-gqa-hd64", {"decode_splitk": 2}),      # residual GEMMs: K over two blocks, atomics
    ("t-f32-ragged", {"decode_splitk": 2}),
    ("125m", {"decode_splitk": 2}),
    ("t-b32-hd128", {"prefill_tile": 1, "attn_decode_chunk": 256}),
    ("t-gqa-hd64", {"decode_fused": 1}),       # attention merge inside the O projection
    ("t-f32-ragged", {"decode_fused": 1}),
    ("125m", {"decode_fused": 1}),
    ("t-gqa-hd128", {"decode_fused": 1, "decode_splitk": 2}),
]


@pytest.mark.parametrize("name,options", CASES, ids=[f"{n}-{o}" for n, o in CASES])
def test_variant_parity(name, options):
    cfg = get_config(name)
    w = gen.weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    log(f"variant {name} {options}: oracle ...")
    ref_logits, ref_tokens = teacher_forced_run(OracleModel(cfg, w), lens, packed, cfg.n_decode)
    log(f"variant {name} {options}: gpu ...")
    gl, gt = run_gpu_teacher_forced(cfg, w, lens, packed, ref_tokens, cfg.n_decode,
                                    options=options)
    rep = judge(name, cfg.dtype, ref_logits, gl, gt)
    log(f"variant {name} {options}: max_abs={rep.max_abs_err:.3e} "
        f"worst_row_rel={rep.worst_rel_row_err:.3e} literal_mismatch={rep.literal_mismatches}")
    assert rep.ok(cfg.dtype), rep


def test_tuner_accepts_only_passing_faster_variants():
    """The tuner (Eq. 1 ordering, Eq. 3 acceptance) on a small workload: the options it ends
    with still match the oracle, and every accepted knob cleared the delta margin with a
    passing in-model check."""
    import numpy as np
    import torch
    from paper_2608_21836_amd import tuner
    from paper_2608_21836_amd.binding import Model, upload_weights
    cfg = get_config("t-gqa-hd64")
    w = gen.weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    model = Model(cfg, upload_weights(cfg, w), max_batch=len(lens),
                  max_prefill_tokens=int(sum(lens)), max_ctx=int(max(lens)) + cfg.n_decode)
    wl = tuner.Workload(list(lens), torch.from_numpy(np.asarray(packed, dtype=np.int32)).cuda(),
                        cfg.n_decode)
    reports = tuner.tune(model, wl, delta=0.02, reps=1, n_check=2, log=log)
    opts = model.options()
    model.close()
    assert {r.option for r in reports} == {k[0] for k in tuner.KNOBS}
    for r in reports:
        if r.accepted:
            c = r.candidates[r.chosen]
            assert c["ok"] and c["ell"] <= 1 - 0.02, r
        assert opts[r.option] == r.chosen
    ref_logits, ref_tokens = teacher_forced_run(OracleModel(cfg, w), lens, packed, cfg.n_decode)
    gl, gt = run_gpu_teacher_forced(cfg, w, lens, packed, ref_tokens, cfg.n_decode, options=opts)
    assert judge(cfg.name, cfg.dtype, ref_logits, gl, gt).ok(cfg.dtype)


@pytest.mark.parametrize("name", ["t-gqa-hd64", "t-f32-ragged", "125m"])
def test_merge_in_o_projection_is_bitwise_the_merge_kernel(name):
    """decode_fused 1 stages the attention merge inside the O projection with the merge
    kernel's arithmetic, so the logits equal the two-kernel path's bit for bit."""
    import numpy as np
    cfg = get_config(name)
    w = gen.weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    nd = min(cfg.n_decode, 24)
    ref_t = np.zeros((nd + 1, len(lens)), dtype=np.int64)      # fixed inputs
    base_l, base_t = run_gpu_teacher_forced(cfg, w, lens, packed, ref_t, nd)
    for graph in (1, 0):
        fl, ft = run_gpu_teacher_forced(cfg, w, lens, packed, ref_t, nd,
                                        options={"decode_fused": 1, "decode_graph": graph})
        assert np.array_equal(fl, base_l) and np.array_equal(ft, base_t), \
            f"graph {graph}: max diff {np.abs(fl - base_l).max()}"
