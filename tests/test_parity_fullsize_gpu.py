"""Parity of the large workloads at full depth, as the benchmark runs them.

Every layer of the model runs, at the workload's real width, batch, ragged prompt lengths and
cache capacity, with the implementation options the tuner accepted for that workload (the
options bench.py applies).  The fp64 oracle's logits come from stored files written by
tests/golden/fullsize_oracle.py (which calls only the oracle and the input generator): the
oracle takes minutes to hours for these sizes, so it runs once per change of its sources, and
a file whose recorded source hash differs from the tree's is refused.

The oracle covers a sample of the sequences (all eight of 1b-gqa, the single one of 7b-mha,
the shortest and the longest of 8b-gqa's 32), teacher-forced: both sides consume the
oracle's greedy tokens.  The other sequences of the batch run free on the GPU with their own
tokens (batch independence is pinned in the oracle tests), so every launch has the shapes of
the real workload.
"""
import os
import sys

import numpy as np
import pytest

from parity import judge, log
from synth import gen, get_config

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
sys.path.insert(0, GOLDEN)
import fullsize_oracle as fx  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21836_amd.binding import load_library
    load_library()


def load_fixture(name):
    """(stored arrays, reference logits [steps + 1, S, V] fp64).  The reference is the 16-bit
    code dequantised, with the eight largest logits of every row replaced by their fp32
    values (exact to ~1e-7 relative, where token decisions are made)."""
    path = fx.fixture_path(name)
    if not os.path.exists(path):
        pytest.fail(f"missing oracle file {path}: python tests/golden/fullsize_oracle.py {name}")
    d = dict(np.load(path, allow_pickle=False))
    if str(d["sources_sha256"]) != fx.sources_sha256():
        pytest.fail(f"{path} was written by other oracle / generator sources than the tree's; "
                    f"regenerate it: python tests/golden/fullsize_oracle.py {name}")
    ref = fx.dequantise(d["row_min"], d["row_max"], d["codes"])
    np.put_along_axis(ref, d["top_ids"].astype(np.int64), d["top_vals"].astype(np.float64),
                      axis=-1)
    return d, ref


def run_gpu(cfg, lens, packed, sel, ref_tokens, steps, options):
    """Prefill of the whole batch, then `steps` decode steps: sequences in `sel` are fed the
    oracle's tokens, the others their own.  Returns the logits and tokens of `sel`."""
    import torch
    from paper_2608_21836_amd.binding import Model, to_device
    B = len(lens)
    workers = max(1, min(16, len(os.sched_getaffinity(0))))
    dev_w = {n: to_device(a, cfg.dtype) for n, a in gen.iter_weights_parallel(cfg, workers)}
    dev_w.update({k: to_device(v, cfg.dtype) for k, v in gen.gains(cfg).items()})
    model = Model(cfg, dev_w, max_batch=B, max_prefill_tokens=int(sum(lens)),
                  max_ctx=int(max(lens)) + cfg.n_decode)
    del dev_w
    torch.cuda.empty_cache()
    for k, v in options.items():
        model.set_option(k, int(v))
    toks = torch.from_numpy(np.asarray(packed, dtype=np.int32)).cuda()
    logits = torch.empty(B, cfg.vocab, dtype=torch.float32, device="cuda")
    nxt = torch.empty(B, dtype=torch.int32, device="cuda")
    model.prefill(lens, toks, nxt, logits)
    torch.cuda.synchronize()
    gl, gt = [logits.cpu().numpy()[sel]], [nxt.cpu().numpy()[sel]]
    inp = torch.empty(B, dtype=torch.int32, device="cuda")
    for k in range(1, steps + 1):
        feed = nxt.cpu().numpy().copy()
        feed[sel] = ref_tokens[k - 1]
        inp.copy_(torch.from_numpy(feed))
        model.decode_step(inp, nxt, logits)
        torch.cuda.synchronize()
        gl.append(logits.cpu().numpy()[sel])
        gt.append(nxt.cpu().numpy()[sel])
    assert model.seq_lengths() == [int(x) + steps for x in lens]
    assert model.device_flags() == 0
    model.close()
    return np.stack(gl), np.stack(gt)


@pytest.mark.parametrize("name", ["1b-gqa", "7b-mha", "8b-gqa"])
def test_full_depth_parity(name):
    from paper_2608_21836_amd.tuner import accepted_options
    d, ref = load_fixture(name)
    cfg = get_config(name)
    lens, packed = gen.prompt_tokens(cfg)
    assert [int(x) for x in d["lens"]] == lens
    assert str(d["prompt_sha256"]) == gen.sha256(np.asarray(packed, dtype=np.int32))
    sel = [int(x) for x in d["seqs"]]
    steps = int(d["steps"])
    options = accepted_options(name)
    log(f"fulldepth {name}: {cfg.n_layers} layers, batch {len(lens)}, {sum(lens)} prompt tokens, "
        f"sequences {sel} teacher-forced for {steps} steps, options {options}")
    gl, gt = run_gpu(cfg, lens, packed, sel, d["tokens"], steps, options)
    rep = judge(name, cfg.dtype, ref, gl, gt, ref_margin=d["margin"], ref_tokens=d["tokens"])
    log(f"fulldepth {name}: rows={rep.rows} max_abs={rep.max_abs_err:.3e} "
        f"worst_row_rel={rep.worst_rel_row_err:.3e} literal_mismatch={rep.literal_mismatches} "
        f"unexplained={rep.unexplained_mismatches} min_margin={float(d['margin'].min()):.3e}")
    for line in rep.details:
        log("  " + line)
    # the stored quantisation error (at most range / 131070 per logit) is taken off the bar
    assert rep.ok(cfg.dtype, quant=1.0 / 131070), rep
