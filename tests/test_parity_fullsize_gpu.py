"""Parity at the large workloads' real width, batch and prompt lengths.

Every kernel launch here has the grid and shapes of the full workload (same d_model, heads,
FFN, vocab, batch, ragged prompt lengths, cache capacity); only the number of identical
decoder layers is cut to two so that the fp64 oracle can follow.  The oracle computes a
sample of the sequences (batch independence is pinned in the oracle tests), teacher-forced
for a few decode steps; the other sequences run free on the GPU with their own tokens.
"""
import numpy as np
import pytest

from oracle import OracleModel, argmax_lowest, split_prompts
from parity import judge, log
from synth import gen, get_config

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21836_amd.binding import load_library
    load_library()


def _sample(name, lens):
    if name == "8b-gqa":   # shortest and longest prompt
        return sorted({int(np.argmin(lens)), int(np.argmax(lens))})
    if len(lens) > 1:
        return [0, len(lens) - 1]
    return [0]


@pytest.mark.parametrize("name", ["1b-gqa", "7b-mha", "8b-gqa"])
def test_full_width_parity(name):
    import torch
    from paper_2608_21836_amd.binding import Model, upload_weights
    n_decode = 4
    cfg = get_config(name).replace(n_layers=2)
    log(f"fullwidth {name}: weights")
    w = gen.weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    B = len(lens)
    sel = _sample(name, lens)
    prompts = split_prompts(lens, packed)

    log(f"fullwidth {name}: oracle on sequences {sel} (lengths {[lens[i] for i in sel]})")
    om = OracleModel(cfg, w)
    ref_l = [om.prefill([prompts[i] for i in sel])]
    ref_t = [argmax_lowest(ref_l[0])]
    for _ in range(n_decode):
        ref_l.append(om.decode(ref_t[-1]))
        ref_t.append(argmax_lowest(ref_l[-1]))
    del om

    log(f"fullwidth {name}: gpu, batch {B}, {sum(lens)} prompt tokens")
    dev_w = upload_weights(cfg, w)
    del w
    model = Model(cfg, dev_w, max_batch=B, max_prefill_tokens=int(sum(lens)),
                  max_ctx=int(max(lens)) + cfg.n_decode)
    del dev_w
    toks = torch.from_numpy(np.asarray(packed, dtype=np.int32)).cuda()
    logits = torch.empty(B, cfg.vocab, dtype=torch.float32, device="cuda")
    nxt = torch.empty(B, dtype=torch.int32, device="cuda")
    model.prefill(lens, toks, nxt, logits)
    torch.cuda.synchronize()
    gl, gt = [logits.cpu().numpy()[sel]], [nxt.cpu().numpy()[sel]]
    inp = torch.empty(B, dtype=torch.int32, device="cuda")
    for k in range(1, n_decode + 1):
        feed = nxt.cpu().numpy().copy()          # free-running for unsampled sequences
        feed[sel] = ref_t[k - 1]                 # teacher-forced for sampled ones
        inp.copy_(torch.from_numpy(feed))
        model.decode_step(inp, nxt, logits)
        torch.cuda.synchronize()
        gl.append(logits.cpu().numpy()[sel])
        gt.append(nxt.cpu().numpy()[sel])
    assert model.device_flags() == 0
    model.close()
    rep = judge(name, cfg.dtype, np.stack(ref_l), np.stack(gl), np.stack(gt))
    log(f"fullwidth {name}: rows={rep.rows} max_abs={rep.max_abs_err:.3e} "
        f"worst_row_rel={rep.worst_rel_row_err:.3e} literal_mismatch={rep.literal_mismatches} "
        f"unexplained={rep.unexplained_mismatches}")
    for d in rep.details:
        log("  " + d)
    assert rep.ok(cfg.dtype), rep
