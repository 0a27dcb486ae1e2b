"""The allocation-free LM head + argmax (ll_op_lmhead_argmax_noalloc) against the entry point
with a caller scratch (ll_op_lmhead_argmax): same logits bitwise and same tokens, on two calls
in a row, the second smaller (the static partials keep the first call's contents)."""
import numpy as np
import pytest

from parity import device_tensor, log, rounded

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21836_amd.binding import load_library
    load_library()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_lmhead_matches_scratch_version(dtype):
    import torch
    from paper_2608_21836_amd.binding import (LLError, op_lmhead_argmax,
                                              op_lmhead_argmax_noalloc, op_repack)
    rng = np.random.default_rng(42)
    # 8b-gqa's LM head at 32 rows (the largest shape the static scratch takes at this vocab
    # is 65 rows), then a smaller call: 3 rows of a 4096-word vocabulary over k = 256
    for rows, vocab, k in ((32, 128256, 4096), (3, 4096, 256)):
        log(f"noalloc lm head {dtype} rows={rows} vocab={vocab} k={k}")
        h = device_tensor(rounded(rng.standard_normal((rows, k)), dtype), dtype)
        w = device_tensor(rounded(rng.standard_normal((vocab, k)) * 0.02, dtype), dtype)
        wt = op_repack(w)
        ref_next, ref_logits = op_lmhead_argmax(h, wt, vocab)
        logits = torch.empty(rows, vocab, dtype=torch.float32, device="cuda")
        nxt = torch.empty(rows, dtype=torch.int32, device="cuda")
        op_lmhead_argmax_noalloc(h, wt, vocab, logits, nxt)
        torch.cuda.synchronize()
        assert torch.equal(logits, ref_logits)
        assert torch.equal(nxt, ref_next)
        # without logits: the tokens alone
        nxt2 = torch.full((rows,), -1, dtype=torch.int32, device="cuda")
        op_lmhead_argmax_noalloc(h, wt, vocab, None, nxt2)
        torch.cuda.synchronize()
        assert torch.equal(nxt2, ref_next)
    # a shape beyond the static scratch is refused before anything is enqueued
    h = torch.zeros(66, 4096, dtype=torch.bfloat16 if dtype == "bf16" else torch.float32,
                    device="cuda")
    with pytest.raises(LLError) as e:
        op_lmhead_argmax_noalloc(h, wt, 128256, None, torch.empty(66, dtype=torch.int32,
                                                                  device="cuda"))
    assert e.value.status == 3   # LL_ERR_CAPACITY
