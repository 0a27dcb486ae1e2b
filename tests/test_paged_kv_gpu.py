"""Paged KV cache (ll_config.kv_page / kv_pages): a pool of pages of 256 positions per layer and
a per-sequence block table, filled as prefill and decode reach new pages.

The paged path runs the same kernels as the contiguous one; only the address of a cached row
changes.  So on the same inputs its logits must equal the contiguous run's bit for bit, and
pass the oracle by the usual rules (parity.py).  The cases cross page boundaries in prefill,
in chunked prefill and in decode, use pools holding exactly the pages the job needs (so pages
are shared out of one pool in a non-identity order), and cover the bf16 and fp32 attention
kernels, ragged batches of 32 and the 125m workload.  Pool exhaustion is checked to leave
the state unchanged."""
import numpy as np
import pytest

from oracle import OracleModel, split_prompts, teacher_forced_run
from parity import (chunk_prompts, judge, log, oracle_chunked_run, run_gpu_chunked,
                    run_gpu_teacher_forced)
from synth import gen, get_config

pytestmark = pytest.mark.gpu

PAGE = 256


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21836_amd.binding import load_library
    load_library()


def _pages(lengths):
    return int(sum((int(x) + PAGE - 1) // PAGE for x in lengths))


def _config(name):
    cfg = get_config(name)
    over = {"t-gqa-hd128": dict(prompt_list=(250, 33, 505), n_decode=10),
            "t-f32-ragged": dict(prompt_list=(250, 65, 2), n_decode=10),
            "t-b32-hd128": dict(prompt_range=(200, 300), n_decode=60)}.get(name)
    return cfg.replace(**over) if over else cfg


@pytest.mark.parametrize("name", ["t-gqa-hd128", "t-f32-ragged", "t-b32-hd128", "125m"])
def test_paged_equals_contiguous_and_oracle(name):
    cfg = _config(name)
    nd = cfg.n_decode
    w = gen.weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    log(f"paged {name}: lens {list(lens)[:8]}..., {nd} steps, oracle ...")
    ref_l, ref_t = teacher_forced_run(OracleModel(cfg, w), lens, packed, nd)
    gl, gt = run_gpu_teacher_forced(cfg, w, lens, packed, ref_t, nd)
    pool = _pages([x + nd for x in lens])
    log(f"paged {name}: pool of {pool} pages")
    pl, pt = run_gpu_teacher_forced(cfg, w, lens, packed, ref_t, nd,
                                    paging={"kv_page": PAGE, "kv_pages": pool})
    assert np.array_equal(pl, gl) and np.array_equal(pt, gt), \
        f"paged differs from contiguous: max {np.abs(pl - gl).max()}"
    rep = judge(f"{name}-paged", cfg.dtype, ref_l, pl, pt)
    log(f"paged {name}: max_abs={rep.max_abs_err:.3e} worst_row_rel={rep.worst_rel_row_err:.3e}")
    assert rep.ok(cfg.dtype), rep


@pytest.mark.parametrize("name,n_chunks", [("t-gqa-hd128", 3), ("t-f32-ragged", 2)])
def test_paged_chunked_prefill(name, n_chunks):
    cfg = get_config(name)
    cfg = cfg.replace(prompt_list=(300, 40, 520) if name == "t-gqa-hd128" else (270, 9, 513))
    w = gen.weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    chunks = chunk_prompts(split_prompts(lens, packed), n_chunks)
    nd = 4
    ref_l, ref_t = oracle_chunked_run(OracleModel(cfg, w), chunks, nd)
    gl, gt = run_gpu_chunked(cfg, w, chunks, ref_t, nd)
    pl, pt = run_gpu_chunked(cfg, w, chunks, ref_t, nd,
                             paging={"kv_page": PAGE, "kv_pages": _pages([x + nd for x in lens])})
    assert np.array_equal(pl, gl) and np.array_equal(pt, gt)
    rep = judge(f"{name}-paged-chunked", cfg.dtype, ref_l, pl, pt)
    assert rep.ok(cfg.dtype), rep


def test_pool_exhaustion_leaves_state_unchanged():
    import torch
    from paper_2608_21836_amd.binding import LL_ERR_CAPACITY, LLError, Model, upload_weights
    cfg = get_config("tiny-f32")
    m = Model(cfg, upload_weights(cfg, gen.weights(cfg)), max_batch=2, max_prefill_tokens=320,
              max_ctx=600, kv_page=PAGE, kv_pages=2)
    assert m.kv_pages() == (0, 2)
    t = torch.zeros(320, dtype=torch.int32, device="cuda")
    with pytest.raises(LLError) as e:          # needs 2 + 1 pages
        m.prefill([300, 10], t)
    assert e.value.status == LL_ERR_CAPACITY
    assert m.kv_pages() == (0, 2) and m.seq_lengths() == []
    nxt, _ = m.prefill([250, 10], t)
    assert m.kv_pages() == (2, 2)
    for _ in range(6):                         # sequence 0 fills its page (positions < 256)
        m.decode_step(nxt, nxt)
    with pytest.raises(LLError) as e:          # position 256 needs a third page
        m.decode_step(nxt, nxt)
    assert e.value.status == LL_ERR_CAPACITY
    assert m.seq_lengths() == [256, 16] and m.kv_pages() == (2, 2)
    m.kv_reset()
    assert m.kv_pages() == (0, 2)
    m.prefill([255, 1], t)
    m.decode_step(nxt, nxt)
    torch.cuda.synchronize()
    assert m.device_flags() == 0
    m.close()
