"""Write-side out-of-bounds guards.

The paper's motivating evidence (Sec. 2.1) includes a latent out-of-bounds access that passes
an isolated check and faults only under another allocation state.  Read-side checks (caches
poisoned with NaN past every sequence's length) live in test_kernels_gpu.py; here every write
is fenced:
  * every region of the workspace layout is followed by a gap that no kernel may write, and
    the workspace itself sits between guard bytes;
  * the caller's outputs (logits, next tokens) sit between guard bytes;
  * every KV-cache position at or past a sequence's final length must stay untouched.
All of it is filled with a byte pattern after the model is loaded and checked after a prefill
and decode steps that reach the cache capacity, at ragged prompt lengths, on the split-K
decode path (32 sequences), in fp32, and with a paged cache.
"""
import numpy as np
import pytest

from parity import log
from synth import gen, get_config

pytestmark = pytest.mark.gpu

PATTERN = 0xA5
GUARD = 4096   # bytes around the workspace and the outputs


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21836_amd.binding import load_library
    load_library()


def _gaps(regions, total):
    """Byte ranges of the workspace that lie outside every region."""
    out, end = [], 0
    for _, off, nb in sorted(regions, key=lambda r: r[1]):
        assert off >= end, "regions overlap"
        if off > end:
            out.append((end, off))
        end = off + nb
    if end < total:
        out.append((end, total))
    return out


def _guarded(torch, n, dtype):
    """A tensor of n elements between GUARD pattern bytes: (whole uint8 buffer, interior)."""
    esize = torch.empty(0, dtype=dtype).element_size()
    buf = torch.full((n * esize + 2 * GUARD,), PATTERN, dtype=torch.uint8, device="cuda")
    return buf, buf[GUARD:GUARD + n * esize].view(dtype)


def _intact(t) -> bool:
    return bool((t == PATTERN).all().item())


@pytest.mark.parametrize("name,paged", [("t-gqa-hd64", False), ("t-b32-hd128", False),
                                        ("t-f32-ragged", False), ("t-gqa-hd128", True)])
def test_no_write_outside_regions(name, paged):
    import torch
    from paper_2608_21836_amd.binding import Model, upload_weights
    cfg = get_config(name)
    lens, packed = gen.prompt_tokens(cfg)
    B, T, nd = len(lens), int(sum(lens)), cfg.n_decode
    max_ctx = max(lens) + nd          # the longest sequence ends exactly at capacity
    paging = {}
    if paged:
        pages = sum((x + nd + 255) // 256 for x in lens)
        paging = {"kv_page": 256, "kv_pages": pages}
    log(f"guards {name}: lens {lens}, {nd} decode steps, max_ctx {max_ctx}, paged {paged}")
    model = Model(cfg, upload_weights(cfg, gen.weights(cfg)), max_batch=B, max_prefill_tokens=T,
                  max_ctx=max_ctx, guard_bytes=GUARD, **paging)
    torch.cuda.synchronize()
    ws, guarded = model.workspace, model.guarded
    regions = model.regions()
    gaps = _gaps(regions, ws.numel())
    assert len(gaps) >= len(regions) - 1   # a gap after every region
    for a, b in gaps:
        ws[a:b].fill_(PATTERN)
    guarded[:GUARD].fill_(PATTERN)
    guarded[-GUARD:].fill_(PATTERN)
    # KV positions past each sequence's final length (contiguous cache)
    eb = 2 if cfg.dtype == "bf16" else 4
    row = cfg.head_dim * eb
    kv = {r[0]: r for r in regions}
    tails = []
    if not paged:
        for cache in ("kcache", "vcache"):
            _, off, nb = kv[cache]
            layer_bytes = B * cfg.n_kv_heads * max_ctx * row
            assert nb == cfg.n_layers * layer_bytes
            view = ws[off:off + nb].view(cfg.n_layers, B, cfg.n_kv_heads, max_ctx * row)
            for b, L in enumerate(lens):
                tail = view[:, b, :, (L + nd) * row:]
                if tail.shape[-1]:
                    tail.fill_(PATTERN)
                    tails.append((cache, b, tail))
    lbuf, logits = _guarded(torch, B * cfg.vocab, torch.float32)
    nbuf, nxt = _guarded(torch, B, torch.int32)
    torch.cuda.synchronize()

    toks = torch.from_numpy(np.asarray(packed, dtype=np.int32)).cuda()
    model.prefill(lens, toks, nxt, logits.view(B, cfg.vocab))
    for _ in range(nd):
        model.decode_step(nxt, nxt, logits.view(B, cfg.vocab))
    torch.cuda.synchronize()
    assert model.seq_lengths() == [x + nd for x in lens]
    assert model.device_flags() == 0

    def before(a):
        return max((r for r in regions if r[1] + r[2] <= a), key=lambda r: r[1] + r[2])[0]
    bad = [f"gap {a}..{b} after region {before(a)}" for a, b in gaps if not _intact(ws[a:b])]
    assert not bad, bad
    assert _intact(guarded[:GUARD]) and _intact(guarded[-GUARD:]), "workspace guard written"
    assert _intact(lbuf[:GUARD]) and _intact(lbuf[-GUARD:]), "logits guard written"
    assert _intact(nbuf[:GUARD]) and _intact(nbuf[-GUARD:]), "next-token guard written"
    for cache, b, tail in tails:
        assert _intact(tail), f"{cache} written past the length of sequence {b}"
    # the outputs themselves were written
    assert not _intact(logits.view(torch.uint8)) and bool(torch.isfinite(logits).all().item())
    log(f"guards {name}: {len(gaps)} gaps, {len(tails)} cache tails intact")
    model.close()
