"""Deployment-time acceptance of implementation variants, after Sec. 3 of the paper.

The paper's loop profiles the real workload, ranks modules by a phase-weighted hotspot score,
qualifies candidate kernels in isolation and admits a candidate into the deployed model only
when the model itself gets faster by a margin.  This module applies the same three rules to
the library's own kernel variants (the ll_option switches of include/ll.h):

  Eq. 1, hotspot score:   s(m) = sum_p w_p * t(m, p) / T(p)
      t(m, p): time of kernel class m in one invocation of phase p; T(p): latency of that
      invocation; w_p: the phase's share of the workload's time (its measured frequency
      times its latency).
  Eq. 2, search utility:  u(c, tau) = t_ref(tau) / t_c(tau) * 1{err(c, tau) <= eps, safe(c, tau)}
      ranks candidates of one task (a kernel class) by their isolated latency, zero when the
      candidate is wrong or failed.
  Eq. 3, deployment acceptance:  c* = argmin_{c in C_dep} l(c),  accepted iff l(c*) <= 1 - delta
      l(c) = L(M[c], W) / L(M, W): the whole workload's latency with the candidate in place
      relative to the current model; C_dep: candidates that pass the in-model check.

The in-model check compares a candidate's logits with output references recorded from the
current model on the same inputs (teacher-forced, so every step sees the same tokens): per
row, max |logit - reference| <= eps * (max - min of the reference row).  Latency is the
workload as the bench runs it: KV reset, prefill of every prompt, free-running greedy decode
steps, timed with stream events.

  python -m paper_2608_21836_amd.tuner --config 125m [--delta 0.01] [--write]
  (a Mamba workload name, e.g. mamba-130m, tunes that model's options)

With --write the accepted (non-default) option values of the workload are stored in
accepted_options.json next to this module; bench.py applies them to that workload, as the
paper deploys accepted patches.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

if __package__ in (None, ""):
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

ACCEPTED_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "accepted_options.json")


def accepted_options(workload: str) -> Dict[str, int]:
    """Option values the tuner accepted for `workload` ({} when none were)."""
    if not os.path.exists(ACCEPTED_PATH):
        return {}
    with open(ACCEPTED_PATH) as f:
        return {k: int(v) for k, v in json.load(f).get(workload, {}).get("options", {}).items()}

# (option, value) pairs whose kernels add partial sums with fp32 atomics: the summation order,
# hence the last bits of the result, can differ between runs.  The tuner may accept them (they
# pass the same in-model check), and the store records them, so that a deployment that needs
# bitwise repeatable runs can leave them out; every other variant is bitwise repeatable.
NONDETERMINISTIC = {("decode_splitk", 2), ("decode_fused", 2)}


def deterministic_options(workload: str) -> Dict[str, int]:
    """accepted_options(workload) without the variants that give up bitwise repeatability."""
    return {k: v for k, v in accepted_options(workload).items()
            if (k, v) not in NONDETERMINISTIC}


# Variants: option name, candidate values (the first is the library default), kernel classes
# whose time the option changes.
KNOBS: List[Tuple[str, Tuple[int, ...], Tuple[str, ...]]] = [
    ("prefill_tile", (0, 1, 2, 3), ("qkv_rope_append", "o_proj_resid", "gate_up_swiglu",
                                    "down_resid")),
    ("prefill_splitk", (1, 0), ("qkv_rope_append", "o_proj_resid", "gate_up_swiglu",
                                "down_resid")),
    ("decode_splitk", (1, 0, 2), ("qkv_rope_append", "o_proj_resid", "gate_up_swiglu",
                               "down_resid")),
    ("attn_decode_chunk", (0, 64, 128, 256), ("attention", "attn_combine")),
    ("decode_fused", (0, 1), ("attention", "attn_combine", "o_proj_resid")),
    ("decode_graph", (1, 0), ("qkv_rope_append", "attention", "attn_combine", "o_proj_resid",
                              "gate_up_swiglu", "down_resid", "lm_head_argmax", "embed",
                              "argmax_reduce", "rmsnorm")),
]


# The same for the Mamba model (include/ll_mamba.h kernel classes).
MAMBA_KNOBS: List[Tuple[str, Tuple[int, ...], Tuple[str, ...]]] = [
    ("decode_fused", (1, 0, 2), ("in_proj", "conv_silu", "x_proj", "scan", "out_proj_resid")),
    ("prefill_tile", (0, 1, 2, 3), ("in_proj", "x_proj", "out_proj_resid")),
    ("prefill_splitk", (1, 0), ("in_proj", "x_proj", "out_proj_resid")),
    ("decode_splitk", (1, 0, 2), ("in_proj", "x_proj", "out_proj_resid")),
    ("decode_graph", (1, 0), ("in_proj", "conv_silu", "x_proj", "scan", "out_proj_resid",
                              "lm_head_argmax", "embed", "argmax_reduce", "rmsnorm")),
]


MAMBA2_KNOBS: List[Tuple[str, Tuple[int, ...], Tuple[str, ...]]] = [
    ("prefill_tile", (0, 1, 2, 3), ("in_proj", "out_proj_resid")),
    ("prefill_splitk", (1, 0), ("in_proj", "out_proj_resid")),
    ("decode_splitk", (1, 0, 2), ("in_proj", "out_proj_resid")),
    ("decode_graph", (1, 0), ("in_proj", "scan", "out_proj_resid", "lm_head_argmax", "embed",
                              "argmax_reduce", "rmsnorm", "gated_rmsnorm")),
]


RG_KNOBS: List[Tuple[str, Tuple[int, ...], Tuple[str, ...]]] = [
    ("prefill_tile", (0, 1, 2, 3), ("in_proj", "gates", "out_proj_resid", "mlp_up", "mlp_down")),
    ("prefill_splitk", (1, 0), ("in_proj", "out_proj_resid", "mlp_up", "mlp_down")),
    ("decode_splitk", (1, 0, 2), ("in_proj", "out_proj_resid", "mlp_up", "mlp_down")),
    ("decode_graph", (1, 0), ("in_proj", "gates", "out_proj_resid", "mlp_up", "mlp_down",
                              "lm_head_argmax", "embed", "argmax_reduce", "rmsnorm")),
]


def hotspot_scores(kernel_ms: Dict[Tuple[str, str], float], phase_ms: Dict[str, float],
                   invocations: Dict[str, int]) -> Dict[str, float]:
    """Eq. 1 over one workload.  kernel_ms[(phase, class)]: that class's summed kernel time
    over the workload; phase_ms[p]: the phase's summed latency; invocations[p]: how often
    the phase ran (1 prefill, N decode steps).  t(m, p) and T(p) are per invocation and
    w_p = phase_ms[p] / sum(phase_ms), so s(m) is the class's share of each phase weighted by
    that phase's share of the workload."""
    total = sum(phase_ms.values())
    score: Dict[str, float] = {}
    for (phase, cls), ms in kernel_ms.items():
        if phase_ms.get(phase, 0.0) <= 0.0 or total <= 0.0:
            continue
        n = max(1, invocations.get(phase, 1))
        t_mp = ms / n
        T_p = phase_ms[phase] / n
        w_p = phase_ms[phase] / total
        score[cls] = score.get(cls, 0.0) + w_p * t_mp / T_p
    return dict(sorted(score.items(), key=lambda kv: -kv[1]))


def search_utility(t_ref: float, t_c: float, err: float, eps: float, safe: bool) -> float:
    """Eq. 2: speed-up over the reference, or 0 for a wrong or unsafe candidate."""
    if not safe or not (err <= eps) or t_c <= 0.0:
        return 0.0
    return t_ref / t_c


def accept(ell: Dict[object, float], ok: Dict[object, bool], delta: float
           ) -> Tuple[Optional[object], bool]:
    """Eq. 3: the passing candidate with the lowest normalised latency, and whether it clears
    the margin (l(c*) <= 1 - delta).  Returns (None, False) when no candidate passes."""
    passing = [c for c in ell if ok.get(c, False)]
    if not passing:
        return None, False
    best = min(passing, key=lambda c: ell[c])
    return best, ell[best] <= 1.0 - delta


def max_row_error(ref, got) -> float:
    """Largest per-row max |got - ref| relative to the reference row's range (inf if any
    value is not finite)."""
    import numpy as np
    ref = np.asarray(ref, dtype=np.float64).reshape(-1, ref.shape[-1])
    got = np.asarray(got, dtype=np.float64).reshape(-1, ref.shape[-1])
    if not np.all(np.isfinite(got)):
        return float("inf")
    span = ref.max(axis=1) - ref.min(axis=1)
    span[span <= 0] = 1.0
    return float((np.abs(got - ref).max(axis=1) / span).max())


@dataclass
class Workload:
    """Inputs of one workload on the device: prompt lengths, packed prompt tokens, decode
    steps."""
    lens: List[int]
    tokens: "object"
    n_decode: int


@dataclass
class KnobReport:
    option: str
    classes: Tuple[str, ...]
    score: float
    baseline_ms: float
    candidates: Dict[int, dict] = field(default_factory=dict)
    chosen: int = 0
    accepted: bool = False


def _job(model, wl: Workload, nxt, reps: int) -> float:
    """Median whole-workload latency (ms) over `reps` runs after one warm-up."""
    import torch
    times = []
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for r in range(reps + 1):
        model.kv_reset()
        e0.record()
        model.prefill(wl.lens, wl.tokens, nxt)
        for _ in range(wl.n_decode):
            model.decode_step(nxt, nxt)
        e1.record()
        e1.synchronize()
        if r:
            times.append(e0.elapsed_time(e1))
    times.sort()
    return times[len(times) // 2]


def reference_outputs(model, wl: Workload, n_check: int):
    """Logits of the prefill and of `n_check` teacher-forced decode steps, and the greedy
    tokens that were fed (the output references of the in-model check)."""
    import torch
    B, V = len(wl.lens), model.mcfg.vocab
    model.kv_reset()
    logits = torch.empty(n_check + 1, B, V, dtype=torch.float32, device="cuda")
    toks = torch.empty(n_check + 1, B, dtype=torch.int32, device="cuda")
    model.prefill(wl.lens, wl.tokens, toks[0], logits[0])
    for k in range(n_check):
        model.decode_step(toks[k], toks[k + 1], logits[k + 1])
    torch.cuda.synchronize()
    return logits.cpu().numpy(), toks


def candidate_outputs(model, wl: Workload, ref_tokens, n_check: int):
    """Logits of the same inputs with the reference tokens fed back (teacher forcing)."""
    import torch
    B, V = len(wl.lens), model.mcfg.vocab
    model.kv_reset()
    logits = torch.empty(n_check + 1, B, V, dtype=torch.float32, device="cuda")
    out = torch.empty(B, dtype=torch.int32, device="cuda")
    model.prefill(wl.lens, wl.tokens, out, logits[0])
    for k in range(n_check):
        model.decode_step(ref_tokens[k], out, logits[k + 1])
    torch.cuda.synchronize()
    return logits.cpu().numpy()


def tune(model, wl: Workload, delta: float = 0.01, eps: float = 2e-2, reps: int = 3,
         n_check: int = 4, knobs=KNOBS, log=print) -> List[KnobReport]:
    """Greedy deployment-time acceptance over the option knobs, in hotspot order.

    Kernel classes are scored with Eq. 1 on the current model; knobs are visited in the order
    of the highest score among the classes they change.  For each knob every candidate value
    is set, checked against the current model's output references and timed on the whole
    workload; the best passing value is kept when it clears Eq. 3's margin, else the knob
    returns to its previous value.  Accepted values stay set for the following knobs (each
    accepted patch becomes part of the current model)."""
    import torch
    B = len(wl.lens)
    nxt = torch.empty(B, dtype=torch.int32, device="cuda")
    # Eq. 1 on the current model
    model.set_kernel_timing(True)
    model.kv_reset()
    e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    e[0].record()
    model.prefill(wl.lens, wl.tokens, nxt)
    e[1].record()
    for _ in range(wl.n_decode):
        model.decode_step(nxt, nxt)
    e[2].record()
    e[2].synchronize()
    kt = model.kernel_timing()
    model.set_kernel_timing(False)
    phase_ms = {"prefill": e[0].elapsed_time(e[1]), "decode": e[1].elapsed_time(e[2])}
    scores = hotspot_scores({k: v[1] for k, v in kt.items()}, phase_ms,
                            {"prefill": 1, "decode": wl.n_decode})
    log(f"[tuner] hotspot scores (Eq. 1): {json.dumps({k: round(v, 4) for k, v in scores.items()})}")
    order = sorted(knobs, key=lambda kn: -max(scores.get(c, 0.0) for c in kn[2]))
    reports = []
    for name, values, classes in order:
        current = model.get_option(name)
        ref_logits, ref_tokens = reference_outputs(model, wl, n_check)
        base = _job(model, wl, nxt, reps)
        rep = KnobReport(name, classes, max(scores.get(c, 0.0) for c in classes), base)
        ell, ok = {}, {}
        for v in values:
            if v == current:
                continue
            try:
                model.set_option(name, v)
            except Exception as ex:  # a value the model cannot take (e.g. a chunk below plan)
                rep.candidates[v] = {"safe": False, "error": str(ex)}
                continue
            got = candidate_outputs(model, wl, ref_tokens, n_check)
            err = max_row_error(ref_logits, got)
            t = _job(model, wl, nxt, reps)
            ell[v], ok[v] = t / base, err <= eps
            rep.candidates[v] = {"ms": round(t, 4), "ell": round(t / base, 4), "err": err,
                                 "ok": ok[v], "utility": round(search_utility(base, t, err, eps, True), 4)}
            model.set_option(name, current)
        best, accepted = accept(ell, ok, delta)
        rep.chosen, rep.accepted = (best, True) if accepted else (current, False)
        model.set_option(name, rep.chosen)
        log(f"[tuner] {name}: baseline {base:.3f} ms, candidates {json.dumps(rep.candidates)}"
            f" -> {'accept ' + str(best) if accepted else 'keep ' + str(current)}")
        reports.append(rep)
    return reports


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--config", default="125m")
    ap.add_argument("--delta", type=float, default=0.01, help="Eq. 3 acceptance margin")
    ap.add_argument("--eps", type=float, default=2e-2, help="in-model logit tolerance")
    ap.add_argument("--reps", type=int, default=3)
    ap.add_argument("--write", action="store_true",
                    help="store the accepted option values in accepted_options.json")
    ap.add_argument("--store", default=ACCEPTED_PATH,
                    help="file --write merges into (default: accepted_options.json here)")
    args = ap.parse_args()
    if args.write and not os.path.exists(args.store):
        # --write merges one workload's entry into the store; starting from an empty file
        # would drop every other workload's accepted options
        print(f"--write: the store {args.store} does not exist (copy the committed "
              "accepted_options.json there first)", file=sys.stderr)
        return 2
    import numpy as np
    import torch
    from synth import gen, get_config
    from synth import mamba as SM
    from synth import mamba2 as S2
    from synth import rglru as SR
    torch.cuda.set_device(0)
    if args.config in SR.RG_CONFIGS or args.config in SR.RG_TEST_CONFIGS:
        from paper_2608_21836_amd.binding import MambaModel, upload_mamba_weights
        cfg = SR.get_rg_config(args.config)
        lens, packed = gen.prompt_tokens(cfg)
        model = MambaModel(cfg, upload_mamba_weights(cfg, SR.weights(cfg)), max_batch=len(lens),
                           max_prefill_tokens=int(sum(lens)))
        knobs = RG_KNOBS
    elif args.config in S2.MAMBA2_CONFIGS or args.config in S2.MAMBA2_TEST_CONFIGS:
        from paper_2608_21836_amd.binding import MambaModel, upload_mamba_weights
        cfg = S2.get_mamba2_config(args.config)
        lens, packed = gen.prompt_tokens(cfg)
        model = MambaModel(cfg, upload_mamba_weights(cfg, S2.weights(cfg)), max_batch=len(lens),
                           max_prefill_tokens=int(sum(lens)))
        knobs = MAMBA2_KNOBS
    elif args.config in SM.MAMBA_CONFIGS or args.config in SM.MAMBA_TEST_CONFIGS:
        from paper_2608_21836_amd.binding import MambaModel, upload_mamba_weights
        cfg = SM.get_mamba_config(args.config)
        lens, packed = gen.prompt_tokens(cfg)
        model = MambaModel(cfg, upload_mamba_weights(cfg, SM.weights(cfg)), max_batch=len(lens),
                           max_prefill_tokens=int(sum(lens)))
        knobs = MAMBA_KNOBS
    else:
        from paper_2608_21836_amd.binding import Model, to_device
        cfg = get_config(args.config)
        lens, packed = gen.prompt_tokens(cfg)
        w = {n: to_device(a, cfg.dtype) for n, a in gen.iter_weights_parallel(cfg, 16)}
        w.update({k: to_device(v, cfg.dtype) for k, v in gen.gains(cfg).items()})
        model = Model(cfg, w, max_batch=len(lens), max_prefill_tokens=int(sum(lens)),
                      max_ctx=max(lens) + cfg.n_decode)
        del w
        knobs = KNOBS
    wl = Workload(list(lens), torch.from_numpy(np.asarray(packed, dtype=np.int32)).cuda(),
                  cfg.n_decode)
    reports = tune(model, wl, args.delta, args.eps, args.reps, knobs=knobs)
    result = {"workload": cfg.name, "delta": args.delta, "options": model.options(),
              "knobs": [{"option": r.option, "score": round(r.score, 4),
                         "baseline_ms": round(r.baseline_ms, 4), "chosen": r.chosen,
                         "accepted": r.accepted, "candidates": r.candidates}
                        for r in reports]}
    print(json.dumps(result))
    model.close()
    if args.write:
        with open(args.store) as f:   # checked to exist before tuning
            store = json.load(f)
        accepted = {r.option: r.chosen for r in reports if r.accepted}
        store[cfg.name] = {
            "delta": args.delta,
            "options": accepted,
            "ell": {r.option: r.candidates[r.chosen]["ell"] for r in reports if r.accepted},
            "nondeterministic": sorted(o for o, v in accepted.items()
                                       if (o, v) in NONDETERMINISTIC)}
        with open(args.store, "w") as f:
            json.dump(store, f, indent=1, sort_keys=True)
            f.write("\n")
    return 0


if __name__ == "__main__":
    sys.exit(main())
