"""Host-side rules of the tuner: the hotspot score (Eq. 1), the search utility (Eq. 2) and
deployment-time acceptance (Eq. 3), on hand-made inputs with known answers."""
import math

import numpy as np
import pytest

from paper_2608_21836_amd import tuner


def test_hotspot_score_weights_phases_by_their_share():
    # prefill 10 ms (1 invocation), decode 30 ms over 10 steps: w = 0.25 / 0.75
    kernel_ms = {("prefill", "gemm"): 6.0, ("prefill", "attn"): 4.0,
                 ("decode", "gemm"): 24.0, ("decode", "attn"): 6.0}
    s = tuner.hotspot_scores(kernel_ms, {"prefill": 10.0, "decode": 30.0},
                             {"prefill": 1, "decode": 10})
    assert s["gemm"] == pytest.approx(0.25 * 0.6 + 0.75 * 0.8)
    assert s["attn"] == pytest.approx(0.25 * 0.4 + 0.75 * 0.2)
    assert list(s) == ["gemm", "attn"]          # ranked
    # scores of a complete partition of both phases sum to 1
    assert sum(s.values()) == pytest.approx(1.0)


def test_hotspot_score_ignores_a_phase_that_did_not_run():
    s = tuner.hotspot_scores({("prefill", "a"): 2.0, ("decode", "a"): 1.0},
                             {"prefill": 4.0, "decode": 0.0}, {"prefill": 1, "decode": 0})
    assert s == {"a": pytest.approx(0.5)}


def test_search_utility():
    assert tuner.search_utility(10.0, 5.0, 1e-3, 1e-2, True) == pytest.approx(2.0)
    assert tuner.search_utility(10.0, 5.0, 2e-2, 1e-2, True) == 0.0      # wrong
    assert tuner.search_utility(10.0, 5.0, 1e-3, 1e-2, False) == 0.0     # unsafe
    assert tuner.search_utility(10.0, 5.0, math.nan, 1e-2, True) == 0.0  # NaN error fails


def test_acceptance_needs_a_passing_candidate_that_clears_delta():
    ell = {"a": 0.97, "b": 0.90, "c": 0.995}
    # b is fastest but fails the in-model check: a is the best passing one
    assert tuner.accept(ell, {"a": True, "b": False, "c": True}, 0.02) == ("a", True)
    # a does not clear a 5 % margin
    assert tuner.accept(ell, {"a": True, "b": False, "c": True}, 0.05) == ("a", False)
    assert tuner.accept(ell, {"a": False, "b": False, "c": False}, 0.0) == (None, False)
    # delta = 0 accepts a tie with the current model
    assert tuner.accept({"x": 1.0}, {"x": True}, 0.0) == ("x", True)


def test_max_row_error_is_relative_to_each_reference_row():
    ref = np.array([[[0.0, 1.0, 2.0]], [[0.0, 10.0, 20.0]]])
    got = ref.copy()
    got[0, 0, 1] += 0.02      # 1 % of row 0's range
    got[1, 0, 2] -= 0.1       # 0.5 % of row 1's range
    assert tuner.max_row_error(ref, got) == pytest.approx(0.01)
    got[1, 0, 0] = np.nan
    assert tuner.max_row_error(ref, got) == math.inf


def test_every_knob_default_is_listed_first():
    # the first candidate of each knob is the library default (ll.h)
    defaults = {"prefill_tile": 0, "prefill_splitk": 1, "decode_splitk": 1,
                "attn_decode_chunk": 0, "decode_fused": 0, "decode_graph": 1}
    assert {k[0]: k[1][0] for k in tuner.KNOBS} == defaults


def test_accepted_options_cover_every_bench_workload():
    """Every bench workload keeps its entry in the store (a --write of one workload merges into
    the file and never drops the others); option names and values are ones the tuner knows, and
    the non-deterministic variants are recorded as such."""
    import json
    with open(tuner.ACCEPTED_PATH) as f:
        store = json.load(f)
    assert set(store) == {"125m", "1b-gqa", "7b-mha", "8b-gqa", "mamba-130m", "mamba2-130m",
                          "rglru-2b"}
    known = {}
    for table in (tuner.KNOBS, tuner.MAMBA_KNOBS, tuner.MAMBA2_KNOBS, tuner.RG_KNOBS):
        for name, values, _ in table:
            known.setdefault(name, set()).update(values)
    for wl, entry in store.items():
        for name, value in entry["options"].items():
            assert value in known[name], (wl, name, value)
        assert set(entry["ell"]) == set(entry["options"]), wl
        assert all(entry["ell"][k] <= 1 - entry["delta"] for k in entry["ell"]), wl
        nd = {k for k, v in entry["options"].items() if (k, v) in tuner.NONDETERMINISTIC}
        assert set(entry["nondeterministic"]) == nd, wl
        assert tuner.deterministic_options(wl) == {k: v for k, v in entry["options"].items()
                                                   if k not in nd}


def test_write_refuses_a_missing_store(tmp_path, monkeypatch):
    import sys
    monkeypatch.setattr(sys, "argv", ["tuner", "--config", "125m", "--write",
                                      "--store", str(tmp_path / "none.json")])
    assert tuner.main() == 2
