"""GPU run of the step-level serving loop (KV append + mixed attention per step,
four policies). Every policy must see the same batches: the same decode-token
count and the same number of prompts finishing prefill; the controller's
steps must be serial, one-launch or a valid candidate split."""
import argparse

import pytest

from paper_2606_04415_amd import serve_sim

from gpu_common import log

pytestmark = pytest.mark.gpu


def test_policies_replay_the_same_stream():
    args = argparse.Namespace(steps=24, seed=3, warm=40, max_active=48, chunk=2048, burst=8, burst_every=10,
                              rate=0.3, fixed_decode_cus=128, per_mix_limits=False)
    res = {}
    for pol in ("serial", "fixed", "controller", "fused"):
        log(f"serve loop: mix long, policy {pol}, 24 steps")
        res[pol] = serve_sim.simulate("long", pol, args, profile=None)
    toks = {p: r["tpot_ms"]["tokens"] for p, r in res.items()}
    firsts = {p: r["ttft_ms"]["n"] for p, r in res.items()}
    assert len(set(toks.values())) == 1 and len(set(firsts.values())) == 1, (toks, firsts)
    assert toks["serial"] > 0 and firsts["serial"] > 0
    assert set(res["serial"]["splits"]) == {"serial"}
    for k in res["controller"]["splits"]:
        assert k in ("serial", "fused") or k in {f"{256 - c}:{c}" for c in range(32, 256, 32)}
    assert set(res["fused"]["splits"]) <= {"serial", "fused"} and "fused" in res["fused"]["splits"]
    for r in res.values():
        assert r["total_ms"] > 0 and r["step_ms"]["max"] < 50.0


def test_timeslice_policy_runs_one_phase_per_step():
    args = argparse.Namespace(steps=24, seed=3, warm=40, max_active=48, chunk=2048, burst=8, burst_every=10,
                              rate=0.3, fixed_decode_cus=128, per_mix_limits=False, decode_share=0.5, ts_decay=0.9)
    log("serve loop: mix long, time-sliced at 40% decode, 24 steps")
    r = serve_sim.simulate("long", "timeslice:0.4", args, profile=None)
    assert set(r["splits"]) == {"decode", "prefill"}, r["splits"]
    assert set(r["device_ms"]) == {"decode", "prefill"}, r["device_ms"]
    assert r["tpot_ms"]["tokens"] > 0 and r["ttft_ms"]["n"] > 0
    # a time-sliced decode token waits for the prefill steps in between
    assert r["tpot_ms"]["p90"] >= r["step_ms"]["p50"] * 0.5
