"""The CU-sweep profiler (the MI355X analog of the paper's bandwidth-vs-
compute-units profile, Sec. 2 Fig. 2, and its split sweeps, Sec. 4.3):
every CU count measured, decode bandwidth rising with the CU count until it
saturates, prefill rate rising, and at every split the co-run output
bit-identical to the serial output of the same plan."""
import pytest

from paper_2606_04415_amd.cusweep import profile_from, sweep

from gpu_common import log

pytestmark = pytest.mark.gpu


def test_sweep_mixed_curves_and_bit_identity():
    counts = [32, 64, 128, 192, 256]
    log(f"CU sweep of the mixed step over {counts}")
    r = sweep("mixed", reps=5, pools=2, counts=counts, corun=True, check_outputs=True)
    assert sorted(r["decode"]) == counts and sorted(r["prefill"]) == counts
    dec = [r["decode"][c]["GBps"] for c in counts]
    pre = [r["prefill"][c]["TFLOPs"] for c in counts]
    log(f"decode GB/s {dec}; prefill TFLOP/s {pre}")
    # decode: rising while far from saturation, and the full device within 10% of the best
    assert dec[0] < dec[1] < dec[2] and dec[-1] >= 0.9 * max(dec)
    assert pre[0] < pre[1] < pre[2] and pre[-1] >= 0.9 * max(pre)
    assert sorted(r["corun_step_us"]) == counts[:-1]
    assert all(r["corun_bitwise_equals_serial"].values()) and len(r["corun_bitwise_equals_serial"]) == 4
    assert r["best_split"]["cus_decode"] in counts
    cus, d, p = profile_from(r)
    assert cus == counts and d == dec and p == pre
