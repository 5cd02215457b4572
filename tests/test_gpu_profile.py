"""GPU tests of the launch timing (sr_profile_start / sr_profile_stop): the events bound to the
kernels at launch, nested inside the backward's fork points, leave every result bit for bit as
it is without timing (filtered: the second stream stays; unfiltered: the weight gradients run on
the caller's stream), and every timed group reports a positive time."""
import numpy as np
import pytest

from paper_2607_02829_amd import abi, inputs

from test_gpu_routed_fused import _bits, _run

pytestmark = pytest.mark.gpu

CASES = {
    "bf16": (inputs.small("pf_a", Hg=10, Wg=21), 2, 52, 0),
    "adaln_bf16": (inputs.small("pf_b", Hg=10, Wg=21, kind="adaln"), 2, 50, 0),
}


def _same(a, b):
    assert np.array_equal(_bits(a["x"]), _bits(b["x"]))
    assert np.array_equal(_bits(a["g"]), _bits(b["g"]))
    for ga, gb in zip(a["grads"], b["grads"]):
        for k in ga:
            assert np.array_equal(_bits(ga[k]), _bits(gb[k])), k
    if "dcond" in a:
        assert np.array_equal(_bits(a["dcond"]), _bits(b["dcond"]))


@pytest.mark.parametrize("case", list(CASES))
@pytest.mark.parametrize("name_filter", ["attn_bwd_dkv", "ln_bwd", ""])
def test_timing_leaves_results_unchanged(case, name_filter):
    w, nb, K, shared = CASES[case]
    print(f"[profile {case} filter={name_filter!r}]", flush=True)
    plain = _run(w, nb, K, shared, True)[0]
    abi.sr_profile_start(name_filter)
    try:
        timed = _run(w, nb, K, shared, True)[0]
    finally:
        prof = abi.sr_profile_stop()
    _same(plain, timed)
    assert prof, "no launch group was timed"
    for name, rec in prof.items():
        assert name_filter in name
        assert rec["launches"] >= 1 and rec["ms"] >= 0.0, (name, rec)
    if name_filter:   # per block: one dK/dV launch group, two LayerNorm backwards
        assert prof[name_filter]["launches"] == {"attn_bwd_dkv": 1, "ln_bwd": 2}[name_filter] * nb
        assert prof[name_filter]["ms"] > 0.0
    else:
        assert prof["attn_bwd_dkv"]["ms"] > 0.0 and prof["ln_bwd"]["ms"] > 0.0
