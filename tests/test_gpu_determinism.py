"""Run-to-run determinism of the HIP path: the backward's weight-gradient work runs on a
second stream concurrently with the input-gradient path, and every reduction is in a fixed
order, so identical calls must give bit-identical outputs.  A race between the two streams
shows up here as outputs that differ between calls (it need not show up as a parity error)."""
import numpy as np
import pytest

from gpu_helpers import gpu_blocks, host_inputs
from paper_2607_02829_amd import inputs

pytestmark = pytest.mark.gpu


def _bits(a):
    a = np.ascontiguousarray(a)
    return a.view(np.uint8) if a.dtype.kind == "f" else a


def _flat(out):
    """name -> array for every output (per-block gradients as b<i>.<param>)."""
    flat = {}
    for k, v in out.items():
        if v is None:
            continue
        if k == "grads":
            for i, g in enumerate(v):
                flat.update({f"b{i}.{p}": a for p, a in g.items()})
        else:
            flat[k] = v
    return flat


@pytest.mark.parametrize("name", ["d025", "edm"])
def test_blocks_fwd_bwd_bitwise_repeatable(name):
    w = inputs.WORKLOADS[name]
    n_blocks = w.n_blocks if name == "d025" else 4
    h, params, cond, dh = host_inputs(w, n_blocks, randomise_affine=True, S=w.K)
    print(f"[{name}] S={w.K} blocks={n_blocks}: three identical forward+backward calls", flush=True)
    runs = [_flat(gpu_blocks(w, w.K, h, params, cond, dh)) for _ in range(3)]
    keys = list(runs[0])
    assert "dh_in" in keys and len(keys) > 10
    for r in runs[1:]:
        diff = [k for k in keys if not np.array_equal(_bits(runs[0][k]), _bits(r[k]))]
        assert not diff, f"outputs differ between identical calls: {diff[:8]}"
