"""The routed step at a batch the stack-buffer limit used to reject: B = 16 samples of the
0.25 deg token grid (L = 16200, K = 4050, D = 1024, two blocks).  Samples interact only through
the weight gradients, so each sample's updated tokens and input gradient must equal, bit for bit,
those of a B = 1 call on that sample alone with its index set -- checked for the first and the
last sample, whose rows lie furthest into the buffers."""
import numpy as np
import pytest

from paper_2607_02829_amd import abi, device, inputs

pytestmark = pytest.mark.gpu


def _step(w, x, g, idx, params):
    import torch
    cfg = device.config_for(w)
    dp = device.DeviceParams(params, w.kind)
    gr = device.DeviceGrads(w, w.n_blocks)
    xd, gd = device.to_device(x), device.to_device(g)
    idd = torch.from_numpy(np.ascontiguousarray(idx)).to("cuda")
    saved, scratch = device.workspace(cfg, w.K)
    abi.sr_routed_blocks_fwd(cfg, w.K, idd, dp.array, None, xd, saved)
    abi.sr_routed_blocks_bwd(cfg, w.K, idd, dp.array, None, saved, gd, gr.array, None, scratch)
    torch.cuda.synchronize()
    out = device.to_host(xd), device.to_host(gd)
    del saved, scratch, xd, gd
    torch.cuda.empty_cache()
    return out


def test_routed_step_at_batch_16_matches_single_samples():
    import torch
    w = inputs.WORKLOADS["d025"].with_(B=16, n_blocks=2)
    rng = np.random.default_rng(11)
    x = inputs.to_storage(rng.standard_normal((w.B, w.L, w.D), dtype=np.float32), w.dtype)
    g = inputs.to_storage(rng.standard_normal((w.B, w.L, w.D), dtype=np.float32), w.dtype)
    params = inputs.params_to_storage(inputs.block_params(w), w.dtype)
    cfg = device.config_for(w)
    idx = torch.empty((w.B, w.K), dtype=torch.int32, device="cuda")
    abi.sr_select_indices(cfg, w.K, abi.SR_SEL_RANDOM, 21, 4, None, None, idx)
    idx = idx.cpu().numpy()
    print(f"[B=16] routed step, L={w.L} K={w.K} D={w.D} blocks={w.n_blocks}", flush=True)
    x16, g16 = _step(w, x, g, idx, params)
    bits = lambda a: np.ascontiguousarray(a).view(np.uint8)
    w1 = w.with_(B=1)
    for b in (0, w.B - 1):
        print(f"[B=16] sample {b} alone", flush=True)
        x1, g1 = _step(w1, x[b:b + 1], g[b:b + 1], idx[b:b + 1], params)
        assert np.array_equal(bits(x1[0]), bits(x16[b])), f"sample {b}: tokens"
        assert np.array_equal(bits(g1[0]), bits(g16[b])), f"sample {b}: input gradient"
    # the call really changed the routed rows of the last sample
    assert not np.array_equal(bits(x16[-1]), bits(x[-1]))
