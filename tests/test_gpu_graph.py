"""HIP graph capture of the fused routed step (selection, sr_routed_blocks_fwd,
sr_routed_blocks_bwd, with the backward's second-stream weight gradients forked and joined
inside the capture): every replay, with eager copies and synchronisations between replays,
equals the eager step bit for bit."""
import pytest

from paper_2607_02829_amd import abi, device, inputs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("w", [inputs.small("graph_s", Hg=10, Wg=21), inputs.WORKLOADS["b5625"]],
                         ids=["small_bf16", "b5625"])
def test_graph_replays_equal_eager(w):
    import torch
    nb, K = w.n_blocks, w.K
    print(f"[graph {w.name}] B={w.B} L={w.L} K={K} blocks={nb}", flush=True)
    params = inputs.params_to_storage(inputs.block_params(w, nb, randomise_affine=True), w.dtype)
    cfg = device.config_for(w, n_blocks=nb)
    dp = device.DeviceParams(params, w.kind)
    gr = device.DeviceGrads(w, nb)
    x0 = device.to_device(inputs.to_storage(inputs.token_field(w), w.dtype))
    g0 = device.to_device(inputs.to_storage(inputs.upstream_grad(w), w.dtype))
    x, g = x0.clone(), g0.clone()
    idx = torch.empty((w.B, K), dtype=torch.int32, device="cuda")
    saved, scratch = device.workspace(cfg, K)

    def step():
        abi.sr_select_indices(cfg, K, abi.SR_SEL_RANDOM, 9, 4, None, None, idx)
        abi.sr_routed_blocks_fwd(cfg, K, idx, dp.array, None, x, saved)
        abi.sr_routed_blocks_bwd(cfg, K, idx, dp.array, None, saved, g, gr.array, None, scratch)

    # eager reference (the first call also creates the library's second stream and events)
    step()
    torch.cuda.synchronize()
    want_x, want_g = x.clone(), g.clone()
    want_gr = [{k: v.clone() for k, v in t.items()} for t in gr.tensors]

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):   # warm-up on the capture stream
        x.copy_(x0); g.copy_(g0)
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    x.copy_(x0); g.copy_(g0)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for rep in range(3):
        x.copy_(x0); g.copy_(g0)
        for t in gr.tensors:
            for v in t.values():
                v.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(x.view(torch.int16), want_x.view(torch.int16)), rep
        assert torch.equal(g.view(torch.int16), want_g.view(torch.int16)), rep
        for i, (a, b) in enumerate(zip(gr.tensors, want_gr)):
            for k in a:
                assert torch.equal(a[k].view(torch.int32), b[k].view(torch.int32)), (rep, i, k)
        # eager work between replays
        step()
        torch.cuda.synchronize()
    print(f"[graph {w.name}] 3 replays equal the eager step", flush=True)
