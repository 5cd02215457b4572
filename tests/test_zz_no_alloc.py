"""The allocation-free selection entry point (sr_select_indices_noalloc) against
sr_select_indices with a caller scratch buffer: identical indices, bit for bit, on two calls
in a row on one GPU (the second with fewer tokens, so stale scores of the first call lie past
the second's extent), for the top-k and the random selector, plus the size limit."""
import numpy as np
import pytest

from paper_2607_02829_amd import abi, device, inputs

pytestmark = pytest.mark.gpu


def _fields(w):
    xt = device.to_device(inputs.to_storage(inputs.token_field(w, 0), w.dtype))
    xp = device.to_device(inputs.to_storage(inputs.token_field(w, 1), w.dtype))
    return xt, xp


def _both(w, K, kind, shared=0, step=0):
    import torch
    cfg = device.config_for(w, idx_shared=shared)
    rows = 1 if shared else w.B
    xt, xp = _fields(w) if kind == abi.SR_SEL_TOPK_DIFFNORM else (None, None)
    ref = torch.full((rows, K), -1, dtype=torch.int32, device="cuda")
    got = torch.full((rows, K), -1, dtype=torch.int32, device="cuda")
    scratch = torch.empty(max(abi.sr_select_scratch_bytes(cfg, kind), 16), dtype=torch.uint8, device="cuda")
    abi.sr_select_indices(cfg, K, kind, 11, step, xt, xp, ref, scratch)
    abi.sr_select_indices_noalloc(cfg, K, kind, 11, step, xt, xp, got)
    torch.cuda.synchronize()
    return got.cpu().numpy(), ref.cpu().numpy()


def test_noalloc_topk_matches_scratch_entry_point_two_calls():
    big = inputs.WORKLOADS["edm"]                                  # 2 x 8192 tokens, D = 1024, bf16
    small = inputs.small("noalloc_small", B=1, Hg=30, Wg=50, D=256, H=4, F=1024)   # 1500 tokens
    for w, K in ((big, big.K), (small, 377)):
        print(f"[noalloc topk] B={w.B} L={w.L} D={w.D} K={K} {w.dtype}", flush=True)
        got, ref = _both(w, K, abi.SR_SEL_TOPK_DIFFNORM)
        assert np.array_equal(got, ref)
        assert np.all(np.diff(got, axis=1) > 0)


def test_noalloc_topk_fp32_shared_and_random():
    w = inputs.small("noalloc_f32", B=3, Hg=20, Wg=37, D=128, H=2, F=512, dtype="f32")
    got, ref = _both(w, 200, abi.SR_SEL_TOPK_DIFFNORM, shared=1)
    assert np.array_equal(got, ref)
    got, ref = _both(w, 99, abi.SR_SEL_RANDOM, step=4)
    assert np.array_equal(got, ref)


def test_noalloc_rejects_more_tokens_than_its_array():
    w = inputs.small("noalloc_limit", B=2, Hg=1, Wg=abi.SR_SELECT_NOALLOC_MAX_TOKENS // 2 + 1, D=64, H=1, F=64)
    cfg = device.config_for(w)
    fake = 1 << 40   # never dereferenced: the size check fails first
    with pytest.raises(abi.SrError) as ei:
        abi.sr_select_indices_noalloc(cfg, 10, abi.SR_SEL_TOPK_DIFFNORM, 0, 0, fake, fake, fake, stream=0)
    assert ei.value.status == abi.SR_EUNSUPPORTED
    assert "without allocation" in abi.sr_last_error()
