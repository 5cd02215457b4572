"""Host-side checks of the C ABI: the library loads, exports every symbol the header
declares, sizes workspaces, and rejects bad arguments before launching anything."""
import os
import re
import subprocess

import pytest

from paper_2607_02829_amd import abi

pytestmark = pytest.mark.cpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sr.h")


def _lib_or_skip():
    try:
        return abi.lib()
    except abi.SrLibraryMissing as e:
        pytest.skip(str(e))


def test_header_symbols_exported():
    _lib_or_skip()
    declared = set(re.findall(r"SR_API\s+[\w\s\*]+?\b(sr_\w+)\s*\(", open(HEADER).read()))
    assert declared == set(abi.EXPORTS)
    out = subprocess.run(["nm", "-D", "--defined-only", abi.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (sr_\w+)", out))
    assert declared <= exported, declared - exported


def _cfg(**kw):
    base = dict(B=2, L=100, D=256, H=4, F=1024, n_blocks=2, dtype=abi.SR_BF16, kind=abi.SR_BLOCK_PRELN,
                ln_eps=1e-6, idx_shared=0)
    base.update(kw)
    return abi.SrConfig(**base)


def test_workspace_sizes_scale_with_tokens():
    _lib_or_skip()
    s1, c1 = abi.sr_workspace_bytes(_cfg(), 25)
    s2, c2 = abi.sr_workspace_bytes(_cfg(), 100)
    assert 0 < s1 < s2 and 0 < c1 < c2
    # saved activations: per token and block the fp32 block input and attention residual (4D + 4D),
    # q, k, v and O (2 x 4D) and the FC1 pre-activation (2F) at least; the LayerNorm outputs and
    # GELU(z) are forward temporaries shared by all blocks (recomputed in the backward)
    assert s2 >= 2 * 2 * 100 * (256 * 16 + 1024 * 2)
    s3, _ = abi.sr_workspace_bytes(_cfg(n_blocks=3), 100)
    s4, _ = abi.sr_workspace_bytes(_cfg(n_blocks=4), 100)
    assert s4 - s3 == s3 - s2 > 0                     # a fixed size per block
    assert s2 - 2 * (s3 - s2) >= 2 * 100 * (256 + 1024) * 2   # plus the shared temporaries


def test_stack_buffer_limit_counts_the_calls_rows():
    # 0.25 deg shape at B = 16: the routed stack's K = 4050 rows per sample stay below the 2 GiB
    # of its fp32 buffers (16 x 4050 x 4096 x 4 bytes), the dense one's L = 16200 rows do not
    _lib_or_skip()
    cfg = _cfg(B=16, L=16200, D=1024, H=16, F=4096, n_blocks=12)
    saved, scratch = abi.sr_workspace_bytes(cfg, 4050)
    assert saved > 0 and scratch > 0
    with pytest.raises(abi.SrError) as ei:
        abi.sr_workspace_bytes(cfg, 16200)
    assert ei.value.status == abi.SR_EUNSUPPORTED and "2 GiB" in abi.sr_last_error()


@pytest.mark.parametrize("kw,status", [
    (dict(D=250), abi.SR_ESHAPE),          # D % H != 0  (250 % 4)
    (dict(D=192, H=4, F=768), abi.SR_EUNSUPPORTED),   # head dim 48
    (dict(dtype=7), abi.SR_EDTYPE),
    (dict(kind=3), abi.SR_EINVAL),
    (dict(B=0), abi.SR_EINVAL),
    (dict(D=96, H=3), abi.SR_EUNSUPPORTED),  # D % 64
])
def test_bad_config_rejected(kw, status):
    _lib_or_skip()
    with pytest.raises(abi.SrError) as ei:
        abi.sr_workspace_bytes(_cfg(**kw), 10)
    assert ei.value.status == status
    assert abi.sr_last_error()


def test_bad_call_arguments_rejected_before_launch():
    _lib_or_skip()
    cfg = _cfg()
    fake = 1 << 40          # aligned, never dereferenced: validation fails first
    with pytest.raises(abi.SrError) as ei:
        abi.sr_gather(cfg, 101, fake, fake, fake, stream=0)       # K > L
    assert ei.value.status == abi.SR_ESHAPE
    with pytest.raises(abi.SrError) as ei:
        abi.sr_gather(cfg, 10, fake + 2, fake, fake, stream=0)    # misaligned x
    assert ei.value.status == abi.SR_EALIGN
    with pytest.raises(abi.SrError) as ei:
        abi.sr_scatter_delta(cfg, 10, None, fake, None, fake, stream=0)
    assert ei.value.status == abi.SR_EINVAL
    with pytest.raises(abi.SrError) as ei:
        abi.sr_select_indices(cfg, 0, abi.SR_SEL_RANDOM, 1, 0, None, None, fake, stream=0)
    assert ei.value.status == abi.SR_ESHAPE
    with pytest.raises(abi.SrError) as ei:
        abi.sr_select_indices(cfg, 10, abi.SR_SEL_TOPK_DIFFNORM, 1, 0, fake, fake, fake, fake, stream=0)
    assert ei.value.status == abi.SR_EWORKSPACE or ei.value.status == abi.SR_EINVAL
    # blocks: workspace too small
    params = (abi.SrBlockParams * 2)()
    for i in range(2):
        for n in abi.PARAM_FIELDS:
            setattr(params[i], n, fake)
    lib = abi.lib()
    import ctypes
    st = lib.sr_sparse_blocks_fwd(ctypes.byref(cfg), 25, params, None, fake, fake + 4096, fake, 16, None, 0, None)
    assert st == abi.SR_EWORKSPACE
    st = lib.sr_sparse_blocks_fwd(ctypes.byref(cfg), 25, params, None, fake, fake, fake, 1 << 40, None, 0, None)
    assert st == abi.SR_EINVAL        # h_out aliases h_in
    ada = _cfg(kind=abi.SR_BLOCK_ADALN)
    st = lib.sr_sparse_blocks_fwd(ctypes.byref(ada), 25, params, None, fake, fake + 4096, fake, 1 << 40, None, 0, None)
    assert st == abi.SR_EINVAL        # adaLN without cond


def test_new_entry_points_reject_bad_arguments_before_launch():
    _lib_or_skip()
    import ctypes
    cfg = _cfg()
    fake = 1 << 40
    lib = abi.lib()
    # attention column sums: block outside [0, n_blocks), S > L, saved too small
    assert lib.sr_attention_colsums(ctypes.byref(cfg), 25, fake, 1 << 40, 2, fake, None) == abi.SR_EINVAL
    assert lib.sr_attention_colsums(ctypes.byref(cfg), 101, fake, 1 << 40, 0, fake, None) == abi.SR_ESHAPE
    assert lib.sr_attention_colsums(ctypes.byref(cfg), 25, fake, 16, 0, fake, None) == abi.SR_EWORKSPACE
    # top-K over score planes: parts < 1, K > L, NULL planes
    assert lib.sr_select_topk_scores(ctypes.byref(cfg), 10, fake, 0, fake, None) == abi.SR_EINVAL
    assert lib.sr_select_topk_scores(ctypes.byref(cfg), 101, fake, 4, fake, None) == abi.SR_ESHAPE
    assert lib.sr_select_topk_scores(ctypes.byref(cfg), 10, None, 4, fake, None) == abi.SR_EINVAL
    # fused routed step: K > L, NULL idx, saved too small, backward without scratch
    params = (abi.SrBlockParams * 2)()
    for i in range(2):
        for n in abi.PARAM_FIELDS:
            setattr(params[i], n, fake)
    grads = (abi.SrBlockGrads * 2)()
    assert lib.sr_routed_blocks_fwd(ctypes.byref(cfg), 101, fake, params, None, fake, fake, 1 << 40, None) == abi.SR_ESHAPE
    assert lib.sr_routed_blocks_fwd(ctypes.byref(cfg), 25, None, params, None, fake, fake, 1 << 40, None) == abi.SR_EINVAL
    assert lib.sr_routed_blocks_fwd(ctypes.byref(cfg), 25, fake, params, None, fake, fake, 16, None) == abi.SR_EWORKSPACE
    st = lib.sr_routed_blocks_bwd(ctypes.byref(cfg), 25, fake, params, None, fake, 1 << 40, fake, grads, None, None, 0,
                                  None)
    assert st in (abi.SR_EINVAL, abi.SR_EWORKSPACE)
    assert abi.sr_last_error()


def test_cross_attention_rejects_bad_arguments_before_launch():
    _lib_or_skip()
    import ctypes
    cfg = _cfg()
    fake = 1 << 40
    lib = abi.lib()
    assert lib.sr_cross_attention_fwd(ctypes.byref(cfg), 0, 10, fake, fake, fake, fake, None) == abi.SR_ESHAPE
    assert lib.sr_cross_attention_fwd(ctypes.byref(cfg), 10, 10, None, fake, fake, fake, None) == abi.SR_EINVAL
    assert lib.sr_cross_attention_bwd(ctypes.byref(cfg), 10, 0, fake, fake, fake, fake, fake, fake, fake, fake,
                                      None) == abi.SR_ESHAPE
    assert lib.sr_cross_attention_bwd(ctypes.byref(cfg), 10, 10, fake, fake, fake, fake, fake, fake, fake, None,
                                      None) == abi.SR_EINVAL


def test_layernorm_and_modulation_pointers_alignment_checked():
    # the row kernels read gamma / beta and W_ada / b_ada with vector loads: a misaligned
    # pointer is rejected before any launch
    _lib_or_skip()
    import ctypes
    fake = 1 << 40
    lib = abi.lib()
    for kind, field in ((abi.SR_BLOCK_PRELN, "ln1_w"), (abi.SR_BLOCK_PRELN, "ln2_b"),
                        (abi.SR_BLOCK_ADALN, "w_ada"), (abi.SR_BLOCK_ADALN, "b_ada")):
        cfg = _cfg(kind=kind)
        params = (abi.SrBlockParams * 2)()
        for i in range(2):
            for n in abi.PARAM_FIELDS:
                setattr(params[i], n, fake)
        setattr(params[1], field, fake + 2)
        st = lib.sr_sparse_blocks_fwd(ctypes.byref(cfg), 25, params, fake, fake, fake + 4096, fake, 1 << 40, None,
                                      0, None)
        assert st == abi.SR_EALIGN, (kind, field)
        assert field.split("_")[0] in abi.sr_last_error() or "aligned" in abi.sr_last_error()


def test_cross_attention_ignores_block_fields():
    # only B, D, H and dtype of cfg are read: block fields that would be invalid for the block
    # calls do not make the asymmetric attention fail
    _lib_or_skip()
    import ctypes
    fake = 1 << 40
    lib = abi.lib()
    cfg = _cfg(L=0, F=0, n_blocks=-1, kind=9, ln_eps=0.0, idx_shared=5)
    # the first failure is the one of the call's own arguments (Sq = 0), not of the ignored fields
    assert lib.sr_cross_attention_fwd(ctypes.byref(cfg), 0, 10, fake, fake, fake, fake, None) == abi.SR_ESHAPE
    assert lib.sr_cross_attention_fwd(ctypes.byref(cfg), 10, 10, None, fake, fake, fake, None) == abi.SR_EINVAL
    assert lib.sr_cross_attention_fwd(ctypes.byref(_cfg(D=96, H=3)), 10, 10, fake, fake, fake, fake,
                                      None) == abi.SR_EUNSUPPORTED


def test_mfma_probe_rejects_null_arguments():
    L = _lib_or_skip()
    assert L.sr_probe_mfma_rate(None, None, None) == abi.SR_EINVAL
    assert "NULL" in abi.lib().sr_last_error().decode()
