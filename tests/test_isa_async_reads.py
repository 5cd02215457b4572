"""The explicit (inline-assembly) LDS fragment reads of the MFMA kernels are only sound if the
compiler never touches their destination registers before the wait that retires them.  build.py
keeps the gfx950 assembly of the sources that use them and refuses a library that breaks this;
here the scan itself is pinned on hand-written sequences, and the kept assembly is rescanned."""
import os

import pytest

from paper_2607_02829_amd import build
from paper_2607_02829_amd.isa_scan import kernel_hazards


def test_scan_flags_a_copy_of_an_in_flight_destination():
    asm = """_Zk:
\tds_read_b128 a[0:3], v1 offset:0
\tv_accvgpr_read_b32 v4, a2
\ts_waitcnt lgkmcnt(0)
\tv_accvgpr_read_b32 v5, a3
.Lfunc_end0:
_Zok:
\tds_read_b128 v[0:3], v9 offset:0
\tds_read_b128 v[4:7], v9 offset:64
\ts_waitcnt lgkmcnt(1)
\tv_add_u32 v10, v0, v1
\ts_waitcnt lgkmcnt(0)
\tv_add_u32 v11, v4, v5
.Lfunc_end1:
_Zw:
\tds_read_b64_tr_b16 v[2:3], v9 offset:0
\tv_mov_b32 v3, 0
\ts_waitcnt lgkmcnt(0)
.Lfunc_end2:
"""
    # a copy before the wait, a read retired by lgkmcnt(1) (in order), a write into a pending register
    assert kernel_hazards(asm) == {"_Zk": 1, "_Zok": 0, "_Zw": 1}


def test_scan_keeps_reads_a_wait_does_not_cover():
    # lgkmcnt(14) with only two reads in flight retires neither: the MFMA reads a register of the
    # first (a list slice that went negative once dropped it)
    asm = """_Zfew:
\tds_read_b128 a[0:3], v1 offset:0
\tds_read_b128 a[4:7], v1 offset:64
\ts_waitcnt lgkmcnt(14)
\tv_mfma_f32_32x32x16_bf16 v[0:15], a[0:3], a[8:11], 0
.Lfunc_end0:
_Zsix:
\tds_read_b128 a[0:3], v1 offset:0
\tds_read_b128 a[4:7], v1 offset:64
\tds_read_b128 a[8:11], v1 offset:128
\ts_waitcnt lgkmcnt(2)
\tv_mfma_f32_32x32x16_bf16 v[0:15], a[0:3], a[12:15], 0
\tv_mfma_f32_32x32x16_bf16 v[16:31], a[4:7], a[12:15], 0
.Lfunc_end1:
"""
    # the second kernel: lgkmcnt(2) retires the first read only, the second MFMA touches the second
    assert kernel_hazards(asm) == {"_Zfew": 1, "_Zsix": 1}


def test_scan_follows_branches_over_waits():
    # the wait sits on the fall-through path only; the branch to .LBB0_2 skips it, so the use
    # after the join still sees the read in flight.  On the second kernel both paths wait.
    asm = """_Zbr:
\tds_read_b128 v[0:3], v9 offset:0
\ts_cbranch_vccz .LBB0_2
\ts_waitcnt lgkmcnt(0)
\tv_mov_b32 v20, 0
.LBB0_2:
\tv_add_u32 v10, v0, v1
\ts_endpgm
.Lfunc_end0:
_Zboth:
\tds_read_b128 v[0:3], v9 offset:0
\ts_waitcnt lgkmcnt(0)
\ts_cbranch_vccz .LBB1_2
\tv_mov_b32 v20, 0
.LBB1_2:
\tv_add_u32 v10, v0, v1
\ts_endpgm
.Lfunc_end1:
"""
    assert kernel_hazards(asm) == {"_Zbr": 1, "_Zboth": 0}


def test_scan_carries_reads_around_loops():
    # a read issued at the bottom of a loop body is still in flight at the top of the next
    # iteration: the use there is flagged unless a wait sits on the back edge
    asm = """_Zloop:
\ts_mov_b32 s0, 4
.LBB0_1:
\tv_add_u32 v10, v0, v1
\tds_read_b128 v[0:3], v9 offset:0
\ts_add_i32 s0, s0, -1
\ts_cmp_lg_u32 s0, 0
\ts_cbranch_scc1 .LBB0_1
\ts_waitcnt lgkmcnt(0)
\ts_endpgm
.Lfunc_end0:
_Zloopok:
\ts_mov_b32 s0, 4
.LBB1_1:
\tv_add_u32 v10, v0, v1
\tds_read_b128 v[0:3], v9 offset:0
\ts_add_i32 s0, s0, -1
\ts_cmp_lg_u32 s0, 0
\ts_waitcnt lgkmcnt(0)
\ts_cbranch_scc1 .LBB1_1
\ts_endpgm
.Lfunc_end1:
"""
    assert kernel_hazards(asm) == {"_Zloop": 1, "_Zloopok": 0}


@pytest.mark.parametrize("src", sorted(build.ASYNC_READS))
def test_built_kernels_keep_in_flight_registers_untouched(src):
    path = build.device_asm_path(src)
    if not os.path.exists(path):
        pytest.skip("library not built here")
    with open(path) as f:
        hz = kernel_hazards(f.read())
    assert hz, "no kernels in the kept assembly"
    assert not {k: v for k, v in hz.items() if v}
