"""The GEMM main loop issues its LDS fragment reads from inline assembly and
places every lgkmcnt wait by hand, so the compiler does not protect the
registers those reads land in.  These tests compile the library's kernels to
gfx950 assembly (on the CPU) and check that no instruction touches the
destination of an LDS read that may still be in flight."""
import os
import shutil

import pytest

from lds_hazards import check, regs
from paper_2606_16264_amd import build

HAVE_HIPCC = shutil.which(build.HIPCC) is not None or os.path.exists(build.HIPCC)

# A dead fragment read in flight when a loop exits, and an epilogue index
# computed into one of its registers before the wait: the hazard that turned
# an epilogue row index into LDS data and faulted the GPU.
BAD = """\
k:
\tds_read_b128 v[0:3], v0
\tds_read_b128 v[4:7], v4
\ts_cbranch_scc0 .LBB0_2
.LBB0_1:
\tv_lshl_or_b32 v6, v22, 2, s1
\ts_waitcnt lgkmcnt(0)
\tglobal_store_short v[18:19], v6, off
.LBB0_2:
\ts_endpgm
.Lfunc_end0:
"""

GOOD = """\
k:
\tds_read_b128 v[0:3], v0
\tds_read_b128 v[4:7], v4
\tv_mov_b32 v8, v9
\ts_waitcnt lgkmcnt(1)
\tv_mov_b32 v10, v1
\ts_waitcnt lgkmcnt(0)
\tv_lshl_or_b32 v6, v22, 2, s1
\ts_endpgm
.Lfunc_end0:
"""

# A loop whose back edge carries reads into the header: the copy at the top
# of the loop reads v2 before the wait.
LOOP = """\
k:
\tds_read_b128 v[0:3], v0
.LBB0_1:
\tv_mov_b32 v20, v2
\ts_waitcnt lgkmcnt(0)
\tds_read_b128 v[0:3], v5
\ts_cbranch_scc0 .LBB0_1
\ts_waitcnt lgkmcnt(0)
\ts_endpgm
.Lfunc_end0:
"""


def test_register_parser():
    assert regs("v[4:7], v9, s[2:3], a0, 0xa3, vcc") == {
        ("v", 4), ("v", 5), ("v", 6), ("v", 7), ("v", 9), ("s", 2), ("s", 3), ("a", 0)}


def test_checker_flags_dead_read_hazard():
    rep = check(BAD)["k"]
    assert rep and rep[0][0] == 6 and ("v", 6) in rep[0][4]


def test_checker_accepts_waited_reads():
    assert check(GOOD)["k"] == []


def test_checker_follows_back_edges():
    rep = check(LOOP)["k"]
    assert any(r[1] == "v_mov_b32" and ("v", 2) in r[4] for r in rep)


@pytest.mark.skipif(not HAVE_HIPCC, reason="hipcc not available")
def test_gemm_kernels_have_no_lds_read_hazard(tmp_path):
    out = build.device_asm("gemm.hip", str(tmp_path / "gemm.s"))
    res = {k: v for k, v in check(open(out).read()).items() if "gemm_kernel" in k}
    # five tile shapes x (four epilogues + the split-K partial store)
    assert len(res) == 25, sorted(res)
    bad = {k: v[:3] for k, v in res.items() if v}
    assert not bad, bad


@pytest.mark.skipif(not HAVE_HIPCC, reason="hipcc not available")
def test_attention_kernels_have_no_lds_read_hazard(tmp_path):
    out = build.device_asm("attention.hip", str(tmp_path / "attention.s"))
    res = {k: v for k, v in check(open(out).read()).items() if "_kernel" in k}
    assert len(res) == 4, sorted(res)
    bad = {k: v[:3] for k, v in res.items() if v}
    assert not bad, bad
