"""The compiled kernels hold no register spill stored under a branch's exec
mask (CPU only: compiles the HIP sources to gfx950 assembly).

A kernel at its register limit once got a spill of a per-lane address stored
in the join block of a statistics branch, before the instruction that
restores the full exec mask: waves that skipped the branch never stored the
value, reloaded garbage after the tile loop and added their gradients at wrong
addresses.  The GPU tests caught it; this check catches the pattern in every
kernel at build time, whether or not a test runs that instance.
"""
import concurrent.futures

import pytest

from paper_2604_20819_amd import build

SOURCES = ["attn_fwd.hip", "attn_bwd.hip", "merge.hip", "stage.hip"]


@pytest.fixture(scope="module")
def asm():
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        return dict(zip(SOURCES, ex.map(build.device_asm, SOURCES)))


def test_detector_finds_the_pattern():
    bad = """
_ZN4cqsa1kEv:                           ; @_ZN4cqsa1kEv
	s_and_saveexec_b64 s[14:15], s[4:5]
	s_cbranch_execz .LBB1_2
	ds_write_b32 v245, v34
.LBB1_2:                                ; %Flow
	scratch_store_dwordx2 off, v[136:137], off offset:20 ; 8-byte Folded Spill
	s_or_b64 exec, exec, s[14:15]
	s_endpgm
.Lfunc_end1:
"""
    good = bad.replace("""	scratch_store_dwordx2 off, v[136:137], off offset:20 ; 8-byte Folded Spill
	s_or_b64 exec, exec, s[14:15]""", """	s_or_b64 exec, exec, s[14:15]
	scratch_store_dwordx2 off, v[136:137], off offset:20 ; 8-byte Folded Spill""")
    assert build.masked_spill_stores(bad) == {"_ZN4cqsa1kEv": 1}
    assert build.masked_spill_stores(good) == {}


@pytest.mark.parametrize("src", SOURCES)
def test_no_spill_under_a_partial_exec_mask(src, asm):
    assert ".amdhsa_kernel" in asm[src]
    assert build.masked_spill_stores(asm[src]) == {}
