"""The build's checks on the persistent kernel's generated code (host only).

paper_2607_18002_amd/build.py refuses a build whose device assembly writes the
data registers of a store wider than 8 bytes with a VALU instruction fewer than
two wait states after the store (gfx950 reads such a store's data after issue),
and one whose kernels copy their arguments to scratch.  These tests pin the
parsers of those checks on hand-written assembly and resource remarks.
"""
import pytest

from paper_2607_18002_amd import build as B


def _refused(asm: str) -> bool:
    try:
        B._store_data_check("t.hip", asm)
    except RuntimeError:
        return True
    return False


def test_store_data_overwrite_is_refused():
    # the sequence found at an epilogue part boundary: store, scheduling-barrier comment, VALU write
    assert _refused("buffer_store_dwordx4 v[34:37], v98, s[28:31], s4 offen sc1\n"
                    "; sched_barrier mask(0x00000000)\n"
                    "v_mul_f32_e32 v34, 0xbfb8aa3b, v18\n")
    # one wait state is not enough; a write of the last data register counts too
    assert _refused("buffer_store_dwordx4 v[4:7], v1, s[0:3], 0 offen sc1\n"
                    "s_mov_b32 s4, 0\n"
                    "v_mov_b32_e32 v7, 0\n")
    # global stores name the address first and the data second
    assert _refused("global_store_dwordx4 v[6:7], v[2:5], off\nv_mov_b32_e32 v3, 0\n")
    assert _refused("global_store_dwordx3 v[6:7], v[2:4], off\nv_add_u32_e32 v4, 1, v4\n")
    # control falls through a label into the next block
    assert _refused("buffer_store_dwordx4 v[4:7], v1, s[0:3], 0 offen\n.LBB0_3:\n; %bb.4:\nv_mov_b32_e32 v4, 0\n")


def test_safe_sequences_pass():
    # two wait states from s_nop 1, or two other instructions, before the write
    assert not _refused("buffer_store_dwordx4 v[34:37], v98, s[28:31], s4 offen sc1\ns_nop 1\n"
                        "v_mul_f32_e32 v34, 0xbfb8aa3b, v18\n")
    assert not _refused("buffer_store_dwordx4 v[4:7], v1, s[0:3], 0 offen sc1\ns_mov_b32 s4, 0\n"
                        "s_mov_b32 s5, 0\nv_mov_b32_e32 v7, 0\n")
    # the address of a global store, an 8-byte store, and another register are free to change
    assert not _refused("global_store_dwordx4 v[6:7], v[2:5], off\nv_lshl_add_u64 v[6:7], v[6:7], 0, s[6:7]\n")
    assert not _refused("buffer_store_dwordx2 v[4:5], v1, s[0:3], 0 offen\nv_mov_b32_e32 v4, 0\n")
    assert not _refused("buffer_store_dwordx4 v[4:7], v1, s[0:3], 0 offen\nv_mov_b32_e32 v8, 0\n")
    # an LDS read into the registers returns long after the store has read them
    assert not _refused("buffer_store_dwordx4 v[40:43], v6, s[40:43], s2 offen sc1\n"
                        "ds_read_b128 v[40:43], v7 offset:7680\n")
    # an unconditional branch ends the look-ahead
    assert not _refused("buffer_store_dwordx4 v[4:7], v1, s[0:3], 0 offen\ns_branch .LBB0_7\n"
                        "v_mov_b32_e32 v4, 0\n")


def test_scratch_copy_of_kernel_arguments_is_refused():
    lines = ["remark: Function Name: _ZN12_GLOBAL__N_110apk_kernelILb0EEEvNS_5KArgsE",
             "remark:     ScratchSize [bytes/lane]: 3632"]
    with pytest.raises(RuntimeError):
        B._scratch_check("ffn.hip", lines)
    B._scratch_check("ffn.hip", [lines[0], "remark:     ScratchSize [bytes/lane]: 0"])
