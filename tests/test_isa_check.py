"""The post-build machine-code check: MFMAs under a possibly-empty EXEC mask (no GPU)."""
import glob
import os

import pytest

from paper_2605_28803_amd import isa_check

HEAD = "0000000000001000 <kern>:\n"


def _dis(*ins):
    return HEAD + "".join(f"\t{i}  // 000000001000: 00000000\n" for i in ins)


MFMA = "v_mfma_i32_32x32x32_i8 v[2:17], v[18:21], v[22:25], v[2:17]"


def test_masked_mfma_without_skip_is_reported():
    hits = isa_check.unguarded_mfma(_dis("s_and_saveexec_b64 s[0:1], s[2:3]", MFMA, "s_or_b64 exec, exec, s[0:1]"))
    assert hits == [("kern", MFMA)]


@pytest.mark.parametrize("guard", ["s_cbranch_execz 4", "s_or_b64 exec, exec, s[0:1]", "s_mov_b64 exec, -1"])
def test_skip_or_restore_clears(guard):
    assert isa_check.unguarded_mfma(_dis("s_and_saveexec_b64 s[0:1], s[2:3]", guard, MFMA)) == []


def test_execnz_fallthrough_and_cmpx_count_as_masked():
    # The fall-through of s_cbranch_execnz runs with EXEC = 0.
    assert len(isa_check.unguarded_mfma(_dis("s_and_saveexec_b64 s[0:1], s[2:3]", "s_cbranch_execnz 8", MFMA))) == 1
    assert len(isa_check.unguarded_mfma(_dis("v_cmpx_lt_i32_e32 vcc, s4, v1", MFMA))) == 1
    assert len(isa_check.unguarded_mfma(_dis("s_andn2_b64 exec, exec, vcc", MFMA))) == 1


def test_unmasked_code_and_function_boundary():
    assert isa_check.unguarded_mfma(_dis(MFMA, "s_and_b64 s[0:1], vcc, s[2:3]", MFMA)) == []
    two = _dis("s_and_saveexec_b64 s[0:1], s[2:3]") + "0000000000002000 <next>:\n\t" + MFMA + "\n"
    assert isa_check.unguarded_mfma(two) == []


def test_built_library_is_clean():
    objs = sorted(glob.glob(os.path.join(os.path.dirname(os.path.dirname(__file__)), "_build", "*.o")))
    if not objs or not isa_check.tools_present():
        pytest.skip("no built objects or no llvm-objcopy / llvm-objdump")
    assert isa_check.check_objects(objs) == []
