"""The library build (CPU only): the helper context kernels of three and four
row blocks come from their own translation unit, compiled with the
matrix-core accumulators in vector registers, and the main unit does not
instantiate them."""
import os
import re

from paper_2608_15797_amd import build

CSRC = os.path.join(os.path.dirname(build.__file__), "csrc")


def test_wide_unit_is_built_apart_with_its_option():
    assert os.path.isfile(build.WIDE)
    assert build.WIDE not in build.sources()
    assert "-amdgpu-mfma-vgpr-form=1" in build.WIDE_FLAGS
    src = open(build.WIDE).read()
    assert "#define KVR_ATTN_WIDE 1" in src and '#include "attn.hip"' in src


def test_main_unit_routes_wide_row_blocks_to_the_wide_unit():
    src = open(os.path.join(CSRC, "attn.hip")).read()
    # No launch of, or occupancy query on, a three- or four-row-block
    # instantiation outside the KVR_ATTN_WIDE part of the file.
    main = src.split("#else  // KVR_ATTN_WIDE")[0]
    assert not re.search(r"launch_prefix<\s*D\s*,\s*[34]\s*,", main)
    assert not re.search(r"prefix_slots<\s*D\s*,\s*[34]\s*,", main)
    assert "launch_prefix_wide(D, 3, p, ent, stream)" in main
    assert "launch_prefix_wide(D, 4, p, ent, stream)" in main
