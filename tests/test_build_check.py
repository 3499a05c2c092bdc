"""The build refuses kernels that need private scratch memory (register
spills): the parser of the compiler's resource-usage remarks, on remark text of
the compiler's form, and the figures of the library as built."""
import os

from paper_2608_28911_amd import build as B

R = "[-Rpass-analysis=kernel-resource-usage]"
TEXT = "\n".join([
    "x.hip:10:1: remark: Function Name: _Z4goodv " + R,
    "x.hip:10:1: remark:     VGPRs: 40 " + R,
    "x.hip:10:1: remark:     ScratchSize [bytes/lane]: 0 " + R,
    "x.hip:20:1: warning: something else",
    "x.hip:30:1: remark: Function Name: _Z5spillv " + R,
    "x.hip:30:1: remark:     VGPRs: 256 " + R,
    "x.hip:30:1: remark:     ScratchSize [bytes/lane]: 24 " + R,
])


def test_remarks_parsed_per_kernel():
    usage, rest = B.parse_remarks(TEXT)
    assert set(usage) == {"_Z4goodv", "_Z5spillv"}
    assert usage["_Z4goodv"]["VGPRs"] == "40"
    assert usage["_Z5spillv"]["ScratchSize [bytes/lane]"] == "24"
    assert rest == ["x.hip:20:1: warning: something else"]


def test_spilling_kernels_found():
    usage, _ = B.parse_remarks(TEXT)
    assert B.spilling(usage) == ["_Z5spillv"]


def test_built_library_has_no_spills():
    path = os.path.join(B.BUILD, "resource_usage.txt")
    if not os.path.exists(path):
        import pytest
        pytest.skip("the library was not built here")
    lines = open(path).read().splitlines()
    assert any("decode_kernel" in l for l in lines)
    for l in lines:
        assert "ScratchSize[bytes/lane]=0" in l, l
