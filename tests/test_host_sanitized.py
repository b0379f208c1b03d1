"""The host library under AddressSanitizer and UndefinedBehaviorSanitizer:
graph construction, partition, patch extraction and union, the tile
schedule, context planning and the error paths (tests/test_host_lib.py) run
against a build whose host C++ is instrumented (device code unchanged); any
sanitizer report aborts the child run.  No device call is made."""
import os
import shutil

import pytest

from paper_2304_00338_amd import build_sanitized as BS

pytestmark = pytest.mark.timeout(900)


@pytest.mark.skipif(not os.path.exists(BS.B.HIPCC) and shutil.which("hipcc") is None, reason="no hipcc")
def test_host_library_under_asan_ubsan():
    lib = BS.build()
    assert os.path.exists(lib)
    assert BS.run_host_tests() == 0
