"""Run the CPU tests of the C ABI (tests/test_abi.py, no GPU) against the
library at the path given on the command line instead of the in-tree build.
Used by the sanitizer test, which starts it in a child process with the
AddressSanitizer runtime preloaded."""
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))
sys.path.insert(0, HERE)

from paper_2609_04910_amd import gauss_sum as gs  # noqa: E402

gs.LIB_PATH = sys.argv[1]
gs.load.__defaults__ = (sys.argv[1], False)  # no torch in the sanitizer run

import pytest  # noqa: E402

sys.exit(pytest.main([os.path.join(HERE, "test_abi.py"), "-q", "-m", "not gpu", "-p", "no:cacheprovider"]))
