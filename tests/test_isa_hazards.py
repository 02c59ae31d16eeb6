"""The built library's gfx950 machine code keeps the wait states a wide store needs before
its data registers are overwritten (CPU: disassembles the code objects built here)."""
import os

import pytest

import paper_2609_32525_amd as fs
from paper_2609_32525_amd.isa_check import WAIT_STATES, check_library


@pytest.mark.skipif(not os.path.exists(fs.lib_path()), reason="libflashslice.so not built")
def test_wide_stores_keep_their_wait_states():
    n, bad = check_library(fs.lib_path())
    assert n > 0
    assert not bad, f"{len(bad)} wide stores overwritten within {WAIT_STATES} wait states: {bad[:5]}"
