"""The build entry point compiles both libraries and imports the package."""
import os

import __graft_entry__ as entry


def test_build_entry_compiles_everything():
    entry.build()
    root = os.path.dirname(os.path.abspath(entry.__file__))
    assert os.path.exists(os.path.join(root, "paper_2512_23236_amd", "libtbe.so"))
    assert os.path.exists(os.path.join(root, "oracle", "liboracle.so"))
    assert callable(entry.smoke)
