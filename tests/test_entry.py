"""The driver's entry points: __graft_entry__.build() compiles the HIP library
and the oracle and loads the library.  Here the HIP compile is stubbed (the
built library is used as it is) so that the rest of build() -- the oracle's
compile, the imports and the load -- runs on the CPU in seconds."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def test_build_entry_runs(monkeypatch):
    import __graft_entry__ as entry
    from paper_2502_02414_amd import build as hip_build
    from paper_2502_02414_amd import binding
    if not os.path.exists(binding.LIB_PATH):
        import pytest
        pytest.skip("libpa.so is not built")
    calls = []
    monkeypatch.setattr(hip_build, "build", lambda verbose=False: calls.append(verbose))
    entry.build()
    assert calls == [True]
    import oracle
    assert os.path.exists(oracle.LIB)
