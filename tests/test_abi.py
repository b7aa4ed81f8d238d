"""CPU checks of the C ABI: the library loads and exports every symbol that
include/mpx.h declares, and the binding covers the same set.  No compute
call is made (there is no GPU here)."""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2507_03312_amd", "libmpx.so")


def declared_functions():
    src = open(os.path.join(ROOT, "include", "mpx.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = set(re.findall(r"\b(mpx_[a-z0-9_]+)\s*\(", src))
    return names


def test_header_declares_the_named_entry_points():
    names = declared_functions()
    for n in ["mpx_cast_to_half", "mpx_linear_fwd", "mpx_linear_bwd", "mpx_unscale_check",
              "mpx_scale_update", "mpx_adamw_masked"]:
        assert n in names


@pytest.mark.skipif(not os.path.exists(LIB), reason="libmpx.so not built")
def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT (mpx_[a-z0-9_]+)$", out, flags=re.M))
    missing = declared_functions() - exported
    assert not missing, missing


@pytest.mark.skipif(not os.path.exists(LIB), reason="libmpx.so not built")
def test_binding_loads_and_covers_the_header():
    from paper_2507_03312_amd import binding
    assert set(binding.EXPORTED) == declared_functions()
    # a pure host call: size queries need no device
    assert binding.mpx_linear_bwd_workspace(64, 512, 1024) > 0
    assert binding.mpx_layernorm_bwd_workspace(100, 384) > 0
