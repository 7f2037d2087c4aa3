"""The C-ABI library loads and exports every entry point include/*.h declares;
host-side calls that need no GPU (sizes, status strings, argument validation
that fails before any launch) behave as documented."""
import ctypes as C
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in sorted(os.listdir(os.path.join(ROOT, "include")))
           if h.endswith(".h")]
LIB = os.path.join(ROOT, "paper_2606_19004_amd", "libditstep.so")


def _ensure_built():
    if not os.path.exists(LIB):
        from paper_2606_19004_amd import build
        build.build()


def declared_functions():
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*([a-z_0-9]+)\s*\(", text, flags=re.M))
    return sorted(names)


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("dit_block_forward", "joint_attention", "flow_step", "group_reward_stats"):
        assert required in names


def test_library_exports_every_declared_symbol():
    _ensure_built()
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True, check=True).stdout
    exported = {l.split()[-1] for l in out.splitlines() if " T " in l}
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, missing
    lib = C.CDLL(LIB)
    for n in declared_functions():
        getattr(lib, n)


def test_binding_covers_every_export():
    _ensure_built()
    from paper_2606_19004_amd import ditstep, planner
    assert set(ditstep.EXPORTS) | set(planner.EXPORTS) == set(declared_functions())
    assert ditstep.dit_abi_version() == 1


def test_host_side_validation_without_gpu():
    _ensure_built()
    from paper_2606_19004_amd import ditstep as d
    lib = d.lib()
    assert lib.dit_status_string(4) == b"NaN or infinite input"
    cfg = d.block_config(3072, 24, 128, 12288, 1024, 256, 32, 32)
    assert d.dit_block_workspace_bytes(cfg, 8) > 8 * 1280 * 12288 * 2
    bad = d.block_config(3072, 24, 100, 12288, 1024, 256, 32, 32)    # hidden != heads * head_dim
    assert d.dit_block_workspace_bytes(bad, 8) == 0
    # every one of these fails validation before touching the device
    assert lib.flow_step(None, None, None, 10, 0.5, 0.6, 0.0, None) == 3            # t_next > t
    assert lib.flow_step(None, None, None, 10, 1.0, 0.9, 0.7, None) == 3            # SDE needs t < 1
    assert lib.flow_step(None, None, None, 10, float("nan"), 0.1, 0.0, None) == 3
    assert lib.flow_step(None, None, None, 0, 0.5, 0.4, 0.0, None) == 0             # empty is a no-op
    assert lib.group_reward_stats(None, 4, 8, 1e-4, 9, None, None, None, None, None, None) == 1   # k > n
    assert lib.group_reward_stats(None, 0, 8, 1e-4, 2, None, None, None, None, None, None) == 0   # no groups
    assert lib.joint_attention(None, None, None, None, 1, 1, 8, 96, 0, 0, 0, 0, 0, 0, 1.0, 1, None) == 5
    assert b"head_dim" in lib.dit_last_error_message()
    w = d.BlockWeights()
    assert lib.dit_block_forward(C.byref(bad), C.byref(w), 1, None, None, None, None, 0, None) == 2
    assert lib.dit_block_forward(C.byref(cfg), C.byref(w), 0, None, None, None, None, 0, None) == 0


@pytest.mark.parametrize("cfg_args,status", [
    ((256, 4, 64, 1024, 64, 16, 8, 8), 0),
    ((256, 4, 64, 1024, 63, 16, 8, 8), 2),      # n_img != grid_h * grid_w
    ((256, 2, 128, 1000, 64, 16, 8, 8), 5),     # mlp_hidden not a multiple of 64
    ((8192, 64, 128, 32768, 64, 16, 8, 8), 5),  # hidden > 4096
])
def test_config_validation(cfg_args, status):
    _ensure_built()
    from paper_2606_19004_amd import ditstep as d
    cfg = d.block_config(*cfg_args)
    n = d.dit_block_workspace_bytes(cfg, 2)
    assert (n > 0) == (status == 0)
