"""Host-side checks of the C ABI library: it loads without a GPU and exports every declared symbol."""
import ctypes
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    src = open(os.path.join(ROOT, "include", "canon.h")).read()
    return sorted(set(re.findall(r"\b(canon_[a-z_0-9]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    import paper_2609_17380_amd.canon as C
    lib = C.lib()
    names = declared_symbols()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    assert C.version() == 1
    assert lib.canon_status_str(-4) == b"workspace too small"


def test_workspace_queries_without_gpu():
    import numpy as np
    import paper_2609_17380_amd.canon as C
    cfg = C.ModelCfg(16, 2048, 16, 128, 8192, 50304, 2048, 4, np.float32(1e-5))
    plan = C.DPPlan(1, 8, 1)
    ws = C.step_workspace_bytes(cfg, plan)
    assert 30e9 < ws < 80e9  # fits one MI355X next to the parameters and moments
    assert C.block_workspace_bytes(cfg, 1) > 0
    bad = C.ModelCfg(16, 2048, 15, 128, 8192, 50304, 2048, 4, np.float32(1e-5))  # heads * head_dim != d
    assert C.step_workspace_bytes(bad, plan) == 0


def test_oracle_and_library_share_no_source():
    lib_src = open(os.path.join(ROOT, "paper_2609_17380_amd", "csrc", "canon_dev.h")).read()
    orc = open(os.path.join(ROOT, "oracle", "canon_ref.c")).read()
    assert "canon_dev.h" not in orc and "canon.h" not in orc.replace("canon_ref.h", "")
    assert "canon_ref" not in lib_src
