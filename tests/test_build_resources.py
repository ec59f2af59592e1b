"""Every GPU kernel of the library keeps its state in registers: no scratch
(private memory) and no spills, as reported by the compiler at build time
(paper_2606_07571_amd/_build/kernel_resources.json, written by build())."""
import json
import os

import pytest

PATH = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                    "paper_2606_07571_amd", "_build", "kernel_resources.json")


def test_no_scratch_no_spills():
    if not os.path.exists(PATH):
        pytest.skip("library not built")
    res = json.load(open(PATH))
    kernels = {k: v for k, v in res.items() if "kernel" in k}
    assert len(kernels) >= 8, sorted(res)
    for name, r in kernels.items():
        assert r.get("ScratchSize [bytes/lane]", 0) == 0, (name, r)
        assert r.get("VGPRs Spill", 0) == 0 and r.get("SGPRs Spill", 0) == 0, (name, r)
