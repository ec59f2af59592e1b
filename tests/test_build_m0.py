"""The GEMM kernels load operand tiles straight into LDS with inline-assembly
buffer loads whose LDS address comes from M0.  The compiler does not see those
loads, so the device code must keep M0 to itself: in the built assembly
(paper_2606_07571_amd/_build/gemm_device.s, written by build()) the only
instruction that names M0 is the helper's `s_mov_b32 m0, s<n>`, always followed
by one wait state and the first load of a group, and every group has four
loads."""
import os
import re

import pytest

PATH = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                    "paper_2606_07571_amd", "_build", "gemm_device.s")


def _kernels(text):
    """{kernel symbol: [instruction lines]} for the GEMM kernels."""
    out, cur = {}, None
    for line in text.splitlines():
        m = re.match(r"^(_Z\S*gemm_kernel\S*):", line)
        if m:
            cur = m.group(1)
            out[cur] = []
            continue
        if cur is None:
            continue
        code = line.split(";", 1)[0].strip()
        if not code or code.startswith(".") or code.endswith(":"):
            continue
        out[cur].append(code)
        if code.startswith("s_endpgm"):
            cur = None
    return out


def test_m0_written_only_by_the_lds_load_helper():
    if not os.path.exists(PATH):
        pytest.skip("library not built")
    kernels = _kernels(open(PATH).read())
    assert len(kernels) >= 4, sorted(kernels)
    for name, ins in kernels.items():
        sets = loads = 0
        for i, code in enumerate(ins):
            if re.search(r"\bm0\b", code):
                assert re.fullmatch(r"s_mov_b32 m0, s\d+", code), (name, code)
                assert ins[i + 1] == "s_nop 0", (name, ins[i:i + 3])
                assert re.fullmatch(r"buffer_load_dwordx4 v\d+, s\[\d+:\d+\], s\d+ offen lds", ins[i + 2]), \
                    (name, ins[i:i + 3])
                sets += 1
            if re.search(r"^buffer_load_dwordx4 .* lds$", code):
                loads += 1
        assert sets > 0 and loads == 4 * sets, (name, sets, loads)
