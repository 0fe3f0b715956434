"""The computed-jump dispatch of the register-tile kernels, checked in the
compiled code object (host-side, no GPU): for every dispatch site the key is
clamped to the table before the jump, the table base resolves to the first
leaf, the leaves sit at the exact power-of-two stride the jump assumes, and
every leaf ends with a branch back.  A wrong stride would send a nonzero to
another leaf's multiply-adds; an unclamped key could leave the table."""
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_1704_07724_amd import build as B  # noqa: E402

LLVM = "/opt/rocm/llvm/bin"


@pytest.fixture(scope="module")
def disassembly(tmp_path_factory):
    if not os.path.exists(B.HIPCC) or not os.path.exists(os.path.join(LLVM, "llvm-objdump")):
        pytest.skip("ROCm toolchain not available")
    B.generate()
    out = tmp_path_factory.mktemp("dispatch")
    texts = {}
    for name in ("sparse_reg.hip", "sparse_res.hip"):
        obj = str(out / (name + ".o"))
        cmd = ([B.HIPCC] + B.DEVICE_FLAGS + B.FILE_FLAGS.get(name, []) +
               ["--offload-device-only", "--no-gpu-bundle-output", "-c", os.path.join(B.CSRC, name), "-o", obj])
        subprocess.run(cmd, check=True, capture_output=True)
        texts[name] = subprocess.run([os.path.join(LLVM, "llvm-objdump"), "-d", "--mcpu=gfx950", obj],
                                     check=True, capture_output=True, text=True).stdout
    return texts


def dispatch_sites(text):
    """(prefix, {leaf index: (address, instructions)}, base address, setup
    instructions) for every dispatch site L<n>_... in a disassembly."""
    sites = {}
    cur = None
    for line in text.splitlines():
        m = re.match(r"^([0-9a-f]+) <(L\d+)_(base|q\d+|end)>:", line)
        if m:
            addr, pre, what = int(m.group(1), 16), m.group(2), m.group(3)
            site = sites.setdefault(pre, {"leaves": {}, "base": None, "setup": []})
            if what == "base":
                site["base"] = addr
                cur = ("base", site, None)
            elif what == "end":
                cur = None
            else:
                q = int(what[1:])
                site["leaves"][q] = (addr, [])
                cur = ("leaf", site, q)
            continue
        m = re.match(r"^\s+(\S+)\s*([^/]*)//\s*([0-9A-F]+):", line)
        if not m or cur is None:
            continue
        ins = (m.group(1), m.group(2).strip(), int(m.group(3), 16))
        if cur[0] == "leaf":
            cur[1]["leaves"][cur[2]][1].append(ins)
        else:
            cur[1]["setup"].append(ins)
    return sites


@pytest.mark.parametrize("name", ["sparse_reg.hip", "sparse_res.hip"])
def test_jump_tables_exact(disassembly, name):
    text = disassembly[name]
    sites = dispatch_sites(text)
    assert sites, "no computed-jump dispatch found"
    lines = text.splitlines()
    for pre, site in sites.items():
        leaves = site["leaves"]
        n = len(leaves)
        assert sorted(leaves) == list(range(n)), pre
        stride = leaves[1][0] - leaves[0][0] if n > 1 else 4
        assert stride & (stride - 1) == 0, (pre, stride)
        for q, (addr, ins) in leaves.items():
            assert addr == leaves[0][0] + q * stride, (pre, q)
            real = [i for i in ins if i[0] != "s_nop"]
            assert real and real[-1][0] == "s_branch", (pre, q)
            assert all(i[0] == "v_fmac_f32_e32" for i in real[:-1]), (pre, q)
            assert 4 * len(real) <= stride, (pre, q)
        # setup: s_add of (first leaf - base), then the jump
        setup = [i for i in site["setup"] if i[0] != "s_nop"]
        assert setup[0][0] == "s_add_u32" and setup[-1][0] == "s_setpc_b64", pre
        off = int(re.findall(r"0x[0-9a-f]+|\d+", setup[0][1].split(",")[-1])[0], 0)
        assert site["base"] + off == leaves[0][0], pre
        # before the base label: the key clamped to the table and scaled
        i = next(k for k, l in enumerate(lines) if ("<%s_base>:" % pre) in l)
        pre_lines = [l for l in lines[i - 6:i] if "\t" in l]
        joined = "\n".join(pre_lines)
        m = re.search(r"s_min_u32 (s\d+), s\d+, (0x[0-9a-f]+|\d+)", joined)
        assert m and int(m.group(2), 0) == n - 1, (pre, joined)
        assert re.search(r"s_lshl_b32 %s, %s, %d" % (m.group(1), m.group(1), stride.bit_length() - 1), joined), pre
