"""What the compiled chunked-prefill kernel looks like, read from the built
library's own gfx950 code object (no GPU needed).

The prefill kernel waits for its direct-to-LDS K/V gathers with hand-counted
``s_waitcnt vmcnt(N)``: N is the number of gathers the step itself issued,
and everything older must have landed. That count is exact only if the
gathers are the only vector-memory loads inside the pipelined loop, since
extra loads issued after the gathers of a step would let older gathers still
be in flight. These tests pin that property on the machine code: the only
vector-memory loads are the gathers and the eight Q^T operand loads before
the loop; block-table entries are scalar loads; nothing spills to scratch.
"""
import os
import re
import shutil
import subprocess

import pytest

import paper_2608_23658_amd.kvattn as K

LLVM = "/opt/rocm/llvm/bin"
MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"
TARGET = "hipv4-amdgcn-amd-amdhsa--gfx950"


def _tool(name):
    p = os.path.join(LLVM, name)
    if not os.path.exists(p):
        pytest.skip(f"{p} is not installed")
    return p


@pytest.fixture(scope="module")
def disassembly(tmp_path_factory):
    """Disassembly of every gfx950 code object bundled into libkvattn.so."""
    if not os.path.exists(K.LIB_PATH):
        pytest.fail("libkvattn.so is not built")
    d = tmp_path_factory.mktemp("codeobj")
    fat = d / "fatbin.bin"
    subprocess.run([_tool("llvm-objcopy"), "-O", "binary", "--only-section=.hip_fatbin",
                    K.LIB_PATH, str(fat)], check=True)
    data = fat.read_bytes()
    starts = [m.start() for m in re.finditer(re.escape(MAGIC), data)]
    assert starts, "no offload bundle in the library"
    text, notes = [], []
    for i, st in enumerate(starts):
        end = starts[i + 1] if i + 1 < len(starts) else len(data)
        part = d / f"bundle{i}.bin"
        part.write_bytes(data[st:end])
        co = d / f"bundle{i}.co"
        r = subprocess.run([_tool("clang-offload-bundler"), "--unbundle", "--type=o",
                            f"--input={part}", f"--targets={TARGET}", f"--output={co}"],
                           capture_output=True)
        if r.returncode != 0 or not co.exists() or co.stat().st_size == 0:
            continue
        dis = subprocess.run([_tool("llvm-objdump"), "-d", str(co)], capture_output=True,
                             text=True, check=True)
        text.append(dis.stdout)
        meta = subprocess.run([_tool("llvm-readelf"), "--notes", str(co)], capture_output=True,
                              text=True, check=True)
        notes.append(meta.stdout)
    shutil.rmtree(d, ignore_errors=True)
    return "\n".join(text), "\n".join(notes)


def _functions(dis, name_part, operands=False):
    """{symbol: [mnemonic, ...]} (or [(mnemonic, operands), ...]) for the
    functions whose name contains name_part."""
    dis = dis[0]
    out, cur = {}, None
    for ln in dis.splitlines():
        m = re.match(r"^[0-9a-f]+ <(.+)>:$", ln)
        if m:
            cur = m.group(1) if name_part in m.group(1) else None
            if cur is not None:
                out[cur] = []
            continue
        if cur is not None:
            code = ln.split("//")[0].strip()
            if not code:
                continue
            mn, _, ops = code.partition(" ")
            out[cur].append((mn, ops.replace(" ", "")) if operands else mn)
    return out


def test_prefill_vector_loads_are_only_the_gathers_and_q(disassembly):
    fns = _functions(disassembly, "prefill_kernel")
    # one instance per group size (1, 2, 4, 8) and block-offset form (shift, multiply)
    assert len(fns) == 8, sorted(fns)
    for name, ins in fns.items():
        vmem = [i for i in ins if re.match(r"(global|buffer|flat|scratch)_", i)]
        loads = [i for i in vmem if "load" in i]
        assert set(loads) <= {"global_load_lds_dwordx4", "global_load_dwordx4"}, (name, set(loads))
        assert loads.count("global_load_dwordx4") == 8, name          # the Q^T operand
        assert loads.count("global_load_lds_dwordx4") >= 8, name      # the K/V gathers
        stores = [i for i in vmem if "store" in i]
        assert set(stores) <= {"global_store_dwordx2"}, (name, set(stores))
        assert not [i for i in ins if i.startswith("scratch_")], name  # no spills
        assert any(i.startswith("s_load_dword") for i in ins), name     # scalar table reads


def test_prefill_q_loads_precede_every_gather(disassembly):
    """The eight Q^T loads come before the first gather, so inside the loop
    every vector-memory load in flight is a gather."""
    for name, ins in _functions(disassembly, "prefill_kernel").items():
        first_gather = ins.index("global_load_lds_dwordx4")
        last_q = max(i for i, x in enumerate(ins) if x == "global_load_dwordx4")
        # the idle-wavefront path issues its gathers without loading Q and
        # comes first or last in the code; the busy path loads Q first
        busy_gathers = [i for i, x in enumerate(ins) if x == "global_load_lds_dwordx4"
                        and i > last_q]
        assert busy_gathers, name
        loads_after = [x for x in ins[last_q + 1:] if re.match(r"(global|buffer|flat)_load", x)]
        assert set(loads_after) == {"global_load_lds_dwordx4"}, (name, first_gather)


def test_prefill_m0_is_saved_and_restored(disassembly):
    """Each pair of gathers sits in one block that saves M0, points it at
    each gather's LDS destination, and restores the saved value, so the
    compiler's own view of M0 stays true outside the block."""
    for name, ins in _functions(disassembly, "prefill_kernel", operands=True).items():
        gathers = [i for i, (mn, _) in enumerate(ins) if mn == "global_load_lds_dwordx4"]
        assert gathers and len(gathers) % 2 == 0, name
        for a, b in zip(gathers[0::2], gathers[1::2]):
            assert b == a + 3, (name, a, b)
            save_mn, save_ops = ins[a - 3]
            assert save_mn == "s_mov_b32" and save_ops.endswith(",m0"), (name, ins[a - 3])
            saved = save_ops.split(",")[0]
            assert ins[a - 2][0] == "s_mov_b32" and ins[a - 2][1].startswith("m0,"), name
            assert ins[b - 2][0] == "s_mov_b32" and ins[b - 2][1].startswith("m0,"), name
            assert ins[b + 1] == ("s_mov_b32", f"m0,{saved}"), (name, ins[b + 1])


def test_no_kernel_spills_registers(disassembly):
    """Every kernel in the library fits its registers: a spill would put
    scratch loads and stores (counted by vmcnt) into the pipelines."""
    notes = disassembly[1]
    names = re.findall(r"\.symbol:\s+(\S+)", notes)
    spills = [int(x) for x in re.findall(r"\.vgpr_spill_count:\s+(\d+)", notes)]
    sspills = [int(x) for x in re.findall(r"\.sgpr_spill_count:\s+(\d+)", notes)]
    assert len(spills) >= 20 and len(spills) == len(sspills)
    assert any("prefill_kernel" in n for n in names)
    assert len(names) == len(spills), (len(names), len(spills))
    bad = [(n, v, sv) for n, v, sv in zip(names, spills, sspills) if v or sv]
    assert not bad, bad
