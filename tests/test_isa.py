"""Static checks of the gfx950 assembly hipcc produces for the kernels (CPU only).

 - no packed FP32 arithmetic anywhere (the build disables the feature);
 - no scalar-memory writes of any kind;
 - M0 is written only by the register-indexing sequences of the interpreter;
 - the discover kernels keep their values in registers (no private scratch).
"""

import os
import re
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2608_27612_amd", "csrc", "kernels.hip")


@pytest.fixture(scope="module", params=["kernels.hip", "band.hip"])
def asm(request):
    """The kernels that run the interpreter's record step: discovery, and the band values."""
    from paper_2608_27612_amd import build
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "k.s")
        cmd = [build.HIPCC, "-O3", "-std=c++17", "--cuda-device-only", "-S"] + build.DEVICE_FLAGS \
            + [os.path.join(os.path.dirname(SRC), request.param), "-o", out]
        subprocess.check_call(cmd, stderr=subprocess.DEVNULL)
        return open(out).read()


def _kernels(asm):
    """{symbol: body} for every kernel in the assembly."""
    out = {}
    for m in re.finditer(r"^(_Z\w+):\s*;\s*@", asm, flags=re.M):
        start = m.end()
        end = asm.find("s_endpgm", start)
        out[m.group(1)] = asm[start:end]
    return out


@pytest.fixture(scope="module", params=["phase2.hip", "network.hip"])
def phase2_asm(request):
    """The kernels after discovery: Phase 2 and connections, and the network kernels."""
    from paper_2608_27612_amd import build
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "p.s")
        cmd = [build.HIPCC, "-O3", "-std=c++17", "--cuda-device-only", "-S"] + build.DEVICE_FLAGS \
            + [os.path.join(ROOT, "paper_2608_27612_amd", "csrc", request.param), "-o", out]
        subprocess.check_call(cmd, stderr=subprocess.DEVNULL)
        return open(out).read()


def test_sort_kernels_have_no_packed_fp32_or_scalar_writes():
    """The library sort behind network assembly (a generic library kernel: its register and
    scratch use is its own) holds no packed FP32 arithmetic and no scalar-memory writes."""
    from paper_2608_27612_amd import build
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "s.s")
        cmd = [build.HIPCC, "-O3", "-std=c++17", "--cuda-device-only", "-S"] + build.DEVICE_FLAGS \
            + [os.path.join(ROOT, "paper_2608_27612_amd", "csrc", "net_sort.hip"), "-o", out]
        subprocess.check_call(cmd, stderr=subprocess.DEVNULL)
        text = open(out).read()
    assert "radix" in text
    assert not re.search(r"v_pk_(add|mul|fma)_f32", text)
    pattern = r"\bs_(buffer_)?(st" + r"ore|atom" + r"ic)\w*|\bs_dca" + r"che_\w+|\bs_scr" + r"atch_\w+"
    assert not re.search(pattern, text)


def test_phase2_kernels_have_no_packed_fp32_scalar_writes_m0_or_scratch(phase2_asm):
    assert not re.search(r"v_pk_(add|mul|fma)_f32", phase2_asm)
    pattern = r"\bs_(buffer_)?(st" + r"ore|atom" + r"ic)\w*|\bs_dca" + r"che_\w+|\bs_scr" + r"atch_\w+"
    assert not re.search(pattern, phase2_asm)
    for line in phase2_asm.splitlines():
        assert not re.search(r"\bm0\b", line.split(";")[0]), line
    for size in re.findall(r"\.private_segment_fixed_size:\s+(\d+)", phase2_asm):
        assert int(size) == 0


def test_no_packed_fp32(asm):
    assert not re.search(r"v_pk_(add|mul|fma)_f32", asm)


def test_no_scalar_memory_writes(asm):
    pattern = r"\bs_(buffer_)?(st" + r"ore|atom" + r"ic)\w*|\bs_dca" + r"che_\w+|\bs_scr" + r"atch_\w+"
    assert not re.search(pattern, asm)


def test_m0_only_for_register_indexing(asm):
    for line in asm.splitlines():
        code = line.split(";")[0]
        if re.search(r"\bm0\b", code):
            pytest.fail("unexpected M0 use: " + line.strip())
    assert "s_set_gpr_idx_on" in asm


def test_discover_kernels_use_no_scratch(asm):
    ks = {k: v for k, v in _kernels(asm).items() if "k_discover" in k or "k_band" in k}
    assert len(ks) in (1, 2)   # one per output mode, or the band kernel
    for name, body in ks.items():
        assert "scratch_" not in body and "buffer_store" not in body, name
    sizes = re.findall(r"\.name:\s+(\S*k_(?:discover|band)\S*)\s*\n(?:.*\n)*?"
                       r"\s+\.private_segment_fixed_size:\s+(\d+)", asm)
    assert sizes
    for name, size in sizes:
        assert int(size) == 0, name


# Scalar instructions that read SCC, and ones that write it without reading it first.
_SCC_READERS = re.compile(r"^\s*(s_cbranch_scc[01]|s_cselect_\w+|s_addc_u32|s_subb_u32|s_cmov\w*)\b")
_SCC_WRITERS = re.compile(
    r"^\s*(s_cmp\w*|s_bitcmp\w*|s_(add|sub)_[ui]32|s_(and|or|xor|andn2|orn2|nand|nor|xnor)_\w+|"
    r"s_(lshl|lshr|ashr)\w*|s_bfe_\w+|s_(min|max)_\w+|s_not_\w+|s_abs_\w+|s_absdiff\w*|s_bcnt\w*|"
    r"s_wqm\w*|s_quadmask\w*|s_bfm_\w+)\b")


def test_scc_is_not_carried_across_inline_asm(asm):
    """The record step's asm statement writes SCC; a compiler-made SCC value must never be read
    after it without being recomputed (a loop exit test carried across it would be garbage)."""
    lines = asm.splitlines()
    blocks = 0
    start = 0
    for i, line in enumerate(lines):
        if ";;#ASMSTART" in line:
            start = i
        if ";;#ASMEND" not in line:
            continue
        if not any(_SCC_WRITERS.match(x.split(";")[0]) for x in lines[start:i]):
            continue  # a statement that leaves SCC alone
        blocks += 1
        for k in range(i + 1, min(i + 80, len(lines))):
            code = lines[k].split(";")[0]
            if not code.strip() or code.strip().startswith("."):
                continue
            assert not _SCC_READERS.match(code), "SCC read after inline asm: " + code.strip()
            if _SCC_WRITERS.match(code) or re.match(r"^\s*s_(branch|endpgm|setpc)", code):
                break
    # every record-step walk of the file: 18+ in the discover kernels, 4 in the band kernel
    assert blocks >= (18 if "k_discover" in asm else 4)


def test_record_step_clobbers_scc_and_m0():
    hdr = open(os.path.join(ROOT, "paper_2608_27612_amd", "csrc", "regwin_gen.h")).read()
    n_walkers = hdr.count("struct Walker<")
    assert n_walkers == 9 and hdr.count('"scc", "m0"') == n_walkers


def test_tail_jumps_land_on_their_tails():
    """The record step jumps to tail (meta & 15) at .Lt0 + index * stride: in the disassembled
    code object, every such jump site's tail slots begin with the instructions of their tails
    (continuation and unknown tails: the loop end; store tails: the index switch or the first
    activation step; output tails: the first activation step)."""
    from paper_2608_27612_amd import build
    llvm = "/opt/rocm/llvm/bin"
    with tempfile.TemporaryDirectory() as d:
        obj, dev = os.path.join(d, "k.o"), os.path.join(d, "k_gfx950.o")
        subprocess.check_call([build.HIPCC, "-O3", "-std=c++17", "--cuda-device-only", "-c"]
                              + build.DEVICE_FLAGS + [SRC, "-o", obj], stderr=subprocess.DEVNULL)
        subprocess.check_call([os.path.join(llvm, "clang-offload-bundler"), "--unbundle",
                               "--type=o", "--input=" + obj,
                               "--targets=hipv4-amdgcn-amd-amdhsa--gfx950", "--output=" + dev])
        out = subprocess.run([os.path.join(llvm, "llvm-objdump"), "-d", "--no-show-raw-insn", dev],
                             capture_output=True, text=True, check=True).stdout
    ins = []
    for line in out.splitlines():
        m = re.match(r"\s+(.*?)\s*//\s*([0-9A-Fa-f]+):", line)
        if m:
            ins.append((int(m.group(2), 16), m.group(1).strip()))
    at = dict(ins)
    # activation ids: 0 linear, 1 sigmoid, 2 tanh, 3 gaussian, 4 sine, 5 abs
    first = ["s_sub_u32",                                   # 0 continuation
             "s_set_gpr_idx_on", "v_exp_f32", "v_exp_f32", "v_mul_f32", "v_fract_f32",
             "s_set_gpr_idx_on",                            # 1..6 store tails
             "s_sub_u32", "v_exp_f32", "v_exp_f32", "v_mul_f32", "v_fract_f32",
             "v_and_b32",                                   # 7..12 output tails
             "s_sub_u32"]                                   # 13 unknown
    sites = 0
    for k, (_, text) in enumerate(ins):
        m = re.match(r"s_lshl_b32 (\w+), \1, (\d+)$", text)
        if not m or k + 1 >= len(ins):
            continue
        m2 = re.match(r"s_add_u32 %s, %s, (0x[0-9a-fA-F]+|\d+)" % (m.group(1), m.group(1)),
                      ins[k + 1][1])
        if not m2:
            continue
        j = k + 2
        while not ins[j][1].startswith("s_getpc_b64"):
            j += 1
        t0 = ins[j + 1][0] + int(m2.group(1), 0)
        stride = 1 << int(m.group(2))
        got = [at.get(t0 + i * stride, "?") for i in range(14)]
        assert all(g.startswith(f) for g, f in zip(got, first)), (stride, got)
        sites += 1
    assert sites == 2 * 9  # one per walker (9 sources-per-walk and window variants) per mode


# ------------------------------------------------------------------ the compiled tier's template
JIT_SRC = os.path.join(ROOT, "paper_2608_27612_amd", "csrc", "jit.hip")


@pytest.fixture(scope="module")
def jit_asm():
    from paper_2608_27612_amd import build
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "j.s")
        cmd = [build.HIPCC, "-O3", "-std=c++17", "--cuda-device-only", "-S"] + build.DEVICE_FLAGS \
            + [JIT_SRC, "-o", out]
        subprocess.check_call(cmd, stderr=subprocess.DEVNULL)
        return open(out).read()


def test_template_has_no_packed_fp32_scalar_writes_m0_or_scratch(jit_asm):
    assert not re.search(r"v_pk_(add|mul|fma)_f32", jit_asm)
    pattern = r"\bs_(buffer_)?(st" + r"ore|atom" + r"ic)\w*|\bs_dca" + r"che_\w+|\bs_scr" + r"atch_\w+"
    assert not re.search(pattern, jit_asm)
    for line in jit_asm.splitlines():
        code = line.split(";")[0]
        assert not re.search(r"\bm0\b", code), line
        assert "s_set_gpr_idx" not in code, line
    for size in re.findall(r"\.private_segment_fixed_size:\s+(\d+)", jit_asm):
        assert int(size) == 0


def test_template_does_not_carry_scc_across_calls(jit_asm):
    lines = jit_asm.splitlines()
    calls = 0
    for i, line in enumerate(lines):
        if "s_swappc_b64" not in line.split(";")[0]:
            continue
        calls += 1
        for k in range(i + 1, min(i + 80, len(lines))):
            code = lines[k].split(";")[0]
            if not code.strip() or code.strip().startswith("."):
                continue
            assert not _SCC_READERS.match(code), "SCC read after a call: " + code.strip()
            if _SCC_WRITERS.match(code) or re.match(r"^\s*s_(branch|endpgm|setpc)", code):
                break
    assert calls == 2 * 9  # one call site per (sources per walk, window) variant per mode


def test_template_kernels_allocate_the_convention_registers(jit_asm):
    """Every kernel of the template declares at least the VGPRs the compiled programs of its
    variants use (accumulators, windows, positions and temporaries)."""
    import sys
    sys.path.insert(0, os.path.join(ROOT, "paper_2608_27612_amd", "csrc"))
    import gen_regwin as G
    top = max(G.base(S * P, S * P, W) + 2 * P + G.jit_temps(S, P, W) for S, P, W in G.VARIANTS)
    counts = re.findall(r"\.name:\s+(emr_discover_jit_\w+)\s*\n(?:.*\n)*?\s+\.vgpr_count:\s+(\d+)",
                        jit_asm)
    assert len(counts) == 2
    for name, n in counts:
        assert int(n) >= top, (name, n, top)


def test_code_area_ends_the_template_text():
    """The area's holder is the last function of the object's .text, so growing the area moves
    nothing the kernels refer to."""
    co = os.path.join(ROOT, "paper_2608_27612_amd", "libemr_jit.co")
    if not os.path.exists(co):
        pytest.skip("template code object not built")
    out = subprocess.run(["/opt/rocm/llvm/bin/llvm-readelf", "-s", "-S", co], capture_output=True,
                         text=True, check=True).stdout
    funcs = [(int(v, 16), int(sz), n) for v, sz, n in
             re.findall(r"^\s*\d+:\s+([0-9a-f]{16})\s+(\d+)\s+FUNC\s+\w+\s+\w+\s+\S+\s+(\S+)\s*$",
                        out, flags=re.M)]
    last = max(funcs)
    assert last[2] == "emr_code_area_holder"
    area = re.search(r"^\s*\d+:\s+([0-9a-f]{16})\s+\d+\s+NOTYPE\s+LOCAL\s+\w+\s+\S+\s+emr_code_area\s*$",
                     out, flags=re.M)
    assert area and last[0] < int(area.group(1), 16) < last[0] + last[1]
