"""The compiled tier's host side (no GPU): the code generator's machine words against the AMDGPU
assembler, the compiled programs' arithmetic (emulated from their listings) against the float64
interpreter of the packed format, the one hazard rule the programs must keep, and the resized
template code object against the ELF tools."""

import os
import re
import subprocess
import sys

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, HERE)
sys.path.insert(0, os.path.join(ROOT, "paper_2608_27612_amd", "csrc"))

import packed_interp as PI  # noqa: E402
import gen_regwin as G  # noqa: E402
from paper_2608_27612_amd import emr, workloads as W  # noqa: E402

LLVM = "/opt/rocm/llvm/bin"
TEMPLATE = os.path.join(ROOT, "paper_2608_27612_amd", "libemr_jit.co")
TEMPLATE_AREA = 4096


def have(tool):
    return os.path.exists(os.path.join(LLVM, tool))


def variants(window):
    """(S, P, W) of every kernel variant a program with this register window can run in."""
    wb = next(w for w in (4, 8, 16, 32) if window <= w)
    return [(S, G.positions_per_lane(S, wb), wb) for S in range(1, G.max_group(wb) + 1)]


def programs(genomes):
    for gi, g in enumerate(genomes):
        st, blob, desc, info, msg = PI.pack(g)
        assert st == 0, msg
        for d in range(2):
            for S, P, Wn in variants(int(info[d][9])):
                yield gi, blob, desc, d, S, P, Wn


def assemble(listing):
    r = subprocess.run([os.path.join(LLVM, "llvm-mc"), "-arch=amdgcn", "-mcpu=gfx950",
                        "-show-encoding"], input=listing, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[:2000]
    enc = []
    for line in r.stdout.split("\n"):
        if "encoding:" in line:
            enc += [int(b, 16) for b in line.split("encoding: [")[1].rstrip("]").split(",")]
    return np.frombuffer(bytes(enc), np.uint32)


POPS = [W.population(11, 12, 20, 60), W.population(12, 4, 40, 120)]


@pytest.mark.skipif(not have("llvm-mc"), reason="no AMDGPU assembler")
@pytest.mark.parametrize("pop", [0, 1])
def test_machine_words_match_the_assembler(pop):
    n = 0
    for gi, blob, desc, d, S, P, Wn in programs(POPS[pop]):
        words, listing = PI.compile_program(blob, desc[d], S, P, Wn)
        ref = assemble(listing)
        assert np.array_equal(ref, words), (gi, d, S, P, Wn)
        n += 1
    assert n > 10


def test_compiled_programs_compute_the_packed_programs():
    """Every instance's output, emulated from the listing, equals the packed program's value at
    that source and position (float64 on both sides; the emulator refuses undefined reads)."""
    rng = np.random.default_rng(5)
    n = 0
    for gi, blob, desc, d, S, P, Wn in programs(POPS[0] + POPS[1][:2]):
        M = S * P
        srcs = [(float(rng.uniform(-1, 1)), float(rng.uniform(-1, 1))) for _ in range(S)]
        x, y = PI.positions(rng, P)
        words, listing = PI.compile_program(blob, desc[d], S, P, Wn)
        V = PI.emulate(listing, PI.bias_rows(blob, desc, d, srcs), x, y, M, Wn)
        for s, (sx, sy) in enumerate(srcs):
            want, _ = PI.interpret(blob, desc, d, sx, sy, x, y)
            got = np.array([V[4 + s * P + j] for j in range(P)])
            assert np.allclose(got, want, rtol=1e-9, atol=1e-9), (gi, d, S, P, Wn, s)
        n += 1
    assert n > 10


def test_shared_nodes_are_evaluated_once_and_a_shared_mark_on_the_output_is_ignored():
    """With S > 1 a node marked shared is evaluated for the first source's instances only (fewer
    instructions than the same program with its marks cleared, same values for every source), and
    a shared mark planted on the output node's first record changes nothing: every source still
    gets its own output."""
    rng = np.random.default_rng(12)
    fewer = planted = 0
    for gi, blob, desc, d, S, P, Wn in programs(POPS[0] + POPS[1][:2]):
        if S == 1:
            continue
        var_off, n_rec = int(desc[d][0]), int(desc[d][1])
        metas = [int(blob[var_off + 16 * r]) for r in range(n_rec)]
        if not any(m & 32 for m in metas):
            continue
        srcs = [(float(rng.uniform(-1, 1)), float(rng.uniform(-1, 1))) for _ in range(S)]
        x, y = PI.positions(rng, P)
        rows = PI.bias_rows(blob, desc, d, srcs)
        want = [PI.interpret(blob, desc, d, sx, sy, x, y)[0] for sx, sy in srcs]
        cleared = blob.copy()
        for r in range(n_rec):
            cleared[var_off + 16 * r] &= ~np.uint32(32)
        w_shared, _ = PI.compile_program(blob, desc[d], S, P, Wn)
        w_full, _ = PI.compile_program(cleared, desc[d], S, P, Wn)
        assert len(w_shared) < len(w_full), (gi, d)
        fewer += 1
        # plant the mark on the output node's first record (the last node's)
        out_first = max(r for r in range(n_rec) if metas[r] & 16)
        bad = blob.copy()
        bad[var_off + 16 * out_first] |= np.uint32(32)
        _, listing = PI.compile_program(bad, desc[d], S, P, Wn)
        V = PI.emulate(listing, rows, x, y, S * P, Wn)
        for s in range(S):
            got = np.array([V[4 + s * P + j] for j in range(P)])
            assert np.allclose(got, want[s], rtol=1e-9, atol=1e-9), (gi, d, s)
        planted += 1
    assert fewer > 5 and planted > 5


def test_programs_load_only_rows_the_caller_did_not_preload():
    """A program whose nodes all start in records 0 .. 3 uses the preloaded rows and loads
    nothing; a longer one loads every row it uses (so it runs right whatever s[40:55] hold)."""
    rng = np.random.default_rng(9)
    seen_long = seen_short = 0
    for gi, blob, desc, d, S, P, Wn in programs(POPS[1] + POPS[0][:6]):
        n_rec = int(desc[d][1])
        if not (int(desc[d][4]) & 1) or n_rec == 0:
            continue
        var_off = int(desc[d][0])
        firsts = [r for r in range(n_rec) if blob[var_off + 16 * r] & 16]
        _, listing = PI.compile_program(blob, desc[d], S, P, Wn)
        loads = [l for l in listing.splitlines() if l.startswith("s_load")]
        if max(firsts) < 4:
            assert not loads
            seen_short += 1
            continue
        seen_long += 1
        srcs = [(float(rng.uniform(-1, 1)), float(rng.uniform(-1, 1))) for _ in range(S)]
        x, y = PI.positions(rng, P)
        V = PI.emulate(listing, PI.bias_rows(blob, desc, d, srcs), x, y, S * P, Wn,
                       stale_rows=True)
        for s, (sx, sy) in enumerate(srcs):
            want, _ = PI.interpret(blob, desc, d, sx, sy, x, y)
            got = np.array([V[4 + s * P + j] for j in range(P)])
            assert np.allclose(got, want, rtol=1e-9, atol=1e-9)
    assert seen_long > 0 and seen_short > 0


def test_uniform_output_program_copies_row_zero():
    g = W.single_cppn(0, 3, 6)[0]
    # no enabled edge leaves x2 or y2: for outgoing queries the output is a per-source constant
    g["enabled"] = np.where(np.isin(g["src"], [2, 3]), 0, 1).astype(np.uint8)
    st, blob, desc, info, msg = PI.pack(g)
    assert st == 0 and not (int(desc[0][4]) & 1)
    words, listing = PI.compile_program(blob, desc[0], 3, 8, 4)
    assert listing.splitlines()[0] == "s_load_dwordx4 s[40:43], s[56:57], 0x0"
    rows = np.zeros(8)
    rows[:3] = [0.25, -1.5, 3.0]
    V = PI.emulate(listing, rows, np.zeros(8), np.zeros(8), 24, 4)
    assert [V[4 + m] for m in range(24)] == [0.25] * 8 + [-1.5] * 8 + [3.0] * 8



def _writes(listing):
    """(opcode, destination VGPR, source text) of every vector instruction in a listing."""
    out = []
    for line in listing.strip().split("\n"):
        op, _, rest = line.partition(" ")
        if op.startswith("v_"):
            dst, _, srcs = rest.partition(",")
            out.append((op, int(dst.strip()[1:]), srcs))
    return out


def test_nodes_without_position_terms_start_with_their_first_edge():
    """A node's bias is folded into its first edge (v_fmamk): no accumulator is set by a move
    and then summed into by v_fmac."""
    fused = 0
    for gi, blob, desc, d, S, P, Wn in programs(POPS[0] + POPS[1]):
        _, listing = PI.compile_program(blob, desc[d], S, P, Wn)
        last = {}
        for op, dst, srcs in _writes(listing):
            if op == "v_fmac_f32_e32":
                assert last.get(dst) != "v_mov_b32_e32", (gi, d, S, P, Wn, dst)
            fused += op == "v_fmamk_f32" and dst < 4 + S * P
            last[dst] = op
    assert fused > 0


def _rec_slots(blob, off):
    """(edge source slots, tail, destination slot) of the record at blob[off]."""
    meta = int(blob[off])
    ne = (meta >> 16) & 15
    srcs = [(int(blob[off + 3 + e // 6]) >> (5 * (e % 6))) & 31 for e in range(ne)]
    return srcs, meta & 15, (meta >> 8) & 31


def _linear_store_counts(blob, desc, d):
    """(linear nodes that store their value, those of them whose own edges read the slot they
    store into) of one program."""
    var_off, n_rec = int(desc[d][0]), int(desc[d][1])
    n = clash = 0
    reads = set()
    for r in range(n_rec):
        srcs, tail, dst = _rec_slots(blob, var_off + 16 * r)
        if int(blob[var_off + 16 * r]) & 16:
            reads = set()
        reads |= set(srcs)
        n += tail == 1
        clash += tail == 1 and dst in reads
    return n, clash


def test_linear_nodes_sum_in_their_destination_slot():
    """A linear node that stores its value sums in its destination slot (no copy from an
    accumulator); one whose own edges read that slot (the packer reuses an input's slot when
    the input dies at the node) keeps the accumulator and copies it; both compute the packed
    program."""
    rng = np.random.default_rng(13)
    in_place = clashing = 0
    for gi, blob, desc, d, S, P, Wn in programs(W.population(21, 60, 20, 60)):
        if not (int(desc[d][4]) & 1):
            continue
        n_lin, n_clash = _linear_store_counts(blob, desc, d)
        if n_lin == 0:
            continue
        M = S * P
        _, listing = PI.compile_program(blob, desc[d], S, P, Wn)
        copies = [w for w in _writes(listing)
                  if w[0] == "v_mov_b32_e32" and re.fullmatch(r"\s*v(\d+)", w[2])
                  and 4 <= int(w[2].strip()[1:]) < 4 + M]
        assert len(copies) == M * n_clash, (gi, d, S, P, Wn)
        srcs = [(float(rng.uniform(-1, 1)), float(rng.uniform(-1, 1))) for _ in range(S)]
        x, y = PI.positions(rng, P)
        V = PI.emulate(listing, PI.bias_rows(blob, desc, d, srcs), x, y, M, Wn)
        for s, (sx, sy) in enumerate(srcs):
            want, _ = PI.interpret(blob, desc, d, sx, sy, x, y)
            got = np.array([V[4 + s * P + j] for j in range(P)])
            assert np.allclose(got, want, rtol=1e-9, atol=1e-9), (gi, d, S, P, Wn, s)
        in_place += n_lin - n_clash
        clashing += n_clash
    assert in_place > 0 and clashing > 0, (in_place, clashing)


TRANS = ("v_exp_f32", "v_rcp_f32", "v_sin_f32")


def test_transcendental_results_are_never_read_by_the_next_instruction():
    for gi, blob, desc, d, S, P, Wn in programs(POPS[0]):
        _, listing = PI.compile_program(blob, desc[d], S, P, Wn)
        lines = listing.strip().split("\n")
        for a, b in zip(lines, lines[1:]):
            if a.startswith(TRANS):
                dst = a.split()[1].rstrip(",")
                assert not re.search(r"(?<![\w])-?%s\b" % dst, b.partition(" ")[2]), (a, b)
        # the caller reads the accumulators right after the return
        assert lines[-1] == "s_setpc_b64 s[58:59]"
        if any(l.startswith(TRANS) for l in lines):
            assert lines[-2] == "s_nop 1"


def test_register_use_stays_inside_the_convention():
    """Only the accumulators, windows, positions (read only, at the registers of the
    convention) and temporaries of the variant, and SGPRs s[40:59]."""
    for gi, blob, desc, d, S, P, Wn in programs(POPS[1] + POPS[0][:4]):
        M = S * P
        X = ((4 + M + 1) & ~1) + M * Wn
        top = X + 2 * P + G.jit_temps(S, P, Wn)
        pos = {X + (j & ~3) + (j & 1) for j in range(P)} | {X + P + (j & ~3) + (j & 2)
                                                             for j in range(P)}
        _, listing = PI.compile_program(blob, desc[d], S, P, Wn)
        for v in re.findall(r"\bv(\d+)\b", listing):
            assert 4 <= int(v) < top
            assert not X <= int(v) < X + 2 * P or int(v) in pos, (gi, d, S, P, Wn, v)
        for op, dst, srcs in _writes(listing):
            assert not X <= dst < X + 2 * P, (gi, d, S, P, Wn, op, dst)
        for s in re.findall(r"\bs(\d+)\b", listing):
            assert 40 <= int(s) <= 59
        for a, b in re.findall(r"s\[(\d+):(\d+)\]", listing):
            assert 40 <= int(a) and int(b) <= 59


def test_bad_variants_are_refused():
    g = W.single_cppn(0, 8, 20)[0]
    st, blob, desc, info, msg = PI.pack(g)
    for S, P, Wn in [(4, 4, 4), (1, 4, 5), (3, 8, 8), (1, 8, 4)]:
        with pytest.raises(ValueError):
            PI.compile_program(blob, desc[0], S, P, Wn)


def readelf(path):
    r = subprocess.run([os.path.join(LLVM, "llvm-readelf"), "-h", "-l", "-S", "-s", "--dyn-syms",
                        path], capture_output=True, text=True)
    assert r.returncode == 0 and "warning" not in r.stderr.lower(), r.stderr
    return r.stdout


def sections(text):
    out = {}
    for m in re.finditer(r"\][ \t]+(\.\S+)[ \t]+\S+[ \t]+([0-9a-f]{16})[ \t]+([0-9a-f]{6,})"
                         r"[ \t]+([0-9a-f]{6,})", text):
        out[m.group(1)] = tuple(int(m.group(k), 16) for k in (2, 3, 4))
    return out


def symbols(text):
    out = {}
    for m in re.finditer(r"^[ \t]*\d+:[ \t]+([0-9a-f]{16})[ \t]+(\d+)[ \t]+\w+[ \t]+\w+[ \t]+\w+"
                         r"[ \t]+\S+[ \t]+(\S+)[ \t]*$", text, flags=re.M):
        out.setdefault(m.group(3), (int(m.group(1), 16), int(m.group(2))))
    return out


@pytest.mark.skipif(not (os.path.exists(TEMPLATE) and have("llvm-readelf")),
                    reason="template code object not built")
@pytest.mark.parametrize("pages", [0, 1, 37])
def test_grown_template_is_a_consistent_code_object(tmp_path, pages):
    img = open(TEMPLATE, "rb").read()
    new = TEMPLATE_AREA + 4096 * pages
    out, off = PI.grow_template(img, TEMPLATE_AREA, new)
    assert len(out) == len(img) + 4096 * pages
    area = np.frombuffer(out[off:off + new], np.uint32)
    assert np.all(area == 0xBF810000)
    p0, p1 = tmp_path / "a.co", tmp_path / "b.co"
    p0.write_bytes(img)
    p1.write_bytes(out)
    t0, t1 = readelf(str(p0)), readelf(str(p1))
    s0, s1 = sections(t0), sections(t1)
    d = 4096 * pages
    assert s1[".text"] == (s0[".text"][0], s0[".text"][1], s0[".text"][2] + d)
    for name, (addr, offs, size) in s0.items():
        if offs > s0[".text"][1]:
            assert s1[name][1] == offs + d and s1[name][2] == size, name
            if addr:
                assert s1[name][0] == addr + d, name
        elif name != ".text":
            assert s1[name] == (addr, offs, size), name
    # section contents are the template's (headers and symbol tables are rewritten and checked
    # below); .text up to the area, and after it, unchanged
    for name in (".note", ".gnu.hash", ".hash", ".dynstr", ".rodata"):
        if name in s0:
            o, n = s0[name][1], s0[name][2]
            assert out[o:o + n] == img[o:o + n], name
    assert out[s0[".text"][1]:off] == img[s0[".text"][1]:off]
    text_end = s0[".text"][1] + s0[".text"][2]
    dyn_off, dyn_size = s0[".dynamic"][1], s0[".dynamic"][2]
    assert out[off + new:text_end + d] == img[off + TEMPLATE_AREA:text_end]
    assert out[dyn_off + d:dyn_off + d + dyn_size] == img[dyn_off:dyn_off + dyn_size]
    y0, y1 = symbols(t0), symbols(t1)
    assert y1["emr_code_area"] == y0["emr_code_area"]
    for k in ("emr_discover_jit_records", "emr_discover_jit_records.kd", "emr_discover_jit_raw"):
        assert y1[k] == y0[k]
    assert y1["emr_code_area_holder"][1] == y0["emr_code_area_holder"][1] + d
    if "_DYNAMIC" in y0:
        assert y1["_DYNAMIC"][0] == y0["_DYNAMIC"][0] + d
    r = subprocess.run([os.path.join(LLVM, "llvm-objdump"), "-d", str(p1)], capture_output=True,
                       text=True)
    assert r.returncode == 0 and "<emr_discover_jit_records>:" in r.stdout


@pytest.mark.skipif(not os.path.exists(TEMPLATE), reason="template code object not built")
def test_template_area_sizes_are_checked():
    img = open(TEMPLATE, "rb").read()
    with pytest.raises(ValueError):
        PI.grow_template(img, TEMPLATE_AREA, TEMPLATE_AREA + 100)   # not whole pages
    with pytest.raises(ValueError):
        PI.grow_template(img, TEMPLATE_AREA - 4, TEMPLATE_AREA)     # wrong area size
    with pytest.raises(ValueError):
        PI.grow_template(img[:1000], TEMPLATE_AREA, TEMPLATE_AREA)  # truncated object


def test_jit_policy_is_validated():
    for p in (emr.EMR_JIT_OFF, emr.EMR_JIT_ALWAYS, emr.EMR_JIT_AUTO):
        emr.emr_set_jit(p)
    for bad in (-1, 3):
        with pytest.raises(emr.EmrError) as e:
            emr.emr_set_jit(bad)
        assert e.value.status == emr.EMR_E_INVAL
