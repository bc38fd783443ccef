"""Test helper: the library's host packer compiled without HIP (tests/shim/pack_shim.cpp), plus a
float64 numpy interpreter of the packed program format. It is a packer test, not an oracle: the
tests compare what it computes from packed programs with the oracle's raw-genome evaluation.
"""

from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SHIM_SRC = os.path.join(HERE, "shim", "pack_shim.cpp")
PACK_SRC = os.path.join(ROOT, "paper_2608_27612_amd", "csrc", "pack.cpp")
JIT_SRC = os.path.join(ROOT, "paper_2608_27612_amd", "csrc", "jit.cpp")
PLAN_SRC = os.path.join(ROOT, "paper_2608_27612_amd", "csrc", "plan.cpp")
JIT_DEPS = [os.path.join(ROOT, "paper_2608_27612_amd", "csrc", f)
            for f in ("jit.h", "emr_internal.h", "pack.h", "plan.h")]
SHIM_LIB = os.path.join(HERE, "shim", "libpackshim.so")

_lib = None


def shim():
    global _lib
    if _lib is None:
        srcs = [SHIM_SRC, PACK_SRC, JIT_SRC, PLAN_SRC]
        if (not os.path.exists(SHIM_LIB)
                or max(os.path.getmtime(s) for s in srcs + JIT_DEPS) > os.path.getmtime(SHIM_LIB)):
            tmp = SHIM_LIB + ".tmp%d" % os.getpid()
            subprocess.check_call(["g++", "-std=c++17", "-O1", "-fPIC", "-shared"] + srcs
                                  + ["-o", tmp])
            os.replace(tmp, SHIM_LIB)
        L = C.CDLL(SHIM_LIB)
        L.shim_pack.restype = C.c_int
        L.shim_pack.argtypes = [C.c_void_p, C.c_void_p, C.c_int64, C.POINTER(C.c_int64), C.c_void_p,
                                C.c_void_p, C.c_char_p, C.c_int]
        L.shim_compile.restype = C.c_int
        L.shim_compile.argtypes = [C.c_void_p, C.c_uint32, C.c_int, C.c_int, C.c_int, C.c_int,
                                   C.c_void_p, C.c_int64, C.POINTER(C.c_int64), C.c_char_p,
                                   C.c_int64, C.c_char_p, C.c_int]
        L.shim_grow.restype = C.c_int
        L.shim_grow.argtypes = [C.c_void_p, C.c_int64, C.c_int64, C.c_int64, C.c_void_p, C.c_int64,
                                C.POINTER(C.c_int64), C.POINTER(C.c_int64), C.c_char_p, C.c_int]
        L.shim_plan_check.restype = C.c_int
        L.shim_plan_check.argtypes = [C.c_void_p, C.c_int32, C.c_int, C.c_void_p, C.c_int32,
                                      C.c_void_p, C.c_int32, C.c_int32, C.c_int,
                                      C.POINTER(C.c_int64), C.c_char_p, C.c_int]
        _lib = L
    return _lib


def pack(genome):
    """Pack one genome on the host. Returns (status, blob, desc[2][4], info[2][12], message)."""
    from paper_2608_27612_amd.emr import _genome_array
    arr, keep = _genome_array([genome])
    cap = 1 << 16
    blob = np.zeros(cap, np.uint32)
    words = C.c_int64()
    desc = np.zeros(16, np.uint32)
    info = np.zeros(24, np.int32)
    msg = C.create_string_buffer(256)
    st = shim().shim_pack(C.byref(arr[0]), blob.ctypes.data, cap, C.byref(words),
                          desc.ctypes.data, info.ctypes.data, msg, 256)
    del keep
    return st, blob[:words.value], desc.reshape(2, 8), info.reshape(2, 12), msg.value.decode()


def _act(a, z):
    if a == 0:
        return z
    if a == 1:
        return 1.0 / (1.0 + np.exp(-z))
    if a == 2:
        return np.tanh(z)
    if a == 3:
        return np.exp(-z * z)
    if a == 4:
        return np.sin(z)
    if a == 5:
        return np.abs(z)
    raise ValueError(a)


def _act_scaled(a, zs):
    """A varying node's activation of its scaled input zs = c z, with the input scales the packer
    applies (sigmoid -log2 e, tanh -2 log2 e, gaussian sqrt(log2 e), sine 1 / (2 pi))."""
    if a == 1:
        return 1.0 / (1.0 + np.exp2(zs))
    if a == 2:
        return 2.0 / (1.0 + np.exp2(zs)) - 1.0
    if a == 3:
        return np.exp2(-zs * zs)
    if a == 4:
        return np.sin(2.0 * np.pi * (zs - np.floor(zs)))
    return _act(a, zs)


def f32(u):
    return float(np.array([u], np.uint32).view(np.float32)[0])


def uniform_part(blob, desc, dir_, sx, sy):
    """The uniform program of `desc[dir_]` for source (sx, sy): its node values U, the output's
    index out_u, and the folded bias of every varying node with the record it starts at."""
    var_off, n_rec, n_steps, uni_off, flags = (int(v) for v in desc[dir_][:5])
    U = np.zeros(5 + 300)
    if dir_ == 0:
        U[0], U[1] = sx, sy
    else:
        U[2], U[3] = sx, sy
    U[4] = 1.0
    n_un, out_u = int(blob[uni_off]), int(blob[uni_off + 1])
    rec = uni_off + 4
    for k in range(n_un):
        act, ne, eo, bb = (int(v) for v in blob[rec + 4 * k: rec + 4 * k + 4])
        z = f32(bb)
        for e in range(ne):
            z += f32(blob[uni_off + eo + 2 * e + 1]) * U[int(blob[uni_off + eo + 2 * e])]
        U[5 + k] = _act(act, np.float64(z))
    fold = rec + 4 * n_un
    folded, fold_rec = [], []
    for t in range(n_steps):
        nf, fo, bb = int(blob[fold + 4 * t]), int(blob[fold + 4 * t + 1]), int(blob[fold + 4 * t + 2])
        z = f32(bb)
        for e in range(nf):
            z += f32(blob[uni_off + fo + 2 * e + 1]) * U[int(blob[uni_off + fo + 2 * e])]
        folded.append(z)
        fold_rec.append(int(blob[fold + 4 * t + 3]))
    return U, out_u, folded, fold_rec


def bias_rows(blob, desc, dir_, sources):
    """The bias rows a group of these sources (x, y pairs, up to 4) sees: row 0 the output
    constants of a uniform output, row 1 + r the folded biases of the node starting at record r
    (what the bind kernel writes), as a flat array of 4 floats per row."""
    n_rec = int(desc[dir_][1])
    rows = np.zeros((n_rec + 2, 4))
    for s, (sx, sy) in enumerate(sources):
        U, out_u, folded, fold_rec = uniform_part(blob, desc, dir_, sx, sy)
        if out_u != 0xFFFFFFFF:
            rows[0, s] = U[out_u]
        for z, r in zip(folded, fold_rec):
            rows[1 + r, s] = z
    return rows.reshape(-1)


def _operand(tok, V, S_):
    if tok.startswith("-v"):
        return -V[int(tok[2:])]
    if tok.startswith("v"):
        return V[int(tok[1:])]
    if tok.startswith("s"):
        return S_[int(tok[1:])]
    if tok.startswith("0x"):
        return f32(int(tok, 16))
    consts = {"0.5": 0.5, "-0.5": -0.5, "1.0": 1.0, "-1.0": -1.0, "2.0": 2.0, "-2.0": -2.0,
              "4.0": 4.0, "-4.0": -4.0, "0.15915494": f32(0x3e22f983)}
    if tok in consts:
        return consts[tok]
    i = int(tok)  # an inline integer constant: its bits as a float
    return f32(i & 0xFFFFFFFF)


def positions(rng, P):
    """P positions in sibling quads (x of child c depends on c & 1, y on c >> 1), as a lane holds
    them."""
    x0, y0 = rng.uniform(-1, 1, (2, P // 4, 2))
    c = np.arange(P) % 4
    q = np.arange(P) // 4
    return x0[q, c & 1], y0[q, c >> 1]


def emulate(listing, rows, x, y, M, W, stale_rows=False):
    """Executes a compiled program's listing on the host in float64 with exact transcendentals:
    `rows` are the group's bias rows (bias_rows), x and y the P positions (sibling quads, as
    `positions` makes them). Returns the VGPR file (a dict). Reading a register that nothing
    wrote raises KeyError, as an interpreter that reads an undefined slot would; only the
    registers of the convention hold positions (x of child c of quad k at X + 4 k + (c & 1), y at
    X + P + 4 k + (c & 2)). With `stale_rows`, s[40:55] start out holding garbage instead of the
    preloaded rows (what a program finds after a longer program of the same chunk ran)."""
    P = len(x)
    X = ((4 + M + 1) & ~1) + M * W
    V = {}
    for j in range(P):
        xj, yj = X + (j & ~3) + (j & 1), X + P + (j & ~3) + (j & 2)
        assert V.setdefault(xj, float(x[j])) == float(x[j]), "not a sibling quad"
        assert V.setdefault(yj, float(y[j])) == float(y[j]), "not a sibling quad"

    # on entry s[40:55] hold the group's bias rows 1 .. 4 (loaded by the caller once per chunk)
    S_ = {40 + k: (float(rows[4 + k]) if 4 + k < len(rows) else 0.0) for k in range(16)}
    if stale_rows:
        S_ = {40 + k: float("nan") for k in range(16)}
    for line in listing.strip().split("\n"):
        op, _, rest = line.partition(" ")
        a = [t.strip() for t in rest.split(",")] if rest else []
        if op == "s_load_dwordx4":
            base = int(a[0][2:].split(":")[0])
            assert a[1] == "s[56:57]"
            off = int(a[2], 16) // 4
            for k in range(4):
                S_[base + k] = float(rows[off + k])
            continue
        if op in ("s_waitcnt", "s_nop"):
            continue
        if op == "s_setpc_b64":
            assert a[0] == "s[58:59]"
            break
        d = int(a[0][1:])
        if op == "v_mov_b32_e32":
            V[d] = _operand(a[1], V, S_)
        elif op == "v_mul_f32_e32":
            V[d] = _operand(a[1], V, S_) * _operand(a[2], V, S_)
        elif op == "v_fmac_f32_e32":
            V[d] = _operand(a[1], V, S_) * _operand(a[2], V, S_) + V[d]
        elif op == "v_fmamk_f32":
            V[d] = _operand(a[1], V, S_) * _operand(a[2], V, S_) + _operand(a[3], V, S_)
        elif op == "v_add_f32_e32":
            V[d] = _operand(a[1], V, S_) + _operand(a[2], V, S_)
        elif op == "v_and_b32_e32":
            assert a[1] == "0x7fffffff"
            V[d] = abs(_operand(a[2], V, S_))
        elif op == "v_exp_f32_e32":
            V[d] = float(np.exp2(_operand(a[1], V, S_)))
        elif op == "v_rcp_f32_e32":
            V[d] = 1.0 / _operand(a[1], V, S_)
        elif op == "v_fract_f32_e32":
            z = _operand(a[1], V, S_)
            V[d] = z - np.floor(z)
        elif op == "v_sin_f32_e32":
            V[d] = float(np.sin(2.0 * np.pi * _operand(a[1], V, S_)))
        elif op == "v_fma_f32":
            V[d] = _operand(a[1], V, S_) * _operand(a[2], V, S_) + _operand(a[3], V, S_)
        elif op == "v_mul_f32_e64":
            V[d] = _operand(a[1], V, S_) * _operand(a[2], V, S_)
        else:
            raise ValueError("unknown instruction: " + line)
    return V


def interpret(blob, desc, dir_, sx, sy, px, py, nodes=None):
    """Evaluate packed program `desc[dir_]` for source (sx, sy) at positions (px, py) (arrays).
    With `nodes` (a list), appends (first record, shared mark, value) for every node in order."""
    var_off, n_rec, n_steps, uni_off, flags = (int(v) for v in desc[dir_][:5])
    # uniform program
    U = np.zeros(5 + 300)
    if dir_ == 0:
        U[0], U[1] = sx, sy
    else:
        U[2], U[3] = sx, sy
    U[4] = 1.0
    n_un, out_u, n_st = int(blob[uni_off]), int(blob[uni_off + 1]), int(blob[uni_off + 2])
    assert n_st == n_steps
    rec = uni_off + 4
    for k in range(n_un):
        act, ne, eo, bb = (int(v) for v in blob[rec + 4 * k: rec + 4 * k + 4])
        z = f32(bb)
        for e in range(ne):  # edge offsets count from uni_off
            z += f32(blob[uni_off + eo + 2 * e + 1]) * U[int(blob[uni_off + eo + 2 * e])]
        U[5 + k] = _act(act, np.float64(z))
    fold = rec + 4 * n_un
    folded = []
    fold_rec = [int(blob[fold + 4 * t + 3]) for t in range(n_steps)]
    for t in range(n_steps):
        nf, fo, bb = int(blob[fold + 4 * t]), int(blob[fold + 4 * t + 1]), int(blob[fold + 4 * t + 2])
        z = f32(bb)
        for e in range(nf):
            z += f32(blob[uni_off + fo + 2 * e + 1]) * U[int(blob[uni_off + fo + 2 * e])]
        folded.append(z)
    if not (flags & 1):
        assert n_steps == 0 and n_rec == 0
        return np.full(len(px), U[out_u]), (flags >> 8) & 0xFF
    window = (flags >> 8) & 0xFF
    assert var_off % 16 == 0
    vals = np.full((max(window, 1), len(px)), np.nan)
    acc = None
    step = 0
    nodes_done = 0
    out = None
    for r in range(n_rec):
        w = blob[var_off + 16 * r: var_off + 16 * r + 16].astype(np.int64)
        meta = int(w[0])
        tail, first = meta & 15, (meta >> 4) & 1
        dst, ne = (meta >> 8) & 31, (meta >> 16) & 15
        assert ne <= 11 and (meta >> 20) == 0 and (meta >> 6) & 3 == 0 and (meta >> 13) & 7 == 0
        assert first or not (meta >> 5) & 1, "a shared mark outside a node's first record"
        if out is not None:
            raise AssertionError("record after the output node")
        if first:
            assert acc is None, "a node starts before the previous one ended"
            assert fold_rec[step] == r, "the node's bias row is not its first record's"
            node_first, node_shared = r, (meta >> 5) & 1
            acc = folded[step] + f32(w[1]) * px + f32(w[2]) * py
        else:
            assert acc is not None and w[1] == 0 and w[2] == 0
        for e in reversed(range(ne)):   # positions n-1 .. 0 hold the edges in edge-list order
            src = (int(w[3 + e // 6]) >> (5 * (e % 6))) & 31
            assert src < window
            v = vals[src]
            assert not np.isnan(v).any(), "read of a slot that holds no live value"
            acc = acc + f32(w[5 + e]) * v
        for e in range(ne, 11):
            assert w[5 + e] == 0 and ((int(w[3 + e // 6]) >> (5 * (e % 6))) & 31) == 0
        if tail == 0:
            continue
        assert 1 <= tail <= 12
        if tail <= 6:
            assert dst < window
            vals[dst] = _act_scaled(tail - 1, acc)
            value = vals[dst]
        else:
            assert not node_shared, "the output node is marked shared"
            out = _act_scaled(tail - 7, acc)
            value = out
        if nodes is not None:
            nodes.append((node_first, node_shared, np.array(value)))
        acc = None
        step += 1
    assert step == n_steps and out is not None
    return out, window


def compile_program(blob, desc, S, P, W):
    """The compiled tier's machine words and assembly listing for one packed program (desc: its
    ProgDesc words) at S sources, P positions per lane and register window W."""
    var_off, n_rec, flags = int(desc[0]), int(desc[1]), int(desc[4])
    rec = np.ascontiguousarray(blob[var_off:var_off + 16 * n_rec], np.uint32)
    if rec.size == 0:
        rec = np.zeros(16, np.uint32)
    cap = 1 << 20
    words = np.zeros(cap, np.uint32)
    n = C.c_int64()
    listing = C.create_string_buffer(1 << 24)
    msg = C.create_string_buffer(256)
    st = shim().shim_compile(rec.ctypes.data, n_rec, flags & 1, S, P, W, words.ctypes.data, cap,
                             C.byref(n), listing, 1 << 24, msg, 256)
    if st != 0:
        raise ValueError("compile failed (%d): %s" % (st, msg.value.decode()))
    return words[:n.value].copy(), listing.value.decode()


def grow_template(img, area_bytes, new_bytes):
    """The template code object bytes with the code area grown; returns (image, area_offset)."""
    src = np.frombuffer(img, np.uint8)
    cap = len(img) + new_bytes + (1 << 16)
    out = np.zeros(cap, np.uint8)
    n = C.c_int64()
    off = C.c_int64()
    msg = C.create_string_buffer(256)
    st = shim().shim_grow(src.ctypes.data, len(img), area_bytes, new_bytes, out.ctypes.data, cap,
                          C.byref(n), C.byref(off), msg, 256)
    if st != 0:
        raise ValueError("grow failed (%d): %s" % (st, msg.value.decode()))
    return out[:n.value].tobytes(), off.value
