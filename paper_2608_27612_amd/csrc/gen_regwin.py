#!/usr/bin/env python3
"""Generates regwin_gen.h: the program-record step of the discover kernel, as inline assembly.

A lane evaluates M = S * P CPPN instances at once (S sources of one genome at P grid positions:
the four children of one or two parent cells).
Instance m = s * P + j keeps
  - its accumulator in v[ACC + m], and
  - its position-dependent node values in a VGPR tuple v[base(m) .. base(m) + W - 1].
Walker<S, P, W>::step() processes one 16-word program record (layout in emr_internal.h) for all M
instances in ONE asm statement, so the accumulators and tuples are bound to their registers at a
single site inside the program loop and the compiler never needs to move them:

  1. first record of a node: acc = bias_s + ax x_j + ay y_j
  2. the record's n edges: a computed jump into 11 fixed-size blocks (entered at block 11 - n);
     each block extracts one slot index (s_bfe_u32 of log2(W) bits, which also confines it to the
     instance's own tuple), sets it as the source-operand index (s_set_gpr_idx_idx) and issues the
     M fused multiply-adds acc_m += w * tuple_m[slot]. The packer stores a node's edges in reverse
     record positions, so they are accumulated in edge-list order.
  3. the tail, through a branch table on meta bits 0..3: the node's activation, whose last
     instruction writes straight into the destination slot of every tuple (DST indexing), or, for
     the output node, the activation in place on the accumulators; nothing for a continuation
     record. The accumulator holds the node's input already multiplied by its activation's input
     scale (the packer scales the weights and biases), which leaves 1 to 4 instructions per
     activation.

The statement declares SCC and M0 as clobbered: its scalar arithmetic writes SCC, and the
register-indexing instructions write M0.

Hazards: the statement is opaque to the compiler's hazard recognizer, so it keeps the one that
applies here itself: a non-transcendental VALU instruction that reads the result of a
transcendental one (v_exp, v_rcp, v_sin) needs one wait state in between; every such pair below
is at least M >= 4 instructions apart, and the output tails end with s_nop 1, since the caller
reads the accumulators next. Branch targets are computed from label differences, so the jump
arithmetic follows the assembler's actual encodings.

Inline assembly needs literal register names, so every variant is spelled out here.
Run from this directory: python gen_regwin.py > regwin_gen.h
"""

ACC = 4
MAX_EDGES = 11
SLOT_BITS = 5


def fits_lane(S, P, W):
    """The positions-per-lane policy of the kernels (emr_internal.h), restated."""
    return S * P * W <= 128 and 16 + S * P + S * P * W + 2 * P + 2 * S <= 168


def positions_per_lane(S, W):
    return next(P for P in (16, 8, 4) if P == 4 or fits_lane(S, P, W))


def max_group(W):
    return next(S for S in (3, 2, 1) if S == 1 or fits_lane(S, 4, W))


# (S, P, W) variants
VARIANTS = [(S, positions_per_lane(S, W), W) for W in (4, 8, 16, 32)
            for S in range(1, max_group(W) + 1)]

ACTS = ["lin", "sig", "tanh", "gau", "sin", "abs"]  # activation ids 0..5


def base(M, m, W):
    first = ACC + M
    first += first & 1  # tuples start on an even register
    return first + m * W


def log2(w):
    return {4: 2, 8: 3, 16: 4, 32: 5}[w]


def bfe_imm(offset, width):
    return "0x%x" % (offset | (width << 16))


# Fixed scalar registers of the walk statement: the current record (16 words), the current bias
# row (4 floats), the record and row pointers, and the computed-jump PC pair.
REC = 40   # s[40:55]: meta, ax, ay, sw0, sw1, w0..w10
ROW = 56   # s[56:59]
RP = 60    # s[60:61]
BP = 62    # s[62:63]
PC = 64    # s[64:65]


def tail_stride(M):
    """Byte stride of the activation tails: a power of two above the longest tail (the tanh
    store, 4 M vector instructions and 6 scalar ones), at 8 bytes per instruction at most."""
    longest = 8 * (4 * M + 6)
    return 1 << (longest - 1).bit_length()


def gen_walker(S, P, W):
    M = S * P
    A = ["v%d" % (ACC + m) for m in range(M)]
    T = ["v%d" % base(M, m, W) for m in range(M)]
    meta, ax, ay = "s%d" % REC, "s%d" % (REC + 1), "s%d" % (REC + 2)
    sw = ["s%d" % (REC + 3), "s%d" % (REC + 4)]
    wt = ["s%d" % (REC + 5 + p) for p in range(MAX_EDGES)]
    bias = ["s%d" % (ROW + s) for s in range(S)]
    pc = "s[%d:%d]" % (PC, PC + 1)
    L = []
    # ---- a program without records (uniform output): the outputs are the constants of row 0
    L += ["s_cmp_lg_u32 %[n], 0",
          "s_cbranch_scc1 .Lstart_%=",
          "s_load_dwordx4 s[%d:%d], s[%d:%d], 0x0" % (ROW, ROW + 3, BP, BP + 1),
          "s_waitcnt lgkmcnt(0)"]
    L += ["v_mov_b32 %s, %s" % (A[s * P + j], bias[s]) for s in range(S) for j in range(P)]
    L += ["s_branch .Ldone_%="]
    # ---- else load record 0 and its row (row 1)
    L += [".Lstart_%=:",
          "s_add_u32 s%d, s%d, 16" % (BP, BP),
          "s_addc_u32 s%d, s%d, 0" % (BP + 1, BP + 1),
          "s_load_dwordx16 s[%d:%d], s[%d:%d], 0x0" % (REC, REC + 15, RP, RP + 1),
          "s_load_dwordx4 s[%d:%d], s[%d:%d], 0x0" % (ROW, ROW + 3, BP, BP + 1)]
    # ---- one record per iteration; its record and row were loaded during the previous one
    L += [".Lrec_%=:",
          "s_waitcnt lgkmcnt(0)",
          "s_add_u32 s%d, s%d, 64" % (RP, RP),
          "s_addc_u32 s%d, s%d, 0" % (RP + 1, RP + 1)]
    # 1. first record of a node: the accumulator starts at bias + ax x + ay y
    L += ["s_bitcmp1_b32 %s, 4" % meta, "s_cbranch_scc0 .Lni_%="]
    if S == 1:
        L.append("v_mov_b32 %%[tb], %s" % bias[0])
        L += ["v_fma_f32 %s, %%[x%d], %s, %%[tb]" % (A[j], j, ax) for j in range(P)]
        L += ["v_fma_f32 %s, %%[y%d], %s, %s" % (A[j], j, ay, A[j]) for j in range(P)]
    else:
        L += ["v_mul_f32 %%[l%d], %s, %%[x%d]" % (j, ax, j) for j in range(P)]
        L += ["v_fma_f32 %%[l%d], %%[y%d], %s, %%[l%d]" % (j, j, ay, j) for j in range(P)]
        L += ["v_add_f32 %s, %s, %%[l%d]" % (A[s * P + j], bias[s], j)
              for s in range(S) for j in range(P)]
    # the row is read: load the next record's
    L += [".Lni_%=:",
          "s_load_dwordx4 s[%d:%d], s[%d:%d], 0x10" % (ROW, ROW + 3, BP, BP + 1),
          "s_add_u32 s%d, s%d, 16" % (BP, BP),
          "s_addc_u32 s%d, s%d, 0" % (BP + 1, BP + 1)]
    # 2. edges: jump to block 11 - n; block i handles record position 10 - i
    L += ["s_bfe_u32 %%[t], %s, 0x40010" % meta,
          "s_min_u32 %%[t], %%[t], %d" % MAX_EDGES,  # a 4-bit count above 11 is clamped
          "s_mul_i32 %[t], %[t], (.Le1_%= - .Le0_%=)",
          "s_sub_u32 %[t], (.Lee_%= - .Lep_%=), %[t]",
          "s_set_gpr_idx_on %[t], gpr_idx(SRC0)",
          "s_getpc_b64 %s" % pc,
          ".Lep_%=:",
          "s_add_u32 s%d, s%d, %%[t]" % (PC, PC),
          "s_addc_u32 s%d, s%d, 0" % (PC + 1, PC + 1),
          "s_setpc_b64 %s" % pc]
    for i in range(MAX_EDGES):
        p = MAX_EDGES - 1 - i
        L.append(".Le%d_%%=:" % i)
        L.append("s_bfe_u32 %%[t], %s, %s" % (sw[p // 6], bfe_imm(SLOT_BITS * (p % 6), log2(W))))
        L.append("s_set_gpr_idx_idx %[t]")
        L += ["v_fma_f32 %s, %s, %s, %s" % (A[m], T[m], wt[p], A[m]) for m in range(M)]
    L += [".Lee_%=:", "s_set_gpr_idx_off"]
    # 3. tail: a computed jump to tail meta & 15 (tails 13..15 do not exist and go to the loop
    # end, like a continuation record); the tails sit at a fixed stride. The record is read once
    # the tail index and the destination slot are taken, so the next record is loaded while the
    # activation runs.
    stride = tail_stride(M)
    L += ["s_and_b32 %%[t], %s, 15" % meta,
          "s_min_u32 %[t], %[t], 13",
          "s_lshl_b32 %%[t], %%[t], %d" % (stride.bit_length() - 1),
          "s_add_u32 %[t], %[t], (.Lt0_%= - .Ltp_%=)",
          "s_bfe_u32 %%[u], %s, %s" % (meta, bfe_imm(8, log2(W))),
          "s_load_dwordx16 s[%d:%d], s[%d:%d], 0x0" % (REC, REC + 15, RP, RP + 1),
          "s_getpc_b64 %s" % pc,
          ".Ltp_%=:",
          "s_add_u32 s%d, s%d, %%[t]" % (PC, PC),
          "s_addc_u32 s%d, s%d, 0" % (PC + 1, PC + 1),
          "s_setpc_b64 %s" % pc]
    # the end of every tail: the next record, or out of the loop
    loop_end = ["s_sub_u32 %[n], %[n], 1",
                "s_cmp_lg_u32 %[n], 0",
                "s_cbranch_scc1 .Lrec_%=",
                "s_branch .Ldone_%="]

    # The activations. pre: in-place steps on the accumulator; final: the last instruction, which
    # writes the destination slot (store tails, DST indexing) or the accumulator (output tails).
    def block(label, pre, final, store):
        out = [".L%s_%%=:" % label]
        for step in pre:
            out += [step.format(a=A[m]) for m in range(M)]
        if store:
            out.append("s_set_gpr_idx_on %[u], gpr_idx(DST)")
            out += [final.format(a=A[m], d=T[m]) for m in range(M)]
            out.append("s_set_gpr_idx_off")
        else:
            out += [final.format(a=A[m], d=A[m]) for m in range(M) if final]
            out.append("s_nop 1")  # the caller reads these next
        return out + loop_end

    # The packer scales every weight and bias feeding a varying node by its activation's input
    # scale (emr_internal.h), so the accumulator holds z' = c z and the tails are short:
    #   sigmoid  c = -log2 e:     1 / (1 + 2^z')
    #   tanh     c = -2 log2 e:   2 / (1 + 2^z') - 1
    #   gaussian c = sqrt(log2 e): 2^-(z'^2)
    #   sine     c = 1 / (2 pi):  v_sin_f32 (the sine of 2 pi times its input) of fract(z'), which
    #                             is exact and in [0, 1)
    defs = {
        "lin": ([], "v_mov_b32 {d}, {a}"),
        "abs": ([], "v_and_b32 {d}, 0x7fffffff, {a}"),
        "sig": (["v_exp_f32 {a}, {a}", "v_add_f32 {a}, 1.0, {a}"], "v_rcp_f32 {d}, {a}"),
        "tanh": (["v_exp_f32 {a}, {a}", "v_add_f32 {a}, 1.0, {a}", "v_rcp_f32 {a}, {a}"],
                 "v_fma_f32 {d}, {a}, 2.0, -1.0"),
        "gau": (["v_mul_f32_e64 {a}, {a}, -{a}"], "v_exp_f32 {d}, {a}"),
        "sin": (["v_fract_f32 {a}, {a}"], "v_sin_f32 {d}, {a}"),
    }
    # tails in index order: 0 continuation; 1..6 activation then store to the destination slot;
    # 7..12 the output node's activation, applied to the accumulators in place; 13 the rest.
    # Each is padded to the stride with never-executed words (s_nop encodings), so tail k starts
    # at .Lt0 + k * stride; the assembler refuses a tail longer than the stride.
    tails = [[".Lx_%=:"] + loop_end]
    for store in (True, False):
        for name in ACTS:  # activation ids 0..5
            pre, final = defs[name]
            if not store and name == "lin":
                tails.append([".Llino_%=:"] + loop_end)
                continue
            tails.append(block(name + ("" if store else "o"), pre, final, store))
    tails.append([".Linv_%=:"] + loop_end)
    assert len(tails) == 14
    for k, body in enumerate(tails):
        assert 8 * sum(1 for l in body if not l.startswith(".")) <= stride, (M, k)
        if k == 0:
            L.append(".Lt0_%=:")
        L += [".Ltb%d_%%=:" % k] + body + [".Lte%d_%%=:" % k,
              ".if .Lte%d_%%= - .Ltb%d_%%= > %d" % (k, k, stride),
              '.error \\"tail longer than its stride\\"',
              ".endif",
              ".fill (%d - (.Lte%d_%%= - .Ltb%d_%%=)) / 4, 4, 0xbf800000" % (stride, k, k)]
    # the last prefetch (one record and one row past the program, inside the tables) is drained
    # before the statement ends: its registers are the compiler's again after it
    L += [".Ldone_%=:", "s_waitcnt lgkmcnt(0)"]

    outs = ['[t] "=&s"(t)', '[u] "=&s"(u)', '[n] "+s"(n)',
            '"+{s[%d:%d]}"(rp)' % (RP, RP + 1), '"+{s[%d:%d]}"(bp)' % (BP, BP + 1)]
    if S == 1:
        outs.append('[tb] "=&v"(tb)')
    else:
        outs += ['[l%d] "=&v"(l[%d])' % (j, j) for j in range(P)]
    outs += ['"+{%s}"(acc[%d])' % (A[m], m) for m in range(M)]
    outs += ['"+{v[%d:%d]}"(v%d)' % (base(M, m, W), base(M, m, W) + W - 1, m) for m in range(M)]
    ins = ['[x%d] "v"(x[%d]), [y%d] "v"(y[%d])' % (j, j, j, j) for j in range(P)]
    clob = ['"scc"', '"m0"'] + ['"s%d"' % r for r in range(REC, ROW + 4)] + \
        ['"s%d"' % PC, '"s%d"' % (PC + 1)]

    body = "\n".join('        "%s\\n"' % l for l in L)
    vec = "f32x%d" % W
    out = []
    out.append("template <> struct Walker<%d, %d, %d> {" % (S, P, W))
    out.append("  static constexpr int M = %d;" % M)
    out.append("  float acc[%d];" % M)
    out.append("  %s %s;" % (vec, ", ".join("v%d" % m for m in range(M))))
    # def(): an empty statement that "defines" the accumulators and windows in their registers.
    # Placed before each walk, it tells the compiler that nothing from a previous walk is live in
    # them (a walk writes every value before reading it), so they cost no initialization and the
    # registers are free for other values between walks.
    defs_ = ['"={%s}"(acc[%d])' % (A[m], m) for m in range(M)]
    defs_ += ['"={v[%d:%d]}"(v%d)' % (base(M, m, W), base(M, m, W) + W - 1, m) for m in range(M)]
    out.append("  __device__ __forceinline__ void def() {")
    out.append('    asm volatile(""')
    out.append("                 : %s);" % ",\n                   ".join(defs_))
    out.append("  }")
    out.append("  // The whole program walk at the P positions (x, y): n records from rec (16 words each);")
    out.append("  // row: the group's bias rows (4 floats each), row 0 holding the outputs of a program")
    out.append("  // without records (n = 0) and row 1 + r the biases of record r.")
    out.append("  __device__ __forceinline__ void walk(uint64_t rec, uint64_t row, uint32_t n, "
               "const float* x, const float* y) {")
    out.append("    uint64_t rp = rec, bp = row;")
    out.append("    uint32_t t, u;")
    out.append("    float tb;" if S == 1 else "    float l[%d];" % P)
    out.append("    asm volatile(")
    out.append(body)
    out.append("        : %s" % ",\n          ".join(outs))
    out.append("        : %s" % ",\n          ".join(ins))
    # SCC is written by the scalar arithmetic, M0 by the indexing instructions; the record, row
    # and PC registers are the statement's own
    out.append("        : %s);" % ", ".join(clob))
    out.append("  }")
    out.append("};")
    return "\n".join(out) + "\n"


# The compiled tier's call convention (restated in emr_internal.h for the host code generator):
# accumulators and value windows where the walker keeps them, the positions right after the
# windows (x at XY .. XY + P - 1, y at XY + P ..), then the generated code's bias copies (one per
# source where they fit below JIT_TOP; for S > 1 the partial sums use accumulators); s[40:55] the
# group's first bias rows (loaded by the caller per chunk, in and out), s[56:57] the group's bias
# row base, s[58:59] the return address.
JIT_ROW, JIT_BP, JIT_RET = 40, 56, 58
JIT_TOP = 148


def jit_temps(S, P, W):
    M = S * P
    return 1 if S == 1 else (S if base(M, M, W) + 2 * P + S <= JIT_TOP else 0)


def gen_jitcall(S, P, W):
    M = S * P
    xy = base(M, M, W)
    tmp0 = xy + 2 * P
    TPW = P // 4
    # the next walk's tile geometry rows (TPW consecutive rows of 4 words) are loaded first, with
    # one load, so they arrive while the program runs; the wait after the return point makes them
    # safe to read (long done by then)
    # s_swappc_b64 jumps to the program and leaves the address of the next instruction (where the
    # program returns to) in s[JIT_RET:JIT_RET+1]
    L = ["s_load_dwordx%d %%[geo], %%[ga], 0x0" % (4 * TPW),
         "s_swappc_b64 s[%d:%d], %%[tgt]" % (JIT_RET, JIT_RET + 1),
         "s_waitcnt lgkmcnt(0)"]
    outs = ['"={v%d}"(acc[%d])' % (ACC + m, m) for m in range(M)]
    outs += ['"=&{v[%d:%d]}"(w%d)' % (base(M, m, W), base(M, m, W) + W - 1, m) for m in range(M)]
    outs += ['"=&{v%d}"(t[%d])' % (tmp0 + k, k) for k in range(jit_temps(S, P, W))]
    outs += ['"+{s[%d:%d]}"(rows)' % (JIT_ROW, JIT_ROW + 15)]
    outs += ['[geo] "=&s"(geo)']
    ins = ['[tgt] "s"(target)', '"{s[%d:%d]}"(bp)' % (JIT_BP, JIT_BP + 1), '[ga] "s"(geo_addr)']
    # position 4 k + c: x depends on c & 1, y on c >> 1; each distinct value is passed once
    ins += ['"{v%d}"(x[%d])' % (xy + j, j) for j in range(P) if j % 4 in (0, 1)]
    ins += ['"{v%d}"(y[%d])' % (xy + P + j, j) for j in range(P) if j % 4 in (0, 2)]
    clob = ['"scc"', '"s%d"' % JIT_RET, '"s%d"' % (JIT_RET + 1)]
    body = "\n".join('        "%s\\n"' % l for l in L)
    out = []
    out.append("template <> struct JitCall<%d, %d, %d> {" % (S, P, W))
    out.append("  typedef uint32_t Geo __attribute__((ext_vector_type(%d)));" % (4 * TPW))
    out.append("  float acc[%d];" % M)
    out.append("  // Runs the compiled program at `target` for the P positions (x, y); bp: the group's bias rows,")
    out.append("  // rows: its rows 1 .. 4 (in and out, see the register convention); geo: the %d words at" % (4 * TPW))
    out.append("  // geo_addr.")
    out.append("  __device__ __forceinline__ void call(uint64_t target, uint64_t bp, const float* x, "
               "const float* y, u32x16& rows, uint64_t geo_addr, Geo& geo) {")
    out.append("    f32x%d %s;" % (W, ", ".join("w%d" % m for m in range(M))))
    if jit_temps(S, P, W):
        out.append("    float t[%d];" % jit_temps(S, P, W))
    out.append("    asm volatile(")
    out.append(body)
    out.append("        : %s" % ",\n          ".join(outs))
    out.append("        : %s" % ",\n          ".join(ins))
    out.append("        : %s);" % ", ".join(clob))
    out.append("  }")
    out.append("};")
    return "\n".join(out) + "\n"


def main():
    print("// Generated by gen_regwin.py (the program-record step of the discover kernel, and the")
    print("// call into a compiled program). Do not edit; regenerate with:")
    print("// python gen_regwin.py > regwin_gen.h")
    print("#pragma once")
    print()
    print("template <int S, int P, int W> struct Walker;")
    print("template <int S, int P, int W> struct JitCall;")
    print()
    for S, P, W in VARIANTS:
        print(gen_walker(S, P, W))
    for S, P, W in VARIANTS:
        print(gen_jitcall(S, P, W))


if __name__ == "__main__":
    main()
