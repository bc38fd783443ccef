// The compiled tier's host side: code generation and the resizing of the template code object.
//
// The code generator translates the records of one packed varying program (emr_internal.h) into
// the instructions the interpreter's record step executes for them (gen_regwin.py): for every
// record, in order,
//   - a node's first record: acc = bias + ax x + ay y (for S = 1 as fma(y, ay, fma(x, ax, bias)),
//     for S > 1 as bias_s + fma(y, ay, ax x)), the bias from the record's bias row;
//   - its edges, from record position n - 1 down to 0: acc_m = fma(w, window_m[slot], acc_m);
//   - its tail: the activation (the packer has scaled its input), stored into the destination
//     slot of every window, or applied in place for the output node.
// A node that takes the same value for every source (marked shared by the packer) is evaluated for
// the first source's instances only, with the operations every source's instances run in the
// interpreter, and the instances of the other sources read its value from the first source's
// registers.
// The slot indices are resolved here, so every vector instruction names fixed registers, and the
// weights are literal operands: no register indexing, no scalar work per edge, and vector
// operands only (which lets the hardware issue the instructions at its higher rate). The result
// is the interpreter's arithmetic, bit for bit.
#include "jit.h"

#include <elf.h>

#include "../../include/emr.h"

#include <cstdio>
#include <cstring>

namespace emr {
namespace jit {
namespace {

// ---------------------------------------------------------------- instruction encoding (gfx950)
// VOP2: op[30:25] vdst[24:17] vsrc1[16:9] src0[8:0]; VOP1: 0x3f[31:25] vdst[24:17] op[16:9]
// src0[8:0]; VOP3: 0x34[31:26] op[25:16] vdst[7:0] | neg[31:29] src2[26:18] src1[17:9] src0[8:0];
// SMEM: 0x30[31:26] op[25:18] imm[17] sdata[12:6] sbase/2[5:0] | offset.
constexpr uint32_t kOpV2Add = 0x01, kOpV2Mul = 0x05, kOpV2And = 0x13, kOpV2Fmamk = 0x17,
                   kOpV2Fmac = 0x3b;
constexpr uint32_t kOpV1Mov = 0x01, kOpV1Fract = 0x1b, kOpV1Exp = 0x20, kOpV1Rcp = 0x22,
                   kOpV1Sin = 0x29;
constexpr uint32_t kOpV3Fma = 0x1cb, kOpV3Mul = 0x105;
constexpr uint32_t kOpSmemX4 = 0x02;
constexpr uint32_t kSrcLiteral = 255;
constexpr uint32_t kWaitLgkm0 = 0xBF8CC07Fu, kNop = 0xBF800000u, kEndpgm = 0xBF810000u;
constexpr uint32_t kSetpc = 0xBE801D00u;

// The inline-constant operand code of a 32-bit pattern, or kSrcLiteral when it needs a literal.
uint32_t inline_code(uint32_t bits) {
  if (bits <= 64u) return 128u + bits;                    // integers 0..64
  if (bits >= 0xFFFFFFF0u) return 192u + (0u - bits);     // integers -1..-16
  switch (bits) {
    case 0x3f000000u: return 240;  //  0.5
    case 0xbf000000u: return 241;  // -0.5
    case 0x3f800000u: return 242;  //  1.0
    case 0xbf800000u: return 243;  // -1.0
    case 0x40000000u: return 244;  //  2.0
    case 0xc0000000u: return 245;  // -2.0
    case 0x40800000u: return 246;  //  4.0
    case 0xc0800000u: return 247;  // -4.0
    case 0x3e22f983u: return 248;  //  1 / (2 pi)
    default: return kSrcLiteral;
  }
}

std::string const_text(uint32_t bits) {
  const uint32_t c = inline_code(bits);
  char b[32];
  if (c >= 128 && c <= 192) {
    std::snprintf(b, sizeof b, "%u", c - 128);
  } else if (c >= 193 && c <= 208) {
    std::snprintf(b, sizeof b, "-%u", c - 192);
  } else {
    static const char* f[] = {"0.5", "-0.5", "1.0", "-1.0", "2.0", "-2.0", "4.0", "-4.0",
                              "0.15915494"};
    if (c >= 240 && c <= 248) return f[c - 240];
    std::snprintf(b, sizeof b, "0x%x", bits);
  }
  return b;
}

class Emitter {
 public:
  Emitter(bool listing, Code* out) : want_(listing), out_(out) {}

  // src0 operands: a VGPR, an SGPR, or a 32-bit constant (their text is made for listings only)
  struct Src {
    uint32_t code;  // 9-bit operand code
    uint32_t lit;   // the constant's bits (for a literal: the literal dword)
    int vgpr;       // the VGPR read, or -1
    int sgpr;       // the SGPR read, or -1
  };
  static Src V(int v) { return {256u + (uint32_t)v, 0, v, -1}; }
  static Src Sg(int s) { return {(uint32_t)s, 0, -1, s}; }
  static Src K(uint32_t bits) { return {inline_code(bits), bits, -1, -1}; }
  static std::string str(const Src& s) {
    if (s.vgpr >= 0) return "v" + std::to_string(s.vgpr);
    if (s.sgpr >= 0) return "s" + std::to_string(s.sgpr);
    return const_text(s.lit);
  }

  void vop2(uint32_t op, const char* name, int vdst, const Src& s0, int vsrc1, bool trans = false) {
    hazard(s0.vgpr, vsrc1, -1);
    put((op << 25) | ((uint32_t)vdst << 17) | ((uint32_t)vsrc1 << 9) | s0.code);
    if (s0.code == kSrcLiteral) put(s0.lit);
    if (want_) text("%s v%d, %s, v%d", name, vdst, str(s0).c_str(), vsrc1);
    wrote(vdst, trans);
  }
  // v_fmamk_f32 vdst, src0, K, vsrc1: vdst = src0 * K + vsrc1
  void fmamk(int vdst, int src0, uint32_t k, int vsrc1) {
    hazard(src0, vsrc1, -1);
    put((kOpV2Fmamk << 25) | ((uint32_t)vdst << 17) | ((uint32_t)vsrc1 << 9) | (256u + (uint32_t)src0));
    put(k);
    text("v_fmamk_f32 v%d, v%d, 0x%x, v%d", vdst, src0, k, vsrc1);
    wrote(vdst, false);
  }
  void vop1(uint32_t op, const char* name, int vdst, const Src& s0, bool trans) {
    hazard(s0.vgpr, -1, -1);
    put(0x7E000000u | ((uint32_t)vdst << 17) | (op << 9) | s0.code);
    if (s0.code == kSrcLiteral) put(s0.lit);
    if (want_) text("%s v%d, %s", name, vdst, str(s0).c_str());
    wrote(vdst, trans);
  }
  // VOP3 with VGPR src0 and inline-constant or VGPR src1 / src2; neg: the NEG field
  void vop3(uint32_t op, const char* name, int vdst, const Src& a, const Src& b, const Src* c,
            uint32_t neg) {
    hazard(a.vgpr, b.vgpr, c ? c->vgpr : -1);
    put(0xD0000000u | (op << 16) | (uint32_t)vdst);
    put((neg << 29) | ((c ? c->code : 0u) << 18) | (b.code << 9) | a.code);
    if (want_ && c)
      text("%s v%d, %s, %s, %s", name, vdst, str(a).c_str(), str(b).c_str(), str(*c).c_str());
    else if (want_)
      text("%s v%d, %s, %s%s", name, vdst, str(a).c_str(), (neg & 2u) ? "-" : "", str(b).c_str());
    wrote(vdst, false);
  }
  void load_x4(int sdata, int sbase, uint32_t offset) {
    put(0xC0000000u | (kOpSmemX4 << 18) | (1u << 17) | ((uint32_t)sdata << 6) | ((uint32_t)sbase >> 1));
    put(offset);
    text("s_load_dwordx4 s[%d:%d], s[%d:%d], 0x%x", sdata, sdata + 3, sbase, sbase + 1, offset);
    last_trans_ = -1;
  }
  void wait_lgkm0() {
    put(kWaitLgkm0);
    line("s_waitcnt lgkmcnt(0)");
    last_trans_ = -1;
  }
  void nop(int n) {
    put(kNop | (uint32_t)n);
    text("s_nop %d", n);
    last_trans_ = -1;
  }
  void setpc(int s) {
    put(kSetpc | (uint32_t)s);
    text("s_setpc_b64 s[%d:%d]", s, s + 1);
    last_trans_ = -1;
  }

 private:
  // A vector instruction that reads the result of the transcendental instruction right before
  // it needs one wait state.
  void hazard(int a, int b, int c) {
    if (last_trans_ >= 0 && (a == last_trans_ || b == last_trans_ || c == last_trans_)) nop(0);
  }
  void wrote(int v, bool trans) { last_trans_ = trans ? v : -1; }
  void put(uint32_t w) { out_->words.push_back(w); }
  void line(const char* s) {
    if (!want_) return;
    out_->listing += s;
    out_->listing += '\n';
  }
  template <typename... A>
  void text(const char* fmt, A... a) {
    if (!want_) return;
    char b[128];
    std::snprintf(b, sizeof b, fmt, a...);
    out_->listing += b;
    out_->listing += '\n';
  }
  bool want_;
  Code* out_;
  int last_trans_ = -1;
};

bool variant_ok(int S, int P, int W) {
  if (W != 4 && W != 8 && W != 16 && W != 32) return false;
  return S >= 1 && S <= max_group(W) && P == positions_per_lane(S, W);
}

}  // namespace

bool compile_program(const uint32_t* rec, uint32_t n_rec, bool output_varies, int S, int P, int W,
                     bool want_listing, Code* out, std::string* msg) {
  if (!variant_ok(S, P, W)) {
    *msg = "no kernel variant for S=" + std::to_string(S) + " P=" + std::to_string(P) +
           " W=" + std::to_string(W);
    return false;
  }
  if (n_rec > kMaxRecords) {
    *msg = "program of " + std::to_string(n_rec) + " records";
    return false;
  }
  out->words.clear();
  out->listing.clear();
  Emitter E(want_listing, out);
  typedef Emitter::Src Src;
  const int M = S * P;
  auto acc = [&](int m) { return kJitAcc + m; };
  auto win = [&](int m, uint32_t k) { return jit_window(M, W, m) + (int)k; };
  const int T = jit_x(M, W) + 2 * P;  // bias copies from T
  // position j's x and y (the convention holds each distinct value of a tile once)
  auto xr = [&](int j) { return jit_xr(M, W, j); };
  auto yr = [&](int j) { return jit_yr(M, W, P, j); };
  auto row = [](uint32_t r, int s) { return kJitRow + 4 * (int)(r % kJitRowBlock) + s; };
  const uint32_t n = output_varies ? n_rec : 0u;

  if (n == 0) {
    // a uniform output: every instance is its source's constant of row 0
    E.load_x4(kJitRow, kJitBp, 0);
    E.wait_lgkm0();
    for (int s = 0; s < S; ++s)
      for (int j = 0; j < P; ++j) E.vop1(kOpV1Mov, "v_mov_b32_e32", acc(s * P + j), Src(Emitter::Sg(kJitRow + s)), false);
    E.setpc(kJitRet);
    return true;
  }

  const uint32_t wmask = (uint32_t)W - 1u;
  // The caller has loaded the rows of records 0 .. kJitRowBlock - 1 (block 0). A program with a
  // node starting later loads those blocks over them, so it loads block 0 itself too: the next
  // walk finds the registers as this one left them.
  bool long_program = false;
  for (uint32_t r = kJitRowBlock; r < n; ++r) long_program |= (rec[16 * (size_t)r] & kRecFirst) != 0;
  int64_t loaded_block = long_program ? -1 : 0;
  const int copies = jit_temps(S, P, W);

  // A linear node that stores its value sums straight into its destination slot (the
  // interpreter sums in the accumulator and copies it there) when none of its own edges reads that
  // slot: the same operations in the same order on other registers. Marked at the node's first
  // record.
  std::vector<uint8_t> in_place(n, 0);
  std::vector<uint8_t> output_node(n, 0);  // at a node's first record: the node is the output
  {
    bool started = false;
    uint32_t first = 0, reads = 0;  // window slots the node's edges read (W <= 32)
    for (uint32_t r = 0; r < n; ++r) {
      const uint32_t meta = rec[16 * (size_t)r];
      if (meta & kRecFirst) {
        started = true;
        first = r;
        reads = 0;
      }
      uint32_t ne = (meta >> kRecEdgeShift) & 15u;
      if (ne > kRecEdges) ne = kRecEdges;
      for (uint32_t q = 0; q < ne; ++q) {
        const uint32_t sw = q < 6 ? rec[16 * (size_t)r + 3] : rec[16 * (size_t)r + 4];
        reads |= 1u << ((sw >> (kSlotBits * (q % 6))) & wmask);
      }
      uint32_t tail = meta & kRecTailMask;
      if (tail > 13) tail = 13;
      if (tail == 0 || tail == 13) continue;
      const uint32_t dst = (meta >> kRecDstShift) & wmask;
      if (started && tail == kRecTailStore + EMR_ACT_LINEAR && !((reads >> dst) & 1u))
        in_place[first] = 1;
      if (started && tail >= kRecTailOutput) output_node[first] = 1;
      started = false;
    }
  }
  bool inplace = false;
  uint32_t node_dst = 0;
  // A node marked shared (kRecShared, with S > 1) takes the same value for every source: it is
  // evaluated for the first source's P instances only, its inputs being shared values too. A
  // window slot that holds a shared value has only the first source's registers written; a read
  // of it by instance s P + j reads instance j's register instead (`shared_slot`, tracked along
  // the straight-line program: a node's store into a slot decides what the slot holds).
  bool shared = false;
  std::vector<uint8_t> shared_slot(W, 0);
  int MM = M;  // instances the current node evaluates
  auto A = [&](int m) { return inplace ? win(m, node_dst) : acc(m); };  // the node's sum
  auto rd = [&](int m, uint32_t k) { return win(shared_slot[k] ? m % P : m, k); };
  // A node without x or y terms starts from its bias: folded into its first edge (one v_fmamk
  // per instance, the fma the interpreter's move + v_fmac computes) when that edge is in the
  // node's first record and the bias is in a VGPR (a copy per source, or one for S = 1).
  bool fuse = false;
  int bias_base = 0, bias_step = 0;  // instance m's bias in v[bias_base + (m / P) * bias_step]
  for (uint32_t r = 0; r < n; ++r) {
    const uint32_t* R = rec + 16 * (size_t)r;
    const uint32_t meta = R[0];
    if (meta & kRecFirst) {
      inplace = in_place[r] != 0;
      node_dst = (meta >> kRecDstShift) & wmask;
      // (every source needs its own output: a shared mark on the output node is not followed)
      shared = S > 1 && (meta & kRecShared) != 0 && !output_node[r];
      MM = shared ? P : M;
      uint32_t ne0 = (meta >> kRecEdgeShift) & 15u;
      if (ne0 > kRecEdges) ne0 = kRecEdges;
      // The bias rows of the first records of this record's block of kJitRowBlock are loaded
      // together (the rows of the records the interpreter reads them for), and waited for once.
      bool wait = false;
      if ((int64_t)(r / kJitRowBlock) != loaded_block) {
        loaded_block = r / kJitRowBlock;
        const uint32_t b0 = kJitRowBlock * (r / kJitRowBlock);
        const uint32_t b1 = b0 + kJitRowBlock < n ? b0 + kJitRowBlock : n;
        for (uint32_t q = b0; q < b1; ++q)
          if (rec[16 * (size_t)q] & kRecFirst) E.load_x4(row(q, 0), kJitBp, 16u * (1u + q));
        wait = true;
      }
      // A zero x or y weight adds nothing: its term is left out. (Positions are never 0 (odd
      // multiples of 2^-level, minus 1), so every product kept is nonzero and the sums equal the
      // interpreter's, which adds the zero terms; only a node bias of -0.0 would come out +0.0
      // there.)
      const bool has_x = R[1] != 0u && R[1] != 0x80000000u, has_y = R[2] != 0u && R[2] != 0x80000000u;
      fuse = false;
      if (S == 1) {
        if (wait) E.wait_lgkm0();
        const int tb = T;
        if (!has_x && !has_y && ne0 > 0) {
          E.vop1(kOpV1Mov, "v_mov_b32_e32", tb, Emitter::Sg(row(r, 0)), false);
          fuse = true;
          bias_base = tb;
          bias_step = 0;
        } else if (!has_x && !has_y) {
          for (int j = 0; j < P; ++j)
            E.vop1(kOpV1Mov, "v_mov_b32_e32", A(j), Emitter::Sg(row(r, 0)), false);
        } else {
          E.vop1(kOpV1Mov, "v_mov_b32_e32", tb, Emitter::Sg(row(r, 0)), false);
          if (has_x)
            for (int j = 0; j < P; ++j) E.fmamk(A(j), xr(j), R[1], tb);
          else
            for (int j = 0; j < P; ++j) E.fmamk(A(j), yr(j), R[2], tb);
          if (has_x && has_y)
            for (int j = 0; j < P; ++j)
              E.vop2(kOpV2Fmac, "v_fmac_f32_e32", A(j), Emitter::K(R[2]), yr(j));
        }
      } else if (!has_x && !has_y && shared) {
        // one bias (a shared node's rows are equal for every source), in the last source's
        // first accumulator, which no value occupies at a node's start
        if (wait) E.wait_lgkm0();
        const int tb = acc((S - 1) * P);
        if (ne0 > 0) {
          E.vop1(kOpV1Mov, "v_mov_b32_e32", tb, Emitter::Sg(row(r, 0)), false);
          fuse = true;
          bias_base = tb;
          bias_step = 0;
        } else {
          for (int j = 0; j < P; ++j)
            E.vop1(kOpV1Mov, "v_mov_b32_e32", A(j), Emitter::Sg(row(r, 0)), false);
        }
      } else if (!has_x && !has_y) {
        if (wait) E.wait_lgkm0();
        if (copies == S) {
          for (int s = 0; s < S; ++s)
            E.vop1(kOpV1Mov, "v_mov_b32_e32", T + s, Emitter::Sg(row(r, s)), false);
          if (ne0 > 0) {
            fuse = true;
            bias_base = T;
            bias_step = 1;
          } else {
            for (int s = 0; s < S; ++s)
              for (int j = 0; j < P; ++j)
                E.vop1(kOpV1Mov, "v_mov_b32_e32", A(s * P + j), Emitter::V(T + s), false);
          }
        } else {
          for (int s = 0; s < S; ++s)
            for (int j = 0; j < P; ++j)
              E.vop1(kOpV1Mov, "v_mov_b32_e32", A(s * P + j), Emitter::Sg(row(r, s)), false);
        }
      } else {
        // the partial sums l_j live in the last source's accumulators (free at a node's start)
        // until every source has added its bias to them. With one position term, l_j has two
        // distinct values per tile, computed once each: position j reads l at ls(j) <= j.
        // (A shared node adds the first source's bias only: the same operations as every
        // source's in a walk of S sources.)
        const int L = acc((S - 1) * P);
        const int ns = shared ? 1 : S;
        auto ls = [&](int j) {
          return L + (has_x && has_y ? j : has_x ? (j & ~3) + (j & 1) : (j & ~3) + (j & 2));
        };
        for (int j = 0; j < P; ++j)
          if (ls(j) == L + j)
            E.vop2(kOpV2Mul, "v_mul_f32_e32", L + j, Emitter::K(has_x ? R[1] : R[2]),
                   has_x ? xr(j) : yr(j));
        if (has_x && has_y)
          for (int j = 0; j < P; ++j)
            E.vop2(kOpV2Fmac, "v_fmac_f32_e32", L + j, Emitter::K(R[2]), yr(j));
        if (wait) E.wait_lgkm0();
        if (copies == S)  // bias copies in VGPRs: the adds read vector operands only
          for (int s = 0; s < ns; ++s)
            E.vop1(kOpV1Mov, "v_mov_b32_e32", T + s, Emitter::Sg(row(r, s)), false);
        // (the last source's sums overwrite l, in decreasing j: l at ls(j) <= j is read first)
        for (int s = 0; s < ns; ++s)
          for (int jj = 0; jj < P; ++jj) {
            const int j = s == S - 1 ? P - 1 - jj : jj;
            const Src b = copies == S ? Emitter::V(T + s) : Emitter::Sg(row(r, s));
            E.vop2(kOpV2Add, "v_add_f32_e32", A(s * P + j), b, ls(j));
          }
      }
    }
    // edges, from record position n - 1 down to 0
    uint32_t ne = (meta >> kRecEdgeShift) & 15u;
    if (ne > kRecEdges) ne = kRecEdges;
    for (uint32_t q = ne; q-- > 0;) {
      const uint32_t sw = q < 6 ? R[3] : R[4];
      const uint32_t slot = (sw >> (kSlotBits * (q % 6))) & wmask;
      const Src w = Emitter::K(R[5 + q]);
      if (fuse) {
        for (int m = 0; m < MM; ++m)
          E.fmamk(A(m), rd(m, slot), R[5 + q], bias_base + (m / P) * bias_step);
        fuse = false;
      } else {
        for (int m = 0; m < MM; ++m) E.vop2(kOpV2Fmac, "v_fmac_f32_e32", A(m), w, rd(m, slot));
      }
    }
    // tail
    uint32_t tail = meta & kRecTailMask;
    if (tail > 13) tail = 13;
    if (tail == 0 || tail == 13) continue;
    const bool store = tail < kRecTailOutput;
    const uint32_t act = store ? tail - kRecTailStore : tail - kRecTailOutput;
    const uint32_t dst = (meta >> kRecDstShift) & wmask;
    auto D = [&](int m) { return store ? win(m, dst) : acc(m); };
    auto each = [&](auto f) {
      for (int m = 0; m < MM; ++m) f(m);
    };
    switch (act) {
      case EMR_ACT_LINEAR:
        if (store && !inplace)
          each([&](int m) { E.vop1(kOpV1Mov, "v_mov_b32_e32", D(m), Emitter::V(acc(m)), false); });
        break;
      case EMR_ACT_ABS:
        each([&](int m) { E.vop2(kOpV2And, "v_and_b32_e32", D(m), Emitter::K(0x7fffffffu), acc(m)); });
        break;
      case EMR_ACT_SIGMOID:  // 1 / (1 + 2^z')
        each([&](int m) { E.vop1(kOpV1Exp, "v_exp_f32_e32", acc(m), Emitter::V(acc(m)), true); });
        each([&](int m) { E.vop2(kOpV2Add, "v_add_f32_e32", acc(m), Emitter::K(0x3f800000u), acc(m)); });
        each([&](int m) { E.vop1(kOpV1Rcp, "v_rcp_f32_e32", D(m), Emitter::V(acc(m)), true); });
        break;
      case EMR_ACT_TANH: {  // 2 / (1 + 2^z') - 1
        each([&](int m) { E.vop1(kOpV1Exp, "v_exp_f32_e32", acc(m), Emitter::V(acc(m)), true); });
        each([&](int m) { E.vop2(kOpV2Add, "v_add_f32_e32", acc(m), Emitter::K(0x3f800000u), acc(m)); });
        each([&](int m) { E.vop1(kOpV1Rcp, "v_rcp_f32_e32", acc(m), Emitter::V(acc(m)), true); });
        const Src two = Emitter::K(0x40000000u), m1 = Emitter::K(0xbf800000u);
        each([&](int m) { E.vop3(kOpV3Fma, "v_fma_f32", D(m), Emitter::V(acc(m)), two, &m1, 0); });
        break;
      }
      case EMR_ACT_GAUSS:  // 2^-(z'^2)
        each([&](int m) {
          E.vop3(kOpV3Mul, "v_mul_f32_e64", acc(m), Emitter::V(acc(m)), Emitter::V(acc(m)), nullptr, 2u);
        });
        each([&](int m) { E.vop1(kOpV1Exp, "v_exp_f32_e32", D(m), Emitter::V(acc(m)), true); });
        break;
      case EMR_ACT_SINE:  // sin(2 pi fract(z'))
        each([&](int m) { E.vop1(kOpV1Fract, "v_fract_f32_e32", acc(m), Emitter::V(acc(m)), false); });
        each([&](int m) { E.vop1(kOpV1Sin, "v_sin_f32_e32", D(m), Emitter::V(acc(m)), true); });
        break;
      default:
        break;  // ids 6..: no activation exists; the interpreter's tail table has none either
    }
    if (store) shared_slot[dst] = shared ? 1 : 0;
  }
  // the caller reads the accumulators next (two wait states cover a transcendental result)
  E.nop(1);
  E.setpc(kJitRet);
  return true;
}

// ---------------------------------------------------------------- the template code object
namespace {
template <typename T>
bool at(const uint8_t* img, size_t n, size_t off, T* out) {
  if (off > n || n - off < sizeof(T)) return false;
  std::memcpy(out, img + off, sizeof(T));
  return true;
}
bool is_dyn_ptr(int64_t tag) {
  switch (tag) {
    case DT_PLTGOT: case DT_HASH: case DT_STRTAB: case DT_SYMTAB: case DT_RELA: case DT_INIT:
    case DT_FINI: case DT_REL: case DT_JMPREL: case DT_INIT_ARRAY: case DT_FINI_ARRAY:
    case DT_GNU_HASH: case DT_VERSYM: case DT_VERDEF: case DT_VERNEED:
      return true;
    default:
      return false;
  }
}
}  // namespace

bool find_area(const uint8_t* img, size_t n, size_t area_bytes, AreaInfo* info, std::string* msg) {
  Elf64_Ehdr eh;
  if (!at(img, n, 0, &eh) || std::memcmp(eh.e_ident, ELFMAG, SELFMAG) != 0 ||
      eh.e_ident[EI_CLASS] != ELFCLASS64 || eh.e_ident[EI_DATA] != ELFDATA2LSB ||
      eh.e_machine != 224 /* EM_AMDGPU */ || eh.e_shentsize != sizeof(Elf64_Shdr) ||
      eh.e_phentsize != sizeof(Elf64_Phdr)) {
    *msg = "template code object: not a 64-bit AMDGPU ELF";
    return false;
  }
  std::vector<Elf64_Shdr> sh(eh.e_shnum);
  for (size_t i = 0; i < sh.size(); ++i)
    if (!at(img, n, eh.e_shoff + i * sizeof(Elf64_Shdr), &sh[i])) {
      *msg = "template code object: truncated section table";
      return false;
    }
  bool found = false;
  for (const Elf64_Shdr& s : sh) {
    if ((s.sh_type == SHT_REL || s.sh_type == SHT_RELA) && s.sh_size > 0) {
      *msg = "template code object has relocations";
      return false;
    }
    if (s.sh_type != SHT_SYMTAB || s.sh_link >= sh.size() || s.sh_entsize != sizeof(Elf64_Sym))
      continue;
    const Elf64_Shdr& str = sh[s.sh_link];
    for (size_t k = 0; k < s.sh_size / sizeof(Elf64_Sym); ++k) {
      Elf64_Sym sym;
      if (!at(img, n, s.sh_offset + k * sizeof(Elf64_Sym), &sym)) break;
      if (sym.st_name >= str.sh_size || str.sh_offset + sym.st_name >= n) continue;
      const char* name = (const char*)img + str.sh_offset + sym.st_name;
      const size_t room = n - (str.sh_offset + sym.st_name);
      if (strnlen(name, room) == room || std::strcmp(name, "emr_code_area") != 0) continue;
      if (sym.st_shndx == SHN_UNDEF || sym.st_shndx >= sh.size()) break;
      const Elf64_Shdr& text = sh[sym.st_shndx];
      if (!(text.sh_flags & SHF_EXECINSTR) || sym.st_value < text.sh_addr ||
          sym.st_value + area_bytes > text.sh_addr + text.sh_size)
        break;
      info->vaddr = sym.st_value;
      info->file_off = text.sh_offset + (sym.st_value - text.sh_addr);
      info->bytes = area_bytes;
      found = info->file_off + area_bytes <= n;
      break;
    }
  }
  if (!found) {
    *msg = "template code object: no code area of the expected size";
    return false;
  }
  for (size_t k = 0; k < area_bytes; k += 4) {
    uint32_t w;
    std::memcpy(&w, img + info->file_off + k, 4);
    if (w != kEndpgm) {
      *msg = "template code object: the code area is not empty";
      return false;
    }
  }
  return true;
}

bool grow_area(const uint8_t* img, size_t n, const AreaInfo& info, size_t new_bytes,
               std::vector<uint8_t>* out, std::string* msg) {
  if (new_bytes < info.bytes || (new_bytes - info.bytes) % 4096 != 0) {
    *msg = "code area sizes differ by a multiple of 4 KiB";
    return false;
  }
  const size_t delta = new_bytes - info.bytes;
  const size_t F = info.file_off + info.bytes;  // insertion point (file)
  const uint64_t V = info.vaddr + info.bytes;   // and its address
  out->assign(img, img + F);
  for (size_t k = 0; k < delta; k += 4) {
    const uint8_t b[4] = {0x00, 0x00, 0x81, 0xbf};  // s_endpgm
    out->insert(out->end(), b, b + 4);
  }
  out->insert(out->end(), img + F, img + n);
  uint8_t* o = out->data();
  const size_t N = out->size();
  auto moved = [&](uint64_t off) { return off >= F ? off + delta : off; };
  Elf64_Ehdr eh;
  std::memcpy(&eh, o, sizeof eh);
  eh.e_phoff = moved(eh.e_phoff);
  eh.e_shoff = moved(eh.e_shoff);
  std::memcpy(o, &eh, sizeof eh);
  for (size_t i = 0; i < eh.e_phnum; ++i) {
    Elf64_Phdr ph;
    const size_t at_off = eh.e_phoff + i * sizeof ph;
    if (at_off + sizeof ph > N) {
      *msg = "truncated program headers";
      return false;
    }
    std::memcpy(&ph, o + at_off, sizeof ph);
    if (ph.p_filesz > 0 || ph.p_memsz > 0) {
      if (ph.p_offset >= F) {
        ph.p_offset += delta;
        if (ph.p_vaddr >= V) {
          ph.p_vaddr += delta;
          ph.p_paddr += delta;
        }
      } else if (F <= ph.p_offset + ph.p_filesz) {
        ph.p_filesz += delta;
        ph.p_memsz += delta;
      }
    }
    std::memcpy(o + at_off, &ph, sizeof ph);
  }
  std::vector<Elf64_Shdr> sh(eh.e_shnum);
  for (size_t i = 0; i < sh.size(); ++i) {
    const size_t at_off = eh.e_shoff + i * sizeof(Elf64_Shdr);
    if (at_off + sizeof(Elf64_Shdr) > N) {
      *msg = "truncated section headers";
      return false;
    }
    Elf64_Shdr& s = sh[i];
    std::memcpy(&s, o + at_off, sizeof s);
    if (s.sh_type != SHT_NULL) {
      if (s.sh_offset >= F) {
        s.sh_offset += delta;
        if ((s.sh_flags & SHF_ALLOC) && s.sh_addr >= V) s.sh_addr += delta;
      } else if (s.sh_type != SHT_NOBITS && F <= s.sh_offset + s.sh_size) {
        s.sh_size += delta;
      }
    }
    std::memcpy(o + at_off, &s, sizeof s);
  }
  for (const Elf64_Shdr& s : sh) {
    if ((s.sh_type == SHT_SYMTAB || s.sh_type == SHT_DYNSYM) && s.sh_entsize == sizeof(Elf64_Sym)) {
      for (size_t k = 0; k < s.sh_size / sizeof(Elf64_Sym); ++k) {
        const size_t off = s.sh_offset + k * sizeof(Elf64_Sym);
        if (off + sizeof(Elf64_Sym) > N) break;
        Elf64_Sym sym;
        std::memcpy(&sym, o + off, sizeof sym);
        if (sym.st_shndx != SHN_UNDEF && sym.st_shndx < SHN_LORESERVE && sym.st_shndx < sh.size() &&
            (sh[sym.st_shndx].sh_flags & SHF_ALLOC)) {
          if (sym.st_value >= V)
            sym.st_value += delta;
          else if (sym.st_value + sym.st_size > V)
            sym.st_size += delta;  // a function that holds the area
        }
        std::memcpy(o + off, &sym, sizeof sym);
      }
    }
    if (s.sh_type == SHT_DYNAMIC) {
      for (size_t k = 0; k < s.sh_size / sizeof(Elf64_Dyn); ++k) {
        const size_t off = s.sh_offset + k * sizeof(Elf64_Dyn);
        if (off + sizeof(Elf64_Dyn) > N) break;
        Elf64_Dyn d;
        std::memcpy(&d, o + off, sizeof d);
        if (is_dyn_ptr(d.d_tag) && d.d_un.d_ptr >= V) d.d_un.d_ptr += delta;
        std::memcpy(o + off, &d, sizeof d);
      }
    }
  }
  return true;
}

}  // namespace jit
}  // namespace emr
