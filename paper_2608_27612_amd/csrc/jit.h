// The compiled tier's host side (no HIP): the code generator that turns one packed varying
// program into gfx950 machine code for the register convention in emr_internal.h, and the
// resizing of the template code object's code area. Loading the result is the runtime's job.
#pragma once
#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "emr_internal.h"

namespace emr {
namespace jit {

// One compiled program: its machine words and, when asked for, an assembly listing (one
// instruction per line, in the syntax of the AMDGPU assembler), for the tests.
struct Code {
  std::vector<uint32_t> words;
  std::string listing;
};

// Compiles the varying program of one (genome, direction) for S sources at P positions per lane
// with register window W: rec points at its n_rec records (16 words each, layout in
// emr_internal.h), output_varies is bit 0 of its ProgDesc flags. The code computes exactly what
// the interpreter's record step computes, instruction for instruction, with the slot indexing
// resolved at compile time and the weights as literal operands, then returns through
// s[kJitRet:kJitRet+1]. Returns false, with *msg, for a variant the kernels do not have or a
// record that the interpreter would reject.
bool compile_program(const uint32_t* rec, uint32_t n_rec, bool output_varies, int S, int P, int W,
                     bool want_listing, Code* out, std::string* msg);

// Where the code area of a template code object lies.
struct AreaInfo {
  size_t file_off = 0;  // file offset of the area's first byte
  uint64_t vaddr = 0;   // its address in the object
  size_t bytes = 0;     // its size in the template
};

// Finds the code area (the local symbol emr_code_area, `area_bytes` long, inside .text) of the
// template object img[0..n) and checks that the object has the layout the resizing assumes.
bool find_area(const uint8_t* img, size_t n, size_t area_bytes, AreaInfo* info, std::string* msg);

// A copy of the template with its code area grown to new_bytes (the template's size plus a
// multiple of 4 KiB): the new bytes are inserted at the area's end and filled with s_endpgm, and
// every file offset, address, size and symbol after them is moved to match.
bool grow_area(const uint8_t* img, size_t n, const AreaInfo& info, size_t new_bytes,
               std::vector<uint8_t>* out, std::string* msg);

}  // namespace jit
}  // namespace emr
