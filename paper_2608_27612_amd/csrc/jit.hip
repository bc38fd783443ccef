// The template code object of the compiled tier. Its kernels run the same discover body as the
// interpreting kernel, but each group's varying program is machine code written at run time into
// the code area at the end of this object's .text (see jit.cpp): a walk calls the group's program
// at the area's address plus the group's code offset, and the program returns to the caller
// through the return address it is handed. The host copies this object, resizes the area to the
// population's code, writes the programs into it and loads the copy as a module.
#include "discover.h"

namespace emr {
// Address of the code area: the PC-relative offset of its label, resolved when this object is
// linked (the same relocation pair the compiler uses for calls).
__device__ __forceinline__ uint64_t code_area_base() {
  uint64_t b;
  asm volatile(
      "s_getpc_b64 s[76:77]\n"
      "s_add_u32 s76, s76, emr_code_area@rel32@lo+4\n"
      "s_addc_u32 s77, s77, emr_code_area@rel32@hi+12\n"
      "s_mov_b64 %0, s[76:77]\n"
      : "=s"(b)
      :
      : "s76", "s77", "scc");
  return b;
}
}  // namespace emr

#define EMR_JIT_PARAMS                                                                          \
  const uint32_t *__restrict__ geo, const uint32_t *__restrict__ blob,                          \
      const emr::Group *__restrict__ groups,                                                    \
      const float *__restrict__ bias_tab, uint64_t *__restrict__ status,                        \
      uint32_t *__restrict__ err, float *__restrict__ raw, emr::DiscoverScalars a

// One kernel per output mode (raw outputs, records to the pool).
extern "C" __global__ void __launch_bounds__(emr::kDiscoverThreads) emr_discover_jit_raw(EMR_JIT_PARAMS) {
  emr::discover_body<emr::kModeRaw, true>(geo, blob, groups, bias_tab, status, err, raw, a,
                                          emr::code_area_base());
}
extern "C" __global__ void __launch_bounds__(emr::kDiscoverThreads) emr_discover_jit_records(EMR_JIT_PARAMS) {
  emr::discover_body<emr::kModeRecords, true>(geo, blob, groups, bias_tab, status, err, raw, a,
                                              emr::code_area_base());
}

// The code area: a never-launched function whose body ends .text. It is filled with s_endpgm,
// and the host grows it to the population's code and keeps at least kJitTailPad bytes of
// s_endpgm after the last program (instruction prefetch reads a little past a program's end).
// This function must stay the last one in this file.
extern "C" __global__ void emr_code_area_holder() {
  asm volatile(
      "s_endpgm\n"
      ".p2align 8\n"
      "emr_code_area:\n"
      ".fill 1024, 4, 0xbf810000\n");
}
