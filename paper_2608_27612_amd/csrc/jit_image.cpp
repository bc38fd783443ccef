// The template code object of the compiled tier (built from jit.hip before this library), embedded
// in the library's read-only data. The build passes its path as EMR_JIT_TEMPLATE.
#include <stdint.h>

#if !defined(__HIP_DEVICE_COMPILE__)
__asm__(
    ".pushsection .rodata\n"
    ".p2align 12\n"
    ".globl emr_jit_template_begin\n"
    ".hidden emr_jit_template_begin\n"
    "emr_jit_template_begin:\n"
    ".incbin \"" EMR_JIT_TEMPLATE "\"\n"
    ".globl emr_jit_template_end\n"
    ".hidden emr_jit_template_end\n"
    "emr_jit_template_end:\n"
    ".popsection\n");
#endif
