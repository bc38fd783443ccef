// The stable key sort of network assembly: the raw edges by their destination's kept node number
// (LSD radix sort, which keeps equal keys in their input order), from rocPRIM. Its own source
// file: the library's own kernels are checked for register and scratch use that a library's
// generic kernels need not follow.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <rocprim/device/device_radix_sort.hpp>

// Sorts n (key, value) pairs on key bits [0, bits) into kout / vout, stably. With tmp == NULL,
// *bytes receives the temporary storage the sort needs and nothing runs.
extern "C" hipError_t emr_net_sort(void* tmp, size_t* bytes, const uint32_t* kin, uint32_t* kout,
                                   const uint32_t* vin, uint32_t* vout, uint32_t n, int bits,
                                   hipStream_t s) {
  if (!bytes || bits < 1 || bits > 32) return hipErrorInvalidValue;
  return rocprim::radix_sort_pairs(tmp, *bytes, kin, kout, vin, vout, n, 0u, (unsigned)bits, s);
}
