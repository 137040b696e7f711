// Size limits of the bf16 GEMM fast path, host-side only (plain C++).
//
// Its operand loads go through 32-bit buffer descriptors whose record size
// is the operand's byte count, and an out-of-range load is sent to byte
// offset 0xFFFFFFF0, which must lie past that size to read zeros; its row
// bases are 32-bit ints.  So every operand it reads -- the caller's tensors
// and the zero-padded or packed copies made for narrow channel counts --
// must have fewer elements than (0xFFFFFFF0 / 2) - 8.  A contraction whose
// operands do not fit takes the general kernel (64-bit offsets) instead.
#pragma once

#include <stdint.h>

namespace ms {
namespace g2 {

constexpr uint32_t kOOB = 0xFFFFFFF0u;   // byte offset beyond any buffer: loads return 0

constexpr bool operand_fits(int64_t elems) {
    return elems >= 0 && elems <= (int64_t)(kOOB / 2) - 8;
}

}  // namespace g2
}  // namespace ms
