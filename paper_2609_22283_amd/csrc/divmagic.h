// Division by a runtime constant through a host-computed magic pair, for
// indices the kernels split per element (tokens into node, frame, row).
#pragma once

#include <cstdint>

namespace sc {

// n / d for n < 2^31: (mulhi(n, mul) + n) >> shift.
struct DivMagic {
  uint32_t mul;
  uint32_t shift;
  uint32_t div;
};

// The magic pair of a divisor d >= 1: shift l = ceil(log2 d), mul =
// floor(2^32 (2^l - d) / d) + 1.
inline DivMagic magic_div(uint32_t d) {
  uint32_t l = 0;
  while ((1ull << l) < d) ++l;
  const uint64_t m = ((1ull << 32) * ((1ull << l) - d)) / d + 1;
  return DivMagic{(uint32_t)m, l, d};
}

}  // namespace sc
