// Prints the binary16 sin/cos table of cp_f16_table.h (host build), one
// hex entry per line, then the divisor reciprocals, then the reciprocals
// keyed by the cosine, for tests/test_f16_table.py.
#include <cstdio>
#include <cstring>

#include "cp_f16_table.h"

int main() {
  static constexpr cp::f16tab::Table t = cp::f16tab::make_table();
  for (uint32_t b = 0; b < cp::f16tab::kEntries; ++b) std::printf("%08x\n", t.v[b]);
  // then the divisor reciprocals, as binary32 bit patterns
  static constexpr cp::f16tab::RecipTable r = cp::f16tab::make_recip_table();
  for (uint32_t k = 0; k < cp::f16tab::kDenEntries; ++k) {
    uint32_t u;
    std::memcpy(&u, &r.v[k], sizeof u);
    std::printf("%08x\n", u);
  }
  static_assert(cp::f16tab::cosines_in_range(cp::f16tab::make_table()), "cosines outside the keyed range");
  static constexpr cp::f16tab::RecipByCos rc = cp::f16tab::make_recip_by_cos_table();
  for (uint32_t k = 0; k < cp::f16tab::kCosEntries; ++k) {
    uint32_t u;
    std::memcpy(&u, &rc.v[k], sizeof u);
    std::printf("%08x\n", u);
  }
  return 0;
}
