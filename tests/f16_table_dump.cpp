// Prints the binary16 sin/cos table of cp_f16_table.h (host build), one
// hex entry per line, for tests/test_f16_table.py.
#include <cstdio>

#include "cp_f16_table.h"

int main() {
  static constexpr cp::f16tab::Table t = cp::f16tab::make_table();
  for (uint32_t b = 0; b < cp::f16tab::kEntries; ++b) std::printf("%08x\n", t.v[b]);
  return 0;
}
