// twiddles.hpp -- host generation of the twiddle table described in plan.hpp.
#pragma once

#include <vector>

namespace rdfft {

struct HostC32 {
  float x, y;
};

// exp(-2 pi i j / M), evaluated in double precision after exact integer reduction of
// j mod M to the first octant, then rounded once to float.
HostC32 unit_root(long long j, long long M);

// The whole table (kTableEntries entries) in the layout of plan.hpp.
std::vector<HostC32> build_twiddle_table();

}  // namespace rdfft
