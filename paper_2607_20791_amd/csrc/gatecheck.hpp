// Compatibility of a probe with one refusal-prefix table entry (Section 3,
// token-level reading): the probe so far q[0..j) followed by token t agrees
// with the entry on their common length; entries shorter than the minimum
// match length and entries owned by another prompt never match.
#pragma once
#include "kernels.hpp"

namespace rgd {
namespace {

RGD_DEV bool entry_matches(const GateArgs& a, int e, int b, const int* q, int j, int t) {
  if (a.owner && a.owner[e] != -1 && a.owner[e] != b) return false;
  const int o0 = a.offsets[e], len = a.offsets[e + 1] - o0;
  if (len < a.min_match) return false;
  const int n = min(len, j + 1);
  for (int i = 0; i < n; ++i)
    if (a.tokens[o0 + i] != (i < j ? q[i] : t)) return false;
  return true;
}

}  // namespace
}  // namespace rgd
