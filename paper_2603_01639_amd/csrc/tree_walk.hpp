// Root-path walk over a parent array, shared by kernels that list a tree
// node's ancestors one by one.  It is constexpr, which makes it callable from
// device code and from plain host C++ alike (the host build is how its bounds
// are tested without a GPU).
#pragma once

#include <stdint.h>

namespace ltd {

// Writes node i, its parent, ..., the root (node 0) to path[0 .. len) and
// returns len.  Each link is clamped into [0, j - 1] before it is followed, so
// the walk strictly descends and stops at the root after at most i + 1
// entries whatever the array holds: a well-formed tree (parents[0] = -1,
// 0 <= parents[j] < j) gives its root path, and a malformed one gives some
// descending path, never a runaway loop or an entry past path[i].
constexpr int root_path(const int32_t* par, int i, int* path) {
  int len = 0;
  int j = i;
  while (true) {
    path[len++] = j;
    if (j <= 0) break;
    const int p = par[j];
    j = p < 0 ? 0 : (p > j - 1 ? j - 1 : p);
  }
  return len;
}

}  // namespace ltd
