// Candidate layouts and the view predicate (see layouts.h).
#include "layouts.h"

#include <algorithm>
#include <set>

#include "graph.h"

namespace fluid {

namespace {

std::vector<int> physical_key(const Shape& shape, const Perm& p) {
  std::vector<int> k;
  for (int d : p)
    if (shape[d] != 1) k.push_back(d);
  return k;
}

// Physical dim sequence `seq` of a tensor whose dims (a, a+1) are the outer
// and inner halves of one coarser dim: drop extent-1 dims, require a to be
// immediately followed by a+1 when both remain, merge them and renumber.
bool collapse(const Perm& seq, const Shape& shape, int a, std::vector<int>* out) {
  std::vector<int> s;
  for (int d : seq)
    if (shape[d] != 1) s.push_back(d);
  const bool both = shape[a] != 1 && shape[a + 1] != 1;
  out->clear();
  for (size_t i = 0; i < s.size();) {
    int d = s[i];
    if (d == a || d == a + 1) {
      if (both) {
        if (d != a || i + 1 >= s.size() || s[i + 1] != a + 1) return false;
        i += 2;
      } else {
        i += 1;
      }
      out->push_back(a);
      continue;
    }
    out->push_back(d < a ? d : d - 1);
    ++i;
  }
  return true;
}

}  // namespace

Perm identity_perm(int rank) {
  Perm p(rank);
  for (int i = 0; i < rank; ++i) p[i] = i;
  return p;
}

std::vector<Perm> layout_list(const Shape& shape) {
  Perm p = identity_perm((int)shape.size());
  std::set<std::vector<int>> seen;
  std::vector<Perm> out;
  do {
    if (seen.insert(physical_key(shape, p)).second) out.push_back(p);
  } while (std::next_permutation(p.begin(), p.end()));
  return out;
}

std::vector<Perm> measured_layout_list(const Shape& shape) {
  std::vector<Perm> all = layout_list(shape);
  if (all.size() <= 6) return all;
  const int r = (int)shape.size();
  std::vector<Perm> out;
  for (const Perm& p : all)
    if (p.back() >= r - 2) out.push_back(p);
  return out;
}

std::vector<int64_t> dense_strides(const Shape& shape, const Perm& perm) {
  std::vector<int64_t> st(shape.size(), 0);
  int64_t acc = 1;
  for (int i = (int)perm.size() - 1; i >= 0; --i) {
    st[perm[i]] = acc;
    acc *= shape[perm[i]];
  }
  return st;
}

bool is_view(int op, const Perm& tperm, const Shape& xs, const Shape& ys, const Perm& lin,
             const Perm& lout) {
  if (op == FLUID_OP_TRANSPOSE) {
    std::vector<int> mapped;
    for (int s : lout)
      if (ys[s] != 1) mapped.push_back(tperm[s]);
    return mapped == physical_key(xs, lin);
  }
  if (op == FLUID_OP_RESHAPE) {
    int a;
    ReshapeKind k = reshape_kind(xs, ys, &a);
    std::vector<int> c;
    switch (k) {
      case ReshapeKind::Same:
        return physical_key(xs, lin) == physical_key(ys, lout);
      case ReshapeKind::Split:
        return collapse(lout, ys, a, &c) && c == physical_key(xs, lin);
      case ReshapeKind::Merge:
        return collapse(lin, xs, a, &c) && c == physical_key(ys, lout);
      default:
        return false;
    }
  }
  return false;
}

}  // namespace fluid
