// Candidate layouts, strides and the zero-copy view predicate.
//
// A layout is a permutation of logical dims listed outermost -> innermost;
// the tensor is stored densely in that order.  Candidates L(e) are all
// permutations in lexicographic order with physically identical ones (equal
// once extent-1 dims are dropped) merged into the first; identity first.
#pragma once

#include <vector>

#include "common.h"

namespace fluid {

std::vector<Perm> layout_list(const Shape& shape);
// The measurement-time candidate list: layout_list, trimmed for tensors with
// more than six candidates to those whose innermost dim is one of the last
// two logical dims.
std::vector<Perm> measured_layout_list(const Shape& shape);
Perm identity_perm(int rank);
// Element stride of every logical dim for a dense tensor stored in `perm`.
std::vector<int64_t> dense_strides(const Shape& shape, const Perm& perm);
// True iff, with input layout `lin` and output layout `lout`, a TRANSPOSE
// (perm) or RESHAPE node's output occupies exactly the input's bytes.
bool is_view(int op, const Perm& tperm, const Shape& xs, const Shape& ys, const Perm& lin,
             const Perm& lout);

}  // namespace fluid
