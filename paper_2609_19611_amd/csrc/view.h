// Merged-dim views of a graph for the separable plan compiler.
//
// The plan keeps each tensor's path-count function as a sum of products of
// one vector per dim.  Some reads couple dims: a reshape that merges dims
// reads x[o // 4, o % 4], a grouped transposed convolution reads its weight
// at [ci, co mod C_out/g] with ci in co's group; one set of variables then
// feeds two dims of the operand, and its counts are not a product over
// those dims.  Such dims are merged: the tensor is viewed with the
// contiguous dims of a group replaced by one dim (row-major over the group,
// so flat indices, and global ids of leaves, are unchanged).  A read of a
// merged tensor indexes the merged dim by the sum of its dims' index
// functions times their strides inside the group, and keeps each dim's own
// index function as a guard (it must be valid for the point to read).  The
// op writing a merged tensor reads in terms of the merged coordinate m:
// dim a of the group is floor(m / st_a) mod s_a.
//
// Merging can make more reads couple (the writer of a merged tensor now
// reads with one variable where it had two), so the partition is grown to
// a fixpoint.  Graphs that need no merge keep the identity partition and an
// unchanged graph.
#pragma once
#include <vector>

#include "graph.h"

namespace dg {

// part[t][d]: the group of dim d of tensor t; groups are contiguous runs of
// dims numbered 0, 1, ... in order.
typedef std::vector<std::vector<int>> DimPartition;

DimPartition identity_partition(const GraphIR& g);

struct MergedView {
  GraphIR ir;          // the graph over merged dims (same tensors and ops)
  DimPartition part;   // the partition it uses
};

// The coarsest partition needed, grown from `start` (identity when null),
// and the graph over it.  Throws Failure(DG_E_UNSUPPORTED_OP) when a merge
// cannot be expressed: a merged dim read through an outer division, or a
// merged coordinate that a read divides at a dim other than the group's
// first.
MergedView merged_view(const GraphIR& g, const DimPartition* start = nullptr);

// The finest partition coarser than both a and b (dims of one tensor).
std::vector<int> join_partition(const std::vector<int>& a, const std::vector<int>& b);

}  // namespace dg
