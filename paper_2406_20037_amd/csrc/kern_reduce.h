// The reduce launch of a split schedule (kern_reduce.hip).
#pragma once

namespace ds {

// Reduction splits across workgroups: at most this many partial slices.
constexpr int kMaxSplits = 32;

// The reduce kernel of a split schedule with `splits` partial slices
// (2..kMaxSplits), else null.
const void *split_reduce_kernel_for(int splits);

}  // namespace ds
