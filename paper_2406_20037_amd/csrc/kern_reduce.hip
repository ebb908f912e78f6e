// The second launch of a split schedule: the sum of the partial outputs in
// split order (a reduction split across workgroups, then its reduction).
#include <array>
#include <utility>

#include "kern_common.h"
#include "kern_reduce.h"

namespace ds {

namespace {

// y[i] = sum over z < S of part[z * n + i], summed in split order.  S is a
// template parameter so every thread issues its S loads before the first add.
template <int S>
__global__ __launch_bounds__(256) void split_reduce_kernel(const float *__restrict__ part,
                                                           float *__restrict__ y, int64_t n) {
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    const bool vec = (n % 4 == 0) && (reinterpret_cast<uintptr_t>(y) % 16 == 0) &&
                     (reinterpret_cast<uintptr_t>(part) % 16 == 0);
    if (vec) {
        const int64_t n4 = n / 4;
        const floatx4 *p4 = reinterpret_cast<const floatx4 *>(part);
        for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n4; i += stride) {
            floatx4 v[S];
#pragma unroll
            for (int z = 0; z < S; ++z) v[z] = p4[z * n4 + i];
            floatx4 s = v[0];
#pragma unroll
            for (int z = 1; z < S; ++z) s += v[z];
            reinterpret_cast<floatx4 *>(y)[i] = s;
        }
    } else {
        for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
            float v[S];
#pragma unroll
            for (int z = 0; z < S; ++z) v[z] = part[z * n + i];
            float s = v[0];
#pragma unroll
            for (int z = 1; z < S; ++z) s += v[z];
            y[i] = s;
        }
    }
}

template <int... S>
constexpr std::array<const void *, sizeof...(S) + 2> split_reduce_table(
    std::integer_sequence<int, S...>) {
    return {nullptr, nullptr, reinterpret_cast<const void *>(&split_reduce_kernel<S + 2>)...};
}
// kSplitReduce[S]: the reduce kernel of S partial slices, 2 <= S <= kMaxSplits
const std::array<const void *, kMaxSplits + 1> kSplitReduce =
    split_reduce_table(std::make_integer_sequence<int, kMaxSplits - 1>{});

}  // namespace

const void *split_reduce_kernel_for(int splits) {
    return splits >= 2 && splits <= kMaxSplits ? kSplitReduce[splits] : nullptr;
}

}  // namespace ds
