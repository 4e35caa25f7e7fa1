// The mixed-degree instantiations of the parity-basis large-degree kernel (spins
// {-1, 0, +1}, L = 9..16, fp32 and bf16 I/O; PAD in forward_pair.h), built with the
// register-minimising scheduling strategy like the equal-degree ones in
// forward_big_parity.hip.
#include <hip/hip_runtime.h>

#include "forward_pair.h"
#include "internal.h"

namespace spingtp {
namespace {

template <int L, typename TIO>
constexpr KernelEntry big_parity_padded_entry() {
    constexpr int W = big_waves<L, true>();
    using B = BigShape<L, true, W>;
    return KernelEntry{B::WAVES, B::UNITS, static_cast<int>(B::LDS_FLOATS * sizeof(float)), 3,
                       &launch_big<L, true, W, false, true, TIO, true>, &launch_big<L, true, W, true, true, TIO, true>};
}

// [dtype][L - 9]: fp32, then bf16 I/O
const KernelEntry kBigParityPadded[2][8] = {
    {big_parity_padded_entry<9, float>(), big_parity_padded_entry<10, float>(),
     big_parity_padded_entry<11, float>(), big_parity_padded_entry<12, float>(),
     big_parity_padded_entry<13, float>(), big_parity_padded_entry<14, float>(),
     big_parity_padded_entry<15, float>(), big_parity_padded_entry<16, float>()},
    {big_parity_padded_entry<9, uint16_t>(), big_parity_padded_entry<10, uint16_t>(),
     big_parity_padded_entry<11, uint16_t>(), big_parity_padded_entry<12, uint16_t>(),
     big_parity_padded_entry<13, uint16_t>(), big_parity_padded_entry<14, uint16_t>(),
     big_parity_padded_entry<15, uint16_t>(), big_parity_padded_entry<16, uint16_t>()}};

}  // namespace

const KernelEntry* find_big_parity_padded_kernel(int L, int dtype) {
    return L >= 9 && L <= 16 && (dtype == 0 || dtype == 1) ? &kBigParityPadded[dtype][L - 9] : nullptr;
}

}  // namespace spingtp
