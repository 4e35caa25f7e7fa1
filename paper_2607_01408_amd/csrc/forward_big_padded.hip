// The mixed-degree instantiations of the large-degree kernel (PAD, forward_pair.h):
// a plan with degrees (L1, L2, Lout) whose rows exceed the direct kernel's runs on the
// kernel of L = max(L1, L2, Lout), 9..16, with x1 and x2 zero-padded as they are staged
// and the product truncated to Lout as it is stored.  Paper basis with spins
// {-1, 0, +1} and spin {0} here; the parity-basis ones, built with the
// register-minimising scheduler like their equal-degree counterparts, are in
// forward_big_parity_padded.hip.  A translation unit of its own so that it compiles
// beside forward.hip.
#include <hip/hip_runtime.h>

#include "forward_pair.h"
#include "internal.h"

namespace spingtp {
namespace {

template <int L, bool SPIN, typename TIO>
constexpr KernelEntry big_padded_entry() {
    constexpr int W = big_waves<L, SPIN>();
    using B = BigShape<L, SPIN, W>;
    return KernelEntry{B::WAVES, B::UNITS, static_cast<int>(B::LDS_FLOATS * sizeof(float)), 3,
                       &launch_big<L, SPIN, W, false, false, TIO, true>,
                       &launch_big<L, SPIN, W, true, false, TIO, true>};
}

template <bool SPIN, typename TIO>
struct PaddedRow {
    KernelEntry e[8] = {big_padded_entry<9, SPIN, TIO>(),  big_padded_entry<10, SPIN, TIO>(),
                        big_padded_entry<11, SPIN, TIO>(), big_padded_entry<12, SPIN, TIO>(),
                        big_padded_entry<13, SPIN, TIO>(), big_padded_entry<14, SPIN, TIO>(),
                        big_padded_entry<15, SPIN, TIO>(), big_padded_entry<16, SPIN, TIO>()};
};

// [spin mode: 0 spin {0}, 1 spins {-1, 0, +1}][dtype: 0 fp32, 1 bf16 I/O]
const PaddedRow<false, float> kPad00;
const PaddedRow<false, uint16_t> kPad01;
const PaddedRow<true, float> kPad10;
const PaddedRow<true, uint16_t> kPad11;

}  // namespace

const KernelEntry* find_big_padded_kernel(int L, int spin_mode, int dtype, bool parity) {
    if (L < 9 || L > 16 || (dtype != 0 && dtype != 1) || (spin_mode != 0 && spin_mode != 1)) return nullptr;
    if (spin_mode == 1 && parity) return find_big_parity_padded_kernel(L, dtype);
    const KernelEntry* row = spin_mode == 0 ? (dtype == 0 ? kPad00.e : kPad01.e) : (dtype == 0 ? kPad10.e : kPad11.e);
    return &row[L - 9];
}

}  // namespace spingtp
