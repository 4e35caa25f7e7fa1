// The parity-basis instantiations of the large-degree forward kernel (L = 9..16,
// spins {-1, 0, +1}, fp32 and bf16 I/O).  They mix the +-1 blocks of each input row as step (A)
// reads them, which doubles that step's register traffic; built in a translation
// unit of their own with the register-minimising scheduling strategy (build.py),
// which measured 22 % (L = 12) to 35 % (L = 16) faster for them and slower for the
// paper-basis kernels, which stay in forward.hip.
#include <hip/hip_runtime.h>

#include "forward_pair.h"
#include "internal.h"

namespace spingtp {
namespace {

template <int L, typename TIO>
constexpr KernelEntry big_parity_entry() {
    constexpr int W = big_waves<L, true>();
    using B = BigShape<L, true, W>;
    return KernelEntry{B::WAVES, B::UNITS, static_cast<int>(B::LDS_FLOATS * sizeof(float)), 3,
                       &launch_big<L, true, W, false, true, TIO>, &launch_big<L, true, W, true, true, TIO>};
}

// [dtype][L - 9]: fp32, then bf16 I/O
const KernelEntry kBigParity[2][8] = {
    {big_parity_entry<9, float>(), big_parity_entry<10, float>(), big_parity_entry<11, float>(),
     big_parity_entry<12, float>(), big_parity_entry<13, float>(), big_parity_entry<14, float>(),
     big_parity_entry<15, float>(), big_parity_entry<16, float>()},
    {big_parity_entry<9, uint16_t>(), big_parity_entry<10, uint16_t>(), big_parity_entry<11, uint16_t>(),
     big_parity_entry<12, uint16_t>(), big_parity_entry<13, uint16_t>(), big_parity_entry<14, uint16_t>(),
     big_parity_entry<15, uint16_t>(), big_parity_entry<16, uint16_t>()}};

}  // namespace

const KernelEntry* find_big_parity_kernel(int L, int dtype) {
    return L >= 9 && L <= 16 && (dtype == 0 || dtype == 1) ? &kBigParity[dtype][L - 9] : nullptr;
}

}  // namespace spingtp
