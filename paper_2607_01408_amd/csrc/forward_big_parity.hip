// The parity-basis instantiations of the large-degree forward kernel (L = 9..16,
// spins {-1, 0, +1}, fp32).  They mix the +-1 blocks of each input row as step (A)
// reads them, which doubles that step's register traffic; built in a translation
// unit of their own with the register-minimising scheduling strategy (build.py),
// which measured 22 % (L = 12) to 35 % (L = 16) faster for them and slower for the
// paper-basis kernels, which stay in forward.hip.
#include <hip/hip_runtime.h>

#include "forward_pair.h"
#include "internal.h"

namespace spingtp {
namespace {

template <int L>
constexpr KernelEntry big_parity_entry() {
    constexpr int W = big_waves<L, true>();
    using B = BigShape<L, true, W>;
    return KernelEntry{B::WAVES, B::UNITS, static_cast<int>(B::LDS_FLOATS * sizeof(float)), 3,
                       &launch_big<L, true, W, false, true>, &launch_big<L, true, W, true, true>};
}

const KernelEntry kBigParity[] = {big_parity_entry<9>(),  big_parity_entry<10>(), big_parity_entry<11>(),
                                  big_parity_entry<12>(), big_parity_entry<13>(), big_parity_entry<14>(),
                                  big_parity_entry<15>(), big_parity_entry<16>()};

}  // namespace

const KernelEntry* find_big_parity_kernel(int L) { return L >= 9 && L <= 16 ? &kBigParity[L - 9] : nullptr; }

}  // namespace spingtp
