// Family 5 instantiations with KS, NT <= 5 (row lengths <= 80) and the lookup of
// the precontracted kernel; the kernel is in forward_pre.h.
#include "forward_pre.h"

namespace spingtp {
namespace {

#define SPINGTP_PRE_ROW(KS)                                                                        \
    {SPINGTP_PRE_PAIR(KS, 1), SPINGTP_PRE_PAIR(KS, 2), SPINGTP_PRE_PAIR(KS, 3), SPINGTP_PRE_PAIR(KS, 4), \
     SPINGTP_PRE_PAIR(KS, 5)}

// [KS - 1][NT - 1][dtype]
const KernelEntry kPreSmall[5][5][2] = {SPINGTP_PRE_ROW(1), SPINGTP_PRE_ROW(2), SPINGTP_PRE_ROW(3),
                                        SPINGTP_PRE_ROW(4), SPINGTP_PRE_ROW(5)};
#undef SPINGTP_PRE_ROW

}  // namespace

const KernelEntry* find_pre_kernel(int L1, int L2, int LO, int ns, int dtype) {
    const int nc1 = ns * (L1 + 1) * (L1 + 1), nc2 = ns * (L2 + 1) * (L2 + 1), nco = ns * (LO + 1) * (LO + 1);
    if (nc1 > kPreMaxNC || nc2 > kPreMaxNC || nco > kPreMaxNC || dtype < 0 || dtype > 1) return nullptr;
    const int ks = (nc1 + 15) / 16, nt = (nco + 15) / 16;
    if (ks <= 5 && nt <= 5) return &kPreSmall[ks - 1][nt - 1][dtype];
    return find_pre_kernel_large(ks, nt, dtype);
}

}  // namespace spingtp
