// Instantiations of the per-channel path-weighted precontracted kernel
// (spingtp_forward_v1_weighted; the kernel is in forward_pre.h with WGT = true).
// The contraction runs over path slots, so KS covers them (up to 480 slots): at
// degree 2 with spins {-1, 0, +1}, 263 slots in the parity basis (KS = 17) and 471
// in the paper basis (KS = 30), whose +-1 blocks are not irreps and split paths.
#include "forward_pre.h"

namespace spingtp {
namespace {

struct PreWeighted {
    int ks, nt;
    KernelEntry e[2];
};

#define SPINGTP_PRE_W_ITEM(KS, NT) \
    PreWeighted { KS, NT, SPINGTP_PRE_W_PAIR(KS, NT) }
#define SPINGTP_PRE_W_ROW(KS) SPINGTP_PRE_W_ITEM(KS, 1), SPINGTP_PRE_W_ITEM(KS, 2), SPINGTP_PRE_W_ITEM(KS, 3)

// ascending in KS, then NT
const PreWeighted kPreWeighted[] = {
    SPINGTP_PRE_W_ROW(1),  SPINGTP_PRE_W_ROW(2),  SPINGTP_PRE_W_ROW(3),  SPINGTP_PRE_W_ROW(4),  SPINGTP_PRE_W_ROW(5),
    SPINGTP_PRE_W_ROW(6),  SPINGTP_PRE_W_ROW(8),  SPINGTP_PRE_W_ROW(11), SPINGTP_PRE_W_ROW(14), SPINGTP_PRE_W_ROW(17),
    SPINGTP_PRE_W_ROW(20), SPINGTP_PRE_W_ROW(24), SPINGTP_PRE_W_ROW(30),
};
#undef SPINGTP_PRE_W_ROW
#undef SPINGTP_PRE_W_ITEM

}  // namespace

const KernelEntry* find_pre_weighted_kernel(int ks_min, int nt_min, int dtype, int* ks, int* nt) {
    if (dtype < 0 || dtype > 1) return nullptr;
    for (const PreWeighted& p : kPreWeighted)
        if (p.ks >= ks_min && p.nt >= nt_min) {
            *ks = p.ks;
            *nt = p.nt;
            return &p.e[dtype];
        }
    return nullptr;
}

}  // namespace spingtp
