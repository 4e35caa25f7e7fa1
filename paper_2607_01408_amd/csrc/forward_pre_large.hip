// Family 5 instantiations with KS or NT in {7, 8, 10} (row lengths 97..160: degree
// 5 or 6 with spins {-1, 0, +1}, degree 4 with spins {-2..2}); the kernel is in
// forward_pre.h.  At KS = NT = 10
// one workgroup holds 147.5 KB of LDS, so one is resident per CU.
#include "forward_pre.h"

namespace spingtp {
namespace {

struct PreLarge {
    int ks, nt;
    KernelEntry e[2];
};

#define SPINGTP_PRE_ITEM(KS, NT) \
    PreLarge { KS, NT, SPINGTP_PRE_PAIR(KS, NT) }

const PreLarge kPreLarge[] = {
    SPINGTP_PRE_ITEM(1, 7),  SPINGTP_PRE_ITEM(2, 7),  SPINGTP_PRE_ITEM(3, 7),  SPINGTP_PRE_ITEM(4, 7),
    SPINGTP_PRE_ITEM(5, 7),  SPINGTP_PRE_ITEM(7, 7),  SPINGTP_PRE_ITEM(10, 7), SPINGTP_PRE_ITEM(1, 10),
    SPINGTP_PRE_ITEM(2, 10), SPINGTP_PRE_ITEM(3, 10), SPINGTP_PRE_ITEM(4, 10), SPINGTP_PRE_ITEM(5, 10),
    SPINGTP_PRE_ITEM(7, 10), SPINGTP_PRE_ITEM(10, 10), SPINGTP_PRE_ITEM(7, 1), SPINGTP_PRE_ITEM(7, 2),
    SPINGTP_PRE_ITEM(7, 3),  SPINGTP_PRE_ITEM(7, 4),  SPINGTP_PRE_ITEM(7, 5),  SPINGTP_PRE_ITEM(10, 1),
    SPINGTP_PRE_ITEM(10, 2), SPINGTP_PRE_ITEM(10, 3), SPINGTP_PRE_ITEM(10, 4), SPINGTP_PRE_ITEM(10, 5),
    SPINGTP_PRE_ITEM(8, 8),  SPINGTP_PRE_ITEM(1, 8),  SPINGTP_PRE_ITEM(2, 8),  SPINGTP_PRE_ITEM(3, 8),
    SPINGTP_PRE_ITEM(5, 8),  SPINGTP_PRE_ITEM(8, 1),  SPINGTP_PRE_ITEM(8, 2),  SPINGTP_PRE_ITEM(8, 3),
    SPINGTP_PRE_ITEM(8, 5),
};
#undef SPINGTP_PRE_ITEM

}  // namespace

const KernelEntry* find_pre_kernel_large(int ks, int nt, int dtype) {
    for (const PreLarge& p : kPreLarge)
        if (p.ks == ks && p.nt == nt) return &p.e[dtype];
    return nullptr;
}

}  // namespace spingtp
