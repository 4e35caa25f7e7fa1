// Internal declarations shared by the plan builder and the kernel launchers.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <vector>

#include "../../include/spingtp.h"
#include "layout.h"

namespace spingtp {

// Launch description of one compiled kernel instantiation.
struct KernelEntry {
    int waves;        // waves (64 lanes) per workgroup
    int units;        // units per workgroup (one per lane)
    int lds_bytes;    // dynamic LDS per workgroup
    int family;       // 1 = register-tiled fixed-degree kernel
    hipError_t (*launch)(const void* x1, const void* x2, void* out, int64_t units, const float* tab,
                         hipStream_t stream);
};

// Finds the instantiation for (L1, L2, Lout, spin mode, dtype); nullptr if none.
const KernelEntry* find_kernel(int L1, int L2, int LO, int spin_mode, int dtype);

// Builds the float64 tables (layout.h) into `out`; returns false on a failed
// self-check.  spin_mode: 0 = {0}, 1 = {-1, 0, +1}.
bool build_tables(int L1, int L2, int LO, int spin_mode, unsigned flags, std::vector<double>& out);

// Dense real tensor of the operation (see spingtp_dense_tensor_host), float64.
void build_dense_tensor(int L1, int L2, int LO, const int* spins, int n_spins, unsigned flags,
                        std::vector<double>& T);

}  // namespace spingtp

struct spingtp_plan_s {
    int L1, L2, LO;
    int spin_mode;
    int n_spins;
    spingtp_dtype dtype;
    unsigned flags;
    int device;
    float* d_tab;
    size_t n_tab;
    const spingtp::KernelEntry* kernel;
};
