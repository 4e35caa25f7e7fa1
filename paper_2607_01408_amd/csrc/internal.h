// Internal declarations shared by the plan builder and the kernel launchers.
#pragma once

#include <hip/hip_runtime_api.h>

#include <array>
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
    int family;       // see spingtp_plan_kernel_info
    // tab: the fp32 plan tables (layout.h); aux: the matrix-core operand tables
    // (build_mfma_operands), nullptr for the vector-ALU families.
    // cpx2: units per row of x2 (1: one x2 row per unit; C: one per edge, shared by
    // its C channels)
    hipError_t (*launch)(const void* x1, const void* x2, void* out, int64_t units, int64_t cpx2, const float* tab,
                         const uint32_t* aux, hipStream_t stream);
    // the instantiation spingtp_backward launches: input-2 lanes take the second
    // copy of the m = 0 mixing (layout.h n0b); nullptr where there is none
    hipError_t (*launch_bwd)(const void* x1, const void* x2, void* out, int64_t units, int64_t cpx2,
                             const float* tab, const uint32_t* aux, hipStream_t stream);
    // the direct kernel (family 6) instead of `launch`: its LDS size comes with the
    // call (the plan's, from its entry table); nullptr for the other families
    hipError_t (*launch_lds)(const void* x1, const void* x2, void* out, int64_t units, int64_t cpx2,
                             const uint32_t* aux, int lds_floats, hipStream_t stream);
};

// Largest row length (n_spins (L+1)^2) of the precontracted kernel: L <= 6 with
// spins {-1, 0, +1}.  Its instantiations cover KS = ceil(NC1/16) and
// NT = ceil(NCO/16) in {1, 2, 3, 4, 5, 7, 10}, and 8 paired with {1, 2, 3, 5, 8}:
// L <= 6 with spins {-1, 0, +1}, L <= 7 with spin {0}, L <= 4 with spins {-2..2}.
constexpr int kPreMaxNC = 147;
// Threads per workgroup of the precontracted kernel (its tensor items are laid out
// for exactly this many threads) and the words of its table header.
constexpr int kPreThreads = 256;
constexpr int kPreHeader = 16;
// k3 rows per kernel block of the large instantiations (KS or NT above 5)
constexpr int kPreBlockRows = 48;

// Direct sparse-tensor kernel (family 6, forward_direct.hip): units per workgroup
// (one wave) and the largest LDS tile it takes (160 KB).
constexpr int kDirectUnits = 64;
constexpr int kDirectWaves = 4;  // waves of a workgroup, sharing its tile, each with a range of outputs
constexpr int kDirectThreads = 64 * kDirectWaves;
constexpr int kDirectMaxLdsFloats = 40960;
// entries per batch of its table, and the longest row its 8-bit entry indices reach
// (a row's zero column sits at index row length)
constexpr int kDirectBatch = 16;
constexpr int kDirectMaxRow = 254;
// The direct kernel for an LDS tile of `lds_floats`; nullptr if it does not fit.
const KernelEntry* find_direct_kernel(int lds_floats, int dtype);
// Entry table of the direct kernel for one role of the tensor T[k1][k2][k3]:
// role 0 (forward) A = x1, B = x2, output k3; role 1 (grad x1) A = grad_out,
// B = x2, output k1; role 2 (grad x2) A = grad_out, B = x1, output k2.  Layout in
// forward_direct.hip; entries per output in ascending (a, b) order, padded to
// batches of 16 with zero entries on the zero column past each row.  *lds_floats:
// the LDS the kernel needs for it (its A and B tiles).
// `dense`: the tensor of build_dense_tensor for these arguments if the caller has
// it (built here otherwise).
void build_direct_table(int L1, int L2, int LO, const int* spins, int n_spins, unsigned flags, int role,
                        std::vector<uint32_t>& out, int* lds_floats, const std::vector<double>* dense = nullptr);

// Finds the instantiation for (L1, L2, Lout, spin mode, dtype); nullptr if none.
// find_kernel returns the vector-ALU kernels, find_mfma_kernel the matrix-core
// kernel where one is built.  parity: the plan's basis is the parity-labelled one
// with an |s| = 1 sector (the large-degree family has a separate instantiation).
const KernelEntry* find_kernel(int L1, int L2, int LO, int spin_mode, int dtype, bool parity);
// The parity-basis large-degree kernel of L1 = L2 = Lout = L (9..16, spins {-1, 0, +1},
// dtype 0 fp32, 1 bf16 I/O; forward_big_parity.hip), nullptr otherwise.
const KernelEntry* find_big_parity_kernel(int L, int dtype);
// The mixed-degree (zero-padded) large-degree kernel of L = max(L1, L2, Lout), 9..16, for
// spin mode 0 or 1 and dtype 0 / 1; its launches take the degree triple as `aux`
// (forward_big_padded.hip, forward_big_parity_padded.hip).  nullptr otherwise.
const KernelEntry* find_big_padded_kernel(int L, int spin_mode, int dtype, bool parity);
const KernelEntry* find_big_parity_padded_kernel(int L, int dtype);
const KernelEntry* find_mfma_kernel(int L1, int L2, int LO, int spin_mode, int dtype);
// The precontracted kernel of spingtp_forward_v1 (x2 shared by the channels of an edge).
const KernelEntry* find_pre_kernel(int L1, int L2, int LO, int n_spins, int dtype);
// The per-channel path-weighted kernel (forward_pre_weighted.hip): the smallest
// instantiation with KS >= ks_min and NT >= nt_min (its KS and NT to *ks, *nt);
// nullptr if none (KS up to 30, NT up to 3).
const KernelEntry* find_pre_weighted_kernel(int ks_min, int nt_min, int dtype, int* ks, int* nt);
// The instantiations with KS or NT in {7, 10} (forward_pre_large.hip); nullptr if none.
const KernelEntry* find_pre_kernel_large(int ks, int nt, int dtype);

// Sparse tensor of the precontracted kernel (forward_pre.h).  Header words NCOL
// (the contraction length: NC1, or the path slots of the per-channel weighted
// table), NC2, NCO, BLK1 = (L1+1)^2, KS = ceil(NCOL/16) (or the instantiation's),
// NT = ceil(NCO/16), IPT, KST = 16 KS + 4, NB3, RB, STRIDE, n_spins, NC1 (x1 row
// length), NPATHS (0 unweighted), the word offset of the path slots (0
// unweighted), 0: the kernel's k3 rows come in NB3 blocks
// of RB rows (one block of 16 NT rows for KS, NT <= 5; kPreBlockRows otherwise).
// Then per block STRIDE x kPreThreads items [item][thread]: IPT items (a multiple
// of 8) for the one-block kernel, STRIDE = IPT; for the blocked kernel IPT is a
// multiple of 16 and 16 zero items follow (STRIDE = IPT + 16), which that kernel
// loads ahead without conditions.  Each item is the two words
// dst | k2 << 16 | last << 24 (dst = (k3 - RB b) KST + k1 within block b) and an
// fp32 value.  An item
// adds value * x2[k2] to the thread's running sum, and `last` stores the sum to the
// transposed edge kernel at LDS index dst = k3 KST + k1 and restarts it.  Whole
// (k1, k3) lists go to one thread (longest first, to the least loaded thread), so
// every entry has one writer; lists are padded with zero items.
// conj_x2: the table of spingtp_backward_v1, whose kernel reads x2 but must use
// J x2 (build_conj_map); false if J cannot be built.
// The table of the per-channel path-weighted kernel (spingtp_forward_v1_weighted):
// the contraction runs over path slots q = (path p, x1 slot k1 of p's input-1
// block), listed path by path (paths in spingtp_paths_host order, k1 ascending);
// entry (q, k3) sums T[k1, k2, k3] x2[k2] over k2 of p's input-2 block, for k3 of
// p's output block.  ks: the instantiation's contraction blocks (16 ks >= the
// number of path slots, written to *n_rows; false otherwise).  One block of rows.
// The path slots follow the items: x1 slot | path << 16.
bool build_pre_tables_channel_weighted(int L1, int L2, int LO, const int* spins, int n_spins, unsigned flags,
                                       int ks, std::vector<uint32_t>& out, int* n_rows);
std::vector<int> slot_blocks(int L, const int* spins, int n_spins);
// dense: the tensor to tabulate (the plan's, e.g. path-weighted); built here when nullptr.
bool build_pre_tables(int L1, int L2, int LO, const int* spins, int n_spins, unsigned flags,
                      std::vector<uint32_t>& out, bool conj_x2 = false, const std::vector<double>* dense = nullptr);

// Per-lane A operands of the matrix-core kernel for L1 = L2 = Lout = L, spins
// {-1, 0, +1}: packed fp16 (hi, lo) words; layout in forward_mfma.hip.
void build_mfma_operands(int L, std::vector<uint32_t>& out);

// Builds the float64 tables (layout.h) into `out`; returns false on a failed
// self-check.  spin_mode: 0 = {0}, 1 = {-1, 0, +1}.  conj_input2: the tables of
// spingtp_backward, where input 2 enters conjugated (its N0 mixing absorbs the
// conjugation map; false if that map is not of the form this needs).
bool build_tables(int L1, int L2, int LO, int spin_mode, unsigned flags, std::vector<double>& out,
                  bool conj_input2 = false);

// Real matrix J of complex conjugation on real-basis coefficients of degree <= L
// (conj of sum x[k] R_k is sum (J x)[k] R_k; App. A.1 conjugation relation), as
// one word per destination slot j: (J x)[j] = +-x[src] with src in the low 16 bits,
// kConjNeg for the sign, kConjZero for slots with l < |s| (written 0).  Returns
// false if J is not a signed permutation.
constexpr uint32_t kConjNeg = 1u << 16;
constexpr uint32_t kConjZero = 1u << 17;
bool build_conj_map(int L, const int* spins, int n_spins, unsigned flags, std::vector<uint32_t>& out);

// Argument checks and launch of one forward kernel (api.cpp).  shared_x2: x2
// holds one row per edge (spingtp_forward_v1), else one per unit.  tab: the
// plan tables to use (the plan's own when nullptr); backward: launch the
// entry's launch_bwd instantiation (the matrix-core and vector-ALU families);
// aux: the operand or tensor table to pass (the plan's own when nullptr).
spingtp_status run_forward(spingtp_plan plan, const KernelEntry* k, const void* x1, const void* x2, void* out,
                           int64_t N, int64_t C, bool shared_x2, void* stream, const float* tab = nullptr,
                           bool backward = false, const uint32_t* aux = nullptr);

// Gradients of the per-channel path-weighted product (backward_v1w.hip).
// Sizes of its table; lds_floats: the LDS of one workgroup (weight, gW, x1 and
// grad_out tiles of 64 rows and the x2 row); lds_unit_bwd, lds_unit_fwd: those of
// the per-unit x2 forms (spingtp_backward_weighted, spingtp_forward_weighted), 0
// where they exceed 160 KB; lds_shared_fwd: that of the entry-list forward with x2
// shared by the channels (spingtp_forward_v1_weighted), 0 where it exceeds 160 KB.
struct Bw1wShape {
    int nc1, nc2, nco, np, lds_floats, lds_unit_bwd, lds_unit_fwd, lds_shared_fwd;
};
constexpr int kBw1wWaves = 4;             // waves of a workgroup, splitting each pass's keys
constexpr int kBw1wMaxLdsFloats = 40960;  // 160 KB
constexpr int kBw1wMaxIndex = 1022;       // 10-bit entry fields; a row's zero column sits at index n
constexpr int kBw1wTargetGroups = 512;    // default workgroup target of bw1w_groups
// Entry lists of the table (layout in backward_v1w.hip); false where an index or the
// LDS tile does not fit.  `dense`: the tensor of build_dense_tensor if the caller has it.
bool build_bwd_v1w_table(int L1, int L2, int LO, const int* spins, int n_spins, unsigned flags,
                         std::vector<uint32_t>& out, Bw1wShape* shape, const std::vector<double>* dense = nullptr);
// Edge ranges of a launch: `groups` ranges of `epg` edges (0, 0 when N or C is 0), for
// about `target` workgroups.
void bw1w_groups(int64_t N, int64_t C, int64_t* groups, int64_t* epg, int target = kBw1wTargetGroups);
// Workspace of a launch, in floats: gx2 partial sums per channel tile and edge, then
// gW partial sums per edge range, path and channel.
size_t bw1w_workspace_floats(int64_t N, int64_t C, const Bw1wShape& s);
// Workspace of the per-unit x2 gradients, in floats: gW partial sums per edge range.
size_t bwcw_workspace_floats(int64_t N, int64_t C, const Bw1wShape& s);
// dtype 0: fp32 x1, x2, grad_out, gx1, gx2; 1: bf16.  Weights and gW are fp32.
// shared_x2: x2 [N][NC2] shared by the channels (spingtp_backward_v1_weighted), else
// x2 [N][C][NC2] per unit (spingtp_backward_weighted).
// x2_stride (shared x2): elements between the x2 (and gx2) rows of consecutive edges,
// 0 for NC2; accumulate_gx1: add gx1 to what grad_x1 holds (the depthwise mode's sum
// over its second-input channels).
hipError_t launch_bwd_v1w(int dtype, bool shared_x2, const void* x1, const void* x2, const float* w, const void* g,
                          void* gx1, void* gx2, float* gw, float* ws, int64_t N, int64_t C, const Bw1wShape& s,
                          const uint32_t* tab, hipStream_t stream, int64_t x2_stride = 0,
                          bool accumulate_gx1 = false);
// out[n][c] = sum_p W[c][p] T_p(x1[n][c], x2[n][c]) (spingtp_forward_weighted), or with
// x2[n] shared by the channels (shared_x2, spingtp_forward_v1_weighted).
// x2_stride, accumulate: as for launch_bwd_v1w (accumulate adds to out).
// nv > 1 (shared_x2 only): nv second-input channels in one launch (the depthwise mode),
// their x2 rows x2v elements apart within an edge's row and their weight slices
// wslice floats apart; the LDS that takes is fwd_cw_lds_floats(s, nv).
constexpr int kFwdCwMaxNv = 4;
hipError_t launch_fwd_cw(int dtype, bool shared_x2, const void* x1, const void* x2, const float* w, void* out,
                         int64_t N, int64_t C, const Bw1wShape& s, const uint32_t* tab, hipStream_t stream,
                         int64_t x2_stride = 0, bool accumulate = false, int nv = 1, int64_t x2v = 0,
                         int64_t wslice = 0);
int fwd_cw_lds_floats(const Bw1wShape& s, int nv);

// Paths of the instruction-weighted product (spingtp_paths_host): the block triples
// (i (L+1) + l of spin index i and degree l, per input and output) on which T has
// a nonzero entry, in ascending lexicographic order.
void tensor_paths(int L1, int L2, int LO, const int* spins, int n_spins, const std::vector<double>& T,
                  std::vector<std::array<int, 3>>& paths);
// T[k1][k2][k3] *= w[p] with p the path of (k1, k2, k3); entries at quadrature
// round-off level are set to 0.
void weight_paths(int L1, int L2, int LO, const int* spins, int n_spins, const std::vector<std::array<int, 3>>& paths,
                  const double* w, std::vector<double>& T);

// Fully connected product (mode uvw): entry tables of spingtp_forward_fully_connected
// (role 0: inputs x1, x2, output out) and of the gradients w.r.t. x1 (role 1: inputs x2
// and grad_out, output grad_x1) and x2 (role 2: inputs x1 and grad_out, output grad_x2);
// "a", "b" and "o" below are the role's first input, second input and output.
// Words: header [kUvwHeader]: n_paths, n_blocks (output blocks reached by a path), the
// row widths of a, b and o, max_d3, first word of the path records, first word of the
// entries.  Then per block (4 words): slot offset o3 of the block in the output row, its
// width d3, first path record, path count.  Per path record (kUvwRec words): path index
// (the weights' leading index), d3, first word of its d3 + 1 entry offsets, then the
// path's block of x1, of x2 and of the forward's output as first slot | width << 16
// each.  The offsets
// (absolute entry numbers) delimit its entries by output component m3; an entry is two
// words: ka | kb << 16 and the fp32 value T (at (k1, k2, k3) = (ka, kb, o3 + m3) for
// role 0, (o3 + m3, ka, kb) for role 1, (ka, o3 + m3, kb) for role 2).
constexpr int kUvwHeader = 8;
constexpr int kUvwRec = 6;
constexpr int kUvwChunk = 8;  // output components per workgroup (the kernel's accumulators)
bool build_uvw_table(int L1, int L2, int LO, const int* spins, int n_spins, unsigned flags,
                     std::vector<uint32_t>& out, const std::vector<double>* dense = nullptr, int role = 0);
// One role's product and channel mixing: out[n][o][k] = sum_p sum_(a, b) weights[p-th block
// + a sa + b sb + o so] R_p[n][(a, b)][k], R_p from xa [N][A][.] and xb [N][B][.]; the
// output (N x O rows of nco floats) is written 0 first.
hipError_t launch_uvw_mix(const float* xa, const float* xb, const float* w, float* out, int64_t N, int A, int B, int O,
                          int64_t sa, int64_t sb, int64_t so, int64_t ps, const uint32_t* table, int n_blocks,
                          int max_d3, int nco, hipStream_t stream);
// grad_w[p][u][v][w] = sum_n sum_(k3 in p) R_p[n][(u, v)][k3] g[n][w][k3] (role-0 table).
hipError_t launch_uvw_grad_w(const float* x1, const float* x2, const float* g, float* gw, int64_t N, int U, int V,
                             int W, const uint32_t* table, int n_paths, int nco, hipStream_t stream);
// grad_x2 through gR_p = W_p g (role-0 table; the blocks of x2 from the role-2 table); LDS
// bytes it needs for blocks of x1 and x2 up to d1max and d2max wide (0 if more than a CU has).
size_t uvw_grad_x2_lds(int d1max, int d2max);
hipError_t launch_uvw_grad_x2(const float* x1, const float* g, const float* w, float* gx2, int64_t N, int U, int V,
                              int W, const uint32_t* table, const uint32_t* table2, int n_blocks2, int n_paths,
                              int nc1, int nc2, int nco, int d1max, int d2max, hipStream_t stream);

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
    uint32_t* d_aux;  // matrix-core operand tables, nullptr for the vector-ALU kernels
    uint32_t* d_pre;  // sparse tensor of the precontracted kernel, nullptr if not used
    uint32_t* d_pre_bwd;  // the same with J x2 (spingtp_backward_v1), nullptr if not used
    uint32_t* d_pre_w;    // the per-channel path-weighted table (SPINGTP_CHANNEL_WEIGHTS), nullptr if not built
    const spingtp::KernelEntry* kernel_v1w;  // its kernel (spingtp_forward_v1_weighted)
    uint32_t* d_bw1w;  // entry lists of spingtp_backward_v1_weighted, nullptr if not built
    spingtp::Bw1wShape bw1w;
    float* d_tab_bwd;  // tables of spingtp_backward (d_tab when equal), nullptr without a backward
    bool own_tab_bwd;  // d_tab_bwd is a separate allocation
    uint32_t* d_dir;     // direct-kernel entry table of the forward (family 6), nullptr if not used
    uint32_t* d_dir_b1;  // direct-kernel tables of the gradients w.r.t. x1 and x2, nullptr unless
    uint32_t* d_dir_b2;  //   the gradients run on the direct kernel
    const spingtp::KernelEntry* kernel_dir;  // the direct kernel of d_dir_b1 and d_dir_b2
    int dir_lds_floats;  // LDS of the direct kernel's tiles (the same for its three tables)
    // entry tables of the fully connected product (SPINGTP_FULLY_CONNECTED, else nullptr):
    // roles 0 (forward), 1 and 2 (gradients w.r.t. x1 and x2), each from word uvw_off[role]
    uint32_t* d_uvw;
    size_t uvw_off[3];
    int uvw_blocks[3], uvw_max_d3[3], uvw_paths;
    // mixed degrees on the large-degree kernel of the largest degree: d_aux holds the
    // degree triples of the forward, the grad_x1 and the grad_x2 launches
    bool padded;
    const uint32_t* deg_bwd(int which) const { return padded ? d_aux + 3 * which : nullptr; }
    const spingtp::KernelEntry* kernel;     // spingtp_forward
    const spingtp::KernelEntry* kernel_v1;  // spingtp_forward_v1 (x2 shared by the channels of an edge)
};
