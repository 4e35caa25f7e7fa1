// Fully connected SpinGTP product (mode uvw of App. E.1; Sec. 3.5 eq. spin_gtp) and its
// gradients on gfx950.
//
// For every path p = (rho1, rho2 -> rho3) the product forms
//   R_p[n, (u, v), m3] = sum over the entries (k1, k2, m3) of p of T x1[n, u, k1] x2[n, v, k2]
// and mixes the channels:
//   out[n, w, o3 + m3] = sum_p sum_(u, v) W[p, u, v, w] R_p[n, (u, v), m3],
// o3 the first slot of rho3.  Per path and over all edges the mixing is a dense product
// [W x UV] . [UV x (edges x d3)], so it runs on the matrix cores with fp32 operands and
// sums (v_mfma_f32_32x32x2_f32): output channels w are the M dimension, the (u, v) pairs
// the K dimension and the 32 edges of a tile the N dimension, with one accumulator per
// output component m3.
//
// The gradients w.r.t. x1 and x2 have the same form with the roles of the three tensor
// axes exchanged (chain rule through R_p and the mixing, g = dL/dout):
//   grad_x1[n, u, k1] = sum_p sum_(v, w) W[p, u, v, w] sum_(k1, k2, k3 in p) T x2[n, v, k2] g[n, w, k3],
//   grad_x2[n, v, k2] = sum_p sum_(u, w) W[p, u, v, w] sum_(k1, k2, k3 in p) T x1[n, u, k1] g[n, w, k3],
// so one kernel serves all three: inputs a and b with A and B channels, the pairs (a, b),
// O output channels, the weight of (p, a, b, o) at p-th block + a sa + b sb + o so, and a
// table of the role (entries ka | kb << 16 by output component).  The weight gradient
//   grad_W[p, u, v, w] = sum_n sum_(m3) R_p[n, (u, v), m3] g[n, w, o3 + m3]
// is the product [UV x (edges x d3)] . [(edges x d3) x W] per path: its own kernel.
//
// Mapping of the mixing kernel.  A workgroup owns 32 edges, one output block, 128 output
// channels and CH of the block's components (1 or 8, chosen per launch); wave i owns
// channels 32 i .. 32 i + 31 of the 128.  For every path into the block and every 32 pairs:
//   (1) the 256 threads form R for 32 pairs x 32 edges x CH components into LDS, laid out
//       [pair][component][edge] (a lane's B operand is one conflict-free LDS read), and the
//       pairs' weight offsets;
//   (2) each wave multiplies: A = W[p, pair, o] from global memory, B = R from LDS, 16 K
//       steps of two pairs per component.
// The accumulators stay in registers across the paths of the block; the tile is written
// once at the end.  Blocks reached by no path and slots with l < |s| hold no entry: a
// fill kernel writes the whole output 0 first, in the same stream.
//
// Mapping of the weight-gradient kernel.  A workgroup owns one path, 32 pairs and 128
// output channels w (32 per wave) and runs over all edges in tiles of 32: the 256
// threads form R for the tile (LDS layout [component][edge][pair], so a lane's A operand
// is a conflict-free read), and each wave accumulates A = R[pair, (edge, m3)] times
// B = g[edge, w, o3 + m3], two edges per K step.  Every element of grad_W belongs to one
// workgroup and is summed in a fixed order: deterministic, no atomics.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "internal.h"

namespace spingtp {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f_ __attribute__((ext_vector_type(4)));

constexpr int kEdges = 32;    // N of the matrix-core product: edges of a tile
constexpr int kPairs = 32;    // (a, b) pairs staged per round (16 K steps of two)
constexpr int kGroupW = 128;  // output channels of a workgroup (4 waves x 32)
constexpr int kThreads = 256;
constexpr int kSmallGrid = 512;  // see launch_uvw_mix
constexpr int kSmallChunk = 1;

__global__ __launch_bounds__(kThreads) void spingtp_fill_zero_kernel(float* __restrict__ out, int64_t n) {
    const int64_t n4 = n >> 2;
    v4f_* o4 = reinterpret_cast<v4f_*>(out);
    const v4f_ z = {0.f, 0.f, 0.f, 0.f};
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n4;
         i += static_cast<int64_t>(gridDim.x) * kThreads)
        o4[i] = z;
    const int64_t t = 4 * n4 + static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (t < n) out[t] = 0.f;
}

// R of pair pr (< A B) at edge n (< N) for the components j < mc of one path record:
// r[j] = sum over the record's entries of component m0 + j of T a[ka] b[kb].
template <int CH>
__device__ __forceinline__ void form_r_rows(const float* ra, const float* rb, const uint32_t* __restrict__ csr,
                                            const uint32_t* __restrict__ ent, int mc, float (&r)[CH]) {
#pragma unroll
    for (int j = 0; j < CH; ++j) {
        if (j < mc) {
            float s = 0.f;
            for (uint32_t k = csr[j]; k < csr[j + 1]; ++k) {
                const uint32_t ix = ent[2 * k];
                s = fmaf(__uint_as_float(ent[2 * k + 1]) * ra[ix & 0xffffu], rb[ix >> 16], s);
            }
            r[j] = s;
        }
    }
}

template <int CH>
__device__ __forceinline__ void form_r(const float* __restrict__ xa, const float* __restrict__ xb, int64_t n, int pr,
                                       int A, int B, int nca, int ncb, const uint32_t* __restrict__ csr,
                                       const uint32_t* __restrict__ ent, int mc, float (&r)[CH]) {
    const int a = pr / B, b = pr - a * B;
    form_r_rows(xa + (n * A + a) * nca, xb + (n * B + b) * ncb, csr, ent, mc, r);
}

// Staging of a path's input blocks in LDS for R.  The pairs c0 .. c0 + 31 take the a rows
// a_lo .. a_lo + n_a - 1 (a_lo = c0 / B) and the b rows (b0 + i) mod B, i < n_b (b0 = c0 mod
// B, n_b = min(B, 32)); n_a + n_b <= 34 for every B.  Blocks up to kStageD wide (degree 3)
// are staged: XS[e][row][k] with rows 0 .. n_a - 1 the a rows and n_a .. the b rows, an odd
// edge stride (the lanes of a wave take consecutive edges).  Each value then comes from
// HBM once per tile instead of once per tensor entry that reads it.
constexpr int kStageD = 7;
constexpr int kStageRows = 34;
constexpr int kStageEdge = kStageRows * kStageD + 1;
constexpr int kStageFloats = kEdges * kStageEdge;

struct StageRows {
    int a_lo, n_a, b0, n_b;
};

__device__ __forceinline__ StageRows stage_rows(int c0, int AB, int B) {
    const int last = (c0 + kPairs < AB ? c0 + kPairs : AB) - 1;
    StageRows s;
    s.a_lo = c0 / B;
    s.n_a = last / B - s.a_lo + 1;
    s.b0 = c0 - s.a_lo * B;
    s.n_b = B < kPairs ? B : kPairs;
    return s;
}

// rows of the tile's edges e0 .. e0 + 31 (zeros past N): a block [oa, oa + da) of xa,
// b block [ob, ob + db) of xb
__device__ __forceinline__ void stage_blocks(const float* __restrict__ xa, const float* __restrict__ xb, int64_t e0,
                                             int64_t N, int A, int B, int nca, int ncb, int oa, int da, int ob,
                                             int db, const StageRows& sr, float* XS, int tid) {
    const int pa = sr.n_a * da, pb = sr.n_b * db;
    for (int it = tid; it < kEdges * pa; it += kThreads) {
        const int e = it / pa, rem = it - e * pa, row = rem / da, k = rem - row * da;
        const int64_t n = e0 + e;
        XS[e * kStageEdge + row * kStageD + k] = n < N ? xa[(n * A + sr.a_lo + row) * nca + oa + k] : 0.f;
    }
    for (int it = tid; it < kEdges * pb; it += kThreads) {
        const int e = it / pb, rem = it - e * pb, row = rem / db, k = rem - row * db;
        const int64_t n = e0 + e;
        int b = sr.b0 + row;
        if (b >= B) b -= B;
        XS[e * kStageEdge + (sr.n_a + row) * kStageD + k] = n < N ? xb[(n * B + b) * ncb + ob + k] : 0.f;
    }
}

// CH: output components per workgroup (the accumulators of a wave)
template <int CH>
__global__ __launch_bounds__(kThreads) void spingtp_uvw_mix_kernel(const float* __restrict__ xa,
                                                                   const float* __restrict__ xb,
                                                                   const float* __restrict__ wt,
                                                                   float* __restrict__ out, int64_t N, int A, int B,
                                                                   int O, int64_t sa, int64_t sb, int64_t so,
                                                                   int64_t ps, const uint32_t* __restrict__ tab,
                                                                   int n_chunks, int nco) {
    __shared__ float R[kPairs * CH * kEdges];
    __shared__ int64_t woff[kPairs];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t e0 = static_cast<int64_t>(blockIdx.x) * kEdges;
    const uint32_t* blk = tab + kUvwHeader + 4 * blockIdx.y;
    const int o3 = static_cast<int>(blk[0]), d3 = static_cast<int>(blk[1]);
    const int rec_first = static_cast<int>(blk[2]), n_rec = static_cast<int>(blk[3]);
    const int og = static_cast<int>(blockIdx.z) / n_chunks;
    const int m0 = (static_cast<int>(blockIdx.z) - og * n_chunks) * CH;
    if (m0 >= d3) return;  // the whole workgroup: this block has fewer components
    const int mc = d3 - m0 < CH ? d3 - m0 : CH;
    const int nca = static_cast<int>(tab[2]), ncb = static_cast<int>(tab[3]);
    const uint32_t* recs = tab + tab[6];
    const uint32_t* ent = tab + tab[7];
    const int AB = A * B;
    const int obase = og * kGroupW + 32 * wave;  // this wave's first output channel
    const bool wave_on = obase < O;
    const int o_lane = obase + (lane & 31);
    const int64_t o_off = static_cast<int64_t>(o_lane) * so;
    const int half = lane >> 5;

    v16f acc[CH];
#pragma unroll
    for (int j = 0; j < CH; ++j) acc[j] = v16f{};

    for (int q = 0; q < n_rec; ++q) {
        const uint32_t* rec = recs + kUvwRec * (rec_first + q);
        const uint32_t* csr = tab + rec[2] + m0;  // entry offsets of components m0 .. m0 + mc
        const float* __restrict__ wp = wt + static_cast<int64_t>(rec[0]) * ps;
        for (int c0 = 0; c0 < AB; c0 += kPairs) {
            // (1) R of pairs c0 .. c0 + 31 for the tile's edges, components m0 .. m0 + mc - 1
            for (int it = tid; it < kPairs * kEdges; it += kThreads) {
                const int pl = it >> 5, e = it & 31;
                const int pr = c0 + pl;
                const int64_t n = e0 + e;
                float r[CH];
#pragma unroll
                for (int j = 0; j < CH; ++j) r[j] = 0.f;
                if (pr < AB && n < N) form_r(xa, xb, n, pr, A, B, nca, ncb, csr, ent, mc, r);
#pragma unroll
                for (int j = 0; j < CH; ++j) R[(pl * CH + j) * kEdges + e] = r[j];
            }
            if (tid < kPairs) {
                const int pr = c0 + tid;
                const int a = pr / B, b = pr - a * B;
                woff[tid] = pr < AB ? a * sa + b * sb : 0;
            }
            __syncthreads();
            // (2) out[o, edge] += W[p, pair, o] R[pair, edge] for each component
            if (wave_on) {
#pragma unroll 2
                for (int kk = 0; kk < kPairs; kk += 2) {
                    const int pr = c0 + kk + half;
                    const float av = (pr < AB && o_lane < O) ? wp[woff[kk + half] + o_off] : 0.f;
                    const float* rb = R + ((kk + half) * CH) * kEdges + (lane & 31);
#pragma unroll
                    for (int j = 0; j < CH; ++j)
                        if (j < mc) acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, rb[j * kEdges], acc[j], 0, 0, 0);
                }
            }
            __syncthreads();
        }
    }

    // (3) accumulator element i of lane l holds channel obase + 8 (i / 4) + 4 (l / 32) + i % 4
    //     and edge e0 + l % 32
    if (!wave_on) return;
    const int64_t n = e0 + (lane & 31);
    if (n >= N) return;
#pragma unroll
    for (int j = 0; j < CH; ++j) {
        if (j >= mc) break;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int o = obase + 8 * (i >> 2) + 4 * half + (i & 3);
            if (o < O) out[(n * O + o) * nco + o3 + m0 + j] = acc[j][i];
        }
    }
}

// kPairs + 1: the row stride of one (component, edge) row of R in the weight-gradient kernel
constexpr int kPairsPad = kPairs + 1;

__global__ __launch_bounds__(kThreads) void spingtp_uvw_grad_w_kernel(const float* __restrict__ x1,
                                                                      const float* __restrict__ x2,
                                                                      const float* __restrict__ g,
                                                                      float* __restrict__ gw, int64_t N, int U, int V,
                                                                      int W, const uint32_t* __restrict__ tab,
                                                                      int nco) {
    __shared__ float R[kUvwChunk * kEdges * kPairsPad];
    __shared__ float XS[kStageFloats];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int half = lane >> 5;
    const uint32_t* rec = tab + tab[6] + kUvwRec * blockIdx.x;  // one path record per workgroup column
    const int p = static_cast<int>(rec[0]), d3 = static_cast<int>(rec[1]), o3 = static_cast<int>(rec[5] & 0xffffu);
    const int nc1 = static_cast<int>(tab[2]), nc2 = static_cast<int>(tab[3]);
    const uint32_t* ent = tab + tab[7];
    const int UV = U * V;
    const int c0 = static_cast<int>(blockIdx.y) * kPairs;
    const int wbase = static_cast<int>(blockIdx.z) * kGroupW + 32 * wave;
    const int w_lane = wbase + (lane & 31);

    // the path's x1 and x2 blocks; staged in LDS per edge tile when both fit and one has
    // degree 2 or more (with blocks of three slots or fewer the direct reads measured faster)
    const int oa = static_cast<int>(rec[3] & 0xffffu), da = static_cast<int>(rec[3] >> 16);
    const int ob = static_cast<int>(rec[4] & 0xffffu), db = static_cast<int>(rec[4] >> 16);
    const bool staged = da <= kStageD && db <= kStageD && (da > 3 || db > 3);
    const StageRows sr = stage_rows(c0, UV, V);

    v16f acc = v16f{};
    for (int64_t e0 = 0; e0 < N; e0 += kEdges) {
        if (staged) {
            stage_blocks(x1, x2, e0, N, U, V, nc1, nc2, oa, da, ob, db, sr, XS, tid);
            __syncthreads();
        }
        for (int m0 = 0; m0 < d3; m0 += kUvwChunk) {
            const int mc = d3 - m0 < kUvwChunk ? d3 - m0 : kUvwChunk;
            const uint32_t* csr = tab + rec[2] + m0;
            // (1) R[component][edge][pair] of the tile
            for (int it = tid; it < kPairs * kEdges; it += kThreads) {
                const int pl = it >> 5, e = it & 31;
                const int pr = c0 + pl;
                const int64_t n = e0 + e;
                float r[kUvwChunk];
#pragma unroll
                for (int j = 0; j < kUvwChunk; ++j) r[j] = 0.f;
                if (pr < UV && n < N) {
                    if (staged) {
                        const int a = pr / V, b = pr - a * V;
                        const int ai = a - sr.a_lo, bi = b >= sr.b0 ? b - sr.b0 : b - sr.b0 + V;
                        const float* xs = XS + e * kStageEdge;
                        form_r_rows(xs + ai * kStageD - oa, xs + (sr.n_a + bi) * kStageD - ob, csr, ent, mc, r);
                    } else {
                        form_r(x1, x2, n, pr, U, V, nc1, nc2, csr, ent, mc, r);
                    }
                }
#pragma unroll
                for (int j = 0; j < kUvwChunk; ++j) R[(j * kEdges + e) * kPairsPad + pl] = r[j];
            }
            __syncthreads();
            // (2) grad_W[pair, w] += R[pair, (edge, m3)] g[edge, w, o3 + m3], edges 2 s + half.
            //     Per edge a lane loads the chunk's components of its (edge, w) row of g
            //     together (adjacent words: the later ones hit the cache the first one
            //     filled), then runs the chunk's products with them.
            if (wbase < W) {
#pragma unroll 2
                for (int s2 = 0; s2 < kEdges; s2 += 2) {
                    const int e = s2 + half;
                    const int64_t n = e0 + e;
                    const bool ok = n < N && w_lane < W;
                    const float* __restrict__ gr = g + (ok ? (n * W + w_lane) * nco + o3 + m0 : 0);
                    float bv[kUvwChunk];
#pragma unroll
                    for (int j = 0; j < kUvwChunk; ++j) bv[j] = (ok && j < mc) ? gr[j] : 0.f;
#pragma unroll
                    for (int j = 0; j < kUvwChunk; ++j)
                        if (j < mc)
                            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(R[(j * kEdges + e) * kPairsPad + (lane & 31)],
                                                                       bv[j], acc, 0, 0, 0);
                }
            }
            __syncthreads();
        }
    }
    // (3) accumulator element i of lane l holds pair c0 + 8 (i / 4) + 4 (l / 32) + i % 4 and
    //     channel w = wbase + l % 32
    if (wbase >= W || w_lane >= W) return;
    float* __restrict__ gp = gw + static_cast<int64_t>(p) * UV * W;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int pr = c0 + 8 * (i >> 2) + 4 * half + (i & 3);
        if (pr < UV) gp[static_cast<int64_t>(pr) * W + w_lane] = acc[i];
    }
}

// grad_x2 in the chain rule's own order (the role-2 form pairs every u with every w):
//   gR_p[n][u][k3]    = sum_w W[p][u][v][w] g[n][w][k3]      (matrix cores: u = M, edges = N, w = K)
//   Z_p[n][k1][k3]    = sum_u x1[n][u][k1] gR_p[n][u][k3]    (a lane: its edge, its 16 u rows;
//                                                             the two half-waves added)
//   grad_x2[n][v][k2] = sum_p sum_(entries (k1, k2, k3) of p) T Z_p[n][k1][k3].
// A workgroup owns 32 edges, one block of x2 (the paths into it: each path has one x2
// block, so the workgroups' slots are disjoint) and one v; wave i takes the u blocks
// 32 i + 128 j and writes its partial Z of one (path, component chunk) item to LDS.  After a
// barrier wave 0 adds the four partials in wave order and scatters the item's entries into
// the LDS tile of the block while the waves compute the next item into the other of two Z
// buffers.  Items in table order: deterministic.
__global__ __launch_bounds__(kThreads) void spingtp_uvw_grad_x2_kernel(const float* __restrict__ x1,
                                                                       const float* __restrict__ g,
                                                                       const float* __restrict__ wt,
                                                                       float* __restrict__ gx2, int64_t N, int U,
                                                                       int V, int W, const uint32_t* __restrict__ tab,
                                                                       const uint32_t* __restrict__ tab2, int n_paths,
                                                                       int nc1, int nc2, int nco, int d1max,
                                                                       int d2max) {
    extern __shared__ float sm[];
    const int zs = kEdges * d1max * kUvwChunk;  // one wave's partial Z: [edge][k1 - o1][component]
    const int st2 = d2max | 1;
    float* Zb = sm;                     // [2 buffers][4 waves][zs]
    float* G2 = sm + 8 * zs;            // [edge][st2]: the tile's grad_x2 slots of the block, this v
    const uint32_t* blk2 = tab2 + kUvwHeader + 4 * blockIdx.y;  // the block (role-2 table)
    const int o2b = static_cast<int>(blk2[0]), d2b = static_cast<int>(blk2[1]);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int half = lane >> 5;
    const int el = lane & 31;
    const int64_t e0 = static_cast<int64_t>(blockIdx.x) * kEdges;
    const int64_t n = e0 + el;
    const bool n_ok = n < N;
    const uint32_t* recs = tab + tab[6];
    const uint32_t* ent = tab + tab[7];
    const int64_t UVW = static_cast<int64_t>(U) * V * W;
    for (int v = blockIdx.z; v < V; v += gridDim.z) {
        for (int i = tid; i < kEdges * st2; i += kThreads) G2[i] = 0.f;
        __syncthreads();
        int step = 0;
        for (int r = 0; r < n_paths; ++r) {
            const uint32_t* rec = recs + kUvwRec * r;
            if (static_cast<int>(rec[4] & 0xffffu) != o2b) continue;  // into another block of x2
            const int p = static_cast<int>(rec[0]), d3 = static_cast<int>(rec[1]);
            const int o1 = static_cast<int>(rec[3] & 0xffffu), d1 = static_cast<int>(rec[3] >> 16);
            const int o3 = static_cast<int>(rec[5] & 0xffffu);
            const float* __restrict__ wp = wt + static_cast<int64_t>(p) * UVW + static_cast<int64_t>(v) * W;
            for (int m0 = 0; m0 < d3; m0 += kUvwChunk, ++step) {
                const int mc = d3 - m0 < kUvwChunk ? d3 - m0 : kUvwChunk;
                float* Zw = Zb + ((step & 1) * 4 + wave) * zs;
                bool first = true;
                for (int ub = 32 * wave; ub < U; ub += 128) {
                    // gR for u = ub .. ub + 31 (rows) and the tile's edges (columns)
                    v16f acc[kUvwChunk];
#pragma unroll
                    for (int j = 0; j < kUvwChunk; ++j) acc[j] = v16f{};
                    const int ua = ub + el;
                    for (int s2 = 0; s2 < W; s2 += 2) {
                        const int wv = s2 + half;
                        const float av = (ua < U && wv < W) ? wp[static_cast<int64_t>(ua) * V * W + wv] : 0.f;
                        const float* gb = g + (n * W + wv) * nco + o3 + m0;
                        const bool b_ok = n_ok && wv < W;
#pragma unroll
                        for (int j = 0; j < kUvwChunk; ++j)
                            if (j < mc) acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, b_ok ? gb[j] : 0.f, acc[j], 0, 0, 0);
                    }
                    // accumulator element i: u = ub + 8 (i / 4) + 4 half + i % 4, edge el
                    for (int k1 = 0; k1 < d1; ++k1) {
                        float xv[16];
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            const int u = ub + 8 * (i >> 2) + 4 * half + (i & 3);
                            xv[i] = (n_ok && u < U) ? x1[(n * U + u) * nc1 + o1 + k1] : 0.f;
                        }
#pragma unroll
                        for (int j = 0; j < kUvwChunk; ++j) {
                            if (j >= mc) break;
                            float z = 0.f;
#pragma unroll
                            for (int i = 0; i < 16; ++i) z = fmaf(xv[i], acc[j][i], z);
                            z += __shfl_xor(z, 32);
                            float* zp = Zw + (el * d1max + k1) * kUvwChunk + j;
                            if (half == 0) *zp = first ? z : *zp + z;
                        }
                    }
                    first = false;
                }
                if (first && half == 0) {  // no u block for this wave: a zero partial
                    for (int k1 = 0; k1 < d1; ++k1)
                        for (int j = 0; j < mc; ++j) Zw[(el * d1max + k1) * kUvwChunk + j] = 0.f;
                }
                __syncthreads();  // the item's four partials are in LDS
                if (wave == 0 && half == 0) {
                    const float* Zi = Zb + (step & 1) * 4 * zs + el * d1max * kUvwChunk;
                    const uint32_t* csr = tab + rec[2] + m0;
                    float* grow = G2 + el * st2;
                    for (int j = 0; j < mc; ++j)
                        for (uint32_t k = csr[j]; k < csr[j + 1]; ++k) {
                            const uint32_t ix = ent[2 * k];
                            const int z_at = static_cast<int>((ix & 0xffffu) - o1) * kUvwChunk + j;
                            const float z = ((Zi[z_at] + Zi[zs + z_at]) + Zi[2 * zs + z_at]) + Zi[3 * zs + z_at];
                            float* gq = grow + (static_cast<int>(ix >> 16) - o2b);
                            *gq = fmaf(__uint_as_float(ent[2 * k + 1]), z, *gq);
                        }
                }
            }
        }
        __syncthreads();  // wave 0's last scatter is done
        for (int i = tid; i < kEdges * d2b; i += kThreads) {
            const int e = i / d2b, c = i - e * d2b;
            if (e0 + e < N) gx2[((e0 + e) * V + v) * nc2 + o2b + c] = G2[e * st2 + c];
        }
        __syncthreads();  // the tile is read before the next v clears it
    }
}

hipError_t fill_zero(float* out, int64_t total, hipStream_t stream) {
    if (total <= 0) return hipSuccess;
    const int64_t want = (total / 4 + kThreads - 1) / kThreads;
    const unsigned g = static_cast<unsigned>(want < 4096 ? (want < 1 ? 1 : want) : 4096);
    hipLaunchKernelGGL(spingtp_fill_zero_kernel, dim3(g), dim3(kThreads), 0, stream, out, total);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_uvw_mix(const float* xa, const float* xb, const float* w, float* out, int64_t N, int A, int B, int O,
                          int64_t sa, int64_t sb, int64_t so, int64_t ps, const uint32_t* table, int n_blocks,
                          int max_d3, int nco, hipStream_t stream) {
    const hipError_t e = fill_zero(out, N * O * nco, stream);
    if (e != hipSuccess) return e;
    if (N == 0 || A == 0 || B == 0 || O == 0 || n_blocks == 0) return hipSuccess;
    const int64_t gx = (N + kEdges - 1) / kEdges;
    const int64_t groups = (O + kGroupW - 1) / kGroupW;
    // One output component per workgroup: each forms R of its own component only, so only
    // the weight reads repeat.  That pays wherever the weights of consecutive output
    // channels are adjacent (so = 1, the forward: 1.6-2.2x faster on the App. E.2 shapes and
    // still 1.6x at 16,384 edges), and for the strided weight reads of the gradient roles
    // only in launches of fewer than kSmallGrid workgroups (measured: B = 1024 1.45x faster,
    // B = 4096 1.24x slower).
    const bool small = so == 1 || gx * n_blocks * groups * ((max_d3 + kUvwChunk - 1) / kUvwChunk) < kSmallGrid;
    const int ch = small ? kSmallChunk : kUvwChunk;
    const int n_chunks = (max_d3 + ch - 1) / ch;
    const int64_t gz = groups * n_chunks;
    if (gx > 0x7fffffff || n_blocks > 65535 || gz > 65535) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(gx), static_cast<unsigned>(n_blocks), static_cast<unsigned>(gz));
    if (small)
        hipLaunchKernelGGL(spingtp_uvw_mix_kernel<kSmallChunk>, grid, dim3(kThreads), 0, stream, xa, xb, w, out, N, A,
                           B, O, sa, sb, so, ps, table, n_chunks, nco);
    else
        hipLaunchKernelGGL(spingtp_uvw_mix_kernel<kUvwChunk>, grid, dim3(kThreads), 0, stream, xa, xb, w, out, N, A,
                           B, O, sa, sb, so, ps, table, n_chunks, nco);
    return hipGetLastError();
}

hipError_t launch_fwd_uvw(const float* x1, const float* x2, const float* w, float* out, int64_t N, int U, int V,
                          int W, const uint32_t* table, int n_blocks, int max_d3, int nco, hipStream_t stream) {
    // pairs (u, v), output channels w: W[p][u][v][w] at u V W + v W + w
    return launch_uvw_mix(x1, x2, w, out, N, U, V, W, static_cast<int64_t>(V) * W, W, 1,
                          static_cast<int64_t>(U) * V * W, table, n_blocks, max_d3, nco, stream);
}

hipError_t launch_uvw_grad_w(const float* x1, const float* x2, const float* g, float* gw, int64_t N, int U, int V,
                             int W, const uint32_t* table, int n_paths, int nco, hipStream_t stream) {
    if (n_paths == 0 || U == 0 || V == 0 || W == 0) return hipSuccess;
    const int64_t gy = (static_cast<int64_t>(U) * V + kPairs - 1) / kPairs;
    const int64_t gz = (W + kGroupW - 1) / kGroupW;
    if (gy > 65535 || gz > 65535) return hipErrorInvalidValue;
    hipLaunchKernelGGL(spingtp_uvw_grad_w_kernel, dim3(static_cast<unsigned>(n_paths), static_cast<unsigned>(gy),
                                                        static_cast<unsigned>(gz)),
                       dim3(kThreads), 0, stream, x1, x2, g, gw, N, U, V, W, table, nco);
    return hipGetLastError();
}

size_t uvw_grad_x2_lds(int d1max, int d2max) {
    const size_t bytes = (static_cast<size_t>(8) * kEdges * d1max * kUvwChunk + kEdges * (d2max | 1)) * sizeof(float);
    return bytes <= 160 * 1024 ? bytes : 0;
}

hipError_t launch_uvw_grad_x2(const float* x1, const float* g, const float* w, float* gx2, int64_t N, int U, int V,
                              int W, const uint32_t* table, const uint32_t* table2, int n_blocks2, int n_paths,
                              int nc1, int nc2, int nco, int d1max, int d2max, hipStream_t stream) {
    // slots of blocks that no path reaches (and l < |s|) stay 0
    const hipError_t e = fill_zero(gx2, N * V * nc2, stream);
    if (e != hipSuccess) return e;
    if (N == 0 || V == 0 || U == 0 || W == 0 || n_paths == 0 || n_blocks2 == 0) return hipSuccess;
    const size_t lds = uvw_grad_x2_lds(d1max, d2max);
    const int64_t gx = (N + kEdges - 1) / kEdges;
    if (lds == 0 || gx > 0x7fffffff || n_blocks2 > 65535) return hipErrorInvalidValue;
    const unsigned gz = static_cast<unsigned>(V < 65535 ? V : 65535);
    hipLaunchKernelGGL(spingtp_uvw_grad_x2_kernel,
                       dim3(static_cast<unsigned>(gx), static_cast<unsigned>(n_blocks2), gz), dim3(kThreads), lds,
                       stream, x1, g, w, gx2, N, U, V, W, table, table2, n_paths, nc1, nc2, nco, d1max, d2max);
    return hipGetLastError();
}

}  // namespace spingtp

namespace {

bool misaligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) != 0; }

}  // namespace

extern "C" spingtp_status spingtp_forward_fully_connected(spingtp_plan plan, const void* x1, const void* x2,
                                                          const float* weights, void* out, int64_t N, int64_t U,
                                                          int64_t V, int64_t W, void* stream) {
    if (plan == nullptr || N < 0 || U < 0 || V < 0 || W < 0) return SPINGTP_ERR_INVALID_ARG;
    if (plan->d_uvw == nullptr || plan->dtype != SPINGTP_FP32) return SPINGTP_ERR_UNSUPPORTED;
    if (U > 65536 || V > 65536 || W > 65536 || U * V > (int64_t{1} << 24)) return SPINGTP_ERR_INVALID_ARG;
    const int64_t nco = static_cast<int64_t>(plan->n_spins) * (plan->LO + 1) * (plan->LO + 1);
    if (N == 0 || W == 0) return SPINGTP_OK;
    if (N > (int64_t{1} << 40) / (W * nco)) return SPINGTP_ERR_INVALID_ARG;
    if (out == nullptr || misaligned(out, 16)) return SPINGTP_ERR_INVALID_ARG;
    if (U > 0 && V > 0 && (x1 == nullptr || x2 == nullptr || weights == nullptr || misaligned(x1, 16) ||
                           misaligned(x2, 16) || misaligned(weights, 4)))
        return SPINGTP_ERR_INVALID_ARG;
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return SPINGTP_ERR_HIP;
    if (cur != plan->device) return SPINGTP_ERR_INVALID_ARG;
    const hipError_t e = spingtp::launch_fwd_uvw(
        static_cast<const float*>(x1), static_cast<const float*>(x2), weights, static_cast<float*>(out), N,
        static_cast<int>(U), static_cast<int>(V), static_cast<int>(W), plan->d_uvw + plan->uvw_off[0],
        plan->uvw_blocks[0], plan->uvw_max_d3[0], static_cast<int>(nco), static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SPINGTP_OK : SPINGTP_ERR_HIP;
}

extern "C" spingtp_status spingtp_backward_fully_connected(spingtp_plan plan, const void* x1, const void* x2,
                                                           const float* weights, const void* grad_out,
                                                           void* grad_x1, void* grad_x2, float* grad_weights,
                                                           int64_t N, int64_t U, int64_t V, int64_t W, void* stream) {
    if (plan == nullptr || N < 0 || U < 0 || V < 0 || W < 0) return SPINGTP_ERR_INVALID_ARG;
    if (plan->d_uvw == nullptr || plan->dtype != SPINGTP_FP32) return SPINGTP_ERR_UNSUPPORTED;
    const int64_t lim = int64_t{1} << 24;
    if (U > 65536 || V > 65536 || W > 65536 || U * V > lim || V * W > lim || U * W > lim)
        return SPINGTP_ERR_INVALID_ARG;
    const int64_t nc1 = static_cast<int64_t>(plan->n_spins) * (plan->L1 + 1) * (plan->L1 + 1);
    const int64_t nc2 = static_cast<int64_t>(plan->n_spins) * (plan->L2 + 1) * (plan->L2 + 1);
    const int64_t nco = static_cast<int64_t>(plan->n_spins) * (plan->LO + 1) * (plan->LO + 1);
    const int64_t widest = nc1 > nc2 ? (nc1 > nco ? nc1 : nco) : (nc2 > nco ? nc2 : nco);
    const int64_t chans = U > V ? (U > W ? U : W) : (V > W ? V : W);
    if (chans > 0 && N > (int64_t{1} << 40) / (chans * widest)) return SPINGTP_ERR_INVALID_ARG;
    // every array that a requested gradient reads or writes
    const bool want1 = grad_x1 != nullptr && N * U > 0, want2 = grad_x2 != nullptr && N * V > 0;
    const bool wantw = grad_weights != nullptr && U * V * W > 0;
    const bool rows = N > 0 && U * V * W > 0;  // the products touch the inputs at all
    if (want2 && spingtp::uvw_grad_x2_lds(2 * plan->L1 + 1, 2 * plan->L2 + 1) == 0)
        return SPINGTP_ERR_UNSUPPORTED;  // its LDS tiles exceed a CU's 160 KB
    if ((want1 && misaligned(grad_x1, 16)) || (want2 && misaligned(grad_x2, 16)) ||
        (wantw && misaligned(grad_weights, 4)))
        return SPINGTP_ERR_INVALID_ARG;
    if (rows && (want1 || want2 || wantw) &&
        (x1 == nullptr || x2 == nullptr || grad_out == nullptr || misaligned(x1, 16) || misaligned(x2, 16) ||
         misaligned(grad_out, 16) || ((want1 || want2) && (weights == nullptr || misaligned(weights, 4)))))
        return SPINGTP_ERR_INVALID_ARG;
    if (!want1 && !want2 && !wantw) return SPINGTP_OK;
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return SPINGTP_ERR_HIP;
    if (cur != plan->device) return SPINGTP_ERR_INVALID_ARG;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    const float* a1 = static_cast<const float*>(x1);
    const float* a2 = static_cast<const float*>(x2);
    const float* g = static_cast<const float*>(grad_out);
    const int u = static_cast<int>(U), v = static_cast<int>(V), w = static_cast<int>(W);
    const int64_t ps = U * V * W;
    hipError_t e = hipSuccess;
    if (want1)  // pairs (v, w) of x2 and grad_out, output channels u
        e = spingtp::launch_uvw_mix(a2, g, weights, static_cast<float*>(grad_x1), N, v, w, u, W, 1, V * W, ps,
                                    plan->d_uvw + plan->uvw_off[1], rows ? plan->uvw_blocks[1] : 0,
                                    plan->uvw_max_d3[1], static_cast<int>(nc1), s);
    if (e == hipSuccess && want2)  // through gR_p = W_p g, then x1 and the entries
        e = spingtp::launch_uvw_grad_x2(a1, g, weights, static_cast<float*>(grad_x2), N, u, v, w, plan->d_uvw,
                                        plan->d_uvw + plan->uvw_off[2], plan->uvw_blocks[2], rows ? plan->uvw_paths : 0,
                                        static_cast<int>(nc1), static_cast<int>(nc2), static_cast<int>(nco),
                                        2 * plan->L1 + 1, 2 * plan->L2 + 1, s);
    if (e == hipSuccess && wantw)
        e = spingtp::launch_uvw_grad_w(a1, a2, g, grad_weights, N, u, v, w, plan->d_uvw + plan->uvw_off[0],
                                       plan->uvw_paths, static_cast<int>(nco), s);
    return e == hipSuccess ? SPINGTP_OK : SPINGTP_ERR_HIP;
}
