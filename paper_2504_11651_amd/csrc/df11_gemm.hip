// Matrix products of a decompressed transformer block on the gfx950 matrix
// cores: y[m] = x[m] * W_m^T for the block's matrices, BF16 inputs, fp32
// accumulation (the consumer of the decoded weights in Sec. 2.3.3; the
// batch-size experiments of Sec. 3 time decompression plus these products).
//
// With at most 64 activation rows the products are bound by streaming the
// weights from HBM, so the design reads every weight once, with 16-byte
// loads, and keeps several kilobytes in flight per wave:
//   - one wavefront computes a tile of 16 output features x all tokens over a
//     contiguous range of k; all matrices of the block share one launch;
//   - per 64 k a lane feeds 2 x 8 BF16 of one weight row (lanes 16g..16g+15
//     take rows 0..15 at k offset 16g) and the matching activations to
//     v_mfma_f32_16x16x32_bf16, twice per 16-token slice; A (tokens) and B
//     (features) use the same assignment of k to lanes, so the dot products
//     cover each k once whatever order the unit sums in;
//   - up to 3 tokens each wave loads its weights straight into that layout
//     and reads its activations from memory; from 4, a workgroup of 4 waves
//     stages each 256-k activation slab in LDS once, and each wave passes
//     its weights through LDS so that every load reads whole cache lines;
//   - a matrix is split into k ranges of about 1024 columns (up to 8
//     tokens) or 4096 columns, or half that where it evens out the work per
//     CU (more tokens); each range of a split matrix writes fp32 partial
//     sums, and a second kernel adds them in a fixed order, so results are
//     deterministic (no atomics).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <vector>

#include "df11.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr uint32_t kTileRows = 16;   // output features per wave
constexpr uint32_t kKStep = 64;      // k per inner step: two MFMAs
constexpr uint32_t kUnroll = 4;      // inner steps whose weight loads are issued together
constexpr uint32_t kKPerIter = kKStep * kUnroll;
// k range of one wave before a matrix is split: short ranges (more
// workgroups in flight) pay off while the products are light; from 9
// tokens the products per weight favour long ranges (whose weights pass
// through LDS), and the split is chosen to balance the CUs
constexpr uint32_t kKTargetFew = 1024;
constexpr uint32_t kKTargetMany = 4096;
constexpr uint32_t kFewTokens = 8;
constexpr uint32_t kSlabMinTokens = 4;  // fewer tokens: activations straight from memory
constexpr uint32_t kWaves = 4;       // waves per workgroup, up to 3 tokens
constexpr uint32_t kSlabWaves = 4;   // waves per workgroup sharing one activation slab
constexpr uint32_t kMax = DF11_MAX_MATRICES;

struct GemmArgs {
    const uint16_t *w;
    float *part;
    uint32_t n_mats;
    uint32_t tokens;
    uint32_t num_tiles;
    uint32_t num_wg;
    uint32_t tile_start[kMax + 1];  // prefix sums of 16-feature tiles per matrix
    uint32_t wg_start[kMax + 1];    // prefix sums of 64-feature workgroup tiles
    uint32_t ksplit[kMax];          // k ranges per matrix
    uint32_t kchunk[kMax];          // k per range (multiple of kKPerIter)
    uint32_t rows[kMax];
    uint32_t cols[kMax];
    uint64_t w_off[kMax];           // weights
    uint64_t part_off[kMax];        // floats (split matrices only)
    const uint16_t *x[kMax];
    float *y[kMax];
};

struct ReduceArgs {
    const float *part;
    uint32_t n_mats;
    uint32_t tokens;
    uint32_t total;                 // outputs of all split matrices
    uint32_t out_start[kMax + 1];   // prefix sums of tokens*rows over split matrices
    uint32_t ksplit[kMax];
    uint32_t rows[kMax];
    uint64_t part_off[kMax];
    float *y[kMax];
};

__device__ __forceinline__ uint32_t umin(uint32_t a, uint32_t b) { return a < b ? a : b; }

__device__ __forceinline__ uint4 load16(const uint16_t *p) {
    return *reinterpret_cast<const uint4 *>(p);
}

__device__ __forceinline__ uint4 masked(uint4 v, uint32_t m) {
    return make_uint4(v.x & m, v.y & m, v.z & m, v.w & m);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

struct Mat {
    uint32_t ksplit, kchunk, rows, cols;
    uint64_t w_off, part_off;
    const uint16_t *x;
    float *y;
};

// Matrix whose work items [start[i], start[i+1]) contain idx (uniform;
// constant-index selects keep the kernel arguments in scalar registers).
__device__ __forceinline__ Mat select_matrix(const GemmArgs &a, const uint32_t (&start)[kMax + 1],
                                             uint32_t idx, uint32_t *first) {
    Mat m{1, 0, 0, 0, 0, 0, nullptr, nullptr};
    *first = 0;
#pragma unroll
    for (uint32_t i = 0; i < kMax; ++i) {
        if (i < a.n_mats && idx >= start[i]) {
            *first = start[i];
            m.ksplit = a.ksplit[i];
            m.kchunk = a.kchunk[i];
            m.rows = a.rows[i];
            m.cols = a.cols[i];
            m.w_off = a.w_off[i];
            m.part_off = a.part_off[i];
            m.x = a.x[i];
            m.y = a.y[i];
        }
    }
    return m;
}

// acc[mt][r] holds the sum over k range s for token 16*mt + 4*g + r and
// feature 16*rb + j: written to y, or to the partial sums of a split matrix.
template <uint32_t MT>
__device__ __forceinline__ void write_tile(const GemmArgs &a, const Mat &m, uint32_t rb, uint32_t s,
                                           uint32_t j, uint32_t g, const f32x4 (&acc)[MT]) {
    const uint32_t feature = rb * kTileRows + j;
#pragma unroll
    for (uint32_t mt = 0; mt < MT; ++mt) {
#pragma unroll
        for (uint32_t r = 0; r < 4; ++r) {
            const uint32_t t = mt * 16u + 4u * g + r;
            if (t >= a.tokens) continue;
            if (m.ksplit == 1) {
                m.y[static_cast<uint64_t>(t) * m.rows + feature] = acc[mt][r];
            } else {
                const uint64_t idx = m.part_off +
                    (static_cast<uint64_t>(rb * m.ksplit + s) * a.tokens + t) * kTileRows + j;
                a.part[idx] = acc[mt][r];
            }
        }
    }
}

// k assignment (the same for both operands): in the 64-k step at kk, MFMA
// half h gives lane group g the 8 values kk + 32h + 8g .. +7, so the four
// lanes of one row read 64 contiguous bytes per load.

// Up to 3 tokens: one wavefront per 16-feature tile, activations read
// straight from memory (a few hundred bytes per k range, cache resident).
__global__ __launch_bounds__(64 * kWaves) void gemm_tiles_kernel(GemmArgs a) {
    const uint32_t lane = threadIdx.x & 63u;
    const uint32_t tile =
        blockIdx.x * kWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (tile >= a.num_tiles) return;
    uint32_t first;
    const Mat m = select_matrix(a, a.tile_start, tile, &first);
    const uint32_t local = tile - first;
    const uint32_t rb = local / m.ksplit;
    const uint32_t s = local - rb * m.ksplit;
    const uint32_t k0 = s * m.kchunk;
    const uint32_t k1 = umin(m.cols, k0 + m.kchunk);

    const uint32_t j = lane & 15u;   // feature row (B) / token row (A) in the slice
    const uint32_t g = lane >> 4;    // k group
    const uint16_t *wrow = a.w + m.w_off + static_cast<uint64_t>(rb * kTileRows + j) * m.cols + 8u * g;
    // rows of x past the last token read token 0 and are masked to zero
    const uint32_t xmask = j < a.tokens ? ~0u : 0u;
    const uint16_t *xrow = m.x + static_cast<uint64_t>(j < a.tokens ? j : 0u) * m.cols + 8u * g;

    f32x4 acc[1] = {f32x4{0.f, 0.f, 0.f, 0.f}};
    auto step = [&](uint32_t kk, uint4 w0, uint4 w1) {
        const uint4 x0 = masked(load16(xrow + kk), xmask);
        const uint4 x1 = masked(load16(xrow + kk + 32u), xmask);
        acc[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(x0), as_bf16x8(w0), acc[0], 0, 0, 0);
        acc[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(x1), as_bf16x8(w1), acc[0], 0, 0, 0);
    };
    uint32_t k = k0;
    for (; k + kKPerIter <= k1; k += kKPerIter) {
        // the weight loads of kUnroll steps are issued before their products
        uint4 W[kUnroll][2];
#pragma unroll
        for (uint32_t u = 0; u < kUnroll; ++u) {
            W[u][0] = load16(wrow + k + u * kKStep);
            W[u][1] = load16(wrow + k + u * kKStep + 32u);
        }
#pragma unroll
        for (uint32_t u = 0; u < kUnroll; ++u) step(k + u * kKStep, W[u][0], W[u][1]);
    }
    for (; k < k1; k += kKStep) step(k, load16(wrow + k), load16(wrow + k + 32u));
    write_tile<1>(a, m, rb, s, j, g, acc);
}

// Four or more tokens: a workgroup of kSlabWaves waves covers 16*kSlabWaves features
// over one k range and stages the activations of each 256-k slab in LDS once
// for all its waves (rows padded by 16 bytes so the 16 lanes of one read
// pass hit distinct banks).
// Each wave's weights pass through 8 KB of LDS of its own: a load
// instruction reads 512 contiguous bytes of each of two rows (8 whole cache
// lines) rather than 64 bytes of each of 16 rows, which streams the
// 4096-column matrices about a tenth faster; written with row r's 16-byte
// piece p at slot (p + r) mod 32, the slab is read back in the matrix-core
// layout without bank conflicts.  Only the wave that writes a weight slab
// reads it, and one wave's LDS accesses complete in order, so the weights
// need no barrier.
constexpr uint32_t kSlabK = kKPerIter;              // k per staged slab
constexpr uint32_t kSlabStride = kSlabK * 2 + 16;   // bytes per token row in LDS
constexpr uint32_t kWaveW = kTileRows * kSlabK * 2; // bytes of one wave's weight slab

// LDS of one workgroup, and the waves per SIMD it leaves room for (at most
// 4): the register hint asks for exactly that many
template <uint32_t MT>
constexpr uint32_t kSlabLds = 16 * MT * kSlabStride + kSlabWaves * kWaveW;
template <uint32_t MT>
constexpr uint32_t kSlabOcc = 160u * 1024u / kSlabLds<MT> < 4u ? 160u * 1024u / kSlabLds<MT> : 4u;

template <uint32_t MT>
__global__ __launch_bounds__(64 * kSlabWaves) __attribute__((amdgpu_waves_per_eu(kSlabOcc<MT>))) void
gemm_slab_kernel(GemmArgs a) {
    __shared__ __attribute__((aligned(16))) uint8_t slab[kSlabLds<MT>];
    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63u;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t wgt = blockIdx.x;  // < num_wg by the grid size
    uint32_t first;
    const Mat m = select_matrix(a, a.wg_start, wgt, &first);
    const uint32_t local = wgt - first;
    const uint32_t rbw = local / m.ksplit;        // 64-feature block
    const uint32_t s = local - rbw * m.ksplit;
    const uint32_t k0 = s * m.kchunk;
    const uint32_t k1 = umin(m.cols, k0 + m.kchunk);
    const uint32_t rb = rbw * kSlabWaves + wave;       // this wave's 16-feature tile
    const bool active = rb * kTileRows < m.rows;   // uniform

    const uint32_t j = lane & 15u;
    const uint32_t g = lane >> 4;

    // slab loading: 16-byte piece q = tid + 64*kSlabWaves*i covers token
    // q / kRowPieces, k offset 8 * (q % kRowPieces) of the slab
    constexpr uint32_t kRowPieces = kSlabK / 8u;
    constexpr uint32_t kPieces = 16u * MT * kRowPieces;
    constexpr uint32_t kPer = kPieces / (64u * kSlabWaves);
    static_assert(kPieces % (64u * kSlabWaves) == 0, "whole pieces per thread");
    // Inside the loop every slab has a next one: its activations are
    // requested first, and each weight register's next load right after the
    // register is written to LDS, so a slab of weights stays in flight;
    // loads complete in order, so the wait for one load never waits for
    // loads issued after it.  Activations are masked when staged, not when
    // they arrive (a use on arrival would wait for every older load).
    uint4 xr[kPer];
    auto slab_piece = [&](uint32_t i, uint32_t k, uint32_t *t, uint32_t *kk) {
        const uint32_t q = tid + 64u * kSlabWaves * i;
        *t = q / kRowPieces;
        *kk = k + 8u * (q % kRowPieces);
        return *t < a.tokens && *kk < k1;
    };
    auto load_slab = [&](uint32_t k) {
#pragma unroll
        for (uint32_t i = 0; i < kPer; ++i) {
            uint32_t t, kk;
            const bool ok = slab_piece(i, k, &t, &kk);
            xr[i] = load16(m.x + static_cast<uint64_t>(ok ? t : 0u) * m.cols + (ok ? kk : k0));
        }
    };
    auto store_slab = [&](uint32_t k) {
#pragma unroll
        for (uint32_t i = 0; i < kPer; ++i) {
            uint32_t t, kk;
            const bool ok = slab_piece(i, k, &t, &kk);
            const uint32_t q = tid + 64u * kSlabWaves * i;
            *reinterpret_cast<uint4 *>(slab + (q / kRowPieces) * kSlabStride + 16u * (q % kRowPieces)) =
                masked(xr[i], ok ? ~0u : 0u);
        }
    };
    // weights: load i of a slab reads rows 2i and 2i+1 of the tile (lane:
    // row 2i + lane/32, 16-byte piece lane%32 of the slab; pieces past the
    // range repeat its last piece).  A plain vector type keeps the eight
    // registers out of private memory.
    typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
    u32x4v W[8];
    u32x4v *wl = reinterpret_cast<u32x4v *>(slab + 16 * MT * kSlabStride + wave * kWaveW);
    const uint32_t half = lane >> 5, pl = lane & 31u;
    const uint16_t *wrow2 =
        a.w + m.w_off + static_cast<uint64_t>(active ? rb * kTileRows + half : 0u) * m.cols;
    auto load_w = [&](uint32_t i, uint32_t k) {
        const uint32_t p = umin(pl, umin(32u, (k1 - k) / 8u) - 1u);
        W[i] = *reinterpret_cast<const u32x4v *>(wrow2 + static_cast<uint64_t>(2u * i) * m.cols + k + 8u * p);
    };
    auto put_w = [&](uint32_t i) {
        const uint32_t r = 2u * i + half;
        wl[r * 32u + ((pl + r) & 31u)] = W[i];
    };
    f32x4 acc[MT];
#pragma unroll
    for (uint32_t mt = 0; mt < MT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    auto products = [&](uint32_t u) {
#pragma unroll
        for (uint32_t mt = 0; mt < MT; ++mt) {
            const uint8_t *row = slab + (16u * mt + j) * kSlabStride + 2u * (kKStep * u + 8u * g);
            const uint4 x0 = *reinterpret_cast<const uint4 *>(row);
            const uint4 x1 = *reinterpret_cast<const uint4 *>(row + 64u);
            const u32x4v w0 = wl[j * 32u + ((8u * u + g + j) & 31u)];
            const u32x4v w1 = wl[j * 32u + ((8u * u + 4u + g + j) & 31u)];
            acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(x0), __builtin_bit_cast(bf16x8, w0),
                                                              acc[mt], 0, 0, 0);
            acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(x1), __builtin_bit_cast(bf16x8, w1),
                                                              acc[mt], 0, 0, 0);
        }
    };

#pragma unroll
    for (uint32_t i = 0; i < 8; ++i) load_w(i, k0);
    load_slab(k0);
    store_slab(k0);
    __syncthreads();
    uint32_t k = k0;
    for (; k + kSlabK < k1; k += kSlabK) {
        const uint32_t kn = k + kSlabK;
        load_slab(kn);
        // each weight register takes the next slab's load as soon as it is
        // in LDS (kept in this order: hoisting the loads would make the
        // compiler copy registers, and each copy waits for its load)
#pragma unroll
        for (uint32_t i = 0; i < 8; ++i) {
            put_w(i);
            __builtin_amdgcn_sched_barrier(0);
            load_w(i, kn);
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (uint32_t u = 0; u < kUnroll; ++u)
            if (active) products(u);
        __syncthreads();  // every wave is done with this slab
        store_slab(kn);
        __syncthreads();
    }
    // the last slab of the range
    const uint32_t steps = umin(kUnroll, (k1 - k) / kKStep);  // uniform
#pragma unroll
    for (uint32_t i = 0; i < 8; ++i) put_w(i);
#pragma unroll
    for (uint32_t u = 0; u < kUnroll; ++u)
        if (active && u < steps) products(u);
    if (active) write_tile<MT>(a, m, rb, s, j, g, acc);
}

// y[t][f] = sum over k ranges s = 0, 1, ... of the partial sums, in that order.
__global__ __launch_bounds__(256) void gemm_reduce_kernel(ReduceArgs a) {
    const uint32_t i = blockIdx.x * 256u + threadIdx.x;
    if (i >= a.total) return;
    uint32_t m = 0;
#pragma unroll
    for (uint32_t q = 1; q < kMax; ++q)
        if (q < a.n_mats && i >= a.out_start[q]) m = q;
    uint32_t start = 0, ksplit = 1, rows = 1;
    uint64_t part_off = 0;
    float *y = nullptr;
#pragma unroll
    for (uint32_t q = 0; q < kMax; ++q) {
        if (q == m) {
            start = a.out_start[q];
            ksplit = a.ksplit[q];
            rows = a.rows[q];
            part_off = a.part_off[q];
            y = a.y[q];
        }
    }
    const uint32_t local = i - start;
    const uint32_t t = local / rows;
    const uint32_t f = local - t * rows;
    const uint32_t rb = f / kTileRows;
    const uint32_t j = f - rb * kTileRows;
    float sum = 0.f;
    for (uint32_t s = 0; s < ksplit; ++s)
        sum += a.part[part_off + (static_cast<uint64_t>(rb * ksplit + s) * a.tokens + t) * kTileRows + j];
    y[static_cast<uint64_t>(t) * rows + f] = sum;
}

// Split of one matrix into about ks_req k ranges, each a whole number of
// slabs (kKPerIter) except the last.
void split_into(uint32_t cols, uint32_t ks_req, uint32_t *ksplit, uint32_t *kchunk) {
    uint32_t kc = (cols + ks_req - 1) / ks_req;
    kc = (kc + kKPerIter - 1) / kKPerIter * kKPerIter;
    *kchunk = kc;
    *ksplit = (cols + kc - 1) / kc;  // no empty range
}

uint32_t base_ranges(uint32_t cols, uint32_t tokens) {
    const uint32_t target = tokens <= kFewTokens ? kKTargetFew : kKTargetMany;
    const uint32_t ks = (cols + target - 1) / target;
    return ks ? ks : 1u;
}

// Estimated bytes moved by the busiest CU for one choice of k ranges per
// matrix: workgroup i runs on CU i mod cus (with many tokens every
// workgroup of the launch is resident at once), moving its weights and,
// for a split matrix, writing its partial sums; the reduce kernel's traffic
// is spread over all CUs.
uint64_t split_cost(const df11_matrix *mats, uint32_t n_mats, uint32_t tokens, uint32_t cus,
                    const uint32_t *ks_req, std::vector<uint64_t> &load) {
    load.assign(cus, 0);
    uint64_t wg = 0, reduce = 0;
    for (uint32_t m = 0; m < n_mats; ++m) {
        uint32_t ks, kc;
        split_into(mats[m].cols, ks_req[m], &ks, &kc);
        const uint32_t rows = mats[m].rows, cols = mats[m].cols;
        for (uint32_t r0 = 0; r0 < rows; r0 += kTileRows * kSlabWaves) {
            const uint64_t nr = rows - r0 < kTileRows * kSlabWaves ? rows - r0 : kTileRows * kSlabWaves;
            for (uint32_t s = 0; s < ks; ++s) {
                const uint64_t len = cols - s * kc < kc ? cols - s * kc : kc;
                load[wg++ % cus] += 2 * nr * len + (ks > 1 ? 4 * nr * tokens : 0);
            }
        }
        if (ks > 1) reduce += 4ull * rows * tokens * (ks + 1);
    }
    uint64_t most = 0;
    for (uint64_t l : load) most = l > most ? l : most;
    return most + reduce / cus;
}

// With many tokens the products per weight are heavy enough that the CU
// holding the most work sets the time: of the choices of 1x or 2x the base
// number of k ranges per matrix, take the one whose busiest CU moves the
// fewest bytes (ties: fewer workgroups).  Cached per device and shapes.
struct SplitEntry {
    int dev;
    uint32_t tokens, n_mats, rows[kMax], cols[kMax], ks_req[kMax];
};
std::mutex g_split_mu;
std::vector<SplitEntry> g_splits;
constexpr size_t kMaxSplits = 64;

int choose_ranges(const df11_matrix *mats, uint32_t n_mats, uint32_t tokens, uint32_t *ks_req) {
    for (uint32_t m = 0; m < n_mats; ++m) ks_req[m] = base_ranges(mats[m].cols, tokens);
    if (tokens <= kFewTokens) return DF11_OK;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return DF11_E_HIP;
    std::lock_guard<std::mutex> lk(g_split_mu);
    for (const SplitEntry &e : g_splits) {
        bool same = e.dev == dev && e.tokens == tokens && e.n_mats == n_mats;
        for (uint32_t m = 0; same && m < n_mats; ++m)
            same = e.rows[m] == mats[m].rows && e.cols[m] == mats[m].cols;
        if (same) {
            for (uint32_t m = 0; m < n_mats; ++m) ks_req[m] = e.ks_req[m];
            return DF11_OK;
        }
    }
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
        return DF11_E_HIP;
    uint32_t base[kMax], trial[kMax], best_mask = 0;
    for (uint32_t m = 0; m < n_mats; ++m) base[m] = ks_req[m];
    std::vector<uint64_t> load;
    uint64_t best = ~0ull, best_wg = ~0ull;
    for (uint32_t mask = 0; mask < (1u << n_mats); ++mask) {
        uint64_t wg = 0;
        for (uint32_t m = 0; m < n_mats; ++m) {
            trial[m] = base[m] << ((mask >> m) & 1u);
            uint32_t ks, kc;
            split_into(mats[m].cols, trial[m], &ks, &kc);
            wg += uint64_t{(mats[m].rows + kTileRows * kSlabWaves - 1) / (kTileRows * kSlabWaves)} * ks;
        }
        const uint64_t c = split_cost(mats, n_mats, tokens, static_cast<uint32_t>(cus), trial, load);
        if (c < best || (c == best && wg < best_wg)) {
            best = c;
            best_wg = wg;
            best_mask = mask;
        }
    }
    SplitEntry e{};
    e.dev = dev;
    e.tokens = tokens;
    e.n_mats = n_mats;
    for (uint32_t m = 0; m < n_mats; ++m) {
        ks_req[m] = base[m] << ((best_mask >> m) & 1u);
        e.rows[m] = mats[m].rows;
        e.cols[m] = mats[m].cols;
        e.ks_req[m] = ks_req[m];
    }
    if (g_splits.size() >= kMaxSplits) g_splits.erase(g_splits.begin());  // oldest goes first
    g_splits.push_back(e);
    return DF11_OK;
}

int check_mats(const df11_matrix *mats, uint32_t n_mats, uint32_t tokens) {
    if (!mats || n_mats == 0 || n_mats > kMax) return DF11_E_INVALID_ARG;
    if (tokens == 0 || tokens > DF11_MAX_TOKENS) return DF11_E_UNSUPPORTED;
    for (uint32_t m = 0; m < n_mats; ++m) {
        const df11_matrix &d = mats[m];
        if (d.rows == 0 || d.cols == 0) return DF11_E_INVALID_ARG;
        if (d.rows % kTileRows || d.cols % kKStep || d.offset % 8) return DF11_E_UNSUPPORTED;
    }
    return DF11_OK;
}

// Partial-sum floats any device's choice of k ranges needs (with many
// tokens, the most the choice between 1x and 2x the base ranges can take).
uint64_t workspace_floats(const df11_matrix *mats, uint32_t n_mats, uint32_t tokens) {
    uint64_t f = 0;
    for (uint32_t m = 0; m < n_mats; ++m) {
        uint32_t ks, kc;
        const uint32_t base = base_ranges(mats[m].cols, tokens);
        split_into(mats[m].cols, tokens <= kFewTokens ? base : 2 * base, &ks, &kc);
        if (ks > 1) f += static_cast<uint64_t>(mats[m].rows) * ks * tokens;
    }
    return f;
}

// Checks every argument and fills the kernel arguments; enqueues nothing.
int plan(const uint16_t *weights, uint64_t n_weights, const df11_matrix *mats, uint32_t n_mats,
         const uint16_t *const *x, uint32_t tokens, float *const *y, void *workspace,
         uint64_t workspace_bytes, GemmArgs *gp, ReduceArgs *rp) {
    int rc = check_mats(mats, n_mats, tokens);
    if (rc) return rc;
    if (!weights || !x || !y || (reinterpret_cast<uintptr_t>(weights) & 15u))
        return DF11_E_INVALID_ARG;
    const uint64_t need = 4 * workspace_floats(mats, n_mats, tokens);
    if (need > workspace_bytes) return DF11_E_BUFFER_TOO_SMALL;
    if (need && (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 15u)))
        return DF11_E_INVALID_ARG;

    for (uint32_t m = 0; m < n_mats; ++m) {
        const df11_matrix &d = mats[m];
        if (d.offset > n_weights || static_cast<uint64_t>(d.rows) * d.cols > n_weights - d.offset)
            return DF11_E_INVALID_ARG;
        if (!x[m] || !y[m] || (reinterpret_cast<uintptr_t>(x[m]) & 15u) ||
            (reinterpret_cast<uintptr_t>(y[m]) & 3u))
            return DF11_E_INVALID_ARG;
    }
    uint32_t ks_req[kMax];
    rc = choose_ranges(mats, n_mats, tokens, ks_req);
    if (rc) return rc;

    GemmArgs g{};
    ReduceArgs r{};
    g.w = weights;
    g.part = static_cast<float *>(workspace);
    r.part = static_cast<const float *>(workspace);
    g.n_mats = r.n_mats = n_mats;
    g.tokens = r.tokens = tokens;
    uint64_t tiles = 0, wgs = 0, part = 0, outs = 0;
    for (uint32_t m = 0; m < n_mats; ++m) {
        const df11_matrix &d = mats[m];
        uint32_t ks, kc;
        split_into(d.cols, ks_req[m], &ks, &kc);
        g.tile_start[m] = static_cast<uint32_t>(tiles);
        g.wg_start[m] = static_cast<uint32_t>(wgs);
        g.ksplit[m] = r.ksplit[m] = ks;
        g.kchunk[m] = kc;
        g.rows[m] = r.rows[m] = d.rows;
        g.cols[m] = d.cols;
        g.w_off[m] = d.offset;
        g.part_off[m] = r.part_off[m] = part;
        g.x[m] = x[m];
        g.y[m] = r.y[m] = y[m];
        r.out_start[m] = static_cast<uint32_t>(outs);
        tiles += static_cast<uint64_t>(d.rows / kTileRows) * ks;
        wgs += static_cast<uint64_t>((d.rows + kTileRows * kSlabWaves - 1) / (kTileRows * kSlabWaves)) * ks;
        if (ks > 1) {
            part += static_cast<uint64_t>(d.rows) * ks * tokens;
            outs += static_cast<uint64_t>(d.rows) * tokens;
        }
        if (tiles > 0xFFFFFFFFull || outs > 0xFFFFFFFFull) return DF11_E_UNSUPPORTED;
    }
    for (uint32_t m = n_mats; m <= kMax; ++m) {
        g.tile_start[m] = static_cast<uint32_t>(tiles);
        g.wg_start[m] = static_cast<uint32_t>(wgs);
        r.out_start[m] = static_cast<uint32_t>(outs);
    }
    g.num_tiles = static_cast<uint32_t>(tiles);
    g.num_wg = static_cast<uint32_t>(wgs);
    r.total = static_cast<uint32_t>(outs);
    *gp = g;
    *rp = r;
    return DF11_OK;
}

int launch(const GemmArgs &g, const ReduceArgs &r, hipStream_t stream) {
    const uint32_t mt = (g.tokens + 15) / 16;
    const dim3 block(64 * kWaves), slab_block(64 * kSlabWaves);
    const dim3 grid_tiles((g.num_tiles + kWaves - 1) / kWaves), grid_wg(g.num_wg);
    switch (mt) {
    case 1:
        if (g.tokens < kSlabMinTokens)
            hipLaunchKernelGGL(gemm_tiles_kernel, grid_tiles, block, 0, stream, g);
        else
            hipLaunchKernelGGL(gemm_slab_kernel<1>, grid_wg, slab_block, 0, stream, g);
        break;
    case 2: hipLaunchKernelGGL(gemm_slab_kernel<2>, grid_wg, slab_block, 0, stream, g); break;
    case 3: hipLaunchKernelGGL(gemm_slab_kernel<3>, grid_wg, slab_block, 0, stream, g); break;
    default: hipLaunchKernelGGL(gemm_slab_kernel<4>, grid_wg, slab_block, 0, stream, g); break;
    }
    if (hipGetLastError() != hipSuccess) return DF11_E_HIP;
    if (r.total) {
        hipLaunchKernelGGL(gemm_reduce_kernel, dim3((r.total + 255) / 256), dim3(256), 0, stream, r);
        if (hipGetLastError() != hipSuccess) return DF11_E_HIP;
    }
    return DF11_OK;
}

// Partial sums of the entry point that allocates nothing: one array per
// GPU, held until the process ends.  Host code never passes the array's name
// to a kernel (on the host it is a stand-in, not a device address); it uses
// the address hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) float scratch[DF11_STATIC_SCRATCH_BYTES / sizeof(float)];

std::mutex g_scratch_mu;
std::vector<void *> g_scratch;  // device address of `scratch`, per device

int scratch_address(void **out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return DF11_E_HIP;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (g_scratch.size() <= static_cast<size_t>(dev)) g_scratch.resize(dev + 1, nullptr);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return DF11_E_HIP;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return DF11_OK;
}

}  // namespace

extern "C" {

int df11_gemm_workspace_bytes(const df11_matrix *mats, uint32_t n_mats, uint32_t tokens,
                              uint64_t *bytes) {
    int rc = check_mats(mats, n_mats, tokens);
    if (rc) return rc;
    if (!bytes) return DF11_E_INVALID_ARG;
    *bytes = 4 * workspace_floats(mats, n_mats, tokens);
    return DF11_OK;
}

int df11_block_gemm(const uint16_t *weights, uint64_t n_weights, const df11_matrix *mats,
                    uint32_t n_mats, const uint16_t *const *x, uint32_t tokens, float *const *y,
                    void *workspace, uint64_t workspace_bytes, hipStream_t stream) {
    GemmArgs g;
    ReduceArgs r;
    int rc = plan(weights, n_weights, mats, n_mats, x, tokens, y, workspace, workspace_bytes, &g, &r);
    if (rc) return rc;
    return launch(g, r, stream);
}

int df11_block_forward(const df11_stream *dev, uint16_t *weights_out, const df11_matrix *mats,
                       uint32_t n_mats, const uint16_t *const *x, uint32_t tokens,
                       float *const *y, void *workspace, uint64_t workspace_bytes,
                       hipStream_t stream) {
    if (!dev) return DF11_E_INVALID_ARG;
    // every argument is checked before anything is enqueued
    GemmArgs g;
    ReduceArgs r;
    int rc = plan(weights_out, dev->sizes.n_elems, mats, n_mats, x, tokens, y, workspace,
                  workspace_bytes, &g, &r);
    if (rc) return rc;
    rc = df11_decode_block(dev, weights_out, stream);
    if (rc) return rc;
    return launch(g, r, stream);
}

int df11_block_forward_noalloc(const df11_stream *dev, uint16_t *weights_out,
                               const df11_matrix *mats, uint32_t n_mats,
                               const uint16_t *const *x, uint32_t tokens, float *const *y,
                               hipStream_t stream) {
    if (!dev) return DF11_E_INVALID_ARG;
    int rc = check_mats(mats, n_mats, tokens);
    if (rc) return rc;
    // every partial sum is written before it is read: nothing to clear
    if (4 * workspace_floats(mats, n_mats, tokens) > DF11_STATIC_SCRATCH_BYTES)
        return DF11_E_BUFFER_TOO_SMALL;
    void *ws = nullptr;
    rc = scratch_address(&ws);
    if (rc) return rc;
    return df11_block_forward(dev, weights_out, mats, n_mats, x, tokens, y, ws,
                              DF11_STATIC_SCRATCH_BYTES, stream);
}

}  // extern "C"
