// Fused decompression and matrix-vector products for one token: the weights
// of a transformer block are decoded on chip (Algorithm 1 of arXiv
// 2504.11651) and multiplied by the activations right away, so the 2 bytes
// per weight of BF16 are never written to memory and read back (the paper
// decompresses each block into a buffer right before its products,
// Sec. 2.3.3; with one token the products are bound by reading weights).
//
// Per 64-chunk block one wavefront decodes exactly as the decode kernel does
// (phase 1, prefix sum, phase 2 into LDS); then, in place of the stores, each
// lane takes its 8-weight groups, assembles the BF16 values, and accumulates
// their dot product with the matching 8 activations (v_dot2c_f32_bf16, fp32
// accumulation).  A block covers at most two matrices and at most three rows
// of each (columns >= 2048), so every lane keeps three partial sums per
// matrix segment; a wave-wide sum turns them into at most 8 partial sums per
// block, written to a workspace.  A second kernel adds, for every output row,
// the partial sums of the blocks that cover it, in block order.  The result
// depends only on the stream and the inputs (fixed summation order).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <type_traits>
#include <vector>

#include "df11.h"
#include "df11_decode_core.h"
#include "df11_tables.h"

namespace {

using namespace df11dec;

constexpr uint32_t kMaxM = DF11_MAX_MATRICES;
constexpr uint32_t kSegSlots = 4;              // partial sums per matrix segment (3 used)
constexpr uint32_t kSlots = 2 * kSegSlots;     // per block
constexpr uint32_t kMinCols = 2048;            // a block (<= 4096 weights) spans <= 3 rows
constexpr uint32_t kMaxBlockElems = 64u * 64u; // 64 chunks of at most 64 codes

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint64_t umin64(uint64_t a, uint64_t b) { return a < b ? a : b; }

// q = n / d for all 32-bit n, by the round-up multiply-and-shift method for
// division by an invariant integer (Granlund and Montgomery, 1994):
// t = mulhi(n, m), q = (t + ((n - t) >> 1)) >> (l - 1), l = ceil(log2 d).
struct Divider {
    uint32_t magic, shift;  // shift = l - 1
};

__host__ __device__ inline uint32_t divide(uint32_t n, Divider dv) {
#if defined(__HIP_DEVICE_COMPILE__)
    const uint32_t t = __umulhi(n, dv.magic);
#else
    const uint32_t t = static_cast<uint32_t>((static_cast<uint64_t>(n) * dv.magic) >> 32);
#endif
    return (t + ((n - t) >> 1)) >> dv.shift;
}

Divider make_divider(uint32_t d) {  // d >= 2
    uint32_t l = 0;
    while ((uint64_t{1} << l) < d) ++l;
    const unsigned __int128 num = (static_cast<unsigned __int128>(1) << 32) *
                                  ((uint64_t{1} << l) - d);
    return Divider{static_cast<uint32_t>(num / d + 1), l - 1};
}

struct GemvArgs {
    DecodeArgs d;
    uint32_t n_mats;
    uint32_t off[kMaxM];  // first weight of each matrix (sorted, disjoint)
    uint32_t end[kMaxM];  // one past its last weight
    uint32_t cols[kMaxM];
    Divider div[kMaxM];   // division by cols
    const uint16_t *x[kMaxM];
    uint32_t row_base[kMaxM];  // index of the matrix's first row among all rows
    float *part;               // kSlots floats per block
    uint32_t *first_block;     // per row: the block holding its first weight
    uint32_t *last_block;      // per row: the block holding its last weight
};

struct ReduceArgs {
    const uint32_t *block_pos;  // B + 1 entries
    const float *part;
    const uint32_t *first_block;
    const uint32_t *last_block;
    uint32_t num_blocks;
    uint32_t n_mats;
    uint32_t row_start[kMaxM + 1];  // prefix sums of rows
    uint32_t off[kMaxM];
    uint32_t cols[kMaxM];
    float *y[kMaxM];
};

template <int kCtrl, int kRowMask, bool kBound>
__device__ __forceinline__ float dpp_f32(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x),
                                                                 kCtrl, kRowMask, 0xF, kBound));
}

// Same row-shift / row-broadcast pattern as the integer scan: lane 63 ends
// with the sum of all 64 lanes, added in a fixed order.
__device__ __forceinline__ float wave_sum(float v) {
    v += dpp_f32<0x111, 0xF, true>(v);
    v += dpp_f32<0x112, 0xF, true>(v);
    v += dpp_f32<0x114, 0xF, true>(v);
    v += dpp_f32<0x118, 0xF, true>(v);
    v += dpp_f32<0x142, 0xA, false>(v);
    v += dpp_f32<0x143, 0xC, false>(v);
    return v;
}

__device__ __forceinline__ float dot8(const uint4 &w, const uint4 &x) {
    float d = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w.x),
                                              __builtin_bit_cast(bf16x2, x.x), 0.f, false);
    d = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w.y),
                                        __builtin_bit_cast(bf16x2, x.y), d, false);
    d = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w.z),
                                        __builtin_bit_cast(bf16x2, x.z), d, false);
    d = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w.w),
                                        __builtin_bit_cast(bf16x2, x.w), d, false);
    return d;
}

// 16-bit lane masks of the elements [a0, a1) of an 8-element group
__device__ __forceinline__ uint4 element_mask(uint32_t a0, uint32_t a1) {
    uint32_t m[4];
#pragma unroll
    for (uint32_t q = 0; q < 4; ++q) {
        const uint32_t lo = (2 * q >= a0 && 2 * q < a1) ? 0x0000FFFFu : 0u;
        const uint32_t hi = (2 * q + 1 >= a0 && 2 * q + 1 < a1) ? 0xFFFF0000u : 0u;
        m[q] = lo | hi;
    }
    return make_uint4(m[0], m[1], m[2], m[3]);
}

// The block's weights [s, e) times the activations of the (at most two)
// matrices they belong to: segment 0 is the matrix holding weight s,
// segment 1 the first matrix that starts inside (s, e).
__device__ __forceinline__ void dot_block(const GemvArgs &g, const Range &r, const uint8_t *buf,
                                          uint32_t lane, const uint2 (&S)[kPre], uint32_t b) {
    const uint32_t s = r.g0 + r.shift, e = r.g0 + r.lim;
    int seg_m[2] = {-1, -1};
#pragma unroll
    for (uint32_t i = 0; i < kMaxM; ++i) {
        if (i < g.n_mats) {
            if (g.off[i] <= s && s < g.end[i]) seg_m[0] = static_cast<int>(i);
            else if (g.off[i] > s && g.off[i] < e && seg_m[1] < 0) seg_m[1] = static_cast<int>(i);
        }
    }
#pragma unroll
    for (uint32_t j = 0; j < 2; ++j) {
        if (seg_m[j] < 0) continue;  // uniform
        const uint32_t m = static_cast<uint32_t>(seg_m[j]);
        const uint32_t off = g.off[m], cols = g.cols[m];
        const uint32_t lo = umax(s, off), hi = umin(e, g.end[m]);
        const uint32_t rlo = divide(lo - off, g.div[m]);
        // starts of the next two rows (the second clamped: past the end of
        // a stream of 2^32 - 1 weights it would wrap)
        const uint32_t b1 = off + (rlo + 1u) * cols;
        const uint32_t b2 = static_cast<uint32_t>(umin64(uint64_t{b1} + cols, 0xFFFFFFFFull));
        const uint16_t *x = g.x[m];
        // rows the segment touches (uniform): one row is the common case
        const uint32_t nrows = divide(hi - 1u - off, g.div[m]) - rlo + 1u;
        float acc[3] = {0.f, 0.f, 0.f};
        auto group = [&](uint32_t gi, uint2 Sg, auto one_row) {
            const uint32_t E = r.g0 + (gi << 3);
            if ((E < lo && lo - E >= 8u) || E >= hi) return;  // (no E + 8: it may wrap)
            const uint32_t row = one_row ? rlo : rlo + (E >= b1 ? 1u : 0u) + (E >= b2 ? 1u : 0u);
            const uint32_t kcol = E - off - row * cols;
            uint4 w = assemble_group(buf, gi, Sg);
            uint4 xv = *reinterpret_cast<const uint4 *>(x + kcol);
            if (E < lo || hi - E < 8u) {  // a group shared with a neighbour: its elements only
                const uint4 mk = element_mask(lo > E ? lo - E : 0u, umin(hi - E, 8u));
                w = make_uint4(w.x & mk.x, w.y & mk.y, w.z & mk.z, w.w & mk.w);
                xv = make_uint4(xv.x & mk.x, xv.y & mk.y, xv.z & mk.z, xv.w & mk.w);
            }
            const float d = dot8(w, xv);
            if (one_row) {
                acc[0] += d;
            } else {
                const uint32_t rr = row - rlo;
                acc[0] += rr == 0u ? d : 0.f;
                acc[1] += rr == 1u ? d : 0.f;
                acc[2] += rr == 2u ? d : 0.f;
            }
        };
        auto all_groups = [&](auto one_row) {
#pragma unroll
            for (int k = 0; k < kPre; ++k) {
                const uint32_t gi = lane + 64u * k;
                if (gi < r.ngroups) group(gi, S[k], one_row);
            }
            for (uint32_t gi = lane + 64u * kPre; gi < r.ngroups; gi += 64u)
                group(gi, *reinterpret_cast<const uint2 *>(g.d.sm + r.g0 + (gi << 3)), one_row);
        };
        if (nrows == 1u) all_groups(std::true_type{});
        else all_groups(std::false_type{});
        const float t0 = wave_sum(acc[0]);
        const float t1 = nrows > 1u ? wave_sum(acc[1]) : 0.f;
        const float t2 = nrows > 2u ? wave_sum(acc[2]) : 0.f;
        if (lane == 63u)
            *reinterpret_cast<float4 *>(g.part + static_cast<uint64_t>(b) * kSlots + j * kSegSlots) =
                make_float4(t0, t1, t2, 0.f);
        if (lane < nrows) {  // rows whose first or last weight is in this block, one per lane
            const uint64_t rs = uint64_t{off} + uint64_t{rlo + lane} * cols;
            if (rs >= lo) g.first_block[g.row_base[m] + rlo + lane] = b;
            if (rs + cols <= hi) g.last_block[g.row_base[m] + rlo + lane] = b;
        }
    }
}

// Same loop as the decode kernel (one wave per block, persistent grid); the
// decoded block goes into dot_block instead of memory.
template <uint32_t W>
__global__ __launch_bounds__(64 * W) void df11_gemv_wave_kernel(GemvArgs g) {
    const DecodeArgs &a = g.d;
    extern __shared__ __align__(16) uint8_t lds[];
    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63u;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // block indices stay scalar
    stage_table_blob(a, lds, tid, 64 * W);
    const Tables tb = stage_tables(a, lds);
    uint8_t *buf = lds + a.table_lds_bytes + wave * a.buf_bytes;
    uint32_t *buf32 = reinterpret_cast<uint32_t *>(buf);
    const uint32_t cap = a.buf_bytes - 8u;
    __syncthreads();

    const uint32_t first_block = xcd_grouped_index(blockIdx.x, gridDim.x) * W + wave;
    const uint32_t stride = gridDim.x * W;
    if (first_block >= a.num_blocks) return;
    ChunkWords cw = load_chunk(a, first_block, first_block * 64u + lane);
    Chunk ch = chunk_setup(a, cw, first_block * 64u + lane);
    Range r = block_range(a, cw);

    for (uint32_t b = first_block; b < a.num_blocks; b += stride) {
        const uint32_t bn = b + stride;
        ChunkWords nxt = cw;
        if (bn < a.num_blocks) nxt = load_chunk(a, bn, bn * 64u + lane);
        uint2 S[kPre];
        prefetch_sm(a, r, lane, 64u, S);

        wave_lds_sync();
        for (uint32_t i = lane; i < (a.buf_bytes >> 4); i += 64u)
            reinterpret_cast<uint4 *>(buf)[i] = make_uint4(0u, 0u, 0u, 0u);

        uint32_t sy[kKeep], npk[(kKeep + 3) / 4], p_rest;
        const uint32_t cnt = decode_count(tb, ch, sy, npk, &p_rest);
        const uint32_t excl = wave_inclusive_scan(cnt) - cnt;
        __builtin_amdgcn_s_setprio(1);
        wave_lds_sync();
        emit_exponents(tb, ch, sy, npk, p_rest, r.shift + excl, buf32, cap);
        wave_lds_sync();

        __builtin_amdgcn_s_setprio(2);
        dot_block(g, r, buf, lane, S, b);
        __builtin_amdgcn_s_setprio(0);
        cw = nxt;
        ch = chunk_setup(a, cw, bn * 64u + lane);
        r = block_range(a, cw);
    }
}

// y[m][row] = sum over the blocks covering the row, in block order, of the
// block's partial sum for that row.
__global__ __launch_bounds__(256) void df11_gemv_reduce_kernel(ReduceArgs ra) {
    const uint32_t i = blockIdx.x * 256u + threadIdx.x;
    if (i >= ra.row_start[ra.n_mats]) return;
    uint32_t m = 0;
#pragma unroll
    for (uint32_t q = 1; q < kMaxM; ++q)
        if (q < ra.n_mats && i >= ra.row_start[q]) m = q;
    uint32_t rs = 0, off = 0, cols = 1;
    float *y = nullptr;
#pragma unroll
    for (uint32_t q = 0; q < kMaxM; ++q) {
        if (q == m) {
            rs = ra.row_start[q];
            off = ra.off[q];
            cols = ra.cols[q];
            y = ra.y[q];
        }
    }
    const uint32_t row = i - rs;
    // every block between the row's first and last holds at least one weight
    // (each 64-bit chunk starts a code), so all of them wrote partial sums
    const uint32_t fb = ra.first_block[i], lb = ra.last_block[i];
    // a block holds >= 128 weights (64 chunks, >= 2 codes each), so a row
    // spans at most cols / 128 + 2 blocks; indices outside that (not written
    // by the decode kernel) give NaN instead of reads out of range
    if (lb >= ra.num_blocks || fb > lb || lb - fb > cols / 128u + 2u) {
        y[row] = __builtin_nanf("");
        return;
    }
    float sum = 0.f;
    for (uint32_t b = fb; b <= lb; ++b) {
        const uint32_t bs = ra.block_pos[b];
        const uint32_t j = off <= bs ? 0u : 1u;
        const uint32_t seg_lo = bs > off ? bs : off;
        const uint32_t rlo = (seg_lo - off) / cols;
        const uint32_t rr = row - rlo;  // 0..2 by construction; checked to keep reads in range
        if (rr < 3u) sum += ra.part[static_cast<uint64_t>(b) * kSlots + j * kSegSlots + rr];
    }
    y[row] = sum;
}

using GemvFn = void (*)(GemvArgs);

GemvFn gemv_kernel(uint32_t W) { return W == 4 ? df11_gemv_wave_kernel<4> : nullptr; }

struct Shape {
    int dev;
    uint32_t lut_bits, buf, W, per_cu;
};
std::mutex g_mu;
std::vector<Shape> g_shapes;
constexpr size_t kMaxShapes = 64;

// workgroup size and resident workgroups per CU for this table and buffer size
int gemv_shape(uint32_t lut_bits, uint32_t buf, uint32_t *W_out, uint32_t *grid_max) {
    int dev = 0, cus = 0, max_lds = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
        return DF11_E_HIP;
    std::lock_guard<std::mutex> lk(g_mu);
    for (const Shape &sh : g_shapes) {
        if (sh.dev == dev && sh.lut_bits == lut_bits && sh.buf == buf) {
            *W_out = sh.W;
            *grid_max = sh.per_cu * static_cast<uint32_t>(cus);
            return DF11_OK;
        }
    }
    const uint32_t tab = static_cast<uint32_t>(df11tab::lds_bytes(lut_bits));
    uint32_t best_W = 0, best_pc = 0, best_waves = 0;
    for (uint32_t W : {4u}) {
        const uint32_t lds = tab + W * buf;
        if (lds > static_cast<uint32_t>(max_lds) || lds > 65536u) continue;
        int pc = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &pc, reinterpret_cast<const void *>(gemv_kernel(W)), static_cast<int>(64 * W),
                lds) != hipSuccess)
            return DF11_E_HIP;
        if (static_cast<uint32_t>(pc) * W > best_waves) {
            best_waves = static_cast<uint32_t>(pc) * W;
            best_W = W;
            best_pc = static_cast<uint32_t>(pc);
        }
    }
    if (!best_waves) return DF11_E_UNSUPPORTED;
    if (g_shapes.size() >= kMaxShapes) g_shapes.clear();
    g_shapes.push_back(Shape{dev, lut_bits, buf, best_W, best_pc});
    *W_out = best_W;
    *grid_max = best_pc * static_cast<uint32_t>(cus);
    return DF11_OK;
}

// partial sums (kSlots floats per block), then first and last block per row
uint64_t workspace_bytes_for(const df11_stream *s, const df11_matrix *mats, uint32_t n_mats) {
    uint64_t rows = 0;
    for (uint32_t m = 0; m < n_mats; ++m) rows += mats[m].rows;
    return 4ull * kSlots * s->sizes.num_blocks + 8ull * rows;
}

int check_gemv(const df11_stream *s, const df11_matrix *mats, uint32_t n_mats) {
    int rc = check_stream(s);
    if (rc) return rc;
    if (s->layout.threads_per_block != 64) return DF11_E_UNSUPPORTED;
    if (!mats || n_mats == 0 || n_mats > kMaxM) return DF11_E_INVALID_ARG;
    uint64_t prev_end = 0;
    for (uint32_t m = 0; m < n_mats; ++m) {
        const df11_matrix &d = mats[m];
        if (d.rows == 0 || d.cols == 0) return DF11_E_INVALID_ARG;
        if (d.cols % 64 || d.cols < kMinCols || d.offset % 8) return DF11_E_UNSUPPORTED;
        const uint64_t size = static_cast<uint64_t>(d.rows) * d.cols;
        if (size < kMaxBlockElems) return DF11_E_UNSUPPORTED;  // a block spans <= 2 matrices
        if (d.offset < prev_end) return DF11_E_UNSUPPORTED;    // sorted and disjoint
        if (d.offset > s->sizes.n_elems || size > s->sizes.n_elems - d.offset)
            return DF11_E_INVALID_ARG;
        prev_end = d.offset + size;
    }
    return DF11_OK;
}

}  // namespace

extern "C" {

int df11_gemv_workspace_bytes(const df11_stream *dev, const df11_matrix *mats, uint32_t n_mats,
                              uint64_t *bytes) {
    if (!dev || !bytes || !mats || n_mats == 0 || n_mats > kMaxM) return DF11_E_INVALID_ARG;
    *bytes = workspace_bytes_for(dev, mats, n_mats);
    return DF11_OK;
}

int df11_block_gemv(const df11_stream *dev, const df11_matrix *mats, uint32_t n_mats,
                    const uint16_t *const *x, float *const *y, void *workspace,
                    uint64_t workspace_bytes, hipStream_t stream) {
    int rc = check_gemv(dev, mats, n_mats);
    if (rc) return rc;
    if (!x || !y) return DF11_E_INVALID_ARG;
    for (uint32_t m = 0; m < n_mats; ++m)
        if (!x[m] || !y[m] || (reinterpret_cast<uintptr_t>(x[m]) & 15u) ||
            (reinterpret_cast<uintptr_t>(y[m]) & 3u))
            return DF11_E_INVALID_ARG;
    const uint64_t need = workspace_bytes_for(dev, mats, n_mats);
    if (workspace_bytes < need) return DF11_E_BUFFER_TOO_SMALL;
    if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 15u)) return DF11_E_INVALID_ARG;
    if (dev->sizes.n_elems == 0) return DF11_OK;

    GemvArgs g{};
    DecodeArgs &a = g.d;
    a.exp = dev->exp;
    a.sm = dev->sm;
    a.gaps = reinterpret_cast<const uint32_t *>(dev->gaps);
    a.block_pos = dev->block_pos;
    a.tables = dev->tables + df11tab::kHeaderBytes;
    a.out = nullptr;  // nothing is stored
    a.total_bits = dev->sizes.total_bits;
    a.n_elems = static_cast<uint32_t>(dev->sizes.n_elems);
    a.num_chunks = static_cast<uint32_t>(dev->sizes.num_chunks);
    a.num_blocks = static_cast<uint32_t>(dev->sizes.num_blocks);
    a.lut_bits = dev->layout.lut_bits;
    a.max_len = dev->sizes.max_code_len;
    a.table_lds_bytes = static_cast<uint32_t>(df11tab::lds_bytes(dev->layout.lut_bits));
    a.buf_bytes = buf_bytes_for(dev->sizes.max_elems_per_block);
    a.twin_bufs = 0;  // not used by the fused kernel
    g.n_mats = n_mats;
    g.part = static_cast<float *>(workspace);
    ReduceArgs ra{};
    ra.block_pos = dev->block_pos;
    ra.part = static_cast<const float *>(workspace);
    ra.num_blocks = a.num_blocks;
    ra.n_mats = n_mats;
    uint64_t rows = 0;
    for (uint32_t m = 0; m < n_mats; ++m) {
        g.off[m] = ra.off[m] = static_cast<uint32_t>(mats[m].offset);
        g.end[m] = static_cast<uint32_t>(mats[m].offset + uint64_t{mats[m].rows} * mats[m].cols);
        g.cols[m] = ra.cols[m] = mats[m].cols;
        g.div[m] = make_divider(mats[m].cols);
        // the divider must agree with plain division at every row start and
        // just before it (a failed check means a bug here, not bad input)
        for (uint32_t t : {0u, 1u, mats[m].rows - 1u, mats[m].rows}) {
            const uint64_t n0 = uint64_t{t} * mats[m].cols;
            if (n0 <= 0xFFFFFFFFull && divide(static_cast<uint32_t>(n0), g.div[m]) != t)
                return DF11_E_UNSUPPORTED;
            if (n0 && n0 - 1 <= 0xFFFFFFFFull &&
                divide(static_cast<uint32_t>(n0 - 1), g.div[m]) != t - 1)
                return DF11_E_UNSUPPORTED;
        }
        g.x[m] = x[m];
        ra.y[m] = y[m];
        ra.row_start[m] = g.row_base[m] = static_cast<uint32_t>(rows);
        rows += mats[m].rows;
    }
    for (uint32_t m = n_mats; m <= kMaxM; ++m) ra.row_start[m] = static_cast<uint32_t>(rows);
    if (rows > 0xFFFFFFFFull) return DF11_E_UNSUPPORTED;
    uint32_t *row_blocks = reinterpret_cast<uint32_t *>(static_cast<uint8_t *>(workspace) +
                                                        4ull * kSlots * a.num_blocks);
    g.first_block = row_blocks;
    g.last_block = row_blocks + rows;
    ra.first_block = g.first_block;
    ra.last_block = g.last_block;

    uint32_t W = 0, grid_max = 0;
    rc = gemv_shape(a.lut_bits, a.buf_bytes, &W, &grid_max);
    if (rc) return rc;
    uint32_t grid = (a.num_blocks + W - 1) / W;
    if (grid > grid_max) grid = grid_max;
    if (!grid) grid = 1;
    const uint32_t lds = a.table_lds_bytes + W * a.buf_bytes;
    hipLaunchKernelGGL(gemv_kernel(W), dim3(grid), dim3(64 * W), lds, stream, g);
    if (hipGetLastError() != hipSuccess) return DF11_E_HIP;
    hipLaunchKernelGGL(df11_gemv_reduce_kernel, dim3(static_cast<uint32_t>((rows + 255) / 256)),
                       dim3(256), 0, stream, ra);
    return hipGetLastError() == hipSuccess ? DF11_OK : DF11_E_HIP;
}

}  // extern "C"
