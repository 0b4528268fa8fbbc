// DFloat11 decompression on gfx950 (Algorithm 1 of arXiv 2504.11651,
// re-designed for CDNA4).
//
// One workgroup decodes one block of T chunks at a time (the paper's
// "thread block"); a persistent grid walks the blocks so the decode tables
// are staged into LDS once per workgroup instead of once per block.
//
// Per block:
//   1. every lane loads its 8-byte chunk of EncodedExponent plus the next
//      4 bytes, and its two 5-bit Gaps (own chunk and next chunk);
//   2. phase 1 (count): starting at the gap, decode with the multi-symbol
//      table until the code start reaches the next chunk's first code;
//   3. workgroup exclusive scan of the counts (wave scan + LDS across waves)
//      gives each lane its output position (Sec. 2.3.2);
//   4. phase 2 (emit): decode again and OR the exponent bytes into an LDS
//      buffer at their output positions.  A lookup may run past the lane's
//      last code; the extra codes are the next lanes' first codes, decoded
//      from the same bits, so they land on their own positions with their
//      own values and need no masking;
//   5. assemble BF16 = sign<<15 | exponent<<7 | mantissa (Algorithm 1) for
//      16 consecutive outputs per lane: one 16-byte PackedSignMantissa load,
//      one 16-byte LDS read, two 16-byte stores -- coalesced, no per-element
//      gather (the paper gathers sign/mantissa per element).
// Integer work only; no MFMA.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <vector>

#include "df11.h"
#include "df11_tables.h"

namespace {

constexpr uint32_t kScanSlots = 16;  // waves per workgroup (<= 1024 threads)
constexpr uint32_t kBufSlack = 32;   // alignment shift (< 16) + over-decoded bytes

struct DecodeArgs {
    const uint8_t *exp;
    const uint8_t *sm;
    const uint32_t *gaps;      // packed Gaps read as 32-bit words
    const uint32_t *block_pos; // B + 1 entries
    const uint8_t *tables;     // LDS image (blob past its header)
    uint16_t *out;
    uint64_t total_bits;
    uint32_t n_elems;
    uint32_t num_chunks;
    uint32_t num_blocks;
    uint32_t lut_bits;
    uint32_t max_len;
    uint32_t table_lds_bytes;
    uint32_t buf_bytes;        // exponent buffer, multiple of 16
};

// 4 stream bytes as loaded (little endian) -> word whose bit j is stream bit j
// (the stream is most-significant-bit first within each byte).
__device__ __forceinline__ uint32_t lsb_first(uint32_t le) {
    return __builtin_bitreverse32(__builtin_bswap32(le));
}

// 32 stream bits starting at bit p (0 <= p < 64) of the 96 bits w0:w1:w2.
__device__ __forceinline__ uint32_t window_at(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t p) {
    const bool upper = p >= 32;
    const uint32_t lo = upper ? w1 : w0;
    const uint32_t hi = upper ? w2 : w1;
    return __builtin_amdgcn_alignbit(hi, lo, p);
}

struct Tables {
    const uint2 *ent;        // K-bit entries: x = exponents, y = meta
    const uint32_t *lj_last; // [33]
    const uint32_t *offset;  // [33]
    const uint8_t *sorted;   // [256]
    uint32_t mask;
    uint32_t lut_bits;
    uint32_t max_len;
};

// Code longer than the table index: canonical length search on the
// left-justified window, then rank within the length.
__device__ __forceinline__ uint2 decode_long(Tables t, uint32_t win) {
    const uint32_t v = __builtin_bitreverse32(win);
    uint32_t L = t.lut_bits + 1;
    while (L < t.max_len && v > t.lj_last[L]) ++L;
    const uint32_t idx = ((v >> (32u - L)) + t.offset[L]) & 255u;
    return make_uint2(t.sorted[idx], L | (1u << 8) | (1u << 16));
}

__device__ __forceinline__ uint2 lookup(Tables t, uint32_t win) {
    uint2 e = t.ent[win & t.mask];
    if (e.y == 0) e = decode_long(t, win);
    return e;
}

__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t v) {
    const uint32_t lane = __lane_id();
#pragma unroll
    for (uint32_t d = 1; d < 64; d <<= 1) {
        const uint32_t t = __shfl_up(v, d, 64);
        if (lane >= d) v += t;
    }
    return v;
}

// 4 sign/mantissa bytes + 4 exponents -> 4 BF16 (two words, low element first).
__device__ __forceinline__ void assemble4(uint32_t S, uint32_t E, uint32_t &o0, uint32_t &o1) {
    const uint32_t lo = (S & 0x7F7F7F7Fu) | ((E << 7) & 0x80808080u);  // (e&1)<<7 | mantissa
    const uint32_t hi = (S & 0x80808080u) | ((E >> 1) & 0x7F7F7F7Fu);  // sign<<7 | e>>1
    o0 = __builtin_amdgcn_perm(hi, lo, 0x05010400u);
    o1 = __builtin_amdgcn_perm(hi, lo, 0x07030602u);
}

template <uint32_t T>
__global__ __launch_bounds__(T) void df11_decode_kernel(DecodeArgs a) {
    extern __shared__ __align__(16) uint8_t lds[];
    const uint32_t tid = threadIdx.x;
    const uint32_t ent_bytes = 8u << a.lut_bits;
    Tables tb;
    tb.ent = reinterpret_cast<const uint2 *>(lds);
    tb.lj_last = reinterpret_cast<const uint32_t *>(lds + ent_bytes);
    tb.offset = tb.lj_last + 33;
    tb.sorted = reinterpret_cast<const uint8_t *>(tb.offset + 33);
    tb.mask = (1u << a.lut_bits) - 1u;
    tb.lut_bits = a.lut_bits;
    tb.max_len = a.max_len;
    uint32_t *wave_sums = reinterpret_cast<uint32_t *>(lds + a.table_lds_bytes);
    uint8_t *buf = lds + a.table_lds_bytes + 4 * kScanSlots;
    uint32_t *buf32 = reinterpret_cast<uint32_t *>(buf);
    const uint32_t buf_dwords = a.buf_bytes >> 2;

    {  // stage the decode tables once per workgroup
        const uint4 *src = reinterpret_cast<const uint4 *>(a.tables);
        uint4 *dst = reinterpret_cast<uint4 *>(lds);
        for (uint32_t i = tid; i < (a.table_lds_bytes >> 4); i += T) dst[i] = src[i];
    }

    const uint32_t lane = tid & 63u;
    const uint32_t wave = tid >> 6;

    for (uint32_t b = blockIdx.x; b < a.num_blocks; b += gridDim.x) {
        __syncthreads();  // tables staged / previous block's buffer consumed
        for (uint32_t i = tid; i < (a.buf_bytes >> 4); i += T)
            reinterpret_cast<uint4 *>(buf)[i] = make_uint4(0u, 0u, 0u, 0u);

        // ---- 1. chunk bits and gaps
        const uint32_t c = b * T + tid;
        const uint2 own = *reinterpret_cast<const uint2 *>(a.exp + 8ull * c);
        const uint32_t nxt = *reinterpret_cast<const uint32_t *>(a.exp + 8ull * c + 8);
        const uint32_t w0 = lsb_first(own.x), w1 = lsb_first(own.y), w2 = lsb_first(nxt);

        const uint64_t gbit = 5ull * c;
        const uint64_t gw = gbit >> 5;
        const uint64_t gv = ((static_cast<uint64_t>(__builtin_bswap32(a.gaps[gw])) << 32) |
                             __builtin_bswap32(a.gaps[gw + 1]))
                            << (static_cast<uint32_t>(gbit) & 31u);
        const uint32_t gap_own = static_cast<uint32_t>(gv >> 59);
        const uint32_t gap_next = static_cast<uint32_t>(gv >> 54) & 31u;

        uint32_t start = 0, end = 0;
        if (c < a.num_chunks) {
            start = gap_own;
            end = (c + 1 < a.num_chunks) ? 64u + gap_next
                                         : static_cast<uint32_t>(a.total_bits - 64ull * c);
            end = min(end, 95u);
        }

        // ---- 2. phase 1: count the codes that start in this chunk
        uint32_t p = start, cnt = 0, last_p = 0, last_meta = 0;
        for (uint32_t it = 0; p < end && it < 96u; ++it) {
            const uint2 e = lookup(tb, window_at(w0, w1, w2, p));
            last_p = p;
            last_meta = e.y;
            p += e.y & 0xFFu;
            cnt += (e.y >> 8) & 0xFFu;
        }
        // codes of the last lookup that start at or past `end` belong to the next chunk
        cnt -= __builtin_popcount((last_meta >> 16) >> min(end - last_p, 31u));

        // ---- 3. output positions: exclusive scan over the workgroup
        const uint32_t incl = wave_inclusive_scan(cnt);
        if (lane == 63u) wave_sums[wave] = incl;
        __syncthreads();
        uint32_t before = 0;
        for (uint32_t w = 0; w < wave; ++w) before += wave_sums[w];
        const uint32_t excl = before + incl - cnt;

        const uint32_t s = min(a.block_pos[b], a.n_elems);
        uint32_t e_end = max(min(a.block_pos[b + 1], a.n_elems), s);
        const uint32_t shift = s & 15u;
        e_end = min(e_end, s + (a.buf_bytes - kBufSlack));
        const uint32_t count = e_end - s;

        // ---- 4. phase 2: exponents into the LDS buffer at their positions
        uint32_t off = shift + excl;
        p = start;
        for (uint32_t it = 0; p < end && it < 96u; ++it) {
            const uint2 e = lookup(tb, window_at(w0, w1, w2, p));
            const uint64_t v = static_cast<uint64_t>(e.x) << ((off & 3u) * 8u);
            const uint32_t dw = min(off >> 2, buf_dwords - 2u);
            atomicOr(&buf32[dw], static_cast<uint32_t>(v));
            atomicOr(&buf32[dw + 1], static_cast<uint32_t>(v >> 32));
            off += (e.y >> 8) & 0xFFu;
            p += e.y & 0xFFu;
        }
        __syncthreads();

        // ---- 5. assemble BF16 and write 16 outputs per lane
        const uint32_t g0 = s - shift;
        const uint32_t ngroups = (shift + count + 15u) >> 4;
        for (uint32_t g = tid; g < ngroups; g += T) {
            const uint32_t j0 = g << 4;  // buffer index of the group
            if (j0 >= shift && j0 + 16u <= shift + count) {
                const uint4 S = *reinterpret_cast<const uint4 *>(a.sm + g0 + j0);
                const uint4 E = reinterpret_cast<const uint4 *>(buf)[g];
                uint4 lo, hi;
                assemble4(S.x, E.x, lo.x, lo.y);
                assemble4(S.y, E.y, lo.z, lo.w);
                assemble4(S.z, E.z, hi.x, hi.y);
                assemble4(S.w, E.w, hi.z, hi.w);
                uint4 *dst = reinterpret_cast<uint4 *>(a.out + g0 + j0);
                dst[0] = lo;
                dst[1] = hi;
            } else {
                for (uint32_t k = 0; k < 16u; ++k) {
                    const uint32_t j = j0 + k;
                    if (j >= shift && j < shift + count) {
                        const uint32_t smb = a.sm[g0 + j];
                        const uint32_t ex = buf[j];
                        a.out[g0 + j] =
                            static_cast<uint16_t>(((smb & 0x80u) << 8) | (ex << 7) | (smb & 0x7Fu));
                    }
                }
            }
        }
    }
}

struct DeviceInfo {
    int cus = 0;
    int max_lds = 0;                         // bytes of LDS one workgroup may use
    uint32_t lds_granted[5] = {0, 0, 0, 0, 0};  // dynamic LDS limit set per kernel
};

std::mutex g_mu;
std::vector<DeviceInfo> g_dev;

using KernelFn = void (*)(DecodeArgs);

KernelFn kernel_for(uint32_t T, int *slot) {
    switch (T) {
        case 64: *slot = 0; return df11_decode_kernel<64>;
        case 128: *slot = 1; return df11_decode_kernel<128>;
        case 256: *slot = 2; return df11_decode_kernel<256>;
        case 512: *slot = 3; return df11_decode_kernel<512>;
        case 1024: *slot = 4; return df11_decode_kernel<1024>;
        default: return nullptr;
    }
}

uint32_t buf_bytes_for(uint32_t max_elems) {
    return (max_elems + kBufSlack + 15u) & ~15u;
}

int check_stream(const df11_stream *s) {
    if (!s) return DF11_E_INVALID_ARG;
    const df11_sizes &z = s->sizes;
    if (s->layout.bytes_per_thread != 8) return DF11_E_UNSUPPORTED;
    int slot;
    if (!kernel_for(s->layout.threads_per_block, &slot)) return DF11_E_UNSUPPORTED;
    if (s->layout.lut_bits < 8 || s->layout.lut_bits > 12) return DF11_E_INVALID_ARG;
    if (z.n_elems == 0) return DF11_OK;
    if (!s->exp || !s->sm || !s->gaps || !s->block_pos || !s->tables) return DF11_E_INVALID_ARG;
    if (z.n_elems > 0xFFFFFFFFull || z.num_blocks > 0xFFFFFFFFull / 1024) return DF11_E_INVALID_ARG;
    if (z.max_code_len > 32 || z.table_bytes != df11tab::blob_bytes(s->layout.lut_bits))
        return DF11_E_INVALID_ARG;
    const uint64_t T = s->layout.threads_per_block;
    if (z.exp_bytes < z.num_blocks * 8 * T + 16) return DF11_E_INVALID_ARG;
    if (z.gap_bytes < 4 * ((5 * (z.num_blocks * T + 1) + 31) / 32 + 2)) return DF11_E_INVALID_ARG;
    if (z.num_chunks > z.num_blocks * T) return DF11_E_INVALID_ARG;
    if (z.max_elems_per_block > 64u * T) return DF11_E_INVALID_ARG;
    if ((reinterpret_cast<uintptr_t>(s->sm) & 15u) || (reinterpret_cast<uintptr_t>(s->exp) & 7u) ||
        (reinterpret_cast<uintptr_t>(s->gaps) & 3u) || (reinterpret_cast<uintptr_t>(s->tables) & 15u) ||
        (reinterpret_cast<uintptr_t>(s->block_pos) & 3u))
        return DF11_E_INVALID_ARG;
    return DF11_OK;
}

int shape_for(const df11_stream *s, KernelFn *fn, uint32_t *grid, uint32_t *block, uint32_t *lds) {
    int slot = 0;
    const uint32_t T = s->layout.threads_per_block;
    *fn = kernel_for(T, &slot);
    const uint32_t tab = static_cast<uint32_t>(df11tab::lds_bytes(s->layout.lut_bits));
    *lds = tab + 4 * kScanSlots + buf_bytes_for(s->sizes.max_elems_per_block);
    *block = T;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return DF11_E_HIP;
    std::lock_guard<std::mutex> lk(g_mu);
    if (g_dev.size() <= static_cast<size_t>(dev)) g_dev.resize(dev + 1);
    DeviceInfo &di = g_dev[dev];
    if (!di.cus) {
        if (hipDeviceGetAttribute(&di.cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            hipDeviceGetAttribute(&di.max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) !=
                hipSuccess)
            return DF11_E_HIP;
    }
    if (*lds > static_cast<uint32_t>(di.max_lds)) return DF11_E_UNSUPPORTED;
    if (*lds > 65536u && di.lds_granted[slot] < *lds) {
        if (hipFuncSetAttribute(reinterpret_cast<const void *>(*fn),
                                hipFuncAttributeMaxDynamicSharedMemorySize,
                                static_cast<int>(*lds)) != hipSuccess)
            return DF11_E_HIP;
        di.lds_granted[slot] = *lds;
    }
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void *>(*fn),
                                                     static_cast<int>(T), *lds) != hipSuccess)
        return DF11_E_HIP;
    if (per_cu < 1) return DF11_E_UNSUPPORTED;
    uint64_t g = static_cast<uint64_t>(di.cus) * static_cast<uint64_t>(per_cu);
    if (g > s->sizes.num_blocks) g = s->sizes.num_blocks;
    *grid = static_cast<uint32_t>(g ? g : 1);
    return DF11_OK;
}

}  // namespace

extern "C" {

int df11_decode_launch_shape(const df11_stream *s, uint32_t *grid, uint32_t *block,
                             uint32_t *lds_bytes) {
    int rc = check_stream(s);
    if (rc) return rc;
    if (!grid || !block || !lds_bytes) return DF11_E_INVALID_ARG;
    KernelFn fn;
    return shape_for(s, &fn, grid, block, lds_bytes);
}

int df11_decode_block(const df11_stream *s, uint16_t *out, hipStream_t stream) {
    int rc = check_stream(s);
    if (rc) return rc;
    if (s->sizes.n_elems == 0) return DF11_OK;
    if (!out || (reinterpret_cast<uintptr_t>(out) & 15u)) return DF11_E_INVALID_ARG;
    KernelFn fn;
    uint32_t grid, block, lds;
    rc = shape_for(s, &fn, &grid, &block, &lds);
    if (rc) return rc;
    DecodeArgs a;
    a.exp = s->exp;
    a.sm = s->sm;
    a.gaps = reinterpret_cast<const uint32_t *>(s->gaps);
    a.block_pos = s->block_pos;
    a.tables = s->tables + df11tab::kHeaderBytes;
    a.out = out;
    a.total_bits = s->sizes.total_bits;
    a.n_elems = static_cast<uint32_t>(s->sizes.n_elems);
    a.num_chunks = static_cast<uint32_t>(s->sizes.num_chunks);
    a.num_blocks = static_cast<uint32_t>(s->sizes.num_blocks);
    a.lut_bits = s->layout.lut_bits;
    a.max_len = s->sizes.max_code_len;
    a.table_lds_bytes = static_cast<uint32_t>(df11tab::lds_bytes(s->layout.lut_bits));
    a.buf_bytes = buf_bytes_for(s->sizes.max_elems_per_block);
    hipLaunchKernelGGL(fn, dim3(grid), dim3(block), lds, stream, a);
    return hipGetLastError() == hipSuccess ? DF11_OK : DF11_E_HIP;
}

}  // extern "C"
