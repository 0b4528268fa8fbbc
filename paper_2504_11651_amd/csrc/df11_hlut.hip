// The paper's own decompression kernel (Algorithm 1 of arXiv 2504.11651 with
// the hierarchical lookup tables of Sec. 2.3.1), built for gfx950 as an
// ablation beside the redesigned decoder in df11_decode.hip.  It decodes the
// same streams (EncodedExponent, PackedSignMantissa, Gaps, BlockOutputPos)
// with the paper's tables (df11_hlut_host.cpp) and keeps the paper's design:
//   - one workgroup of T threads per block of T chunks (n = 8 bytes each),
//     launched over all blocks; the block's EncodedExponent bytes, the LUTs
//     and CodeLengths are staged in LDS;
//   - phase 1: from its gap, each thread decodes one code per step -- a
//     32-bit window, LUT_1 on its first byte, pointer entries (240..255)
//     leading to LUT_(257-v) on the next byte, CodeLengths for the advance --
//     and counts the codes that start in its chunk;
//   - a work-efficient (Blelloch) exclusive scan of the counts in LDS;
//   - phase 2: each thread decodes its codes again, reads each element's
//     sign/mantissa byte from PackedSignMantissa at its output position (one
//     byte per element) and writes the BF16 into a write buffer in LDS;
//   - the block's outputs are copied from the buffer to HBM with coalesced
//     stores.
// The write buffer is offset by BlockOutputPos[b] mod 8 elements so that the
// copy can use 16-byte stores for whole 8-element groups (the paper copies
// element by element; the offset changes no value).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <vector>

#include "df11.h"
#include "df11_decode_core.h"

namespace {

struct HlutArgs {
    const uint8_t *exp;
    const uint8_t *sm;
    const uint32_t *gaps;
    const uint32_t *block_pos;
    const uint8_t *luts;  // k * 256 bytes, then CodeLengths[256]
    uint16_t *out;
    uint64_t total_bits;
    uint32_t n_elems;
    uint32_t num_chunks;
    uint32_t num_luts;
    uint32_t buf_elems;   // write buffer capacity in elements (multiple of 8)
};

// 32 stream bits starting at bit q of the staged bytes, first bit in bit 31.
__device__ __forceinline__ uint32_t window_msb(const uint32_t *stage32, uint32_t q) {
    const uint64_t w = (static_cast<uint64_t>(__builtin_bswap32(stage32[q >> 5])) << 32) |
                       __builtin_bswap32(stage32[(q >> 5) + 1]);
    return static_cast<uint32_t>((w << (q & 31u)) >> 32);
}

// One code from the window: LUT_1 on byte 1, then pointer entries lead to the
// table that decodes the next byte (at most 4 bytes, a 32-bit code).
// Returns the exponent; *len = its code length (at least 1).
__device__ __forceinline__ uint32_t decode_one(const uint8_t *luts, uint32_t k, uint32_t win,
                                               uint32_t *len) {
    uint32_t e = luts[win >> 24];
    for (uint32_t i = 1; e >= 240u && i < 4u; ++i) {
        const uint32_t t = min(256u - e, k - 1u);  // LUT_(257-e), 0-based, kept in range
        e = luts[(t << 8) + ((win >> (24u - 8u * i)) & 255u)];
    }
    const uint32_t l = luts[(k << 8) + e];
    *len = l ? l : 1u;
    return e;
}

template <uint32_t T>
__global__ __launch_bounds__(T) void df11_hlut_kernel(HlutArgs a) {
    extern __shared__ __align__(16) uint8_t lds[];
    const uint32_t tid = threadIdx.x;
    const uint32_t b = blockIdx.x;
    const uint32_t lut_bytes = (a.num_luts + 1u) << 8;
    uint8_t *luts = lds;
    uint32_t *stage32 = reinterpret_cast<uint32_t *>(lds + lut_bytes);  // 8T + 16 bytes
    uint32_t *scan = stage32 + (2u * T + 4u);                          // T words
    uint16_t *wbuf = reinterpret_cast<uint16_t *>(scan + T);           // buf_elems

    // tables and this block's EncodedExponent bytes (plus the 16 that follow)
    for (uint32_t i = tid; i < (lut_bytes >> 4); i += T)
        reinterpret_cast<uint4 *>(luts)[i] = reinterpret_cast<const uint4 *>(a.luts)[i];
    const uint2 *src = reinterpret_cast<const uint2 *>(a.exp + 8ull * T * b);
    for (uint32_t i = tid; i < T + 2u; i += T) reinterpret_cast<uint2 *>(stage32)[i] = src[i];

    const uint32_t c = b * T + tid;
    const uint64_t gw = (5ull * c) >> 5;
    const uint64_t gv = ((static_cast<uint64_t>(__builtin_bswap32(a.gaps[gw])) << 32) |
                         __builtin_bswap32(a.gaps[gw + 1]))
                        << ((5u * c) & 31u);
    const uint32_t gap = static_cast<uint32_t>(gv >> 59);
    // codes of this chunk start in [gap, end): the chunk's 64 bits, and not
    // past the end of the stream
    uint32_t end = 0;
    if (c < a.num_chunks) {
        const uint64_t rest = a.total_bits - 64ull * c;
        end = rest < 64u ? static_cast<uint32_t>(rest) : 64u;
    }
    const uint32_t bp0 = min(a.block_pos[b], a.n_elems);
    const uint32_t bp1 = max(min(a.block_pos[b + 1], a.n_elems), bp0);
    __syncthreads();

    // phase 1: count
    uint32_t count = 0;
    for (uint32_t p = gap; p < end;) {
        uint32_t len;
        decode_one(luts, a.num_luts, window_msb(stage32, 64u * tid + p), &len);
        p += len;
        ++count;
    }

    // Blelloch exclusive scan of the counts
    scan[tid] = count;
    __syncthreads();
    for (uint32_t d = 1; d < T; d <<= 1) {  // up-sweep
        const uint32_t i = (tid + 1) * 2 * d - 1;
        if (i < T) scan[i] += scan[i - d];
        __syncthreads();
    }
    if (tid == 0) scan[T - 1] = 0;
    __syncthreads();
    for (uint32_t d = T >> 1; d >= 1; d >>= 1) {  // down-sweep
        const uint32_t i = (tid + 1) * 2 * d - 1;
        if (i < T) {
            const uint32_t left = scan[i - d];
            scan[i - d] = scan[i];
            scan[i] += left;
        }
        __syncthreads();
    }

    // phase 2: decode again, gather sign/mantissa per element, write buffer
    const uint32_t shift = bp0 & 7u;
    uint32_t pos = bp0 + scan[tid];
    for (uint32_t p = gap; p < end; ++pos) {
        uint32_t len;
        const uint32_t e = decode_one(luts, a.num_luts, window_msb(stage32, 64u * tid + p), &len);
        p += len;
        const uint32_t j = pos - bp0 + shift;
        if (pos < bp1 && j < a.buf_elems) {
            const uint32_t smb = a.sm[pos];
            wbuf[j] = static_cast<uint16_t>(((smb & 0x80u) << 8) | ((e & 0xFFu) << 7) | (smb & 0x7Fu));
        }
    }
    __syncthreads();

    // coalesced copy of [bp0, bp1): whole 8-element groups as 16-byte stores
    const uint32_t lim = min(shift + (bp1 - bp0), a.buf_elems);
    const uint32_t g0 = bp0 - shift;
    const uint32_t full_lo = shift ? 1u : 0u, full_hi = max(lim >> 3, full_lo);
    for (uint32_t g = full_lo + tid; g < full_hi; g += T)
        *reinterpret_cast<uint4 *>(a.out + g0 + 8u * g) = reinterpret_cast<const uint4 *>(wbuf)[g];
    if (tid < 16u && lim) {
        const uint32_t el = (tid < 8u ? 0u : ((lim + 7u) / 8u - 1u) * 8u) + (tid & 7u);
        const uint32_t g = el >> 3;
        const bool full = g >= full_lo && g < full_hi;
        if (!full && (tid < 8u || g != 0u) && el >= shift && el < lim) a.out[g0 + el] = wbuf[el];
    }
}

using HlutFn = void (*)(HlutArgs);

HlutFn hlut_kernel(uint32_t T) {
    switch (T) {
        case 64: return df11_hlut_kernel<64>;
        case 128: return df11_hlut_kernel<128>;
        case 256: return df11_hlut_kernel<256>;
        case 512: return df11_hlut_kernel<512>;
        case 1024: return df11_hlut_kernel<1024>;
        default: return nullptr;
    }
}

std::mutex g_hlut_mu;
std::vector<uint32_t> g_hlut_lds;  // per device and T slot: dynamic LDS granted so far

uint32_t slot_of(uint32_t T) { return T == 64 ? 0 : T == 128 ? 1 : T == 256 ? 2 : T == 512 ? 3 : 4; }

}  // namespace

extern "C" int df11_decode_block_hlut(const df11_stream *s, const uint8_t *luts, uint32_t num_luts,
                                      uint16_t *out, hipStream_t stream) {
    int rc = df11dec::check_stream(s);
    if (rc) return rc;
    if (num_luts < 1 || num_luts > 17) return DF11_E_INVALID_ARG;
    if (s->sizes.n_elems == 0) return DF11_OK;
    if (!luts || (reinterpret_cast<uintptr_t>(luts) & 15u) || !out ||
        (reinterpret_cast<uintptr_t>(out) & 15u))
        return DF11_E_INVALID_ARG;
    const uint32_t T = s->layout.threads_per_block;
    HlutFn fn = hlut_kernel(T);
    if (!fn) return DF11_E_UNSUPPORTED;
    HlutArgs a;
    a.exp = s->exp;
    a.sm = s->sm;
    a.gaps = reinterpret_cast<const uint32_t *>(s->gaps);
    a.block_pos = s->block_pos;
    a.luts = luts;
    a.out = out;
    a.total_bits = s->sizes.total_bits;
    a.n_elems = static_cast<uint32_t>(s->sizes.n_elems);
    a.num_chunks = static_cast<uint32_t>(s->sizes.num_chunks);
    a.num_luts = num_luts;
    a.buf_elems = (s->sizes.max_elems_per_block + 8u + 7u) & ~7u;
    const uint32_t lds = ((num_luts + 1u) << 8) + (8u * T + 16u) + 4u * T + 2u * a.buf_elems;
    int dev = 0, max_lds = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
        return DF11_E_HIP;
    if (lds > static_cast<uint32_t>(max_lds)) return DF11_E_UNSUPPORTED;
    if (lds > 65536u) {
        std::lock_guard<std::mutex> lk(g_hlut_mu);
        const size_t idx = static_cast<size_t>(dev) * 5 + slot_of(T);
        if (g_hlut_lds.size() <= idx) g_hlut_lds.resize(idx + 1, 0);
        if (g_hlut_lds[idx] < lds) {
            if (hipFuncSetAttribute(reinterpret_cast<const void *>(fn),
                                    hipFuncAttributeMaxDynamicSharedMemorySize,
                                    static_cast<int>(lds)) != hipSuccess)
                return DF11_E_HIP;
            g_hlut_lds[idx] = lds;
        }
    }
    hipLaunchKernelGGL(fn, dim3(static_cast<uint32_t>(s->sizes.num_blocks)), dim3(T), lds, stream, a);
    return hipGetLastError() == hipSuccess ? DF11_OK : DF11_E_HIP;
}
