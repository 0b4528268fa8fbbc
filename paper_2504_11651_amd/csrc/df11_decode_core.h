// Building blocks of the DFloat11 decoder shared by the kernels that decode
// a stream (Algorithm 1 of arXiv 2504.11651): stream loads, table lookups,
// the two decode phases, the wave prefix sum and BF16 assembly, plus the
// host-side descriptor check.  Included by the decode kernels and by the
// fused decode-and-multiply kernel.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

#include "df11.h"
#include "df11_tables.h"

namespace df11dec {


constexpr uint32_t kScanSlots = 16;  // waves per workgroup (<= 1024 threads)
// Exponent buffer bytes past the largest block: alignment shift (< 8), codes
// decoded past a block's end, and the 4 bytes per kept lookup that a lane may
// store past a clamped start offset.
constexpr uint32_t kBufSlack = 128;

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
    uint32_t twin_bufs;        // T >= 256: two block buffers alternate (else one)
};

__device__ __forceinline__ uint32_t umin(uint32_t a, uint32_t b) { return a < b ? a : b; }
__device__ __forceinline__ uint32_t umax(uint32_t a, uint32_t b) { return a > b ? a : b; }

// 4 stream bytes as loaded (little endian) -> word whose bit j is stream bit j
// (the stream is most-significant-bit first within each byte).
__device__ __forceinline__ uint32_t lsb_first(uint32_t le) {
    return __builtin_bitreverse32(__builtin_bswap32(le));
}

// 32 bits starting at bit p (0 <= p < 64) of the 96 bits w0:w1:w2.
__device__ __forceinline__ uint32_t window_at(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t p) {
    const bool upper = p >= 32;
    const uint32_t lo = upper ? w1 : w0;
    const uint32_t hi = upper ? w2 : w1;
    return __builtin_amdgcn_alignbit(hi, lo, p);
}

// The kernels declare no static LDS, so the dynamically sized LDS (and the
// decode table at its start) begins at group-segment offset 0; table entries
// are read through LDS byte offsets.
__device__ __forceinline__ uint2 lds_entry(uint32_t byte_offset) {
    const uint64_t v = *(__attribute__((address_space(3))) const uint64_t *)
        static_cast<uintptr_t>(byte_offset);
    return make_uint2(static_cast<uint32_t>(v), static_cast<uint32_t>(v >> 32));
}

struct Tables {
    // K-bit entries (8 bytes: x = exponents, y = meta) at LDS offset 0
    const uint32_t *lj_last; // [33]
    const uint32_t *offset;  // [33]
    const uint8_t *sorted;   // [256]
    uint32_t addr_mask;      // (2^K - 1) << 3: entry byte offset from a shifted window
    uint32_t lut_bits;
    uint32_t max_len;
};

__device__ __forceinline__ Tables stage_tables(const DecodeArgs &a, uint8_t *lds) {
    Tables tb;
    const uint32_t ent_bytes = 8u << a.lut_bits;
    tb.lj_last = reinterpret_cast<const uint32_t *>(lds + ent_bytes);
    tb.offset = tb.lj_last + 33;
    tb.sorted = reinterpret_cast<const uint8_t *>(tb.offset + 33);
    tb.addr_mask = ((1u << a.lut_bits) - 1u) << 3;
    tb.lut_bits = a.lut_bits;
    tb.max_len = a.max_len;
    return tb;
}

// Code longer than the table index: canonical length search on the
// left-justified window, then rank within the length.
__device__ __forceinline__ uint2 decode_long(const Tables &t, uint32_t win) {
    const uint32_t v = __builtin_bitreverse32(win);
    uint32_t L = t.lut_bits + 1;
    while (L < t.max_len && v > t.lj_last[L]) ++L;
    const uint32_t idx = ((v >> (32u - L)) + t.offset[L]) & 255u;
    return make_uint2(t.sorted[idx], L | (1u << 8) | (1u << 16));
}

// Inclusive prefix sum over the 64 lanes of a wave: four row shifts give the
// sums within each row of 16 lanes, two row broadcasts carry row totals.
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t v) {
    v += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x111, 0xF, 0xF, true));
    v += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x112, 0xF, 0xF, true));
    v += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x114, 0xF, 0xF, true));
    v += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x118, 0xF, 0xF, true));
    v += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x142, 0xA, 0xF, false));
    v += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x143, 0xC, 0xF, false));
    return v;
}

// Orders this wave's LDS accesses (other lanes' writes become visible to
// later reads: LDS executes a wave's instructions in order; this keeps the
// compiler from moving accesses across).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// 4 sign/mantissa bytes + 4 exponents -> 4 BF16 (two words, low element first).
__device__ __forceinline__ void assemble4(uint32_t S, uint32_t E, uint32_t &o0, uint32_t &o1) {
    const uint32_t lo = (S & 0x7F7F7F7Fu) | ((E << 7) & 0x80808080u);  // (e&1)<<7 | mantissa
    const uint32_t hi = (S & 0x80808080u) | ((E >> 1) & 0x7F7F7F7Fu);  // sign<<7 | e>>1
    o0 = __builtin_amdgcn_perm(hi, lo, 0x05010400u);
    o1 = __builtin_amdgcn_perm(hi, lo, 0x07030602u);
}

// Raw global words one lane needs for chunk c of block b: the chunk's 8
// bytes, the next 4 bytes, the two 32-bit words holding Gaps[c] and
// Gaps[c+1], and the block's two BlockOutputPos entries.
struct ChunkWords {
    uint32_t x, y, z, g0, g1, bp0, bp1;
};

__device__ __forceinline__ ChunkWords load_chunk(const DecodeArgs &a, uint32_t b, uint32_t c) {
    ChunkWords r;
    // BlockOutputPos is read-only for the whole launch and its index is
    // uniform: through the constant address space these are scalar loads,
    // which keep the vector memory path for the streams
    const __attribute__((address_space(4))) uint32_t *bp =
        (const __attribute__((address_space(4))) uint32_t *)a.block_pos;
    r.bp0 = bp[b];
    r.bp1 = bp[b + 1];
    const uint2 own = *reinterpret_cast<const uint2 *>(a.exp + 8ull * c);
    r.x = own.x;
    r.y = own.y;
    r.z = *reinterpret_cast<const uint32_t *>(a.exp + 8ull * c + 8);
    const uint64_t gw = (5ull * c) >> 5;
    r.g0 = a.gaps[gw];
    r.g1 = a.gaps[gw + 1];
    return r;
}

// Lookups kept in registers between the count phase and the write phase;
// a chunk needing more (short codes, 4 per lookup) continues in a loop.
constexpr int kKeep = 10;
// 8-element output groups whose sign/mantissa bytes are fetched at block start.
constexpr int kPre = 4;

// One chunk's decode state.  w*: the chunk's bits (word j bit i = stream bit
// 32j+i); s*: the same bits moved up by 3, so that a window taken from s* at
// bit p holds stream bits p.. at bits 3.. and masking it gives the byte
// offset of the table entry directly.
struct Chunk {
    uint32_t w0, w1, w2, s0, s1, s2, start, end;
};

__device__ __forceinline__ Chunk chunk_setup(const DecodeArgs &a, const ChunkWords &cw, uint32_t c) {
    Chunk ch;
    ch.w0 = lsb_first(cw.x);
    ch.w1 = lsb_first(cw.y);
    ch.w2 = lsb_first(cw.z);
    ch.s0 = ch.w0 << 3;
    ch.s1 = __builtin_amdgcn_alignbit(ch.w1, ch.w0, 29);
    ch.s2 = __builtin_amdgcn_alignbit(ch.w2, ch.w1, 29);
    const uint64_t gv = ((static_cast<uint64_t>(__builtin_bswap32(cw.g0)) << 32) |
                         __builtin_bswap32(cw.g1))
                        << ((5u * c) & 31u);
    const uint32_t gap_own = static_cast<uint32_t>(gv >> 59);
    const uint32_t gap_next = static_cast<uint32_t>(gv >> 54) & 31u;
    ch.start = 0;
    ch.end = 0;
    if (c < a.num_chunks) {
        ch.start = gap_own;
        const uint32_t e = (c + 1 < a.num_chunks) ? 64u + gap_next
                                                  : static_cast<uint32_t>(a.total_bits - 64ull * c);
        ch.end = min(e, 95u);
    }
    return ch;
}

__device__ __forceinline__ uint2 lookup(const Tables &t, const Chunk &ch, uint32_t p) {
    const uint32_t ws = window_at(ch.s0, ch.s1, ch.s2, p);
    uint2 e = lds_entry(ws & t.addr_mask);
    if (e.y == 0u) e = decode_long(t, window_at(ch.w0, ch.w1, ch.w2, p));
    return e;
}

// ---- two chunks per lane (blocks of 128 chunks decoded by one wavefront) ----

// Raw global words for the chunk pair (c, c+1), c even: their 16 bytes (one
// 128-bit load), the next 4 bytes, the two 32-bit words holding Gaps[c],
// Gaps[c+1] and Gaps[c+2], and the block's two BlockOutputPos entries.
struct PairWords {
    uint32_t x0, x1, x2, x3, z, g0, g1, bp0, bp1;
};

__device__ __forceinline__ PairWords load_pair(const DecodeArgs &a, uint32_t b, uint32_t c) {
    PairWords r;
    const __attribute__((address_space(4))) uint32_t *bp =
        (const __attribute__((address_space(4))) uint32_t *)a.block_pos;
    r.bp0 = bp[b];
    r.bp1 = bp[b + 1];
    // EncodedExponent is only 8-byte aligned (its stated alignment), and the
    // type says so; the load stays one 16-byte load
    typedef uint32_t u32x4_a8 __attribute__((ext_vector_type(4), aligned(8)));
    const u32x4_a8 own = *reinterpret_cast<const u32x4_a8 *>(a.exp + 8ull * c);
    r.x0 = own.x;
    r.x1 = own.y;
    r.x2 = own.z;
    r.x3 = own.w;
    r.z = *reinterpret_cast<const uint32_t *>(a.exp + 8ull * c + 16);
    const uint64_t gw = (5ull * c) >> 5;
    r.g0 = a.gaps[gw];
    r.g1 = a.gaps[gw + 1];
    return r;
}

// Decode state of chunks c (A) and c+1 (B).  B's window words start at the
// pair's third word; their low 3 shifted-in bits come from A's bits and only
// ever sit below a window's table index, which is masked off.
__device__ __forceinline__ void pair_setup(const DecodeArgs &a, const PairWords &pw, uint32_t c,
                                           Chunk &A, Chunk &B) {
    const uint32_t w0 = lsb_first(pw.x0), w1 = lsb_first(pw.x1), w2 = lsb_first(pw.x2),
                   w3 = lsb_first(pw.x3), w4 = lsb_first(pw.z);
    const uint32_t s2 = __builtin_amdgcn_alignbit(w2, w1, 29);
    A.w0 = w0;
    A.w1 = w1;
    A.w2 = w2;
    A.s0 = w0 << 3;
    A.s1 = __builtin_amdgcn_alignbit(w1, w0, 29);
    A.s2 = s2;
    B.w0 = w2;
    B.w1 = w3;
    B.w2 = w4;
    B.s0 = s2;
    B.s1 = __builtin_amdgcn_alignbit(w3, w2, 29);
    B.s2 = __builtin_amdgcn_alignbit(w4, w3, 29);
    const uint64_t gv = ((static_cast<uint64_t>(__builtin_bswap32(pw.g0)) << 32) |
                         __builtin_bswap32(pw.g1))
                        << ((5u * c) & 31u);
    const uint32_t gap_a = static_cast<uint32_t>(gv >> 59);
    const uint32_t gap_b = static_cast<uint32_t>(gv >> 54) & 31u;
    const uint32_t gap_c = static_cast<uint32_t>(gv >> 49) & 31u;
    A.start = A.end = B.start = B.end = 0;
    if (c < a.num_chunks) {
        A.start = gap_a;
        const uint32_t e = (c + 1 < a.num_chunks) ? 64u + gap_b
                                                  : static_cast<uint32_t>(a.total_bits - 64ull * c);
        A.end = min(e, 95u);
    }
    if (c + 1 < a.num_chunks) {
        B.start = gap_b;
        const uint32_t e = (c + 2 < a.num_chunks)
                               ? 64u + gap_c
                               : static_cast<uint32_t>(a.total_bits - 64ull * (c + 1));
        B.end = min(e, 95u);
    }
}

// Phase 1 for both chunks of a pair at once: each step takes one lookup of
// A and one of B, which are independent, so their LDS round trips overlap.
// Otherwise as decode_count, per chunk.
template <int N>
__device__ __forceinline__ void decode_count_pair(const Tables &t, const Chunk &A, const Chunk &B,
                                                  uint32_t (&syA)[N], uint32_t (&npkA)[(N + 3) / 4],
                                                  uint32_t (&syB)[N], uint32_t (&npkB)[(N + 3) / 4],
                                                  uint32_t *restA, uint32_t *restB,
                                                  uint32_t *cntA, uint32_t *cntB) {
#pragma unroll
    for (int k = 0; k < (N + 3) / 4; ++k) npkA[k] = npkB[k] = 0u;
    uint32_t pA = A.start, pB = B.start, cA = 0, cB = 0;
    uint32_t lpA = 0, lmA = 0, lpB = 0, lmB = 0;
    constexpr uint32_t sel[4] = {0x03020105u, 0x03020500u, 0x03050100u, 0x05020100u};
#pragma unroll
    for (int k = 0; k < N; ++k) {
        const bool actA = pA < A.end, actB = pB < B.end;
        syA[k] = syB[k] = 0u;
        if (__builtin_amdgcn_ballot_w64(actA || actB) == 0) continue;  // wave-uniform skip
        const uint32_t wsA = window_at(A.s0, A.s1, A.s2, pA);
        const uint32_t wsB = window_at(B.s0, B.s1, B.s2, pB);
        uint2 eA = lds_entry(wsA & t.addr_mask);
        uint2 eB = lds_entry(wsB & t.addr_mask);
        if (actA && eA.y == 0u) eA = decode_long(t, window_at(A.w0, A.w1, A.w2, pA));
        if (actB && eB.y == 0u) eB = decode_long(t, window_at(B.w0, B.w1, B.w2, pB));
        const uint32_t mA = actA ? eA.y : 0u, mB = actB ? eB.y : 0u;
        syA[k] = eA.x;
        syB[k] = eB.x;
        npkA[k / 4] = __builtin_amdgcn_perm(mA, npkA[k / 4], sel[k % 4]);  // byte k%4 <- count
        npkB[k / 4] = __builtin_amdgcn_perm(mB, npkB[k / 4], sel[k % 4]);
        lpA = actA ? pA : lpA;
        lmA = actA ? mA : lmA;
        lpB = actB ? pB : lpB;
        lmB = actB ? mB : lmB;
        pA += eA.y & 0xFFu;  // done chunks only move further past their end
        pB += eB.y & 0xFFu;
        cA += (mA >> 8) & 0xFFu;
        cB += (mB >> 8) & 0xFFu;
    }
    *restA = pA;
    *restB = pB;
    for (uint32_t it = 0; pA < A.end && it < 96u; ++it) {
        const uint2 e = lookup(t, A, pA);
        lpA = pA;
        lmA = e.y;
        pA += e.y & 0xFFu;
        cA += (e.y >> 8) & 0xFFu;
    }
    for (uint32_t it = 0; pB < B.end && it < 96u; ++it) {
        const uint2 e = lookup(t, B, pB);
        lpB = pB;
        lmB = e.y;
        pB += e.y & 0xFFu;
        cB += (e.y >> 8) & 0xFFu;
    }
    *cntA = cA - __builtin_popcount((lmA >> 16) >> min(A.end - lpA, 31u));
    *cntB = cB - __builtin_popcount((lmB >> 16) >> min(B.end - lpB, 31u));
}

// Phase 1: decode the codes that start in the chunk, keep up to kKeep
// lookups (exponent words in sy, code counts one byte each in npk), and
// count the codes.  Returns the count; *p_rest = where decoding stopped.
__device__ __forceinline__ uint32_t decode_count(const Tables &t, const Chunk &ch,
                                                 uint32_t (&sy)[kKeep],
                                                 uint32_t (&npk)[(kKeep + 3) / 4],
                                                 uint32_t *p_rest) {
#pragma unroll
    for (int k = 0; k < (kKeep + 3) / 4; ++k) npk[k] = 0u;
    uint32_t p = ch.start, cnt = 0, last_p = 0, last_meta = 0;
#pragma unroll
    for (int k = 0; k < kKeep; ++k) {
        const bool act = p < ch.end;
        sy[k] = 0u;
        if (__builtin_amdgcn_ballot_w64(act) == 0) continue;  // wave-uniform skip
        const uint32_t ws = window_at(ch.s0, ch.s1, ch.s2, p);
        uint2 e = lds_entry(ws & t.addr_mask);
        if (act && e.y == 0u) e = decode_long(t, window_at(ch.w0, ch.w1, ch.w2, p));
        const uint32_t m = act ? e.y : 0u;
        sy[k] = e.x;
        constexpr uint32_t sel[4] = {0x03020105u, 0x03020500u, 0x03050100u, 0x05020100u};
        npk[k / 4] = __builtin_amdgcn_perm(m, npk[k / 4], sel[k % 4]);  // byte k%4 <- count
        last_p = act ? p : last_p;
        last_meta = act ? m : last_meta;
        p += e.y & 0xFFu;  // done lanes only move further past `end`
        cnt += (m >> 8) & 0xFFu;
    }
    *p_rest = p;
    for (uint32_t it = 0; p < ch.end && it < 96u; ++it) {
        const uint2 e = lookup(t, ch, p);
        last_p = p;
        last_meta = e.y;
        p += e.y & 0xFFu;
        cnt += (e.y >> 8) & 0xFFu;
    }
    // codes of the last lookup that start at or past `end` belong to the next chunk
    return cnt - __builtin_popcount((last_meta >> 16) >> min(ch.end - last_p, 31u));
}

// OR 4 exponent bytes into the zeroed buffer at byte offset off.
__device__ __forceinline__ void or_exponents(uint32_t *buf32, uint32_t off, uint32_t syms) {
    const uint64_t v = static_cast<uint64_t>(syms) << ((off & 3u) << 3);
    atomicOr(&buf32[off >> 2], static_cast<uint32_t>(v));
    atomicOr(&buf32[(off >> 2) + 1], static_cast<uint32_t>(v >> 32));
}

// Phase 2: exponents into the LDS buffer at output offset off (the kept
// lookups, then the rest of a long chunk by decoding again).  A valid entry
// holds at most 4 codes, so 3 bits of each kept count suffice; with the start
// clamped, the kept lookups stay inside the buffer whatever the metadata and
// tables hold; the rest are clamped one by one.
template <int N>
__device__ __forceinline__ void emit_exponents(const Tables &t, const Chunk &ch,
                                               const uint32_t (&sy)[N],
                                               const uint32_t (&npk)[(N + 3) / 4],
                                               uint32_t p_rest, uint32_t off, uint32_t *buf32,
                                               uint32_t cap_bytes) {
    off = umin(off, cap_bytes - 8u * N);
#pragma unroll
    for (int k = 0; k < N; ++k) {
        const uint32_t n = (npk[k / 4] >> (8 * (k % 4))) & 7u;
        if (n != 0u) {
            or_exponents(buf32, off, sy[k]);
            off += n;
        }
    }
    uint32_t p = p_rest;
    for (uint32_t it = 0; p < ch.end && it < 96u; ++it) {
        const uint2 e = lookup(t, ch, p);
        off = umin(off, cap_bytes);
        or_exponents(buf32, off, e.x);
        off += (e.y >> 8) & 0xFFu;
        p += e.y & 0xFFu;
    }
}

// A block's output range, clamped to the buffer and the tensor.  Outputs
// are handled in 8-element groups aligned to the tensor: group g of the
// block covers buffer bytes [8g, 8g+8), i.e. outputs g0 + 8g .. g0 + 8g + 7;
// the block owns buffer bytes [shift, lim).  Only the first and the last
// group can be partial (shared with the neighbouring block): the groups
// [full_lo, full_hi) are whole.
struct Range {
    uint32_t s, shift, lim, g0, ngroups, full_lo, full_hi;
};

__device__ __forceinline__ Range block_range(const DecodeArgs &a, uint32_t bp0, uint32_t bp1) {
    Range r;
    r.s = umin(static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(bp0)), a.n_elems);
    uint32_t e = umax(umin(static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(bp1)), a.n_elems), r.s);
    // at most the buffer's worth; the room above r.s is clamped so the sum
    // cannot wrap for a stream ending near 2^32 weights
    e = umin(e, r.s + umin(a.buf_bytes - kBufSlack, 0xFFFFFFFFu - r.s));
    r.shift = r.s & 7u;
    r.lim = r.shift + (e - r.s);
    r.g0 = r.s - r.shift;
    r.ngroups = (r.lim + 7u) >> 3;
    r.full_lo = r.shift ? 1u : 0u;
    r.full_hi = umax(r.lim >> 3, r.full_lo);
    return r;
}

__device__ __forceinline__ Range block_range(const DecodeArgs &a, const ChunkWords &cw) {
    return block_range(a, cw.bp0, cw.bp1);
}

__device__ __forceinline__ bool full_group(const Range &r, uint32_t g) {
    return g - r.full_lo < r.full_hi - r.full_lo;  // full_lo <= g < full_hi
}

// Sign/mantissa bytes of groups first, first+step, ... (P of them).  The
// buffer is zero padded past n_elems to a multiple of 16 bytes, so a whole
// group can be read even where the block starts or ends inside it.
template <int P>
__device__ __forceinline__ void prefetch_sm(const DecodeArgs &a, const Range &r, uint32_t first,
                                            uint32_t step, uint2 (&S)[P]) {
    const uint32_t last = umax(r.ngroups, 1u) - 1u;  // groups past the block reread its last one
#pragma unroll
    for (int k = 0; k < P; ++k) {
        const uint32_t g = umin(first + k * step, last);
        S[k] = *reinterpret_cast<const uint2 *>(a.sm + r.g0 + (g << 3));
    }
}

// Edge elements: threads 0..7 take element t of the block's first group,
// threads 8..15 element t-8 of its last group.  Buffer byte of thread t's
// element (inside [0, 8*ngroups) whenever the block has a group).
__device__ __forceinline__ uint32_t edge_byte(const Range &r, uint32_t t) {
    return (t < 8u ? 0u : (umax(r.ngroups, 1u) - 1u) << 3) + (t & 7u);
}

// The sign/mantissa byte of this thread's edge element (threads 0..15),
// fetched when the block starts like the groups' bytes.
__device__ __forceinline__ uint32_t prefetch_edge_sm(const DecodeArgs &a, const Range &r,
                                                     uint32_t t) {
    uint32_t v = 0;
    if (t < 16u) v = a.sm[r.g0 + edge_byte(r, t)];
    return v;
}

// 8 outputs of group g from its sign/mantissa bytes and the exponent buffer.
__device__ __forceinline__ uint4 assemble_group(const uint8_t *buf, uint32_t g, uint2 Sg) {
    const uint2 E = reinterpret_cast<const uint2 *>(buf)[g];
    uint4 o;
    assemble4(Sg.x, E.x, o.x, o.y);
    assemble4(Sg.y, E.y, o.z, o.w);
    return o;
}

// One 16-byte non-temporal store of a whole group (the output is written
// once and not read back by this kernel).
__device__ __forceinline__ void store_group(const DecodeArgs &a, const Range &r, uint32_t g,
                                            const uint4 &o) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 ov = {o.x, o.y, o.z, o.w};
    __builtin_nontemporal_store(ov, reinterpret_cast<u32x4 *>(a.out + r.g0 + (g << 3)));
}

// Assemble and store every whole group of the block: groups first + k*step.
// The first P use the bytes fetched when the block started.  Loads and
// stores share one in-order counter on this GPU, so all of those groups are
// assembled (their loads waited for) before the first store is issued;
// otherwise each wait would also wait for the stores issued before it.
// Then the elements of the (at most two) partial groups that this block
// owns go out as one 2-byte store instruction over threads 0..15.
template <int P>
__device__ __forceinline__ void assemble_block(const DecodeArgs &a, const Range &r,
                                               const uint8_t *buf, uint32_t first, uint32_t step,
                                               const uint2 (&S)[P], uint32_t edge_sm) {
    uint4 O[P];
#pragma unroll
    for (int k = 0; k < P; ++k) {
        const uint32_t g = first + k * step;
        O[k] = make_uint4(0u, 0u, 0u, 0u);
        if (full_group(r, g)) O[k] = assemble_group(buf, g, S[k]);
    }
#pragma unroll
    for (int k = 0; k < P; ++k) {
        const uint32_t g = first + k * step;
        if (full_group(r, g)) store_group(a, r, g, O[k]);
    }
    for (uint32_t g = first + P * step; g < r.full_hi; g += step)
        if (full_group(r, g))
            store_group(a, r, g,
                        assemble_group(buf, g, *reinterpret_cast<const uint2 *>(a.sm + r.g0 + (g << 3))));
    if (first < 16u) {
        const uint32_t t = first;
        const uint32_t el = edge_byte(r, t);
        const uint32_t g = el >> 3;
        // the last group is taken by threads 8..15 only when it is not also the first
        const bool mine = r.ngroups != 0u && !full_group(r, g) && (t < 8u || g != 0u) &&
                          el >= r.shift && el < r.lim;
        if (mine) {
            const uint32_t e = buf[el];
            a.out[r.g0 + el] = static_cast<uint16_t>(((edge_sm & 0x80u) << 8) | (e << 7) |
                                                     (edge_sm & 0x7Fu));
        }
    }
}

// Workgroups are dispatched to the 8 XCDs round robin and each XCD has its
// own L2.  Within every run of 32 workgroups this numbering gives the 4 that
// share an XCD neighbouring indices, so neighbouring blocks, which share the
// cache lines at their boundaries, are mostly decoded under one L2, while
// the blocks in flight still form one contiguous window of the stream.  A
// bijection of [0, n): a trailing partial run keeps its own numbers.
__device__ __forceinline__ uint32_t xcd_grouped_index(uint32_t g, uint32_t n) {
    constexpr uint32_t kXcds = 8u, kPer = 4u, kRun = kXcds * kPer;
    const uint32_t base = g - g % kRun;
    if (base + kRun > n) return g;
    return base + (g % kXcds) * kPer + (g % kRun) / kXcds;
}

__device__ __forceinline__ void stage_table_blob(const DecodeArgs &a, uint8_t *lds, uint32_t tid,
                                                 uint32_t nthreads) {
    const uint4 *src = reinterpret_cast<const uint4 *>(a.tables);
    uint4 *dst = reinterpret_cast<uint4 *>(lds);
    for (uint32_t i = tid; i < (a.table_lds_bytes >> 4); i += nthreads) dst[i] = src[i];
}

// ---- host side ------------------------------------------------------------

inline bool layout_supported(uint32_t T) {
    return T == 64 || T == 128 || T == 256 || T == 512 || T == 1024;
}

inline uint32_t buf_bytes_for(uint32_t max_elems) {
    return (max_elems + kBufSlack + 15u) & ~15u;
}

inline int check_stream(const df11_stream *s) {
    if (!s) return DF11_E_INVALID_ARG;
    const df11_sizes &z = s->sizes;
    if (s->layout.bytes_per_thread != 8) return DF11_E_UNSUPPORTED;
    if (!layout_supported(s->layout.threads_per_block)) return DF11_E_UNSUPPORTED;
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
    if (z.sm_bytes < ((z.n_elems + 15) & ~uint64_t{15}) + 16) return DF11_E_INVALID_ARG;
    if ((reinterpret_cast<uintptr_t>(s->sm) & 15u) || (reinterpret_cast<uintptr_t>(s->exp) & 7u) ||
        (reinterpret_cast<uintptr_t>(s->gaps) & 3u) || (reinterpret_cast<uintptr_t>(s->tables) & 15u) ||
        (reinterpret_cast<uintptr_t>(s->block_pos) & 3u))
        return DF11_E_INVALID_ARG;
    return DF11_OK;
}

}  // namespace df11dec
