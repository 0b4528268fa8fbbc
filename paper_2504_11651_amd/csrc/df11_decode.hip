// DFloat11 decompression on gfx950 (Algorithm 1 of arXiv 2504.11651,
// re-designed for CDNA4).
//
// A block of T chunks (the paper's "thread block") is decoded by one
// wavefront when T = 64 (a chunk per lane) or T = 128 (two adjacent chunks
// per lane, decoded as two interleaved lookup chains) -- the block's prefix
// sum is then a wave-level DPP scan and no workgroup barrier is needed, so
// the waves of a CU drift into different phases and decode overlaps memory
// streaming -- or, when T >= 256, by one workgroup: T threads with a chunk
// each (T = 256, 512), or T/2 threads whose waves take 128 of the chunks as
// lane pairs (T = 1024).  The grid is persistent:
// decode tables are staged into LDS once per workgroup and shared by all of
// its waves.
//
// Per block:
//   1. every lane loads its 8-byte chunk of EncodedExponent plus the next
//      4 bytes (or its two chunks' 16 bytes plus the next 4), and the 5-bit
//      Gaps of its chunks and of the next chunk;
//   2. phase 1 (count): starting at the gap, decode with the multi-symbol
//      table until the code start reaches the next chunk's first code;
//   3. exclusive scan of the counts (wave DPP scan, plus LDS across waves
//      for T >= 256) gives each lane its output position (Sec. 2.3.2);
//   4. phase 2 (emit): replay the lookups phase 1 kept in registers (a
//      chunk that needed more decodes its remaining codes again) and OR the
//      exponent bytes into an LDS buffer at their output positions.  The
//      waves of a CU run this phase at a higher priority than decoding, and
//      step 5 higher still.  A lookup may run past the lane's
//      last code; the extra codes are the next lanes' first codes, decoded
//      from the same bits, so they land on their own positions with their
//      own values and need no masking;
//   5. assemble BF16 = sign<<15 | exponent<<7 | mantissa (Algorithm 1) for
//      8 consecutive outputs per lane and step: one 8-byte PackedSignMantissa
//      load (issued when the block starts), one 8-byte LDS read, one 16-byte
//      store; consecutive lanes take consecutive groups, so a wave stores
//      1 KiB contiguous per instruction.  The block's first and last group
//      may be shared with its neighbours; their elements go out as one
//      2-byte store over 16 lanes.  No per-element gather (the paper
//      gathers sign/mantissa per element).
// Integer work only; no MFMA.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <vector>

#include "df11.h"
#include "df11_decode_core.h"
#include "df11_tables.h"

namespace {

using namespace df11dec;

// T = 64: every wave owns whole blocks; W waves per workgroup share the tables.
template <uint32_t W>
__global__ __launch_bounds__(64 * W) void df11_decode_wave_kernel(DecodeArgs a) {
    extern __shared__ __align__(16) uint8_t lds[];
    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63u;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // block indices stay scalar
    const uint32_t first_block = xcd_grouped_index(blockIdx.x, gridDim.x) * W + wave;
    const uint32_t stride = gridDim.x * W;
    // the first block's words are requested before the tables are staged,
    // so the two memory round trips overlap
    ChunkWords cw{};
    if (first_block < a.num_blocks) cw = load_chunk(a, first_block, first_block * 64u + lane);
    stage_table_blob(a, lds, tid, 64 * W);
    const Tables tb = stage_tables(a, lds);
    uint8_t *buf = lds + a.table_lds_bytes + wave * a.buf_bytes;
    uint32_t *buf32 = reinterpret_cast<uint32_t *>(buf);
    const uint32_t cap = a.buf_bytes - 8u;
    __syncthreads();
    if (first_block >= a.num_blocks) return;
    Chunk ch = chunk_setup(a, cw, first_block * 64u + lane);
    Range r = block_range(a, cw);

    for (uint32_t b = first_block; b < a.num_blocks; b += stride) {
        // loads for this block's assembly and the next block's decode
        const uint32_t bn = b + stride;
        ChunkWords nxt = cw;
        if (bn < a.num_blocks) nxt = load_chunk(a, bn, bn * 64u + lane);
        uint2 S[kPre];
        prefetch_sm(a, r, lane, 64u, S);
        const uint32_t edge_sm = prefetch_edge_sm(a, r, lane);

        wave_lds_sync();  // this wave's reads of the previous block are issued
        for (uint32_t i = lane; i < (a.buf_bytes >> 4); i += 64u)
            reinterpret_cast<uint4 *>(buf)[i] = make_uint4(0u, 0u, 0u, 0u);

        uint32_t sy[kKeep], npk[(kKeep + 3) / 4], p_rest;
        const uint32_t cnt = decode_count(tb, ch, sy, npk, &p_rest);
        const uint32_t excl = wave_inclusive_scan(cnt) - cnt;
        // Waves near their memory phase issue first: the CU's decoding waves
        // (priority 0) fill the gaps, and the loads and stores of the waves
        // that have finished decoding reach the memory system sooner.
        __builtin_amdgcn_s_setprio(1);
        wave_lds_sync();
        emit_exponents(tb, ch, sy, npk, p_rest, r.shift + excl, buf32, cap);
        wave_lds_sync();

        __builtin_amdgcn_s_setprio(2);
        assemble_block(a, r, buf, lane, 64u, S, edge_sm);
        __builtin_amdgcn_s_setprio(0);
        cw = nxt;
        ch = chunk_setup(a, cw, bn * 64u + lane);
        r = block_range(a, cw);
    }
}

// Lookups kept per chunk and sign/mantissa groups fetched at block start
// when a lane owns two chunks (a 128-chunk block holds about twice the
// outputs of a 64-chunk one).
constexpr int kKeepPair = 10;
constexpr int kPrePair = 7;

// T = 128: one wave per block as well, lane l owning chunks 2l and 2l+1 of
// it.  Its 16 bytes come in one 128-bit load, the two chunks decode
// interleaved (independent table lookups in flight together), and the
// block's count scan, buffer, edges and positions are shared by twice the
// outputs.
template <uint32_t W>
__global__ __launch_bounds__(64 * W) void df11_decode_pair_kernel(DecodeArgs a) {
    extern __shared__ __align__(16) uint8_t lds[];
    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63u;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t first_block = xcd_grouped_index(blockIdx.x, gridDim.x) * W + wave;
    const uint32_t stride = gridDim.x * W;
    PairWords pw{};
    if (first_block < a.num_blocks) pw = load_pair(a, first_block, first_block * 128u + 2u * lane);
    stage_table_blob(a, lds, tid, 64 * W);
    const Tables tb = stage_tables(a, lds);
    uint8_t *buf = lds + a.table_lds_bytes + wave * a.buf_bytes;
    uint32_t *buf32 = reinterpret_cast<uint32_t *>(buf);
    const uint32_t cap = a.buf_bytes - 8u;
    __syncthreads();
    if (first_block >= a.num_blocks) return;
    Chunk A, B;
    pair_setup(a, pw, first_block * 128u + 2u * lane, A, B);
    Range r = block_range(a, pw.bp0, pw.bp1);

    for (uint32_t b = first_block; b < a.num_blocks; b += stride) {
        const uint32_t bn = b + stride;
        PairWords nxt = pw;
        if (bn < a.num_blocks) nxt = load_pair(a, bn, bn * 128u + 2u * lane);
        uint2 S[kPrePair];
        prefetch_sm(a, r, lane, 64u, S);
        const uint32_t edge_sm = prefetch_edge_sm(a, r, lane);

        wave_lds_sync();
        for (uint32_t i = lane; i < (a.buf_bytes >> 4); i += 64u)
            reinterpret_cast<uint4 *>(buf)[i] = make_uint4(0u, 0u, 0u, 0u);

        uint32_t syA[kKeepPair], npkA[(kKeepPair + 3) / 4], syB[kKeepPair],
            npkB[(kKeepPair + 3) / 4], restA, restB, cntA, cntB;
        decode_count_pair(tb, A, B, syA, npkA, syB, npkB, &restA, &restB, &cntA, &cntB);
        const uint32_t cnt = cntA + cntB;
        const uint32_t excl = wave_inclusive_scan(cnt) - cnt;
        __builtin_amdgcn_s_setprio(1);
        wave_lds_sync();
        emit_exponents(tb, A, syA, npkA, restA, r.shift + excl, buf32, cap);
        emit_exponents(tb, B, syB, npkB, restB, r.shift + excl + cntA, buf32, cap);
        wave_lds_sync();

        __builtin_amdgcn_s_setprio(2);
        assemble_block(a, r, buf, lane, 64u, S, edge_sm);
        __builtin_amdgcn_s_setprio(0);
        pw = nxt;
        pair_setup(a, pw, bn * 128u + 2u * lane, A, B);
        r = block_range(a, pw.bp0, pw.bp1);
    }
}

// T = 1024: one workgroup of T/2 threads per block, each wave decoding 128
// chunks as lane pairs like the kernel above.  The waves' counts meet in
// LDS, every wave ORs its exponents into one block buffer, and the workgroup
// assembles the block together.  Where LDS holds two block buffers they
// alternate between blocks: a buffer is cleared while the other is still
// being assembled, so a block needs two barriers (counts, then exponents).
// With one buffer, a third barrier waits for the previous block's assembly.
template <uint32_t T>
__global__ __launch_bounds__(T / 2) void df11_decode_block_pair_kernel(DecodeArgs a) {
    constexpr uint32_t NT = T / 2;
    extern __shared__ __align__(16) uint8_t lds[];
    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63u;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    PairWords pw{};
    if (blockIdx.x < a.num_blocks) pw = load_pair(a, blockIdx.x, blockIdx.x * T + 2u * tid);
    stage_table_blob(a, lds, tid, NT);
    const Tables tb = stage_tables(a, lds);
    uint32_t *wave_sums = reinterpret_cast<uint32_t *>(lds + a.table_lds_bytes);
    uint8_t *const buf0 = lds + a.table_lds_bytes + 4 * kScanSlots;
    const uint32_t cap = a.buf_bytes - 8u;
    __syncthreads();
    if (blockIdx.x >= a.num_blocks) return;
    Chunk A, B;
    pair_setup(a, pw, blockIdx.x * T + 2u * tid, A, B);
    Range r = block_range(a, pw.bp0, pw.bp1);

    uint32_t parity = 0;
    for (uint32_t b = blockIdx.x; b < a.num_blocks; b += gridDim.x) {
        const uint32_t bn = b + gridDim.x;
        PairWords nxt = pw;
        if (bn < a.num_blocks) nxt = load_pair(a, bn, bn * T + 2u * tid);
        uint2 S[kPrePair];
        prefetch_sm(a, r, tid, NT, S);
        const uint32_t edge_sm = prefetch_edge_sm(a, r, tid);

        // with two buffers this one was last read two blocks ago, before the
        // previous block's barriers
        if (!a.twin_bufs) __syncthreads();  // the previous block is assembled
        uint8_t *buf = buf0 + (a.twin_bufs ? parity : 0u) * a.buf_bytes;
        uint32_t *buf32 = reinterpret_cast<uint32_t *>(buf);
        for (uint32_t i = tid; i < (a.buf_bytes >> 4); i += NT)
            reinterpret_cast<uint4 *>(buf)[i] = make_uint4(0u, 0u, 0u, 0u);

        uint32_t syA[kKeepPair], npkA[(kKeepPair + 3) / 4], syB[kKeepPair],
            npkB[(kKeepPair + 3) / 4], restA, restB, cntA, cntB;
        decode_count_pair(tb, A, B, syA, npkA, syB, npkB, &restA, &restB, &cntA, &cntB);
        const uint32_t cnt = cntA + cntB;
        const uint32_t incl = wave_inclusive_scan(cnt);
        if (lane == 63u) wave_sums[wave] = incl;
        __syncthreads();  // every wave's count is in, the buffer is cleared
        uint32_t before = 0;
        for (uint32_t w = 0; w < wave; ++w) before += wave_sums[w];
        const uint32_t off = r.shift + before + incl - cnt;
        emit_exponents(tb, A, syA, npkA, restA, off, buf32, cap);
        emit_exponents(tb, B, syB, npkB, restB, off + cntA, buf32, cap);
        __syncthreads();  // the block's exponents are all in the buffer

        assemble_block(a, r, buf, tid, NT, S, edge_sm);
        parity ^= 1u;
        pw = nxt;
        pair_setup(a, pw, bn * T + 2u * tid, A, B);
        r = block_range(a, pw.bp0, pw.bp1);
    }
}

// T = 256, 512: one workgroup of T threads per block, a chunk per thread.
// (Two chunks per lane would halve the waves of a workgroup, and the tables
// staged per workgroup would then cap the waves per CU.)
template <uint32_t T>
__global__ __launch_bounds__(T) void df11_decode_block_kernel(DecodeArgs a) {
    extern __shared__ __align__(16) uint8_t lds[];
    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63u;
    const uint32_t wave = tid >> 6;
    stage_table_blob(a, lds, tid, T);
    const Tables tb = stage_tables(a, lds);
    uint32_t *wave_sums = reinterpret_cast<uint32_t *>(lds + a.table_lds_bytes);
    uint8_t *buf = lds + a.table_lds_bytes + 4 * kScanSlots;
    uint32_t *buf32 = reinterpret_cast<uint32_t *>(buf);
    const uint32_t cap = a.buf_bytes - 8u;

    if (blockIdx.x >= a.num_blocks) return;
    ChunkWords cw = load_chunk(a, blockIdx.x, blockIdx.x * T + tid);
    Chunk ch = chunk_setup(a, cw, blockIdx.x * T + tid);
    Range r = block_range(a, cw);

    for (uint32_t b = blockIdx.x; b < a.num_blocks; b += gridDim.x) {
        const uint32_t bn = b + gridDim.x;
        ChunkWords nxt = cw;
        if (bn < a.num_blocks) nxt = load_chunk(a, bn, bn * T + tid);
        uint2 S[kPre];
        prefetch_sm(a, r, tid, T, S);
        const uint32_t edge_sm = prefetch_edge_sm(a, r, tid);

        __syncthreads();  // tables staged / previous block's buffer consumed
        for (uint32_t i = tid; i < (a.buf_bytes >> 4); i += T)
            reinterpret_cast<uint4 *>(buf)[i] = make_uint4(0u, 0u, 0u, 0u);

        uint32_t sy[kKeep], npk[(kKeep + 3) / 4], p_rest;
        const uint32_t cnt = decode_count(tb, ch, sy, npk, &p_rest);

        const uint32_t incl = wave_inclusive_scan(cnt);
        if (lane == 63u) wave_sums[wave] = incl;
        __syncthreads();
        uint32_t before = 0;
        for (uint32_t w = 0; w < wave; ++w) before += wave_sums[w];
        emit_exponents(tb, ch, sy, npk, p_rest, r.shift + before + incl - cnt, buf32, cap);
        __syncthreads();

        assemble_block(a, r, buf, tid, T, S, edge_sm);
        cw = nxt;
        ch = chunk_setup(a, cw, bn * T + tid);
        r = block_range(a, cw);
    }
}

using KernelFn = void (*)(DecodeArgs);

struct LaunchShape {
    uint32_t threads, lut_bits, buf;  // key
    KernelFn fn;
    uint32_t block, lds, per_cu, waves_per_group, twin_bufs;
};

struct DeviceInfo {
    int cus = 0;
    int max_lds = 0;                 // bytes of LDS one workgroup may use
    uint32_t lds_granted[11] = {};   // dynamic LDS limit set per kernel instance (slot)
    std::vector<LaunchShape> shapes; // launch shapes already worked out
};

std::mutex g_mu;
std::vector<DeviceInfo> g_dev;

constexpr uint32_t kWaveChoices[4] = {4, 8, 12, 16};
// Waves per SIMD for a long stream: 5 beats 4 and 6 (a sixth adds contention
// for memory and LDS, not throughput).  A short stream takes every wave that
// fits when that removes a round of blocks per wave (its tail dominates).
constexpr uint64_t kLongWavesPerSimd = 5;
constexpr uint64_t kShortRounds = 4;
constexpr size_t kMaxShapes = 64;  // cached launch shapes per device

KernelFn wave_kernel(uint32_t W) {
    switch (W) {
        case 4: return df11_decode_wave_kernel<4>;
        case 8: return df11_decode_wave_kernel<8>;
        case 12: return df11_decode_wave_kernel<12>;
        case 16: return df11_decode_wave_kernel<16>;
        default: return nullptr;
    }
}

KernelFn pair_kernel(uint32_t W) {
    switch (W) {
        case 4: return df11_decode_pair_kernel<4>;
        case 8: return df11_decode_pair_kernel<8>;
        case 12: return df11_decode_pair_kernel<12>;
        case 16: return df11_decode_pair_kernel<16>;
        default: return nullptr;
    }
}

// Slots of lds_granted: 0-3 wave kernels, 4-7 pair kernels, 8-10 below.
KernelFn block_kernel(uint32_t T, int *slot) {
    switch (T) {
        case 256: *slot = 8; return df11_decode_block_kernel<256>;
        case 512: *slot = 9; return df11_decode_block_kernel<512>;
        case 1024: *slot = 10; return df11_decode_block_pair_kernel<1024>;
        default: return nullptr;
    }
}

// Lets a kernel use `lds` bytes of dynamic LDS and returns how many of its
// workgroups fit on one CU (0 when none does).
int fit(DeviceInfo &di, int slot, KernelFn fn, uint32_t threads, uint32_t lds, int *per_cu) {
    *per_cu = 0;
    if (lds > static_cast<uint32_t>(di.max_lds)) return DF11_OK;
    if (lds > 65536u && di.lds_granted[slot] < lds) {
        if (hipFuncSetAttribute(reinterpret_cast<const void *>(fn),
                                hipFuncAttributeMaxDynamicSharedMemorySize,
                                static_cast<int>(lds)) != hipSuccess)
            return DF11_E_HIP;
        di.lds_granted[slot] = lds;
    }
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(per_cu, reinterpret_cast<const void *>(fn),
                                                     static_cast<int>(threads), lds) != hipSuccess)
        return DF11_E_HIP;
    return DF11_OK;
}

int shape_for(const df11_stream *s, KernelFn *fn, uint32_t *grid, uint32_t *block, uint32_t *lds,
              uint32_t *twin_bufs) {
    const uint32_t T = s->layout.threads_per_block;
    const uint32_t K = s->layout.lut_bits;
    const uint32_t tab = static_cast<uint32_t>(df11tab::lds_bytes(K));
    const uint32_t buf = buf_bytes_for(s->sizes.max_elems_per_block);
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
    const LaunchShape *found = nullptr;
    for (const LaunchShape &ls : di.shapes)
        if (ls.threads == T && ls.lut_bits == K && ls.buf == buf) found = &ls;
    if (!found) {
        LaunchShape ls{T, K, buf, nullptr, 0, 0, 0, 1, 0};
        if (T == 64 || T == 128) {
            // one wave per block: most resident waves per CU; fewer waves per
            // workgroup on a tie
            int best_waves = 0;
            for (int i = 0; i < 4; ++i) {
                const uint32_t W = kWaveChoices[i];
                const KernelFn fn = T == 64 ? wave_kernel(W) : pair_kernel(W);
                int pc = 0;
                int rc = fit(di, T == 64 ? i : 4 + i, fn, 64 * W, tab + W * buf, &pc);
                if (rc) return rc;
                if (pc * static_cast<int>(W) > best_waves) {
                    best_waves = pc * static_cast<int>(W);
                    ls.fn = fn;
                    ls.block = 64 * W;
                    ls.lds = tab + W * buf;
                    ls.per_cu = static_cast<uint32_t>(pc);
                    ls.waves_per_group = W;
                }
            }
            if (!best_waves) return DF11_E_UNSUPPORTED;
        } else if (T == 1024) {
            int slot = 0, pc = 0;
            ls.fn = block_kernel(T, &slot);
            ls.block = T / 2;
            ls.twin_bufs = 1;
            ls.lds = tab + 4 * kScanSlots + 2 * buf;  // two block buffers
            int rc = fit(di, slot, ls.fn, T / 2, ls.lds, &pc);
            if (rc) return rc;
            if (pc < 1) {  // one buffer (very compressible streams: large blocks)
                ls.twin_bufs = 0;
                ls.lds = tab + 4 * kScanSlots + buf;
                rc = fit(di, slot, ls.fn, T / 2, ls.lds, &pc);
                if (rc) return rc;
            }
            if (pc < 1) return DF11_E_UNSUPPORTED;
            ls.per_cu = static_cast<uint32_t>(pc);
        } else {
            int slot = 0, pc = 0;
            ls.fn = block_kernel(T, &slot);
            ls.block = T;
            ls.lds = tab + 4 * kScanSlots + buf;
            int rc = fit(di, slot, ls.fn, T, ls.lds, &pc);
            if (rc) return rc;
            if (pc < 1) return DF11_E_UNSUPPORTED;
            ls.per_cu = static_cast<uint32_t>(pc);
        }
        if (di.shapes.size() >= kMaxShapes) di.shapes.erase(di.shapes.begin());  // oldest goes
        di.shapes.push_back(ls);
        found = &di.shapes.back();
    }
    *fn = found->fn;
    *block = found->block;
    *lds = found->lds;
    *twin_bufs = found->twin_bufs;
    const uint64_t W = found->waves_per_group;
    const uint64_t nb = s->sizes.num_blocks;
    const uint64_t blocks_needed = (nb + W - 1) / W;
    uint64_t per_cu = found->per_cu;
    const uint64_t cap = kLongWavesPerSimd * 4 / W;  // 4 SIMDs per CU
    if (T <= 128 && cap >= 1 && per_cu > cap) {
        const uint64_t cus = static_cast<uint64_t>(di.cus);
        const uint64_t rounds_all = (nb + cus * per_cu * W - 1) / (cus * per_cu * W);
        const uint64_t rounds_cap = (nb + cus * cap * W - 1) / (cus * cap * W);
        if (!(rounds_all < rounds_cap && rounds_all <= kShortRounds)) per_cu = cap;
    }
    uint64_t g = static_cast<uint64_t>(di.cus) * per_cu;
    if (g > blocks_needed) g = blocks_needed;
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
    uint32_t twin;
    return shape_for(s, &fn, grid, block, lds_bytes, &twin);
}

int df11_decode_block(const df11_stream *s, uint16_t *out, hipStream_t stream) {
    int rc = check_stream(s);
    if (rc) return rc;
    if (s->sizes.n_elems == 0) return DF11_OK;
    if (!out || (reinterpret_cast<uintptr_t>(out) & 15u)) return DF11_E_INVALID_ARG;
    KernelFn fn;
    uint32_t grid, block, lds, twin;
    rc = shape_for(s, &fn, &grid, &block, &lds, &twin);
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
    a.twin_bufs = twin;
    hipLaunchKernelGGL(fn, dim3(grid), dim3(block), lds, stream, a);
    return hipGetLastError() == hipSuccess ? DF11_OK : DF11_E_HIP;
}

}  // extern "C"
