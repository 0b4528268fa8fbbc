// Host half of the DFloat11 codec: code book, encoder, decode tables and
// stream validation (arXiv 2504.11651, Sec. 2.3 and Algorithm 1).
//
// The encoder is the offline step of the method (the paper compresses one
// transformer block per CPU thread); here it is parallel over element
// ranges so large blocks encode in seconds.
#include <algorithm>
#include <array>
#include <atomic>
#include <cstdint>
#include <cstring>
#include <thread>
#include <vector>

#include "df11.h"
#include "df11_tables.h"

namespace {

constexpr uint64_t kMinPerThread = 1u << 20;

unsigned worker_count(uint64_t work) {
    unsigned hw = std::thread::hardware_concurrency();
    if (hw == 0) hw = 1;
    hw = std::min(hw, 32u);
    uint64_t by_work = work / kMinPerThread;
    if (by_work < 1) by_work = 1;
    return static_cast<unsigned>(std::min<uint64_t>(hw, by_work));
}

template <class F>
void parallel_for(unsigned parts, F &&fn) {
    if (parts <= 1) {
        fn(0u);
        return;
    }
    std::vector<std::thread> pool;
    pool.reserve(parts);
    for (unsigned p = 0; p < parts; ++p) pool.emplace_back([&fn, p] { fn(p); });
    for (auto &t : pool) t.join();
}

inline unsigned exp_field(uint16_t w) { return (w >> 7) & 0xFFu; }

// ---------------------------------------------------------------------------
// Code lengths
// ---------------------------------------------------------------------------

// Huffman by the two-queue method: leaves sorted by (count, value) in one
// queue, merged nodes in creation order in the other; on equal weight the
// leaf queue wins.  Returns the depth of each used symbol (depth may exceed
// 32; the caller applies the cap).
unsigned huffman_depths(const uint64_t *counts, unsigned *depth) {
    struct Leaf {
        uint64_t w;
        int sym;
    };
    std::vector<Leaf> leaves;
    for (int s = 0; s < 256; ++s)
        if (counts[s]) leaves.push_back({counts[s], s});
    std::fill(depth, depth + 256, 0u);
    const size_t m = leaves.size();
    if (m == 0) return 0;
    if (m == 1) {
        depth[leaves[0].sym] = 1;
        return 1;
    }
    std::sort(leaves.begin(), leaves.end(), [](const Leaf &a, const Leaf &b) {
        return a.w != b.w ? a.w < b.w : a.sym < b.sym;
    });
    // node ids: 0..m-1 leaves (sorted order), m.. merged nodes
    std::vector<uint64_t> weight(2 * m - 1);
    std::vector<int> parent(2 * m - 1, -1);
    for (size_t i = 0; i < m; ++i) weight[i] = leaves[i].w;
    size_t qa = 0, qb = m, next = m;
    auto pop = [&]() -> size_t {
        bool leaf_ok = qa < m;
        bool node_ok = qb < next;
        if (leaf_ok && (!node_ok || weight[qa] <= weight[qb])) return qa++;
        return qb++;
    };
    for (size_t k = 0; k + 1 < m; ++k) {
        size_t a = pop();
        size_t b = pop();
        weight[next] = weight[a] + weight[b];
        parent[a] = parent[b] = static_cast<int>(next);
        ++next;
    }
    // depth of a node = depth of its parent + 1; parents have larger ids
    std::vector<unsigned> d(2 * m - 1, 0);
    unsigned maxd = 0;
    for (size_t i = 2 * m - 1; i-- > 0;) {
        if (parent[i] >= 0) d[i] = d[parent[i]] + 1;
    }
    for (size_t i = 0; i < m; ++i) {
        depth[leaves[i].sym] = d[i];
        maxd = std::max(maxd, d[i]);
    }
    return maxd;
}

// Length-limited optimal lengths by package-merge (Larmore & Hirschberg).
// Lists are built from the deepest level up; the selection of the first
// 2m-2 items of the last list is propagated down as "how many items of each
// list are taken", and a symbol's length is the number of lists whose taken
// prefix contains its leaf.
int package_merge(const uint64_t *counts, unsigned cap, unsigned *len_out) {
    struct Leaf {
        uint64_t w;
        int sym;
    };
    std::vector<Leaf> leaves;
    for (int s = 0; s < 256; ++s)
        if (counts[s]) leaves.push_back({counts[s], s});
    std::fill(len_out, len_out + 256, 0u);
    const size_t m = leaves.size();
    if (m == 0) return DF11_OK;
    if (m == 1) {
        len_out[leaves[0].sym] = 1;
        return DF11_OK;
    }
    if (cap < 32 && (uint64_t{1} << cap) < m) return DF11_E_CAP_INFEASIBLE;
    std::sort(leaves.begin(), leaves.end(), [](const Leaf &a, const Leaf &b) {
        return a.w != b.w ? a.w < b.w : a.sym < b.sym;
    });
    std::vector<std::vector<uint64_t>> wt(cap);
    std::vector<std::vector<uint8_t>> is_leaf(cap);
    wt[0].resize(m);
    is_leaf[0].assign(m, 1);
    for (size_t i = 0; i < m; ++i) wt[0][i] = leaves[i].w;
    for (unsigned lv = 1; lv < cap; ++lv) {
        const auto &pw = wt[lv - 1];
        size_t npk = pw.size() / 2;
        size_t i = 0, j = 0;
        wt[lv].reserve(m + npk);
        is_leaf[lv].reserve(m + npk);
        while (i < m || j < npk) {
            uint64_t pkw = j < npk ? pw[2 * j] + pw[2 * j + 1] : 0;
            if (j >= npk || (i < m && leaves[i].w <= pkw)) {
                wt[lv].push_back(leaves[i].w);
                is_leaf[lv].push_back(1);
                ++i;
            } else {
                wt[lv].push_back(pkw);
                is_leaf[lv].push_back(0);
                ++j;
            }
        }
    }
    std::vector<size_t> leaves_taken(cap, 0);
    size_t take = 2 * m - 2;
    for (unsigned lv = cap; lv-- > 0;) {
        size_t nl = 0;
        for (size_t k = 0; k < take; ++k) nl += is_leaf[lv][k];
        leaves_taken[lv] = nl;
        take = 2 * (take - nl);
    }
    for (size_t r = 0; r < m; ++r) {
        unsigned l = 0;
        for (unsigned lv = 0; lv < cap; ++lv) l += (r < leaves_taken[lv]) ? 1u : 0u;
        len_out[leaves[r].sym] = l;
    }
    return DF11_OK;
}

// Canonical codes: count codes per length, first code per length, then
// hand out consecutive codes in exponent order within each length.
int assign_canonical(const uint8_t *len, uint32_t *code) {
    uint64_t per_len[33] = {0};
    for (int s = 0; s < 256; ++s) {
        if (len[s] > 32) return DF11_E_INVALID_ARG;
        if (len[s]) per_len[len[s]]++;
    }
    uint64_t first[34] = {0};
    uint64_t c = 0;
    for (unsigned l = 1; l <= 32; ++l) {
        c = (c + per_len[l - 1]) << 1;
        if (l == 1) c = 0;
        first[l] = c;
        if (per_len[l] && c + per_len[l] > (uint64_t{1} << l)) return DF11_E_INVALID_ARG;
    }
    uint64_t next[33];
    std::memcpy(next, first, sizeof(next));
    for (int s = 0; s < 256; ++s) {
        code[s] = 0;
        if (len[s]) code[s] = static_cast<uint32_t>(next[len[s]]++);
    }
    return DF11_OK;
}

uint64_t ceil_div(uint64_t a, uint64_t b) { return (a + b - 1) / b; }

bool layout_ok(const df11_layout *lay) {
    if (!lay) return false;
    if (lay->bytes_per_thread < 4 || lay->bytes_per_thread > 64) return false;
    if (lay->threads_per_block < 64 || lay->threads_per_block > 1024 ||
        lay->threads_per_block % 64)
        return false;
    if (lay->lut_bits < 8 || lay->lut_bits > 12) return false;
    return true;
}

}  // namespace

extern "C" {

const char *df11_strerror(int status) {
    switch (status) {
        case DF11_OK: return "ok";
        case DF11_E_INVALID_ARG: return "invalid argument";
        case DF11_E_CAP_INFEASIBLE: return "code length cap too small for the alphabet";
        case DF11_E_BUFFER_TOO_SMALL: return "buffer too small";
        case DF11_E_CORRUPT: return "corrupt stream";
        case DF11_E_HIP: return "HIP runtime error";
        case DF11_E_UNSUPPORTED: return "layout not supported by the decoder";
        default: return "unknown status";
    }
}

int df11_codebook_from_counts(const uint64_t counts[256], uint32_t max_code_len,
                              df11_codebook *out) {
    if (!counts || !out || max_code_len < 1 || max_code_len > 32) return DF11_E_INVALID_ARG;
    std::memset(out, 0, sizeof(*out));
    unsigned depth[256];
    unsigned maxd = huffman_depths(counts, depth);
    if (maxd > max_code_len) {
        int rc = package_merge(counts, max_code_len, depth);
        if (rc) return rc;
    }
    unsigned used = 0, maxl = 0;
    for (int s = 0; s < 256; ++s) {
        out->count[s] = counts[s];
        out->len[s] = static_cast<uint8_t>(depth[s]);
        if (depth[s]) {
            ++used;
            maxl = std::max(maxl, depth[s]);
        }
    }
    out->num_symbols = used;
    out->max_code_len = maxl;
    return assign_canonical(out->len, out->code);
}

int df11_build_codebook(const uint16_t *bf16, uint64_t n, uint32_t max_code_len,
                        df11_codebook *out) {
    if ((n && !bf16) || !out) return DF11_E_INVALID_ARG;
    unsigned parts = worker_count(n);
    std::vector<std::array<uint64_t, 256>> part_counts(parts);
    parallel_for(parts, [&](unsigned p) {
        auto &c = part_counts[p];
        c.fill(0);
        uint64_t lo = n * p / parts, hi = n * (p + 1) / parts;
        for (uint64_t i = lo; i < hi; ++i) c[exp_field(bf16[i])]++;
    });
    uint64_t counts[256] = {0};
    for (auto &c : part_counts)
        for (int s = 0; s < 256; ++s) counts[s] += c[s];
    return df11_codebook_from_counts(counts, max_code_len, out);
}

int df11_default_layout(uint64_t n, df11_layout *out) {
    if (!out) return DF11_E_INVALID_ARG;
    out->bytes_per_thread = 8;
    out->threads_per_block = n >= DF11_LARGE_STREAM_ELEMS ? 128 : 64;
    out->lut_bits = 11;
    return DF11_OK;
}

int df11_encoded_sizes(const df11_codebook *cb, const df11_layout *lay, df11_sizes *out) {
    if (!cb || !out || !layout_ok(lay)) return DF11_E_INVALID_ARG;
    uint64_t n = 0, bits = 0;
    for (int s = 0; s < 256; ++s) {
        if (cb->count[s] && !cb->len[s]) return DF11_E_INVALID_ARG;
        n += cb->count[s];
        bits += cb->count[s] * cb->len[s];
    }
    if (n > 0xFFFFFFFFull) return DF11_E_INVALID_ARG;  // BlockOutputPos is 32-bit
    if (cb->max_code_len > 32 || 8u * lay->bytes_per_thread < cb->max_code_len)
        return DF11_E_INVALID_ARG;
    std::memset(out, 0, sizeof(*out));
    const uint64_t n_bytes = lay->bytes_per_thread, T = lay->threads_per_block;
    out->n_elems = n;
    out->total_bits = bits;
    out->num_chunks = ceil_div(bits, 8 * n_bytes);
    out->num_blocks = ceil_div(out->num_chunks, T);
    out->exp_bytes = out->num_blocks * n_bytes * T + 16;
    out->sm_bytes = ((n + 15) & ~uint64_t{15}) + 16;  // zero padded for 16-byte reads
    out->gap_bytes = 4 * (ceil_div(5 * (out->num_blocks * T + 1), 32) + 2);
    out->block_pos_bytes = 4 * (out->num_blocks + 1);
    out->table_bytes = df11tab::blob_bytes(lay->lut_bits);
    out->max_code_len = cb->max_code_len;
    return DF11_OK;
}

int df11_encode(const uint16_t *bf16, uint64_t n, const df11_codebook *cb, const df11_layout *lay,
                uint8_t *exp, uint64_t exp_cap, uint8_t *sm, uint64_t sm_cap, uint8_t *gaps,
                uint64_t gap_cap, uint32_t *block_pos, uint64_t block_pos_cap, df11_sizes *out) {
    if ((n && !bf16) || !sm || !cb || !exp || !gaps || !block_pos || !out)
        return DF11_E_INVALID_ARG;
    df11_sizes sz;
    int rc = df11_encoded_sizes(cb, lay, &sz);
    if (rc) return rc;
    if (sz.n_elems != n) return DF11_E_INVALID_ARG;
    if (exp_cap < sz.exp_bytes || sm_cap < sz.sm_bytes || gap_cap < sz.gap_bytes ||
        block_pos_cap < sz.block_pos_bytes)
        return DF11_E_BUFFER_TOO_SMALL;

    const uint64_t chunk_bits = 8ull * lay->bytes_per_thread;
    const uint64_t block_bits = chunk_bits * lay->threads_per_block;
    const uint64_t slots = sz.num_blocks * lay->threads_per_block + 1;
    const uint64_t B = sz.num_blocks;
    const uint8_t *len = cb->len;
    const uint32_t *code = cb->code;

    // pass 1: bits per element range, and a check that the data matches cb
    unsigned parts = worker_count(n);
    std::vector<uint64_t> seg_bits(parts + 1, 0);
    std::atomic<bool> bad{false};
    parallel_for(parts, [&](unsigned p) {
        uint64_t lo = n * p / parts, hi = n * (p + 1) / parts, b = 0;
        for (uint64_t i = lo; i < hi; ++i) {
            unsigned l = len[exp_field(bf16[i])];
            if (!l) bad = true;
            b += l;
        }
        seg_bits[p + 1] = b;
    });
    if (bad) return DF11_E_INVALID_ARG;
    for (unsigned p = 0; p < parts; ++p) seg_bits[p + 1] += seg_bits[p];
    if (seg_bits[parts] != sz.total_bits) return DF11_E_INVALID_ARG;

    // zero the stream (padding included) and the unpacked gap slots
    std::vector<uint8_t> gap_slot(slots, 0);
    parallel_for(worker_count(sz.exp_bytes), [&](unsigned p) {
        unsigned P = worker_count(sz.exp_bytes);
        uint64_t lo = sz.exp_bytes * p / P, hi = sz.exp_bytes * (p + 1) / P;
        std::memset(exp + lo, 0, hi - lo);
    });

    // pass 2: pack codes, split sign/mantissa, record gaps and block starts.
    // A chunk (block) boundary X is owned by the first element whose code
    // start is >= X, so every slot is written by exactly one thread.
    std::vector<uint8_t> head(parts, 0), tail(parts, 0);
    std::vector<uint8_t> has_head(parts, 0), has_tail(parts, 0);
    parallel_for(parts, [&](unsigned p) {
        uint64_t lo = n * p / parts, hi = n * (p + 1) / parts;
        if (lo >= hi) return;
        uint64_t pos = seg_bits[p];
        uint64_t prev = lo ? pos - len[exp_field(bf16[lo - 1])] : 0;
        bool first_elem_global = (lo == 0);
        // bit writer: acc holds nacc pending bits (right aligned)
        uint64_t acc = 0;
        unsigned nacc = static_cast<unsigned>(pos & 7);
        uint64_t byte_at = pos >> 3;
        bool first_byte = (pos & 7) != 0;
        for (uint64_t i = lo; i < hi; ++i) {
            const uint16_t w = bf16[i];
            const unsigned e = exp_field(w);
            sm[i] = static_cast<uint8_t>(((w >> 8) & 0x80u) | (w & 0x7Fu));
            // boundaries in (prev, pos] are owned by element i
            uint64_t c0 = (first_elem_global && i == 0) ? 0 : prev / chunk_bits + 1;
            for (uint64_t c = c0; c * chunk_bits <= pos; ++c)
                gap_slot[c] = static_cast<uint8_t>(pos - c * chunk_bits);
            uint64_t b0 = (first_elem_global && i == 0) ? 0 : prev / block_bits + 1;
            for (uint64_t b = b0; b * block_bits <= pos && b <= B; ++b)
                block_pos[b] = static_cast<uint32_t>(i);
            const unsigned l = len[e];
            acc = (acc << l) | code[e];
            nacc += l;
            while (nacc >= 8) {
                uint8_t byte = static_cast<uint8_t>(acc >> (nacc - 8));
                if (first_byte) {
                    head[p] = byte;
                    has_head[p] = 1;
                    first_byte = false;
                } else {
                    exp[byte_at] = byte;
                }
                ++byte_at;
                nacc -= 8;
            }
            prev = pos;
            pos += l;
        }
        if (nacc) {
            uint8_t byte = static_cast<uint8_t>(acc << (8 - nacc));
            if (first_byte) {
                head[p] = byte;
                has_head[p] = 1;
            } else {
                tail[p] = byte;
                has_tail[p] = 1;
            }
        }
    });
    std::memset(sm + n, 0, sz.sm_bytes - n);
    for (unsigned p = 0; p < parts; ++p) {
        uint64_t lo = n * p / parts, hi = n * (p + 1) / parts;
        if (lo >= hi) continue;
        if (has_head[p]) exp[seg_bits[p] >> 3] |= head[p];
        if (has_tail[p]) exp[seg_bits[p + 1] >> 3] |= tail[p];
    }
    // boundaries after the last code start: the end of the stream is a start
    {
        uint64_t total = sz.total_bits;
        uint64_t last = n ? total - len[exp_field(bf16[n - 1])] : 0;
        uint64_t c0 = n ? last / chunk_bits + 1 : 0;
        for (uint64_t c = c0; c < slots && c * chunk_bits <= total; ++c)
            gap_slot[c] = static_cast<uint8_t>(total - c * chunk_bits);
        uint64_t b0 = n ? last / block_bits + 1 : 0;
        for (uint64_t b = b0; b <= B; ++b) block_pos[b] = static_cast<uint32_t>(n);
    }
    // pack the gaps, 5 bits each, most significant first; 8 slots = 5 bytes
    std::memset(gaps, 0, sz.gap_bytes);
    const uint64_t groups = ceil_div(slots, 8);
    unsigned gparts = worker_count(groups * 64);
    parallel_for(gparts, [&](unsigned p) {
        uint64_t lo = groups * p / gparts, hi = groups * (p + 1) / gparts;
        for (uint64_t g = lo; g < hi; ++g) {
            uint64_t v = 0;
            for (unsigned k = 0; k < 8; ++k) {
                uint64_t c = 8 * g + k;
                v = (v << 5) | (c < slots ? (gap_slot[c] & 31u) : 0u);
            }
            for (unsigned k = 0; k < 5; ++k) gaps[5 * g + k] = static_cast<uint8_t>(v >> (32 - 8 * k));
        }
    });
    uint32_t max_per_block = 0;
    for (uint64_t b = 0; b < B; ++b)
        max_per_block = std::max(max_per_block, block_pos[b + 1] - block_pos[b]);
    sz.max_elems_per_block = max_per_block;
    *out = sz;
    return DF11_OK;
}

int df11_build_tables(const df11_codebook *cb, uint32_t lut_bits, uint8_t *tables,
                      uint64_t table_cap) {
    if (!cb || !tables || lut_bits < 8 || lut_bits > 12) return DF11_E_INVALID_ARG;
    if (table_cap < df11tab::blob_bytes(lut_bits)) return DF11_E_BUFFER_TOO_SMALL;
    return df11tab::build(cb->len, cb->code, cb->max_code_len, lut_bits, tables);
}

int df11_validate(const df11_stream *s) {
    if (!s) return DF11_E_INVALID_ARG;
    const df11_sizes &z = s->sizes;
    if (!layout_ok(&s->layout)) return DF11_E_INVALID_ARG;
    if (z.n_elems && (!s->exp || !s->sm || !s->gaps || !s->block_pos || !s->tables))
        return DF11_E_INVALID_ARG;
    const uint64_t n_bytes = s->layout.bytes_per_thread, T = s->layout.threads_per_block;
    if (z.max_code_len > 32 || z.max_code_len > 8 * n_bytes) return DF11_E_CORRUPT;
    if (z.n_elems > 0xFFFFFFFFull || z.sm_bytes != ((z.n_elems + 15) & ~uint64_t{15}) + 16)
        return DF11_E_CORRUPT;
    if (z.num_chunks != ceil_div(z.total_bits, 8 * n_bytes)) return DF11_E_CORRUPT;
    if (z.num_blocks != ceil_div(z.num_chunks, T)) return DF11_E_CORRUPT;
    if (z.exp_bytes != z.num_blocks * n_bytes * T + 16) return DF11_E_CORRUPT;
    if (z.gap_bytes != 4 * (ceil_div(5 * (z.num_blocks * T + 1), 32) + 2)) return DF11_E_CORRUPT;
    if (z.block_pos_bytes != 4 * (z.num_blocks + 1)) return DF11_E_CORRUPT;
    if (z.table_bytes != df11tab::blob_bytes(s->layout.lut_bits)) return DF11_E_CORRUPT;
    if (z.n_elems == 0) return DF11_OK;
    if (z.total_bits < z.n_elems || z.total_bits > 32 * z.n_elems) return DF11_E_CORRUPT;
    // BlockOutputPos
    const uint32_t *bp = s->block_pos;
    if (bp[0] != 0 || bp[z.num_blocks] != z.n_elems) return DF11_E_CORRUPT;
    uint32_t mx = 0;
    for (uint64_t b = 0; b < z.num_blocks; ++b) {
        if (bp[b + 1] < bp[b]) return DF11_E_CORRUPT;
        mx = std::max(mx, bp[b + 1] - bp[b]);
        if (static_cast<uint64_t>(bp[b + 1] - bp[b]) > 8 * n_bytes * T) return DF11_E_CORRUPT;
    }
    if (mx != z.max_elems_per_block) return DF11_E_CORRUPT;
    // Gaps: every slot below the code-length cap; slots past the end are 0
    const uint64_t slots = z.num_blocks * T + 1;
    const uint32_t lim = z.max_code_len ? z.max_code_len : 1;
    for (uint64_t c = 0; c < slots; ++c) {
        uint64_t bit = 5 * c;
        unsigned v = 0;
        for (unsigned j = 0; j < 5; ++j, ++bit)
            v = (v << 1) | ((s->gaps[bit >> 3] >> (7 - (bit & 7))) & 1u);
        if (v >= lim && !(v == 0)) return DF11_E_CORRUPT;
        if (8 * n_bytes * c > z.total_bits && v) return DF11_E_CORRUPT;
        if (8 * n_bytes * c <= z.total_bits && 8 * n_bytes * c + v > z.total_bits)
            return DF11_E_CORRUPT;
    }
    return df11tab::check(s->tables, s->layout.lut_bits, z.max_code_len);
}

}  // extern "C"
