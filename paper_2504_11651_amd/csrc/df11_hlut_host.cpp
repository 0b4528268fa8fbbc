// Hierarchical lookup tables of the paper's own decoder (Sec. 2.3.1 and the
// appendix on compact lookup tables), for the ablation kernel in
// df11_hlut.hip.
//
// The canonical Huffman tree is cut into subtrees of height b (b = 8 for the
// decoder): table LUT_1 is indexed by the first b bits of the window; an
// entry holds either the exponent whose code is a prefix of those bits, or,
// when the bits are the prefix of longer codes, a pointer to the table that
// decodes the next b bits.  Pointers are the exponent values 240..255, which
// the paper reserves for this (they are magnitudes of 2^113 and above): value
// v points to LUT_(257 - v), so LUT_2 .. LUT_17 can be referenced.  A code
// book that uses an exponent of 240 or more, or that needs more than 17
// tables, cannot be expressed this way (DF11_E_UNSUPPORTED).  CodeLengths
// maps each exponent to its code length.
//
// Blob: LUT_1 .. LUT_k (2^b bytes each, in the order the tables are created:
// breadth first from the root), then CodeLengths[256].
#include <cstdint>
#include <cstring>
#include <vector>

#include "df11.h"

namespace {

constexpr uint32_t kMaxLuts = 17;     // LUT_1 plus the 16 pointer values
constexpr uint32_t kFirstPointer = 240;

struct Prefix {
    uint64_t bits;   // the first `depth` bits of every code below this table
    uint32_t depth;  // multiple of b
};

}  // namespace

extern "C" int df11_build_hlut_tables(const df11_codebook *cb, uint32_t level_bits,
                                      uint8_t *tables, uint64_t table_cap, uint32_t *num_luts) {
    if (!cb || !num_luts || level_bits < 1 || level_bits > 8 || cb->max_code_len > 32)
        return DF11_E_INVALID_ARG;
    const uint32_t b = level_bits, ent = 1u << b;
    for (int s = 0; s < 256; ++s) {
        if (cb->len[s] > 32) return DF11_E_INVALID_ARG;
        if (cb->len[s] && s >= static_cast<int>(kFirstPointer)) return DF11_E_UNSUPPORTED;
    }
    std::vector<Prefix> todo{{0, 0}};
    std::vector<uint8_t> luts;
    for (size_t t = 0; t < todo.size(); ++t) {
        const Prefix pre = todo[t];
        const uint32_t d = pre.depth + b;  // bits resolved once this table is read
        const size_t base = luts.size();
        luts.resize(base + ent, 0);
        for (uint32_t x = 0; x < ent; ++x) {
            const uint64_t s = (pre.bits << b) | x;  // d bits
            bool done = false, longer = false;
            for (int e = 0; e < 256 && !done; ++e) {
                const uint32_t l = cb->len[e];
                if (!l) continue;
                const uint64_t c = cb->code[e];
                if (l <= d) {
                    // the code is a prefix of s, and it starts below this table
                    if (l > pre.depth && (s >> (d - l)) == c) {
                        luts[base + x] = static_cast<uint8_t>(e);
                        done = true;
                    }
                } else if ((c >> (l - d)) == s) {
                    longer = true;  // s is a proper prefix of this code
                }
            }
            if (done || !longer) continue;  // no code at all: an unreachable entry (0)
            if (todo.size() >= kMaxLuts) return DF11_E_UNSUPPORTED;
            luts[base + x] = static_cast<uint8_t>(257u - (todo.size() + 1));
            todo.push_back({s, d});
        }
    }
    const uint32_t k = static_cast<uint32_t>(todo.size());
    *num_luts = k;
    const uint64_t need = static_cast<uint64_t>(k) * ent + 256;
    if (!tables || table_cap < need) return DF11_E_BUFFER_TOO_SMALL;
    std::memcpy(tables, luts.data(), luts.size());
    for (int e = 0; e < 256; ++e) tables[luts.size() + e] = cb->len[e];
    return DF11_OK;
}
