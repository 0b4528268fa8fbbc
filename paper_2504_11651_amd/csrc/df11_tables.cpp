// Builds and checks the decode-table blob described in df11_tables.h.
#include "df11_tables.h"

#include <cstring>
#include <vector>

#include "df11.h"

namespace df11tab {

namespace {

struct Canon {
    uint64_t per_len[33];
    uint64_t first[33];
    uint32_t base[33];  // symbols with a shorter code
    uint8_t sorted[256];
    unsigned nsym;
};

void canon_from_lengths(const uint8_t *len, Canon &cn) {
    std::memset(&cn, 0, sizeof(cn));
    for (int s = 0; s < 256; ++s)
        if (len[s]) cn.per_len[len[s]]++;
    uint64_t c = 0;
    unsigned k = 0;
    for (unsigned l = 1; l <= 32; ++l) {
        c = (c + cn.per_len[l - 1]) << 1;
        if (l == 1) c = 0;
        cn.first[l] = c;
        cn.base[l] = k;
        for (int s = 0; s < 256; ++s)
            if (len[s] == l) cn.sorted[k++] = static_cast<uint8_t>(s);
    }
    cn.nsym = k;
}

// First code of the window bits [pos, K) of x (window bit j = bit j of x,
// read first to last); returns its length, 0 when no whole code fits.
unsigned first_code(const Canon &cn, uint32_t x, unsigned pos, unsigned K, unsigned *sym) {
    uint64_t c = 0;
    for (unsigned l = 1; pos + l <= K; ++l) {
        c = (c << 1) | ((x >> (pos + l - 1)) & 1u);
        if (cn.per_len[l] && c >= cn.first[l] && c < cn.first[l] + cn.per_len[l]) {
            *sym = cn.sorted[cn.base[l] + (c - cn.first[l])];
            return l;
        }
    }
    return 0;
}

void put32(uint8_t *p, uint32_t v) { std::memcpy(p, &v, 4); }
uint32_t get32(const uint8_t *p) {
    uint32_t v;
    std::memcpy(&v, p, 4);
    return v;
}

}  // namespace

int build(const uint8_t *len, const uint32_t *code, uint32_t max_len, uint32_t K, uint8_t *blob) {
    (void)code;  // canonical codes follow from the lengths
    Canon cn;
    canon_from_lengths(len, cn);
    std::memset(blob, 0, blob_bytes(K));
    put32(blob + 0, kMagic);
    put32(blob + 4, K);
    put32(blob + 8, max_len);
    uint8_t *ent = blob + kHeaderBytes;
    const uint32_t nent = 1u << K;
    for (uint32_t x = 0; x < nent; ++x) {
        uint32_t syms = 0, mask = 0;
        unsigned pos = 0, n = 0;
        while (n < 4) {
            unsigned s = 0;
            unsigned l = first_code(cn, x, pos, K, &s);
            if (!l) break;
            syms |= s << (8 * n);
            mask |= 1u << pos;
            ++n;
            pos += l;
        }
        uint32_t meta = n ? (pos | (n << 8) | (mask << 16)) : 0u;
        put32(ent + 8ull * x, syms);
        put32(ent + 8ull * x + 4, meta);
    }
    uint8_t *esc = ent + entry_bytes(K);
    for (unsigned l = 0; l < kEscWords; ++l) {
        uint32_t lj = 0xFFFFFFFFu, off = 0;
        if (l >= 1 && l <= max_len) {
            uint64_t lim = (cn.first[l] + cn.per_len[l]) << (32 - l);
            lj = static_cast<uint32_t>(lim - 1);
            off = cn.base[l] - static_cast<uint32_t>(cn.first[l]);
        }
        put32(esc + 4 * l, lj);
        put32(esc + 4 * (kEscWords + l), off);
    }
    std::memcpy(esc + 8 * kEscWords, cn.sorted, 256);
    return DF11_OK;
}

int check(const uint8_t *blob, uint32_t K, uint32_t max_len) {
    if (get32(blob) != kMagic || get32(blob + 4) != K || get32(blob + 8) != max_len ||
        max_len > 32)
        return DF11_E_CORRUPT;
    // The code the blob describes, read back from its escape arrays: the
    // canonical codes of length L are [first[L], end[L]) with end[L] =
    // (lj_last[L] + 1) >> (32 - L) and first[L+1] = 2 * end[L].  Below the
    // shortest length (first = 0, no code yet) lj_last is 2^32 - 1, which
    // at the longest length instead means end = 2^L (a complete code).
    const uint8_t *esc = blob + kHeaderBytes + entry_bytes(K);
    const uint8_t *sorted = esc + 8 * kEscWords;
    uint8_t len[256] = {0};
    uint64_t first = 0, nsym = 0, kraft = 0;  // kraft: sum of 2^(32-L), exact in 64 bits
    for (unsigned l = 1; l <= max_len; ++l) {
        const uint32_t lj = get32(esc + 4 * l);
        const uint64_t end = (first == 0 && lj == 0xFFFFFFFFu && l < max_len)
                                 ? 0
                                 : (static_cast<uint64_t>(lj) + 1) >> (32 - l);
        if (end < first || end > (uint64_t{1} << l)) return DF11_E_CORRUPT;
        const uint64_t count = end - first;
        if (nsym + count > 256) return DF11_E_CORRUPT;
        for (uint64_t i = 0; i < count; ++i) {
            const uint8_t sym = sorted[nsym + i];
            // exponents of one length in increasing order, each used once
            if (len[sym] || (i && sym <= sorted[nsym + i - 1])) return DF11_E_CORRUPT;
            len[sym] = static_cast<uint8_t>(l);
        }
        kraft += count << (32 - l);
        nsym += count;
        first = end << 1;
    }
    // a complete prefix code (Kraft sum 1) for two or more symbols; a lone
    // symbol has the one-bit code 0
    if (nsym == 0 || (nsym == 1 ? len[sorted[0]] != 1 : kraft != (uint64_t{1} << 32)))
        return DF11_E_CORRUPT;
    if (len[sorted[nsym - 1]] != max_len) return DF11_E_CORRUPT;
    // everything else (the K-bit entries, offsets, padding) follows from the
    // lengths: rebuild and compare byte for byte
    std::vector<uint8_t> again(blob_bytes(K));
    if (build(len, nullptr, max_len, K, again.data()) != DF11_OK) return DF11_E_CORRUPT;
    return std::memcmp(again.data(), blob, again.size()) ? DF11_E_CORRUPT : DF11_OK;
}

}  // namespace df11tab
