// Host-only cross-check of the library's host codec (df11_host.cpp,
// df11_tables.cpp) against the CPU oracle (oracle/df11_oracle.c), built with
// sanitizers: AddressSanitizer + UndefinedBehaviorSanitizer, or
// ThreadSanitizer for the multi-threaded histogram and encoder.  Test
// infrastructure: tests/test_sanitize.py compiles and runs it.
//
// For each seeded input and layout: the library builds the code book,
// stream, metadata and tables and validates them; the oracle does every step
// of the format by its own definitions (Sec. 2.3, 2.3.2, Algorithm 1); the
// two must agree byte for byte, and the oracle's bit-serial and
// metadata-driven decodes of the library's stream must give back the input.
// Exit status 0 = all agree; messages on stderr name the failing case.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "df11.h"

extern "C" {
int dfo_histogram(const uint16_t *w, uint64_t n, uint64_t counts[256]);
int dfo_code_lengths(const uint64_t counts[256], unsigned max_len, uint8_t lengths[256]);
int dfo_canonical_codes(const uint8_t lengths[256], uint32_t codes[256]);
int dfo_layout(uint64_t total_bits, unsigned n_bytes, unsigned threads, uint64_t *num_chunks,
               uint64_t *num_blocks, uint64_t *exp_bytes, uint64_t *gap_bytes);
int dfo_encode(const uint16_t *w, uint64_t n, const uint8_t lengths[256],
               const uint32_t codes[256], uint8_t *exp, uint64_t exp_cap, uint8_t *sm,
               uint64_t *total_bits);
int dfo_metadata(const uint16_t *w, uint64_t n, const uint8_t lengths[256], unsigned n_bytes,
                 unsigned threads, uint8_t *gaps, uint64_t slots, uint32_t *block_pos,
                 uint64_t bp_count);
int dfo_pack_gaps(const uint8_t *gaps, uint64_t slots, uint8_t *packed, uint64_t packed_bytes);
int dfo_decode_serial(const uint8_t *exp, uint64_t total_bits, const uint8_t *sm, uint64_t n,
                      const uint8_t lengths[256], uint16_t *out);
int dfo_decode_blocks(const uint8_t *exp, uint64_t total_bits, const uint8_t *sm, uint64_t n,
                      const uint8_t lengths[256], unsigned n_bytes, unsigned threads,
                      const uint8_t *gaps, const uint32_t *block_pos, uint64_t first_block,
                      uint64_t num_blocks, uint16_t *out);
}

namespace {

int failures = 0;

#define EXPECT(cond, ...)                                        \
    do {                                                         \
        if (!(cond)) {                                           \
            std::fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
            std::fprintf(stderr, __VA_ARGS__);                   \
            std::fprintf(stderr, "\n");                          \
            ++failures;                                          \
            return;                                              \
        }                                                        \
    } while (0)

// splitmix64: seeded input only
struct Rng {
    uint64_t s;
    uint64_t next() {
        uint64_t z = (s += 0x9E3779B97F4A7C15ull);
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        return z ^ (z >> 31);
    }
    double uniform() { return (next() >> 11) * (1.0 / 9007199254740992.0); }
};

uint16_t to_bf16(float f) {  // round to nearest, ties to even
    uint32_t u;
    std::memcpy(&u, &f, 4);
    return static_cast<uint16_t>((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

std::vector<uint16_t> make_input(int kind, uint64_t n, uint64_t seed) {
    Rng r{seed};
    std::vector<uint16_t> w(n);
    for (uint64_t i = 0; i < n; ++i) {
        switch (kind) {
            case 0: {  // N(0, 0.02^2) by Box-Muller
                const double u1 = r.uniform() + 1e-300, u2 = r.uniform();
                w[i] = to_bf16(static_cast<float>(0.02 * std::sqrt(-2 * std::log(u1)) *
                                                  std::cos(6.283185307179586 * u2)));
                break;
            }
            case 1: w[i] = static_cast<uint16_t>(i * 40503u + seed); break;  // every pattern
            case 2: w[i] = 0x3F80; break;                                   // one exponent
            default: {  // geometric exponents: long codes, forces small caps to bind
                unsigned e = 100;
                while (e < 140 && (r.next() & 1)) ++e;
                w[i] = static_cast<uint16_t>((r.next() & 0x807Fu) | (e << 7));
            }
        }
    }
    return w;
}

void check(int kind, uint64_t n, uint64_t seed, unsigned cap, df11_layout lay) {
    const std::vector<uint16_t> w = make_input(kind, n, seed);
    df11_codebook cb;
    int rc = df11_build_codebook(w.data(), n, cap, &cb);
    EXPECT(rc == DF11_OK, "kind %d n %llu: build_codebook %d", kind, (unsigned long long)n, rc);
    df11_sizes z;
    EXPECT(df11_encoded_sizes(&cb, &lay, &z) == DF11_OK, "encoded_sizes");
    std::vector<uint8_t> exp(z.exp_bytes), sm(z.sm_bytes), gaps(z.gap_bytes), tab(z.table_bytes);
    std::vector<uint32_t> bp(z.num_blocks + 1);
    df11_sizes out;
    rc = df11_encode(w.data(), n, &cb, &lay, exp.data(), exp.size(), sm.data(), sm.size(),
                     gaps.data(), gaps.size(), bp.data(), 4 * bp.size(), &out);
    EXPECT(rc == DF11_OK, "encode %d", rc);
    EXPECT(df11_build_tables(&cb, lay.lut_bits, tab.data(), tab.size()) == DF11_OK, "tables");
    df11_stream st{exp.data(), sm.data(), gaps.data(), bp.data(), tab.data(), out, lay};
    if (n) EXPECT(df11_validate(&st) == DF11_OK, "validate");

    // the oracle, step by step
    uint64_t counts[256];
    uint8_t len[256];
    uint32_t codes[256];
    EXPECT(dfo_histogram(w.data(), n, counts) == 0, "oracle histogram");
    if (n == 0) return;
    EXPECT(dfo_code_lengths(counts, cap, len) == 0, "oracle lengths");
    EXPECT(dfo_canonical_codes(len, codes) == 0, "oracle codes");
    for (int s = 0; s < 256; ++s) {
        EXPECT(cb.count[s] == counts[s] && cb.len[s] == len[s] && (!len[s] || cb.code[s] == codes[s]),
               "kind %d n %llu: code book differs at exponent %d", kind, (unsigned long long)n, s);
    }
    uint64_t C, B, exp_bytes, gap_bytes, tb = 0;
    dfo_layout(out.total_bits, lay.bytes_per_thread, lay.threads_per_block, &C, &B, &exp_bytes,
               &gap_bytes);
    EXPECT(C == out.num_chunks && B == out.num_blocks && exp_bytes == out.exp_bytes &&
               gap_bytes == out.gap_bytes, "layout");
    std::vector<uint8_t> oexp(exp_bytes), osm(n);
    EXPECT(dfo_encode(w.data(), n, len, codes, oexp.data(), exp_bytes, osm.data(), &tb) == 0,
           "oracle encode");
    EXPECT(tb == out.total_bits, "total bits");
    EXPECT(oexp == exp, "kind %d n %llu: EncodedExponent differs", kind, (unsigned long long)n);
    EXPECT(std::memcmp(osm.data(), sm.data(), n) == 0, "PackedSignMantissa differs");
    const uint64_t slots = B * lay.threads_per_block + 1;
    std::vector<uint8_t> ogaps(slots), opacked(gap_bytes);
    std::vector<uint32_t> obp(B + 1);
    EXPECT(dfo_metadata(w.data(), n, len, lay.bytes_per_thread, lay.threads_per_block,
                        ogaps.data(), slots, obp.data(), B + 1) == 0, "oracle metadata");
    EXPECT(dfo_pack_gaps(ogaps.data(), slots, opacked.data(), gap_bytes) == 0, "pack");
    EXPECT(opacked == gaps, "Gaps differ");
    EXPECT(obp == bp, "BlockOutputPos differs");

    std::vector<uint16_t> dec(n, 0x5555);
    EXPECT(dfo_decode_serial(exp.data(), out.total_bits, sm.data(), n, len, dec.data()) == 0,
           "oracle serial decode");
    EXPECT(dec == w, "serial round trip");
    std::fill(dec.begin(), dec.end(), 0x5555);
    EXPECT(dfo_decode_blocks(exp.data(), out.total_bits, sm.data(), n, len, lay.bytes_per_thread,
                             lay.threads_per_block, ogaps.data(), bp.data(), 0, B, dec.data()) == 0,
           "oracle block decode");
    EXPECT(dec == w, "block round trip");
}

}  // namespace

int main(int argc, char **argv) {
    // argv[1] = "large" adds inputs big enough for the encoder's threads
    const bool large = argc > 1 && std::strcmp(argv[1], "large") == 0;
    const uint64_t sizes[] = {0, 1, 7, 64, 1000, 65537, 300000};
    const df11_layout lays[] = {{8, 64, 11}, {8, 256, 8}, {8, 1024, 12}, {4, 128, 10}};
    uint64_t seed = 1;
    for (int kind = 0; kind < 4; ++kind)
        for (uint64_t n : sizes)
            for (const df11_layout &lay : lays) {
                if (8 * lay.bytes_per_thread < 32 && kind == 3) continue;  // codes past 32 bits
                check(kind, n, seed++, 32, lay);
                if (kind == 3 && lay.bytes_per_thread == 8) check(kind, n, seed++, 12, lay);
            }
    if (large) {
        check(0, 5u << 20, 99, 32, {8, 64, 11});
        check(3, 3u << 20, 98, 14, {8, 256, 12});
    }
    std::printf("%s: %d failures\n", large ? "host_check large" : "host_check", failures);
    return failures ? 1 : 0;
}
