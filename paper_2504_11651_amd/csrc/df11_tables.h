// Decode-table blob of this library (internal).
//
// The paper decodes with a flat 2^L prefix table plus a CodeLengths table
// (appendix on lookup-table decoding), split into a hierarchy of 256-entry
// tables to fit GPU SRAM (Sec. 2.3.1).  This library uses one K-bit table
// (8 <= K <= 12) whose entry decodes up to four whole codes at once, and a
// canonical length search for the rare codes longer than K bits.
//
// Blob layout (little endian):
//   [0, 16)                header: magic "DFLT", K, max code length, 0
//   [16, 16 + 8*2^K)       entries, one uint64 per K-bit window:
//                            bits  0..31  up to four exponents, first in the
//                                         low byte, unused bytes zero
//                            bits 32..39  bits consumed by those codes
//                            bits 40..47  number of codes (0 = escape)
//                            bits 48..59  code start mask: bit j set when a
//                                         decoded code starts j bits into
//                                         the window
//                          window bit j = stream bit (start + j), so the
//                          first stream bit is the least significant bit
//   then uint32 lj_last[33]  lj_last[L] = largest 32-bit left-justified
//                            window whose code has length <= L
//   then uint32 offset[33]   index of the first length-L code in sym_sorted
//                            minus the first length-L code (mod 2^32)
//   then uint8 sym_sorted[256] exponents ordered by (length, value)
//   zero padding to a multiple of 16 bytes.
// Everything after the header is copied to LDS verbatim by the decoder.
#pragma once
#include <cstdint>

namespace df11tab {

constexpr uint32_t kMagic = 0x544C4644u;  // "DFLT"
constexpr uint32_t kHeaderBytes = 16;
constexpr uint32_t kEscWords = 33;

inline uint64_t entry_bytes(uint32_t lut_bits) { return 8ull << lut_bits; }
inline uint64_t lds_bytes(uint32_t lut_bits) {
    uint64_t b = entry_bytes(lut_bits) + 2 * 4 * kEscWords + 256;
    return (b + 15) & ~uint64_t{15};
}
inline uint64_t blob_bytes(uint32_t lut_bits) { return kHeaderBytes + lds_bytes(lut_bits); }

int build(const uint8_t *len, const uint32_t *code, uint32_t max_len, uint32_t lut_bits,
          uint8_t *blob);
// DF11_OK when the blob is exactly what build() makes for some code book
// with this table width and longest code: its escape arrays describe a
// canonical code that is a complete prefix code (Kraft sum 1; one symbol:
// a one-bit code), and every other byte equals the rebuilt blob's.
int check(const uint8_t *blob, uint32_t lut_bits, uint32_t max_len);

}  // namespace df11tab
