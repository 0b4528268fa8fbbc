/*
 * DFloat11 CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously-correct C implementation of what the DFloat11
 * decompression path computes (arXiv 2504.11651).  Only the test-suite,
 * the smoke check and the benchmark's CPU-baseline leg load it.  It shares
 * no code, header, table or constant with the product library: it is built
 * by its own command from this single file.
 *
 * Every step follows a passage of the paper:
 *   - BF16 field split ............ Sec. 2.1, Eq. (1); Algorithm 1 (assembly
 *                                   of sign, exponent and mantissa)
 *   - exponent histogram .......... Sec. 2.2 / 2.3 (Huffman tree built from the
 *                                   distribution of exponents)
 *   - Huffman code lengths ........ Sec. 2.1 "Entropy coding" (optimal prefix
 *                                   code, repeatedly merge the two lightest)
 *   - length cap (<= 32 bits) ..... Sec. 2.3.1 and 2.3.2 (L ranges 24..32;
 *                                   gaps fit 5 bits because L <= 32).  The paper
 *                                   does not say how the cap is enforced; the
 *                                   oracle uses package-merge (Larmore and
 *                                   Hirschberg 1990) when plain Huffman is deeper.
 *   - canonical code assignment ... Appendix "dual lookup table" worked example
 *                                   (A=0, B=100, C=101, D=110, E=1110, F=1111)
 *   - encoding .................... Sec. 2.3: codes tightly bit-packed into the
 *                                   byte array EncodedExponent (MSB first);
 *                                   sign+mantissa kept raw in PackedSignMantissa
 *   - Gaps / BlockOutputPos ....... Sec. 2.3.2 and Algorithm 1, computed by brute
 *                                   force from the code start positions
 *   - bit-serial tree decode ...... Appendix "dual lookup table": walk the
 *                                   Huffman tree one bit at a time
 *   - metadata-driven decode ...... Algorithm 1 semantics (each thread decodes the
 *                                   codes that start in its n-byte chunk; output
 *                                   position = block position + earlier counts)
 *
 * Conventions where the paper is silent (each is a stated reading):
 *   - stream bit k lives in byte k/8, bit 7-(k%8) (most significant first);
 *   - Huffman ties: among equal weights a leaf is taken before an internal
 *     node, leaves in increasing symbol order, internal nodes in creation
 *     order; package-merge ties: leaf before package;
 *   - one used symbol gets code length 1;
 *   - Gaps[c] = (first code start >= 8n*c, with total_bits counted as a start)
 *     - 8n*c, and 0 for a chunk that starts past total_bits;
 *   - BlockOutputPos has B+1 entries, BlockOutputPos[b] = number of codes that
 *     start before bit 8nT*b.
 *
 * Return codes: 0 = ok, negative = error (see DFO_E_* below).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define DFO_OK 0
#define DFO_E_ARG (-1)
#define DFO_E_CAP (-2)
#define DFO_E_SPACE (-3)
#define DFO_E_STREAM (-4)

/* ------------------------------------------------------------------ */
/* BF16 fields, Eq. (1): 1 sign bit, 8 exponent bits, 7 mantissa bits  */
/* ------------------------------------------------------------------ */
static unsigned exponent_of(uint16_t w) { return (w >> 7) & 0xFFu; }
static unsigned sign_of(uint16_t w) { return (w >> 15) & 1u; }
static unsigned mantissa_of(uint16_t w) { return w & 0x7Fu; }

/* PackedSignMantissa byte: sign in bit 7, mantissa in bits 6..0
 * (Algorithm 1 masks the byte with 0b10000000 and 0b01111111). */
static uint8_t sign_mantissa_byte(uint16_t w) {
    return (uint8_t)((sign_of(w) << 7) | mantissa_of(w));
}

/* Reassembly, Algorithm 1: (Sign << 8) | (Exponent << 7) | Mantissa with
 * Sign = byte & 0x80 and Mantissa = byte & 0x7F. */
static uint16_t assemble(uint8_t sm, unsigned e) {
    unsigned sign = sm & 0x80u;
    unsigned mant = sm & 0x7Fu;
    return (uint16_t)((sign << 8) | (e << 7) | mant);
}

/* ------------------------------------------------------------------ */
/* Exponent histogram                                                  */
/* ------------------------------------------------------------------ */
int dfo_histogram(const uint16_t *w, uint64_t n, uint64_t counts[256]) {
    if (!counts || (n && !w)) return DFO_E_ARG;
    for (int s = 0; s < 256; ++s) counts[s] = 0;
    for (uint64_t i = 0; i < n; ++i) counts[exponent_of(w[i])] += 1;
    return DFO_OK;
}

/* ------------------------------------------------------------------ */
/* Textbook Huffman: repeatedly merge the two lightest nodes.          */
/* O(m^2) selection, on purpose: easy to check by eye.                 */
/* ------------------------------------------------------------------ */
typedef struct {
    uint64_t weight;
    int is_internal; /* 0 leaf, 1 internal */
    int order;       /* leaf: symbol value; internal: creation index */
    int child[2];    /* internal only: node indices */
    int alive;
} hnode;

/* a < b in the tie-break order: weight, then leaf before internal, then order */
static int hnode_less(const hnode *a, const hnode *b) {
    if (a->weight != b->weight) return a->weight < b->weight;
    if (a->is_internal != b->is_internal) return a->is_internal < b->is_internal;
    return a->order < b->order;
}

static void set_depths(const hnode *nodes, int idx, unsigned depth, unsigned *depth_of_sym) {
    if (!nodes[idx].is_internal) {
        depth_of_sym[nodes[idx].order] = depth;
        return;
    }
    set_depths(nodes, nodes[idx].child[0], depth + 1, depth_of_sym);
    set_depths(nodes, nodes[idx].child[1], depth + 1, depth_of_sym);
}

/* Unconstrained Huffman code lengths.  Returns the maximum length, 0 when
 * no symbol is used.  Lengths are written as unsigned (they can exceed 32). */
int dfo_huffman_lengths(const uint64_t counts[256], unsigned lengths[256]) {
    hnode nodes[512];
    int nn = 0, used = 0;
    for (int s = 0; s < 256; ++s) lengths[s] = 0;
    for (int s = 0; s < 256; ++s) {
        if (counts[s] == 0) continue;
        nodes[nn].weight = counts[s];
        nodes[nn].is_internal = 0;
        nodes[nn].order = s;
        nodes[nn].alive = 1;
        ++nn;
        ++used;
    }
    if (used == 0) return 0;
    if (used == 1) {
        lengths[nodes[0].order] = 1;
        return 1;
    }
    int created = 0;
    for (int step = 0; step < used - 1; ++step) {
        int pick[2];
        for (int k = 0; k < 2; ++k) {
            int best = -1;
            for (int i = 0; i < nn; ++i) {
                if (!nodes[i].alive) continue;
                if (best < 0 || hnode_less(&nodes[i], &nodes[best])) best = i;
            }
            nodes[best].alive = 0;
            pick[k] = best;
        }
        nodes[nn].weight = nodes[pick[0]].weight + nodes[pick[1]].weight;
        nodes[nn].is_internal = 1;
        nodes[nn].order = created++;
        nodes[nn].child[0] = pick[0];
        nodes[nn].child[1] = pick[1];
        nodes[nn].alive = 1;
        ++nn;
    }
    unsigned depth[256] = {0};
    set_depths(nodes, nn - 1, 0, depth);
    unsigned maxlen = 0;
    for (int s = 0; s < 256; ++s) {
        if (counts[s] == 0) continue;
        lengths[s] = depth[s];
        if (depth[s] > maxlen) maxlen = depth[s];
    }
    return (int)maxlen;
}

/* ------------------------------------------------------------------ */
/* Package-merge: optimal code lengths under a maximum length.         */
/* Items of each list are leaves (one symbol) or packages of two items */
/* of the previous list; a symbol's length is the number of selected   */
/* items that contain it.                                              */
/* ------------------------------------------------------------------ */
typedef struct {
    uint64_t weight;
    int sym;  /* >= 0 for a leaf */
    int a, b; /* package: indices into the previous list */
} pmitem;

static void pm_count(pmitem **lists, int level, int idx, unsigned *len) {
    const pmitem *it = &lists[level][idx];
    if (it->sym >= 0) {
        len[it->sym] += 1;
        return;
    }
    pm_count(lists, level - 1, it->a, len);
    pm_count(lists, level - 1, it->b, len);
}

int dfo_package_merge(const uint64_t counts[256], unsigned max_len, unsigned lengths[256]) {
    int syms[256];
    int m = 0;
    for (int s = 0; s < 256; ++s) lengths[s] = 0;
    for (int s = 0; s < 256; ++s)
        if (counts[s]) syms[m++] = s;
    if (m == 0) return DFO_OK;
    if (m == 1) {
        lengths[syms[0]] = 1;
        return DFO_OK;
    }
    if (max_len < 1 || max_len > 63) return DFO_E_ARG;
    if (max_len < 63 && ((uint64_t)1 << max_len) < (uint64_t)m) return DFO_E_CAP;
    /* leaves sorted by (count, symbol): insertion sort */
    for (int i = 1; i < m; ++i) {
        int s = syms[i], j = i - 1;
        while (j >= 0 && (counts[syms[j]] > counts[s] ||
                          (counts[syms[j]] == counts[s] && syms[j] > s))) {
            syms[j + 1] = syms[j];
            --j;
        }
        syms[j + 1] = s;
    }
    pmitem **lists = (pmitem **)calloc(max_len, sizeof(pmitem *));
    int *sizes = (int *)calloc(max_len, sizeof(int));
    if (!lists || !sizes) return DFO_E_SPACE;
    for (unsigned lv = 0; lv < max_len; ++lv) {
        lists[lv] = (pmitem *)malloc(sizeof(pmitem) * (size_t)(2 * m));
        if (!lists[lv]) return DFO_E_SPACE;
    }
    /* level 0 = deepest level: the leaves alone */
    for (int i = 0; i < m; ++i) {
        lists[0][i].weight = counts[syms[i]];
        lists[0][i].sym = syms[i];
        lists[0][i].a = lists[0][i].b = -1;
    }
    sizes[0] = m;
    for (unsigned lv = 1; lv < max_len; ++lv) {
        /* packages of consecutive pairs of the previous list */
        int npk = sizes[lv - 1] / 2;
        int li = 0, pi = 0, out = 0;
        while (li < m || pi < npk) {
            int take_leaf;
            if (li >= m) take_leaf = 0;
            else if (pi >= npk) take_leaf = 1;
            else {
                uint64_t pw = lists[lv - 1][2 * pi].weight + lists[lv - 1][2 * pi + 1].weight;
                take_leaf = counts[syms[li]] <= pw; /* tie: leaf first */
            }
            pmitem *it = &lists[lv][out++];
            if (take_leaf) {
                it->weight = counts[syms[li]];
                it->sym = syms[li];
                it->a = it->b = -1;
                ++li;
            } else {
                it->weight = lists[lv - 1][2 * pi].weight + lists[lv - 1][2 * pi + 1].weight;
                it->sym = -1;
                it->a = 2 * pi;
                it->b = 2 * pi + 1;
                ++pi;
            }
        }
        sizes[lv] = out;
    }
    int take = 2 * m - 2;
    for (int i = 0; i < take; ++i) pm_count(lists, (int)max_len - 1, i, lengths);
    for (unsigned lv = 0; lv < max_len; ++lv) free(lists[lv]);
    free(lists);
    free(sizes);
    return DFO_OK;
}

/* Code lengths with the cap: plain Huffman when its depth fits, otherwise
 * package-merge.  Writes 0 for unused symbols. */
int dfo_code_lengths(const uint64_t counts[256], unsigned max_len, uint8_t lengths[256]) {
    unsigned l[256];
    if (!counts || !lengths || max_len < 1 || max_len > 32) return DFO_E_ARG;
    int depth = dfo_huffman_lengths(counts, l);
    if ((unsigned)depth > max_len) {
        int rc = dfo_package_merge(counts, max_len, l);
        if (rc) return rc;
    }
    for (int s = 0; s < 256; ++s) lengths[s] = (uint8_t)l[s];
    return DFO_OK;
}

/* ------------------------------------------------------------------ */
/* Canonical codes: order symbols by (length, symbol value); the first */
/* gets 0, the next (previous + 1) shifted left by the length step.    */
/* ------------------------------------------------------------------ */
int dfo_canonical_codes(const uint8_t lengths[256], uint32_t codes[256]) {
    if (!lengths || !codes) return DFO_E_ARG;
    for (int s = 0; s < 256; ++s) codes[s] = 0;
    uint64_t code = 0;
    unsigned prev_len = 0;
    int first = 1;
    for (unsigned len = 1; len <= 32; ++len) {
        for (int s = 0; s < 256; ++s) {
            if (lengths[s] != len) continue;
            if (first) {
                code = 0;
                first = 0;
            } else {
                code = (code + 1) << (len - prev_len);
            }
            prev_len = len;
            if (code >> len) return DFO_E_STREAM; /* over-full: not a prefix code */
            codes[s] = (uint32_t)code;
        }
    }
    return DFO_OK;
}

/* ------------------------------------------------------------------ */
/* Layout sizes (n = bytes per thread, T = threads per block)           */
/* ------------------------------------------------------------------ */
static uint64_t ceil_div(uint64_t a, uint64_t b) { return (a + b - 1) / b; }

int dfo_layout(uint64_t total_bits, unsigned n_bytes, unsigned threads, uint64_t *num_chunks,
               uint64_t *num_blocks, uint64_t *exp_bytes, uint64_t *gap_bytes) {
    if (n_bytes == 0 || threads == 0) return DFO_E_ARG;
    uint64_t C = ceil_div(total_bits, 8ull * n_bytes);
    uint64_t B = ceil_div(C, threads);
    if (num_chunks) *num_chunks = C;
    if (num_blocks) *num_blocks = B;
    /* every thread of every block reads its n bytes plus 16 bytes past them */
    if (exp_bytes) *exp_bytes = B * n_bytes * threads + 16;
    /* gap slots 0 .. B*T inclusive, 5 bits each, whole 32-bit words, two spare words */
    if (gap_bytes) *gap_bytes = 4 * (ceil_div(5 * (B * threads + 1), 32) + 2);
    return DFO_OK;
}

/* ------------------------------------------------------------------ */
/* Encoder                                                             */
/* ------------------------------------------------------------------ */
static void put_bit(uint8_t *buf, uint64_t k, unsigned bit) {
    if (bit) buf[k >> 3] |= (uint8_t)(0x80u >> (k & 7));
}

static unsigned get_bit(const uint8_t *buf, uint64_t k) {
    return (buf[k >> 3] >> (7 - (k & 7))) & 1u;
}

/* Writes EncodedExponent (exp_cap bytes, zero padded) and PackedSignMantissa
 * (n bytes).  *total_bits receives the number of code bits. */
int dfo_encode(const uint16_t *w, uint64_t n, const uint8_t lengths[256], const uint32_t codes[256],
               uint8_t *exp_out, uint64_t exp_cap, uint8_t *sm_out, uint64_t *total_bits) {
    if ((n && (!w || !sm_out)) || !lengths || !codes || (exp_cap && !exp_out) || !total_bits)
        return DFO_E_ARG;
    uint64_t bits = 0;
    for (uint64_t i = 0; i < n; ++i) {
        unsigned e = exponent_of(w[i]);
        if (lengths[e] == 0) return DFO_E_ARG; /* exponent missing from the codebook */
        bits += lengths[e];
    }
    if (ceil_div(bits, 8) > exp_cap) return DFO_E_SPACE;
    memset(exp_out, 0, exp_cap);
    uint64_t k = 0;
    for (uint64_t i = 0; i < n; ++i) {
        unsigned e = exponent_of(w[i]);
        unsigned len = lengths[e];
        for (unsigned j = 0; j < len; ++j) put_bit(exp_out, k++, (codes[e] >> (len - 1 - j)) & 1u);
        sm_out[i] = sign_mantissa_byte(w[i]);
    }
    *total_bits = bits;
    return DFO_OK;
}

/* ------------------------------------------------------------------ */
/* Metadata by brute force from the list of code start positions.      */
/* gaps: one byte per slot c = 0 .. B*T (B*T+1 slots)                  */
/* block_pos: B+1 entries                                              */
/* ------------------------------------------------------------------ */
int dfo_metadata(const uint16_t *w, uint64_t n, const uint8_t lengths[256], unsigned n_bytes,
                 unsigned threads, uint8_t *gaps, uint64_t gap_slots, uint32_t *block_pos,
                 uint64_t block_slots) {
    if ((n && !w) || !lengths || !gaps || !block_pos || n_bytes == 0 || threads == 0)
        return DFO_E_ARG;
    if (n > 0xFFFFFFFFull) return DFO_E_ARG;
    uint64_t *starts = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)(n + 1));
    if (!starts) return DFO_E_SPACE;
    uint64_t pos = 0;
    for (uint64_t i = 0; i < n; ++i) {
        starts[i] = pos;
        pos += lengths[exponent_of(w[i])];
    }
    uint64_t total_bits = pos;
    starts[n] = total_bits; /* the end of the stream counts as a start */
    uint64_t C, B;
    dfo_layout(total_bits, n_bytes, threads, &C, &B, NULL, NULL);
    if (gap_slots != B * threads + 1 || block_slots != B + 1) {
        free(starts);
        return DFO_E_SPACE;
    }
    const uint64_t chunk_bits = 8ull * n_bytes;
    uint64_t j = 0; /* first start >= current boundary */
    for (uint64_t c = 0; c < gap_slots; ++c) {
        uint64_t boundary = chunk_bits * c;
        if (boundary > total_bits) {
            gaps[c] = 0;
            continue;
        }
        while (starts[j] < boundary) ++j;
        uint64_t g = starts[j] - boundary;
        if (g > 31) {
            free(starts);
            return DFO_E_STREAM;
        }
        gaps[c] = (uint8_t)g;
    }
    /* starts are strictly increasing (every code has length >= 1), so the
     * number of codes starting before a boundary is the index of the first
     * start at or past it */
    const uint64_t block_bits = chunk_bits * threads;
    uint64_t i = 0;
    for (uint64_t b = 0; b <= B; ++b) {
        uint64_t boundary = block_bits * b;
        while (i < n && starts[i] < boundary) ++i;
        block_pos[b] = (uint32_t)i;
    }
    free(starts);
    return DFO_OK;
}

/* 5-bit fields, most significant bit first, slot c at packed bits [5c, 5c+5). */
int dfo_pack_gaps(const uint8_t *gaps, uint64_t slots, uint8_t *packed, uint64_t packed_bytes) {
    if ((slots && !gaps) || (packed_bytes && !packed)) return DFO_E_ARG;
    if (ceil_div(5 * slots, 8) > packed_bytes) return DFO_E_SPACE;
    memset(packed, 0, packed_bytes);
    for (uint64_t c = 0; c < slots; ++c) {
        if (gaps[c] > 31) return DFO_E_ARG;
        for (unsigned j = 0; j < 5; ++j) put_bit(packed, 5 * c + j, (gaps[c] >> (4 - j)) & 1u);
    }
    return DFO_OK;
}

/* ------------------------------------------------------------------ */
/* Explicit binary Huffman tree built from the canonical codes.        */
/* node 0 = root; child[x][bit] = node index, or -1 - symbol for leaf.  */
/* ------------------------------------------------------------------ */
typedef struct {
    int child[2];
} tnode;

static int build_tree(const uint8_t lengths[256], tnode **out_nodes) {
    uint32_t codes[256];
    int rc = dfo_canonical_codes(lengths, codes);
    if (rc) return rc;
    int cap = 1;
    for (int s = 0; s < 256; ++s) cap += lengths[s];
    tnode *nodes = (tnode *)malloc(sizeof(tnode) * (size_t)cap);
    if (!nodes) return DFO_E_SPACE;
    int nn = 1;
    nodes[0].child[0] = nodes[0].child[1] = 0; /* 0 = empty (root is never a child) */
    for (int s = 0; s < 256; ++s) {
        unsigned len = lengths[s];
        if (!len) continue;
        int cur = 0;
        for (unsigned j = 0; j < len; ++j) {
            unsigned bit = (codes[s] >> (len - 1 - j)) & 1u;
            if (j + 1 == len) {
                if (nodes[cur].child[bit] != 0) {
                    free(nodes);
                    return DFO_E_STREAM; /* not prefix free */
                }
                nodes[cur].child[bit] = -1 - s;
            } else {
                int nx = nodes[cur].child[bit];
                if (nx < 0) {
                    free(nodes);
                    return DFO_E_STREAM;
                }
                if (nx == 0) {
                    nx = nn++;
                    nodes[nx].child[0] = nodes[nx].child[1] = 0;
                    nodes[cur].child[bit] = nx;
                }
                cur = nx;
            }
        }
    }
    *out_nodes = nodes;
    return DFO_OK;
}

/* Walks the tree from bit position *k; returns the symbol or a negative error. */
static int walk(const tnode *nodes, const uint8_t *exp, uint64_t total_bits, uint64_t *k) {
    int cur = 0;
    for (;;) {
        if (*k >= total_bits) return DFO_E_STREAM;
        int nx = nodes[cur].child[get_bit(exp, *k)];
        *k += 1;
        if (nx < 0) return -1 - nx;
        if (nx == 0) return DFO_E_STREAM;
        cur = nx;
    }
}

/* Decode the first code of a bit pattern (first bit = bit nbits-1 of pattern).
 * Returns the symbol and its length, used to read tables off the tree. */
int dfo_decode_prefix(uint64_t pattern, unsigned nbits, const uint8_t lengths[256], int *symbol,
                      unsigned *length) {
    if (nbits == 0 || nbits > 64 || !symbol || !length) return DFO_E_ARG;
    tnode *nodes;
    int rc = build_tree(lengths, &nodes);
    if (rc) return rc;
    uint8_t buf[8];
    memset(buf, 0, sizeof buf);
    for (unsigned j = 0; j < nbits; ++j) put_bit(buf, j, (unsigned)(pattern >> (nbits - 1 - j)) & 1u);
    uint64_t k = 0;
    int s = walk(nodes, buf, nbits, &k);
    free(nodes);
    if (s < 0) return s;
    *symbol = s;
    *length = (unsigned)k;
    return DFO_OK;
}

/* Bit-serial decode of a whole stream: n symbols, one tree step per bit. */
int dfo_decode_serial(const uint8_t *exp, uint64_t total_bits, const uint8_t *sm, uint64_t n,
                      const uint8_t lengths[256], uint16_t *out) {
    if ((n && (!exp || !sm || !out)) || !lengths) return DFO_E_ARG;
    tnode *nodes;
    int rc = build_tree(lengths, &nodes);
    if (rc) return rc;
    uint64_t k = 0;
    for (uint64_t i = 0; i < n; ++i) {
        int e = walk(nodes, exp, total_bits, &k);
        if (e < 0) {
            free(nodes);
            return e;
        }
        out[i] = assemble(sm[i], (unsigned)e);
    }
    free(nodes);
    return k == total_bits ? DFO_OK : DFO_E_STREAM;
}

/* Metadata-driven decode of blocks [first_block, first_block + num_blocks):
 * for every chunk c of those blocks start at 8n*c + Gaps[c], decode while the
 * code start lies inside the chunk and before total_bits, and place the
 * symbols at BlockOutputPos[b] + (codes of earlier chunks of the same block).
 * gaps = one byte per slot (unpacked).  out has n entries (full output). */
int dfo_decode_blocks(const uint8_t *exp, uint64_t total_bits, const uint8_t *sm, uint64_t n,
                      const uint8_t lengths[256], unsigned n_bytes, unsigned threads,
                      const uint8_t *gaps, const uint32_t *block_pos, uint64_t first_block,
                      uint64_t num_blocks, uint16_t *out) {
    if (!lengths || !gaps || !block_pos || n_bytes == 0 || threads == 0) return DFO_E_ARG;
    uint64_t C, B;
    dfo_layout(total_bits, n_bytes, threads, &C, &B, NULL, NULL);
    if (first_block + num_blocks > B) return DFO_E_ARG;
    tnode *nodes;
    int rc = build_tree(lengths, &nodes);
    if (rc) return rc;
    const uint64_t chunk_bits = 8ull * n_bytes;
    for (uint64_t b = first_block; b < first_block + num_blocks; ++b) {
        uint64_t pos = block_pos[b];
        for (unsigned t = 0; t < threads; ++t) {
            uint64_t c = b * threads + t;
            if (c >= C) break;
            uint64_t k = chunk_bits * c + gaps[c];
            uint64_t chunk_end = chunk_bits * (c + 1);
            while (k < chunk_end && k < total_bits) {
                int e = walk(nodes, exp, total_bits, &k);
                if (e < 0 || pos >= n) {
                    free(nodes);
                    return DFO_E_STREAM;
                }
                out[pos] = assemble(sm[pos], (unsigned)e);
                ++pos;
            }
        }
        if (pos != block_pos[b + 1]) {
            free(nodes);
            return DFO_E_STREAM;
        }
    }
    free(nodes);
    return DFO_OK;
}
