/*
 * df11.h -- C ABI of the DFloat11 codec for MI355X (gfx950).
 *
 * DFloat11 (arXiv 2504.11651) stores a BF16 tensor losslessly as
 *   - EncodedExponent:    the 8-bit exponents, Huffman coded and tightly
 *                         bit-packed (Sec. 2.3);
 *   - PackedSignMantissa: one raw byte per weight, sign in bit 7 and the 7
 *                         mantissa bits in bits 6..0 (Sec. 2.3, Algorithm 1);
 *   - Gaps:               per n-byte chunk of EncodedExponent, the bit offset
 *                         of the first code that starts in it, 5 bits each
 *                         (Sec. 2.3.2);
 *   - BlockOutputPos:     per block of T chunks, the index of its first output
 *                         element (Sec. 2.3.2, Algorithm 1);
 *   - decode tables:      the code book in table form (Sec. 2.3.1).
 * Decompression (Algorithm 1) turns these back into bit-identical BF16.
 *
 * Byte-level format (every reading of the paper is listed here):
 *   - stream bit k is bit 7-(k%8) of byte k/8 (first code bit = most
 *     significant); codes are canonical, ordered by (length, exponent value);
 *     total_bits = sum of the code lengths; the stream is zero padded to
 *     exp_bytes = B*n*T + 16 bytes;
 *   - chunk c covers stream bits [8n*c, 8n*(c+1)); C = ceil(total_bits/8n)
 *     chunks; B = ceil(C/T) blocks;
 *   - Gaps[c] = (first code start >= 8n*c, the end of the stream counting as
 *     a start) - 8n*c, for c = 0 .. B*T (B*T+1 slots); 0 for a chunk past the
 *     end; slot c occupies packed bits [5c, 5c+5), most significant first, in
 *     gap_bytes = 4*(ceil(5*(B*T+1)/32)+2) bytes;
 *   - BlockOutputPos[b] = number of codes starting before bit 8n*T*b, for
 *     b = 0 .. B (B+1 entries; the last is n_elems);
 *   - PackedSignMantissa holds n_elems bytes followed by zero padding up to
 *     sm_bytes = (n_elems rounded up to 16) + 16, so whole 8-byte groups can
 *     always be read;
 *   - all 256 exponent values are codable (the paper's format reserves
 *     240..255 as table pointers; this one does not need to);
 *   - code lengths are capped at max_code_len <= 32 (gaps fit 5 bits); when
 *     plain Huffman is deeper, optimal capped lengths come from package-merge.
 *   - the decode-table blob (table_bytes) is this library's own layout,
 *     built from the code book by df11_build_tables; it is opaque to callers.
 *
 * Memory ownership: the caller allocates and frees every buffer.  Host
 * functions take host pointers; df11_decode_block, df11_block_gemm and
 * df11_block_forward take device pointers (inside df11_stream, and for the
 * weights, activations, outputs and workspace).  The library keeps no
 * per-call state and allocates no device memory; its one device-side array,
 * the partial sums of df11_block_forward_noalloc, is a fixed-size static
 * array of DF11_STATIC_SCRATCH_BYTES per GPU.
 *
 * Errors: every function returns DF11_OK (0) or a negative DF11_E_* code;
 * nothing is thrown across the ABI.  df11_strerror names a code.
 */
#ifndef DF11_H
#define DF11_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DF11_OK 0
#define DF11_E_INVALID_ARG (-1)       /* null pointer, bad size, bad layout */
#define DF11_E_CAP_INFEASIBLE (-2)    /* 2^max_code_len < number of symbols */
#define DF11_E_BUFFER_TOO_SMALL (-3)  /* an output capacity is too small */
#define DF11_E_CORRUPT (-4)           /* df11_validate found an inconsistency */
#define DF11_E_HIP (-5)               /* HIP runtime or launch failure */
#define DF11_E_UNSUPPORTED (-6)       /* layout the decoder was not built for */

/* Code book: histogram of the exponents, canonical code per exponent. */
typedef struct {
    uint32_t max_code_len; /* longest code in use (0 when no symbol is used) */
    uint32_t num_symbols;  /* exponent values with a non-zero count */
    uint64_t count[256];   /* histogram of exponent values */
    uint8_t len[256];      /* code length in bits, 0 = value not used */
    uint32_t code[256];    /* canonical code, right aligned in len bits */
} df11_codebook;

/* Work partition of the stream (Sec. 2.3.2). */
typedef struct {
    uint32_t bytes_per_thread;  /* n: bytes of EncodedExponent per thread (decoder: 8) */
    uint32_t threads_per_block; /* T: threads per block, a multiple of 64, <= 1024 */
    uint32_t lut_bits;          /* width of the first-level decode table index, 8..12 */
} df11_layout;

/* Sizes of one encoded stream. */
typedef struct {
    uint64_t n_elems;             /* BF16 weights */
    uint64_t total_bits;          /* sum of code lengths */
    uint64_t num_chunks;          /* C */
    uint64_t num_blocks;          /* B */
    uint64_t exp_bytes;           /* EncodedExponent bytes incl. padding */
    uint64_t sm_bytes;            /* PackedSignMantissa buffer: n_elems bytes, zero padded to
                                     a multiple of 16, plus 16 */
    uint64_t gap_bytes;           /* packed Gaps bytes */
    uint64_t block_pos_bytes;     /* 4 * (B + 1) */
    uint64_t table_bytes;         /* decode-table blob bytes */
    uint32_t max_elems_per_block; /* max of BlockOutputPos[b+1]-BlockOutputPos[b]; set by df11_encode */
    uint32_t max_code_len;        /* longest code in the book */
} df11_sizes;

/* One encoded stream.  For df11_decode_block the pointers are device
 * pointers; for df11_validate they are host pointers. */
typedef struct {
    const uint8_t *exp;        /* EncodedExponent, sizes.exp_bytes */
    const uint8_t *sm;         /* PackedSignMantissa, sizes.sm_bytes */
    const uint8_t *gaps;       /* packed Gaps, sizes.gap_bytes */
    const uint32_t *block_pos; /* BlockOutputPos, B + 1 entries */
    const uint8_t *tables;     /* decode-table blob, sizes.table_bytes */
    df11_sizes sizes;
    df11_layout layout;
} df11_stream;

/* Histogram of the exponents of n BF16 weights (bit patterns), optimal code
 * lengths capped at max_code_len (1..32), canonical codes (Sec. 2.3; the
 * Huffman tree of Sec. 2.1; cap: Sec. 2.3.2).  Host.  Ties between equal
 * weights are broken leaf first, then by exponent value, then by creation
 * order, so the result is deterministic. */
int df11_build_codebook(const uint16_t *bf16, uint64_t n, uint32_t max_code_len,
                        df11_codebook *out);

/* Same, from a given histogram (no weights needed).  Host. */
int df11_codebook_from_counts(const uint64_t counts[256], uint32_t max_code_len,
                              df11_codebook *out);

/* The layout df11_decode_block decodes fastest for a stream of n weights:
 * n = 8 bytes per thread and an 11-bit table index, with T = 128 threads per
 * block from DF11_LARGE_STREAM_ELEMS weights up (one wavefront decodes a
 * block, two chunks per lane) and T = 64 below (a shorter stream then
 * finishes in fewer rounds of blocks).  T is a format parameter the paper
 * leaves open (Sec. 2.3.2); it is recorded in the stream.  Host.  Returns
 * DF11_E_INVALID_ARG for a null out. */
#define DF11_LARGE_STREAM_ELEMS (192ull << 20)
int df11_default_layout(uint64_t n, df11_layout *out);

/* Buffer sizes for encoding the weights counted in cb with layout lay.
 * max_elems_per_block is left 0 (it depends on the data).  Host. */
int df11_encoded_sizes(const df11_codebook *cb, const df11_layout *lay, df11_sizes *out);

/* Encode n weights (Sec. 2.3): writes EncodedExponent (exp, zero padded),
 * PackedSignMantissa (sm), packed Gaps and BlockOutputPos (Sec. 2.3.2).
 * Each *_cap is the capacity of the buffer in bytes.  The weights must match
 * the histogram in cb.  Fills *out (including max_elems_per_block).  Host,
 * multi-threaded. */
int df11_encode(const uint16_t *bf16, uint64_t n, const df11_codebook *cb, const df11_layout *lay,
                uint8_t *exp, uint64_t exp_cap, uint8_t *sm, uint64_t sm_cap, uint8_t *gaps,
                uint64_t gap_cap, uint32_t *block_pos, uint64_t block_pos_cap, df11_sizes *out);

/* Decode-table blob for cb with a lut_bits-wide first-level table
 * (Sec. 2.3.1 and the appendix on lookup-table decoding).  Host. */
int df11_build_tables(const df11_codebook *cb, uint32_t lut_bits, uint8_t *tables,
                      uint64_t table_cap);

/* Consistency check of a stream held in HOST memory: sizes agree with the
 * layout, Gaps < max_code_len, BlockOutputPos starts at 0, never decreases,
 * ends at n_elems, and agrees with max_elems_per_block, the table blob is
 * well formed.  Returns DF11_E_CORRUPT on the first violation.  Host. */
int df11_validate(const df11_stream *host_view);

/* Decompress one stream into n_elems BF16 values at out (device memory,
 * 2*n_elems bytes, 16-byte aligned) -- the whole of Algorithm 1 on the GPU.
 * All stream pointers are device pointers.  One transformer block encoded
 * as one stream decodes in one launch (Sec. 2.3.3).  The work is enqueued
 * on `stream` and the call returns without waiting; buffers must stay alive
 * until the stream has executed it.  n_elems == 0 launches nothing.
 * T = 64 and 128 decode one block per wavefront (T = 128 with two chunks
 * per lane), T = 256, 512 and 1024 one block per workgroup.
 * Returns DF11_E_UNSUPPORTED for bytes_per_thread != 8, for threads_per_block
 * outside {64, 128, 256, 512, 1024}, or when no workgroup of the launch fits
 * the device's LDS; DF11_E_INVALID_ARG for a null or misaligned pointer (exp
 * 8-byte, sm and tables 16-byte, gaps and block_pos 4-byte aligned) or
 * inconsistent sizes; DF11_E_HIP when the launch fails. */
int df11_decode_block(const df11_stream *dev, uint16_t *out, hipStream_t stream);

/* Launch shape df11_decode_block would use on the current device for this
 * stream: workgroups, threads per workgroup and LDS bytes per workgroup. */
int df11_decode_launch_shape(const df11_stream *dev, uint32_t *grid, uint32_t *block,
                             uint32_t *lds_bytes);

/* ---- Decode-then-GEMM block driver (Sec. 2.3.3 and the batch-size
 * experiments of Sec. 3: a transformer block is decompressed into a BF16
 * workspace right before its matrix multiplications, and the decoded
 * weights are discarded afterwards). */

#define DF11_MAX_MATRICES 8 /* matrices per block call */
#define DF11_MAX_TOKENS 64  /* activation rows per call */

/* One weight matrix inside a block of BF16 weights: rows x cols, row-major
 * ([out features, in features]), starting `offset` weights into the block.
 * Requirements: rows a multiple of 16, cols a multiple of 64, offset a
 * multiple of 8 (16-byte aligned rows). */
typedef struct {
    uint64_t offset;
    uint32_t rows;
    uint32_t cols;
} df11_matrix;

/* Device workspace bytes df11_block_gemm / df11_block_forward need for these
 * matrices at this many tokens: room for the fp32 partial sums of the
 * matrices whose cols are split into k ranges (0 when none is).  Above 8
 * tokens the split is chosen per device to balance its compute units; the
 * value covers every choice, so it depends only on the shapes.  Host, no
 * device access. */
int df11_gemm_workspace_bytes(const df11_matrix *mats, uint32_t n_mats, uint32_t tokens,
                              uint64_t *bytes);

/* For every matrix m: y[m] = x[m] * W_m^T, i.e.
 *   y[m][t][r] = sum_k x[m][t][k] * W_m[r][k],
 * BF16 products accumulated in fp32 on the matrix cores, fp32 output.
 *   weights:   device, n_weights BF16 values (the block);
 *   mats:      host array of n_mats (1..DF11_MAX_MATRICES) descriptors, each
 *              inside [0, n_weights);
 *   x:         host array of n_mats device pointers, x[m] is tokens x cols_m
 *              BF16 row-major, 16-byte aligned;
 *   y:         host array of n_mats device pointers, y[m] is tokens x rows_m
 *              fp32 row-major, 4-byte aligned;
 *   tokens:    1..DF11_MAX_TOKENS;
 *   workspace: device, at least df11_gemm_workspace_bytes (may be null when
 *              that is 0), 16-byte aligned.
 * The result depends only on the inputs and shapes (fixed summation order, no
 * atomics), so equal weights give bit-identical y.  Enqueued on `stream`;
 * returns without waiting.  DF11_E_UNSUPPORTED for shapes outside the
 * requirements above, DF11_E_BUFFER_TOO_SMALL for a short workspace. */
int df11_block_gemm(const uint16_t *weights, uint64_t n_weights, const df11_matrix *mats,
                    uint32_t n_mats, const uint16_t *const *x, uint32_t tokens, float *const *y,
                    void *workspace, uint64_t workspace_bytes, hipStream_t stream);

/* df11_decode_block(dev, weights_out, stream) followed by
 * df11_block_gemm(weights_out, dev->sizes.n_elems, ...) on the same stream:
 * one transformer block decompressed into the caller's BF16 workspace
 * (weights_out, 2*n_elems bytes) and consumed by its matrix products. */
int df11_block_forward(const df11_stream *dev, uint16_t *weights_out, const df11_matrix *mats,
                       uint32_t n_mats, const uint16_t *const *x, uint32_t tokens,
                       float *const *y, void *workspace, uint64_t workspace_bytes,
                       hipStream_t stream);

/* ---- The same, allocating nothing: for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).
 *
 * df11_block_forward with the fp32 partial sums held in a fixed array of
 * DF11_STATIC_SCRATCH_BYTES that the library keeps on each GPU it runs on
 * until the process ends, instead of a caller workspace.  The caller still
 * passes the stream, the decoded-weight buffer, activations and outputs.
 * The array's device address is looked up once per device, on the first
 * call with that device current; no call allocates device memory.
 *   returns DF11_E_BUFFER_TOO_SMALL when these matrices at this many tokens
 *   need more partial sums than the array holds (df11_gemm_workspace_bytes
 *   > DF11_STATIC_SCRATCH_BYTES): the Llama-3-8B block shapes fit at every
 *   token count up to DF11_MAX_TOKENS, the Llama-3.1-70B block up to 20;
 *   otherwise the same arguments, checks and results as df11_block_forward
 *   (bit-identical outputs).
 * All calls on one GPU share its array: calls that overlap in time on one
 * GPU (two streams, two host threads) race on it and must be serialised by
 * the caller. */
#define DF11_STATIC_SCRATCH_BYTES (32u << 20)

int df11_block_forward_noalloc(const df11_stream *dev, uint16_t *weights_out,
                               const df11_matrix *mats, uint32_t n_mats,
                               const uint16_t *const *x, uint32_t tokens, float *const *y,
                               hipStream_t stream);

/* ---- Fused decode-and-multiply for one token (decode-time products without
 * a decoded copy of the block: the decompression of Algorithm 1 feeds the
 * products of Sec. 2.3.3 directly, so the BF16 weights never reach memory).
 *
 * For every matrix m: y[m][r] = sum_k x[m][k] * W_m[r][k] with one
 * activation row, BF16 products accumulated in fp32 (bf16 dot-product
 * instructions), W_m decoded from the stream on chip.
 *   dev:       device stream, layout with threads_per_block = 64;
 *   mats:      host array of n_mats (1..DF11_MAX_MATRICES) descriptors, sorted
 *              by offset and disjoint, inside [0, n_elems); each with cols a
 *              multiple of 64 and >= 2048, offset a multiple of 8, and at
 *              least 4096 weights;
 *   x:         host array of device pointers, x[m] = cols_m BF16, 16-byte aligned;
 *   y:         host array of device pointers, y[m] = rows_m fp32, 4-byte aligned;
 *   workspace: device, >= df11_gemv_workspace_bytes (8 floats per stream
 *              block plus 8 bytes per output row), 16-byte aligned.
 * The summation order is fixed by the stream's blocks (deterministic; it is
 * not the order df11_block_gemm uses, so results agree with it to rounding,
 * not bit for bit).  Enqueued on `stream`.  DF11_E_UNSUPPORTED for shapes or
 * layouts outside the requirements above. */
int df11_gemv_workspace_bytes(const df11_stream *dev, const df11_matrix *mats, uint32_t n_mats,
                              uint64_t *bytes);
int df11_block_gemv(const df11_stream *dev, const df11_matrix *mats, uint32_t n_mats,
                    const uint16_t *const *x, float *const *y, void *workspace,
                    uint64_t workspace_bytes, hipStream_t stream);

/* ---- The paper's own decoder, as an ablation (Sec. 2.3.1 hierarchical
 * lookup tables; Sec. 2.3.2 and Algorithm 1 two-phase kernel; appendix on
 * compact lookup tables).  It decodes the same streams as df11_decode_block
 * with the paper's tables and kernel design, so the two designs can be
 * compared on the same hardware and data.
 *
 * df11_build_hlut_tables: the Huffman tree of cb cut into subtrees of height
 * level_bits (8 for the decoder; 1..8 accepted), one table of 2^level_bits
 * exponent bytes per subtree, LUT_1 for the root; an entry is the exponent
 * whose code is a prefix of the bits read so far, or a pointer v in 240..255
 * to LUT_(257-v) which decodes the next level_bits bits.  Writes LUT_1 ..
 * LUT_k in creation order (breadth first), then CodeLengths[256] (the code
 * length of every exponent), (k << level_bits) + 256 bytes in all; *num_luts
 * = k.  Host.  DF11_E_UNSUPPORTED when cb uses an exponent of 240 or more
 * (the paper's format reserves them as pointers) or needs more than
 * DF11_HLUT_MAX_LUTS tables; DF11_E_BUFFER_TOO_SMALL (with *num_luts set)
 * when table_cap is short. */
#define DF11_HLUT_MAX_LUTS 17
#define DF11_HLUT_MAX_BYTES ((DF11_HLUT_MAX_LUTS + 1) * 256)
int df11_build_hlut_tables(const df11_codebook *cb, uint32_t level_bits, uint8_t *tables,
                           uint64_t table_cap, uint32_t *num_luts);

/* df11_decode_block_hlut: decompress stream dev into out (device, 2*n_elems
 * bytes, 16-byte aligned) with the paper's kernel: one workgroup of T =
 * dev->layout.threads_per_block threads per block, tables and the block's
 * EncodedExponent bytes staged in LDS, phase 1 decodes one code per step
 * through the table hierarchy and counts, a Blelloch scan gives each thread
 * its output position, phase 2 decodes again and gathers each element's
 * sign/mantissa byte into an LDS write buffer, then coalesced stores.  luts:
 * device copy of df11_build_hlut_tables's output at level_bits 8 (16-byte
 * aligned, (num_luts + 1) * 256 bytes), num_luts its k (1..17).  dev->tables
 * is not used.  Enqueued on `stream`; DF11_E_INVALID_ARG / DF11_E_UNSUPPORTED
 * as df11_decode_block. */
int df11_decode_block_hlut(const df11_stream *dev, const uint8_t *luts, uint32_t num_luts,
                           uint16_t *out, hipStream_t stream);

/* Static description of a status code. */
const char *df11_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* DF11_H */
