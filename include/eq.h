/*
 * libeq -- EntQuant inference-time decoding on AMD Instinct MI355X (gfx950).
 *
 * Paper: "Float8@2bits: Entropy Coding Enables Data-Free Model Compression"
 * (EntQuant, arXiv 2601.22787).  The weights of a linear layer stay in VRAM
 * as an entropy-coded bitstream z with BF16 per-output-row scales S and ANS
 * metadata M (Sec. 2.2, "Weight encoding"); Alg. 2 decodes them on the fly:
 *   w   <- ANS^-1(z, M)            entropy decoding        (eq_decode_codes)
 *   W_q <- view(w)                 row-major [M rows, N cols]
 *   W_hat = s_i * W_q              dequantiser, Sec. 2.1   (eq_decode_bf16)
 *   y   <- QMatMul(W_q, S, x) + b  y = x W_hat^T + b       (eq_decode_gemv)
 * The decode+GEMV entry point fuses all three steps and never materialises
 * the weights.
 *
 * Container (".eqc", one compressed layer; little-endian; every section
 * 256-byte aligned).  Header, 256 bytes:
 *   0 "EQC1"  4 version=1  8 header_bytes=256  12 base_format (1 = E4M3FN,
 *   2 = Int8: the Float8 default and the Int8 alternative of Sec. 3.5)
 *   16 rows M  20 cols N  24 chunk_syms C  28 n_chunks = ceil(M*N/C)
 *   32 lanes W  36 prob_bits P  40 n_syms K  44 flags=0
 *   48 total_words (u64)  56 padded_words (u64)  64 seed (u64)
 *   72 alpha (f32)  76 target_bits (f32)  80 entropy_bits (f32)
 *   88.. u64 byte offsets of the sections scale, sym, freq, chunk_off,
 *   chunk_state, words; 136 file_bytes (u64).
 * Sections:
 *   scale       u16[M]       BF16 bit patterns, one scale per output row
 *   sym         u8[K]        codes present, strictly ascending: E4M3FN bytes
 *                            (never a NaN), or Int8 two's complement bytes in
 *                            [-127, 127] (never 0x80)
 *   freq        u16[K]       frequencies, >= 1, summing to 2^P
 *   chunk_off   u32[n+1]     first stream word of each chunk; [n] = total_words
 *   chunk_state u32[n*W]     initial decoder state of every lane of every chunk
 *   words       u16[padded_words]  all chunks' streams, then >= 1024 zero words
 * Coder (the paper's ANS library is closed; this is interleaved rANS after
 * Duda 2014 with Giesen's interleaving): symbol k of chunk c is element
 * c*C + k of the row-major code matrix and belongs to lane k mod W at step
 * k div W.  A step first decodes every active lane
 *   slot = x mod 2^P;  symbol s with cum_s <= slot < cum_s + f_s;
 *   x = f_s * (x >> P) + slot - cum_s
 * then, in ascending lane order, each active lane with x < 2^16 takes the
 * next word: x = (x << 16) | word.  After the last step every lane is at
 * 2^16 and the chunk's words are used up exactly.
 *
 * Version 2 (written by eqe_encode2, eq_encode.h; header field 4 = 2) keeps
 * the header and sections above with these differences:
 *   36 prob_bits = R, the frequency resolution (10..12); 40 n_syms = the
 *   size of the phrase alphabet; 84 tile_cols TC (a multiple of 4); 32 lanes
 *   = tile rows TR; 24 chunk_syms = TR * TC; 144 n_quads, 148 n_pairs,
 *   152 n_singles (their sum is n_syms); 156 the encoder's dictionary
 *   threshold (informative).
 *   Chunk c is the tile of rows [b TR, b TR + TR) and columns [t TC, t TC +
 *   TC) (cut at the matrix edge), b = c div NT, t = c mod NT, NT =
 *   ceil(N / TC); state s of the chunk codes row b TR + s of the tile.
 *   sym section: u8[n_syms][4], symbol k's codes in position order (quads
 *   first, then pairs, then single codes; unused bytes 0); freq: u16 f_k >= 1
 *   summing to 2^R.  A step decodes, for every state whose row segment is not
 *   yet complete, slot = x mod 2^16, the symbol k with 2^(16-R) cum_k <= slot
 *   < 2^(16-R) (cum_k + f_k), x = F_k (x >> 16) + slot - 2^(16-R) cum_k with
 *   F_k = 2^(16-R) f_k, and appends its 4, 2 or 1 codes to the segment; then
 *   those states in ascending order take the next word when x < 2^16.
 *   Row order (44 flags bit 0; other bits 0): the tiles are cut over the rows
 *   in a stored order, the section at byte offset 160 (u64; 0 without the
 *   flag), u32[M], giving the matrix row of stored row k (a permutation).
 *   Chunk c's rows are then stored rows [b TR, b TR + TR): state s codes a
 *   segment of matrix row order[b TR + s].  Scales stay in matrix order, and
 *   every output is in matrix order.  The encoder sorts rows by their phrase
 *   count, so that a tile's states finish at nearly the same step.
 *   Decoding a version-2 layer without a row order to codes or BF16 needs
 *   2 * TR * N < 2^31.
 *
 * Conventions for every entry point below:
 *  - Device pointers are allocated and owned by the caller; the library never
 *    allocates, frees or synchronises (except eq_get_status, which waits on
 *    the given stream).  The one piece of device memory it holds itself is
 *    eq_decode_gemv_noalloc's static scratch, part of its code object.
 *  - Calls are asynchronous on `stream` and reentrant; different layers or
 *    outputs may be processed on several streams at once.
 *  - Return codes: EQ_OK, EQ_EINVAL (null pointer, size or range),
 *    EQ_EFORMAT (container header or sections inconsistent), EQ_EHIP (a HIP
 *    launch or runtime call failed), EQ_ESCRATCH (eq_decode_gemv_noalloc
 *    only: the call needs more than the library's static scratch).  Stream
 *    corruption found while decoding on the device is recorded in the
 *    layer's status word (EQ_ECORRUPT via eq_get_status); outputs of a
 *    corrupted chunk are then unspecified, but no access ever leaves the
 *    container or the output buffers.
 */
#ifndef EQ_H
#define EQ_H
#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define EQ_OK 0
#define EQ_EINVAL (-1)
#define EQ_EFORMAT (-2)
#define EQ_EHIP (-3)
#define EQ_ECORRUPT (-4)
#define EQ_ESCRATCH (-5)

/* A validated view of one container in device memory (filled by eq_layer_init). */
typedef struct eq_layer {
  uint32_t rows, cols;       /* M output rows, N input columns                    */
  uint32_t chunk_syms;       /* C                                                  */
  uint32_t n_chunks;
  uint32_t lanes;            /* W: 64, 128 or 256                                  */
  uint32_t prob_bits;        /* P: 8..12                                           */
  uint32_t n_syms;           /* K: 1..256                                          */
  uint32_t base_format;      /* 1 = E4M3FN, 2 = Int8 (value v(q) of a code q)      */
  uint64_t total_words, padded_words;
  const uint16_t *scale;     /* device: the container's sections                   */
  const uint8_t *sym;
  const uint16_t *freq;
  const uint32_t *chunk_off;
  const uint32_t *chunk_state;
  const uint16_t *words;
  uint32_t *lut;             /* device scratch, eq_lut_bytes() bytes, caller-owned */
  int32_t *status;           /* device int32, caller-owned                         */
  uint32_t version;          /* container version, 1 or 2                          */
  uint32_t tile_cols;        /* version 2: tile columns TC (tile rows = lanes)     */
  uint32_t n_quads, n_pairs, n_singles; /* version 2: alphabet parts (sum n_syms) */
  const uint32_t *row_order; /* version 2, device: the order section, or null      */
} eq_layer;

/* Bytes of device scratch the decode tables of a layer need (either
 * container version). */
size_t eq_lut_bytes(void);

/* Validate the container `host_blob` (blob_bytes long, host memory) and fill
 * *L with pointers into `dev_blob`, a device copy of the same bytes.  The
 * host copy is read only during the call.  `dev_blob` and `dev_lut`
 * (eq_lut_bytes() bytes) must be 256-byte aligned (EQ_EINVAL otherwise);
 * `dev_lut` and `dev_status` (one int32) are device scratch owned by the
 * caller and tied to this layer.  Checks: magic/version/base format, sizes
 * and section bounds, 8 <= P <= 12 (the kernels multiply f by x >> P with
 * 24-bit operands), ascending symbols valid in the base format, frequencies
 * >= 1 summing to 2^P, monotone chunk offsets ending at total_words,
 * padding >= 1024 words, initial states in [2^16, 2^32), a version-2 row
 * order that is a permutation of the rows, scales finite with
 * magnitude in [2^-117, 2^120) (so every dequantised product s * v(q), an
 * 8-bit by at most 7-bit significand product, is exact in fp32).
 * Returns EQ_OK, EQ_EINVAL or EQ_EFORMAT. */
int eq_layer_init(eq_layer *L, const void *host_blob, uint64_t blob_bytes, const void *dev_blob,
                  void *dev_lut, int32_t *dev_status);

/* Build the layer's decode tables on the device (slot -> symbol/frequency/
 * offset, code -> value in the base format; Sec. 2.2 metadata M) and clear its status
 * word.  Must run (on the same stream, or be complete) before any decode. */
int eq_layer_prepare(const eq_layer *L, hipStream_t stream);

/* Alg. 2, entropy decoding and view: decode every chunk; codes[k] is the
 * code (E4M3FN or Int8 byte) of element k of the row-major M x N matrix
 * (M*N bytes, device). */
int eq_decode_codes(const eq_layer *L, uint8_t *codes, hipStream_t stream);

/* Alg. 2's entropy decoding and view plus the dequantiser of Sec. 2.1:
 * w[i*N + j] = bf16(s_i * v(q_ij)), the exact product rounded once to
 * nearest-even (M*N BF16 bit patterns, device). */
int eq_decode_bf16(const eq_layer *L, uint16_t *w, hipStream_t stream);

/* Workspace bytes eq_decode_gemv needs for batch B (1..8). */
size_t eq_gemv_workspace_bytes(const eq_layer *L, uint32_t B);

/* Alg. 2 fused: y[b][i] = s_i * sum_j v(q_ij) x[b][j] + bias[i] for
 * b < B <= 8, without materialising the weights.  x is [B][N] BF16 (device),
 * bias is [M] BF16 or NULL (2-byte alignment suffices), y is [B][M] fp32
 * (device).  Results are reproducible run to run: partial sums are always
 * added in a fixed order.  The row sum is
 * accumulated in fp32 and scaled by s_i once, as QMatMul(W_q, S, x) does.
 * ws/ws_bytes: device workspace of at least eq_gemv_workspace_bytes(L, B). */
int eq_decode_gemv(const eq_layer *L, const uint16_t *x, uint32_t B, const uint16_t *bias,
                   float *y, void *ws, size_t ws_bytes, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * eq_decode_gemv with the workspace taken from a static array of
 * EQ_NOALLOC_SCRATCH_BYTES in the library's code object instead of `ws`.
 * The call allocates nothing.  Each device holds one such array from the
 * first call on it until the process ends, and every call on that device
 * uses it: calls that overlap on one device (several streams or threads)
 * race and must be serialised by the caller.  Returns EQ_ESCRATCH when
 * eq_gemv_workspace_bytes(L, B) exceeds EQ_NOALLOC_SCRATCH_BYTES (checked on
 * the host before any device work), otherwise what eq_decode_gemv returns;
 * results are identical to eq_decode_gemv's. */
#define EQ_NOALLOC_SCRATCH_BYTES (32u << 20)
int eq_decode_gemv_noalloc(const eq_layer *L, const uint16_t *x, uint32_t B,
                           const uint16_t *bias, float *y, hipStream_t stream);

/* Block-wise decompression (Sec. 2.2, paragraph "Block-Wise Decompression
 * Pipeline": all compressed matrices of a transformer block are decoded
 * together, ahead of the block's forward pass).  Decodes layers L[0..n-1]
 * (host array of n views, 1 <= n <= 8) to BF16: layer i to w[i] (device, its
 * M*N BF16 values), as eq_decode_bf16 does, with identical results.  One
 * launch decodes all layers when all are version 2 (any tile heights), or
 * all version 1 with one lane count and rows that are whole steps (N a
 * multiple of W), which keeps more chunks in flight per compute unit;
 * otherwise each layer gets its own launch, in order. */
int eq_decode_bf16_multi(const eq_layer *const *L, uint16_t *const *w, uint32_t n,
                         hipStream_t stream);

/* Block-wise decompression to the base format (Sec. 2.2, "Block-Wise
 * Decompression Pipeline": the paper decodes a block's weights into one
 * Float8 buffer per device, which its W8A16 GEMM reads).  Decodes layers
 * L[0..n-1] (host array of n views, 1 <= n <= 8) to one-byte codes: layer i
 * to codes[i] (device, its M*N codes, as eq_decode_codes writes them), with
 * identical results.  One launch decodes all layers when all are version 2
 * (any tile heights), or all version 1 with one lane count, one base format
 * and rows that are whole steps; otherwise each layer gets its own launch,
 * in order.  The codes feed eq_gemm_codes. */
int eq_decode_codes_multi(const eq_layer *const *L, uint8_t *const *codes, uint32_t n,
                          hipStream_t stream);

/* Workspace bytes eq_decode_gemv_multi needs: the sum of the layers'
 * eq_gemv_workspace_bytes(L[i], B); 0 if an argument is invalid. */
size_t eq_gemv_multi_workspace_bytes(const eq_layer *const *L, uint32_t n, uint32_t B);

/* Fused decode-GEMV of n layers (1 <= n <= 8) that read the same input, such
 * as the query/key/value or gate/up projections of a block (Alg. 2 for each
 * layer, decoded block-wise as in Sec. 2.2): y[i][b][r] = s_r * sum_j
 * v(q_rj) x[b][j] + bias[i][r] for layer i.  All layers must have the same
 * N; x is [B][N] BF16 (device, B <= 8); bias is NULL or a host array of n
 * device pointers (each [M_i] BF16 or NULL); y is a host array of n device
 * pointers ([B][M_i] fp32).  ws/ws_bytes: device workspace of at least
 * eq_gemv_multi_workspace_bytes(L, n, B); layer i uses the slice after those
 * of layers 0..i-1.  Results equal eq_decode_gemv's for each layer.  One
 * launch serves all layers when they share a container version and lane
 * count (version 1: rows that are whole steps and activations that fit LDS;
 * version 2: the tile height); otherwise each layer is run by a launch of
 * its own. */
int eq_decode_gemv_multi(const eq_layer *const *L, uint32_t n, const uint16_t *x, uint32_t B,
                         const uint16_t *const *bias, float *const *y, void *ws,
                         size_t ws_bytes, hipStream_t stream);

/* Prefill (B > 8 tokens): the linear layer y = x W_hat^T + b on the matrix
 * cores (Sec. 2.1), from the decoded codes.  The paper decompresses a
 * block's weights to a Float8 buffer and runs an FP8-weight / 16-bit
 * activation GEMM (Sec. 2.2 block-wise pipeline, App. A.1); these entry
 * points do the same with one byte per weight: eq_decode_codes writes the
 * codes, eq_gemm_codes converts them to BF16 in registers, multiplies with
 * MFMA (fp32 accumulation) and applies s_i and the bias once per output.
 * Requirements: N (cols) a multiple of 16; codes and x 16-byte aligned. */

/* Workspace bytes of eq_gemm_codes for B tokens: room for the partial sums
 * when the input columns are cut into slices (split-K, chosen when the
 * output tiles alone would leave compute units idle); 0 when no slicing is
 * needed (or on bad arguments). */
size_t eq_gemm_codes_workspace_bytes(const eq_layer *L, uint32_t B);

/* Workspace bytes of eq_decode_gemm for B tokens: the M*N codes, rounded up
 * to 256, then eq_gemm_codes_workspace_bytes(L, B); for B <= 8 at least
 * eq_gemv_workspace_bytes(L, B) too. */
size_t eq_gemm_workspace_bytes(const eq_layer *L, uint32_t B);

/* y[t][i] = s_i * sum_j v(codes[i][j]) x[t][j] + bias[i] for t < B, any
 * B >= 1.  codes is [M][N] (the output of eq_decode_codes for this layer,
 * device), x is [B][N] BF16 (device), bias is [M] BF16 or NULL, y is
 * [B][M] fp32 (device), ws/ws_bytes a device workspace of at least
 * eq_gemm_codes_workspace_bytes(L, B) bytes (4-byte aligned; may be NULL
 * when that is 0).  Sliced sums are added in slice order, so results do
 * not depend on timing.  Returns EQ_OK, EQ_EINVAL or EQ_EHIP. */
int eq_gemm_codes(const eq_layer *L, const uint8_t *codes, const uint16_t *x, uint32_t B,
                  const uint16_t *bias, float *y, void *ws, size_t ws_bytes,
                  hipStream_t stream);

/* Alg. 2 for a batch of B tokens: eq_decode_codes into the start of ws (at
 * least eq_gemm_workspace_bytes(L, B) bytes, device, 16-byte aligned), then
 * eq_gemm_codes with the rest of ws.  For B <= 8 it runs eq_decode_gemv
 * instead (with ws as its workspace), which is faster at such batches and
 * gives that call's results. */
int eq_decode_gemm(const eq_layer *L, const uint16_t *x, uint32_t B, const uint16_t *bias,
                   float *y, void *ws, size_t ws_bytes, hipStream_t stream);

/* Wait for `stream`, then report EQ_ECORRUPT if any decode since the last
 * eq_layer_prepare found a chunk whose stream or terminal states did not
 * check out, else EQ_OK (or EQ_EHIP). */
int eq_get_status(const eq_layer *L, hipStream_t stream);

/* Static description of a return code. */
const char *eq_strerror(int code);

#ifdef __cplusplus
}
#endif
#endif
