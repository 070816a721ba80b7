/*
 * hufflm.h - C ABI of the Huff-LLM bf16 weight codec and its fused
 * decode-GEMV for AMD gfx950 (MI355X).
 *
 * Method: Huff-LLM (arXiv 2502.00922). A bf16 weight is split 1-4-4-7
 * (Sec. 5.1): sign and 7 mantissa bits are kept raw; the 8 exponent bits are
 * two 4-bit symbols, each coded with a per-matrix Huffman code (Sec. 3.1,
 * Sec. 5.1). Compression runs once, offline, on the CPU (Sec. 3.1). Weights
 * stay compressed in memory and are decoded only where they are multiplied
 * (Sec. 1 contributions, Sec. 3.2): here inside y = W x, so that HBM carries
 * only compressed bytes.
 *
 * ---------------------------------------------------------------------------
 * HLF1 container (all integers little-endian)
 * ---------------------------------------------------------------------------
 * W is row-major [rows][cols]; weight i = r*cols + c.
 * Fields of a weight w: s = w>>15, eh = (w>>11)&15, el = (w>>7)&15, m = w&127.
 *
 * Codebooks, one per field per matrix: histogram of the field over the whole
 * matrix; Huffman code lengths from a binary heap keyed (weight, kind, id),
 * kind 0 = leaf with id = symbol, kind 1 = internal node with id = creation
 * order, the two smallest keys merged first; if the longest code exceeds lmax
 * the lengths are replaced by package-merge lengths (items sorted by
 * (weight, symbol); lmax-1 rounds of pairing consecutive items and stable
 * merging with the leaves by (weight, kind); the first 2(n-1) items of the
 * last list are taken; length = occurrences). A field with one present
 * symbol has length 0 and emits no bits. With a joint limit pair_max (see
 * hl_build_codebook) the two fields' limits are a and min(lmax, pair_max - a)
 * for the a of least total code length. Code values are canonical (RFC 1951
 * Sec. 3.2.2 assignment).
 *
 * Tiling: segment (r, cs) is W[r][cs*S .. cs*S+S) (S divides cols, S % 8 == 0,
 * 8 <= S <= 512, L = cols/S segments per row). A group is GR rows x GC
 * consecutive column segments, GR*GC = 64 (GR = group_rows, a power of two,
 * with GC dividing L): row block rb is rows GR*rb .. GR*rb+G-1 (G = GR, or
 * fewer in the last block), column block cb is segments cb*GC .. cb*GC+GC-1,
 * and group g = rb*(L/GC) + cb. Its N = G*GC segments are numbered
 * mu = j*G + i for row offset i < G and segment offset j < GC; a 64-wide
 * wavefront decodes one group, one segment per lane. Segments are numbered in
 * group order: group g starts at segment GR*rb*L + cb*GC*G.
 *
 * Stream: for each weight of a segment in order, code(el) then code(eh),
 * each emitted most-significant bit first; the stream is packed least
 * significant bit first (bit k is bit k%8 of byte k/8). Segment mu of a group
 * occupies stored(mu) = base + seg_len[mu] bits: its codes, then zero bits up
 * to that length. base is the least code-bit count among the group's
 * segments, or the greatest minus 255 when they span more than 255 bits (the
 * shorter segments are then padded to base), so that every seg_len fits one
 * byte. The segments of a group are concatenated in mu order; each group
 * stream starts on a 16-byte boundary and is zero-padded to a multiple of 128
 * bits. (The paper's decoder reads one stream serially, Sec. 3.2, and needs
 * no lengths; here every segment is decoded from its own start.)
 *
 * Layout (sections start at 64-byte boundaries, zero padding between):
 *   0      header (128 bytes, below)
 *   off_seg_bits  uint8 seg_len[n_seg]      stored bits of each segment over
 *                                           its group's base
 *   off_grp_off   uint32 grp_meta[2n_grp+1] group g: [2g] stream start in
 *                                           16-byte units from off_stream,
 *                                           [2g+1] base; [2n_grp] the end
 *   off_stream    group streams
 *   off_raw       uint8 raw[n]: (s<<7)|m; group g starts at S times its first
 *                 segment number; weight t of segment mu is at ((t/8)*N + mu)*8
 *                 + t%8 within the group
 *   total_bytes = off_raw + n
 * Header: u32 magic 0x31464C48 ('HLF1'), u16 version 2, u8 lmax, u8 flags,
 *   u64 rows, u64 cols, u32 seg_len, u32 group_rows (GR), u64 n_seg,
 *   u64 n_grp, u64 off_seg_bits, u64 off_grp_off, u64 off_stream,
 *   u64 off_raw, u64 total_bytes, u32 max_grp_units, u8 eh_nsym, u8 el_nsym,
 *   u8 eh_single, u8 el_single, u8 eh_len[16], u8 el_len[16].
 *
 * flags 0 is the split format above. flags 1 is the whole-exponent format:
 * the exponent byte e = (w>>7)&255 is one symbol of a single per-matrix code
 * over 256 symbols (the same Huffman, package-merge and canonical rules, with
 * lmax in [8, 13]), and the stream holds code(e) for each weight of a segment
 * in order, most-significant bit first. Its 256 code lengths (u8, indexed by
 * e) follow the header at byte 128, so off_seg_bits = 384. Header bytes
 * 92..93 hold the u16 count of present exponent values, byte 94 the value
 * when it is the only one (else 0), bytes 95..127 are zero. Everything else
 * (tiling, padding, offsets, raw plane) is as in the split format. The split
 * follows the paper's split-size analysis (Sec. 3.1): an 8-bit symbol is
 * costly for a single-cycle CAM match, not for a table lookup in local memory.
 *
 * flags 2 is the float16 format, the paper's {1,5,5,5} split (Sec. 3.1,
 * Sec. 3.2): a float16 weight w is sign s = w>>15 (kept raw), exponent
 * e = (w>>10)&31, mantissa-high mh = (w>>5)&31 and mantissa-low ml = w&31;
 * e, mh and ml each have a per-matrix code over 32 symbols (the same rules,
 * lmax in [5, 12]). The stream holds code(ml), code(e), code(mh) for each
 * weight of a segment in order, each most-significant bit first. A 128-byte
 * section after the header holds three records (e, mh, ml) of u8 nsym,
 * u8 single, u8 len[32], then zeros; off_seg_bits = 256; header bytes 92..127
 * are zero. The raw plane holds only signs: byte k*(S/8) + t/8, bit t%8 is the
 * sign of weight t of the segment numbered k in group order, and
 * total_bytes = off_raw + n/8.
 *
 * ---------------------------------------------------------------------------
 * Conventions of the ABI
 * ---------------------------------------------------------------------------
 * Pointers named *_dev are device (HBM) pointers; all others are host. The
 * caller owns every buffer; the library allocates no device memory and keeps
 * no state across calls. `stream` is a hipStream_t (NULL = default stream).
 * Launch functions are asynchronous: they validate arguments on the host,
 * enqueue kernels and return; HL_EHIP reports a failed launch. Corruption
 * that only the device could see is not reported: kernels clamp every read
 * to the container, so a damaged stream gives wrong weights, never a fault.
 * No function throws; all are reentrant.
 */
#ifndef HUFFLM_H
#define HUFFLM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HL_OK = 0,
  HL_EINVAL = 1,        /* bad argument (null pointer, size, range) */
  HL_ENOMEM = 2,        /* output buffer too small / host allocation failed */
  HL_ECORRUPT = 3,      /* container fails validation */
  HL_EUNSUPPORTED = 4,  /* valid request this build does not handle */
  HL_EHIP = 5           /* HIP runtime error */
} hl_status;

typedef enum { HL_F32 = 0, HL_BF16 = 1, HL_F16 = 2 } hl_dtype;

#define HL_MAGIC 0x31464C48u
#define HL_VERSION 2u
#define HL_HEADER_BYTES 128u
#define HL_GROUP_SEGS 64u
#define HL_MAX_BATCH 16u
#define HL_LUT_BYTES 49440u   /* decode tables of the largest format (float16) */
#define HL_LEN8_BYTES 256u    /* whole-exponent code lengths after the header */
#define HL_LMAX8_MIN 8u
#define HL_LMAX8_MAX 13u
#define HL_CB16_BYTES 128u    /* float16 code tables after the header */
#define HL_LMAX16_MIN 5u
#define HL_LMAX16_MAX 12u
#define HL_PAIR_MAX 11u       /* the fused kernel's table window: pairs of codes up to it take the fast form */
#define HL_NOALLOC_SCRATCH_BYTES (4u << 20)  /* scratch of hl_decode_gemv_noalloc, per GPU */

typedef enum { HL_FORMAT_SPLIT = 0, HL_FORMAT_WHOLE_EXPONENT = 1, HL_FORMAT_FP16 = 2 } hl_format;

typedef struct {
  uint8_t nsym;     /* symbols present in the field (1..16) */
  uint8_t single;   /* the symbol when nsym == 1, else 0 */
  uint8_t len[16];  /* code length per symbol; 0 = absent (or the only one) */
} hl_field_code;

typedef struct {
  uint32_t lmax;    /* code-length limit used to build the lengths, 4..15 */
  hl_field_code eh; /* exponent bits 7..4 */
  hl_field_code el; /* exponent bits 3..0 */
} hl_codebook;

/* Whole-exponent code (format 1). */
typedef struct {
  uint32_t lmax;      /* code-length limit used to build the lengths, 8..13 */
  uint16_t nsym;      /* exponent values present (1..256) */
  uint8_t single;     /* the value when nsym == 1, else 0 */
  uint8_t reserved;   /* 0 */
  uint8_t len[256];   /* code length per exponent value; 0 = absent (or the only one) */
} hl_codebook8;

/* One 5-bit field of the float16 format. */
typedef struct {
  uint8_t nsym;     /* symbols present (1..32) */
  uint8_t single;   /* the symbol when nsym == 1, else 0 */
  uint8_t len[32];  /* code length per symbol; 0 = absent (or the only one) */
} hl_field_code5;

/* Float16 codes (format 2). */
typedef struct {
  uint32_t lmax;       /* code-length limit used to build the lengths, 5..12 */
  hl_field_code5 e;    /* exponent, bits 14..10 */
  hl_field_code5 mh;   /* mantissa bits 9..5 */
  hl_field_code5 ml;   /* mantissa bits 4..0 */
} hl_codebook16;

/* Non-owning view of one container resident in device memory. */
typedef struct {
  const uint8_t* blob_dev;   /* whole container */
  uint32_t* lut_dev;         /* HL_LUT_BYTES, filled by hl_tensor_prepare */
  uint64_t rows, cols, n_seg, n_grp, total_bytes;
  uint64_t off_seg_bits, off_grp_off, off_stream, off_raw;
  uint32_t seg_len, grp_rows, lmax, max_grp_units;
  uint32_t max_seg_bits;     /* the longest stored segment (base + seg_len) */
  uint32_t format;           /* hl_format: which of cb / cb8 / cb16 is in use (the others are zero) */
  hl_codebook cb;
  hl_codebook8 cb8;
  hl_codebook16 cb16;
} hl_tensor;

/* Text of a status code (static storage). */
const char* hl_status_str(hl_status s);

/* Segment length the encoder uses for `cols` when asked for 0: among the
 * multiples of 8 in [8, 128] that divide cols with cols/S a multiple of 4
 * (16-row groups), the one nearest to 64 by ratio, the larger on a tie; if
 * there is none, among the multiples of 8 in [8, 512] that divide cols, the
 * one nearest to 128; 0 if there is none. */
uint32_t hl_default_seg_len(uint64_t cols);

/* Per-matrix codebooks of the two exponent fields (Sec. 5.1) from n bf16
 * bit patterns. Each code is limited to lmax bits, lmax in [4, 15] (12
 * matches the maximum code length the paper reports, Sec. 5.2). With
 * pair_max > 0 the longest eh code plus the longest el code is also at most
 * pair_max bits, so that one window of pair_max bits holds every weight's two
 * codes (the decoder's window match of Sec. 3.2 applied to the pair one
 * table lookup decodes): among the splits a + (pair_max - a) of the limit,
 * a = 0 .. lmax, the codes of least total length (each the length-limited
 * optimum for its limit), the smallest a on a tie. 11 is the fused kernel's
 * table window (HL_PAIR_MAX); 0 = no joint limit. Errors: HL_EINVAL for
 * n == 0, null pointers, lmax out of range, pair_max above 30 or too small
 * for the alphabets. */
hl_status hl_build_codebook(const uint16_t* w_bf16, size_t n, uint32_t lmax, uint32_t pair_max,
                            hl_codebook* out);

/* Group rows the encoder uses when asked for 0: 16 (16 rows x 4 segments)
 * when 4 divides the segments per row, else 32, else 64. */
uint32_t hl_default_grp_rows(uint64_t cols, uint32_t seg_len);

/* Encode W [rows][cols] (bf16 bit patterns, host) into an HLF1 container
 * (Sec. 3.1: once, offline, on the CPU). seg_len 0 selects
 * hl_default_seg_len(cols); grp_rows 0 selects hl_default_grp_rows. With
 * out == NULL, *out_bytes receives the exact size; otherwise *out_bytes is the
 * capacity of `out` on entry and the size written on return (HL_ENOMEM if too
 * small). nthreads 0 = the CPUs of the calling process's affinity mask (at most 64); the
 * output does not depend on nthreads.
 * Errors: HL_EINVAL (shape, seg_len, grp_rows, a weight whose field has no
 * code in `cb`). */
hl_status hl_encode(const uint16_t* w_bf16, uint64_t rows, uint64_t cols,
                    const hl_codebook* cb, uint32_t seg_len, uint32_t grp_rows,
                    uint32_t nthreads, void* out, size_t* out_bytes);

/* Whole-exponent code (format 1) of n bf16 bit patterns: one code over the
 * 256 exponent values (the 8-bit symbols of the split-size analysis,
 * Sec. 3.1), built by the same rules as hl_build_codebook. lmax in [8, 13]
 * (the decode table's 13-bit window then matches every code in one lookup).
 * Errors: HL_EINVAL for n == 0, null pointers or lmax out of range. */
hl_status hl_build_codebook8(const uint16_t* w_bf16, size_t n, uint32_t lmax,
                             hl_codebook8* out);

/* Encode W into an HLF1 container of the whole-exponent format (flags 1).
 * Arguments, size query and errors as hl_encode. */
hl_status hl_encode8(const uint16_t* w_bf16, uint64_t rows, uint64_t cols,
                     const hl_codebook8* cb, uint32_t seg_len, uint32_t grp_rows,
                     uint32_t nthreads, void* out, size_t* out_bytes);

/* Float16 codes (format 2, the paper's {1,5,5,5} split, Sec. 3.1) of n
 * float16 bit patterns: one code per 5-bit field, built by the same rules as
 * hl_build_codebook. lmax in [5, 12]. Errors: HL_EINVAL for n == 0, null
 * pointers or lmax out of range. */
hl_status hl_build_codebook16(const uint16_t* w_f16, size_t n, uint32_t lmax,
                              hl_codebook16* out);

/* Encode a float16 matrix W [rows][cols] into an HLF1 container of the
 * float16 format (flags 2). Arguments, size query and errors as hl_encode. */
hl_status hl_encode16(const uint16_t* w_f16, uint64_t rows, uint64_t cols,
                      const hl_codebook16* cb, uint32_t seg_len, uint32_t grp_rows,
                      uint32_t nthreads, void* out, size_t* out_bytes);

/* Full structural check of a container held in host memory: header, section
 * offsets, codebooks (Kraft sum exactly 1, lengths <= lmax), per-group
 * stream sizes against the stored segment lengths (base + seg_len, each at
 * most S times the longest code of a weight). O(n_seg). Returns HL_OK or
 * HL_ECORRUPT. */
hl_status hl_validate(const void* blob_host, size_t blob_bytes);

/* Build a device view of a container copied to `blob_dev` (blob_bytes long)
 * from its host copy `blob_host` (the same bytes), which is fully validated
 * (as hl_validate, O(n_seg)): the compressed weights stay resident in device
 * memory in this form and are never expanded there (Sec. 1 contributions:
 * weights kept compressed in memory, decompressed only to be multiplied).
 * lut_dev must point to HL_LUT_BYTES of device memory that the view uses
 * from now on. blob_dev and lut_dev must be 16-byte aligned (the kernels
 * copy both in 16-byte pieces). Errors: HL_EINVAL (also for a misaligned
 * pointer), HL_ECORRUPT. */
hl_status hl_tensor_view(const void* blob_dev, const void* blob_host,
                         size_t blob_bytes, uint32_t* lut_dev, hl_tensor* out);

/* Fill t->lut_dev on the device: the joint decode table of the two codes for
 * a 13-bit window (the decoder's L_max-bit window match of Sec. 3.2) and the
 * per-length canonical tables used for pairs longer than the window. In the
 * whole-exponent format the table decodes the one exponent code (never
 * longer than the window) and the per-length tables are zero. */
hl_status hl_tensor_prepare(const hl_tensor* t, void* stream);

/* Device buffers of the calls below (x, decoded weights, workspaces, plain
 * bf16 weights) are read or written in 16-byte pieces and must be 16-byte
 * aligned (any hipMalloc or torch allocation is); float32 outputs must be
 * 4-byte aligned. A misaligned pointer gives HL_EINVAL. */

/* Decode the whole matrix to bf16 bit patterns (float16 for the float16
 * format), out_dev[rows*cols] (row-major): the decoder of Sec. 3.2 (window
 * match, symbol, pointer advance by the code length, concatenation with the
 * raw sign and mantissa) without the product; the layer-wise full
 * decompression the paper contrasts with its own (Sec. 1, Sec. 2.1).
 * Bit-exact with the encoder's input. Errors: HL_EINVAL (also for a
 * misaligned out_dev). */
hl_status hl_decode(const hl_tensor* t, uint16_t* out_dev, void* stream);

/* Bytes of device workspace hl_decode_gemv may use for `t` at this batch
 * (the tiled activations of larger batches and the cross-block partial sums;
 * 0 on bad arguments). */
size_t hl_gemv_workspace_bytes(const hl_tensor* t, uint32_t batch);

/* y[b][r] = sum_k W[r][k] * x[b][k] for b < batch, decoding W on the fly in
 * registers (Sec. 3.2: weights are decompressed only to be multiplied).
 * x_dev: [batch][cols] float32 or bf16; y_dev: [batch][rows] float32 (fully
 * written). fp32 accumulation; every output is summed in a fixed order, so
 * results do not vary between runs. batch in [1, 16].
 * workspace_dev: hl_gemv_workspace_bytes(t, batch) bytes, zero-filled by the
 * caller once before first use; each call leaves it ready for the next. Calls
 * that may run concurrently need separate workspaces. With NULL (or too
 * small) the product is still computed, with less parallelism for matrices
 * with few rows. Errors: HL_EINVAL (also for misaligned x, y or workspace). */
hl_status hl_decode_gemv(const hl_tensor* t, const void* x_dev, hl_dtype x_dtype,
                         uint32_t batch, float* y_dev, void* workspace_dev,
                         size_t workspace_bytes, void* stream);

/* hl_decode_gemv without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops that
 * forbid allocation): the tiled activations and partial sums go to a scratch
 * array of HL_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it
 * runs on until the process ends (its address is looked up on the first call
 * on a GPU). No device memory is allocated or freed. The arrival counters a
 * split product uses are zeroed by a small kernel on `stream` before it (no
 * memset). Every call on one GPU shares that GPU's scratch: calls that overlap
 * on one GPU (other streams, other host threads) race and give wrong results.
 * Arguments and results as hl_decode_gemv; the same kernels run, so outputs
 * equal hl_decode_gemv's bit for bit. Errors: those of hl_decode_gemv, and
 * HL_EUNSUPPORTED when the product would need more than
 * HL_NOALLOC_SCRATCH_BYTES of scratch. */
hl_status hl_decode_gemv_noalloc(const hl_tensor* t, const void* x_dev, hl_dtype x_dtype,
                                 uint32_t batch, float* y_dev, void* stream);

/* The products of up to 4 matrices that share x, y_devs[m][b][r] =
 * sum_k W_m[r][k] * x[b][k] (a decode step's q, k and v projections, or its
 * gate and up projections), as hl_decode_gemv computes each. ts[m]: views
 * with the same number of columns. When every matrix is in a bf16 format with
 * 16-row groups and segments of 64 weights, x is bf16 and the
 * matrices have at least one row block per CU together, one launch decodes
 * them all: its blocks are divided among the matrices in proportion to their
 * row blocks, so the launch and first-load latency of small matrices is paid
 * once. Otherwise the matrices are multiplied one after another with
 * hl_decode_gemv. workspace_dev: at least the largest
 * hl_gemv_workspace_bytes(ts[m], batch), under hl_decode_gemv's rules.
 * Errors: HL_EINVAL (also for matrices with different column counts), and
 * those of hl_decode_gemv. */
hl_status hl_decode_gemv_multi(const hl_tensor* const* ts, uint32_t count, const void* x_dev,
                               hl_dtype x_dtype, uint32_t batch, float* const* y_devs,
                               void* workspace_dev, size_t workspace_bytes, void* stream);

/* Bytes of device workspace hl_decode_gemm needs for `tokens` activation rows:
 * up to 64 tokens the partial sums of up to one range per column block of
 * four segments (on the persistent kernel's matrices, up to 64 tokens, only
 * the tiled activations use it), beyond that the decoded weights
 * (rows * cols * 2); 0 for tensors it does not take. */
size_t hl_gemm_workspace_bytes(const hl_tensor* t, uint32_t tokens);

/* Prefill product Y[n][r] = sum_k W[r][k] * X[n][k] for n < tokens (many
 * activation rows; the paper's prompts of tens of tokens, Sec. 4). Up to 64
 * tokens on matrices with at least one 16-row block per compute unit, the
 * persistent fused decode-GEMV multiplies each decoded 8-weight step with
 * one, two or four 16-token tiles (the activations first copied to the
 * workspace in chunks of 16 rows per tile; four tiles for S = 64 and stream
 * columns of 16 words or more); otherwise, up to 64 tokens, each 16-row x 4-segment
 * weight tile is decoded once per chunk of up to 128 tokens and multiplied
 * with all of them on the matrix cores (Sec. 3.2: weights decompressed only
 * to be multiplied); every output summed in a fixed order; beyond that, where the product is compute-bound (Sec. 5), the
 * matrix is decoded once into the workspace (hl_decode) and multiplied by
 * hipBLASLt. x_dev: [tokens][cols] bf16; y_dev: [tokens][rows] float32 (fully
 * written); fp32 accumulation. bf16 formats (split or whole exponent) with
 * 16-row groups and S = 32 or 64; others give HL_EUNSUPPORTED.
 * workspace_dev: hl_gemm_workspace_bytes(t, tokens) bytes (no initial
 * contents needed); calls that may run concurrently need separate
 * workspaces. Errors: HL_EINVAL (also for a missing or short workspace). */
hl_status hl_decode_gemm(const hl_tensor* t, const void* x_dev, hl_dtype x_dtype, uint32_t tokens,
                         float* y_dev, void* workspace_dev, size_t workspace_bytes, void* stream);

/* Uncompressed comparator: the same product from plain bf16 W [rows][cols]
 * in device memory. */
hl_status hl_gemv_bf16(const uint16_t* w_dev, uint64_t rows, uint64_t cols,
                       const void* x_dev, hl_dtype x_dtype, uint32_t batch,
                       float* y_dev, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* HUFFLM_H */
