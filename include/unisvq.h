/*
 * unisvq.h -- C ABI of libunisvq, the MI355X (gfx950) inference path of
 * UniSVQ 2-bit affine-lattice quantised linear layers.
 *
 * The operation (paper "UniSVQ: 2-bit Unified Scalar-Vector Quantization"):
 *   A weight matrix W (N output features x K input features) is stored as
 *   integer codes q in {0,1,2,3}.  Every d = 4 consecutive input columns of
 *   one output row form a vector, rebuilt as an affine image of its lattice
 *   point:   w_hat = A q + B,  A in R^{4x4}, B in R^4          (Sec. 3.1, Eq. 4)
 *   Vector i of a row covers input columns 4i..4i+3           (Sec. 3.2.3, Eq. 8)
 *   and the layer output is  Y = X W_hat^T                     (Sec. 2.1, Eq. 1)
 *   The affine map commutes with the matrix product (Sec. 3.1; Sec. 3.2.3,
 *   Eq. 9), so the kernels never materialise W_hat in memory.
 *   Granularity: one (A, B) pair per (output row, group of 128 input
 *   columns), stored as fp16 -- 40 bytes per set (Sec. 3.1).  The paper's
 *   one-pair-per-matrix setting (Sec. 4.2) is the special case where all
 *   pairs are equal.
 *
 * Conventions shared by every entry point
 *   - Pointers named "device" are device memory owned by the caller; the
 *     library never allocates, frees or keeps them.  Host pointers are named.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All
 *     work is enqueued asynchronously on it; no call synchronises.
 *   - Returns UNISVQ_OK (0) or a negative unisvq_status.  Argument errors are
 *     detected on the host before anything is enqueued (so they can be tested
 *     without a GPU).  A failed launch returns UNISVQ_EHIP.  Faults inside a
 *     kernel surface at the caller's next synchronisation.
 *   - Outputs are overwritten, never accumulated into.
 *   - Thread-safe: no global mutable state besides the kernels' dynamic-LDS
 *     limits, raised on first use once per (kernel, device) -- on the device
 *     current when the call is made.
 *   - Shapes: N % 16 == 0, K % 128 == 0, N >= 16, K >= 128, M >= 1.
 *
 * ---------------------------------------------------------------------------
 * Packed weight format, version 1 (bytes little endian)
 *   Canonical inputs: Q uint8 [N][K] (values 0..3); A fp16 [N][K/128][4][4],
 *   A[r][g][a][b] multiplies q_b into output component a; B fp16 [N][K/128][4].
 *   Total size N*K/4 + N*(K/128)*40 bytes (4.5 bits per weight), no padding.
 *
 *   Row block rb (rows 16rb..16rb+15) occupies (K/128)*1152 consecutive bytes
 *   starting at rb*(K/128)*1152.  Within it, groups g = 0..K/128-1 are taken
 *   in pairs: packet p holds groups 2p and 2p+1 (2304 bytes, at p*2304); when
 *   K/128 is odd a final half packet holds the last group (1152 bytes).
 *   Slot s = 0..63 of a packet stands for row r = 16rb + s/4 and component
 *   b = s%4.
 *     full packet at offset P, j = 0 for group 2p, j = 1 for group 2p+1:
 *       P +        16s + 8j   8-byte code field F(r, 2p+j, b)
 *       P + 1024 + 16s + 8j   A[r][2p+j][a][b] for a = 0..3, fp16 each
 *       P + 2048 +  4s + 2j   B[r][2p+j][b], fp16
 *     half packet at offset P (group g):
 *       P +        8s         F(r, g, b)
 *       P +  512 + 8s         A[r][g][0..3][b]
 *       P + 1024 + 2s         B[r][g][b]
 *   Code field F(r, g, b): 64-bit little-endian word whose bits 2v, 2v+1 hold
 *   Q[r][128g + 4v + b], v = 0..31 (component b of the group's 32 vectors).
 *
 *   One packet slot is exactly the data one lane of a 64-lane wavefront
 *   consumes, so every load of the matrix-vector kernel is a fully coalesced
 *   16-byte-per-lane read.
 * ---------------------------------------------------------------------------
 * Codes-only format with row-shared affine parameters (the paper's own
 * setting: one (A, B) pair per weight matrix, Sec. 3.1 and Sec. 4.2; also
 * one pair per 128-column group shared by all rows)
 *   affine_groups Ga = 1 (one pair) or K/128 (one per group); group g uses
 *   pair (Ga == 1 ? 0 : g).  Canonical inputs: Q as above, A fp16 [Ga][4][4],
 *   B fp16 [Ga][4].
 *   Codes: format v1 without its A and B areas -- row block rb occupies
 *   (K/128)*512 bytes at rb*(K/128)*512; packet p (groups 2p, 2p+1) is 1024
 *   bytes at p*1024 with F(r, 2p+j, b) at P + 16s + 8j; a final half packet
 *   (odd K/128) is 512 bytes with F(r, g, b) at P + 8s.  N*K/4 bytes (2 bits
 *   per weight).
 *   Shared affine block: 80-byte records, one per pair of groups (a single
 *   record, holding pair 0 for both of its groups, when Ga = 1):
 *       R*80 + 16b + 8j        A[2R+j][a][b] for a = 0..3, fp16 each
 *       R*80 + 64 + 4b + 2j    B[2R+j][b], fp16
 *   a group past the last (odd K/128, Ga = K/128) holds zeros.  Lane
 *   (beta, b) of a wavefront reads exactly its A column and B values, as from
 *   a full-format packet.
 * ---------------------------------------------------------------------------
 * Variant codes-only format: b-bit codes (b = 2 or 3; Sec. 5.2.5, where only
 * the integer vectors widen) and d-dimensional vectors (d = 4 or 8; Sec.
 * 5.2.3), with row-shared pairs as the paper keeps them (one per weight
 * matrix, Sec. 4.2, or one per 128-column group).  Canonical inputs: Q uint8
 * [N][K] (0..2^b-1); A fp16 [Ga][d][d] (A[a][b] multiplies q_b into output
 * component a), B fp16 [Ga][d]; Ga = 1 or K/128, group g uses pair (Ga == 1
 * ? 0 : g).  Vector i of a row covers input columns d*i .. d*i+d-1.
 *   Codes: a group of a row block takes CB = 512 (b = 2) or 768 (b = 3) bytes;
 *   row block rb starts at rb*(K/128)*CB; packet p (groups 2p, 2p+1) is 2*CB
 *   bytes at p*2*CB, a final half packet (odd K/128) CB bytes.  Slot s = 0..63
 *   stands for row r = 16rb + s/4 and lane index j = s%4; its 32 codes of
 *   group g are numbered (h, u), h = 0..1, u = 0..15:
 *     d = 4: Q[r][128g + 4(16h + u) + j]   (vector 16h+u, component j)
 *     d = 8: Q[r][128g + 8u + 4h + j]      (vector u, component 4h+j)
 *   Low field (8 bytes): 32-bit word h, bits 2u, 2u+1 = bits 0, 1 of code (h, u).
 *   High field (b = 3, 4 bytes): bit 8n + 4m + 2h + p = bit 2 of code
 *   (h, u = 4n + 2m + p).  Full packet at P: low field of group 2p+jj at
 *   P + 16s + 8jj, high field at P + 1024 + 8s + 4jj; half packet: low at
 *   P + 8s, high at P + 512 + 4s.  N*K*b/8 bytes.  (b = 2, d = 4 is exactly the
 *   codes-only format above and is served by the *_shared entry points.)
 *   Shared affine block: records of RB = 160 (d = 4) or 576 (d = 8) bytes, one
 *   per pair of groups (a single record when Ga = 1); record R serves groups
 *   2R + jj with pair pi = (Ga == 1 ? 0 : 2R + jj), zeros for a group past the
 *   last.  Inside a record, fp16 each:
 *     lane view (read by the matrix-vector kernel):
 *       d = 4: A[pi][a][j] at 16j + 8jj + 2a;  B[pi][j] at 64 + 4j + 2jj
 *       d = 8: A[pi][a][4h+j] at 64j + 32jj + 16h + 2a;  B[pi][4h+j] at 256 + 8j + 4jj + 2h
 *     row view (read by the tiled product's weight decode), at V = 80 (d = 4)
 *     or 288 (d = 8), E = 2(d*d + d):
 *       A[pi][a][b] at V + jj*E + 2(d*a + b);  B[pi][a] at V + jj*E + 2*d*d + 2a
 * ---------------------------------------------------------------------------
 */
#ifndef UNISVQ_H
#define UNISVQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define UNISVQ_FORMAT_VERSION 1
#define UNISVQ_GROUP 128   /* input columns per (A, B) set */
#define UNISVQ_DIM 4       /* vector dimension d */
#define UNISVQ_ROW_BLOCK 16

typedef enum {
    UNISVQ_OK = 0,
    UNISVQ_EINVAL = -1,     /* null pointer, M < 1, unknown dtype value */
    UNISVQ_ESHAPE = -2,     /* N % 16 != 0, K % 128 != 0, N < 16 or K < 128 */
    UNISVQ_EUNSUP = -3,     /* valid but unsupported combination (dtype pair, M too large for gemv) */
    UNISVQ_EALIGN = -4,     /* a pointer lacks the alignment stated for it */
    UNISVQ_EHIP = -5,       /* the HIP runtime reported an error at launch */
    UNISVQ_EWORKSPACE = -6, /* workspace smaller than unisvq_gemm_workspace_bytes() */
    UNISVQ_ESCRATCH = -7    /* the product needs more than the fixed scratch of unisvq_gemm_noalloc */
} unisvq_status;

typedef enum {
    UNISVQ_F16 = 0,   /* IEEE binary16 */
    UNISVQ_BF16 = 1,  /* bfloat16 */
    UNISVQ_F32 = 2    /* IEEE binary32 (outputs only) */
} unisvq_dtype;

/* Library and format version (UNISVQ_FORMAT_VERSION). */
int unisvq_version(void);

/* Human-readable name of a status code (static string, never NULL). */
const char* unisvq_status_string(int status);

/* Bytes of the packed buffer for an N x K matrix (format block above);
 * 0 when the shape is invalid.  Host-only, no GPU needed. */
size_t unisvq_packed_bytes(int64_t N, int64_t K);

/* Pack canonical codes and affine parameters into the packed format.
 *   codes     device uint8  [N][K], values 0..3 (Sec. 3.2.2: unsigned codes,
 *             the centring constant lives in B)
 *   A         device fp16 bits [N][K/128][4][4]
 *   B         device fp16 bits [N][K/128][4]
 *   packed    device, unisvq_packed_bytes(N, K) bytes, 16-byte aligned
 *   bad_codes device int32 or NULL: if given, the number of codes above 3 is
 *             ADDED to *bad_codes (the caller zeroes it); such codes are stored
 *             modulo 4.
 * A bit-exact permutation: values are never converted or rounded. */
int unisvq_pack(int64_t N, int64_t K, const uint8_t* codes, const uint16_t* A, const uint16_t* B,
                void* packed, int32_t* bad_codes, void* stream);

/* Exact inverse of unisvq_pack (codes come back in 0..3).  All device. */
int unisvq_unpack(int64_t N, int64_t K, const void* packed, uint8_t* codes, uint16_t* A, uint16_t* B,
                  void* stream);

/* Decode-phase product y = x * W_hat^T for a few tokens (Eq. 1 with Eq. 4/8).
 *   packed  device, packed N x K matrix, 16-byte aligned
 *   x       device [M][K] row-major, dtype x_dtype (F16 or BF16), 16-byte aligned
 *   y       device [M][N] row-major, dtype y_dtype (F16, BF16 or F32)
 *   M       1..4 tokens (UNISVQ_EUNSUP above that; use unisvq_gemm).  The
 *           kernel stages x in LDS: UNISVQ_EUNSUP also when 576 bytes per
 *           token and 256-column packet, M * ceil(K / 256) * 576, plus up to
 *           2 KB of working space exceed the 160 KB of LDS (the largest K is
 *           17920 for M = 4, 36096 for M = 2, 72192 for M = 1);
 *           unisvq_gemm takes any K.
 * Per (row, group) the kernel contracts the activations with the integer
 * codes on the matrix cores and applies A and B to that small result
 * (the affine map commutes with the product, Sec. 3.1), accumulating in fp32
 * and rounding once to y_dtype. */
int unisvq_gemv(int64_t N, int64_t K, const void* packed, int64_t M, const void* x, int x_dtype,
                void* y, int y_dtype, void* stream);

/* One product of a batched decode-phase call. */
typedef struct {
    int64_t N, K;        /* shape of this weight matrix (N % 16 == 0, K % 128 == 0) */
    const void* packed;  /* device, packed N x K matrix, 16-byte aligned */
    const void* x;       /* device [M][K], 16-byte aligned */
    void* y;             /* device [M][N] */
} unisvq_gemv_problem;

#define UNISVQ_MAX_BATCH 8

/* Several independent decode-phase products y_i = x_i * W_hat_i^T in one
 * launch (same M, x_dtype and y_dtype for all).  A decoder layer's query,
 * key and value projections, or its gate and up projections, read the same
 * activations and are independent -- one launch serves them all, which at
 * batch 1 saves a kernel launch per extra matrix.
 *   problems  HOST array of `count` descriptors (1..UNISVQ_MAX_BATCH); read
 *             before the call returns, so the caller may reuse it at once
 *   others    as unisvq_gemv.  Every descriptor is validated before launch. */
int unisvq_gemv_batched(const unisvq_gemv_problem* problems, int count, int64_t M, int x_dtype,
                        int y_dtype, void* stream);

/* Device workspace unisvq_gemm needs for this product, in bytes (0: none):
 * for BF16 activations an fp16 copy of x (M*K*2 bytes, rounded up to 256;
 * above 16 tokens sized for the copy in 16-token tiles, so M counts rounded
 * up to a multiple of 16) and one fp32 scale per token (rounded up to 256);
 * above 16 tokens, for products with too few output tiles to fill the GPU,
 * fp32 partial sums of a split along K (splits*M*N*4 bytes).  From 17 to 32
 * tokens the size covers either kernel below (the one taken may use less).  0 also for an invalid shape, M < 1 or an
 * unknown x_dtype.  Host-only, no GPU needed. */
size_t unisvq_gemm_workspace_bytes(int64_t N, int64_t K, int64_t M, int x_dtype);

/* Prefill product y = x * W_hat^T for any M >= 1 (Eq. 1 with Eq. 4/8).
 * Arguments as unisvq_gemv; x_dtype F16 or BF16, y_dtype F16, BF16 or F32.
 * Up to 3 tokens the matrix-vector kernel of unisvq_gemv computes it (its
 * faster range; the workspace then goes unused), unless K is too long for
 * that kernel's LDS.  Up to 16 tokens -- and up to 32 when the product has
 * fewer than 64 tiles of 128 output rows, where the alternative would split
 * K many ways -- one launch of the small-batch kernel computes it: each
 * wavefront decodes 16-row x 128-column tiles into its own LDS region and
 * multiplies them with all tokens at once; the wavefronts of a workgroup
 * split K and add their sums in a fixed order (no workspace beyond the bf16
 * copy below).  Otherwise each
 * workgroup decodes a 128-row x 128-column weight tile at a time into
 * LDS (every vector A q + B in fp32 from the exact integer codes, rounded
 * once to fp16) and multiplies it with its tokens on the matrix cores
 * (fp16 x fp16, fp32 accumulation); decoded weights never reach global
 * memory.  bf16 activations are first scaled per token by a power of two
 * into [2^14, 2^15) and stored as fp16 in the workspace -- exact for every
 * element within 2^28 of its token's largest magnitude -- and the scale is
 * undone on the fp32 result.  When M is small the K range is split across
 * workgroups and a second kernel sums the fp32 partials in a fixed order
 * (results are reproducible run to run).
 *   BF16 activations need K <= 65536 (UNISVQ_EUNSUP above).
 *   workspace  device, >= unisvq_gemm_workspace_bytes(N, K, M, x_dtype)
 *              bytes, 16-byte aligned (UNISVQ_EWORKSPACE if missing or
 *              smaller, UNISVQ_EALIGN if misaligned); may be NULL when that
 *              size is 0.  Overwritten; the caller owns it. */
int unisvq_gemm(int64_t N, int64_t K, const void* packed, int64_t M, const void* x, int x_dtype,
                void* y, int y_dtype, void* workspace, size_t workspace_bytes, void* stream);

/* Device workspace unisvq_gemm_batched needs for these problems and M, in
 * bytes: the 256-byte-aligned sum of unisvq_gemm_workspace_bytes of each
 * problem (problem i uses its own slice, in order).  0 when none is needed or
 * for invalid arguments.  problems: HOST array of `count` descriptors.
 * Host-only. */
size_t unisvq_gemm_batched_workspace_bytes(const unisvq_gemv_problem* problems, int count, int64_t M, int x_dtype);

/* Several independent products y_i = x_i * W_hat_i^T of the same M and
 * dtypes (a decoder's query, key and value projections, or its gate and up
 * projections, at a small batch).  For M <= 16 all of them run in ONE launch
 * (of the matrix-vector kernel up to 3 tokens, as unisvq_gemm does, else of
 * the small-batch kernel), with the results of unisvq_gemm on each bit for
 * bit; so also from 17 to 32 tokens when all the batch's rows make fewer than
 * 64 tiles of 128 (unisvq_gemm's rule applied to the whole batch); otherwise
 * in ONE launch of the tiled product, planned over the whole
 * batch, plus one reduction launch when the batch's tiles leave CUs idle and
 * K is split -- the same arithmetic as unisvq_gemm, but the K split (and so
 * the grouping of the fp32 partial sums) follows the batch, so results can
 * differ from single calls in the last bits (bf16 activations first pass
 * through the per-problem pre-pass into their workspace slice; activations
 * above 2 GiB fall back to one product at a time, as single calls).
 *   problems   HOST array of `count` descriptors (1..UNISVQ_MAX_BATCH), read
 *              before the call returns; packed format v1 weights; every
 *              descriptor is validated before anything is enqueued
 *   workspace  device, >= unisvq_gemm_batched_workspace_bytes(...) bytes,
 *              16-byte aligned (UNISVQ_EWORKSPACE / UNISVQ_EALIGN); may be
 *              NULL when that size is 0 */
int unisvq_gemm_batched(const unisvq_gemv_problem* problems, int count, int64_t M, int x_dtype, int y_dtype,
                        void* workspace, size_t workspace_bytes, void* stream);

/* unisvq_gemm for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same kernels, arguments (minus the workspace), results and errors, with the
 * workspace taken from a scratch array of the library itself --
 * unisvq_noalloc_scratch_bytes() (32 MiB) per device, held until the process
 * ends; no call allocates or frees anything.  The first call on a device looks
 * the array's device address up (with that device current).
 *   UNISVQ_ESCRATCH (before any launch) when the product needs more than the
 *   scratch, i.e. unisvq_gemm_workspace_bytes(N, K, M, x_dtype) exceeds it:
 *   with bf16 activations the fp16 copy of x takes M*K*2 bytes (M rounded up
 *   to 16 above 16 tokens), and a product split along K takes splits*M*N*4.
 * Every call on a device shares that device's scratch, so calls that overlap
 * on one device (different streams, different host threads) race; calls in
 * order on one stream do not.  Nothing in the scratch needs to start at zero:
 * each call writes every byte it reads. */
size_t unisvq_noalloc_scratch_bytes(void);
int unisvq_gemm_noalloc(int64_t N, int64_t K, const void* packed, int64_t M, const void* x, int x_dtype, void* y,
                        int y_dtype, void* stream);

/* ---- Row-shared affine parameters (codes-only format block above) ---- */

/* Bytes of the codes-only buffer for an N x K matrix (N*K/4); 0 when the
 * shape is invalid.  Host-only. */
size_t unisvq_codes_bytes(int64_t N, int64_t K);

/* Bytes of the shared affine block: 80 for affine_groups == 1, else
 * 80*ceil(K/256) for affine_groups == K/128; 0 for any other value or an
 * invalid K.  Host-only. */
size_t unisvq_shared_affine_bytes(int64_t K, int64_t affine_groups);

/* Pack codes and row-shared pairs (all device):
 *   codes          uint8 [N][K], values 0..3
 *   A, B           fp16 bits [affine_groups][4][4] and [affine_groups][4]
 *   packed_codes   unisvq_codes_bytes(N, K) bytes, 16-byte aligned
 *   packed_affine  unisvq_shared_affine_bytes(K, affine_groups) bytes, 16-byte aligned
 *   bad_codes      as unisvq_pack
 * UNISVQ_EINVAL when affine_groups is neither 1 nor K/128.  Bit exact. */
int unisvq_pack_shared(int64_t N, int64_t K, int64_t affine_groups, const uint8_t* codes, const uint16_t* A,
                       const uint16_t* B, void* packed_codes, void* packed_affine, int32_t* bad_codes,
                       void* stream);

/* Exact inverse of unisvq_pack_shared.  All device. */
int unisvq_unpack_shared(int64_t N, int64_t K, int64_t affine_groups, const void* packed_codes,
                         const void* packed_affine, uint8_t* codes, uint16_t* A, uint16_t* B, void* stream);

/* unisvq_gemv with codes-only weights and row-shared pairs: the same
 * arithmetic, M and K limits, dtypes and error behaviour; only the 2-bit
 * codes stream from memory (the shared block is read from cache).
 * packed_codes and packed_affine 16-byte aligned. */
int unisvq_gemv_shared(int64_t N, int64_t K, int64_t affine_groups, const void* packed_codes,
                       const void* packed_affine, int64_t M, const void* x, int x_dtype, void* y, int y_dtype,
                       void* stream);

/* One product of a batched call with row-shared pairs. */
typedef struct {
    int64_t N, K, affine_groups;
    const void* packed_codes;   /* device, 16-byte aligned */
    const void* packed_affine;  /* device, 16-byte aligned */
    const void* x;              /* device [M][K], 16-byte aligned */
    void* y;                    /* device [M][N] */
} unisvq_gemv_shared_problem;

/* unisvq_gemv_batched for row-shared pairs (each problem has its own). */
int unisvq_gemv_shared_batched(const unisvq_gemv_shared_problem* problems, int count, int64_t M, int x_dtype,
                               int y_dtype, void* stream);

/* unisvq_gemm with codes-only weights and row-shared pairs: the same decode
 * (A q + B exactly in fp32, one rounding to fp16), tiling, K split, bf16
 * handling and workspace -- size it with unisvq_gemm_workspace_bytes. */
int unisvq_gemm_shared(int64_t N, int64_t K, int64_t affine_groups, const void* packed_codes,
                       const void* packed_affine, int64_t M, const void* x, int x_dtype, void* y, int y_dtype,
                       void* workspace, size_t workspace_bytes, void* stream);

/* Device workspace unisvq_gemm_shared_fold needs, in bytes: the folded
 * activations in fp16 (16-token tiles: M rounded up to a multiple of 16,
 * times K*2, rounded up to 256), one fp32 scale and one fp32 bias term per
 * token (each array rounded up to 256), and the fp32 partial sums when the
 * product is split along K (small M).  0 for an invalid shape or M < 1.
 * Host-only. */
size_t unisvq_gemm_fold_workspace_bytes(int64_t N, int64_t K, int64_t M);

/* Prefill product with row-shared pairs computed through the fold of Eq. 9
 * (Sec. 3.2.3): with A, B shared by the rows, y = sum_v (x_v A) q_v +
 * sum_v x_v B, so a pre-pass forms x'_v = A^T x_v for every 4-column vector
 * v of x (the pair of v's group; fp32 from the fp16 pair, then a per-token
 * power-of-two scale into [2^14, 2^15) and one rounding to fp16) and the
 * per-token bias term c = sum_v x_v . B (fp32, fixed summation order); the
 * tiled kernel then multiplies x' by the bare 2-bit codes on the matrix cores
 * (fp16 operands: the codes are exact, fp32 accumulation) and adds c.  No
 * weight is ever decoded.  The result differs from unisvq_gemm_shared only
 * in rounding (x' is rounded instead of the decoded weight).
 *   Arguments as unisvq_gemm_shared; any M >= 1, x_dtype F16 or BF16,
 *   y_dtype F16, BF16 or F32; (M rounded up to 16) * K * 2 must not exceed
 *   2^31 - 1 bytes (UNISVQ_EUNSUP otherwise).
 *   workspace  device, >= unisvq_gemm_fold_workspace_bytes(N, K, M) bytes,
 *              16-byte aligned (UNISVQ_EWORKSPACE if missing or smaller,
 *              UNISVQ_EALIGN if misaligned).  Overwritten; the caller owns it. */
int unisvq_gemm_shared_fold(int64_t N, int64_t K, int64_t affine_groups, const void* packed_codes,
                            const void* packed_affine, int64_t M, const void* x, int x_dtype, void* y, int y_dtype,
                            void* workspace, size_t workspace_bytes, void* stream);

/* ---- Format variants (variant codes-only format block above) ----
 * (b, d) = (3, 4), (2, 8) or (3, 8); any other pair is UNISVQ_EUNSUP (b = 2,
 * d = 4 uses the *_shared entry points). */

/* Bytes of the variant codes for an N x K matrix (N*K*bits/8); 0 for an
 * invalid shape or an unsupported (bits, d).  Host-only. */
size_t unisvq_var_codes_bytes(int64_t N, int64_t K, int bits, int d);

/* Bytes of the variant shared affine block: RB for affine_groups == 1, else
 * RB*ceil(K/256) for affine_groups == K/128 (RB = 160 for d = 4, 576 for
 * d = 8); 0 for anything else.  Host-only. */
size_t unisvq_var_affine_bytes(int64_t K, int64_t affine_groups, int bits, int d);

/* Pack codes and row-shared pairs into the variant format (all device):
 *   codes          uint8 [N][K], values 0..2^bits-1
 *   A, B           fp16 bits [affine_groups][d][d] and [affine_groups][d]
 *   packed_codes   unisvq_var_codes_bytes(N, K, bits, d) bytes, 16-byte aligned
 *   packed_affine  unisvq_var_affine_bytes(K, affine_groups, bits, d) bytes, 16-byte aligned
 *   bad_codes      as unisvq_pack (codes >= 2^bits counted, stored modulo 2^bits)
 * UNISVQ_EINVAL when affine_groups is neither 1 nor K/128.  Bit exact. */
int unisvq_var_pack(int64_t N, int64_t K, int bits, int d, int64_t affine_groups, const uint8_t* codes,
                    const uint16_t* A, const uint16_t* B, void* packed_codes, void* packed_affine,
                    int32_t* bad_codes, void* stream);

/* Exact inverse of unisvq_var_pack (A and B read from the lane view).  All device. */
int unisvq_var_unpack(int64_t N, int64_t K, int bits, int d, int64_t affine_groups, const void* packed_codes,
                      const void* packed_affine, uint8_t* codes, uint16_t* A, uint16_t* B, void* stream);

/* Decode-phase product with variant weights: the matrix-vector kernel with
 * T = sum_v x_v q_v^T per (row, group, token) formed on the matrix cores --
 * for d = 8 as four 4 x 4 quadrants, for 3-bit codes as the low part plus 4
 * times the high bit (q = lo + 4 hi) accumulated in the same chain -- then
 * sum A o T + B . xbar in fp32, one rounding to y_dtype.  M 1..4, dtypes,
 * LDS limit on K and errors as unisvq_gemv; packed_codes, packed_affine and x
 * 16-byte aligned. */
int unisvq_var_gemv(int64_t N, int64_t K, int bits, int d, int64_t affine_groups, const void* packed_codes,
                    const void* packed_affine, int64_t M, const void* x, int x_dtype, void* y, int y_dtype,
                    void* stream);

/* Several independent variant products in one launch (all with the same
 * bits and d; descriptors as unisvq_gemv_shared_batched, HOST array of
 * 1..UNISVQ_MAX_BATCH entries). */
int unisvq_var_gemv_batched(const unisvq_gemv_shared_problem* problems, int count, int bits, int d, int64_t M,
                            int x_dtype, int y_dtype, void* stream);

/* Device workspace unisvq_var_gemm needs (bytes; 0: none): the bf16 copy of
 * x as for unisvq_gemm, and fp32 partial sums when the K range is split
 * (every M goes to the tiled kernel here, so small M splits K).  Host-only. */
size_t unisvq_var_gemm_workspace_bytes(int64_t N, int64_t K, int64_t M, int x_dtype);

/* Prefill product with variant weights, any M: the tiled kernel of
 * unisvq_gemm with the variant decode (every vector A q + B exactly in fp32
 * on the matrix cores -- d = 8 as two output halves of two chained 4-column
 * steps, 3-bit codes as lo + 4 hi -- rounded once to fp16 in LDS).  Dtypes,
 * bf16 handling, K split and errors as unisvq_gemm; workspace sized by
 * unisvq_var_gemm_workspace_bytes. */
int unisvq_var_gemm(int64_t N, int64_t K, int bits, int d, int64_t affine_groups, const void* packed_codes,
                    const void* packed_affine, int64_t M, const void* x, int x_dtype, void* y, int y_dtype,
                    void* workspace, size_t workspace_bytes, void* stream);

/* ---- Nearest-codeword quantisation (Sec. 3.2.2, without Hessian feedback) ----
 * Codes of the affine-lattice point closest to each vector of d = 4
 * consecutive weights of a row: q* = argmin over the 256 codes q of
 * ||A q + B - w||^2, where (A, B) is the vector's pair.  The decision is taken
 * in fp64 with a fixed operation order (c_a = B_a + A_a0 q_0 + ... + A_a3 q_3
 * left to right, e_a = c_a - w_a, d = fma(e_a, e_a, d) for a = 0..3), and ties
 * go to the lowest index q_0 + 4 q_1 + 16 q_2 + 64 q_3.
 *   W              device fp32 [N][K], 16-byte aligned
 *   A, B           device fp16 bits: affine_groups == 0 -> one pair per (row,
 *                  group), [N][K/128][4][4] and [N][K/128][4]; affine_groups
 *                  == 1 or K/128 -> row-shared pairs [affine_groups][4][4] and
 *                  [affine_groups][4]; any other value: UNISVQ_EINVAL
 *   codes          device uint8 [N][K] (0..3), 4-byte aligned; pack it with
 *                  unisvq_pack or unisvq_pack_shared */
int unisvq_quantize(int64_t N, int64_t K, const float* W, const uint16_t* A, const uint16_t* B,
                    int64_t affine_groups, uint8_t* codes, void* stream);

/* ---- LDLQ: nearest-codeword rounding with Hessian error feedback (Sec. 3.2.2, Eq. 7) ----
 * Vectors of d = 4 consecutive columns are rounded left to right; before
 * vector j (columns 4j..4j+3) is rounded its weights are moved by the errors of
 * all earlier columns,  u_c = W[r][4j+c] + sum_{k < 4j} E[r][k] U[k][4j+c],
 * E = W - W_hat, and u is rounded with the decision of unisvq_quantize (fp64,
 * same operation order, ties to the lowest index).  U is the unit upper
 * block-triangular factor of H = U D U^T (4 x 4 identity blocks on the
 * diagonal, D block diagonal; H the layer's input Hessian, regularised by
 * mu I with mu = 0.01 in Sec. 4.2), e.g. from unisvq_ldl.  Each sum is
 * evaluated as one fma chain in increasing k from 0, then u = W + sum, so the
 * codes are those of a plain sequential evaluation bit for bit.
 *   W          device fp32 [N][K], 16-byte aligned
 *   U          device fp64 [K][K] row-major, 16-byte aligned; only U[k][c] with
 *              k < 4 floor(c / 4) is read
 *   A, B       device fp16 bits, pair layouts as unisvq_quantize (affine_groups
 *              0: per (row, group); 1 or K/128: row-shared)
 *   codes      device uint8 [N][K] (0..3), 4-byte aligned
 *   workspace  device, >= unisvq_ldlq_workspace_bytes(N, K) bytes (fp64 running
 *              feedback and one block of errors), 16-byte aligned; overwritten
 * Work: K/128 pairs of launches (each block of 128 columns: rounding with
 * in-block feedback, then the feedback to every later column). */
size_t unisvq_ldlq_workspace_bytes(int64_t N, int64_t K);
int unisvq_ldlq(int64_t N, int64_t K, const float* W, const double* U, const uint16_t* A, const uint16_t* B,
                int64_t affine_groups, uint8_t* codes, void* workspace, size_t workspace_bytes, void* stream);

/* ---- Block LDL^T factorisation of the Hessian for LDLQ (Sec. 3.2.2, Eq. 7) ----
 * The factor unisvq_ldlq takes: H = U D U^T with U unit upper
 * block-triangular (4 x 4 identity blocks on the diagonal, zeros below them)
 * and D block diagonal (4 x 4 blocks), U's off-diagonal entries being Eq. 7's
 * feedback coefficients.  Computed in fp64 from the last pivot block to the
 * first (D_j = S_jj, U[0:j, j] = S[0:j, j] D_j^-1, S[0:j, 0:j] -= U[0:j, j] D_j
 * U[0:j, j]^T, S the part not yet factorised), blocked over 64-column panels;
 * results differ from another LDL^T or Cholesky-based factorisation only by
 * rounding.
 *   K          128 <= K <= 32768, K % 128 == 0 (UNISVQ_ESHAPE otherwise)
 *   H          device fp64 [K][K] row-major, 16-byte aligned, symmetric
 *              positive definite (e.g. regularised by mu I); only the upper
 *              triangle H[a][b], a <= b, is read
 *   U          device fp64 [K][K] row-major, 16-byte aligned, written in full;
 *              U == H factorises in place (H is then overwritten), any other
 *              overlap is UNISVQ_EINVAL
 *   D          device fp64 [K/4][4][4], or NULL
 *   info       device int32, or NULL: set to 0, or to 1 + the index of the
 *              first pivot block found not positive definite (blocks are taken
 *              last to first), after which U and D are meaningless.  The launches
 *              are asynchronous: read it after synchronising the stream.
 *   workspace  device, >= unisvq_ldl_workspace_bytes(K) bytes (K x 64 fp64 and
 *              the panel's pivot inverses), 16-byte aligned; overwritten
 * Work: one set-up launch and 3 K/64 - 2 launches of the panel steps.
 * unisvq_ldl_workspace_bytes returns 0 for a K outside the range above. */
size_t unisvq_ldl_workspace_bytes(int64_t K);
int unisvq_ldl(int64_t K, const double* H, double* U, double* D, int32_t* info, void* workspace,
               size_t workspace_bytes, void* stream);

/* ---- Randomized Hadamard transform around the product (Sec. 3.2.1, Eq. 5) ----
 * The weights are quantised in the rotated basis W_rot = U S_U W S_V V (S_U,
 * S_V random sign diagonals, U, V Hadamard matrices normalised to be
 * orthogonal), so a layer computes y = ((x S_V V) W_rot^T) U S_U:
 *   mode 0 (input side):   y = (x diag(signs)) H_n / sqrt(n)    -> feeds the product
 *   mode 1 (output side):  y = (x H_n / sqrt(n)) diag(signs)    -> after the product
 * for M rows of length n.  Hadamard matrix of order n: n = 2^k * m with the
 * largest k such that m = 1 or m = q + 1 for a prime power q = p^e = 3 (mod 4),
 * e <= 3; H_n = P_m (x) S_{2^k} (Kronecker; index i = i_m * 2^k + i_2), S the
 * Sylvester matrix (entry (-1)^popcount(i & j)) and P Paley's first
 * construction I + [[0, 1^T], [-1, Q]] with Q[a][b] = chi(a - b) over GF(q),
 * field elements being the base-p digit vectors of their indices taken as
 * polynomials modulo the first monic irreducible polynomial of degree e
 * (coefficient vectors counted with the constant term fastest), chi the
 * quadratic character.  Examples: 4096 = 2^12; 11008 = 2^5 * 344 (q = 7^3);
 * 28672 = 2^10 * 28 (q = 3^3).  Computed in fp32, rounded once to y_dtype.
 *   n        1..32768 with such a factorisation (UNISVQ_EUNSUP otherwise)
 *   M        1..65535 rows
 *   x        device [M][n], x_dtype F16, BF16 or F32 (aligned to its element)
 *   signs    device int8 [n], each +1 or -1
 *   y        device [M][n], y_dtype F16, BF16 or F32; must not overlap x */
int unisvq_rht(int64_t n, int64_t M, const void* x, int x_dtype, const int8_t* signs, int mode, void* y,
               int y_dtype, void* stream);

/* The input side of a rotated layer fused into the decode-phase product
 * (Eq. 5): y_i = ((x_i diag(signs_i)) H_K / sqrt(K)) W_rot,i^T for each
 * problem of the batch, with the transformed activations computed inside the
 * product's own launch (each workgroup transforms the rows in LDS while its
 * first weight packets are in flight) instead of by a separate unisvq_rht
 * call.  The transform follows unisvq_rht mode 0 with y_dtype = x_dtype and
 * the same arithmetic, so the result equals unisvq_rht followed by
 * unisvq_gemv_batched on its output bit for bit.  The output-side transform
 * (U S_U) stays a separate unisvq_rht mode 1 call: it needs all N outputs.
 *   problems  as unisvq_gemv_batched: packed format v1 weights (per (row,
 *             group) pairs), x in the original basis; every K the same, 4096
 *             or 8192 (UNISVQ_EUNSUP otherwise)
 *   signs     HOST array of `count` device pointers, signs[i] = int8 [K] (+-1),
 *             the input-side signs S_V of problem i
 *   M         1..4; x_dtype F16 or BF16 (x' is rounded to it); y_dtype as
 *             unisvq_gemv */
int unisvq_gemv_rht_batched(const unisvq_gemv_problem* problems, int count, int64_t M, int x_dtype, int y_dtype,
                            const int8_t* const* signs, void* stream);

/* ---- Bandwidth reference (not part of the method) ----
 * A plain read of `count` device byte ranges in one launch, with the 16-byte
 * non-temporal loads the decode kernels stream their weights with (8 KB per
 * workgroup of 128 threads; a thread issues all four of its loads before
 * using any).  Timed over the buffers of a product launch it gives the read
 * rate those bytes reach in the same launch structure.
 *   ranges      HOST array of 1..UNISVQ_MAX_BATCH descriptors, read before
 *               the call returns; each ptr device, 16-byte aligned, bytes a
 *               multiple of 16 in [0, 2^31) (UNISVQ_EINVAL otherwise)
 *   store       0: nothing is written (sink may be NULL) -- the pure read;
 *               1: each wavefront stores the XOR of the 32-bit words it read
 *               to its own sink word, so the XOR of all sink words equals the
 *               XOR of all words of the ranges (checkable on the host; the
 *               stores, about 4 bytes per KB read, are of the order of a
 *               product's output)
 *   sink        device uint32 [sink_words], 4-byte aligned; overwritten
 *   sink_words  >= unisvq_read_sink_words(ranges, count) when store = 1 (2
 *               words per 8 KB of each range, rounded up), else
 *               UNISVQ_EWORKSPACE */
typedef struct {
    const void* ptr;
    int64_t bytes;
} unisvq_byte_range;

int64_t unisvq_read_sink_words(const unisvq_byte_range* ranges, int count);
int unisvq_read_bytes(const unisvq_byte_range* ranges, int count, int store, uint32_t* sink, int64_t sink_words,
                      void* stream);

#ifdef __cplusplus
}
#endif

#endif /* UNISVQ_H */
