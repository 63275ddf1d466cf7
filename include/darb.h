/*
 * darb.h -- C ABI of the MI355X (gfx950) DARB library.
 *
 * DARB (density-adaptive regular-block pruning, Ren et al., AAAI-20) stores a
 * pruned weight matrix W [M x N] as follows (section 3.2):
 *   - every row r has a power-of-two block size b_r chosen from its irregular-
 *     pruning row density;
 *   - the row is split into ceil(N / b_r) blocks of b_r columns (the last one
 *     may be shorter);
 *   - each block keeps exactly one weight, its largest-magnitude element
 *     (block-max weight masking, section 3.1), together with that element's
 *     position inside the block (a log2(b_r)-bit index, held either in one
 *     byte or bit-packed, see darb_pack_offsets).
 *
 * Storage order ("grouped layout"): rows are grouped by block size, smallest
 * block size first, rows of one group in ascending original index, and the
 * blocks of a row in ascending order.  Row r's retained weights are
 * values[row_start[r] + k], k < ceil(N / b_r); its block k covers columns
 * [k*b_r, k*b_r + b_r) and keeps column k*b_r + offsets[row_start[r] + k].
 * Grouping by block size follows the paper's remark that power-of-two density
 * groups make the storage regular: every group is one dense 2-D array.
 *
 * Conventions for every call:
 *   - Return value 0 on success, a negative DARB_E_* code otherwise; on error
 *     no output is written and darb_last_error() returns a detail string
 *     (thread-local).  No C++ exception crosses this boundary.
 *   - "device" pointers are HIP device memory of the current device (for
 *     example a torch CUDA tensor's data_ptr()); "host" pointers are ordinary
 *     host memory.  All buffers are owned by the caller; the library never
 *     allocates device memory.
 *   - stream is a hipStream_t (NULL = the null stream).  Device calls only
 *     enqueue work on it and return; the caller synchronises before reading
 *     outputs.  Calls on different streams that write the same buffers race.
 *   - A plan is host memory created by darb_plan_create and released by
 *     darb_plan_destroy.  One plan may be used from several threads for device
 *     calls once uploaded; create/upload/destroy are not thread-safe.
 *   - Sizes: 1 <= M < 2^31, 1 <= N <= 2^31 - 256 (a plan's products form column
 *     indices in 32 bits); block sizes are powers of two in [1, 128].
 */
#ifndef DARB_H
#define DARB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DARB_OK 0
#define DARB_E_INVALID (-1)      /* null pointer, bad size, bad bound, bad density, bad stride */
#define DARB_E_DTYPE (-2)        /* dtype or dtype combination not supported */
#define DARB_E_NOT_UPLOADED (-3) /* device call on a plan without device metadata */
#define DARB_E_HIP (-4)          /* a HIP runtime call or kernel launch failed */
#define DARB_E_NOMEM (-5)        /* host allocation failed */
#define DARB_E_WORKSPACE (-6)    /* workspace too small */

typedef enum { DARB_F32 = 0, DARB_F16 = 1 } darb_dtype;

/* Rounding of a row density to a power-of-two fraction (section 3.2). */
typedef enum {
    /* always round the density up: b_r = largest power of two with b_r * d_r <= 1 */
    DARB_ROUND_FLOOR = 0,
    /* the paper's rule: round up when d_r >= D (the matrix density), down when d_r < D */
    DARB_ROUND_PAPER = 1
} darb_round;

typedef struct darb_plan darb_plan;

/* One block-size group of the grouped layout. */
typedef struct {
    int32_t log2b;      /* block size is 1 << log2b                       */
    int32_t reserved;
    int64_t first_row;  /* index in storage order of the group's first row */
    int64_t rows;       /* rows in the group                               */
    int64_t first_elem; /* slot of the group's first retained weight       */
    int64_t nblk;       /* retained weights per row = ceil(N / b)          */
    int64_t first_word; /* packed offsets: the group's first 32-bit word   */
} darb_bin;

typedef struct {
    int64_t M, N;
    int64_t nnz;             /* retained weights = sum_r ceil(N / b_r)    */
    int64_t workspace_bytes; /* device workspace darb_plan_upload needs   */
    int64_t packed_words;    /* uint32 words of the bit-packed offsets    */
    int32_t nbins;           /* non-empty block-size groups, <= 8         */
    int32_t reserved;
    darb_bin bins[8];        /* ascending block size                      */
} darb_plan_info_t;

/*
 * Block sizes and layout from row densities (section 3.2).
 *   row_density  host fp64 [M], each in [0, 1]: the fraction of row r that
 *                irregular magnitude pruning keeps (section 3.1 obtains it from
 *                the irregular mask without pruning for real).
 *   matrix_density  D in [0, 1], the whole matrix's kept fraction; used by
 *                DARB_ROUND_PAPER only (a row with d_r == D rounds up).
 *   round_mode   a darb_round value.
 *   b_min, b_max powers of two, 1 <= b_min <= b_max <= 128; the block size is
 *                clamped to [b_min, b_max].  A row of density 0 gets b_max.
 *   out          receives the new plan (host memory), or NULL on error.
 * 1 <= M < 2^31, 1 <= N <= 2^31 - 256, and the plan may hold at most 2^55
 * retained weights.
 * Errors: DARB_E_INVALID, DARB_E_NOMEM.
 */
int darb_plan_create(int64_t M, int64_t N, const double *row_density, double matrix_density,
                     int round_mode, int b_min, int b_max, darb_plan **out);

/*
 * darb_plan_create from kept counts: row_density[r] = row_count[r] / N and
 * matrix_density = kept / (M * N), as produced by darb_prune_counts.
 *   row_count  host int64 [M], each in [0, N];  kept in [0, M * N]
 * Errors: DARB_E_INVALID, DARB_E_NOMEM.
 */
int darb_plan_create_counts(int64_t M, int64_t N, const int64_t *row_count, int64_t kept,
                            int round_mode, int b_min, int b_max, darb_plan **out);

/*
 * The plan built on the device, from kept counts in device memory (the flow of
 * section 3.2 from the irregular mask to block sizes, with darb_prune_counts' output
 * left where it is).  The same block-size rule as darb_plan_create_counts, in both
 * rounding modes and with the same results; the storage order and the per-row table
 * are written straight into `workspace`, which becomes the plan's device workspace
 * (the plan comes back uploaded on the current device; darb_plan_upload is refused
 * for it).  Only the group sizes (32 int64) travel to the host, so the call waits for
 * `stream`.  darb_plan_export copies the tables back from the device.
 *   row_count  device int64 [M], 8-byte aligned, each in [0, N] (as darb_prune_counts
 *              writes them; larger values count as N, negative ones as 0)
 *   kept       the matrix's kept count k, in [0, M * N] (D = k / (M N))
 *   workspace  device, 256-byte aligned, >= darb_plan_device_workspace(M) bytes; it must
 *              stay allocated and unmodified while the plan is used
 * Other arguments as for darb_plan_create.
 * Errors: DARB_E_INVALID, DARB_E_WORKSPACE, DARB_E_NOMEM, DARB_E_HIP.
 */
int darb_plan_device_workspace(int64_t M, int64_t *bytes);
int darb_plan_create_device(int64_t M, int64_t N, const int64_t *row_count, int64_t kept,
                            int round_mode, int b_min, int b_max, void *workspace,
                            int64_t workspace_bytes, void *stream, darb_plan **out);

/* Sizes and groups of a plan.  Errors: DARB_E_INVALID (null pointer). */
int darb_plan_info(const darb_plan *plan, darb_plan_info_t *info);

/*
 * Copy the plan's host metadata out.  Any output may be NULL to skip it.
 *   log2b      host uint8 [M]: log2 of each original row's block size
 *   row_start  host int64 [M]: first slot of each original row
 *   perm       host int32 [M]: original index of the row stored i-th
 */
int darb_plan_export(const darb_plan *plan, uint8_t *log2b, int64_t *row_start, int32_t *perm);

/*
 * Copy the plan's device metadata (the storage order and a per-row table of
 * first slot and block size) into a caller-owned device workspace of at least
 * info.workspace_bytes bytes (256-byte aligned) on `stream`, wait for the copy
 * to finish, and remember the workspace for later device calls on the current
 * device.  The workspace must stay allocated and unmodified while the plan is
 * used on the device.  Re-uploading to another workspace is allowed.
 * Errors: DARB_E_INVALID, DARB_E_WORKSPACE, DARB_E_NOMEM, DARB_E_HIP.
 */
int darb_plan_upload(darb_plan *plan, void *workspace, int64_t workspace_bytes, void *stream);

/* Release a plan (NULL is ignored).  Does not touch the device workspace. */
void darb_plan_destroy(darb_plan *plan);

/*
 * BMWM encode (section 3.1, with section 3.2's per-row block size): for every
 * row and block keep the element whose magnitude is largest -- magnitude is the
 * stored bit pattern with the sign bit cleared, compared as an unsigned
 * integer, so equal magnitudes (including +0 / -0) go to the lowest column --
 * and write its bits and its in-block index.
 *   wdtype   DARB_F32 or DARB_F16
 *   W        device [M x ldw] row-major, ldw >= N (elements)
 *   values   device [nnz] of wdtype, grouped layout
 *   offsets  device uint8 [nnz], grouped layout
 * Errors: DARB_E_INVALID, DARB_E_DTYPE, DARB_E_NOT_UPLOADED, DARB_E_HIP.
 */
int darb_encode(const darb_plan *plan, int wdtype, const void *W, int64_t ldw, void *values,
                uint8_t *offsets, void *stream);

/*
 * Decode to the masked dense matrix: W_out[r, c] = the retained value if c is
 * row r's kept column of its block, +0.0 otherwise.  Every element of the
 * [M x N] region is written.  Used to check the format against dense products.
 *   W_out    device [M x ldw] of wdtype, ldw >= N
 * Errors: DARB_E_INVALID, DARB_E_DTYPE, DARB_E_NOT_UPLOADED, DARB_E_HIP.
 */
int darb_decode(const darb_plan *plan, int wdtype, const void *values, const uint8_t *offsets,
                void *W_out, int64_t ldw, void *stream);

/*
 * y = W_darb x (sections 2 and 3.2: only retained weights are read, each
 * block's offset selects the one activation it multiplies).  Products and
 * sums in fp32; y is overwritten.
 *   (wdtype, xdtype) in {(F32, F32), (F16, F16), (F16, F32)}
 *   x  device [N] of xdtype;  y  device fp32 [M], original row order
 * Errors: DARB_E_INVALID, DARB_E_DTYPE, DARB_E_NOT_UPLOADED, DARB_E_HIP.
 */
int darb_spmv(const darb_plan *plan, int wdtype, const void *values, const uint8_t *offsets,
              int xdtype, const void *x, float *y, void *stream);

/*
 * Y = W_darb X for a batch of B activation vectors (same definition as
 * darb_spmv, column by column).  X is [N x B] row-major with leading dimension
 * ldx >= B (the B values of one input feature are contiguous); Y is fp32
 * [M x B] row-major with ldy >= B, overwritten.  B >= 1.
 * Errors: DARB_E_INVALID, DARB_E_DTYPE, DARB_E_NOT_UPLOADED, DARB_E_HIP.
 */
int darb_spmm(const darb_plan *plan, int wdtype, const void *values, const uint8_t *offsets,
              int xdtype, int64_t B, const void *X, int64_t ldx, float *Y, int64_t ldy,
              void *stream);

/*
 * Bit-packed offsets (section 4.2: the kept weight's position inside a block of
 * size b needs log2 b bits, not a byte).  Layout: inside each block-size group
 * (log2 b = l) the retained weights are numbered j = 0, 1, ... in storage order
 * and cut into runs of 32; run j / 32 occupies l consecutive uint32 words, and
 * weight j's index is bits (j % 32) * l ... (j % 32) * l + l - 1 of its run read
 * as one little-endian bit string (bit i of the run is bit i % 32 of word i / 32).
 * Groups follow each other in ascending block size starting at word
 * bins[g].first_word; a group with b = 1 has no words (every index is 0).  The
 * whole form is info.packed_words words, which may be 0 (then `packed` may be
 * NULL).  `packed` is device memory, 4-byte aligned.
 *
 * darb_pack_offsets converts the byte offsets darb_encode writes (every one must
 * be < b; only its low log2 b bits are stored) to the packed form, overwriting
 * every packed word; darb_unpack_offsets converts back, writing all nnz bytes.
 * Errors: DARB_E_INVALID, DARB_E_NOT_UPLOADED, DARB_E_HIP.
 */
int darb_pack_offsets(const darb_plan *plan, const uint8_t *offsets, uint32_t *packed,
                      void *stream);
int darb_unpack_offsets(const darb_plan *plan, const uint32_t *packed, uint8_t *offsets,
                        void *stream);

/*
 * darb_spmv and darb_spmm reading the offsets in the packed form above.  Every
 * other argument, and the result bit for bit, is as for the byte-offset calls.
 * Errors: DARB_E_INVALID, DARB_E_DTYPE, DARB_E_NOT_UPLOADED, DARB_E_HIP.
 */
int darb_spmv_packed(const darb_plan *plan, int wdtype, const void *values,
                     const uint32_t *packed, int xdtype, const void *x, float *y, void *stream);
int darb_spmm_packed(const darb_plan *plan, int wdtype, const void *values,
                     const uint32_t *packed, int xdtype, int64_t B, const void *X, int64_t ldx,
                     float *Y, int64_t ldy, void *stream);

/*
 * INT8 retained weights.  Section 4.2's storage accounting assumes weights
 * quantised to INT8 without fixing a scheme; this one is symmetric with one fp32
 * scale per row.  For row r with a = max |v| over its retained values (fp32, fp16
 * widened exactly): inv = 127 / a, code q = rint(v * inv) (ties to even) clamped to
 * [-127, 127], scale s_r = a / 127 -- each a single correctly rounded fp32
 * operation, so the codes are exact.  Rows with a < 2^-120 (127 / a would
 * overflow) get s_r = 0 and all-zero codes.  Values must be finite.
 *   darb_quantize_i8
 *     values   device, the format's values (wdtype DARB_F32 or DARB_F16), nnz
 *     codes    device int8 [nnz], slot order like values, overwritten
 *     scales   device fp32 [M], indexed by original row, overwritten
 *   darb_spmv_i8 / darb_spmm_i8: y[r] = s_r * sum_k q[r,k] * x[k * b_r + off[r,k]],
 *     summed in fp32 and scaled once; as darb_spmv / darb_spmm (same layouts, x/X
 *     fp32 or fp16, Y fp32) with the offsets from exactly one of `offsets` (one byte
 *     each) and `packed` (darb_pack_offsets' words; with offsets NULL, packed may be
 *     NULL only when the plan has no packed words).  Passing both is an error.
 * Errors: DARB_E_INVALID, DARB_E_DTYPE, DARB_E_NOT_UPLOADED, DARB_E_HIP.
 */
int darb_quantize_i8(const darb_plan *plan, int wdtype, const void *values, int8_t *codes,
                     float *scales, void *stream);
int darb_spmv_i8(const darb_plan *plan, const int8_t *codes, const float *scales,
                 const uint8_t *offsets, const uint32_t *packed, int xdtype, const void *x,
                 float *y, void *stream);
int darb_spmm_i8(const darb_plan *plan, const int8_t *codes, const float *scales,
                 const uint8_t *offsets, const uint32_t *packed, int xdtype, int64_t B,
                 const void *X, int64_t ldx, float *Y, int64_t ldy, void *stream);

/*
 * Irregular magnitude pruning, the step DARB starts from (section 3.2: the
 * irregular mask is computed only to measure each row's density; irregular
 * pruning keeps the K largest-magnitude weights, section 2).  Keeps the k
 * elements of W with the largest magnitude -- the stored bits with the sign
 * cleared, compared as unsigned integers, as in darb_encode; among equal
 * magnitudes the lower flat index r * N + c first -- and writes how many each
 * row keeps.  No mask is materialised.
 *   wdtype     DARB_F32 or DARB_F16
 *   W          device [M x ldw] row-major, ldw >= N (elements)
 *   k          0 <= k <= M * N
 *   counts     device int64 [M], 8-byte aligned, overwritten
 *   workspace  device, 256-byte aligned, >= the size darb_prune_workspace
 *              returns (about M*N/4 bytes: room for the keys whose leading digit
 *              lies in a small bracket around the threshold's, which the later
 *              passes read instead of W when W has 64 MiB or more); its contents
 *              on entry do not change the counts (a workspace last used by this
 *              call runs fastest: it leaves the part the next call's sample adds
 *              into at zero; other contents may cost that call passes over W)
 * Work is enqueued on `stream` only (several kernels, no host synchronisation);
 * calls sharing a workspace must not overlap.
 * Errors: DARB_E_INVALID, DARB_E_DTYPE, DARB_E_WORKSPACE, DARB_E_HIP.
 */
int darb_prune_workspace(int64_t M, int64_t N, int wdtype, int64_t *bytes);
int darb_prune_counts(int64_t M, int64_t N, int wdtype, const void *W, int64_t ldw, int64_t k,
                      int64_t *counts, void *workspace, int64_t workspace_bytes, void *stream);

/*
 * darb_prune_counts for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the same
 * arguments and the same counts, bit for bit, without the workspace.  Its scratch
 * is a fixed 8 MiB array in the library's device code, one per device, held until
 * the process ends; the first call on a device looks up that device's copy (no
 * allocation).  The array holds the per-row counters (16 bytes per row), so M is
 * limited to 483 296 rows (larger M: DARB_E_INVALID, naming the limit);
 * the rest is candidate room, and a matrix whose candidates do not fit takes more
 * passes over W with the same result.  Every call on a device shares its array and
 * leaves its contents there (each call clears what must start at zero), so calls
 * that overlap on one device -- on different streams or threads -- race.
 * Errors: DARB_E_INVALID, DARB_E_DTYPE, DARB_E_HIP.
 */
int darb_prune_counts_noalloc(int64_t M, int64_t N, int wdtype, const void *W, int64_t ldw,
                              int64_t k, int64_t *counts, void *stream);

/*
 * One LSTM layer over a sequence with DARB-stored weights (the recurrent
 * models of section 4.1): no bias, gate order (i, f, g, o),
 *   gates_t = W_ih x_t + W_hh h_{t-1},
 *   c_t = sigmoid(f) * c_{t-1} + sigmoid(i) * tanh(g),  h_t = sigmoid(o) * tanh(c_t).
 * W_ih is [4H x I] and W_hh is [4H x H], both of wdtype, each with its own
 * uploaded plan.  The input products of all steps are computed first as one
 * darb_spmm with B = T * batch.  Each time step is then one launch: a workgroup per
 * hidden unit computes the unit's four gate rows of W_hh h_{t-1} and the cell
 * (batch <= 64 and a multiple of 4, or batch <= 16; W_hh rows of at most 512
 * retained weights); other shapes run
 * the recurrent product and the cell as two launches.  Both give the same result
 * within the product tolerance; the call is deterministic.  The workspace also
 * holds the second buffer of h that the steps alternate with `h`.
 *   x_seq      device fp32 [I x T*batch], column t*batch + n
 *   h_seq      device fp32 [H x T*batch], receives h_t in columns t*batch + n
 *   h, c       device fp32 [H x batch], initial state in, final state out
 *   workspace  device fp32, 16-byte aligned, at least 4H*T*batch + 4H*batch floats
 *              (darb_lstm_workspace)
 * Errors: DARB_E_INVALID, DARB_E_DTYPE, DARB_E_NOT_UPLOADED, DARB_E_HIP.
 */
int darb_lstm_layer(const darb_plan *wih_plan, const void *wih_values,
                    const uint8_t *wih_offsets, const darb_plan *whh_plan,
                    const void *whh_values, const uint8_t *whh_offsets, int wdtype,
                    int64_t H, int64_t T, int64_t batch, const float *x_seq, float *h_seq,
                    float *h, float *c, float *workspace, int64_t workspace_floats,
                    void *stream);

/* Workspace floats darb_lstm_layer needs for (H, T, batch).  Errors: DARB_E_INVALID. */
int darb_lstm_workspace(int64_t H, int64_t T, int64_t batch, int64_t *floats);

/*
 * Measurement helpers (not part of DARB).  darb_stream_read reads `bytes`
 * bytes (a multiple of 16, 16-byte aligned) of device memory and writes one
 * float per workgroup derived from them into `sink` (device, >= 8192 floats)
 * so the reads cannot be elided; darb_stream_copy copies `bytes` bytes
 * (multiple of 16, both 16-byte aligned).  They give the HBM read and copy
 * rates the DARB kernels are compared with.
 */
int darb_stream_read(const void *buf, int64_t bytes, float *sink, void *stream);
/*
 * The same read in other launch shapes, to find the fastest plain read of a given
 * size: `threads` per workgroup (64, 128, 256, 512 or 1024) each issuing `vectors`
 * 16-byte loads (1, 2, 4 or 8; the pairs 64/1, 64/2, 128/1, 128/2, 128/8, 512/8
 * and 1024/8 are not built) before using any of them.  The loaded data decides
 * whether anything is written to `sink` (device, >= 8192 floats); real data never
 * produces the value that would, so the launch is the read alone.
 * Errors: DARB_E_INVALID (also for a shape that is not built), DARB_E_HIP.
 */
int darb_stream_read_shape(const void *buf, int64_t bytes, int threads, int vectors, float *sink,
                           void *stream);
int darb_stream_copy(void *dst, const void *src, int64_t bytes, void *stream);

/* Text for a DARB_E_* code (static storage). */
const char *darb_strerror(int code);

/* Detail of the last error on the calling thread ("" if none). */
const char *darb_last_error(void);

/* Library version as major*10000 + minor*100 + patch. */
int darb_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DARB_H */
