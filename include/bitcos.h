/*
 * bitcos.h -- C ABI of libbitcos: ternary GEMV over the BITCOS layout on MI355X (gfx950).
 *
 * BITCOS (paper "Breaking the 1.58-bit Barrier for Ternary LLMs", Sec. II-A)
 * stores a ternary matrix W in {-1, 0, +1}^{N x K} as
 *   - a presence bitmap with one bit per weight, set where the weight is
 *     non-zero, and
 *   - a sign vector with one bit per NON-ZERO weight, in the same tensor order
 *     (the j-th sign bit belongs to the j-th set bit of the bitmap; a set sign
 *     bit means -1, Sec. II-D Eq. (4)),
 * which costs 2 - z bits per weight at zero density z (Eq. (1)).  Beside the
 * two streams the blob carries non-negative fp16 scales (one per 128 weights
 * along K, or one per tensor) and 32-bit sign offsets, one per "unit" of
 * rows, telling where each unit enters the sign stream (the paper leaves the
 * storage of stream entry points open, Sec. II-D; these offsets are metadata
 * outside the 2 - z payload).
 *
 * The GEMV computes y = (S (.) W) x for one activation row (batch 1 decode):
 *   y[n] = sum_g S[n, g] * a[g] * sum_{k in group g} W[n, k] * x[k]
 * with int8 activations accumulated exactly in int32 and the group scale
 * applied once per group (Sec. II-C), or bf16 activations accumulated in
 * fp32.  Two same-GPU baselines use fixed-rate layouts: five trits per byte,
 * 26 bytes per 128 weights (Sec. I), and 2 bits per weight (Table I).
 *
 * Layouts (all little-endian; every section starts at a 256-byte boundary
 * of the blob and the blob length is a multiple of 256 bytes):
 *   BITCOS  section 0  bitmap   u32[N*K/32]; bit b of word w is weight
 *                               32w + b of W in row-major (n, k) order.
 *           section 1  signs    u32[ceil(nnz/32)] LSB-first sign stream,
 *                               then 16 zero bytes (the GEMV may read them).
 *           section 2  offsets  u32[ceil(N/unit_rows) + 1]; entry u is the
 *                               number of non-zeros in rows
 *                               [0, u*unit_rows); the last entry is nnz.
 *           section 3  scales   fp16[N][K/128] (group 128) or fp16[1].
 *   TRIT5   section 0  codes    26-byte blocks, row-major [N][K/128]; byte j
 *                               of a block holds weights 5j..5j+4 of the
 *                               block as sum_t (w+1) * 3^t (a missing weight
 *                               past 127 is the digit 1), then 16 zero bytes.
 *           section 3  scales   as BITCOS.
 *   BIT2    section 0  codes    u32 per 16 weights, row-major; weight
 *                               k0 + 4t + b (k0 = 16 * word) has the code
 *                               w + 1 at bits [8b + 2t, 8b + 2t + 1].
 *           section 3  scales   as BITCOS.
 *
 * Conventions for every function:
 *   - Return BITCOS_OK (0) or a negative status; nothing aborts or prints.
 *     bitcos_strerror() names a status.  All validation happens before any
 *     device work is enqueued.
 *   - The caller owns every host and device buffer and the stream; the
 *     library allocates nothing on the device, keeps no mutable global state
 *     and is safe to call from several threads.  The one exception is the
 *     fixed per-GPU workspace of bitcos_pack_device_noalloc (see there).
 *   - Device pointers are plain device addresses (e.g. a torch tensor's
 *     data_ptr()); `stream` is a hipStream_t passed as void* (NULL = the
 *     default stream).  GEMV calls are asynchronous and never synchronise.
 *   - Host pointers are ordinary host memory.
 */
#ifndef BITCOS_H
#define BITCOS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
#define BITCOS_OK 0
#define BITCOS_E_ARG (-1)          /* null pointer, bad size/shape/enum      */
#define BITCOS_E_VALUE (-2)        /* weight outside {-1,0,1}, bad scale, corrupt blob */
#define BITCOS_E_SPACE (-3)        /* destination capacity too small          */
#define BITCOS_E_HIP (-4)          /* HIP launch/runtime error                */
#define BITCOS_E_UNSUPPORTED (-5)  /* shape/dtype/batch without a kernel      */

/* ---- enums ------------------------------------------------------------- */
#define BITCOS_LAYOUT_VERSION 1u

#define BITCOS_FMT_BITCOS 1
#define BITCOS_FMT_TRIT5 2
#define BITCOS_FMT_BIT2 3

#define BITCOS_SEC_BITMAP 0   /* BITCOS */
#define BITCOS_SEC_SIGNS 1    /* BITCOS */
#define BITCOS_SEC_OFFSETS 2  /* BITCOS */
#define BITCOS_SEC_CODES 0    /* TRIT5, BIT2 */
#define BITCOS_SEC_SCALES 3   /* all formats */

#define BITCOS_X_I8 1         /* activations int8 [m][K]                 */
#define BITCOS_X_BF16 2       /* activations bfloat16 bit patterns [m][K] */

#define BITCOS_MAX_M 16        /* most activation rows per GEMV call      */

#define BITCOS_Y_F32 1        /* y float32 [m][N], scaled                 */
#define BITCOS_Y_I32_RAW 2    /* y int32 [m][N] = sum_k W x, unscaled (int8 x only) */
/* Accumulating forms of the two: the result is added onto what y already
 * holds (y += ...), e.g. to sum the partial products of a matrix stored as
 * column blocks (a split of K: block c holds columns [c Kc, (c+1) Kc) as a
 * matrix of its own).  Every output element is added once per call, so calls
 * that follow one another on a stream add in that order (deterministic). */
#define BITCOS_Y_F32_ADD 3
#define BITCOS_Y_I32_RAW_ADD 4

/* Plain-old-data description of one packed matrix.  Filled by *_plan();
 * passed by pointer to pack/unpack/gemv.  Section offsets are relative to the
 * blob start. */
typedef struct bitcos_layout {
  uint32_t version;        /* BITCOS_LAYOUT_VERSION                           */
  uint32_t format;         /* BITCOS_FMT_*                                    */
  int32_t n;               /* output rows N (>= 1)                            */
  int32_t k;               /* reduction length K                              */
  int32_t group;           /* 128: one scale per 128 weights of a row; 0: one per tensor */
  int32_t unit_rows;       /* BITCOS: rows per sign-offset entry; 0 otherwise */
  uint64_t nnz;            /* number of non-zero weights                     */
  uint64_t sec_off[4];     /* byte offset of each section (0 if unused)      */
  uint64_t sec_bytes[4];   /* byte length of each section (0 if unused)      */
  uint64_t total_bytes;    /* blob length (multiple of 256)                  */
  uint64_t payload_bits;   /* format symbols + 16-bit scales, no metadata    */
} bitcos_layout;

/* Name of a status code (static string; never NULL). */
const char* bitcos_strerror(int status);

/* BITCOS_LAYOUT_VERSION of the library. */
uint32_t bitcos_version(void);

/* ---- BITCOS -------------------------------------------------------------
 * bitcos_plan: validate W (host int8 [n][k], row-major, values in {-1,0,1})
 * and fill *out.  group is 128 (k % 128 == 0) or 0 (one scale per tensor,
 * k % 32 == 0).  unit_rows >= 1 sets the rows per sign offset; 0 picks the
 * library default (1: one offset per row, which every kernel can use).  Errors: E_ARG,
 * E_VALUE (a weight outside {-1,0,1}).  Paper: Sec. II-A. */
int bitcos_plan(const int8_t* w, int32_t n, int32_t k, int32_t group, int32_t unit_rows,
                bitcos_layout* out);

/* bitcos_pack: write the whole blob for W and its scales (host fp16 bit
 * patterns, [n][k/128] or [1]; finite and non-negative) into host memory
 * dst of `cap` bytes (>= L->total_bytes).  Bytes are a deterministic
 * function of (W, scales, *L); padding is zero.  Errors: E_ARG, E_VALUE
 * (bad weight or scale, W not the one planned), E_SPACE.  Paper: Sec. II-A
 * (a presence bit per weight, a sign bit per non-zero in the same row-major
 * order, 2 - z bits per weight by Eq. (1)); the fp16 scale per 128-weight
 * group is the deployed models' convention of Sec. I and Table I. */
int bitcos_pack(const int8_t* w, const uint16_t* scales_f16, const bitcos_layout* L, void* dst,
                size_t cap);

/* bitcos_unpack: exact inverse of bitcos_pack on a host blob of
 * `blob_bytes` bytes: writes W (host int8 [n][k]) and the scales (host
 * fp16 bits).  Verifies the bitmap popcount against nnz and every unit
 * offset; E_VALUE on a mismatch.  Paper: Sec. II-A and Fig. 1 (the j-th
 * stored sign belongs to the j-th set bit of the bitmap); the weight is
 * w = p - 2n of Eq. (2), Sec. II-C. */
int bitcos_unpack(const bitcos_layout* L, const void* blob, size_t blob_bytes, int8_t* w_out,
                  uint16_t* scales_out);

/* bitcos_gemv: y = (S (.) W) x on the device, enqueued on `stream`.
 *   blob_dev  device copy of the packed blob (L->total_bytes bytes).
 *   m         number of activation rows, 1..BITCOS_MAX_M.  m = 1 is batch-1
 *             decode.  2 <= m <= 16 runs the small-batch kernel (every
 *             decoded weight multiplied against all m rows on the matrix
 *             cores) when the layout has one sign offset per row and
 *             k % 128 == 0; other layouts run m batch-1 launches.  At m = 1
 *             rows longer than the batch-1 kernels take (bf16 k > 16384,
 *             int8 k > 32768) run the small-batch kernel too, with such
 *             layouts; others return E_UNSUPPORTED.
 *   x_dev     device activations [m][k]: int8 (BITCOS_X_I8) or bf16 bits
 *             (BITCOS_X_BF16), row-major.
 *   xscale_dev  NULL (a = 1) or device fp32 [m][k/128] per-group activation
 *             scales a (int8 activations quantised per group of 128).
 *   y_dev     device output [m][n], overwritten: fp32 (BITCOS_Y_F32) or the
 *             unscaled int32 row sums (BITCOS_Y_I32_RAW, int8 x only, exact);
 *             or added onto (BITCOS_Y_F32_ADD, BITCOS_Y_I32_RAW_ADD).
 * int8 x accumulates exactly in int32 per group and applies the scale once per
 * group in fp32; with one scale per tensor and no xscale the full int32 row
 * sum is multiplied once.  bf16 x accumulates in fp32.
 * Errors: E_ARG (also m outside 1..BITCOS_MAX_M), E_UNSUPPORTED (dtype or
 * shape without a kernel), E_HIP.  Paper: Sec. II-C (ternary weights
 * w = p - 2n, Eq. (2), contracted against int8 activations into int32 with
 * the group scale applied once per group) and Sec. II-B / II-D (the same
 * contraction with floating-point activations); the GEMV of a decode step,
 * Sec. III. */
int bitcos_gemv(const bitcos_layout* L, const void* blob_dev, int32_t m, const void* x_dev,
                int32_t x_dtype, const float* xscale_dev, void* y_dev, int32_t y_mode,
                void* stream);

/* ---- five-trit baseline (26 B per 128 weights; Sec. I) -------------------
 * Same conventions as the BITCOS functions; k % 128 == 0 always (the block is
 * 128 weights whatever the scale group). */
int trit5_plan(const int8_t* w, int32_t n, int32_t k, int32_t group, bitcos_layout* out);
int trit5_pack(const int8_t* w, const uint16_t* scales_f16, const bitcos_layout* L, void* dst,
               size_t cap);
int trit5_unpack(const bitcos_layout* L, const void* blob, size_t blob_bytes, int8_t* w_out,
                 uint16_t* scales_out);
int trit5_gemv(const bitcos_layout* L, const void* blob_dev, int32_t m, const void* x_dev,
               int32_t x_dtype, const float* xscale_dev, void* y_dev, int32_t y_mode,
               void* stream);

/* ---- 2-bit baseline (2 bits per weight; Table I) ------------------------ */
int bit2_plan(const int8_t* w, int32_t n, int32_t k, int32_t group, bitcos_layout* out);
int bit2_pack(const int8_t* w, const uint16_t* scales_f16, const bitcos_layout* L, void* dst,
              size_t cap);
int bit2_unpack(const bitcos_layout* L, const void* blob, size_t blob_bytes, int8_t* w_out,
                uint16_t* scales_out);
int bit2_gemv(const bitcos_layout* L, const void* blob_dev, int32_t m, const void* x_dev,
              int32_t x_dtype, const float* xscale_dev, void* y_dev, int32_t y_mode,
              void* stream);

/* ---- batched GEMVs (one persistent launch for a list of matrices) -------
 * A decode step runs many GEMVs; launching each on its own leaves the GPU
 * idle between small kernels.  A batch runs a list of GEMVs of ONE format and
 * ONE tile (bitcos_describe reports per_lane and seg_lanes) as a single
 * persistent launch: every wave takes a contiguous range of the list's work
 * units.  Each GEMV keeps the single-call semantics above (its own x, xscale
 * and y; y overwritten), with the same number m of activation rows.
 *
 * bitcos_batch_bytes: bytes of a batch table for `count` GEMVs (0 if count < 1).
 *
 * bitcos_batch_build: fill a host table (table_bytes >= bitcos_batch_bytes)
 * for `count` GEMVs of m activation rows each (1..BITCOS_MAX_M): layouts[i]
 * (host), blobs_dev[i], x_dev[i] ([m][k]), y_dev[i] ([m][n]) (device
 * pointers), xscale_dev NULL or an array of per-GEMV device pointers
 * ([m][k/128]; entries may be NULL).  The table records the device pointers:
 * they must stay valid while the table is in use.  m > 1 takes BITCOS
 * layouts with one sign offset per row and k % 128 == 0 (the small-batch
 * kernel); so does m = 1 when layouts[0]'s rows are longer than the batch-1
 * tiles (bitcos_describe reports BITCOS_KERNEL_SMALL_BATCH).  Errors: E_ARG,
 * E_SPACE, E_UNSUPPORTED (mixed formats or tiles: build one batch per tile;
 * a small-batch table with another layout).
 *
 * bitcos_gemv_batch: copy of the table in device memory (16-byte aligned,
 * unchanged since built) plus the host table it was copied from; enqueues
 * one launch on `stream`.  Errors: E_ARG, E_UNSUPPORTED, E_HIP. */
size_t bitcos_batch_bytes(int32_t count);
int bitcos_batch_build(int32_t count, int32_t m, const bitcos_layout* layouts,
                       const void* const* blobs_dev,
                       const void* const* x_dev, const float* const* xscale_dev,
                       void* const* y_dev, int32_t x_dtype, int32_t y_mode, void* table,
                       size_t table_bytes);
int bitcos_gemv_batch(const void* table_host, const void* table_dev, void* stream);

/* ---- activation quantisation --------------------------------------------
 * bitcos_quantize_act: int8 activations for the int8 GEMV path, quantised per
 * group of 128 (Sec. II-C).  The paper does not state the rule; this one is
 * symmetric absmax: for every row r and group g,
 *   a[r][g] = max|x| / 127 in fp32 (1 for an all-zero group),
 *   q[r][k] = clamp(round_half_even(x / a), -127, 127), divisions IEEE fp32.
 * x_bf16_dev: device bf16 bits [m][k]; q_dev: device int8 [m][k]; scale_dev:
 * device fp32 [m][k/128] (pass it as the GEMV's xscale_dev).  k % 128 == 0.
 * Asynchronous on `stream`.  Errors: E_ARG, E_UNSUPPORTED, E_HIP. */
int bitcos_quantize_act(const void* x_bf16_dev, int32_t m, int32_t k, int8_t* q_dev,
                        float* scale_dev, void* stream);

/* ---- partial outputs of split rows --------------------------------------
 * bitcos_add_partials: y[i] += parts[0 * n + i] + parts[1 * n + i] + ... +
 * parts[(nparts - 1) * n + i] for i < n, one fp32 addition per part, left to
 * right.  For rows too long for one batch-1 tile, computed as column blocks
 * (the row sum over K of Sec. II-C taken block by block): the first block's
 * GEMV writes y (BITCOS_Y_F32), block c + 1's writes slice c of a device
 * buffer [nparts][n] (also BITCOS_Y_F32), so every block can run in one
 * launch, and this call adds the slices in block order -- the same fp32
 * additions in the same order as the accumulating mode (BITCOS_Y_F32_ADD)
 * with one launch per block.  y_dev and parts_dev are device fp32 buffers of
 * n and nparts * n elements that do not overlap; several GEMVs' outputs can
 * be summed in one call when their y and slices are laid out alike.
 * Asynchronous on `stream`; allocates nothing.  Errors: E_ARG (null pointer,
 * nparts < 1, n < 1), E_HIP. */
int bitcos_add_partials(float* y_dev, const float* parts_dev, int32_t nparts, int64_t n, void* stream);

/* ---- device-side BITCOS packer ------------------------------------------
 * The same blob bytes as bitcos_plan + bitcos_pack (Sec. II-A: presence
 * bitmap and compacted sign vector in row-major order, the unit offsets and
 * the scales), computed on the GPU from W already in device memory.  Both
 * calls enqueue on `stream` and wait for it before returning (the plan has
 * to read the non-zero count back).
 *
 * bitcos_plan_device_workspace: bytes of device workspace for an n-row
 *   matrix (0 if n < 1): a 16-byte header and n + 1 row offsets.
 *
 * bitcos_plan_device: W is device int8 [n][k], row-major; group / unit_rows
 *   as bitcos_plan (n*k < 2^31).  ws_dev: caller device memory of ws_bytes
 *   >= bitcos_plan_device_workspace(n); it receives the row offsets the pack
 *   call reuses.  Fills *out exactly as bitcos_plan would.  Errors: E_ARG,
 *   E_SPACE (workspace), E_VALUE (a weight outside {-1,0,1}), E_UNSUPPORTED
 *   (shape), E_HIP.
 *
 * bitcos_pack_device: writes the blob into dst_dev (device, cap >=
 *   L->total_bytes) from the same W, the device fp16 scales ([n][k/128] or
 *   [1], finite and non-negative) and the workspace of the plan call for this
 *   W and *L.  Errors: E_ARG (a layout this plan would not give), E_SPACE,
 *   E_VALUE (bad scale, or W differs from the planned one: then the blob is
 *   incomplete but nothing outside it is written), E_UNSUPPORTED, E_HIP. */
size_t bitcos_plan_device_workspace(int32_t n);
int bitcos_plan_device(const int8_t* w_dev, int32_t n, int32_t k, int32_t group, int32_t unit_rows,
                       void* ws_dev, size_t ws_bytes, bitcos_layout* out, void* stream);
int bitcos_pack_device(const int8_t* w_dev, const uint16_t* scales_dev, const bitcos_layout* L,
                       void* ws_dev, size_t ws_bytes, void* dst_dev, size_t cap, void* stream);

/* ---- device-side packing without allocation ------------------------------
 * For callers that cannot allocate device memory (code under graph capture
 * of its neighbours, serving loops and harnesses that forbid hipMalloc):
 * bitcos_plan_device + bitcos_pack_device in one call, with the plan's
 * workspace in a fixed array the library keeps in every GPU it runs on
 * (about 1 MiB each, held until the process ends) instead of a caller
 * buffer.  Nothing is allocated: the caller passes W, the scales and dst.
 *
 * bitcos_pack_device_noalloc: W device int8 [n][k], scales_dev device fp16
 *   ([n][k/128] or [1]), group / unit_rows as bitcos_plan; fills *out as
 *   bitcos_plan would and writes the blob into dst_dev (cap bytes) -- the
 *   same bytes as bitcos_pack.  Waits for `stream` before returning (the
 *   plan reads the non-zero count back).
 *   Errors: E_ARG, E_SPACE (n > BITCOS_NOALLOC_MAX_ROWS, checked before any
 *   device work; or cap < out->total_bytes, with *out filled so the caller
 *   can size dst and call again), E_VALUE, E_UNSUPPORTED, E_HIP.
 *   Every call on one GPU uses that GPU's one workspace: calls that overlap
 *   in time on one GPU (other threads, other streams) race and must be
 *   serialised by the caller; calls on different GPUs do not interact. */
#define BITCOS_NOALLOC_MAX_ROWS 262144
int bitcos_pack_device_noalloc(const int8_t* w_dev, const uint16_t* scales_dev, int32_t n, int32_t k,
                               int32_t group, int32_t unit_rows, bitcos_layout* out, void* dst_dev, size_t cap,
                               void* stream);

/* ---- launch description (for measurement) ---------------------------------
 * Fills the kernel configuration a GEMV on this layout would launch with,
 * for a call (or a batch of such layouts) without activation scales: words
 * (or blocks) per lane, lanes per row segment, rows per wave step, waves and
 * workgroups, and which kernel runs (BITCOS_KERNEL_*).  Errors as for the
 * GEMV. */
#define BITCOS_KERNEL_GENERAL 1     /* BITCOS, any rows per sign offset                          */
#define BITCOS_KERNEL_STREAMING 2   /* BITCOS batch 1, group scales: v_dot2 / v_dot4 multiply    */
#define BITCOS_KERNEL_MATRIX 3      /* BITCOS batch 1, one scale per tensor: multiply on MFMA    */
#define BITCOS_KERNEL_SMALL_BATCH 4 /* BITCOS, 2..16 activation rows on MFMA (and batch-1 rows   \
                                       longer than the batch-1 tiles)                             */
#define BITCOS_KERNEL_FIXED 5       /* five-trit or 2-bit                                        */
typedef struct bitcos_launch_info {
  int32_t per_lane;        /* BITCOS: 32-weight words per lane; TRIT5: 128-blocks; BIT2: 16-weight words */
  int32_t seg_lanes;       /* lanes that share one row: a power of two, or 20
                              (five-trit, rows of 20 or 40 blocks)             */
  int32_t rows_per_step;   /* rows a wave covers per step = 64 / seg_lanes,
                              rounded down                                     */
  int32_t lanes_used;      /* lanes per row that hold weights                   */
  int64_t waves;           /* work units (rows_per_step rows each); a persistent
                              launch runs at most the resident waves, each
                              taking a share of the units                      */
  int64_t workgroups;      /* waves / 4, rounded up (a nominal 256-thread
                              grouping; the kernels' own workgroups hold 8 to
                              16 waves)                                        */
  int32_t kernel;          /* BITCOS_KERNEL_*                                   */
  int32_t reserved;
} bitcos_launch_info;

int bitcos_describe(const bitcos_layout* L, int32_t m, int32_t x_dtype, bitcos_launch_info* out);

#ifdef __cplusplus
}
#endif

#endif /* BITCOS_H */
