/* spconv.h - C ABI of the MI355X (gfx950) sparse-convolution library.
 *
 * Implements the two sparse convolutions of Graham & van der Maaten,
 * "Submanifold Sparse Convolutional Networks":
 *   SC(m, n, f, s)   an output site is active when any input site of its
 *                    f^d receptive field is active; output extent
 *                    (l - f + s) / s; inactive inputs count as zero
 *                    (Section 3, definition of SC);
 *   VSC(m, n, f, 1)  input padded by (f - 1)/2, output active exactly where
 *                    the central input site is active, so the output set is
 *                    the input set (Section 3, definition of VSC).
 * Each layer has two phases (Section 4, Implementation): building the rule
 * book R = (R_i) of (input row, output row) pairs per filter offset i, and
 * the forward multiply-add, which starts from a zero output and adds
 * (input row R_i(j,1)) x W^i into output row R_i(j,2).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Sites.   A site is a tuple of D = 1 + d int32 coordinates; coordinate 0 is
 *          the sample index in a batch.  Filters and strides are per
 *          dimension with f[0] = s[0] = 1, so samples never interact.
 *          1 <= spatial_size[j] <= 65535; every coordinate must satisfy
 *          0 <= c_j < spatial_size[j].  2 <= D <= 4.
 * Offsets. Filter offsets o in prod_j [0, f_j) are flattened row-major, last
 *          dimension fastest: i = sum_j o_j prod_{l>j} f_l; K = prod_j f_j.
 *          W^i multiplies the input site y + o - (f-1)/2 (VSC) or s*y + o
 *          (SC) for output site y: a cross-correlation, no filter flip.
 * Rows.    VSC output row r is input row r.  SC output rows are numbered in
 *          lexicographic order of the output site (sample first).
 *          Pairs inside R_i are ordered along the Z-order (Morton) curve of
 *          their output site: sample first, then the coordinates' bits level
 *          by level from the most significant, coordinate 1 first within a
 *          level (the order the forward walks its output tiles).
 * Memory.  coords, x, w, bias, y are device pointers owned by the caller:
 *          contiguous, row-major, 16-byte aligned.  Host pointers are marked
 *          "host".  A rule book owns its device memory (taken on the build
 *          stream from the library's allocator, see spconv_set_allocator)
 *          until spconv_rulebook_destroy.  A feature pointer whose row count
 *          is zero may be NULL (an SC book's output rows count as zero only
 *          once the book is synchronised; before, their bound counts).
 * Streams. `stream` is a hipStream_t passed as void*; NULL is the null
 *          stream.  All work is enqueued on it.
 * Errors.  Every call returns a spconv_status; nothing is printed and
 *          nothing aborts.  Argument errors are detected on the host before
 *          any work is enqueued.
 */
#ifndef SPCONV_H
#define SPCONV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SPCONV_OK = 0,
  SPCONV_EINVAL = -1, /* bad argument, dtype, shape or rule-book kind       */
  SPCONV_EDUP = -2,   /* a site appears twice in the input coordinates      */
  SPCONV_ERANGE = -3, /* a coordinate lies outside [0, spatial_size)         */
  SPCONV_ENOMEM = -4, /* device allocation failed                            */
  SPCONV_ECAP = -5,   /* hash table full (only with a forced tiny capacity)  */
  SPCONV_EHIP = -6,   /* a HIP runtime call failed                           */
  SPCONV_ESCRATCH = -7 /* the call needs more than the library's fixed scratch
                        * array (spconv_backward_weight_noalloc)             */
} spconv_status;

typedef enum { SPCONV_F32 = 0, SPCONV_BF16 = 1 } spconv_dtype;
typedef enum { SPCONV_VSC = 0, SPCONV_SC = 1 } spconv_kind;
/* Layer operations for the gradients: the two convolutions and the
 * deconvolution DC(.,.,f,s), which runs on the rule book of the
 * SC(.,.,f,s) it inverts (Section 3). */
typedef enum { SPCONV_OP_VSC = 0, SPCONV_OP_SC = 1, SPCONV_OP_DC = 2 } spconv_op;
/* Sparse pooling (Section 3: MP(f,s) and AP(f,s), variants of SC). */
typedef enum { SPCONV_POOL_MAX = 0, SPCONV_POOL_AVG = 1 } spconv_pool_mode;

/* Build flags. */
enum {
  /* Return as soon as the work is enqueued.  Device-detected errors
   * (EDUP, ERANGE, ECAP) are then reported by spconv_rulebook_status. */
  SPCONV_BUILD_ASYNC = 1,
  /* SC only: also build the transposed rule book (every pair reversed),
   * which spconv_dc_forward and the SC input gradient walk. */
  SPCONV_BUILD_TRANSPOSE = 2
};

typedef struct spconv_rulebook_s* spconv_rulebook;

/* Build the rule book of one layer (Section 4: map the active sites to rows,
 * then list for every filter offset the (input row, output row) pairs; VSC
 * re-uses the input site set as its output set).  The site map is a dense
 * index grid when the grid is small enough, else a hash table; the result
 * does not depend on which.
 *
 *   kind          SPCONV_VSC or SPCONV_SC
 *   D             coordinates per site, 2..4 (sample index + d spatial)
 *   coords        device int32 [N][D], distinct sites
 *   N             number of active input sites, >= 0 (0 gives an empty book)
 *   spatial_size  host int32 [D], grid extent; spatial_size[0] = batch size
 *   f, s          host int32 [D], filter size and stride; f[0] = s[0] = 1;
 *                 VSC needs every f_j odd and every s_j = 1
 *   flags         0 (wait for the device result), SPCONV_BUILD_ASYNC, and for
 *                 SC optionally SPCONV_BUILD_TRANSPOSE (OR-ed)
 *   stream        hipStream_t as void*
 *   out           receives the handle; NULL on any error
 *
 * Errors: EINVAL (arguments), EDUP, ERANGE, ECAP (device-detected; with
 * flags = 0 they are returned here and nothing is kept), ENOMEM, EHIP.
 * The rule book is immutable once built; any number of forwards, on any
 * stream ordered after the build, may use it (Section 4: one rule book
 * serves every layer with the same sparsity pattern). */
int spconv_build_rulebook(int kind, int D, const int32_t* coords, int64_t N,
                          const int32_t* spatial_size, const int32_t* f,
                          const int32_t* s, unsigned flags, void* stream,
                          spconv_rulebook* out);

/* Build the rule book of the next layer on the output sites of an SC rule
 * book (Section 5's networks stack VSC and SC layers level by level): the
 * sites are parent's output coordinates in parent's row order, the grid is
 * parent's output grid, and the site count stays on the device, so with
 * SPCONV_BUILD_ASYNC a whole chain of levels is built without the host
 * waiting once.  kind, f, s, flags and stream as spconv_build_rulebook
 * (SPCONV_BUILD_TRANSPOSE not accepted here).  Until the book is
 * synchronised its input row count is a bound (spconv_rulebook_bounds); the
 * forward reads the real counts on the device.  parent must outlive the
 * enqueued build (destroying it later on the same stream is enough).  Grids
 * too large for the dense-grid path make this call wait for parent's count
 * and build as spconv_build_rulebook does.  Errors: EINVAL (parent not SC,
 * TRANSPOSE, as spconv_build_rulebook), and the build's own. */
int spconv_build_rulebook_on(spconv_rulebook parent, int kind, const int32_t* f,
                             const int32_t* s, unsigned flags, void* stream,
                             spconv_rulebook* out);

/* Host-side bounds, known without waiting for the device: input rows and
 * output rows the book's buffers are sized for (for allocating layer outputs
 * ahead of an asynchronous build).  Errors: EINVAL (NULL). */
int spconv_rulebook_bounds(spconv_rulebook rb, int64_t* n_in_bound, int64_t* n_out_bound);

/* Wait for the build and return its device-detected status (OK, EDUP,
 * ERANGE or ECAP).  Needed only after an SPCONV_BUILD_ASYNC build. */
int spconv_rulebook_status(spconv_rulebook rb);

/* Sizes of a rule book (waits for the build).  Any output may be NULL.
 *   n_in, n_out       active input / output sites
 *   K                 number of filter offsets, prod f_j
 *   out_spatial_size  host int32 [D]: VSC = input size; SC = floor((l-f)/s)+1
 *   pair_off          host int64 [K+1]: pair_off[i+1] - pair_off[i] = k_i,
 *                     the length of R_i (Section 4, rule book). */
int spconv_rulebook_query(spconv_rulebook rb, int64_t* n_in, int64_t* n_out,
                          int64_t* K, int32_t* out_spatial_size,
                          int64_t* pair_off);

/* Copy the output sites and the rule book into caller buffers (device).
 *   out_coords  device int32 [n_out][D] or NULL
 *   pairs       device int32 [pair_off[K]][2] or NULL: (input row, output
 *               row), R_0 first, each R_i in Z-order of the output site.
 * Enqueued on `stream` after the build. */
int spconv_rulebook_export(spconv_rulebook rb, int32_t* out_coords,
                           int32_t* pairs, void* stream);

/* Device pointer to the rule book's own output sites, int32 [n_out][D],
 * valid until the rule book is destroyed (lets an SC output feed the next
 * build without a copy). */
int spconv_rulebook_out_coords(spconv_rulebook rb, const int32_t** coords);

/* Forward pass of a VSC layer (Section 4: zero the output, then for every
 * offset i and pair j add x[R_i(j,1)] W^i into y[R_i(j,2)]; plus bias).
 *   rb      a rule book of kind SPCONV_VSC
 *   in_dt   dtype of x and w: SPCONV_F32 or SPCONV_BF16
 *   x       device [n_in][C_in]
 *   w       device [K][C_in][C_out] (W^i is w[i], an m x n matrix)
 *   bias    device fp32 [C_out] or NULL; added once at every output site
 *   out_dt  dtype of y: SPCONV_F32 or SPCONV_BF16
 *   y       device [n_out][C_out], fully overwritten
 * Accumulation is fp32, in ascending offset order, without atomics, so
 * repeated calls give bit-identical results; the result is rounded once to
 * out_dt (round to nearest even).  Nothing is allocated; the call is
 * asynchronous on `stream`.  Errors: EINVAL (kind, dtype, C < 1, NULL). */
int spconv_vsc_forward(spconv_rulebook rb, int in_dt, const void* x,
                       const void* w, const float* bias, int out_dt, void* y,
                       int C_in, int C_out, void* stream);

/* Forward pass of an SC layer; arguments as spconv_vsc_forward, with rb of
 * kind SPCONV_SC and y of n_out rows (Section 3 / Section 4). */
int spconv_sc_forward(spconv_rulebook rb, int in_dt, const void* x,
                      const void* w, const float* bias, int out_dt, void* y,
                      int C_in, int C_out, void* stream);

/* Forward pass of a VSC or SC layer with its block epilogue fused into the
 * single store of the output.  The networks of Section 5 follow each
 * convolution with batch normalisation and a ReLU acting on the active
 * sites only, and their residual blocks add the block input back before the
 * last ReLU; at inference the batch normalisation is an affine map per
 * channel.  For every output row r and channel n:
 *   z = acc[r][n] * scale[n] + shift[n] + residual[r][n]
 *   y[r][n] = relu ? (z < 0 ? 0 : z) : z          (NaN stays NaN)
 * computed in fp32 and rounded once to out_dt.
 *   rb        rule book of kind SPCONV_VSC or SPCONV_SC
 *   scale     device fp32 [C_out] or NULL (= 1)
 *   shift     device fp32 [C_out] or NULL (= 0); with scale NULL this is the
 *             bias of spconv_vsc_forward
 *   residual  device [n_out][C_out] of dtype out_dt, or NULL (= 0); it may
 *             be y itself (in place), but must not overlap y otherwise
 *   relu      0 or 1
 * Other arguments, ordering, determinism and ownership as
 * spconv_vsc_forward.  Errors: EINVAL (kind, dtype, C < 1, NULL, relu not
 * 0/1, alignment: x, w, y, residual 16 bytes, scale and shift 4 bytes). */
int spconv_forward_fused(spconv_rulebook rb, int in_dt, const void* x, const void* w,
                         const float* scale, const float* shift, const void* residual,
                         int relu, int out_dt, void* y, int C_in, int C_out, void* stream);

/* Sparse max- or average-pooling (Section 3: MP(f,s) takes the maximum of
 * the zero vector and the input vectors of the receptive field, AP(f,s)
 * f^-d times the sum of the active input vectors; both are variants of
 * SC(.,.,f,s) and run on its rule book).
 *   rb      a rule book of kind SPCONV_SC (its f and s are the pooling's)
 *   mode    SPCONV_POOL_MAX or SPCONV_POOL_AVG
 *   dt      dtype of x and y (SPCONV_F32 or SPCONV_BF16)
 *   x       device [n_in][C];  y  device [n_out][C], fully overwritten
 * MP compares with IEEE maxNum (a NaN input is ignored) and is exact; AP
 * sums in fp32 in ascending offset order and divides once by prod_j f_j
 * (f^-d for non-square fields), rounded once to dt.  Asynchronous, allocates
 * nothing.  Errors: EINVAL (kind, dtype, mode, C < 1, NULL, alignment). */
int spconv_pool_forward(spconv_rulebook rb, int mode, int dt, const void* x, void* y,
                        int C, void* stream);

/* Deconvolution DC(.,.,f,s) (Section 3: the inverse of SC(.,.,f,s); its
 * active output sites are the SC input sites, every connection reversed):
 * y[a] = bias + sum_i sum_{(a,b) in R_i} x[b] W^i.
 *   rb      the SC(.,.,f,s) rule book, built with SPCONV_BUILD_TRANSPOSE
 *   x       device [n_out][C_in] (features on the SC output sites)
 *   w       device [K][C_in][C_out]; bias fp32 [C_out] or NULL
 *   y       device [n_in][C_out] (rows in the SC input order), overwritten
 * Accumulation, rounding and determinism as spconv_vsc_forward.  For
 * f = s the first such call on a book reads its pair offsets once (a wait);
 * later calls are asynchronous.
 * Errors: EINVAL (kind, no transposed book, dtype, C < 1, NULL). */
int spconv_dc_forward(spconv_rulebook rb, int in_dt, const void* x, const void* w,
                      const float* bias, int out_dt, void* y, int C_in, int C_out,
                      void* stream);

/* Gradient with respect to the input of a layer (the networks of Section 5
 * are trained by SGD): every pair runs in the opposite direction with W^i
 * transposed.  C_in, C_out and w ([K][C_in][C_out]) are the layer's.
 *   op SPCONV_OP_VSC (VSC book):  dy [n_out][C_out] -> dx [n_in][C_in]
 *   op SPCONV_OP_SC  (SC book built with SPCONV_BUILD_TRANSPOSE):
 *                                 dy [n_out][C_out] -> dx [n_in][C_in]
 *   op SPCONV_OP_DC  (SC book):   dy [n_in][C_out]  -> dx [n_out][C_in]
 * dt is the dtype of dy and w, out_dt that of dx.  fp32 accumulation in a
 * fixed order, rounded once; deterministic; allocates nothing; asynchronous
 * (for op SC with f = s the first such call on a book reads its pair offsets
 * once, as spconv_dc_forward).
 * Errors: EINVAL (op / book mismatch, missing transposed book, dtype, NULL). */
int spconv_backward_data(spconv_rulebook rb, int op, int dt, const void* dy, const void* w,
                         int out_dt, void* dx, int C_in, int C_out, void* stream);

/* Workspace bytes spconv_backward_weight needs for this book, op and shape
 * (waits for the build).  Errors: EINVAL. */
int spconv_backward_weight_workspace(spconv_rulebook rb, int op, int C_in, int C_out,
                                     size_t* bytes);

/* Gradients of the weights and the bias of a layer:
 *   dw[i][c][n] = sum_{(a,b) in R_i} x[a][c] dy[b][n]        (VSC, SC)
 *   dw[i][c][n] = sum_{(a,b) in R_i} x[b][c] dy[a][n]        (DC)
 *   db[n]       = sum over the layer's output rows of dy[.][n]
 *   x, dy     device, dtype dt, shaped as the layer's input and output
 *             gradient (see spconv_backward_data)
 *   dw        device fp32 [K][C_in][C_out], overwritten; db fp32 [C_out] or NULL
 *   workspace device scratch of at least spconv_backward_weight_workspace
 *             bytes, owned by the caller (its contents are overwritten)
 * Each R_i is summed in fixed chunks, and the chunks in ascending order:
 * deterministic, no atomics.  Allocates nothing; asynchronous, except that
 * a book built with SPCONV_BUILD_ASYNC is waited for once here (the bias
 * gradient needs its output count on the host).
 * Errors: EINVAL (op / book mismatch, dtype, NULL, workspace too small). */
int spconv_backward_weight(spconv_rulebook rb, int op, int dt, const void* x, const void* dy,
                           float* dw, float* db, int C_in, int C_out, void* workspace,
                           size_t workspace_bytes, void* stream);

/* Size of the library's fixed device scratch array (one per GPU the library
 * runs on, held until the process ends): 128 MiB. */
#define SPCONV_NOALLOC_SCRATCH_BYTES (128u << 20)

/* spconv_backward_weight for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same gradients, the same kernels and the same results,
 * bit for bit, with the partial sums kept in the library's fixed scratch
 * array instead of a caller workspace.  Arguments as spconv_backward_weight
 * without the workspace; the book's device must be the current device.
 * Allocates nothing (no hipMalloc, hipFree or allocating library routine).
 * Every call on one GPU shares that GPU's array: calls that overlap on one
 * GPU (on different streams, or from different host threads) race and must
 * be ordered by the caller; nothing in the array needs to start at zero.  A
 * book built with SPCONV_BUILD_ASYNC is waited for once, as in
 * spconv_backward_weight (under graph capture, synchronise the book first).
 * Errors: those of spconv_backward_weight; ESCRATCH when the partials
 * (spconv_backward_weight_workspace bytes) exceed
 * SPCONV_NOALLOC_SCRATCH_BYTES; EINVAL when the book's device is not
 * current. */
int spconv_backward_weight_noalloc(spconv_rulebook rb, int op, int dt, const void* x,
                                   const void* dy, float* dw, float* db, int C_in, int C_out,
                                   void* stream);

/* Device memory of the rule books.  Every allocation the library makes (a
 * rule book's persistent block and the transient buffers of a build) comes
 * from alloc(bytes, stream, ctx) and goes back through
 * release(ptr, stream, ctx), both on the build stream and stream-ordered
 * there (a caching allocator may hand the memory to later work on that
 * stream).  A rule book keeps the pair it was built with, so a change applies
 * to later builds only.  Both NULL (the default): the library's own block
 * cache (see spconv_release_cached_memory).  An alloc that returns NULL makes
 * the build return ENOMEM
 * after releasing everything it had taken.  Ownership: the library calls
 * release exactly once for every non-NULL pointer alloc returned.  Errors:
 * EINVAL when only one of the two functions is given.  Set it while no build
 * is running on another thread. */
int spconv_set_allocator(void* (*alloc)(size_t bytes, void* stream, void* ctx),
                         void (*release)(void* ptr, void* stream, void* ctx), void* ctx);

/* The default allocator keeps the device memory that rule books and builds
 * give back (on their build stream) and hands it to later requests of up to
 * the block's size on any stream: an event recorded where the block was given
 * back is waited for on the new stream (on the device; the host never waits),
 * so the blocks of a book rebuilt every step are reused without driver calls.
 * When a fresh hipMalloc fails, the idle blocks of that device are freed and
 * the allocation is tried once more.  spconv_release_cached_memory frees every
 * idle block on every device (waiting for the work that last used each) and
 * stores the bytes freed in *released (may be NULL); blocks of live rule books
 * stay.  Always SPCONV_OK.  Another allocator in the same process (a caching
 * one such as torch's) cannot take memory held idle here: call this first, or
 * route the library through that allocator with spconv_set_allocator. */
int spconv_release_cached_memory(int64_t* released);

/* Bytes of device memory on `device` that the default allocator has handed
 * out (live rule books and running builds) and holds idle.  Either pointer
 * may be NULL.  Errors: EINVAL for a device index out of range, EHIP. */
int spconv_memory_stats(int device, int64_t* in_use, int64_t* cached);

/* Release a rule book.  Stream-ordered: the memory is given back on the
 * build stream after the build stream's own work and after the latest work
 * that any other stream enqueued on this book (every call that takes the
 * book records, on a stream other than the build stream, an event there
 * that the release waits on).  The host does not wait.  NULL is a no-op. */
void spconv_rulebook_destroy(spconv_rulebook rb);

/* Static string naming a status code. */
const char* spconv_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* SPCONV_H */
