/*
 * isc.h -- C ABI of the sparse-input ("inverse sparse") convolution library
 * for AMD Instinct MI355X (gfx950).
 *
 * Method: Shi & Chu, "Speeding up Convolutional Neural Networks By Exploiting
 * the Sparsity of Rectifier Units" (arXiv 1704.07724).  The input of a
 * convolution is the output of a ReLU (Eq. 2), so most of its entries are
 * zero; the sparse path lists the nonzero inputs (ISC step 1, Sec. "Sparse
 * Convolution") and multiplies only those with K-contiguous weight vectors
 * (ISC step 2), accumulating an output tile that is written out transposed
 * to NCHW (ISC step 3).  The dense path is the matrix-multiplication
 * formulation M_K x M_I = M_O of Fig. 3 (the im2col matrix M_I times the
 * filter matrix M_K), the paper's baseline; here M_I is gathered from the
 * input inside the GEMM rather than written out.  A dispatcher picks one by measured input sparsity.
 *
 * Conventions shared by every entry point
 *   - All tensors are fp32 (indices int32/uint32), dense and row-major:
 *     input  x  N x C x H x W   (NCHW)
 *     filter w  K x C x R x S   (KCRS)
 *     output y  N x K x Ho x Wo (NCHW),
 *     Ho = floor((H + 2P - R)/T) + 1, Wo = floor((W + 2P - S)/T) + 1.
 *   - Device pointers are caller-owned HIP device allocations on the current
 *     device; the library allocates no device memory.  Work is enqueued on the
 *     given HIP stream (hipStream_t passed as void*, NULL = default stream)
 *     and the call returns without waiting, unless stated otherwise.
 *   - Return value: ISC_OK (0) or one of the positive status codes below.
 *     Arguments are validated on the host before anything is enqueued; on a
 *     validation error nothing is enqueued and no output is touched.  No C++
 *     exception crosses the ABI and nothing is printed.
 *   - Limits: every dimension >= 1, stride >= 1, pad >= 0, Ho and Wo >= 1,
 *     H and W <= 65535, and N*C*H*W, N*K*Ho*Wo, K*C*R*S and N*Ho*Wo each
 *     below 2^31 elements; when C*R*S >= 2^16 the dense path materialises
 *     the im2col matrix (C*R*S rows of N*Ho*Wo rounded up to 256 columns),
 *     which must then be below 2^31 elements too.  Float pointers must be 4-byte aligned, workspaces 256-byte
 *     aligned.
 *   - Calls that share a workspace must not overlap in time (same stream, or
 *     synchronised).
 */
#ifndef ISC_H
#define ISC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Parameters of one convolution: the paper's Tab. 1 ("Parameters of
 * Convolution") with the batch N added.  stride is T, pad is P (the same on
 * both axes and on both sides). */
typedef struct isc_conv_desc {
    int32_t N;      /* images in the batch */
    int32_t C;      /* input feature maps */
    int32_t H, W;   /* input height and width (H_in, W_in) */
    int32_t K;      /* output feature maps */
    int32_t R, S;   /* filter height and width */
    int32_t stride; /* T */
    int32_t pad;    /* P, zero padding */
} isc_conv_desc;

/* Which path isc_conv2d runs. */
typedef enum isc_path {
    ISC_PATH_AUTO = 0,   /* count the nonzero inputs, then sparse if the count is
                            within the limit (the per-shape crossover, or a
                            caller's sparsity threshold), else dense */
    ISC_PATH_SPARSE = 1, /* compaction + zero-skipping convolution */
    ISC_PATH_DENSE = 2   /* MFMA GEMM of Fig. 3 (im2col gathered in the GEMM) */
} isc_path;

/* One entry of the nonzero list of ISC step 1: the value (bit-exact copy of
 * the input) and its position in its plane, yx = (row << 16) | column. */
typedef struct isc_nz {
    float v;
    uint32_t yx;
} isc_nz;

enum isc_status {
    ISC_OK = 0,
    ISC_ERR_NULL = 1,      /* a required pointer is NULL */
    ISC_ERR_SHAPE = 2,     /* a dimension < 1, stride < 1, pad < 0, or Ho/Wo < 1 */
    ISC_ERR_LIMIT = 3,     /* a size exceeds the int32 / 16-bit limits above */
    ISC_ERR_WORKSPACE = 4, /* workspace smaller than isc_workspace_size */
    ISC_ERR_ALIAS = 5,     /* output overlaps an input or the workspace */
    ISC_ERR_PATH = 6,      /* path not an isc_path value */
    ISC_ERR_DEVICE = 7,    /* no device, or the current device is not gfx950 */
    ISC_ERR_HIP = 8,       /* a HIP runtime call failed */
    ISC_ERR_ALIGN = 9,     /* pointer misaligned */
    ISC_ERR_ARG = 10       /* other bad argument (threshold outside [0,1], ...) */
};

/* Per-call plan overrides, in the manner of a DNN library's per-call
 * algorithm argument, for measurements and tests.  Every field 0 means "the
 * library chooses"; a forced value the shape cannot take is ignored (the
 * library's own choice runs), so isc_sparse_plan reports what a call would
 * actually run.  A NULL pointer stands for all zeros.  Nothing in the
 * environment changes a plan: the library reads no environment variables. */
typedef struct isc_tuning {
    int32_t kernel;        /* sparse kernel (an isc_kernel value) to run when it
                              takes the shape */
    int32_t rows;          /* output rows of a wavefront's tile */
    int32_t cols;          /* output columns of a wavefront's tile */
    int32_t maps_per_lane; /* output maps per lane (64 * this per wavefront) */
    int32_t phases;        /* channel phases of the filter-resident kernel */
    int32_t waves;         /* wavefronts per workgroup of the filter-ring kernel */
    int32_t wide_loads;    /* 1: the register-weight kernel loads its weights
                              through a buffer resource on one map group too */
    int32_t gemm_split;    /* -1: the dense GEMM never splits its reduction,
                              and ws needs no room for its partial sums
                              (which isc_workspace_size counts) */
    int32_t reserved;      /* must be 0 */
} isc_tuning;

/* threshold value that asks AUTO for the library's per-shape crossover (the
 * sparsity at which the zero-skipping path starts to beat the dense path for
 * this shape on this GPU) instead of a fixed sparsity. */
#define ISC_THRESHOLD_CROSSOVER (-1.0f)

/* Output extent (Sec. "Sparsity of ReLUs" output-size formula, read as
 * floor((H + 2P - R)/T) + 1; the printed (H + 2P - R + 1)/T agrees at T = 1).
 * Host-only.  Ho/Wo receive the sizes.  Errors: NULL, SHAPE. */
int isc_out_shape(const isc_conv_desc *d, int32_t *Ho, int32_t *Wo);

/* Bytes of device workspace isc_conv2d needs for this descriptor and path
 * (AUTO needs the sparse and dense buffers; the dense path needs an im2col
 * buffer only when C*R*S >= 2^16, and the partial sums of its GEMM's split
 * reduction where the GEMM splits: small grids, and grids of 128 x 128
 * tiles that a split spreads more evenly over the CUs).  Host-only.
 * Errors: NULL, SHAPE, LIMIT, PATH. */
int isc_workspace_size(const isc_conv_desc *d, int32_t path, size_t *bytes);

/* The convolution of Eq. 1 (Sec. "Sparsity of ReLUs"), extended with batch,
 * stride T and zero padding P, no bias and no activation:
 *   y[n,k,i,j] = sum_{c,r,s} w[k,c,r,s] * x[n,c,i*T+r-P,j*T+s-P]
 * (x taken as 0 outside the map).
 *   x, w: device inputs (read only).  y: device output, fully written.
 *   ws, ws_bytes: device workspace, at least isc_workspace_size(d, path)
 *     bytes, 256-byte aligned; contents on entry are ignored.
 *   path: isc_path.  threshold: the sparsity (fraction of zero inputs,
 *     Sec. "Sparse Convolution") at or above which AUTO takes the sparse
 *     path (the paper's experiments use 0.9: Abstract, Sec. "Experiments"),
 *     or ISC_THRESHOLD_CROSSOVER for the library's per-shape crossover.
 *     The decision is made on the device from the count of the input's
 *     nonzeros, with no host synchronisation; isc_decision and
 *     isc_read_decision read it back.
 *   stream: hipStream_t or NULL.
 * A value counts as zero iff its bits with the sign cleared are zero.
 * fp32 throughout; the sparse path accumulates in fp32 in an order of its
 * own, the dense path in MFMA order.  Errors: NULL, SHAPE, LIMIT, WORKSPACE,
 * ALIAS, PATH, ARG, ALIGN, DEVICE, HIP. */
int isc_conv2d(const isc_conv_desc *d, const float *x, const float *w, float *y,
               void *ws, size_t ws_bytes, int32_t path, float threshold,
               void *stream);

/* isc_conv2d with plan overrides (tuning may be NULL: isc_conv2d itself).
 * Errors: as isc_conv2d; ARG for a nonzero reserved field. */
int isc_conv2d_tuned(const isc_conv_desc *d, const float *x, const float *w, float *y,
                     void *ws, size_t ws_bytes, int32_t path, float threshold,
                     const isc_tuning *tuning, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * isc_conv2d with its workspace taken from a buffer the library keeps in
 * device memory, ISC_NOALLOC_SCRATCH_BYTES on every GPU it runs on, held
 * until the process ends.  The caller passes only inputs and outputs; the
 * call allocates nothing.  Every call on one GPU shares that GPU's buffer:
 * calls that overlap in time on one GPU (on different streams without
 * synchronisation, or from several threads) race and must not be made; the
 * buffer needs no clearing (the path writes every word it reads).
 *   x, w, y, path, threshold, stream: as for isc_conv2d.
 * Where the dense GEMM's split reduction would not fit in the buffer with
 * the rest of the workspace, the GEMM runs unsplit (as with tuning
 * gemm_split = -1).
 * Errors: as isc_conv2d (no WORKSPACE); LIMIT also when the workspace this
 * descriptor and path need without the split reduction exceeds
 * ISC_NOALLOC_SCRATCH_BYTES. */
#define ISC_NOALLOC_SCRATCH_BYTES (16u << 20)
int isc_conv2d_noalloc(const isc_conv_desc *d, const float *x, const float *w, float *y,
                       int32_t path, float threshold, void *stream);

/* The per-shape crossover AUTO uses under ISC_THRESHOLD_CROSSOVER: the
 * smallest input sparsity (fraction of zero inputs, the definition under
 * Tab. 2) at which it takes the sparse path, from models of both paths'
 * times on this GPU for the plans this descriptor gets; 2.0 when the sparse
 * path is never expected to win, or only past a sparsity of 0.95, where
 * keeping the choice open (the count and the gated launch of the path not
 * taken, on every call) costs more than it could save (for example 1x1
 * filters at large batch).  Host-only.  Errors: NULL, SHAPE, LIMIT. */
int isc_crossover_sparsity(const isc_conv_desc *d, double *sparsity);

/* After isc_conv2d has completed on `stream` (this call synchronises the
 * stream): the number of nonzero inputs the compaction counted (UINT64_MAX
 * if the call ran the dense path only) and the path taken (ISC_PATH_SPARSE
 * or ISC_PATH_DENSE).  ws/ws_bytes as passed to isc_conv2d.  Errors: NULL,
 * WORKSPACE, HIP. */
int isc_decision(const isc_conv_desc *d, const void *ws, size_t ws_bytes,
                 uint64_t *nnz_total, int32_t *path_taken, void *stream);

/* The same record read by the host once the caller has synchronised the
 * call that wrote it (this call waits for nothing): the path taken
 * (ISC_PATH_SPARSE or ISC_PATH_DENSE) and the input's nonzero count behind
 * the decision (sparsity = 1 - nnz / (N*C*H*W), the definition under Tab. 2
 * and the density rho of Sec. "Sparse Convolution"; UINT64_MAX when no
 * count was taken).  ws: the workspace the call used (its first 16 bytes
 * hold the record).  Errors: NULL, DEVICE, HIP. */
int isc_read_decision(const void *ws, int32_t *path, uint64_t *nnz);

/* ---- Layer chains: the rectifier of Eq. 2 in the convolution's epilogue ----
 *
 * In a network the input of a convolution is the rectified output of the
 * layer before (Eq. 2, Sec. "Sparsity of ReLUs"), and its sparsity is what
 * the dispatcher needs.  isc_conv2d_relu applies the rectifier where y is
 * written and counts the nonzeros of the rectified y in the same pass, into
 * a census: one count per workgroup of the kernel that wrote y, behind a
 * header that names the entries they cover (layout private to the library;
 * no counter to clear, no atomics).  Given to the next layer as x_census,
 * it replaces that layer's count of its input, so a chain of layers reads
 * every activation once and writes it once, with no separate ReLU pass. */

/* Bytes of the census of the output of a convolution with descriptor d
 * (the layer that writes it).  Host-only.  Errors: NULL, SHAPE, LIMIT. */
int isc_census_size(const isc_conv_desc *d, size_t *bytes);

/* y = max(0, conv(x, w)): the convolution of isc_conv2d, then the rectifier
 * of Eq. 2 on every entry (v > 0 ? v : +0, so -0 and NaN give +0), with the
 * nonzero count of y written to y_census.
 *   x, w, y, ws, ws_bytes, path, threshold, stream: as for isc_conv2d (the
 *     workspace size is isc_workspace_size's).
 *   x_census, x_census_bytes: the census an isc_conv2d_relu call wrote for
 *     x (16-byte aligned), or NULL.  AUTO then decides from it instead of
 *     counting x.  A census that does not cover exactly N*C*H*W entries
 *     (never written, or written for another shape) leaves the count
 *     unknown and AUTO runs the dense path: y is right either way.  Shapes
 *     whose sparse path runs over compacted lists (isc_sparse_kernel not
 *     FUSED, FUSED_REG or FUSED_RING) count x while listing it and ignore
 *     x_census.
 *   wt: the repacked filter of isc_repack_filter for K, C, R, S of d
 *     (16-byte aligned), or NULL to repack w into the workspace on every
 *     call.  Used by the on-the-fly sparse kernels.
 *   y_census, y_census_bytes: at least isc_census_size(d) bytes, 16-byte
 *     aligned, or NULL for no census.
 *   tuning: plan overrides, or NULL.
 * The on-the-fly sparse kernels and the GEMM kernels rectify and count as
 * they store y; after a kernel over compacted lists, one more launch
 * rectifies y in place and counts it.  y must not overlap x, w, wt, ws or a
 * census; y_census must not overlap any other argument.
 * Errors: as isc_conv2d; WORKSPACE also for a census smaller than needed;
 * ALIGN for a misaligned census or wt. */
int isc_conv2d_relu(const isc_conv_desc *d, const float *x, const void *x_census,
                    size_t x_census_bytes, const float *w, const float *wt, float *y,
                    void *y_census, size_t y_census_bytes, void *ws, size_t ws_bytes,
                    int32_t path, float threshold, const isc_tuning *tuning, void *stream);

/* After the call that wrote `census` has completed on `stream` (this call
 * synchronises the stream): the number of entries the census covers and how
 * many of them are nonzero.  bytes: the census buffer's size.  Errors:
 * NULL, WORKSPACE (bytes below the header), ARG (the buffer holds no
 * census), DEVICE, HIP. */
int isc_census_read(const void *census, size_t bytes, uint64_t *elems, uint64_t *nnz,
                    void *stream);

/* ISC step 1 (Sec. "Sparse Convolution"): list the nonzero inputs of every
 * (n, c) plane with their row and column, in row-major order.
 *   row_ptr: device int32[N*C*(H+1)]; row_ptr[p*(H+1) + y] = nonzeros of
 *     plane p = n*C + c in rows < y (plane-relative), so row_ptr[p*(H+1)+H]
 *     is the plane's count.
 *   nz: device isc_nz[N*C*H*W]; entry e of plane p at nz[p*H*W + e]; slots
 *     past the plane's count are not written.
 *   nnz_total: device uint64, set to the total count (cleared by the call).
 * The output is unique and bit-exact (values are bit copies).  Filter fields
 * of d (K, R, S, stride, pad) must be valid but are otherwise unused.
 * Errors: NULL, SHAPE, LIMIT, ALIAS, ALIGN, DEVICE, HIP. */
int isc_compact(const isc_conv_desc *d, const float *x, int32_t *row_ptr,
                isc_nz *nz, uint64_t *nnz_total, void *stream);

/* Bytes isc_repack_filter writes for this descriptor (K, C, R, S used).
 * Host-only.  Errors: NULL, SHAPE, LIMIT. */
int isc_repacked_filter_size(const isc_conv_desc *d, size_t *bytes);

/* ISC step 2's filter layout (Sec. "Sparse Convolution": the kernel matrix
 * stored column-major, so that for one input channel and tap the weights of
 * consecutive output maps are contiguous and can be fetched together), with
 * the output-map dimension zero padded to a multiple of 64:
 *   wt[((c*R + r)*S + s)*Kp + k] = w[k, c, r, s],  Kp = ceil(K/64)*64,
 *   0 for K <= k < Kp.
 *   w: device K x C x R x S; wt: device buffer of isc_repacked_filter_size
 *   bytes, 16-byte aligned, must not overlap w.
 * Only K, C, R, S of d are used (all must be valid).  Errors: NULL, SHAPE,
 * LIMIT, ALIAS, ALIGN, DEVICE, HIP. */
int isc_repack_filter(const isc_conv_desc *d, const float *w, float *wt, void *stream);

/* ISC steps 2 and 3 (Sec. "Sparse Convolution") on lists that isc_compact
 * produced for the same input shape: for every nonzero x[n,c,y,x] and every
 * filter tap (r, s) that reaches a valid output, add x * wt[c,r,s,k] to
 * y[n, k, (y+P-r)/T, (x+P-s)/T]; then y holds the convolution of Eq. 1.
 *   row_ptr, nz: as written by isc_compact for N, C, H, W of d (read only;
 *     nz must have 256 readable entries past N*C*H*W -- isc_conv2d's
 *     workspace does; a caller's own buffer of N*C*H*W + 256 entries does).
 *   wt: the repacked filter of isc_repack_filter (16-byte aligned).
 *   y: device output N x K x Ho x Wo, fully written, must not overlap the
 *     inputs.
 *   tuning: plan overrides (kernel, rows, maps_per_lane, phases), or NULL.
 * One launch, no workspace, deterministic (each output is summed by one
 * lane in list order).  Several convolutions of the same input (for example
 * the branches of an inception block) can share one compaction.  Errors:
 * NULL, SHAPE, LIMIT (no LDS tiling fits the shape), ALIAS, ALIGN, DEVICE,
 * HIP. */
int isc_sparse_conv(const isc_conv_desc *d, const int32_t *row_ptr, const isc_nz *nz,
                    const float *wt, float *y, const isc_tuning *tuning, void *stream);

/* ISC steps 1-3 (Sec. "Sparse Convolution") in one launch with no workspace:
 * each wavefront compacts the input rows it needs on the fly (a ballot of
 * the zero test over its window, scanned in row-major order) and multiplies
 * each nonzero by the K-contiguous weight vectors of step 2, which it holds
 * in registers.  The filter is resident in LDS when it fits (K <= 64:
 * ISC_KERNEL_FUSED), streamed from L2 into each wavefront's registers at
 * stride 1 with at most 16 output columns (ISC_KERNEL_FUSED_REG, one
 * workgroup per group of 64 output maps: taken there when K > 64, when the
 * filter does not fit in LDS, or when every wavefront of the resident plan
 * would own its channels alone), and streamed through LDS otherwise
 * (ISC_KERNEL_FUSED_RING).  The kernels isc_conv2d's sparse path runs when
 * isc_sparse_kernel reports either (isc_conv2d repacks the filter itself, in
 * the launch that counts the nonzeros); no sparse/dense decision here.
 *   x: device input as for isc_conv2d.
 *   wt: the repacked filter of isc_repack_filter for K, C, R, S of d.
 *   y: device output N x K x Ho x Wo, fully written, must not overlap x or
 *     wt.
 *   tuning: plan overrides, or NULL.
 * Deterministic (fixed summation order per output).  Errors: NULL, SHAPE,
 * LIMIT (shape not eligible: a square 1x1, 3x3 or 5x5 filter at stride 1,
 * or a 3x3 or 5x5 filter at stride 2 with K <= 64, a filter that fits in LDS
 * and at most 8 output columns), ALIAS, ALIGN, DEVICE, HIP. */
int isc_sparse_conv_fused(const isc_conv_desc *d, const float *x, const float *wt, float *y,
                          const isc_tuning *tuning, void *stream);

/* Which kernel isc_conv2d's sparse path runs for this descriptor, reported in
 * *kernel: ISC_KERNEL_FUSED, ISC_KERNEL_FUSED_REG or ISC_KERNEL_FUSED_RING
 * (compaction on the fly, isc_sparse_conv_fused; filter resident in LDS,
 * each wavefront's own channels' weights streamed to registers -- for plans
 * whose wavefronts share no input channel, at stride 1 and at most 16
 * output columns, any K -- or filter streamed through LDS), else
 * the kernel over compacted lists that isc_sparse_conv also runs:
 * ISC_KERNEL_RESIDENT (filter resident in LDS), ISC_KERNEL_RING (filter
 * streamed through LDS) or ISC_KERNEL_GENERIC (any filter and stride);
 * ISC_KERNEL_NONE if no sparse kernel fits (AUTO then runs dense).
 * Host-only.  Errors: NULL, SHAPE, LIMIT. */
enum isc_kernel {
    ISC_KERNEL_NONE = 0,
    ISC_KERNEL_FUSED = 1,
    ISC_KERNEL_RESIDENT = 2,
    ISC_KERNEL_RING = 3,
    ISC_KERNEL_GENERIC = 4,
    ISC_KERNEL_FUSED_RING = 5,
    ISC_KERNEL_FUSED_REG = 6
};
int isc_sparse_kernel(const isc_conv_desc *d, int32_t *kernel);

/* The whole plan of the sparse path for this descriptor under the given
 * overrides (tuning may be NULL): the kernel, its wavefront tile (rows x
 * cols x 64*maps_per_lane output maps), the channel phases per tile, the
 * wavefronts per workgroup and the workgroups of its launch.  Host-only.
 * Errors: NULL, SHAPE, LIMIT, ARG (nonzero reserved field). */
typedef struct isc_plan {
    int32_t kernel;         /* isc_kernel value; ISC_KERNEL_NONE: no sparse kernel fits */
    int32_t rows, cols;     /* output tile of one wavefront */
    int32_t maps_per_lane;  /* output maps per lane */
    int32_t phases;         /* channel phases summed per tile (1: none) */
    int32_t waves;          /* wavefronts per workgroup */
    int64_t workgroups;     /* workgroups of the launch */
} isc_plan;
int isc_sparse_plan(const isc_conv_desc *d, const isc_tuning *tuning, isc_plan *plan);

/* ---- Training: the weight gradient with zero skipping ----
 *
 * The paper measures the sparsity of the rectified inputs during training
 * (Sec. "Sparsity of ReLUs").  The gradient of Eq. 1 with respect to the
 * filter multiplies every input by output gradients, so a zero input adds
 * nothing: isc_conv2d_dw visits the nonzero inputs only, each meeting the
 * K-contiguous vector of output gradients it reaches (ISC step 2 with the
 * roles of filter and output exchanged). */

/* Bytes of device workspace isc_conv2d_dw needs (per-range partial sums).
 * Host-only.  Errors: NULL, SHAPE, LIMIT (not stride 1 with a square 1x1,
 * 3x3 or 5x5 filter). */
int isc_conv2d_dw_workspace_size(const isc_conv_desc *d, size_t *bytes);

/*   dw[k,c,r,s] = sum_{n,i,j} dy[n,k,i,j] * x[n, c, i*T + r - P, j*T + s - P]
 * (x taken as 0 outside the map), stride T = 1.
 *   x: device input N x C x H x W; dy: device output gradient N x K x Ho x Wo
 *     (read only).
 *   dw: device K x C x R x S, fully written; must not overlap x, dy or ws.
 *   ws, ws_bytes: workspace of isc_conv2d_dw_workspace_size bytes, 256-byte
 *     aligned; contents on entry are ignored.
 *   tuning: plan overrides (rows, maps_per_lane), or NULL; the workspace
 *     size holds for every override.
 * Two launches: one wavefront per 64 or 128 output maps, a few input channels
 * and a range of output rows sums in registers over the nonzero inputs of
 * its range; the ranges' sums are then added in order.  fp32, deterministic.
 * Errors: NULL, SHAPE, LIMIT, WORKSPACE, ALIAS, ALIGN, DEVICE, HIP. */
int isc_conv2d_dw(const isc_conv_desc *d, const float *x, const float *dy, float *dw,
                  void *ws, size_t ws_bytes, const isc_tuning *tuning, void *stream);

/* The unrolled input matrix M_I of the matrix-multiplication formulation
 * (Sec. "Sparse Convolution", Fig. 3), with the batch as extra columns:
 *   col[(c*R + r)*S + s][(n*Ho + i)*Wo + j] = x[n, c, i*T + r - P, j*T + s - P]
 * (0 outside the map), row stride ldc >= N*Ho*Wo elements; columns
 * [N*Ho*Wo, ldc) of every row are set to 0.  Bit-exact copy.
 * Errors: NULL, SHAPE, LIMIT, ALIAS, ALIGN, ARG (ldc too small), DEVICE, HIP. */
int isc_im2col(const isc_conv_desc *d, const float *x, float *col, int64_t ldc,
               void *stream);

/* The GEMM of Fig. 3 on its own: c[m][n] = sum_k a[m][k] * b[k][n] for
 * m < M, n < Ncols, k < Kd, fp32 inputs and accumulation on the fp32 matrix
 * cores.  Row-major with leading dimensions lda >= Kd, ldb >= Ncols,
 * ldc >= Ncols (elements).  Errors: NULL, SHAPE, LIMIT, ALIAS, ALIGN,
 * DEVICE, HIP. */
int isc_gemm_f32(int32_t M, int32_t Ncols, int32_t Kd, const float *a, int64_t lda,
                 const float *b, int64_t ldb, float *c, int64_t ldc, void *stream);

/* Short text for a status code (static storage). */
const char *isc_status_str(int status);

/* Library version, for logs. */
const char *isc_version(void);

#ifdef __cplusplus
}
#endif

#endif /* ISC_H */
