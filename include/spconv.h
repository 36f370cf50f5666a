/*
 * spconv.h - fused sparse direct convolution on MI355X (gfx950).
 *
 * C ABI of libspconv.so. The operation is the sparse direct convolution of the
 * paper's "Optimizing Sparse Neural Networks" section (paragraph "Sparse
 * Convolution with CSR"): the filter of shape (K, C, R, S) is viewed as a
 * K x (C*R*S) matrix and its rows are compressed (CSR); for every output channel
 * k and every nonzero (offset, coeff) of row k, each output pixel accumulates
 * coeff times the padded input at the pixel's position plus the offset. The
 * output is the dense convolution written in the paper's DSL section (read as a
 * cross-correlation over the zero-padded input, no filter flip) followed, when
 * requested, by the ReLU and 2x2 max-pool of its "Conv-Relu-Maxpool" block
 * (section "Evaluation"), all fused into one kernel and one store.
 *
 * Layouts are NCHW, fp32, row-major. Hp = H + 2*pad, Wp = W + 2*pad,
 * Ho = (Hp - R)/stride + 1, Wo = (Wp - S)/stride + 1 (floor); with the pool flag
 * the stored output is Ho/2 x Wo/2 (floor: an odd last row/column is dropped).
 *
 * Every call returns an int status (SPCONV_OK or a negative code) and never
 * throws. Argument checks happen on the host before any GPU work is queued.
 * The caller owns every buffer; the library keeps no state, so calls on
 * different streams may run concurrently.
 */
#ifndef SPCONV_H
#define SPCONV_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define SPCONV_OK 0
#define SPCONV_EINVAL (-1)    /* invalid argument; nothing was queued */
#define SPCONV_ECAPACITY (-2) /* output arrays too small for the nonzeros (pack) */
#define SPCONV_EHIP (-3)      /* a HIP call or kernel launch failed */

/* Flags for spconv_forward. Any other bit is SPCONV_EINVAL. */
#define SPCONV_RELU 1u       /* out = max(pre, 0) */
#define SPCONV_MAXPOOL2X2 2u /* 2x2 window, stride 2, applied after the ReLU */
/* The input is the unpadded [N][C][H][W] tensor: the kernel forms the zero
 * border itself while staging the input in LDS, so no padded copy is made
 * (the pad step fused into the convolution). Stride-1 plans and the dense
 * path only: a layer whose plan (spconv_plan) is SPCONV_KERNEL_GENERIC gets
 * SPCONV_EINVAL. The results are bit-identical to the padded input's. */
#define SPCONV_UNPADDED_INPUT 4u

/*
 * CSR filter (paper, "Sparse Convolution with CSR": flatten (K, C, k, k) to
 * (K, C*k*k), compress the rows). Besides the flattened column the entries carry
 * the paper's input offset, lowered for a padded plane of Hp x Wp:
 *   colidx[j] = c*R*S + r*S + s
 *   offset[j] = c*Hp*Wp + r*Wp + s      (index inside one padded C x Hp x Wp image)
 * Within a row, entries are in increasing colidx order. Pointers are host
 * memory for spconv_pack_csr and device memory for spconv_forward; the struct
 * itself is always a host object.
 */
typedef struct spconv_csr {
    int32_t K, C, R, S; /* filter shape */
    int32_t Hp, Wp;     /* padded plane the offsets were lowered for */
    int64_t nnz;        /* number of entries, < 2^31 */
    const int32_t *rowptr; /* [K+1]; rowptr[0] = 0, non-decreasing, rowptr[K] = nnz */
    const int32_t *colidx; /* [nnz]; not read by spconv_forward (may be NULL there) */
    const int32_t *offset; /* [nnz] */
    const float *vals;     /* [nnz]; the filter values, bit-copied */
} spconv_csr;

/*
 * spconv_pack_csr - host-side CSR packing of a dense-stored sparse filter.
 *
 * w      [K][C][R][S] fp32, host.
 * mask   [K][C][R][S] bytes, host, nullable. With a mask, every position whose
 *        byte is nonzero is an entry (an explicit 0.0 value is kept); without
 *        one, every value that compares unequal to 0.0f is an entry (-0.0 is
 *        dropped, NaN kept).
 * Hp, Wp padded plane the offsets are lowered for; requires Hp >= R, Wp >= S.
 * rowptr [K+1] int32, host, nullable only in the count phase.
 * colidx, offset, vals  [capacity] host arrays. If all three are NULL the call
 *        only counts: *nnz_out receives the number of entries (and rowptr is
 *        filled when given).
 * capacity  length of colidx/offset/vals; if the filter has more entries the
 *        call returns SPCONV_ECAPACITY, sets *nnz_out to the count and writes
 *        nothing else.
 * nnz_out   host, required.
 * Errors: SPCONV_EINVAL for NULL w/nnz_out, non-positive sizes, Hp < R,
 * Wp < S, an offset or entry count that does not fit int32, or a partial set
 * of output arrays.
 */
int spconv_pack_csr(const float *w, const uint8_t *mask, int K, int C, int R, int S, int Hp, int Wp,
                    int32_t *rowptr, int32_t *colidx, int32_t *offset, float *vals, int64_t capacity,
                    int64_t *nnz_out);

/*
 * spconv_pad_input - zero-padded copy of an NCHW tensor (device, asynchronous).
 *
 * The padded input is what the paper's CSR loop indexes with its offsets: it
 * reads in[pixel + offset] with no bounds test, which needs the zero border.
 *   out_padded[n][c][y+pad][x+pad] = in[n][c][y][x], border = +0.0.
 * in          [N][C][H][W] fp32, device.
 * out_padded  [N][C][H+2pad][W+2pad] fp32, device, must not overlap `in`.
 * stream      HIP stream the copy is queued on (0 = the null stream).
 * Errors: SPCONV_EINVAL (NULL pointer, N/C/H/W < 1, pad < 0, a padded plane
 * of 2^31 - 4096 elements or more, element count >= 2^40); SPCONV_EHIP when the
 * launch fails.
 */
int spconv_pad_input(const float *in, int N, int C, int H, int W, int pad, float *out_padded, hipStream_t stream);

/*
 * spconv_resize_pad_input - bilinear resize of an NCHW tensor written straight
 * into the zero-padded layout spconv_forward reads (device, asynchronous).
 *
 * The resize step that precedes the convolution in the Resize-Conv-ReLU-Maxpool
 * block of the paper's evaluation (Evaluation, deep learning benchmarks), done in
 * the same pass as the padding so the block needs no separate pad pass. The
 * paper does not name the interpolation; this is bilinear with pixel centres
 * aligned (align_corners = false): output pixel (y, x) samples the input at
 *   sy = max((y + 1/2) * Hin / H - 1/2, 0),  sx = max((x + 1/2) * Win / W - 1/2, 0)
 * from taps y0 = floor(sy), y1 = min(y0 + 1, Hin - 1) (x likewise) with weights
 * (1 - ty, ty), ty = sy - y0:
 *   out_padded[n][c][y+pad][x+pad] = sum over the 2x2 taps of weight * in[n][c][yi][xi],
 *   border = +0.0.
 * Coordinates are exact integer ratios; the interpolation is fp32 in the form
 * a + t*(b - a), so an axis whose size does not change is copied exactly
 * (H == Hin and W == Win reproduce spconv_pad_input bit for bit).
 * in          [N][C][Hin][Win] fp32, device.
 * out_padded  [N][C][H+2pad][W+2pad] fp32, device, must not overlap `in`.
 * stream      HIP stream the pass is queued on (0 = the null stream).
 * Errors: SPCONV_EINVAL (NULL pointer, N/C/Hin/Win/H/W < 1, pad < 0, a side
 * above 16384, a padded plane of 2^31 elements or more, input or output
 * element count >= 2^40); SPCONV_EHIP when the launch fails.
 */
int spconv_resize_pad_input(const float *in, int N, int C, int Hin, int Win, int H, int W, int pad,
                            float *out_padded, hipStream_t stream);

/*
 * spconv_forward - fused sparse convolution + bias + ReLU + 2x2 max-pool
 * (device, asynchronous, one kernel, one store per output element).
 *
 *   pre[n,k,y,x] = bias[k] + sum_{j in row k} vals[j] *
 *                  in_padded[n*C*Hp*Wp + (y*stride)*Wp + x*stride + offset[j]]
 *   o   = (flags & SPCONV_RELU) ? max(pre, 0) : pre
 *   out = (flags & SPCONV_MAXPOOL2X2) ? max over a,b in {0,1} of o[n,k,2i+a,2j+b] : o
 *
 * in_padded  [N][C][Hp][Wp] fp32, device: the zero-bordered input (as written by
 *            spconv_pad_input); with SPCONV_UNPADDED_INPUT the [N][C][H][W]
 *            input itself.
 * csr        host struct whose arrays are in device memory; csr->K/C/R/S must
 *            equal K/C/R/S and csr->Hp/Wp must equal H+2pad / W+2pad. The array
 *            contents must be a valid CSR as produced by spconv_pack_csr for
 *            these Hp/Wp; they are not re-validated on the device.
 * bias       [K] fp32, device, nullable (zero bias).
 * out        [N][K][Ho][Wo] fp32 (or [N][K][Ho/2][Wo/2] with the pool flag),
 *            device, must not overlap the inputs. Every element is written.
 * stream     HIP stream the kernel is queued on (0 = the null stream).
 * Summation order inside one output is unspecified (fp32 arithmetic; results
 * are reproducible run to run for a given device and shape).
 * Errors: SPCONV_EINVAL (NULL pointer, sizes < 1, stride < 1, pad < 0, shape
 * mismatch with csr, nnz outside [0, 2^31),
 * unknown flag bits, SPCONV_UNPADDED_INPUT with a plan other than the
 * stride-1 kernel, empty output,
 * Ho or Wo < 2 with the pool flag, C*Hp*Wp >= 2^31); SPCONV_EHIP when the
 * launch fails.
 */
int spconv_forward(const float *in_padded, int N, int C, int H, int W, const spconv_csr *csr, int K, int R, int S,
                   int stride, int pad, const float *bias, uint32_t flags, float *out, hipStream_t stream);

/*
 * Options of spconv_forward_ex (and of spconv_plan / spconv_forward_dense):
 * where the fused output goes, what is added before the activation, and a
 * planning hint. A zero-initialised struct (or NULL) gives spconv_forward's
 * behaviour.
 *
 * out_pad   >= 0. The stored output planes carry a border of out_pad zeros:
 *           out is [N][K][Hs+2*out_pad][Ws+2*out_pad] (Hs x Ws the stored plane:
 *           Ho x Wo, or Ho/2 x Wo/2 pooled), the value of (n,k,i,j) at row
 *           i+out_pad, column j+out_pad, and every border element is written
 *           with +0.0 by the same launch. With out_pad equal to the next
 *           layer's pad, out is that layer's in_padded: the zero-padding pass
 *           between chained layers disappears (the paper fuses consecutive
 *           operators, "Evaluation").
 * residual  nullable, device. A tensor on the convolution's own output grid,
 *           added to the pre-activation before ReLU and pooling:
 *             pre[n,k,y,x] += residual[n][k][y+residual_pad][x+residual_pad]
 *           over planes of (Ho+2*residual_pad) x (Wo+2*residual_pad). This is
 *           the shortcut of a ResNet basic block (the paper's ResNet benchmark,
 *           "Evaluation"), read straight from a padded block input when
 *           residual_pad equals that input's pad. Must not overlap out.
 * residual_pad >= 0, ignored without a residual.
 * max_row_nnz  planning hint, 0 = unknown: the largest CSR row's entry count
 *           (rowptr[k+1] - rowptr[k] over k). The CSR arrays live in device
 *           memory and the planner never reads them back (that would need a
 *           synchronous copy inside an asynchronous call), so this is how it
 *           learns that a filter's rows are skewed, where pairing heavy and
 *           light output channels on one wave pays. It only steers the choice
 *           of tiling: results do not depend on it. Must lie in [0, nnz]
 *           (spconv_forward_dense ignores it).
 * lowered  nullable, device: the filter as the entry stream spconv_pack_lowered
 *           writes for this very call (same N, C, H, W, K, R, S, stride, pad,
 *           flags and max_row_nnz), 16-byte aligned. With it the stride-1
 *           kernel reads its entries ready-made, with scalar loads, instead of
 *           decoding the CSR rows itself (same results bit for bit);
 *           csr->offset and csr->vals are then not read. Calls whose plan is
 *           not the stride-1 kernel get SPCONV_EINVAL.
 * lowered_words  number of int32 words of `lowered`; must equal
 *           spconv_lowered_size for the call (SPCONV_EINVAL otherwise).
 * Both borders are limited so that one padded plane has fewer than 2^31
 * elements.
 */
typedef struct spconv_options {
    int32_t out_pad;
    int32_t residual_pad;
    const float *residual;
    int64_t max_row_nnz;
    const int32_t *lowered;
    int64_t lowered_words;
} spconv_options;

/*
 * spconv_forward_ex - spconv_forward with options (device, asynchronous, one
 * kernel, one store per output element including the border).
 *
 *   pre = bias[k] + sum_j vals[j] * in_padded[...]      (as spconv_forward)
 *         + residual[n,k,y,x]                           (opt->residual != NULL)
 *   o   = RELU ? max(pre, 0) : pre;   q = MAXPOOL2X2 ? 2x2 max of o : o
 *   out[n][k][i+out_pad][j+out_pad] = q[n,k,i,j];  border of out = +0.0
 *
 * opt: host struct, nullable (= all zero). Other arguments, layouts and errors
 * as spconv_forward; additionally SPCONV_EINVAL for a negative out_pad or
 * residual_pad, a padded output or residual plane of 2^31 elements or more, or
 * max_row_nnz outside [0, nnz].
 */
int spconv_forward_ex(const float *in_padded, int N, int C, int H, int W, const spconv_csr *csr, int K, int R, int S,
                      int stride, int pad, const float *bias, uint32_t flags, const spconv_options *opt, float *out,
                      hipStream_t stream);

/*
 * Lowered entry stream (host packing). The CSR walk of the paper's "Sparse
 * Convolution with CSR" loop re-bases every entry's offset to the kernel's
 * staged input tile and splits it by tap parity before use; for a fixed layer
 * and launch plan that work is the same on every call, so it can be done once
 * on the host. The stream holds, for each (output-channel tile, wave, row slot,
 * input-channel chunk) of the plan, a header of four int32
 *   {start, n_even, n_odd, k}
 * (k = the output channel of the slot, K for an empty slot; start = index of
 * the slot's first entry of that chunk), followed by every CSR entry once as
 * an int32 pair (LDS index of the pixel pair the tap reads for virtual pixel 0
 * of the chunk, the value's bits), the even-parity taps of a (slot, chunk)
 * before its odd ones, each in CSR order; then 16 zero pairs of padding. With
 * the plan's spconv_plan_info, entry (c, r, s) of the chunk starting at
 * channel c0 = chunk * channels_per_chunk has LDS index t = (c - c0) *
 * lds_channel_floats + r * lds_row_pitch + s + lds_col_shift; its parity is
 * t's, and the stored index is t rounded down to even (the kernel reads the
 * aligned pixel pair there). Headers are ordered by (tile, wave, slot, chunk),
 * entries by (tile, wave, slot, chunk, parity).
 * Its layout is a function of the plan, so it is valid only for the call
 * arguments it was packed for.
 */

/*
 * spconv_lowered_size - int32 words of the lowered stream for a forward call
 * with these arguments (host only; csr's arrays are not read):
 *   4 * tiles * 16 * channels_per_wave * chunks + 2 * (nnz + 16).
 * Errors: those of spconv_forward_ex's argument checks (opt->lowered is not
 * looked at); SPCONV_EINVAL for a NULL words or a plan other than the
 * stride-1 kernel.
 */
int spconv_lowered_size(int N, int C, int H, int W, const spconv_csr *csr, int K, int R, int S, int stride, int pad,
                        uint32_t flags, const spconv_options *opt, int64_t *words);

/*
 * spconv_pack_lowered - write the lowered stream (host). csr's arrays are host
 * memory here: rowptr, colidx and vals are read (offset is not), and checked
 * to be a valid CSR of a (K, C*R*S) matrix (rowptr starts at 0, does not
 * decrease and ends at nnz; colidx strictly increasing within a row and below
 * C*R*S). Output channels are assigned to the (wave, slot) pairs of each
 * channel tile so that the waves' entries are even within every chunk: ranked
 * by entry count and dealt in snake order, then refined by swaps of rows
 * between waves (deterministic); the header's k names each slot's channel.
 * lowered  host array of capacity int32 words; spconv_lowered_size words are
 *          written.
 * Errors: as spconv_lowered_size; SPCONV_EINVAL for a NULL lowered or an
 * invalid CSR; SPCONV_ECAPACITY when capacity is below spconv_lowered_size
 * (nothing written).
 */
int spconv_pack_lowered(int N, int C, int H, int W, const spconv_csr *csr, int K, int R, int S, int stride, int pad,
                        uint32_t flags, const spconv_options *opt, int32_t *lowered, int64_t capacity);

/* Kernel families reported by spconv_plan. */
#define SPCONV_KERNEL_STRIDE1 1 /* stride 1: channel-chunked LDS staging, lanes own padded-width pixels */
#define SPCONV_KERNEL_GENERIC 2 /* any stride */
#define SPCONV_KERNEL_DENSE 3   /* dense filter on the matrix cores (spconv_forward_dense) */
/* spconv_kernel_variants only: the stride-1 tilings also built to run several
 * work items per workgroup with a lowered stream (the launch takes that form
 * when the plan has more work items than launch_workgroups). */
#define SPCONV_KERNEL_STRIDE1_TILED 4

typedef struct spconv_plan_info {
    int32_t kernel;                /* SPCONV_KERNEL_STRIDE1, _GENERIC or _DENSE */
    int32_t pixels_per_lane;       /* virtual output pixels per lane per image; dense: 32-pixel blocks per wave */
    int32_t images_per_group;      /* images sharing one workgroup's tile */
    int32_t channels_per_wave;     /* output channels (CSR rows) per wave; generic kernel: per workgroup */
    int32_t tile_rows;             /* output rows per spatial tile */
    int32_t tiles_per_image;       /* spatial tiles per image */
    int32_t channels_per_chunk;    /* input channels staged in LDS at a time */
    int32_t chunks;                /* LDS chunks per tile */
    int32_t workgroups;            /* work items: (image group, spatial tile, channel tile) */
    int32_t threads_per_workgroup;
    int64_t lds_bytes;             /* dynamic LDS per workgroup */
    /* Stride-1 kernel (0 otherwise): where tap (r, s) of input channel c of a
     * chunk starting at channel c0 sits in the staged tile, as an LDS float
     * index for virtual pixel 0:  (c - c0)*lds_channel_floats + r*lds_row_pitch
     * + s + lds_col_shift. */
    int32_t lds_channel_floats;
    int32_t lds_row_pitch;
    int32_t lds_col_shift;
    /* Grid of the launch: one workgroup per work item, or, for the stride-1
     * kernel with a lowered stream (opt->lowered non-NULL; not read here)
     * on a tiling of SPCONV_KERNEL_STRIDE1_TILED with more than 256 work
     * items, 256 workgroups (one per CU) that take the work items in turn. */
    int32_t launch_workgroups;
    /* Stride-1 kernel with a lowered stream (opt->lowered non-NULL), unpooled,
     * one image per tile: virtual pixels per row-spanning tile. Tile t of an
     * image then covers its virtual pixels [t * tile_pixels, (t+1) *
     * tile_pixels) (pixel y*lds_row_pitch + x), starting in any column, and
     * tile_rows is the most output rows such a tile touches. 0: tiles of
     * tile_rows whole rows. */
    int32_t tile_pixels;
} spconv_plan_info;

/*
 * spconv_plan - the launch plan spconv_forward_ex would use for these arguments
 * (host only, queues nothing). Takes the same arguments as spconv_forward_ex
 * without the buffers and applies the same checks (opt nullable; its
 * max_row_nnz steers the plan, and whether lowered is non-NULL selects the
 * lowered-stream launch, whose tiles may span rows); csr's arrays are not read. Meant for tests,
 * tools and reports that need to know which kernel variant and tiling run.
 * Errors: those of spconv_forward_ex's argument checks; SPCONV_EINVAL for a
 * NULL info.
 */
int spconv_plan(int N, int C, int H, int W, const spconv_csr *csr, int K, int R, int S, int stride, int pad,
                uint32_t flags, const spconv_options *opt, spconv_plan_info *info);

/*
 * spconv_kernel_variants - the compiled instances of one kernel family (host
 * only), for tests and reports that must show every instance the planners can
 * pick has been run. Each instance is a 4-tuple of int32:
 *   SPCONV_KERNEL_STRIDE1  (pixels_per_lane, images_per_group, channels_per_wave, pool)
 *   SPCONV_KERNEL_STRIDE1_TILED  the same tuple, for the tilings built to run
 *                          several work items per workgroup
 *   SPCONV_KERNEL_GENERIC  (pixels_per_lane, 0, channels_per_workgroup, pool)
 *   SPCONV_KERNEL_DENSE    (R, S, pixel blocks per wave, pool)
 * with pool 0 or 1 and the other fields as spconv_plan_info reports them.
 * variants  host array of 4*capacity int32, nullable when capacity is 0; the
 *           first min(count, capacity) tuples are written.
 * count     host, required: receives the number of instances.
 * Errors: SPCONV_EINVAL for an unknown family, a NULL count, a negative
 * capacity, or a NULL variants with capacity > 0.
 */
int spconv_kernel_variants(int32_t kernel, int32_t *variants, int32_t capacity, int32_t *count);

/*
 * Dense path. Above some density, skipping zeros no longer pays: the same
 * fused convolution computed with every filter tap on the matrix cores
 * (fp32 MFMA, so the arithmetic stays fp32 like the sparse path) is faster.
 * The paper reports that its sparse kernels beat the dense ones only below a
 * break-even density (Evaluation, sparse versus dense, on its CPUs); these
 * calls give the same choice on MI355X: spconv_select_path predicts which
 * path is faster for a layer, spconv_forward_dense runs the dense one.
 */
#define SPCONV_PATH_SPARSE 1
#define SPCONV_PATH_DENSE 2

/*
 * spconv_dense_size - floats of the packed dense filter (host):
 *   ceil(C/2) * R * S * Kp * 2,  Kp = K rounded up to a multiple of 32 when
 *   K <= 128, of 128 otherwise.
 * Errors: SPCONV_EINVAL for a NULL floats, sizes < 1, or 2^40 floats or more.
 */
int spconv_dense_size(int K, int C, int R, int S, int64_t *floats);

/*
 * spconv_pack_dense - the filter in the order spconv_forward_dense reads it
 * (host): for channel pair cp = c/2, tap t = r*S + s and output channel k,
 *   packed[((cp*R*S + t)*Kp + k)*2 + c%2] = w[k][c][r][s]
 * for the entries spconv_pack_csr keeps (same mask rule), 0.0 everywhere else
 * (absent entries, k >= K, the pad channel of an odd C).
 * w       [K][C][R][S] fp32, host.   mask  same shape, or NULL (see pack_csr).
 * packed  host array of packed_len floats, written in full.
 * Errors: SPCONV_EINVAL (NULL w/packed, bad sizes); SPCONV_ECAPACITY when
 * packed_len < spconv_dense_size (nothing written).
 */
int spconv_pack_dense(const float *w, const uint8_t *mask, int K, int C, int R, int S, float *packed,
                      int64_t packed_len);

/*
 * spconv_forward_dense - spconv_forward_ex computed from the packed dense
 * filter (device, asynchronous): same padded (or, with SPCONV_UNPADDED_INPUT,
 * unpadded) input, bias, flags, options (max_row_nnz ignored), output layout
 * and ordering; the result is the same convolution up
 * to fp32 summation order. Stride 1 only (the stride is not an argument);
 * filters 3x3 and 1x1.
 * packed  device copy of spconv_pack_dense's output for this K, C, R, S.
 * Errors: SPCONV_EINVAL (NULL in_padded/packed/out, sizes < 1, pad < 0, a
 * filter other than 3x3 or 1x1, unknown flags, pool with Ho or Wo < 2,
 * C*Hp*Wp >= 2^31, a packed filter of 2^31 bytes or more, bad border
 * options as in spconv_forward_ex, or no tiling
 * that fits the kernel: the padded row wider than 255 floats, 127 with pool);
 * SPCONV_EHIP when the launch fails.
 */
int spconv_forward_dense(const float *in_padded, int N, int C, int H, int W, const float *packed, int K, int R, int S,
                         int pad, const float *bias, uint32_t flags, const spconv_options *opt, float *out,
                         hipStream_t stream);

/*
 * spconv_dense_plan - the launch plan spconv_forward_dense would use (host
 * only, same checks). Errors: those of spconv_forward_dense; NULL info.
 */
int spconv_dense_plan(int N, int C, int H, int W, int K, int R, int S, int pad, uint32_t flags,
                      spconv_plan_info *info);

/*
 * spconv_select_path - which path is predicted faster for this layer on
 * MI355X (host only): SPCONV_PATH_DENSE when the dense kernel applies (stride
 * 1, 3x3 or 1x1, a plan exists) and the filter density nnz / (K*C*R*S) is
 * above the break-even density measured on MI355X for the output's size
 * (0.24 at 14x14, 0.43 at 56x56, log-linear in Ho*Wo between and beyond,
 * clamped to [0.2, 0.5]; the paper's CPU figure is 43.5%); otherwise
 * SPCONV_PATH_SPARSE.
 * Errors: SPCONV_EINVAL for a NULL path, sizes < 1, stride < 1, pad < 0, nnz
 * outside [0, K*C*R*S], unknown flags.
 */
int spconv_select_path(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int64_t nnz,
                       uint32_t flags, int *path);

/*
 * spconv_output_shape - stored output plane size for the given layer (host).
 * The convolution's output grid is that of the paper's dense convolution
 * written in its DSL section (an output pixel for every position where the
 * R x S filter fits), taken over the zero-padded input:
 *   Ho = (H + 2*pad - R)/stride + 1,  Wo = (W + 2*pad - S)/stride + 1  (floor);
 * with SPCONV_MAXPOOL2X2 the 2x2, stride-2 max-pool of the Conv-Relu-Maxpool
 * block (Evaluation) halves both, dropping an odd last row/column.
 * Writes *Ho, *Wo (pooled sizes when flags has SPCONV_MAXPOOL2X2).
 * Errors: SPCONV_EINVAL for NULL outputs, H/W/R/S/stride < 1, pad < 0, unknown
 * flags, or an empty (pooled) output.
 */
int spconv_output_shape(int H, int W, int R, int S, int stride, int pad, uint32_t flags, int *Ho, int *Wo);

/*
 * spconv_strerror - static, human-readable text for one of this library's
 * status codes (SPCONV_OK, SPCONV_EINVAL, SPCONV_ECAPACITY, SPCONV_EHIP; any
 * other value gives a generic text). Not an operation of the paper: the
 * status codes are this C ABI's own. Never NULL; the text must not be freed.
 */
const char *spconv_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* SPCONV_H */
