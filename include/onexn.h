/*
 * onexn: 1xN-pruned convolution on AMD Instinct MI355X (gfx950).
 *
 * C ABI of libonexn.so.  Plain pointers and sizes only.
 *
 * The method is 1xN pruning (Lin et al., "1xN Pattern for Pruning
 * Convolutional Neural Networks", arXiv 2105.14713).  A layer's weight W has
 * shape [n][m][kh][kw] (n output channels, m input channels; Sec. 3.1).  Seen
 * as the m x n matrix Omega of kh x kw kernels (Sec. 3.2), each row is cut
 * into G = ceil(n/N) col-groups of N consecutive output kernels; one such
 * 1xN block is the pruning unit.  The last col-group is ragged when N does
 * not divide n: its rows at and beyond n do not exist (they score 0 and are
 * stored as 0).
 *
 * Common conventions
 *   - Weights are OIHW, row-major: w[((j*m + k)*kh + q)*kw + r].
 *   - bf16 values are raw IEEE bfloat16 bit patterns in uint16_t.
 *   - The caller owns every buffer.  No function keeps a pointer after it
 *     returns.  Host functions are re-entrant and thread-safe.
 *   - On error nothing is written to the outputs of host functions, and the
 *     conv call enqueues nothing.  onexn_last_error() gives a message for the
 *     last failure on the calling thread.
 */
#ifndef ONEXN_H
#define ONEXN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    ONEXN_OK = 0,
    ONEXN_ERR_NULL = 1,        /* a required pointer is NULL */
    ONEXN_ERR_ARG = 2,         /* a scalar is out of range, or perm/mask/t are inconsistent */
    ONEXN_ERR_SHAPE = 3,       /* sizes give an empty or overflowing output */
    ONEXN_ERR_DTYPE = 4,       /* unknown dtype, or a dtype combination that is not allowed */
    ONEXN_ERR_UNSUPPORTED = 5, /* valid request this build does not implement */
    ONEXN_ERR_BUFSIZE = 6,     /* an index or size does not fit the int32 BSR arrays */
    ONEXN_ERR_HIP = 7          /* the HIP runtime reported an error */
} onexn_status;

typedef enum { ONEXN_F32 = 0, ONEXN_BF16 = 1 } onexn_dtype;
typedef enum { ONEXN_NCHW = 0, ONEXN_NHWC = 1 } onexn_layout;
typedef enum { ONEXN_ACT_NONE = 0, ONEXN_ACT_RELU = 1, ONEXN_ACT_RELU6 = 2 } onexn_act;

/*
 * Mask building (host, synchronous).
 *
 * Does, in the paper's order:
 *  1. Filter rearrangement (Sec. 3.3, Fig. 2): if `rearrange` is non-zero,
 *     order the filters by decreasing l1 norm sum_{k,q,r} |W[j][k][q][r]|;
 *     equal norms keep ascending original index.  perm[j'] = original index
 *     of the filter at rearranged position j' (identity if rearrange == 0).
 *     The caller applies the same permutation to the next layer's input
 *     channels, W2[:, perm], and to any per-channel parameters of this layer.
 *  2. Block scores (Sec. 3.2, Eq. 4-5): the l1 norm of each 1xN block of the
 *     rearranged weights, summed in fp64 over block rows i < N, then q, r.
 *  3. Per-layer top-(1-p) selection (Eq. 1, the solution of Eq. 5, Sec. 4.1):
 *     of the K = m*G blocks, floor(p*K + 0.5) (clamped to [0, K]) are
 *     pruned; the t = K - pruned blocks with the largest scores are kept,
 *     equal scores keeping the lower row-major index k*G + g.
 *
 * w:     host [n][m][kh][kw] in wdt.
 * N:     block length, 1 <= N; p: pruning rate in [0, 1].
 * perm:  out, host int32[n].
 * mask:  out, host uint8[m][G] (row-major by input channel k): 1 = kept.
 * t:     out, number of kept blocks.
 * Errors: NULL, DTYPE, ARG (non-positive size, N < 1, p not in [0,1]),
 *         BUFSIZE (n*m*kh*kw or m*G beyond 2^31 - 1).
 */
onexn_status onexn_build_mask(const void* w, onexn_dtype wdt, int32_t n, int32_t m, int32_t kh,
                              int32_t kw, int32_t N, double p, int32_t rearrange, int32_t* perm,
                              uint8_t* mask, int64_t* t);

/*
 * Mask building on the GPU (device, asynchronous): the same three steps as
 * onexn_build_mask (Sec. 3.3 filter rearrangement, Sec. 3.2 / Eq. 4-5 block
 * l1 scores, Eq. 1 / Sec. 4.1 per-layer top-(1-p) selection), for weights
 * already on the device.  perm and mask equal onexn_build_mask's bit for bit
 * (the same fp64 sums in the same order and the same tie rules).
 *
 * w_dev:    device [n][m][kh][kw] in wdt.
 * perm_dev: out, device int32[n];  mask_dev: out, device uint8[m][G] (every
 *           byte written).
 * t:        out, HOST int64: the kept count, set before the call returns
 *           (it depends only on m * G and p).
 * workspace_dev, workspace_bytes: device scratch of at least
 *           onexn_mask_workspace_bytes(n, m, N) bytes, 8-byte aligned, owned by
 *           the caller; nothing in it needs initialising, and it must not be
 *           reused until the work enqueued here has finished.
 * stream:   hipStream_t (NULL = the null stream).  Enqueues four kernels and
 *           returns without waiting.
 * Errors:   NULL, DTYPE, ARG (sizes, N < 1, p outside [0, 1], misaligned
 *           workspace), BUFSIZE (too small a workspace, layer beyond int32
 *           indexing), HIP (launch failed).  On an error nothing is enqueued
 *           (a HIP error may leave earlier kernels of the call enqueued).
 *           Unlike the host function, NaN weights are not detected: their
 *           norms order above every number, perm stays a permutation and the
 *           mask keeps exactly t blocks.
 */
size_t onexn_mask_workspace_bytes(int32_t n, int32_t m, int32_t N);
onexn_status onexn_build_mask_dev(const void* w_dev, onexn_dtype wdt, int32_t n, int32_t m,
                                  int32_t kh, int32_t kw, int32_t N, double p, int32_t rearrange,
                                  int32_t* perm_dev, uint8_t* mask_dev, int64_t* t,
                                  void* workspace_dev, size_t workspace_bytes, void* stream);

/*
 * onexn_build_mask_dev without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid hipMalloc).  Same arguments (minus the workspace),
 * results and errors as onexn_build_mask_dev; it allocates nothing.  The
 * workspace is a fixed 8 MiB array in the library that each GPU holds from
 * the library's load until the process ends: layers needing more
 * (onexn_mask_workspace_bytes(n, m, N) > 8 MiB) fail with
 * ONEXN_ERR_BUFSIZE.  Every call on a GPU shares that GPU's array: calls
 * whose work overlaps on one GPU (on different streams, or from several
 * threads without ordering) race on it and give undefined results.
 */
onexn_status onexn_build_mask_dev_noalloc(const void* w_dev, onexn_dtype wdt, int32_t n, int32_t m,
                                          int32_t kh, int32_t kw, int32_t N, double p,
                                          int32_t rearrange, int32_t* perm_dev, uint8_t* mask_dev,
                                          int64_t* t, void* stream);

/*
 * BSR packing (host, synchronous): Sec. 3.4 and Fig. 3.
 *
 * Encodes Omega-bar = rearranged W masked by `mask` (Eq. 6) into
 *   P: int32[G+1]   start of col-group g in D and I; P[0] = 0, P[G] = t
 *                   (0-based; the paper's P is 1-based with last entry t+1);
 *   I: int32[t]     input channel k of each stored block, ascending within
 *                   a col-group;
 *   D: [t][N][kh][kw] in wdt, block z = the kernels of output channels
 *                   gN .. gN+N-1 (rearranged order) for input channel I[z];
 *                   rows at and beyond n are 0.
 * perm and mask are the outputs of onexn_build_mask (any permutation and any
 * 0/1 mask are accepted); t must equal the number of ones in mask.
 * Errors: NULL, DTYPE, ARG (perm not a permutation of 0..n-1, mask entry not
 *         0/1, t inconsistent), BUFSIZE.
 */
onexn_status onexn_pack(const void* w, onexn_dtype wdt, int32_t n, int32_t m, int32_t kh,
                        int32_t kw, int32_t N, const int32_t* perm, const uint8_t* mask,
                        int64_t t, int32_t* P, int32_t* I, void* D);

/*
 * Forward convolution of a 1xN-pruned layer (device, asynchronous).
 *
 * Computes the block-wise decode of Eq. 8, which equals the dense product of
 * Eq. 7 with Omega-bar: for every output pixel and col-group g,
 *   Y[pixel][gN .. gN+N-1] = sum_{z=P[g]}^{P[g+1]-1} X[pixel, I[z]] . D[z]
 * where for a kh x kw kernel X[pixel, c] is the input patch of channel c under
 * the output pixel (stride, zero padding) and "." the patch-kernel inner
 * product.  Output channels are in rearranged order (no un-permute).
 * Accumulation is fp32.
 *
 * P_dev, I_dev, D_dev: device BSR arrays from onexn_pack (G+1, t, t*N*kh*kw
 *         entries).  P is clamped to [0, t] and entries of I outside [0, m)
 *         contribute nothing, so malformed arrays cannot cause out-of-bounds
 *         reads.  With I not ascending within a col-group the result is
 *         unspecified (still no out-of-bounds access).
 * x_dev:  device input [batch][m][H][W] (NCHW) or [batch][H][W][m] (NHWC).
 * y_dev:  device output [batch][n][Ho][Wo] or [batch][Ho][Wo][n] (same layout
 *         as x), Ho = (H + 2*pad_h - kh)/stride_h + 1, likewise Wo.  Every
 *         element is written.  y must not overlap x, P, I or D.
 * dtypes: wdt == xdt (F32 or BF16); ydt == xdt or F32.
 * stream: hipStream_t to enqueue on (NULL = the null stream).  The call
 *         validates its arguments, launches, and returns without waiting.
 * Supported: N in {1, 2, 4, 8, 16, 32}; 1 <= kh, kw <= 16; stride 1..8;
 *         0 <= pad < 16; m*H*W and n*Ho*Wo below 2^31 (per image).
 * Errors: NULL, DTYPE, ARG, SHAPE (Ho or Wo < 1), UNSUPPORTED, HIP (launch
 *         failed).  batch == 0 is a no-op after the checks; x and y may then
 *         be NULL.  Argument errors enqueue nothing.  A layer computed in two
 *         launches (an output fill, then the convolution) that gets HIP from
 *         the second may have left y zeroed.
 */
onexn_status onexn_conv2d_fwd(const int32_t* P_dev, const int32_t* I_dev, const void* D_dev,
                              onexn_dtype wdt, int32_t n, int32_t m, int32_t kh, int32_t kw,
                              int32_t N, int64_t t, const void* x_dev, onexn_dtype xdt,
                              onexn_layout layout, int32_t batch, int32_t H, int32_t W,
                              int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                              void* y_dev, onexn_dtype ydt, void* stream);

/*
 * The same convolution with a fused epilogue in its store stage (device,
 * asynchronous): for output channel o (rearranged order) and every pixel,
 *   y = act(scale[o] * acc + bias[o])
 * computed in fp32 from the fp32 accumulator, then rounded to ydt.  This is
 * the per-channel affine map of a batch norm folded for inference (or a plain
 * bias) followed by ReLU or ReLU6, the layer-to-layer step of the networks
 * the paper prunes (Sec. 4.1).  Sec. 3.3 requires that every per-channel
 * parameter of the layer follows the filter rearrangement: scale and bias are
 * indexed by the rearranged channel, i.e. scale_dev[o] = scale_orig[perm[o]],
 * and the next layer takes its input channels as W2[:, perm]; the network is
 * then unchanged.
 *
 * scale_dev, bias_dev: device fp32[n], or NULL for 1 and 0.  act: ONEXN_ACT_*.
 * Every other argument, the result layout and the errors are those of
 * onexn_conv2d_fwd (plus ARG for an unknown act); with NULL, NULL,
 * ONEXN_ACT_NONE the result equals onexn_conv2d_fwd's bit for bit.  A k x k
 * layer whose output is at most 16 MB may run as the split convolution
 * (fill, convolution) followed by a pass that applies the epilogue to y; a
 * HIP error from that last launch may leave y holding the sums without it.
 */
onexn_status onexn_conv2d_fwd_fused(const int32_t* P_dev, const int32_t* I_dev, const void* D_dev,
                                    onexn_dtype wdt, int32_t n, int32_t m, int32_t kh, int32_t kw,
                                    int32_t N, int64_t t, const void* x_dev, onexn_dtype xdt,
                                    onexn_layout layout, int32_t batch, int32_t H, int32_t W,
                                    int32_t stride_h, int32_t stride_w, int32_t pad_h,
                                    int32_t pad_w, void* y_dev, onexn_dtype ydt,
                                    const float* scale_dev, const float* bias_dev, onexn_act act,
                                    void* stream);

/*
 * Backward of the 1xN-pruned convolution (device, asynchronous), for
 * fine-tuning with the pattern fixed (Sec. 4.1): the pruned weights stay
 * zero, so only the kept blocks' weights get a gradient.  NCHW only.
 *
 * onexn_conv2d_bwd_data: the input gradient, the adjoint of Eq. 7 through
 *   Omega-bar:  dX[b][c][ih][iw] = sum over kept blocks z with I[z] = c, rows i
 *   and taps (q, r) landing on (ih, iw) of D[z][i][q][r] * dY[b][gN+i][oh][ow].
 *   dy_dev [batch][n][Ho][Wo] (rearranged channel order, as the forward's y)
 *   in dydt == wdt; dx_dev [batch][m][H][W] in dxdt (dydt or F32).  Every dx
 *   element is written.  Layers with more than 2048 col-groups: UNSUPPORTED.
 * onexn_conv2d_bwd_weight: the gradient of the kept blocks in D's layout,
 *   dD[z][i][q][r] = sum_{b,oh,ow} dY[b][gN+i][oh][ow] * X[b][I[z]][oh*sh-ph+q][ow*sw-pw+r],
 *   fp32 [t][N][kh][kw] (rows gN+i >= n get 0); x_dev [batch][m][H][W] and
 *   dy_dev in xdt (F32 or BF16).
 * Both accumulate in fp32.  The input gradient, and the weight gradient of
 * every layer except those below, sum in a fixed order (results do not vary
 * run to run).  For fp32 layers at N = 16 or 32 with few tiles of (kept
 * block, tap) pairs, and fp32 layers at N = 2, 4, 8 with few (32 x 32
 * channel tile, tap) items (fewer than four workgroups per CU), the
 * weight gradient
 * splits the pixels over workgroups and adds their sums with atomics into the
 * zeroed dD, so the last bits can vary run to run; setting the tuning
 * "bwd_split" to 1 makes it one range per item (fixed order, slower).  Such
 * a call launches a fill of dD first: a HIP error from its second launch may
 * leave dD zeroed.  The input gradient of a stride-2 3x3 fp32 layer at
 * N = 16/32 is four launches, one per parity class of input pixels: a HIP
 * error from a later one leaves the earlier classes' dx entries written.
 * Arguments, ownership, the int32 size limits and the errors are those of
 * onexn_conv2d_fwd; P, I, D are the forward's BSR arrays.
 */
onexn_status onexn_conv2d_bwd_data(const int32_t* P_dev, const int32_t* I_dev, const void* D_dev,
                                   onexn_dtype wdt, int32_t n, int32_t m, int32_t kh, int32_t kw,
                                   int32_t N, int64_t t, const void* dy_dev, onexn_dtype dydt,
                                   int32_t batch, int32_t H, int32_t W, int32_t stride_h,
                                   int32_t stride_w, int32_t pad_h, int32_t pad_w, void* dx_dev,
                                   onexn_dtype dxdt, void* stream);
onexn_status onexn_conv2d_bwd_weight(const int32_t* P_dev, const int32_t* I_dev, int32_t n, int32_t m,
                                     int32_t kh, int32_t kw, int32_t N, int64_t t, const void* x_dev,
                                     onexn_dtype xdt, const void* dy_dev, int32_t batch, int32_t H,
                                     int32_t W, int32_t stride_h, int32_t stride_w, int32_t pad_h,
                                     int32_t pad_w, float* dD_dev, void* stream);

/*
 * Fully connected layer (device, asynchronous): Sec. 3.1 treats an FC layer
 * as the kh = kw = 1 case, so its weight [n][m] is packed like a 1x1 conv
 * (onexn_build_mask / onexn_pack with kh = kw = 1) and
 *   Y[b][gN .. gN+N-1] = sum_{z=P[g]}^{P[g+1]-1} X[b][I[z]] * D[z]   (Eq. 8)
 * for every sample b and col-group g; output features in rearranged order.
 *
 * layout: ONEXN_NHWC: x_dev is [batch][m] (one row per sample), y_dev
 *         [batch][n];  ONEXN_NCHW: x_dev is [m][batch] (one row per feature,
 *         the samples contiguous), y_dev [n][batch] -- the layout in which
 *         every gathered row is read with coalesced loads.
 * D_dev: [t][N] (the [t][N][1][1] of onexn_pack).  scale_dev, bias_dev, act:
 *         the fused epilogue of onexn_conv2d_fwd_fused (NULL, NULL,
 *         ONEXN_ACT_NONE for none).  dtypes, errors and ownership as for the
 *         convolution.
 */
onexn_status onexn_fc_fwd(const int32_t* P_dev, const int32_t* I_dev, const void* D_dev,
                          onexn_dtype wdt, int32_t n, int32_t m, int32_t N, int64_t t,
                          const void* x_dev, onexn_dtype xdt, onexn_layout layout, int32_t batch,
                          void* y_dev, onexn_dtype ydt, const float* scale_dev,
                          const float* bias_dev, onexn_act act, void* stream);

/*
 * Kernel-choice and launch-shape overrides (host, process-wide).
 *
 * Not part of the method: these let a caller reach a particular kernel variant
 * (tests of every variant's parity) or compare variants (A/B timing).  The
 * library never reads the environment; until a name is set, and after it is
 * set to -1, the dispatch rules decide.  Names and values:
 *   "kernel"      1: generic gather kernels for every layer
 *   "pw_kernel"   1x1 fp32 N = 16/32: 1 resident tile, 3 register operands
 *   "pwb_kernel"  1x1 bf16 N = 32: 1 register-gathered, 2 LDS-staged
 *   "bwd_kernel"  backward: 1 general kernels for every layer, 2 the stride-2
 *                 3x3 input gradient with all nine taps per pixel (instead of
 *                 one launch per parity class of input pixels), 3 the 1x1
 *                 weight gradient staged one pixel per access (instead of
 *                 16-byte pixel quads)
 *   "pw_wgs", "pwb_gp", "pwb_rp", "pwb_wgs", "direct_kdb", "direct_tile",
 *   "fma_tpw", "fma_no_v4", "fma_tile", "kxk_split", "kxk_tp", "kxkf_split",
 *   "nhwc_tile", "bwd_split":
 *                 tile shapes, workgroup counts and pipeline depths of the
 *                 kernel families (a value the family cannot use falls back to
 *                 its default, or makes the conv call fail with UNSUPPORTED).
 * The setting applies to conv calls that start after it returns; changing it
 * while another thread is inside onexn_conv2d_fwd gives that call either value.
 * Errors: NULL, ARG (unknown name, value < -1).
 */
onexn_status onexn_set_tuning(const char* name, int32_t value);

/* Static name of a status code ("ONEXN_OK", ...); "ONEXN_UNKNOWN" otherwise. */
const char* onexn_status_string(onexn_status s);

/* Message describing the last error on the calling thread ("" if none).
 * The pointer stays valid until the next onexn call on the same thread. */
const char* onexn_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ONEXN_H */
