/*
 * ifq.h -- C ABI of the integrated fixed-point quantized convolution library
 * for AMD Instinct MI355X (gfx950).
 *
 * The library implements one "quantized substructure" of IFQ-Net
 * (Integrated Fixed-point Quantization Networks for Embedded Vision):
 *
 *   a    = W_b (x) X_q                       integer part of Eq. (1):
 *                                            +-1 weights convolved with k-bit
 *                                            activation codes, int32 sums
 *   code = #{ i : s*a > T_i }                Eq. (7)/(8): the float data of
 *                                            conv, BN (Eq. 2) and quantizer
 *                                            (Eq. 3) composed into per-channel
 *                                            integer thresholds (Sec. 3.2)
 *   y    = max over a window of codes        Eq. (4), applied to the codes
 *
 * Conventions shared by every entry point:
 *  - Status codes are ifq_status values; IFQ_OK is 0. INVALID_ARGUMENT,
 *    UNSUPPORTED and INSUFFICIENT_BUFFER are decided before any launch, so
 *    nothing has been launched and no output written; IFQ_ERR_HIP reports a
 *    failed launch (for a stack, earlier layers may have been launched). A
 *    text for the last error of the calling thread is in ifq_last_error().
 *  - Every argument is validated on the host before any launch. Device faults
 *    and kernel errors surface at the caller's next synchronisation.
 *  - Device functions are asynchronous on the caller's stream. The caller owns
 *    all memory (device and host); the library never allocates device memory
 *    and keeps no state between calls beyond its loaded code object.
 *  - Tensors are dense. Codes are unsigned: layout IFQ_LAYOUT_I8_NHWC
 *    stores one code per byte; IFQ_LAYOUT_U2_NHWC_PACKED stores four 2-bit
 *    codes per byte along C (channel c in bits 2*(c%4)..2*(c%4)+1 of byte
 *    c/4; C must be a multiple of 4); IFQ_LAYOUT_U2_BLOCK64 stores 2-bit
 *    codes in channel blocks of 64: the tensor is [n][c/64][h][w] cells of
 *    16 bytes, each cell holding channels 64b .. 64b+63 of one pixel packed
 *    as in IFQ_LAYOUT_U2_NHWC_PACKED (C must be a multiple of 64). In that
 *    layout the 64 channels of one filter tap for a run of consecutive
 *    output pixels are one contiguous span, so the convolution's gathers
 *    are contiguous loads. IFQ_LAYOUT_I32_NHWC holds int32 sums.
 *  - No C++ exception crosses this interface. All functions are reentrant.
 */
#ifndef IFQ_H_
#define IFQ_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define IFQ_API __attribute__((visibility("default")))

typedef int32_t ifq_status;

#define IFQ_OK 0
#define IFQ_ERR_INVALID_ARGUMENT (-1)   /* a value is out of its domain     */
#define IFQ_ERR_UNSUPPORTED (-2)        /* valid but not implemented combo  */
#define IFQ_ERR_HIP (-3)                /* a HIP launch or query failed     */
#define IFQ_ERR_INSUFFICIENT_BUFFER (-4)/* a caller buffer is too small     */

#define IFQ_LAYOUT_I8_NHWC 0
#define IFQ_LAYOUT_U2_NHWC_PACKED 1
#define IFQ_LAYOUT_I32_NHWC 2
#define IFQ_LAYOUT_U2_BLOCK64 3

#define IFQ_POOL_VALID 0 /* ho = (h-k)/stride + 1, windows fully inside       */
#define IFQ_POOL_SAME 1  /* ho = ceil(h/stride), windows clipped bottom/right */

#define IFQ_JOIN_NONE 0
#define IFQ_JOIN_IDENTITY 1 /* shortcut = the block input codes             */
#define IFQ_JOIN_CONV 2     /* shortcut = int32 sums of a 1x1 downsample conv */
#define IFQ_JOIN_CONV_FUSED 3 /* shortcut = the downsample's input codes; the
                                 1x1 downsample conv runs inside this conv  */

#define IFQ_LAYER_CONV 0
#define IFQ_LAYER_POOL 1
#define IFQ_LAYER_CONV_POOL 2 /* conv with its max-pool fused (see ifq_conv_pool_forward) */
#define IFQ_LAYER_CONV_FP4 3  /* conv on the fp4 path (see ifq_conv_forward_fp4) */
#define IFQ_LAYER_CONV_POOL_FP4 4 /* CONV_POOL on the fp4 path (ifq_conv_pool_forward_fp4) */

#define IFQ_MAX_THRESHOLDS 15 /* 2^4 - 1: codes of up to 4 bits */

/*
 * One quantized convolution (Eq. 1 with the epilogue of Eq. 7/8).
 *   n, h, w        batch and input spatial size
 *   c_in, c_out    channels
 *   kh, kw         filter size; stride and pad apply to both axes, the
 *                  padded input positions hold code 0 (the level 0 is the
 *                  real value 0)
 *   in_bits        bits per input code, 1..8 (codes 0 .. 2^in_bits - 1)
 *   out_bits       0: the output is the int32 sum a itself (no quantizer);
 *                  1..4: the output is a code with 2^out_bits - 1 thresholds
 *   in_layout      IFQ_LAYOUT_I8_NHWC; or, when in_bits == 2,
 *                  IFQ_LAYOUT_U2_NHWC_PACKED (c_in % 16 == 0) or
 *                  IFQ_LAYOUT_U2_BLOCK64 (c_in % 64 == 0)
 *   out_layout     IFQ_LAYOUT_I32_NHWC iff out_bits == 0; otherwise
 *                  IFQ_LAYOUT_I8_NHWC, or when out_bits == 2
 *                  IFQ_LAYOUT_U2_NHWC_PACKED (c_out % 4 == 0) or
 *                  IFQ_LAYOUT_U2_BLOCK64 (c_out % 64 == 0)
 * Output size: ho = (h + 2*pad - kh)/stride + 1, wo likewise.
 */
typedef struct ifq_conv_desc {
  int32_t n, h, w;
  int32_t c_in, c_out;
  int32_t kh, kw, stride, pad;
  int32_t in_bits, out_bits;
  int32_t in_layout, out_layout;
} ifq_conv_desc;

/*
 * Parameters of the threshold fold of one layer (Sec. 3.2, Eq. 6 -> Eq. 7).
 * All arrays are host arrays of c_out doubles; nullable ones take the default
 * in brackets.
 *   alpha[c] > 0     scale of filter c (W = alpha * W_b, Eq. 1)
 *   beta_in > 0      step of the input codes (X = beta * X_q, Eq. 1)
 *   bias    [0]      conv bias b (Eq. 1)
 *   mean    [0], var [1], gamma [1], bn_beta [0], eps
 *                    batch normalisation Y_bn = gamma*(Y - mean)/sqrt(var+eps)
 *                    + bn_beta (Eq. 2 with its scale read as the standard
 *                    deviation and the affine scale/shift included)
 *   q_thr[i]         the 2^out_bits - 1 quantizer thresholds of Eq. (3),
 *                    strictly increasing (equality goes to the lower code)
 *   k                contraction length kh*kw*c_in; with in_bits it bounds the
 *                    sums: |a| <= B = k * (2^in_bits - 1)
 */
typedef struct ifq_fold_params {
  int32_t c_out;
  int32_t in_bits;
  int32_t out_bits;
  int32_t reserved;
  int64_t k;
  const double* alpha;
  double beta_in;
  const double* bias;
  const double* mean;
  const double* var;
  const double* gamma;
  const double* bn_beta;
  double eps;
  const double* q_thr;
} ifq_fold_params;

/*
 * Residual join of a basic block (not part of the paper; used by the
 * ResNet-shaped stack). The quantizer input is the main branch after its BN
 * plus the dequantized shortcut:
 *   z = gamma*(alpha*beta_in*a + bias - mean)/sqrt(var+eps) + bn_beta + sc
 *   sc = beta_x * x_q                                   (IFQ_JOIN_IDENTITY)
 *   sc = gamma_d*(alpha_d*beta_x*d + bias_d - mean_d)/sqrt(var_d+eps_d)
 *        + bn_beta_d                                    (IFQ_JOIN_CONV)
 * with a the block's conv2 sum, x_q the block input code and d the 1x1
 * downsample sum. ifq_fold_join writes per channel {p, q, cc} such that
 * z = fma(p, a, fma(q, s, cc)) with s = x_q or d. Nullable: bias, bias_d
 * [0]. The _d arrays are ignored for IFQ_JOIN_IDENTITY.
 */
typedef struct ifq_join_params {
  int32_t c_out;
  int32_t kind;
  const double* alpha;
  double beta_in;
  const double* bias;
  const double* mean;
  const double* var;
  const double* gamma;
  const double* bn_beta;
  double eps;
  double beta_x;
  const double* alpha_d;
  const double* bias_d;
  const double* mean_d;
  const double* var_d;
  const double* gamma_d;
  const double* bn_beta_d;
  double eps_d;
} ifq_join_params;

/*
 * Device-side join operand of ifq_conv_forward.
 *   kind      IFQ_JOIN_NONE, IFQ_JOIN_IDENTITY, IFQ_JOIN_CONV or
 *             IFQ_JOIN_CONV_FUSED
 *   layout    layout of shortcut: codes (I8, U2 or BLOCK64) for IDENTITY,
 *             I32 for CONV, BLOCK64 codes for CONV_FUSED
 *   shortcut  IDENTITY, CONV: device tensor [n][ho][wo][c_out] (block input
 *             codes, or the downsample conv's int32 sums d);
 *             CONV_FUSED: the downsample conv's input codes, of shape
 *             down.{n, h, w, c_in}
 *   coef      IFQ_JOIN_CONV / CONV_FUSED: device array [c_out][3] written by
 *             ifq_fold_join (NULL for IDENTITY)
 *   table     IFQ_JOIN_IDENTITY: device array [c_out][4][2^out_bits]
 *             written by ifq_fold_join_table with x_bits = 2 (the shortcut
 *             codes are 2-bit; NULL for CONV)
 *   n_q       number of quantizer thresholds, 2^out_bits - 1
 *   sc_bits   IFQ_JOIN_IDENTITY: bit width of the shortcut codes, 0 meaning
 *             2. Only 2-bit shortcut codes are supported (the table holds 4
 *             shortcut levels and the kernels read 2 bits per code): any
 *             other width returns IFQ_ERR_UNSUPPORTED. With an I8_NHWC
 *             shortcut every code must be below 4; larger values are not
 *             detected on the device. In a stack, a shortcut slot written
 *             by a layer whose out_bits is not 2 is rejected the same way.
 *             Ignored for the other kinds.
 *   q_thr     the quantizer thresholds of Eq. (3), strictly increasing
 *   down_w, down
 *             IFQ_JOIN_CONV_FUSED only (else ignored): the downsample conv's
 *             packed weights (ifq_pack_weights of down) and its descriptor:
 *             1x1, pad 0, 2-bit BLOCK64 input, int32 output (out_bits 0),
 *             c_out and output size equal to the conv's. Its sums d are
 *             computed inside the conv's kernel and never stored, so the
 *             join reads neither d nor anything from an extra launch. It
 *             needs a 3x3 pad-1 conv with 2-bit BLOCK64 input and output;
 *             shapes the kernel does not cover return IFQ_ERR_UNSUPPORTED.
 */
typedef struct ifq_join {
  int32_t kind;
  int32_t layout;
  const void* shortcut;
  const double* coef;
  const int32_t* table;
  int32_t n_q;
  int32_t sc_bits;
  double q_thr[IFQ_MAX_THRESHOLDS];
  const void* down_w;
  ifq_conv_desc down;
} ifq_join;

/*
 * Integer max-pool on codes (Eq. 4 applied after the quantizer; for channels
 * with a positive BN scale this equals pooling the conv output first).
 *   n, h, w, c     input tensor; bits: code width; layout I8, or U2 or
 *                  BLOCK64 (bits 2); the output has the same layout
 *   k, stride      square window; mode IFQ_POOL_VALID or IFQ_POOL_SAME
 */
typedef struct ifq_pool_desc {
  int32_t n, h, w, c;
  int32_t k, stride;
  int32_t mode;
  int32_t bits;
  int32_t layout;
} ifq_pool_desc;

/*
 * One layer of a stack (Sec. 3.1: a network is a chain of substructures).
 *   kind        IFQ_LAYER_CONV, IFQ_LAYER_POOL, IFQ_LAYER_CONV_POOL (conv
 *               without join whose codes go through pool before dst; its
 *               pool desc describes the conv's output as for
 *               ifq_conv_pool_forward), IFQ_LAYER_CONV_FP4 (conv on the fp4
 *               path; w_packed is its ifq_pack_weights_fp4 blob, a fused
 *               join's down_w the down conv's) or IFQ_LAYER_CONV_POOL_FP4
 *               (CONV_POOL on the fp4 path)
 *   src, dst    tensor slots: 0 is the stack input x, 1 the stack output y,
 *               2 .. n_slots-1 live in the caller's workspace
 *   join_src    slot of the join shortcut (conv layers with join.kind != 0),
 *               else -1; join.shortcut is ignored inside a stack
 *   conv        shape of a conv layer; w_packed/thr as for ifq_conv_forward
 *   pool        shape of a pool layer, or the fused pool of a CONV_POOL layer
 */
typedef struct ifq_layer {
  int32_t kind;
  int32_t src;
  int32_t dst;
  int32_t join_src;
  ifq_conv_desc conv;
  const void* w_packed;
  const int32_t* thr;
  ifq_join join;
  ifq_pool_desc pool;
} ifq_layer;

/*
 * A layer chain run on one stream.
 *   events   optional array of n_layers + 1 HIP events; when non-null,
 *            events[i] is recorded before layer i and events[n_layers] after
 *            the last layer (per-layer timing)
 */
typedef struct ifq_stack {
  int32_t n_layers;
  int32_t n_slots;
  const ifq_layer* layers;
  hipEvent_t* events;
} ifq_stack;

/* Library version string, e.g. "ifq 1.0.0 gfx950". Host. */
IFQ_API const char* ifq_version(void);

/* Text of the last non-OK status of the calling thread ("" if none). Host. */
IFQ_API const char* ifq_last_error(void);

/* Bytes of a dense NHWC tensor in the given layout (0 if invalid). Host. */
IFQ_API size_t ifq_tensor_bytes(int64_t n, int64_t h, int64_t w, int64_t c,
                                int32_t layout);

/*
 * Output spatial size of a conv descriptor (Eq. 1 with stride and zero
 * padding). Host. Returns IFQ_ERR_INVALID_ARGUMENT for an invalid desc.
 */
IFQ_API ifq_status ifq_conv_output_dims(const ifq_conv_desc* d, int32_t* ho,
                                        int32_t* wo);

/*
 * Bytes of the device-ready weight blob of a layer (W_b of Eq. 1 as +-1
 * int8 rows plus per-row sums), 0 for an invalid desc. Host.
 */
IFQ_API size_t ifq_packed_weight_bytes(const ifq_conv_desc* d);

/*
 * Pack the binary filters W_b of Eq. (1) for the device. Host only.
 *   w_oihw     host int8 [c_out][c_in][kh][kw], every value +1 or -1
 *              (alpha is not part of it: it is folded into the thresholds)
 *   dst        host buffer of at least ifq_packed_weight_bytes(d) bytes; the
 *              caller uploads it unchanged and passes it as w_packed
 * Errors: INVALID_ARGUMENT (bad desc, a value other than +-1; dst untouched),
 * INSUFFICIENT_BUFFER.
 */
IFQ_API ifq_status ifq_pack_weights(const ifq_conv_desc* d,
                                    const int8_t* w_oihw, void* dst,
                                    size_t dst_bytes);

/*
 * Threshold fold of Sec. 3.2 (Eq. 6 -> Eq. 7 -> floor; Eq. 8 for k bits).
 * Host only. For channel c it writes the record
 *   thr_out[c*R + 0]      s = +1, or -1 when gamma < 0 (the division by the
 *                         negative BN scale flips every inequality)
 *   thr_out[c*R + i]      T_i = clamp(floor(s * t_i), -B-1, B), i = 1..R-1
 * with R = 2^out_bits and t_i = ((q_i - bn_beta)*sd/gamma + mean - bias) /
 * (alpha*beta_in), sd = sqrt(var+eps), evaluated in fp64 in exactly that
 * order. For every integer a, #{i : s*a > T_i} is the code Eq. (3) assigns to
 * BN(alpha*beta_in*a + bias). gamma == 0 gives the constant code
 * #{i : bn_beta > q_i}. thr_out holds c_out * 2^out_bits int32 (host).
 * Errors: INVALID_ARGUMENT (alpha <= 0, beta_in <= 0, var+eps <= 0, NaN,
 * q_thr not strictly increasing, out_bits outside 1..4, in_bits outside 1..8).
 */
IFQ_API ifq_status ifq_fold_thresholds(const ifq_fold_params* p,
                                       int32_t* thr_out);

/*
 * Compact thresholds of a uniform quantizer (Sec. 3.2, Eq. 8): with
 * q_i = i*base + offset for i = 1 .. 2^out_bits - 1, the moved thresholds of
 * a channel are t_i = i*base' + offset', so one record per channel serves
 * every bit width. In fp64, in exactly this order (sd = sqrt(var + eps),
 * ab = alpha*beta_in):
 *   base'   = ((base * sd) / gamma) / ab
 *   offset' = ((((offset - bn_beta) * sd) / gamma + mean) - bias) / ab
 *   s       = +1 (gamma > 0), -1 (gamma < 0), or 0 (gamma == 0: every code is
 *             cstar = #{i : bn_beta > i*base + offset})
 */
typedef struct ifq_thr_compact {
  double base;
  double offset;
  int32_t s;
  int32_t cstar;
} ifq_thr_compact;

/*
 * Fold one layer into compact records (host). p as for ifq_fold_thresholds,
 * except that p->q_thr is not read: base > 0 and offset define the
 * quantizer. out: host array of p->c_out records.
 * Errors: INVALID_ARGUMENT as ifq_fold_thresholds, and base <= 0 or a
 * non-finite base or offset.
 */
IFQ_API ifq_status ifq_fold_thresholds_compact(const ifq_fold_params* p, double base,
                                               double offset, ifq_thr_compact* out);

/*
 * Expand compact records into the records ifq_conv_forward takes (Eq. 8 with
 * a floor per threshold; the floor of i*base' + offset' is not affine in i,
 * so it is taken for each i). Asynchronous on stream, device memory:
 *   recs   c_out records (ifq_fold_thresholds_compact)
 *   thr    c_out * 2^out_bits int32: {s, T_1 .. T_{R-1}} per channel with
 *          T_i = clamp(floor(s * (i*base' + offset')), -B-1, B), the product
 *          i*base' rounded before the sum; s = 0 becomes s = +1 with
 *          T_i = -B-1 for i <= cstar and B above, B = k*(2^in_bits - 1)
 * Errors: INVALID_ARGUMENT (NULL, c_out < 1, bits or k out of range), HIP.
 */
IFQ_API ifq_status ifq_expand_thresholds(const ifq_thr_compact* recs, int32_t c_out,
                                         int32_t in_bits, int64_t k, int32_t out_bits,
                                         int32_t* thr, hipStream_t stream);

/*
 * Join coefficients (see ifq_join_params), fp64 in this order:
 *   p  = (gamma * (alpha*beta_in)) / sd
 *   c2 = (gamma * (bias - mean)) / sd + bn_beta
 *   q  = beta_x (identity) or (gamma_d * (alpha_d*beta_x)) / sd_d
 *   cd = 0 (identity) or (gamma_d * (bias_d - mean_d)) / sd_d + bn_beta_d
 *   coef_out[c*3 + 0..2] = {p, q, c2 + cd}
 * Host only. Errors: INVALID_ARGUMENT (bad kind, alpha <= 0, var+eps <= 0,
 * NaN, beta <= 0).
 */
IFQ_API ifq_status ifq_fold_join(const ifq_join_params* p, double* coef_out);

/*
 * Integer thresholds of an identity join (the idea of Eq. 6 -> 7 applied to
 * the join: the fixed-point test moves onto the integer sum). For channel c
 * and shortcut code x in 0 .. X-1 (X = 2^x_bits) the record
 *   table_out[(c*X + x)*R + 0]   s = +1, or -1 when the join's p < 0
 *   table_out[(c*X + x)*R + i]   T_i, i = 1 .. R-1     (R = 2^out_bits)
 * satisfies, for every integer a with |a| <= B = k * (2^in_bits - 1),
 *   #{i : s*a > T_i} == #{i : fma(p, a, fma(q, x, cc)) > q_thr[i-1]}
 * with {p, q, cc} of ifq_fold_join (p->kind must be IFQ_JOIN_IDENTITY) and
 * the fma evaluated in fp64. fma is correctly rounded, so the left side of
 * each comparison is monotone in a and every T_i is found by bisection of
 * that predicate; the table is exact, not an approximation. p == 0 gives a
 * constant code. Host only; table_out holds c_out * X * R int32.
 * Errors: INVALID_ARGUMENT (as ifq_fold_join, bad bits, k < 1, q_thr not
 * strictly increasing).
 */
IFQ_API ifq_status ifq_fold_join_table(const ifq_join_params* p, int32_t in_bits,
                                       int64_t k, int32_t x_bits, int32_t out_bits,
                                       const double* q_thr, int32_t* table_out);

/*
 * Name of the kernel variant ifq_conv_forward launches for d with join
 * (nullable: no join; only its kind and descriptors are read, no pointer is
 * dereferenced), as a static string: the kernel's symbol as a profiler lists
 * it, or "" for an invalid desc or one with no output pixels (nothing is
 * launched). Host; for profiling and benchmarks.
 */
IFQ_API const char* ifq_conv_kernel_name(const ifq_conv_desc* d, const ifq_join* join);

/*
 * Kernel variants of the register-blocked 3x3 conv kernels, for autotuning
 * and per-variant parity tests (the same contraction, Eq. 1, and the same
 * epilogues as ifq_conv_forward): conv_w2 (one output tile per workgroup),
 * conv_wp (persistent: a workgroup keeps the weights of its 64 output
 * channels in LDS and runs a range of pixel tiles) and conv_wv (persistent
 * with the weights in LDS too, but each wave runs its own range of pixels
 * with its own input windows and no barrier after the prologue; c_out %
 * 64 == 0; conv_wvh the same with 32 output channels per workgroup, for
 * weights of up to 256 input channels in its slab). All take 3x3 pad-1 convs of stride 1 or 2 on 2-bit BLOCK64
 * codes with c_in % 64 == 0, 2-bit output (U2 or BLOCK64, c_out % 32 == 0,
 * 27 * c_in <= 32766), no pool, and thresholds or an identity join with a
 * 2-bit shortcut (c_out % 64 == 0); conv_w2 also a join with a fused 1x1
 * downsample on BLOCK64 codes of at most 256 channels. Each variant further
 * needs its weights and input windows to fit its LDS budget.
 *   ifq_conv_variant_count   number of variants (host)
 *   ifq_conv_variant_fp4     1 if variant computes the sums exactly on the
 *                            fp4 scaled MFMA, as ifq_conv_forward_fp4 (its
 *                            w_packed, and a fused join's down_w, are then
 *                            ifq_pack_weights_fp4 blobs), 0 if on the int8
 *                            MFMA, -1 if variant is out of range (host)
 *   ifq_conv_variant_name    the kernel variant `variant` would launch for
 *                            d and join (join nullable; no pointer in it is
 *                            dereferenced), or "" if it cannot take the
 *                            layer or d has no pixels (host)
 *   ifq_conv_forward_variant ifq_conv_forward (same arguments, no
 *                            workspace) on that variant, asynchronous on
 *                            stream; IFQ_ERR_UNSUPPORTED where it cannot
 *                            take the layer. Errors as ifq_conv_forward.
 */
IFQ_API int32_t ifq_conv_variant_count(void);
IFQ_API int32_t ifq_conv_variant_fp4(int32_t variant);
IFQ_API const char* ifq_conv_variant_name(const ifq_conv_desc* d, const ifq_join* join,
                                          int32_t variant);
IFQ_API ifq_status ifq_conv_forward_variant(const ifq_conv_desc* d, const void* x,
                                            const void* w_packed, const int32_t* thr,
                                            const ifq_join* join, void* y, int32_t* acc_dump,
                                            int32_t variant, hipStream_t stream);

/*
 * The contraction of Eq. (1) split over K across workgroups, on one int8
 * variant of the register-blocked kernel (conv_w2, variants below
 * ifq_conv_variant_count() - 2 with ifq_conv_variant_fp4 0), for tests and
 * tuning: ksplit workgroups per output tile, each over c_in/64/ksplit of the
 * channel blocks, their int32 partial tiles added by the last to arrive,
 * which runs the threshold epilogue (Eq. 7/8; no join). ifq_conv_forward
 * takes such a split where its planner predicts one faster.
 *   ifq_conv_split_workspace_bytes  workspace bytes of that launch, or 0 if
 *                                   the variant cannot take the layer with
 *                                   that split (ksplit 2 or 4 dividing the
 *                                   variant's K groups into c_in/64) (host)
 *   ifq_conv_forward_split          the launch, asynchronous on stream; ws
 *                                   as for ifq_conv_forward (zero-filled
 *                                   before its first use). Errors:
 *                                   UNSUPPORTED where the variant cannot take
 *                                   the layer with that split, else as
 *                                   ifq_conv_forward.
 */
IFQ_API size_t ifq_conv_split_workspace_bytes(const ifq_conv_desc* d, int32_t variant,
                                              int32_t ksplit);
IFQ_API ifq_status ifq_conv_forward_split(const ifq_conv_desc* d, const void* x,
                                          const void* w_packed, const int32_t* thr, void* y,
                                          int32_t* acc_dump, int32_t variant, int32_t ksplit,
                                          void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Device workspace bytes ifq_conv_forward needs for d (may be 0). Host.
 * Non-zero where the planner splits the contraction of Eq. (1) over K
 * across workgroups (3x3 layers with the threshold epilogue that fill too
 * few workgroups): the workspace holds one int32 partial tile per split and
 * tile, and at its start a 64 KiB region of per-tile arrival counters. That
 * region must be zero before the workspace's first use (hipMemset once);
 * every call leaves it zero again, so a workspace serves any number of
 * calls (on one stream at a time). The sums stay exact: integer addition
 * is associative.
 */
IFQ_API size_t ifq_conv_workspace_bytes(const ifq_conv_desc* d);

/*
 * One quantized substructure on the GPU, asynchronous on stream.
 *   x          device input [n][h][w][c_in] in d->in_layout
 *   w_packed   device copy of ifq_pack_weights(d, ...), 16-byte aligned
 *   thr        device copy of ifq_fold_thresholds(...) for this layer,
 *              16-byte aligned; must be NULL iff out_bits == 0 or
 *              join->kind != IFQ_JOIN_NONE
 *   join       nullable; residual join in place of the thresholds
 *   y          device output [n][ho][wo][c_out] in d->out_layout
 *   acc_dump   nullable device int32 [n][ho][wo][c_out]: also receives the
 *              raw sums a
 *   ws         device workspace of ws_bytes >= ifq_conv_workspace_bytes(d),
 *              zero-filled before its first use (see there)
 * Errors: INVALID_ARGUMENT, UNSUPPORTED, INSUFFICIENT_BUFFER, HIP.
 */
IFQ_API ifq_status ifq_conv_forward(const ifq_conv_desc* d, const void* x,
                                    const void* w_packed, const int32_t* thr,
                                    const ifq_join* join, void* y,
                                    int32_t* acc_dump, void* ws,
                                    size_t ws_bytes, hipStream_t stream);

/*
 * The conv of ifq_conv_forward with its contraction (Eq. 1, integer part) on
 * the fp4 (e2m1) scaled matrix instructions, for the 3x3 layers of the
 * windowed kernel with the 2-bit threshold or identity-join epilogue. The codes 0..3 are the
 * e2m1 values c/2 and the weights +-2.0, so every product and partial sum is
 * an exact integer in fp32, and the output is bit-identical to
 * ifq_conv_forward's. Weights come from ifq_pack_weights_fp4.
 * Covered: in_layout BLOCK64, in_bits 2, 3x3, pad 1, stride 1 or 2,
 * c_in % 64 == 0, out_bits 2 in a 2-bit layout, c_out % 32 == 0, and no join
 * (thr as for ifq_conv_forward), an identity join with a 2-bit packed
 * shortcut, or a fused downsample join whose down_w is the 1x1 conv's
 * ifq_pack_weights_fp4 blob (join as for ifq_conv_forward, thr NULL); the
 * 128-channel tiles of the windowed kernel only; otherwise UNSUPPORTED
 * (ifq_conv_fp4_kernel_name returns ""). Asynchronous.
 * Errors: INVALID_ARGUMENT, UNSUPPORTED, HIP.
 */
IFQ_API ifq_status ifq_conv_forward_fp4(const ifq_conv_desc* d, const void* x,
                                        const void* w_fp4, const int32_t* thr,
                                        const ifq_join* join, void* y, hipStream_t stream);

/* Name of the kernel ifq_conv_forward_fp4 launches for d and join (nullable),
 * "" if none. Host. */
IFQ_API const char* ifq_conv_fp4_kernel_name(const ifq_conv_desc* d, const ifq_join* join);

/*
 * ifq_conv_pool_forward with the contraction on the fp4 path (as
 * ifq_conv_forward_fp4; w_fp4 from ifq_pack_weights_fp4): the same pooled
 * codes. Covered where both a fused-pool plan and an fp4 instance of the
 * windowed kernel exist; otherwise UNSUPPORTED (the name query returns "").
 * Errors: INVALID_ARGUMENT, UNSUPPORTED, HIP.
 */
IFQ_API ifq_status ifq_conv_pool_forward_fp4(const ifq_conv_desc* d, const ifq_pool_desc* p,
                                             const void* x, const void* w_fp4,
                                             const int32_t* thr, void* y, hipStream_t stream);
IFQ_API const char* ifq_conv_pool_fp4_kernel_name(const ifq_conv_desc* d,
                                                  const ifq_pool_desc* p);

/*
 * Bytes of the fp4 weight blob of a layer (0 unless in_bits 2, c_in % 64 == 0
 * and a 2-bit packed input layout), and its packing from the same OIHW +-1
 * int8 weights as ifq_pack_weights: per 32-row block and K64 step, 1 KB of
 * 64 lanes x 32 nibbles (+-2.0 as 0x4 / 0xC), in the order the kernel's
 * nibble expansion of the codes gives K; a zero block of 1 KB at the end.
 * Host only. Errors as ifq_pack_weights.
 */
IFQ_API size_t ifq_packed_weight_bytes_fp4(const ifq_conv_desc* d);
IFQ_API ifq_status ifq_pack_weights_fp4(const ifq_conv_desc* d, const int8_t* w_oihw,
                                        void* dst, size_t dst_bytes);

/*
 * Conv (Eq. 1, thresholds of Eq. 7-8) and max-pool (Eq. 4) in one kernel: the
 * codes of each output tile are pooled in the conv's epilogue and only the
 * pooled tensor reaches HBM. The paper pools the conv output before BN and
 * the quantizer; the code of a channel is monotone in its integer sum
 * (non-increasing where the sign s is -1), so pooling the codes gives the
 * same result as pooling the sums with max (s = +1) or min (s = -1) and
 * thresholding once. Asynchronous on stream.
 *   d          conv as for ifq_conv_forward, codes out (out_bits 1..8), no join
 *   p          the pool over the conv's output: n, h, w, c equal to the conv's
 *              n, ho, wo, c_out; bits = d->out_bits; layout = d->out_layout;
 *              any window, stride and mode of ifq_maxpool_codes. A kernel
 *              covers it where its tiles can hold whole rows of windows
 *              (VALID, k == stride, ho and wo multiples of k) or whole images
 *   x, w_packed, thr   as for ifq_conv_forward
 *   y          device [n][pho][pwo][c_out] codes in d->out_layout, pho and pwo
 *              as ifq_maxpool_codes gives them
 * Errors: INVALID_ARGUMENT (a desc invalid or the two inconsistent),
 * UNSUPPORTED (no fused kernel covers the shape: ifq_conv_pool_kernel_name
 * returns ""; run ifq_conv_forward and ifq_maxpool_codes instead), HIP.
 */
IFQ_API ifq_status ifq_conv_pool_forward(const ifq_conv_desc* d, const ifq_pool_desc* p,
                                         const void* x, const void* w_packed,
                                         const int32_t* thr, void* y, hipStream_t stream);

/*
 * Name of the kernel ifq_conv_pool_forward launches for d and p, as
 * ifq_conv_kernel_name; "" when the pair is invalid or not covered. Host.
 */
IFQ_API const char* ifq_conv_pool_kernel_name(const ifq_conv_desc* d,
                                              const ifq_pool_desc* p);

/*
 * Max-pool on codes (Eq. 4), asynchronous on stream. x, y device tensors in
 * d->layout; y is [n][ho][wo][c]. Errors: INVALID_ARGUMENT, UNSUPPORTED, HIP.
 */
IFQ_API ifq_status ifq_maxpool_codes(const ifq_pool_desc* d, const void* x,
                                     void* y, hipStream_t stream);

/*
 * Convert a code tensor of n images of h x w pixels and c channels between
 * any two of IFQ_LAYOUT_I8_NHWC, IFQ_LAYOUT_U2_NHWC_PACKED (c % 4 == 0) and
 * IFQ_LAYOUT_U2_BLOCK64 (c % 64 == 0), asynchronous; src and dst must not
 * overlap. Converting to a 2-bit layout keeps the low two bits of each code.
 * Errors: INVALID_ARGUMENT, HIP.
 */
IFQ_API ifq_status ifq_convert_codes(int64_t n, int64_t h, int64_t w, int32_t c,
                                     int32_t src_layout, int32_t dst_layout,
                                     const void* src, void* dst,
                                     hipStream_t stream);

/*
 * Device workspace bytes of a stack: at its start the conv workspace shared
 * by the layers (the K-split counters and partial tiles, as for
 * ifq_conv_workspace_bytes; at least the 64 KiB counter region), then the
 * work slots (256-byte aligned). Zero-fill it before its first use; runs
 * leave the counter region zero, so one workspace serves any stacks.
 */
IFQ_API size_t ifq_stack_workspace_bytes(const ifq_stack* s);

/*
 * Where work slot `slot` (2 .. n_slots-1) of a stack lives in the workspace:
 * its byte offset and capacity (the largest tensor any layer writes to it).
 * After ifq_run_stack a slot holds the tensor its last writer produced, in
 * that layer's output layout. Host. Errors: INVALID_ARGUMENT.
 */
IFQ_API ifq_status ifq_stack_slot_info(const ifq_stack* s, int32_t slot,
                                       size_t* offset, size_t* bytes);

/*
 * Run a layer chain (Sec. 3.1) on one stream with no host synchronisation.
 * All layers are validated before the first launch. x is slot 0, y slot 1;
 * ws holds the other slots. Errors: as ifq_conv_forward / ifq_maxpool_codes,
 * plus INVALID_ARGUMENT for a slot read before it is written.
 */
IFQ_API ifq_status ifq_run_stack(const ifq_stack* s, const void* x, void* y,
                                 void* ws, size_t ws_bytes,
                                 hipStream_t stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops, harnesses that forbid hipMalloc): ifq_run_stack
 * with the work slots in a workspace of ifq_static_workspace_bytes() bytes
 * (64 MiB) that the library keeps in a device array, one per GPU, for the
 * life of the process. The caller still passes x and y (device pointers, as
 * for ifq_run_stack). Calls nothing that allocates or frees device memory.
 * Every call on one GPU shares that GPU's array and leaves the last call's
 * slot contents in it (nothing in it needs clearing: every slot is written
 * before it is read, and the K-split counter region at its start is zero
 * from the library's load and again after every run), so calls that
 * overlap on one GPU (two streams, two
 * threads) race and must be serialised by the caller. Errors: as
 * ifq_run_stack, INSUFFICIENT_BUFFER when ifq_stack_workspace_bytes(s)
 * exceeds the static workspace (nothing is launched), HIP_ERROR when the
 * array's device address cannot be looked up on the current device.
 */
IFQ_API ifq_status ifq_run_stack_static(const ifq_stack* s, const void* x, void* y,
                                        hipStream_t stream);

/* Bytes of the static workspace of ifq_run_stack_static. Host. */
IFQ_API size_t ifq_static_workspace_bytes(void);

#ifdef __cplusplus
}
#endif

#endif /* IFQ_H_ */
