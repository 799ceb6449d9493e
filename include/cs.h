/*
 * cs.h - C ABI of the Complementary Sparsity sparse-sparse layer for AMD
 * Instinct MI355X (gfx950).
 *
 * The method (Hunter, Spracklen and Ahmad, "Two Sparsities Are Better Than
 * One", Section 3) overlays N sparse weight kernels whose supports do not
 * collide into one dense packed kernel that stores, per slot, a weight value
 * and a Kernel ID (Combine, Sections 3.1-3.2 step 1, Section 3.3.1).  At run
 * time only the non-zero activations are visited (Select, Section 3.2 step 2);
 * each is multiplied by the packed weights at its index (Multiply, step 3),
 * each product goes to the accumulator of its Kernel ID (Route, step 4,
 * Section 3.3.2) and is summed (Sum, step 5).  k-WTA (Section 3.3.3) then
 * keeps the k largest outputs, which become the next layer's sparse input.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Status: every function returns a cs_status (0 = success, < 0 = error).
 *    All argument checks are synchronous, run on the host and happen before
 *    any HIP call, so a bad argument never launches work and needs no GPU.
 *    A HIP launch or runtime failure returns CS_ERR_DEVICE; the library clears
 *    the HIP error state it observed.  No C++ exception crosses this ABI.
 *  - Ownership: the caller owns every buffer.  The GPU entry points never
 *    allocate, free or synchronise; they enqueue kernels on `stream` (a
 *    hipStream_t passed as void*, NULL = the default stream) and return.
 *    Outputs are completely overwritten.  Inputs and outputs must not alias.
 *  - "host" pointers are ordinary CPU memory; "device" pointers are GPU memory
 *    of the current HIP device.
 *  - Layouts are dense row-major.  Images are NHWC.  Conv weights are OHWI,
 *    flattened per output channel to r = kh*kw*c_in slots with slot
 *    i = (ky*kw + kx)*c_in + c (taps major, channels inner; Section 5.1 treats
 *    a 3x3 conv as nine 1x1 convs).
 *  - Packed sets: output channel o belongs to set (group) g = o / n and has
 *    Kernel ID kid = o - g*n; the n kernels of a set are n contiguous output
 *    channels.  G = d_out / n packed kernels.
 *  - Integer path: int8 activations and weights, int32 accumulation and bias
 *    (Section 4: weights and activations quantised to 8 bits).  Float path:
 *    fp32 throughout.  Integer sums wrap modulo 2^32 on overflow (the
 *    configurations used stay below 2^31 by a wide margin).
 */
#ifndef CS_H_
#define CS_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CS_OK = 0,
  CS_ERR_ARG = -1,        /* null pointer, negative/zero size, bad enum value   */
  CS_ERR_SHAPE = -2,      /* sizes inconsistent or beyond the supported limits   */
  CS_ERR_DTYPE = -3,      /* unsupported dtype or dtype combination              */
  CS_ERR_COLLISION = -4,  /* cs_pack: two kernels of one set share a slot        */
  CS_ERR_WORKSPACE = -5,  /* workspace missing or smaller than required          */
  CS_ERR_DEVICE = -6,     /* HIP launch or runtime error                         */
  CS_ERR_UNSUPPORTED = -7 /* not available in this build of the library          */
} cs_status;

typedef enum { CS_I8 = 0, CS_I32 = 1, CS_F32 = 2 } cs_dtype;

/* Supported limits (checked, CS_ERR_SHAPE beyond them). */
#define CS_MAX_ROW 65535   /* row length / c_in: indices are stored as uint16  */
#define CS_MAX_N 32        /* kernels per packed set                           */
#define CS_MAX_KWTA_ROW 2048 /* row length of cs_kwta                           */

/*
 * Augmented packed tensor (Section 3.3.1: each packed weight carries the
 * Kernel ID that routes its products; Figure 8(b)).  aug[i][g], i < r slots,
 * g < G sets, row-major, one entry per (slot, set):
 *   CS_I8 : uint16_t  = (uint8_t)value | (kid << 8)
 *   CS_F32: cs_aug_f32 {float value; uint32_t kid;}   (8 bytes)
 * kid is local to the set, in [0, n).  A slot no kernel of the set uses (a
 * hole) holds value 0, kid 0.
 */
typedef struct {
  float value;
  uint32_t kid;
} cs_aug_f32;

/*
 * cs_pack - Combine (Section 3.1/3.2 step 1, Figure 7): overlay each set of n
 * kernels into one packed kernel with its Kernel IDs.  Offline, HOST memory
 * only, no HIP call.
 *
 *  wt      CS_I8 or CS_F32: element type of w.
 *  w       host [d_out][r] dense weights; an exact zero is an absent weight.
 *  n       complement factor, 1 <= n <= CS_MAX_N, must divide d_out.
 *  aug     host [r][G] out, G = d_out / n, augmented entries as above:
 *          value = w[g*n + kid][i] for the one kernel of set g non-zero at i.
 *  holes   out (may be NULL): number of (i, g) slots no kernel of g uses.
 *  bad_g, bad_i  out (may be NULL): on CS_ERR_COLLISION, the first colliding
 *          (set, slot) in set-major, slot-minor order; -1 otherwise.
 *  Errors: CS_ERR_ARG (null w/aug, d_out/r < 1), CS_ERR_SHAPE (n does not
 *  divide d_out, n > CS_MAX_N), CS_ERR_DTYPE, CS_ERR_COLLISION (aug is then
 *  unspecified).
 */
int cs_pack(cs_dtype wt, const void* w, int d_out, int r, int n, void* aug, int64_t* holes,
            int* bad_g, int* bad_i);

/*
 * cs_compact - the sparse representation of Select (Section 3.2 step 2: the
 * non-zero activations with their indices; Figure 10 passes winners "along
 * with their indices").  DEVICE memory.
 *
 *  xt      CS_I8 or CS_F32.
 *  x       device [rows][c] dense activations.
 *  idx     device [rows][c] out (uint16): per row, the indices of the non-zero
 *          elements in ascending order in idx[row][0 .. cnt[row]-1]; the rest
 *          of the row is left untouched.
 *  val     device [rows][c] out (same dtype as x): the matching values.
 *  cnt     device [rows] out (int32): number of non-zeros of each row.
 *  A float -0.0 counts as zero.  rows may be 0 (nothing is launched).
 *  Errors: CS_ERR_ARG, CS_ERR_DTYPE, CS_ERR_SHAPE (c > CS_MAX_ROW), CS_ERR_DEVICE.
 */
int cs_compact(cs_dtype xt, const void* x, int64_t rows, int c, uint16_t* idx, void* val,
               int32_t* cnt, void* stream);

/*
 * cs_mrs_conv2d - Multiply, Route and Sum (Section 3.2 steps 3-5, Sections
 * 3.3.1-3.3.2) of a convolution whose input is already in cs_compact form.
 * DEVICE memory.  For each output pixel and each non-zero (c, v) of every
 * input pixel under the kernel window at tap (ky, kx), slot
 * i = (ky*kw + kx)*c_in + c; for each set g the product v * aug[i][g].value
 * is added to output channel g*n + aug[i][g].kid.  Then bias, the optional 2x2
 * stride-2 max-pool (Table 1), then the NHWC store.
 *
 *  xt      CS_I8 (int8 lists and weights, int32 bias and y) or CS_F32.
 *  idx, lval, cnt  device lists of the b*h*w input pixels as cs_compact or
 *          cs_kwta_lists write them, row stride `cap` (cap >= 1 entries): every
 *          index < c_in; a count above cap is read as cap.  Row strides that
 *          are multiples of 4 take the fast path (4 entries per load).
 *  b, h, w, c_in   input geometry; kh, kw >= 1; stride >= 1; pad >= 0.
 *          ho = (h + 2*pad - kh)/stride + 1, wo likewise, both >= 1.
 *  aug     device augmented packed tensor [kh*kw*c_in][G] from cs_pack
 *          (every kid < n), element type of xt.
 *  c_out, n  n divides c_out, 1 <= n <= CS_MAX_N.
 *  bias    device [c_out] (int32 / fp32) or NULL for none.
 *  pool    1 (none) or 2 (2x2 stride-2 max-pool; ho and wo must be even).
 *  y       device NHWC [b][ho/pool][wo/pool][c_out] out (int32 / fp32).
 *  Errors: CS_ERR_ARG, CS_ERR_DTYPE, CS_ERR_SHAPE, CS_ERR_DEVICE.
 */
int cs_mrs_conv2d(cs_dtype xt, const uint16_t* idx, const void* lval, const int32_t* cnt, int cap,
                  int b, int h, int w, int c_in, int kh, int kw, int stride, int pad,
                  const void* aug, int c_out, int n, const void* bias, int pool, void* y,
                  void* stream);

/*
 * cs_mrs_kwta_conv2d - one whole layer: cs_mrs_conv2d followed by k-WTA along
 * the channels of every output pixel (Section 2.2.2: exactly the top k
 * activations propagate; Section 3.3.3 local k-WTA), with the winners sent on
 * as (index, value) lists (Figure 10) or as a dense masked tensor.  DEVICE
 * memory.  A layer with one output vector per sample (a linear layer: window
 * = the whole unpadded map, output 1 x 1, no pool; at most 1024 input pixels)
 * runs as one kernel with one workgroup per sample, the table read from
 * global memory; a layer whose packed table fits one workgroup's LDS runs as
 * one kernel with the table in LDS; in both the sums need not reach HBM.
 * Otherwise cs_mrs_conv2d and cs_kwta / cs_kwta_lists run back to back on
 * `stream`.
 *
 *  xt .. pool   as cs_mrs_conv2d.
 *  y       device NHWC [b][ho/pool][wo/pool][c_out] (int32 / fp32), always
 *          required: with keep_sums = 1 it holds the sums after pool and bias
 *          on return; with keep_sums = 0 it is scratch and its contents are
 *          unspecified.
 *  k       winners per output pixel, 0 <= k <= c_out; ties go to the lower
 *          channel index; fp32 compares numerically (-0.0 == +0.0).
 *  ot      output dtype: CS_F32 for fp32 input; CS_I32 (the sums themselves)
 *          or CS_I8 (requantised, clamp(v >> shift, -127, 127)) for int8.
 *  shift   0 .. 31, used with ot == CS_I8.
 *  out     device [b][ho/pool][wo/pool][c_out] of ot: winners kept, the rest
 *          zero.  NULL when lists are written instead.
 *  oidx, oval, ocnt, ocap  list output (NULL when out is given): per output
 *          pixel, oidx/oval [rows][ocap] (uint16 / ot) hold the winners whose
 *          output value is non-zero in ascending channel order and ocnt[row]
 *          their number; ocap >= k.
 *  Exactly one of out and oidx must be non-NULL.
 *  Errors: CS_ERR_ARG, CS_ERR_DTYPE, CS_ERR_SHAPE (k > c_out, ocap < k, or
 *  c_out > CS_MAX_KWTA_ROW), CS_ERR_DEVICE.
 */
int cs_mrs_kwta_conv2d(cs_dtype xt, const uint16_t* idx, const void* lval, const int32_t* cnt,
                       int cap, int b, int h, int w, int c_in, int kh, int kw, int stride, int pad,
                       const void* aug, int c_out, int n, const void* bias, int pool, void* y,
                       int keep_sums, int k, cs_dtype ot, int shift, void* out, uint16_t* oidx,
                       void* oval, int32_t* ocnt, int ocap, void* stream);

/*
 * cs_mrs_kwta_units_conv2d - cs_mrs_kwta_conv2d with the k-WTA applied in
 * units: every `unit` consecutive channels of an output pixel keep their own
 * k winners (Section 5: channels partitioned into independent modules, each
 * with its own k-WTA; the ResNet-50 stages use units of 64 channels).  fp32
 * only (unit == c_out: exactly cs_mrs_kwta_conv2d, any dtype, ot = the sums'
 * dtype).  DEVICE memory.  One kernel when the layer runs on the table-block
 * kernel with the selection on the lanes' own accumulators (no pooling,
 * power-of-two sets and kernels per set, n <= 16, c_out <= 256, a unit a
 * power-of-two number of a pixel's lanes); otherwise cs_mrs_conv2d and
 * cs_kwta on the [rows * c_out / unit][unit] view of y, dense output only.
 *
 *  xt .. keep_sums, out  as cs_mrs_kwta_conv2d (xt == CS_F32, output fp32).
 *  k       winners per unit, 0 <= k <= unit; ties go to the lower channel index.
 *  unit    channels per unit, dividing c_out.
 *  oidx, oval, ocnt, ocap  one list per output pixel with the winners of all
 *          its units in ascending channel order; ocap >= k * c_out / unit.
 *  Errors: CS_ERR_ARG, CS_ERR_DTYPE (xt != CS_F32 with unit != c_out),
 *  CS_ERR_SHAPE (unit does not divide c_out, k > unit, ocap too small, or
 *  lists asked for a layer the single kernel does not take), CS_ERR_DEVICE.
 */
int cs_mrs_kwta_units_conv2d(cs_dtype xt, const uint16_t* idx, const void* lval,
                             const int32_t* cnt, int cap, int b, int h, int w, int c_in, int kh,
                             int kw, int stride, int pad, const void* aug, int c_out, int n,
                             const void* bias, int pool, void* y, int keep_sums, int k, int unit,
                             void* out, uint16_t* oidx, void* oval, int32_t* ocnt, int ocap,
                             void* stream);

/*
 * cs_mrs_plan - how cs_mrs_conv2d / cs_mrs_kwta_conv2d would run a layer with
 * these sizes (operands assumed aligned as torch allocates them).  Host only;
 * no HIP call.  For tests and tuning.
 *
 *  xt .. pool  as cs_mrs_kwta_conv2d; cap: list row stride; k: winners, or -1
 *          for cs_mrs_conv2d (sums only).
 *  info    host int64[11] out: [0] path (0 one lane per output, 1 table-slice
 *          kernel, 2 fused layer kernel, 3 one workgroup per sample: a layer
 *          whose window is the whole unpadded input map, output 1 x 1, no
 *          pool - a linear layer; 4 input-stationary int8 convolution; 5 one
 *          wavefront per item: a 1x1 layer with many items and a k-WTA over
 *          rows of more than 128 or k > 32; 6 fp32 layer without pooling,
 *          sets and kernels per set powers of two, n <= 16, c_out <= 256:
 *          tiles complete in the channel dimension with the packed table
 *          streamed through LDS in blocks of rows, k-WTA in the epilogue);
 *          for path 6: [1] k-WTA selection (1-3 four lanes per row with
 *          top-8/16/32 lists, 4 sixteen lanes per row, 5 the lanes that
 *          summed a pixel, on their own accumulators, bit by bit, 6-8 the
 *          same four lanes with top-8/16/32 lists), [2] table rows per
 *          block, [3] blocks, [6]
 *          workgroups, [7] LDS bytes, [8] sets per lane; for paths 3 and
 *          5: [6] workgroups, [7] LDS bytes per workgroup, [8] entry slices
 *          per packed set; for path 4: [2] output rows per band, [6]
 *          workgroups, [7] LDS bytes, [8] sets per lane; for path 2: [1] tile mode (0 rows of
 *          items, 1 image rectangles), [2] items (mode 0) or pooled rows
 *          (mode 1) per tile, [3] pooled columns per tile (mode 1), [4] list
 *          chunks staged in LDS at most, [5] input pixels per tile at most,
 *          [6] workgroups, [7] LDS bytes per workgroup, [8] log2 of the lanes
 *          sharing one output's taps or chunks, [9] k-WTA selection variant;
 *          [10] 1 when k-WTA runs as a kernel of its own after the sums.
 *  Errors: CS_ERR_ARG, CS_ERR_DTYPE, CS_ERR_SHAPE.
 */
int cs_mrs_plan(cs_dtype xt, int cap, int b, int h, int w, int c_in, int kh, int kw, int stride,
                int pad, int c_out, int n, int pool, int k, int64_t* info);

/*
 * cs_linear - a whole sparse-sparse linear layer: cs_compact of x into the
 * workspace, then Multiply/Route/Sum (a linear layer is the 1x1 convolution
 * of 1x1 images).  DEVICE memory.
 *
 *  x       device [batch][d_in] (int8 or fp32), d_in <= CS_MAX_ROW.
 *  aug     device augmented packed tensor [d_in][G] from cs_pack of [d_out][d_in].
 *  bias    device [d_out] or NULL.   y  device [batch][d_out] out.
 *  ws      device workspace of at least cs_workspace_bytes(0, xt, batch, d_in)
 *          bytes, 256-byte aligned; its contents on entry do not matter.
 *  Errors: as cs_compact and cs_mrs_conv2d, plus CS_ERR_WORKSPACE.
 */
int cs_linear(cs_dtype xt, const void* x, int batch, int d_in, const void* aug, int d_out, int n,
              const void* bias, void* y, void* ws, size_t ws_bytes, void* stream);

/*
 * cs_conv2d - a whole sparse-sparse conv layer: cs_compact of the b*h*w input
 * pixels (rows of c_in) into the workspace, then cs_mrs_conv2d.  Arguments as
 * cs_mrs_conv2d with x a device NHWC [b][h][w][c_in] tensor; ws must hold at
 * least cs_workspace_bytes(1, xt, b*h*w, c_in) bytes.
 */
int cs_conv2d(cs_dtype xt, const void* x, int b, int h, int w, int c_in, int kh, int kw,
              int stride, int pad, const void* aug, int c_out, int n, const void* bias, int pool,
              void* y, void* ws, size_t ws_bytes, void* stream);

/*
 * cs_conv2d_noalloc - cs_conv2d for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same computation and result, bit for bit, but the
 * compaction lists go to a scratch area the library holds instead of a
 * workspace the caller passes in.
 *
 *  Arguments as cs_conv2d without ws / ws_bytes (linear layers: b = batch,
 *  h = w = kh = kw = stride = 1, pad = 0, pool = 1).
 *  Scratch: a static device array of CS_NOALLOC_SCRATCH_BYTES per GPU, part
 *  of the library's code object, held from the library's load until the
 *  process ends; its address is looked up once per device on the first call
 *  made with that device current.  Nothing is allocated, freed or cleared by
 *  a call; every scratch byte the kernels read was written earlier in the
 *  same call.  All calls on one GPU share that GPU's scratch, so calls whose
 *  execution overlaps on one GPU (concurrent streams, host threads) race and
 *  must be serialised by the caller.
 *  Errors: as cs_conv2d; CS_ERR_WORKSPACE when the lists of the b*h*w input
 *  rows need more than CS_NOALLOC_SCRATCH_BYTES (cs_workspace_bytes(1, xt,
 *  b*h*w, c_in) is that need); CS_ERR_DEVICE if the scratch address cannot be
 *  obtained.
 */
#define CS_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int cs_conv2d_noalloc(cs_dtype xt, const void* x, int b, int h, int w, int c_in, int kh, int kw,
                      int stride, int pad, const void* aug, int c_out, int n, const void* bias,
                      int pool, void* y, void* stream);

/*
 * cs_mrs_kwta_chain2 - two layers of a chain's tail: a layer with k-WTA whose
 * output is one vector per sample (a linear layer, or a conv whose pooled map
 * is 1 x 1), then a linear layer without k-WTA on its requantised winners
 * (Figure 10: the winners go on with their indices).  When the first layer
 * runs one workgroup per sample (as cs_mrs_plan reports, path 3) both run in
 * one kernel: every winner (channel i, value v) adds v times the second
 * layer's packed row i into LDS accumulators, and the winners never leave the
 * chip (their lists are still written); otherwise cs_mrs_kwta_conv2d and
 * cs_mrs_conv2d run back to back on `stream`.  DEVICE memory.
 *
 *  xt .. ocap   as cs_mrs_kwta_conv2d, with xt == ot == CS_I8 and list
 *          output (oidx, oval, ocnt, ocap; no dense out).
 *  aug2, c_out2, n2, bias2   the second layer (cs_pack of [c_out2][c_out]
 *          int8 weights; bias2 int32 [c_out2] or NULL).
 *  y2      device int32 [b][c_out2] out: the second layer's sums.
 *  Errors: as cs_mrs_kwta_conv2d; CS_ERR_SHAPE when the first layer's output
 *  is not one vector per sample.
 */
int cs_mrs_kwta_chain2(cs_dtype xt, const uint16_t* idx, const void* lval, const int32_t* cnt,
                       int cap, int b, int h, int w, int c_in, int kh, int kw, int stride, int pad,
                       const void* aug, int c_out, int n, const void* bias, int pool, void* y,
                       int keep_sums, int k, cs_dtype ot, int shift, uint16_t* oidx, void* oval,
                       int32_t* ocnt, int ocap, const void* aug2, int c_out2, int n2,
                       const void* bias2, void* y2, void* stream);

/*
 * cs_mrs_kwta_chain3 - three layers of a chain's tail (Figure 10: every
 * layer's winners go on to the next with their indices): an int8 convolution
 * with k-WTA and lists, a layer with k-WTA whose window is that layer's whole
 * pooled map (one output vector per sample), and a linear layer without k-WTA
 * on its winners.  The result is that of cs_mrs_kwta_conv2d on the first
 * layer followed by cs_mrs_kwta_chain2 on its lists (input shape b x hp x wp x
 * c_out, window hp x wp, stride 1, no padding, no pool, where hp x wp is the
 * first layer's pooled map).  When the first layer runs input-stationary with
 * one workgroup per image and the second one workgroup per sample, the three
 * run in one kernel: each workgroup writes its image's lists, then (after a
 * workgroup barrier) reads them back as the second layer's input and feeds
 * the third layer on chip; otherwise the two calls run back to back on
 * `stream`.  DEVICE memory.
 *
 *  xt .. ocap   the first layer as cs_mrs_kwta_conv2d, with xt == ot == CS_I8
 *          and list output (oidx, oval, ocnt, ocap).
 *  aug2, c_out2, n2, bias2, y2, k2, shift2, oidx2, oval2, ocnt2, ocap2   the
 *          second layer (cs_pack of [c_out2][hp*wp*c_out] int8 weights in the
 *          (y, x, channel) slot order; bias2 int32 or NULL; y2 int32
 *          [b][c_out2] sums, written when keep_sums; k-WTA k2 with
 *          requantisation shift2, lists of capacity ocap2 >= k2).
 *  aug3, c_out3, n3, bias3, y3   the third layer as cs_mrs_kwta_chain2's
 *          second (y3: int32 [b][c_out3]).
 *  Errors: as cs_mrs_kwta_conv2d and cs_mrs_kwta_chain2 (CS_ERR_ARG for a
 *  missing buffer or a bad k, shift or keep_sums; CS_ERR_SHAPE for sizes).
 */
int cs_mrs_kwta_chain3(cs_dtype xt, const uint16_t* idx, const void* lval, const int32_t* cnt,
                       int cap, int b, int h, int w, int c_in, int kh, int kw, int stride, int pad,
                       const void* aug, int c_out, int n, const void* bias, int pool, void* y,
                       int keep_sums, int k, cs_dtype ot, int shift, uint16_t* oidx, void* oval,
                       int32_t* ocnt, int ocap, const void* aug2, int c_out2, int n2,
                       const void* bias2, void* y2, int k2, int shift2, uint16_t* oidx2,
                       void* oval2, int32_t* ocnt2, int ocap2, const void* aug3, int c_out3,
                       int n3, const void* bias3, void* y3, void* stream);

/*
 * cs_conv2d_dense_kwta_chain3 - a whole chain shaped like the keyword-spotting
 * network of Section 4: the dense-input first layer (as cs_conv2d_dense_kwta,
 * int8, list output), then the three layers of cs_mrs_kwta_chain3 on its lists
 * (input shape b x hp x wp x c_out, where hp x wp is the first layer's pooled
 * map).  The result is that of those two calls.  When the first layer's
 * matrix-core kernel can take a whole image per workgroup and the three-layer
 * tail runs in one kernel (cs_mrs_kwta_chain3's condition, or: the second
 * layer has eight list slots per pixel (ocap == 8), a square 3x3 or 5x5
 * window, four sets (c_out2 == 4 * n2 <= 64), the first layer pools 2x2 and
 * the second layer's output map fits in LDS, which runs it output-stationary),
 * all four layers run in one kernel, one workgroup per image, the phases
 * separated by workgroup barriers and the lists between them read back from
 * L2; otherwise the two calls run back to back on `stream`.  The result does
 * not depend on the path (integer sums).  DEVICE memory.
 *
 *  xt .. ocap   the first layer as cs_conv2d_dense_kwta (xt == ot == CS_I8,
 *          list output oidx/oval/ocnt/ocap, no dense out).
 *  kh2 .. ocap2   the second layer (a conv over the first one's lists) as the
 *          first layer of cs_mrs_kwta_chain3: window, stride, padding, packed
 *          table, c_out2, n2, bias, pool, sums y2, k-WTA k2 / shift2 and lists.
 *  aug3 .. ocap3   the third layer (window = the second one's whole pooled map)
 *          as cs_mrs_kwta_chain3's second.
 *  aug4, c_out4, n4, bias4, y4   the last linear layer, as its third.
 *  keep_sums applies to the first three layers' sums y, y2, y3.
 *  Errors: as cs_conv2d_dense_kwta and cs_mrs_kwta_chain3.
 */
int cs_conv2d_dense_kwta_chain3(
    cs_dtype xt, const void* x, int b, int h, int w, int c_in, int kh, int kw, int stride, int pad,
    const void* aug, int c_out, int n, const void* bias, int pool, void* y, int keep_sums, int k,
    cs_dtype ot, int shift, uint16_t* oidx, void* oval, int32_t* ocnt, int ocap, int kh2, int kw2,
    int stride2, int pad2, const void* aug2, int c_out2, int n2, const void* bias2, int pool2,
    void* y2, int k2, int shift2, uint16_t* oidx2, void* oval2, int32_t* ocnt2, int ocap2,
    const void* aug3, int c_out3, int n3, const void* bias3, void* y3, int k3, int shift3,
    uint16_t* oidx3, void* oval3, int32_t* ocnt3, int ocap3, const void* aug4, int c_out4, int n4,
    const void* bias4, void* y4, void* stream);

/*
 * cs_conv2d_dense_blocks - the sparse-dense variant with block Complementary
 * Sparsity (Section 3.1: complementary patterns made of blocks; Section 5: a
 * stem whose block is one input pixel's RGB values; Section 4: a first layer
 * on dense input runs sparse-dense).  DEVICE memory, int8 activations and
 * weights, int32 sums.  A block is one tap's c_in channels: the c_in products
 * of a (tap, set) pair are summed first (one 4-way int8 dot product) and the
 * sum is routed once by the block's Kernel ID, so an output pixel costs
 * kh*kw*(c_out/n) dot products and routed adds.  No compaction, no workspace.
 *
 *  x       device NHWC [b][h][w][c_in] int8, dense; 1 <= c_in <= 4.
 *  aug     device [kh*kw*c_in][c_out/n] uint16 (cs_pack_blocks with b = c_in:
 *          value in the low byte).
 *  kidb    device [kh*kw][c_out/n] uint8: each block's Kernel ID (< n), as
 *          cs_pack_blocks writes it.
 *  bias    device int32 [c_out] or NULL.
 *  y       device NHWC [b][ho][wo][c_out] int32 out: the sums plus bias.
 *  Errors: CS_ERR_ARG, CS_ERR_SHAPE (c_in > 4, c_out/n sets too many for one
 *  workgroup, the input under one tile - kh rows of (P-1)*stride + kw
 *  pixels, P = 256 / lanes per pixel output pixels - over 1024 pixels, or
 *  the tile's LDS over 64 KB), CS_ERR_DEVICE.
 */
int cs_conv2d_dense_blocks(const int8_t* x, int b, int h, int w, int c_in, int kh, int kw,
                           int stride, int pad, const uint16_t* aug, const uint8_t* kidb,
                           int c_out, int n, const int32_t* bias, int32_t* y, void* stream);

/*
 * cs_conv2d_dense - the sparse-dense variant (Section 3.1: Combine, Multiply,
 * Route, Sum with dense activations; Section 4 runs the first layer of the
 * keyword-spotting network this way because its input is dense).  DEVICE
 * memory.  Same arguments and result as cs_conv2d, but x is read densely (no
 * compaction, no workspace).  Supported shapes (else CS_ERR_SHAPE): n == 1
 * (every set holds one dense kernel), c_out == 64, kh*kw*c_in <= 32 and an
 * input patch per output item ((pool-1)*stride + kh) * ((pool-1)*stride + kw)
 * * c_in <= 64 values.
 */
int cs_conv2d_dense(cs_dtype xt, const void* x, int b, int h, int w, int c_in, int kh, int kw,
                    int stride, int pad, const void* aug, int c_out, int n, const void* bias,
                    int pool, void* y, void* stream);

/*
 * cs_conv2d_dense_kwta - the whole dense-input first layer: cs_conv2d_dense
 * followed by k-WTA along the channels of every output pixel, with the
 * winners emitted as lists or densely, as cs_mrs_kwta_conv2d does for a
 * sparse input.  DEVICE memory.  For int8 with k <= 32 the convolution runs
 * on the matrix cores (int8 MFMA; the dense contraction of Section 3.1's
 * sparse-dense case) in the same kernel as the pool, the selection and the
 * output, and the sums need not reach HBM; otherwise cs_conv2d_dense and
 * cs_kwta / cs_kwta_lists run back to back on `stream`.
 *
 *  xt .. pool   as cs_conv2d_dense (n == 1, c_out == 64, kh*kw*c_in <= 32; the
 *          two-kernel path, taken for fp32 or k > 32, also needs the pooled
 *          window to hold at most 64 values, else CS_ERR_SHAPE).
 *  y, keep_sums, k, ot, shift, out, oidx, oval, ocnt, ocap   as
 *          cs_mrs_kwta_conv2d.
 *  Errors: CS_ERR_ARG, CS_ERR_DTYPE, CS_ERR_SHAPE, CS_ERR_DEVICE.
 */
int cs_conv2d_dense_kwta(cs_dtype xt, const void* x, int b, int h, int w, int c_in, int kh, int kw,
                         int stride, int pad, const void* aug, int c_out, int n, const void* bias,
                         int pool, void* y, int keep_sums, int k, cs_dtype ot, int shift, void* out,
                         uint16_t* oidx, void* oval, int32_t* ocnt, int ocap, void* stream);

/* Output tile side of the reordering kernel (CS_REORDER_TILE^2 pixels). */
#define CS_REORDER_TILE 8

/*
 * cs_reorder_table - the packed kernel in Kernel-ID order, for reordering
 * the activations instead of routing the products (Section 3.2: reordering
 * the incoming activations as the alternative to routing the element-wise
 * products).  Offline, HOST memory only, no HIP call.  For every output
 * o = g*n + kid the table lists the slots i of set g with kid[i][g] == kid and
 * a non-zero value (the support of kernel o), in ascending slot order, as
 * pairs (byte offset of slot i in cs_conv2d_reorder_kwta's input tile,
 * value bits): slot i = (ky*kw + kx)*c_in + c has offset
 * 4*((ky*(CS_REORDER_TILE + kw - 1) + kx)*(c_in + 1) + c).
 *
 *  aug     host [kh*kw*c_in][c_out/n] cs_aug_f32 entries (cs_pack, CS_F32).
 *  smax    in/out: with table == NULL, receives the longest support (>= 1);
 *          else the entries per output the table has room for (>= that).
 *  table   host [c_out][smax][2] int32 out (may be NULL), outputs shorter
 *          than smax padded with (0, 0.0f).
 *  Errors: CS_ERR_ARG (null aug/smax, sizes < 1, a kid >= n), CS_ERR_SHAPE
 *  (n does not divide c_out, n > CS_MAX_N, kh*kw*c_in > CS_MAX_ROW, smax too
 *  small).
 */
int cs_reorder_table(const void* aug, int kh, int kw, int c_in, int c_out, int n, int* smax,
                     int32_t* table);

/*
 * cs_pack_blocks - Combine for Complementary Sparsity with blocks of
 * non-zeros (Section 3.1: complementary patterns made of blocks; Section 5's
 * stem treats a pixel's 3 RGB inputs as one block).  Slots j*b .. j*b+b-1 form
 * block j (for conv weights in (tap, channel) slot order and b dividing c_in,
 * a block is b consecutive channels of one tap); every kernel's support must
 * be a union of whole blocks, complementary within each set block by block.
 * Offline, HOST memory only, no HIP call.
 *
 *  wt, w, d_out, r, n, aug   as cs_pack (aug is the per-slot augmented
 *          tensor every layer call reads); b divides r.
 *  kidb    host [r/b][G] uint8 out: the Kernel ID of each (block, set) - one
 *          routing decision for the block's b products (0 for a hole).
 *  holes   out (may be NULL): (block, set) pairs no kernel uses.
 *  bad_g, bad_i  out (may be NULL): on CS_ERR_SHAPE for a split block, the
 *          kernel and the block; on CS_ERR_COLLISION, the set and the block.
 *  Errors: CS_ERR_ARG, CS_ERR_DTYPE, CS_ERR_SHAPE (n does not divide d_out,
 *  n > CS_MAX_N, b does not divide r, a support splits a block),
 *  CS_ERR_COLLISION.
 */
int cs_pack_blocks(cs_dtype wt, const void* w, int d_out, int r, int n, int b, void* aug,
                   uint8_t* kidb, int64_t* holes, int* bad_g, int* bad_i);

/*
 * cs_pack_channels - Combine along the channel dimension (Section 3.1: sets
 * of kernels can be overlaid in the filter or in the channel dimension).  In
 * every filter, each group of n consecutive input channels holds n kh x kw
 * slices with disjoint supports; they are overlaid into one dense kh x kw
 * slice whose slots keep the weight and the channel ID (which slice, 0..n-1).
 * Offline, HOST memory only, no HIP call.
 *
 *  wt      CS_F32 or CS_I8.  w host [c_out][kh][kw][c_in] dense filters (0 =
 *          absent).
 *  n       channels per group, 1 <= n <= CS_MAX_N, dividing c_in.
 *  packed  host [c_out][c_in/n][kh][kw] out, cs_aug_f32 (CS_F32) or uint16
 *          (CS_I8: value byte | channel ID << 8) entries, kid = channel ID:
 *          value = w[o][y][x][q*n + cid] for the one channel of group q that
 *          is non-zero at (y, x); holes hold 0, 0.
 *  holes   out (may be NULL): packed slots no channel uses.
 *  bad_o, bad_i  out (may be NULL): on CS_ERR_COLLISION the first colliding
 *          filter and packed slot (q*kh + y)*kw + x, in that order; else -1.
 *  Errors: CS_ERR_ARG, CS_ERR_DTYPE, CS_ERR_SHAPE (n does not divide c_in,
 *  n > CS_MAX_N), CS_ERR_COLLISION (packed then unspecified).
 */
int cs_pack_channels(cs_dtype wt, const void* w, int c_out, int kh, int kw, int c_in, int n,
                     void* packed, int64_t* holes, int* bad_o, int* bad_i);

/*
 * cs_channel_table - the table cs_conv2d_channels reads for an int8
 * channel-overlaid layer (cs_pack_channels, CS_I8) run with stride `stride`.
 * Offline, HOST memory only, no HIP call.  Filter o's row holds, with S =
 * (c_in/n)*kh*kw packed slots and S4 = ceil(S/4): first 4*S4 offsets, slot
 * i = (q*kh + y)*kw + x at [i] (padding slots 0): off = (y*sw + x)*cp + q*n +
 * cid, the byte offset of the slot's input (tap (y, x), channel q*n + cid)
 * from the first input pixel of an output pixel's window in the kernel's
 * staged tile (sw = 63*stride + kw pixels per staged row, cp = c_in bytes per
 * pixel when c_in/4 is odd, else c_in + 4); then S4 words, word j holding the
 * weights of slots 4j .. 4j+3 in its bytes (0 for padding slots).
 *
 *  packed  host [c_out][c_in/n][kh][kw] uint16 (cs_pack_channels, CS_I8).
 *  table   host int32 [c_out][5 * S4] out.
 *  Errors: CS_ERR_ARG (null pointers, sizes < 1, a channel ID >= n),
 *  CS_ERR_SHAPE (n does not divide c_in, c_in not a multiple of 4, n >
 *  CS_MAX_N, the staged tile reaching 2^23 bytes).
 */
int cs_channel_table(const uint16_t* packed, int kh, int kw, int c_in, int c_out, int n,
                     int stride, int32_t* table);

/*
 * cs_conv2d_channels - an int8 dense-input conv layer with Complementary
 * Sparsity overlaid in the channel dimension (Section 3.1): every output is
 * the dot product of its filter's packed slots with the input gathered at
 * each slot's channel (q*n + channel ID) - no routing, the products of a
 * filter all go to its own output.  DEVICE memory (except the scalars).
 * Output tiles of 64 pixels of one output row, one pixel per lane, the
 * filters split over the four wavefronts of a workgroup; the tile's input
 * rows staged in LDS with the pixel stride of cs_channel_table.
 *
 *  x       device NHWC [b][h][w][c_in] int8, dense, 4-byte aligned; c_in a
 *          multiple of 4.
 *  table   device copy of cs_channel_table's table for this stride.
 *  c_out   16, 32, 64 or 128; n as packed.
 *  bias    device int32 [c_out] or NULL.
 *  y       device NHWC [b][ho][wo][c_out] int32 out (16-byte aligned): sums + bias.
 *  Errors: CS_ERR_ARG, CS_ERR_SHAPE (c_out, c_in or n unsupported, the staged
 *  tile over 64 KB of LDS), CS_ERR_DEVICE.
 */
int cs_conv2d_channels(const int8_t* x, int b, int h, int w, int c_in, int kh, int kw, int stride,
                       int pad, const int32_t* table, int c_out, int n, const int32_t* bias,
                       int32_t* y, void* stream);

/*
 * cs_reorder_table_channels - cs_reorder_table for a channel-overlaid layer
 * (cs_pack_channels): every filter's packed slots (q, y, x) with a non-zero
 * value read channel q*n + cid at tap (y, x), so the filter's table lists
 * them with that slot's byte offset in cs_conv2d_reorder_kwta's input tile;
 * the layer then runs as any reordered layer.  Offline, HOST memory only.
 *  packed  host [c_out][c_in/n][kh][kw] cs_aug_f32 (cs_pack_channels).
 *  smax, table   as cs_reorder_table.
 *  Errors: CS_ERR_ARG (null packed/smax, sizes < 1, a channel ID >= n),
 *  CS_ERR_SHAPE (n does not divide c_in, n > CS_MAX_N, kh*kw*c_in >
 *  CS_MAX_ROW, smax too small).
 */
int cs_reorder_table_channels(const void* packed, int kh, int kw, int c_in, int c_out, int n,
                              int* smax, int32_t* table);

/*
 * cs_conv2d_reorder_kwta - a dense-input fp32 conv layer computed by
 * reordering instead of routing: every output reads the activations at its
 * kernel's support (cs_reorder_table) and sums their products in a register;
 * then k-WTA along the channels of every output pixel as cs_mrs_kwta_conv2d.
 * Same sums as cs_conv2d_dense_kwta / cs_conv2d + cs_mrs_kwta_conv2d up to
 * fp32 rounding order.  DEVICE memory (except the scalars).
 *
 *  xt      CS_F32.  x device NHWC [b][h][w][c_in] dense activations.
 *  kh, kw, pad   window and zero padding; stride 1, no pooling.
 *  table, smax   device copy of cs_reorder_table's table for this layer, with
 *          smax a multiple of 8 (CS_ERR_SHAPE otherwise).
 *  c_out   must be 64; c_in <= 64.
 *  bias    device [c_out] (may be NULL).
 *  y, keep_sums  device [b][ho][wo][c_out] sums, written when keep_sums == 1
 *          (16-byte aligned).
 *  k       winners per pixel, 0 <= k <= 32 or k == c_out; ot CS_F32.
 *  out | (oidx, oval, ocnt, ocap)   exactly one: dense [b][ho][wo][c_out]
 *          output (winners keep their value, the rest 0; 16-byte aligned), or
 *          lists as cs_mrs_kwta_conv2d with ocap >= k and a multiple of 4,
 *          oidx 8-byte and oval 16-byte aligned.
 *  Errors: CS_ERR_ARG, CS_ERR_DTYPE, CS_ERR_SHAPE, CS_ERR_DEVICE.
 */
int cs_conv2d_reorder_kwta(cs_dtype xt, const void* x, int b, int h, int w, int c_in, int kh,
                           int kw, int pad, const int32_t* table, int smax, int c_out,
                           const void* bias, void* y, int keep_sums, int k, cs_dtype ot,
                           void* out, uint16_t* oidx, void* oval, int32_t* ocnt, int ocap,
                           void* stream);

/*
 * cs_kwta - k-WTA (Section 2.2.2: exactly the top k activations propagate;
 * Section 3.3.3: global k-WTA over a vector after linear layers, local k-WTA
 * along the channels of each pixel after conv layers - both are this call
 * with one row per vector or per pixel).  DEVICE memory.
 *
 *  it      CS_I32 or CS_F32: dtype of `in`.
 *  in      device [rows][c], 1 <= c <= CS_MAX_KWTA_ROW, 0 <= k <= c.
 *  Each row keeps exactly k elements: the k largest, equal values going to
 *  the lower index; fp32 compares numerically (-0.0 ties +0.0; NaN is not
 *  supported).  Winners keep their value (even if <= 0), the rest become 0.
 *  ot      == it: out holds the masked values.
 *          CS_I8 with it == CS_I32: out holds requantised winners
 *          clamp(v >> shift, -127, 127) (arithmetic shift), 0 elsewhere.
 *  shift   0..31, used only for CS_I8 output.
 *  out     device [rows][c] out.  rows may be 0.
 *  Errors: CS_ERR_ARG, CS_ERR_DTYPE, CS_ERR_SHAPE, CS_ERR_DEVICE.
 */
int cs_kwta(cs_dtype it, const void* in, int64_t rows, int c, int k, cs_dtype ot, int shift,
            void* out, void* stream);

/*
 * cs_kwta_lists - k-WTA whose winners go to the next layer as (index, value)
 * lists (Figure 10: the values that pass are sent on "along with their
 * indices"; Section 3.2: the next layer's Select is this list).  DEVICE memory.
 * Same selection and dtype rules as cs_kwta (exactly k, ties to the lower
 * index, optional int8 requantisation), but instead of a dense row it writes,
 * per row, the winners whose output value is non-zero in ascending index
 * order: idx[row][0 .. cnt[row]-1] (uint16), val[row][..] (dtype ot),
 * cnt[row] (int32), row stride `cap` >= k.  Entries past cnt are untouched.
 * These lists feed cs_mrs_conv2d directly (its cap argument = this cap).
 *  Errors: as cs_kwta; CS_ERR_SHAPE if cap < k.
 */
int cs_kwta_lists(cs_dtype it, const void* in, int64_t rows, int c, int k, cs_dtype ot, int shift,
                  uint16_t* idx, void* val, int32_t* cnt, int cap, void* stream);

/*
 * cs_workspace_bytes - workspace cs_linear (op 0) or cs_conv2d (op 1) needs
 * for `rows` input rows (batch, or b*h*w pixels) of c_in elements of dtype
 * xt.  Returns 0 for invalid arguments.  Host only.
 */
size_t cs_workspace_bytes(int op, cs_dtype xt, int64_t rows, int c_in);

/*
 * cs_product_count - the number of weight x activation products the
 * multiply-route-sum kernels have formed on the current device since the
 * last reset (Section 3.2 and Figure 1: only pairs of a non-zero activation
 * and a non-zero packed weight are multiplied, so the work falls with the
 * product of the two densities).  Only the counting build of the library
 * (libcs_count.so, compiled with CS_COUNT_PRODUCTS) keeps the count: each
 * kernel adds the products of its live list entries to one device counter.
 * The dense-input matrix-core layers are not counted (they are dense
 * contractions, not routed products).
 *
 *  count  out (host, may be NULL): the count, read after the device has
 *         finished all work queued before the call.
 *  reset  non-zero: set the counter to 0 after reading it.
 *
 * Synchronises the current device.  Errors: CS_ERR_UNSUPPORTED in the
 * product build (libcs.so), CS_ERR_DEVICE.
 */
int cs_product_count(unsigned long long* count, int reset);

/*
 * cs_phase_stamps - per-phase wall-clock sums of the stamping build of the
 * library (libcs_stamps.so, compiled with CS_PHASE_STAMPS; a measurement
 * aid: where the time of a layer kernel goes).  At the end of each phase of
 * the one-kernel keyword-spotting chain and of each tile of the table-block
 * kernel, thread 0 of the workgroup adds the constant-rate wall clock to the
 * phase's slot, and at each start one to the count slot (chain: slots 0-13
 * in phase order, count 15; table-block kernel: 16 tile start, 17 products,
 * 18 epilogue, count 31, inside its k-WTA on the lanes' own columns 19
 * threshold search, 20 winner masks, and 21 the summed time of a tile's table
 * blocks' products).  (slot[b] - slot[a]) / count / clock is the mean time
 * from point a to point b, slot[21] / count / clock a mean duration.
 *
 *  acc        out (host): the first n slots, read after the device has
 *             finished all work queued before the call; n in 0..32.
 *  reset      non-zero: set every slot to 0 after reading.
 *  clock_khz  out (host, may be NULL): the wall clock's rate in kHz.
 *
 * Synchronises the current device.  Errors: CS_ERR_ARG (n outside 0..32, or
 * acc NULL with n > 0), CS_ERR_UNSUPPORTED outside the stamping build,
 * CS_ERR_DEVICE.
 */
int cs_phase_stamps(unsigned long long* acc, int n, int reset, int* clock_khz);

/* cs_status_str - static, never-NULL description of a status code. */
const char* cs_status_str(int status);

#ifdef __cplusplus
}
#endif

#endif /* CS_H_ */
