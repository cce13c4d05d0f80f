/*
 * mdlstm.h — C ABI of the packed four-direction MDLSTM layer for MI355X (gfx950).
 *
 * What is computed (Maillette de Buy Wenniger, Schomaker, Way, "No Padding
 * Please: Efficient Neural Handwriting Recognition"):
 *
 *   - Example packing (Section V-A; Algorithm 1 in Appendix B): variable-size
 *     examples are bucketed by height, rows are filled greedily with the widest
 *     example that still fits, and examples are tiled within and across rows
 *     with one separating pixel; a binary mask marks example pixels.
 *   - The four-direction 2D MDLSTM layer (Section III, Section IV-B): per scan
 *     direction d and cell, with left/top predecessors L and T in d's frame,
 *         a   = Wx_d x + b_d + U_d [h_L ; h_T]       5H rows, gates in the order
 *                                                    (i, f_L, f_T, o, g)
 *         c   = sig(a_i) tanh(a_g) + sig(a_fL) c_L + sig(a_fT) c_T
 *         h   = sig(a_o) tanh(c)
 *     Direction 0 scans from the top-left, 1 from the top-right, 2 from the
 *     bottom-left, 3 from the bottom-right. State handed over by a predecessor
 *     outside the cell's rectangle or with mask 0 is zero (Section V, binary
 *     masking), so a packed canvas gives every example exactly the result it
 *     has alone.
 *
 * Conventions shared by every entry point:
 *   - Canvas tensors are row-major [canvas_h][canvas_w][channels] ("HWC"),
 *     unskewed; the input-skewing of Section IV-A is index arithmetic inside
 *     the kernels.
 *   - Pointers named d_* are DEVICE memory of the current HIP device; all
 *     other pointers are HOST memory. The caller owns every buffer; the library
 *     allocates no memory of its own (its one static device array, the scratch
 *     of mdlstm_pack_layout_noalloc, is described there) and keeps no pointer
 *     after returning (workspace addresses serve as lookup keys only, never
 *     dereferenced).
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream). Work
 *     is enqueued on it asynchronously unless stated otherwise.
 *   - Every argument is validated on the host before any HIP call; on error
 *     nothing is enqueued and mdlstm_last_error() describes the problem.
 *   - Calls are reentrant given distinct workspaces.
 */
#ifndef MDLSTM_H
#define MDLSTM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MDLSTM_OK = 0,
    MDLSTM_ERR_INVALID_ARG = 1, /* NULL pointer, negative size, bad descriptor   */
    MDLSTM_ERR_TOO_WIDE = 2,    /* an example is wider than the canvas          */
    MDLSTM_ERR_BAD_LAYOUT = 3,  /* rectangles overlap or leave the canvas       */
    MDLSTM_ERR_WORKSPACE = 4,   /* workspace or output buffer too small         */
    MDLSTM_ERR_UNSUPPORTED = 5, /* hidden size / dtype / rectangle height not built */
    MDLSTM_ERR_DEVICE = 6,      /* a HIP call failed; message has the HIP string */
    MDLSTM_ERR_NUMERIC = 7      /* non-finite outputs, reported only when the
                                   environment sets MDLSTM_CHECK_FINITE=1 (see mdlstm_forward) */
} mdlstm_status;

/* Storage type of x, y, weights, dx and the saved gates. Accumulation and the
 * saved cell state are always fp32; weight gradients are always fp32. */
typedef enum { MDLSTM_F32 = 0, MDLSTM_BF16 = 1 } mdlstm_dtype;

/* A rectangle of the canvas: top-left corner (y0, x0), height h, width w. */
typedef struct {
    int32_t y0, x0, h, w;
} mdlstm_rect;

/* One MDLSTM layer. Supported: F32 with 1 <= hidden <= 64, BF16 with
 * 1 <= hidden <= 128, and 1 <= c_in <= 256 (UNSUPPORTED beyond). The kernels
 * are built for F32 hidden in {4, 8, 16, 32, 64}, BF16 hidden in {32, 64,
 * 128}, and c_in a multiple of 4 (F32) or 8 (BF16). Other sizes (the paper's
 * 2, 10 and 50 hidden units, a single input channel) run on the next built
 * shape: the call copies the weights and, when those sizes differ, x, y and
 * dy into zero-padded copies in the workspace and copies y, dx and the
 * weight gradients back. A padded unit has zero weights, so its gates stay at
 * 1/2, its cell candidate, state and output at 0 and its gradients at 0; a
 * padded input channel is 0. The results are those of the layer's own sizes
 * (bit for bit those of the built shape on zero-padded operands); the copies
 * cost workspace and a few extra passes over x and y.
 *
 * memory_states = 1 adds the memory-state matrices of Appendix A (three per
 * predecessor memory state S1 = c_L and S2 = c_T, next to the five per
 * predecessor hidden state). Reading: both states feed the input gate and the
 * two forget gates through V_d (3H x 2H, rows i, f_L, f_T; columns c_L, c_T):
 *     a = Wx_d x + b_d + U_d [h_L ; h_T] + [V_d [c_L ; c_T] ; 0 ; 0]
 * The recurrent weight argument then holds U [4][5H][2H] immediately followed
 * by V [4][3H][2H] (one buffer), and the backward writes dU followed by dV the
 * same way. Built for F32 with hidden 16 or 32 (hidden 1 to 15 and 17 to 31
 * padded as above; UNSUPPORTED for BF16 and above 32); the per-diagonal
 * schedule (mdlstm_forward_stepwise) is not built for it.
 * 0 (or a descriptor initialised with its first three fields) is the plain
 * cell. */
typedef struct {
    int32_t c_in;
    int32_t hidden;
    int32_t dtype;         /* mdlstm_dtype */
    int32_t memory_states; /* 0 or 1 */
} mdlstm_layer_desc;

/* Largest rectangle height the wavefront kernels accept. */
#define MDLSTM_MAX_RECT_H 64

/* Most rectangles (examples) one call takes (UNSUPPORTED beyond). */
#define MDLSTM_MAX_RECTS (1 << 24)

/* Device workspace needed by mdlstm_pack_layout / mdlstm_pack_data /
 * mdlstm_unpack_data for n examples. */
size_t mdlstm_pack_workspace_bytes(int32_t n);

/*
 * Example packing, placement and mask (Section V-A steps 1-3; Algorithm 1).
 *
 * heights[n], widths[n] (host): example sizes, all >= 1.
 * canvas_w: width of the canvas; every example must fit (else TOO_WIDE).
 * rects[n] (host, out): rects[k] is the placement of ORIGINAL example k.
 * canvas_h (host, out): height of the packed canvas (0 when n == 0).
 * d_mask (device, out, may be NULL): uint8 [canvas_h][canvas_w], 1 on example
 *   pixels and 0 on separators and slack; needs mask_bytes >= canvas_h*canvas_w
 *   (else WORKSPACE, with rects and canvas_h still written). With NULL only the
 *   placement is computed, so a caller can learn canvas_h, allocate, and call again.
 * d_workspace: mdlstm_pack_workspace_bytes(n) bytes of device memory.
 *
 * Placement runs as a kernel on `stream`, and the call waits for it because
 * rects and canvas_h are host outputs. The mask is written asynchronously; the
 * workspace must stay untouched until the stream has passed the mask kernel.
 * Readings of the paper this follows: buckets in ascending height; ties in
 * width broken by original index; the fit test counts a separator only between
 * two examples; a partial row is flushed when its bucket runs empty.
 */
mdlstm_status mdlstm_pack_layout(int32_t n, const int32_t* heights, const int32_t* widths,
                                 int32_t canvas_w, mdlstm_rect* rects, int32_t* canvas_h,
                                 uint8_t* d_mask, size_t mask_bytes,
                                 void* d_workspace, size_t workspace_bytes, void* stream);

/* Most examples one mdlstm_pack_layout_noalloc call places. */
#define MDLSTM_NOALLOC_MAX_N 4096

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * placement and mask as mdlstm_pack_layout, with the same arguments, results
 * (bit for bit) and errors, but no workspace argument. Its device scratch (the
 * uploaded sizes and the placement, 4 * (6n + 1) bytes) lives in a static
 * array of MDLSTM_NOALLOC_MAX_N * 24 + 4 bytes that each GPU the library runs
 * on holds until the process ends; the call allocates neither device nor heap
 * memory (host staging is a per-thread static buffer).
 * n > MDLSTM_NOALLOC_MAX_N is refused with UNSUPPORTED before any HIP call.
 * Every call on one GPU shares that GPU's array, and the mask kernel reads it
 * after the call returns: calls that overlap on one GPU (other threads, or
 * another stream before this call's mask kernel has run) race. Nothing in the
 * array needs to start at zero: every call writes what it reads.
 */
mdlstm_status mdlstm_pack_layout_noalloc(int32_t n, const int32_t* heights, const int32_t* widths,
                                         int32_t canvas_w, mdlstm_rect* rects, int32_t* canvas_h,
                                         uint8_t* d_mask, size_t mask_bytes, void* stream);

/*
 * Last-minute batch padding layout (Section VI-B): every example padded to the
 * batch maximum height and width; tiles stacked vertically with no separators.
 * tiles[n] (host, out) are the scheduling rectangles, place[n] (host, out) the
 * example extents (top-left of each tile). canvas_h/canvas_w (host, out).
 * d_mask (device, out, may be NULL): 1 on example pixels, 0 on padding.
 * Host-only computation plus an asynchronous mask kernel.
 */
mdlstm_status mdlstm_pad_layout(int32_t n, const int32_t* heights, const int32_t* widths,
                                mdlstm_rect* tiles, mdlstm_rect* place,
                                int32_t* canvas_h, int32_t* canvas_w,
                                uint8_t* d_mask, size_t mask_bytes,
                                void* d_workspace, size_t workspace_bytes, void* stream);

/*
 * Scatter (Section V-A step 3) / gather (unpacking, Section V-A last paragraph).
 * d_examples[k] (host array of device pointers): example k, HWC [h][w][c]
 *   with (h, w) = (rects[k].h, rects[k].w), storage dtype `dt`.
 * rects[n] (host): where example k sits on the canvas (disjoint, inside).
 * d_canvas: [canvas_h][canvas_w][c]. pack_data overwrites the whole canvas,
 *   zero outside the rectangles; unpack_data reads it and overwrites each example.
 */
mdlstm_status mdlstm_pack_data(int32_t n, const void* const* d_examples, const mdlstm_rect* rects,
                               int32_t canvas_h, int32_t canvas_w, int32_t c, int32_t dt,
                               void* d_canvas, void* d_workspace, size_t workspace_bytes,
                               void* stream);
mdlstm_status mdlstm_unpack_data(int32_t n, void* const* d_examples, const mdlstm_rect* rects,
                                 int32_t canvas_h, int32_t canvas_w, int32_t c, int32_t dt,
                                 const void* d_canvas, void* d_workspace, size_t workspace_bytes,
                                 void* stream);

/* Device workspace needed by mdlstm_forward followed by mdlstm_backward
 * (with the zero-padded copies of a shape between the built ones); 0 when the
 * descriptor is invalid or unsupported, or the canvas or the number of
 * rectangles is out of range (mdlstm_last_error says which). */
size_t mdlstm_workspace_bytes(const mdlstm_layer_desc* desc, int32_t canvas_h, int32_t canvas_w,
                              int32_t n_rects);

/*
 * Forward pass of the four-direction layer over a canvas.
 *
 * Every device pointer of mdlstm_forward and mdlstm_backward must be 16-byte
 * aligned (INVALID_ARG otherwise).
 * d_x: [canvas_h][canvas_w][c_in], storage dtype.
 * d_mask: uint8 [canvas_h][canvas_w]; a cell is valid iff its mask byte is
 *   nonzero AND it lies inside one of the rectangles.
 * rects[n_rects] (host): scheduling rectangles; the recurrence of every
 *   direction restarts at each rectangle edge. Must be inside the canvas,
 *   pairwise disjoint, with h <= MDLSTM_MAX_RECT_H (else BAD_LAYOUT /
 *   UNSUPPORTED). Packed canvases pass the example placements; padded canvases
 *   pass the tiles and carry the true extents in the mask.
 * d_wx: [4][5H][c_in], d_u: [4][5H][2H] (columns 0..H-1 multiply h_L,
 *   H..2H-1 multiply h_T), d_b: [4][5H]; storage dtype; gate order (i, f_L,
 *   f_T, o, g) along 5H.
 * d_y (out): [canvas_h][canvas_w][4H], channel d*H + j; 0 at invalid cells.
 * d_workspace: mdlstm_workspace_bytes(...) bytes; keeps the gates and the cell
 *   state for mdlstm_backward, so it must not be modified in between.
 * Asynchronous on `stream`. Debug mode: with MDLSTM_CHECK_FINITE=1 in the
 * environment the call also counts the non-finite values of y and of the
 * cell state at the cells whose mask byte is set (the plain cell's state can
 * grow without bound, Section III),
 * waits for the count, and returns MDLSTM_ERR_NUMERIC when it is not zero.
 * Debug mode: with MDLSTM_POISON_WORKSPACE=1 in the environment,
 * mdlstm_forward, mdlstm_backward and the head calls first fill the
 * floating-point workspace sections they write before reading (gates, cell
 * states, partial sums; all bits set, NaN in every storage type) so that a
 * read of a value the call did not write shows as NaN in the results; index
 * sections are not touched. Results are identical with and without it.
 */
mdlstm_status mdlstm_forward(const mdlstm_layer_desc* desc, int32_t canvas_h, int32_t canvas_w,
                             const void* d_x, const uint8_t* d_mask,
                             int32_t n_rects, const mdlstm_rect* rects,
                             const void* d_wx, const void* d_u, const void* d_b,
                             void* d_y, void* d_workspace, size_t workspace_bytes, void* stream);

/*
 * The same forward pass with the wavefront run as one kernel launch per local
 * anti-diagonal (launch s advances every unit by its diagonal s, reading the
 * state of diagonal s - 1 back from y and the workspace) instead of one
 * persistent launch: the alternative schedule of Section IV-A, kept for
 * comparison. Same arguments, contract and results (bit for bit) as
 * mdlstm_forward. The launches are recorded once into a HIP graph, which is
 * replayed while the arguments (pointers, sizes, rectangles) stay the same; the
 * graph of the last call is kept per calling thread until the next call with
 * different arguments.
 */
mdlstm_status mdlstm_forward_stepwise(const mdlstm_layer_desc* desc, int32_t canvas_h, int32_t canvas_w,
                                      const void* d_x, const uint8_t* d_mask,
                                      int32_t n_rects, const mdlstm_rect* rects,
                                      const void* d_wx, const void* d_u, const void* d_b,
                                      void* d_y, void* d_workspace, size_t workspace_bytes, void* stream);

/*
 * Backward pass: gradients of L = sum(Y * dY) after an mdlstm_forward with the
 * same arguments and workspace (reverse anti-diagonal sweep, then weight and
 * input gradient reductions).
 * d_y: the forward output; d_dy: [canvas_h][canvas_w][4H], ignored at invalid cells.
 * d_dx (out): [canvas_h][canvas_w][c_in] storage dtype, 0 at invalid cells.
 * d_dwx [4][5H][c_in], d_du [4][5H][2H], d_db [4][5H] (out, fp32): sums over
 *   all valid cells, OVERWRITTEN (not accumulated); fixed reduction order, so
 *   repeated calls give bitwise-identical results.
 * The gates saved in the workspace are overwritten by their gradients. The
 * rectangle ids the forward call staged in the workspace are reused when the
 * layer shape, canvas and rectangles are the same (the library remembers, per
 * workspace address, what the last forward call staged there).
 * Asynchronous on `stream`.
 */
mdlstm_status mdlstm_backward(const mdlstm_layer_desc* desc, int32_t canvas_h, int32_t canvas_w,
                              const void* d_x, const uint8_t* d_mask,
                              int32_t n_rects, const mdlstm_rect* rects,
                              const void* d_wx, const void* d_u, const void* d_b,
                              const void* d_y, const void* d_dy,
                              void* d_dx, float* d_dwx, float* d_du, float* d_db,
                              void* d_workspace, size_t workspace_bytes, void* stream);

/*
 * 1 if mdlstm_backward computes the input and weight gradients of this layer
 * shape in one kernel (reading the gate gradients once), 0 if in two (input
 * gradient, then weight gradients), -1 for a descriptor mdlstm_backward
 * refuses. Host-only; for profilers that attribute time to the kernels.
 */
int32_t mdlstm_gradients_fused(const mdlstm_layer_desc* desc);

/*
 * Stack glue (Section V-B, Fig. 1): a multi-layer network keeps every layer
 * on a packed canvas. Between two MDLSTM layers a block-strided convolution
 * (stride equal to its bh x bw kernel, so blocks never overlap) with tanh maps
 * one layer's output canvas onto the next layer's input canvas, where each
 * example occupies a rectangle bh times lower and bw times narrower (packed
 * again with mdlstm_pack_layout). It is grouped by scan direction: group d
 * reads the H channels d*H + j of the block's pixels, input index
 * (dy*bw + dx)*H + j, and writes og channels d*og + o:
 *   out[p'][d*og + o] = tanh(b[d][o] + sum_{dy,dx,j} W[d][o][(dy*bw+dx)*H + j]
 *                                      * y[pixel (by*bh + dy, bx*bw + dx)][d*H + j])
 * All glue tensors are fp32. The convolutions support bh x bw = 2 x 4 (the
 * paper's block), hidden in {4, 8, 16, 32, 64} and og in {4, 8, 16, 32} with
 * 4*og*bh*bw*hidden <= 16384 (else UNSUPPORTED).
 */

/* Workspace of mdlstm_pack_blocks (hidden = og = 0) and of the block
 * convolutions for n examples. */
size_t mdlstm_blocks_workspace_bytes(int32_t n, int32_t hidden, int32_t og);

/*
 * Block reshape of the stack input: image k (device, HWC fp32
 * [rects[k].h*bh][rects[k].w*bw][c]) becomes [rects[k].h][rects[k].w][bh*bw*c],
 * channel (dy*bw + dx)*c + ch, written into rectangle rects[k] of d_canvas
 * [canvas_h][canvas_w][bh*bw*c]; the rest of the canvas is set to zero.
 * d_images: host array of n device pointers. Rectangles must be disjoint and
 * inside the canvas (BAD_LAYOUT).
 */
mdlstm_status mdlstm_pack_blocks(int32_t n, const float* const* d_images, int32_t c, int32_t bh, int32_t bw,
                                 const mdlstm_rect* rects, int32_t canvas_h, int32_t canvas_w, float* d_canvas,
                                 void* d_workspace, size_t workspace_bytes, void* stream);

/*
 * Grouped block convolution forward. in_rects[k] (host) is example k on the
 * input canvas d_y [in_h][in_w][4*hidden]; out_rects[k] (host) on the output
 * canvas d_out [out_h][out_w][4*og], with in_rects[k].h == bh*out_rects[k].h
 * and in_rects[k].w == bw*out_rects[k].w (BAD_LAYOUT otherwise). d_w
 * [4][og][bh*bw*hidden], d_b [4][og]. d_out is overwritten: the formula above
 * inside the output rectangles, zero elsewhere.
 */
mdlstm_status mdlstm_block_conv_forward(int32_t n, int32_t hidden, int32_t og, int32_t bh, int32_t bw,
                                        const mdlstm_rect* in_rects, int32_t in_h, int32_t in_w, const float* d_y,
                                        const float* d_w, const float* d_b, const mdlstm_rect* out_rects,
                                        int32_t out_h, int32_t out_w, float* d_out, void* d_workspace,
                                        size_t workspace_bytes, void* stream);

/*
 * Grouped block convolution backward: gradients of sum(out * dout).
 * d_out: the forward output; d_dout: its gradient (read inside the output
 * rectangles only). d_dy (out) [in_h][in_w][4*hidden]: input gradient inside
 * the input rectangles, zero elsewhere. d_dw [4][og][bh*bw*hidden] and d_db
 * [4][og] (out): OVERWRITTEN, summed over all blocks of all examples in a fixed
 * order (bitwise reproducible).
 */
mdlstm_status mdlstm_block_conv_backward(int32_t n, int32_t hidden, int32_t og, int32_t bh, int32_t bw,
                                         const mdlstm_rect* in_rects, int32_t in_h, int32_t in_w, const float* d_y,
                                         const float* d_w, const mdlstm_rect* out_rects, int32_t out_h,
                                         int32_t out_w, const float* d_out, const float* d_dout, float* d_dy,
                                         float* d_dw, float* d_db, void* d_workspace, size_t workspace_bytes,
                                         void* stream);

/*
 * Output layer and CTC loss (Section II, Overview: the model ends in a
 * fully-connected layer shared across the four directions and is trained with
 * connectionist temporal classification; Section V-B: that layer is the 1 x 1
 * case of the block-strided layers, so it runs on the packed canvas).
 *
 * For example i at rects[i] = (y0, x0, h, w) of the last MDLSTM layer's output
 * canvas d_y [canvas_h][canvas_w][4*hidden] (channel d*hidden + j), frame
 * t = 0 .. w - 1 is canvas column x0 + t and
 *   logits[off_i + t][k] = sum_{y < h} sum_{d < 4} (W h_d(y0 + y, x0 + t) + b)[k]
 * with the shared W [classes][hidden], b [classes]: the layer applied to every
 * cell of every direction, summed over the directions and the example's rows.
 * off_i = w_0 + ... + w_{i-1}: frames are stored example after example, in
 * the order of rects. Class 0 is the CTC blank. All tensors are fp32.
 * Built: hidden a multiple of 4 in [4, 64], 2 <= classes <= 128.
 */
typedef struct {
    int32_t hidden;
    int32_t classes;
} mdlstm_head_desc;

/* Workspace of the head calls for these examples: with label_lens NULL, what
 * mdlstm_head_forward and mdlstm_head_backward need; with the label lengths,
 * what mdlstm_ctc_loss needs as well (one workspace serves all three). 0 when
 * the descriptor, a rectangle or a label length (0 to min(960, the example's
 * width)) is invalid. */
size_t mdlstm_head_workspace_bytes(const mdlstm_head_desc* desc, int32_t n, const mdlstm_rect* rects,
                                   const int32_t* label_lens);

/*
 * logits (out, device) [frames][classes] as above, frames = sum of rects[i].w.
 * rects (host): inside the canvas and pairwise disjoint (BAD_LAYOUT). The
 * per-frame sums over rows and directions stay in the workspace for
 * mdlstm_head_backward, which must follow before the workspace is reused for
 * another forward call. Asynchronous on `stream`.
 */
mdlstm_status mdlstm_head_forward(const mdlstm_head_desc* desc, int32_t canvas_h, int32_t canvas_w,
                                  const float* d_y, int32_t n, const mdlstm_rect* rects,
                                  const float* d_w, const float* d_b, float* d_logits,
                                  void* d_workspace, size_t workspace_bytes, void* stream);

/*
 * CTC loss (Graves et al. 2006) of every example and its gradient with respect
 * to the logits, computed in double precision.
 * label_lens[n], labels (host): example i's target sequence is the next
 * label_lens[i] entries of labels, each a class in [1, classes); at most 960
 * labels per example (UNSUPPORTED), and the sequence must fit its frames:
 * label_lens[i] + (number of adjacent repeats) <= rects[i].w (INVALID_ARG
 * otherwise, as no frame path would exist).
 * d_losses (out) [n]: -ln p(label_i | frames of example i).
 * d_dlogits (out) [frames][classes]: gradient of sum_i loss_i.
 * The workspace must hold mdlstm_head_workspace_bytes with the label lengths.
 * Asynchronous on `stream`.
 */
mdlstm_status mdlstm_ctc_loss(const mdlstm_head_desc* desc, int32_t n, const mdlstm_rect* rects,
                              const int32_t* label_lens, const int32_t* labels, const float* d_logits,
                              float* d_losses, float* d_dlogits, void* d_workspace, size_t workspace_bytes,
                              void* stream);

/*
 * Gradients of sum(logits * dlogits) after mdlstm_head_forward on the same
 * workspace: d_dy (out) [canvas_h][canvas_w][4*hidden] holds W^T dlogits[off_i
 * + t] at every row of example i's column x0 + t, in every direction, and zero
 * outside the rectangles (the upstream gradient of the MDLSTM layer's
 * backward); d_dw [classes][hidden] and d_db [classes] (out) are OVERWRITTEN,
 * summed over all frames in a fixed order. Asynchronous on `stream`.
 */
mdlstm_status mdlstm_head_backward(const mdlstm_head_desc* desc, int32_t canvas_h, int32_t canvas_w, int32_t n,
                                   const mdlstm_rect* rects, const float* d_w, const float* d_dlogits,
                                   float* d_dy, float* d_dw, float* d_db,
                                   void* d_workspace, size_t workspace_bytes, void* stream);

/* Message for the last non-OK status returned on the calling thread. */
const char* mdlstm_last_error(void);

/*
 * Optional kernel-boundary timing (profiling hook, off by default).
 * events[n] (host array of hipEvent_t handles owned by the caller). While set,
 * mdlstm_forward and mdlstm_backward called on this thread record them on
 * their stream at kernel boundaries:
 *   [0] before the projection   [1] after the projection   [2] after zeroing
 *   invalid output rows (the persistent forward wavefront zeroes them itself
 *   when the batch has at least a unit per CU; then [2] follows [1] directly)
 *   [3] after the forward wavefront
 *   [4] before the backward wavefront  [5] after it  [6] after the input
 *   gradient  [7] after the weight gradients. Where one kernel computes both
 *   gradients (fp32 (hidden, c_in) in {(4, 4), (4, 8), (8, 8), (16, 8), (16, 16),
 *   (32, 16), (32, 32)}, bf16 (32, 16) and (32, 32)) [6] is recorded
 *   right after [5] and [6]..[7] spans the fused kernel.
 * n must be 0 (disable) or 8; a NULL entry is not recorded (each record
 * costs the stream a few microseconds, so a caller timing whole steps records
 * only the boundaries it needs). The handles must stay valid while set.
 */
mdlstm_status mdlstm_set_phase_events(int32_t n, void* const* events);

#ifdef __cplusplus
}
#endif

#endif /* MDLSTM_H */
