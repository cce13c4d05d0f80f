// Internal launcher interface between the C-ABI host layer and the HIP kernels.
// All launchers enqueue on `stream` and return the hipError_t of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace mdl {

struct LayerGeom {
    int c_in, hidden, dtype;  // dtype: 0 fp32, 1 bf16
    int canvas_h, canvas_w;
    int64_t n_cells;          // canvas_h * canvas_w
};

// --- packing -------------------------------------------------------------
// Placement of n examples; sizes in d_hw[2n] (heights then widths), result
// d_rects[4n] (y0,x0,h,w by original index) and d_rects[4n] = canvas_h.
hipError_t launch_pack_place(int n, int canvas_w, const int32_t* d_hw, int32_t* d_out,
                             int32_t* d_scratch, hipStream_t s);
// mask[canvas] = 1 inside any of the rects, else 0.
hipError_t launch_mask(int n, const int32_t* d_rects, int canvas_h, int canvas_w, uint8_t* d_mask,
                       hipStream_t s);
// rect id per cell (-1 outside every rect); also zeroes the two counters at
// d_zero2 (the wavefront unit queue) when n > 0 and d_zero2 is not NULL.
hipError_t launch_rect_ids(int n, const int32_t* d_rects, int canvas_h, int canvas_w, int32_t* d_rid,
                           unsigned* d_zero2, hipStream_t s);
// scatter/gather of n HWC examples of c channels, element size esize (2 or 4).
hipError_t launch_scatter(int n, const void* const* d_ptrs, const int32_t* d_rects, int canvas_h,
                          int canvas_w, int c, int esize, void* d_canvas, int max_h, hipStream_t s);
hipError_t launch_gather(int n, void* const* d_ptrs, const int32_t* d_rects, int canvas_w, int c,
                         int esize, const void* d_canvas, int max_h, hipStream_t s);

// --- forward ---------------------------------------------------------------
// Z[p][20H] = Wx_all[20H][C] x[p] + b_all, for the cells of every 64-cell
// chunk that holds a cell of a rectangle (d_rid: rectangle id per cell, -1
// outside; NULL: every chunk).
hipError_t launch_projection(const LayerGeom& g, const void* d_x, const void* d_wx, const void* d_b,
                             const int32_t* d_rid, void* d_z, hipStream_t s);
// Count the non-finite values of n elements (dtype 0 fp32, 1 bf16) into
// *d_count (added to; the caller zeroes it).
hipError_t launch_fill_u32(void* d, int64_t n_words, uint32_t v, hipStream_t s);
// Block remap between a layer's own sizes and its padded built sizes (k_pad.hip):
// dst[o][rb*rd + j][cb*cd + k] = src[o][rb*rs + j][cb*cs + k] where j < min(rs, rd) and
// k < min(cs, cd), else 0; es = element bytes (2 or 4).
hipError_t launch_remap(const void* src, void* dst, int es, int64_t outer, int rblocks, int rs, int rd, int cblocks,
                        int cs, int cd, hipStream_t s);
hipError_t launch_count_nonfinite(const void* d, int64_t n_cells, int row, const uint8_t* d_mask, int dtype,
                                  unsigned long long* d_count, hipStream_t s);
// Zero the rows of a [n_cells][width] tensor (storage dtype) whose cell is invalid.
hipError_t launch_zero_invalid(const LayerGeom& g, int width, const uint8_t* d_mask,
                               const int32_t* d_rid, void* d_t, hipStream_t s);
// Forward anti-diagonal wavefront over n_units units (rectangle, direction)
// in the order of d_units. d_queue: two device counters, zero on entry (the
// workgroups take units from the first, a fixed number per CU, and count
// themselves out on the second; the last one out zeroes both again). With
// d_rid set, the output rows of cells outside every rectangle or masked are
// zeroed first.
hipError_t launch_wavefront_fwd(const LayerGeom& g, int nt, int n_units, const int32_t* d_units,
                                const int32_t* d_rects, const uint8_t* d_mask, const int32_t* d_rid,
                                const void* d_u, void* d_z, float* d_c, void* d_y, unsigned* d_queue, hipStream_t s);

// The forward wavefront as one launch per local diagonal (diagonal s of every
// unit in launch s), recorded as a chain of max_steps kernel nodes into an
// instantiated graph; same results as launch_wavefront_fwd.
hipError_t build_wavefront_fwd_graph(const LayerGeom& g, int nt, int n_units, int max_steps, const int32_t* d_units,
                                     const int32_t* d_rects, const uint8_t* d_mask, const void* d_u, void* d_z,
                                     float* d_c, void* d_y, hipGraphExec_t* exec);

// --- backward --------------------------------------------------------------
hipError_t launch_wavefront_bwd(const LayerGeom& g, int nt, int n_units, const int32_t* d_units,
                                const int32_t* d_rects, const uint8_t* d_mask, const void* d_u,
                                const void* d_dy, void* d_z, const float* d_c, unsigned* d_queue, hipStream_t s);
// Input and weight gradients as tiled MFMA products (any built shape), in
// two launches: first a validity byte per cell (d_flags, n_cells bytes),
// Wx_all transposed (d_wxt) and the input gradient; then the weight
// gradients from chunk partials (d_part) summed in a fixed order (it reads
// the validity bytes of the first).
size_t big_flags_bytes(const LayerGeom& g);
size_t big_wxt_bytes(const LayerGeom& g);
size_t big_partial_bytes(const LayerGeom& g);
hipError_t launch_bwd_big_dx(const LayerGeom& g, const void* d_dz, const void* d_wx, const uint8_t* d_mask,
                             const int32_t* d_rid, void* d_dx, uint8_t* d_flags, void* d_wxt, hipStream_t s);
hipError_t launch_bwd_big_dw(const LayerGeom& g, const void* d_dz, const void* d_x, const void* d_y,
                             const uint8_t* d_flags, float* d_part, float* d_dwx, float* d_du, float* d_db,
                             hipStream_t s);
// Input and weight gradients together, staged through LDS by canvas-row
// strips (the shapes strip_supported lists). d_vid: strip_vid_bytes of
// workspace for a validity id per cell.
bool strip_supported(const LayerGeom& g);
size_t strip_partial_bytes(const LayerGeom& g);
size_t strip_vid_bytes(const LayerGeom& g);
hipError_t launch_bwd_strip(const LayerGeom& g, const void* d_dz, const void* d_x, const void* d_y,
                            const void* d_wx, const uint8_t* d_mask, const int32_t* d_rid, int32_t* d_vid,
                            void* d_dx, float* d_part, float* d_dwx, float* d_du, float* d_db, hipStream_t s);

// --- stack glue (block reshape, grouped block convolution) -----------------
// d_blk_off[n + 1]: first block of each example (prefix sum of out_h*out_w).
hipError_t launch_pack_blocks(int n, const float* const* d_imgs, const int32_t* d_blk_off, int total_blocks,
                              const int32_t* d_rects, int canvas_w, int c, int bh, int bw, float* d_canvas,
                              hipStream_t s);
struct ConvArgs {
    int n, total_blocks, hidden, og, bh, bw;
    const int32_t* blk_off;
    const int32_t* in_rects;
    int in_w;
    const int32_t* out_rects;
    int out_w;
    const float* y;     // [in canvas][4H]
    const float* w;     // [4][og][bh*bw*H]
    const float* b;     // [4][og]
    float* out;         // [out canvas][4*og] (forward output; backward input)
    const float* dout;  // backward: gradient of out
    float* dy;          // backward: gradient of y (only rectangle pixels written)
    float* dw;          // backward: [4][og][bh*bw*H]
    float* db;          // backward: [4][og]
    float* partial;     // backward: conv_partial_bytes
};
bool conv_supported(int hidden, int og, int bh, int bw);
int conv_chunks(int total_blocks);
size_t conv_partial_bytes(int hidden, int og, int bh, int bw, int total_blocks);
hipError_t launch_block_conv(bool fwd, const ConvArgs& a, hipStream_t s);
// Fill n floats with zero.
hipError_t launch_zero_f32(float* d, int64_t n, hipStream_t s);

// --- layer with memory-state matrices (fp32, H = 16 or 32) -----------------
struct MemArgs {
    const int32_t* units;   // unit order (4 * rect + direction), one workgroup each
    const int32_t* rects;   // [n_rects][4]
    const uint8_t* mask;
    const float* u;         // [4][5H][2H]
    const float* v;         // [4][3H][2H]
    float* z;               // pre-activations -> activated gates (forward) -> gate gradients (backward)
    float* c;               // cell states [cells][4H]
    float* y;               // forward output [cells][4H]
    const float* dy;        // backward input [cells][4H]
    int canvas_w;
    float* dvpart;          // backward: [units][3H][2H] partials
};
bool mem_supported(const LayerGeom& g);
size_t mem_partial_bytes(const LayerGeom& g, int n_units);
hipError_t launch_wavefront_mem(bool fwd, const LayerGeom& g, int n_units, const MemArgs& a, hipStream_t s);
hipError_t launch_dv_reduce(const LayerGeom& g, int n_units, const int32_t* d_units, const float* d_part, float* d_dv,
                            hipStream_t s);

// --- output layer shared by the directions, row collapse, CTC loss ---------
struct HeadArgs {
    int H, K, canvas_w;
    int n_tiles;                 // tiles of head_tile_frames() frames
    int frames;                  // frames of all examples
    const float* y;              // forward: the last layer's output canvas [canvas][4H]
    const int32_t* rects;        // [n][4] example rectangles on that canvas
    const int32_t* frame_off;    // [n + 1] first frame of each example
    const int32_t* tiles;        // [n_tiles][2] (example, first frame)
    const float* w;              // [K][H]
    const float* b;              // [K]
    float* logits;               // forward output [frames][K]
    float* S;                    // column sums [frames][H + 4], forward output, backward input
    const float* dlogits;        // backward input [frames][K]
    float* dy;                   // backward output canvas [canvas][4H]
    float* part;                 // backward: weight-gradient partials
    float* dw;                   // backward output [K][H]
    float* db;                   // backward output [K]
};
struct CtcArgs {
    int n, K, nm;                // examples, classes, states per lane of the scan (a power of two, 64 nm >= S)
    int64_t frames;
    const int32_t* frame_off;    // [n + 1]
    const int32_t* lab_off;      // [n + 1]
    const int32_t* labels;       // concatenated labels
    const int32_t* occ;          // per label: next occurrence of its class in the example | first-occurrence bit 30
    const float* logits;         // [frames][K]
    double* y;                   // workspace [frames][K]: softmax
    double* am;                  // workspace [frames][64 nm]: forward variables, mantissas
    int32_t* ae;                 //   and exponents
    double* bm;                  // workspace [frames][64 nm]: backward variables, mantissas
    int32_t* be;                 //   and exponents
    float* losses;               // [n]
    float* dlogits;              // [frames][K]
};
int head_tile_frames();
int head_dw_chunk_frames();
size_t head_fwd_lds(int H, int K);
size_t head_bwd_lds(int H, int K);
size_t head_dw_lds(int H, int K);
int ctc_states_per_lane(int max_labels);
hipError_t launch_head_fwd(const HeadArgs& a, hipStream_t s);
hipError_t launch_ctc(const CtcArgs& a, hipStream_t s);
// zeroes the dy canvas (canvas_floats floats), then writes the rectangles
hipError_t launch_head_bwd(const HeadArgs& a, int64_t canvas_floats, hipStream_t s);

}  // namespace mdl
