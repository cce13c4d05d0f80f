// Host side of the C ABI declared in include/mdlstm.h: argument and layout
// validation (always before the first HIP call), workspace planning, unit
// ordering and kernel dispatch.
#include "mdlstm.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

#include "kernels.hpp"

namespace {

thread_local std::string g_last_error;
thread_local hipEvent_t g_phase_events[8];
thread_local bool g_phase_on = false;

hipError_t mark(int i, hipStream_t s) {
    return g_phase_on && g_phase_events[i] ? hipEventRecord(g_phase_events[i], s) : hipSuccess;
}

mdlstm_status fail(mdlstm_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

mdlstm_status device_fail(hipError_t e, const char* where) {
    return fail(MDLSTM_ERR_DEVICE, "%s: %s", where, hipGetErrorString(e));
}

#define HIP_OR_FAIL(expr)                                     \
    do {                                                      \
        hipError_t _e = (expr);                               \
        if (_e != hipSuccess) return device_fail(_e, #expr);  \
    } while (0)

constexpr int32_t kMaxDim = (1 << 21) - 1;  // largest canvas side / example side
constexpr int32_t kMaxPackN = 4096;         // placement keys in LDS; a placed bit per key, 64 per lane
constexpr int32_t kMaxRects = MDLSTM_MAX_RECTS;  // rectangles per call (unit ids 4k + d stay within int32)

size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

// Device buffers are accessed with 16-byte vector loads and stores.
bool misaligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) != 0; }

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// Debug mode of the forward pass: MDLSTM_CHECK_FINITE=1 in the environment
// (read at every call, so a process can switch it on and off).
bool check_finite_requested() {
    const char* v = std::getenv("MDLSTM_CHECK_FINITE");
    return v && v[0] == '1' && v[1] == 0;
}

// Debug mode: MDLSTM_POISON_WORKSPACE=1 fills the floating-point sections of
// a workspace that a call writes before it reads them with NaN (all bits
// set: NaN as fp32, bf16 and fp64) at the start of the call, so that a read
// of anything the call has not written shows in its results. Index and
// offset sections are left alone.
bool poison_requested() {
    const char* v = std::getenv("MDLSTM_POISON_WORKSPACE");
    return v && v[0] == '1' && v[1] == 0;
}

mdlstm_status poison(char* ws, size_t from, size_t to, hipStream_t s) {
    if (to > from) HIP_OR_FAIL(mdl::launch_fill_u32(ws + from, (int64_t)((to - from) / 4), 0xffffffffu, s));
    return MDLSTM_OK;
}

// ---------------------------------------------------------------------------
// Layer descriptor and workspace plan.
// ---------------------------------------------------------------------------
// A shape the kernels are built for.
mdlstm_status check_built(const mdlstm_layer_desc* d) {
    if (!d) return fail(MDLSTM_ERR_INVALID_ARG, "desc is NULL");
    if (d->dtype != MDLSTM_F32 && d->dtype != MDLSTM_BF16)
        return fail(MDLSTM_ERR_INVALID_ARG, "dtype %d is not MDLSTM_F32 or MDLSTM_BF16", d->dtype);
    if (d->c_in < 1 || d->hidden < 1) return fail(MDLSTM_ERR_INVALID_ARG, "c_in and hidden must be positive");
    if (d->memory_states != 0 && d->memory_states != 1)
        return fail(MDLSTM_ERR_INVALID_ARG, "memory_states %d is not 0 or 1", d->memory_states);
    if (d->memory_states && (d->dtype != MDLSTM_F32 || (d->hidden != 16 && d->hidden != 32)))
        return fail(MDLSTM_ERR_UNSUPPORTED, "memory-state matrices are built for F32 with hidden 16 or 32");
    if (d->dtype == MDLSTM_F32) {
        const int h = d->hidden;
        if (!(h == 4 || h == 8 || h == 16 || h == 32 || h == 64))
            return fail(MDLSTM_ERR_UNSUPPORTED, "fp32 hidden size %d not built (4, 8, 16, 32, 64)", h);
        if (d->c_in % 4 || d->c_in < 4 || d->c_in > 256)
            return fail(MDLSTM_ERR_UNSUPPORTED, "fp32 c_in %d must be a multiple of 4 in [4, 256]", d->c_in);
    } else {
        const int h = d->hidden;
        if (!(h == 32 || h == 64 || h == 128))
            return fail(MDLSTM_ERR_UNSUPPORTED, "bf16 hidden size %d not built (32, 64, 128)", h);
        if (d->c_in % 8 || d->c_in < 8 || d->c_in > 256)
            return fail(MDLSTM_ERR_UNSUPPORTED, "bf16 c_in %d must be a multiple of 8 in [8, 256]", d->c_in);
    }
    return MDLSTM_OK;
}

// The kernels' shape for a layer: the hidden size padded to the next built
// size (fp32 4, 8, 16, 32, 64; bf16 32, 64, 128; with memory-state matrices at
// least 16), c_in to a multiple of the MFMA K step (4 fp32, 8 bf16). Padded
// hidden units and input channels carry zero weights, which leaves the
// layer's results unchanged (k_pad.hip).
mdlstm_status inner_desc(const mdlstm_layer_desc* d, mdlstm_layer_desc* in) {
    if (!d) return fail(MDLSTM_ERR_INVALID_ARG, "desc is NULL");
    if (d->dtype != MDLSTM_F32 && d->dtype != MDLSTM_BF16)
        return fail(MDLSTM_ERR_INVALID_ARG, "dtype %d is not MDLSTM_F32 or MDLSTM_BF16", d->dtype);
    if (d->c_in < 1 || d->hidden < 1) return fail(MDLSTM_ERR_INVALID_ARG, "c_in and hidden must be positive");
    if (d->memory_states != 0 && d->memory_states != 1)
        return fail(MDLSTM_ERR_INVALID_ARG, "memory_states %d is not 0 or 1", d->memory_states);
    const bool f32 = d->dtype == MDLSTM_F32;
    const int hmax = f32 ? 64 : 128;
    if (d->hidden > hmax) return fail(MDLSTM_ERR_UNSUPPORTED, "%s hidden size %d: at most %d", f32 ? "fp32" : "bf16",
                                      d->hidden, hmax);
    if (d->c_in > 256) return fail(MDLSTM_ERR_UNSUPPORTED, "c_in %d: at most 256", d->c_in);
    int hp = f32 ? 4 : 32;
    while (hp < d->hidden) hp *= 2;
    if (d->memory_states && f32) hp = std::max(hp, 16);
    const int kq = f32 ? 4 : 8;
    *in = mdlstm_layer_desc{(d->c_in + kq - 1) / kq * kq, hp, d->dtype, d->memory_states};
    return check_built(in);
}

bool same_shape(const mdlstm_layer_desc* a, const mdlstm_layer_desc& b) {
    return a->c_in == b.c_in && a->hidden == b.hidden;
}

struct Plan {
    size_t z, c, rid, rects, units, part, flags, wxt, dvpart, queue, check, total;
};

mdl::LayerGeom geom(const mdlstm_layer_desc* d, int32_t ch, int32_t cw) {
    mdl::LayerGeom g;
    g.c_in = d->c_in;
    g.hidden = d->hidden;
    g.dtype = d->dtype;
    g.canvas_h = ch;
    g.canvas_w = cw;
    g.n_cells = (int64_t)ch * cw;
    return g;
}

Plan plan(const mdlstm_layer_desc* d, int32_t ch, int32_t cw, int32_t nr) {
    const mdl::LayerGeom g = geom(d, ch, cw);
    const size_t es = d->dtype == MDLSTM_BF16 ? 2 : 4;
    const size_t H = (size_t)d->hidden;
    Plan p;
    size_t off = 0;
    p.z = off;
    off += align_up((size_t)g.n_cells * 20 * H * es);
    p.c = off;
    off += align_up((size_t)g.n_cells * 4 * H * 4);
    p.rid = off;
    off += align_up((size_t)g.n_cells * 4);
    p.rects = off;
    off += align_up((size_t)(nr > 0 ? nr : 1) * 16);
    p.units = off;
    off += align_up((size_t)(nr > 0 ? nr : 1) * 16);
    p.part = off;
    const bool strip = mdl::strip_supported(g);
    off += align_up(strip ? mdl::strip_partial_bytes(g) : mdl::big_partial_bytes(g));
    p.flags = off;  // tiled gradient path: a validity byte per cell; strip path: a validity id per cell
    off += align_up(strip ? mdl::strip_vid_bytes(g) : mdl::big_flags_bytes(g));
    p.wxt = off;
    off += strip ? 0 : align_up(mdl::big_wxt_bytes(g));
    p.dvpart = off;  // memory-state matrices: a dV partial per unit
    off += d->memory_states ? align_up(mdl::mem_partial_bytes(g, 4 * (nr > 0 ? nr : 1))) : 0;
    p.queue = off;  // unit queue: next unit, workgroups done
    off += align_up(8);
    p.check = off;  // non-finite count of the debug mode
    off += align_up(8);
    p.total = off;
    return p;
}

// Sections of the padded copies at the front of the workspace (the kernels'
// plan follows them); none when the layer is a built shape. x and dx are
// copied only when c_in is padded, y and dy only when the hidden size is.
struct PadPlan {
    bool active = false, pad_c = false, pad_h = false;
    size_t wx = 0, u = 0, b = 0, x = 0, y = 0, dy = 0, dx = 0, dwx = 0, du = 0, db = 0, total = 0;
};

PadPlan pad_plan(const mdlstm_layer_desc* d, const mdlstm_layer_desc& in, int32_t ch, int32_t cw) {
    PadPlan q;
    if (same_shape(d, in)) return q;
    q.active = true;
    q.pad_c = in.c_in != d->c_in;
    q.pad_h = in.hidden != d->hidden;
    const size_t es = d->dtype == MDLSTM_BF16 ? 2 : 4, cells = (size_t)ch * (size_t)cw;
    const size_t H = (size_t)in.hidden, C = (size_t)in.c_in;
    const size_t nu = 4 * 5 * H * 2 * H + (d->memory_states ? 4 * 3 * H * 2 * H : 0);
    size_t off = 0;
    q.wx = off;
    off += align_up(4 * 5 * H * C * es);
    q.u = off;
    off += align_up(nu * es);
    q.b = off;
    off += align_up(4 * 5 * H * es);
    q.x = off;
    off += q.pad_c ? align_up(cells * C * es) : 0;
    q.dx = off;
    off += q.pad_c ? align_up(cells * C * es) : 0;
    q.y = off;
    off += q.pad_h ? align_up(cells * 4 * H * es) : 0;
    q.dy = off;
    off += q.pad_h ? align_up(cells * 4 * H * es) : 0;
    q.dwx = off;
    off += align_up(4 * 5 * H * C * 4);
    q.du = off;
    off += align_up(nu * 4);
    q.db = off;
    off += align_up(4 * 5 * H * 4);
    q.total = off;
    return q;
}

// ---------------------------------------------------------------------------
// Rectangle validation: inside the canvas, height within the kernel limit,
// pairwise disjoint. Sorted by y0, a rectangle can only overlap those that
// start fewer than MDLSTM_MAX_RECT_H rows before it.
// ---------------------------------------------------------------------------
mdlstm_status check_rects(int32_t n, const mdlstm_rect* r, int32_t ch, int32_t cw, int32_t* max_h,
                          int32_t limit_h = MDLSTM_MAX_RECT_H) {
    if (n < 0) return fail(MDLSTM_ERR_INVALID_ARG, "n_rects is negative");
    if (n > kMaxRects) return fail(MDLSTM_ERR_UNSUPPORTED, "%d rectangles; at most %d per call", n, kMaxRects);
    if (n > 0 && !r) return fail(MDLSTM_ERR_INVALID_ARG, "rects is NULL");
    int32_t mh = 0;
    for (int32_t k = 0; k < n; ++k) {
        const mdlstm_rect& a = r[k];
        if (a.h < 1 || a.w < 1) return fail(MDLSTM_ERR_BAD_LAYOUT, "rect %d has size %dx%d", k, a.h, a.w);
        if (a.y0 < 0 || a.x0 < 0 || (int64_t)a.y0 + a.h > ch || (int64_t)a.x0 + a.w > cw)
            return fail(MDLSTM_ERR_BAD_LAYOUT, "rect %d (%d,%d,%d,%d) leaves the %dx%d canvas", k, a.y0, a.x0, a.h,
                        a.w, ch, cw);
        if (a.h > limit_h)
            return fail(MDLSTM_ERR_UNSUPPORTED, "rect %d is %d high; at most %d is supported", k, a.h, limit_h);
        mh = std::max(mh, a.h);
    }
    std::vector<int32_t> order(n);
    for (int32_t k = 0; k < n; ++k) order[k] = k;
    std::sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
        return r[a].y0 != r[b].y0 ? r[a].y0 < r[b].y0 : a < b;
    });
    for (int32_t i = 0; i < n; ++i) {
        const mdlstm_rect& a = r[order[i]];
        for (int32_t j = i + 1; j < n; ++j) {
            const mdlstm_rect& b = r[order[j]];
            if (b.y0 >= a.y0 + a.h) break;
            if (b.x0 < a.x0 + a.w && a.x0 < b.x0 + b.w)
                return fail(MDLSTM_ERR_BAD_LAYOUT, "rects %d and %d overlap", order[i], order[j]);
        }
    }
    *max_h = mh;
    return MDLSTM_OK;
}

// Units (rect, direction) ordered longest first (h + w - 1 steps), so the
// in-order workgroup dispatcher starts the critical-path units first.
std::vector<int32_t> unit_order(int32_t n, const mdlstm_rect* r) {
    std::vector<int32_t> u(4 * (size_t)n);
    for (int32_t k = 0; k < n; ++k)
        for (int d = 0; d < 4; ++d) u[4 * (size_t)k + d] = 4 * k + d;
    std::stable_sort(u.begin(), u.end(), [&](int32_t a, int32_t b) {
        return r[a >> 2].h + r[a >> 2].w > r[b >> 2].h + r[b >> 2].w;
    });
    return u;
}

struct Common {
    mdl::LayerGeom g;
    Plan p;
    int nt;
    int memory;
    char* ws;
};

mdlstm_status prepare(const mdlstm_layer_desc* desc, int32_t ch, int32_t cw, const void* d_x, const uint8_t* d_mask,
                      int32_t n_rects, const mdlstm_rect* rects, const void* d_wx, const void* d_u,
                      const void* d_b, void* d_workspace, size_t ws_bytes, Common* out) {
    mdlstm_status st = check_built(desc);
    if (st != MDLSTM_OK) return st;
    if (ch < 0 || cw < 0 || ch > kMaxDim || cw > kMaxDim)
        return fail(MDLSTM_ERR_INVALID_ARG, "canvas %dx%d out of range", ch, cw);
    int32_t max_h = 0;
    st = check_rects(n_rects, rects, ch, cw, &max_h);
    if (st != MDLSTM_OK) return st;
    const int64_t cells = (int64_t)ch * cw;
    if (cells > 0 && (!d_x || !d_mask)) return fail(MDLSTM_ERR_INVALID_ARG, "x or mask is NULL");
    if (!d_wx || !d_u || !d_b) return fail(MDLSTM_ERR_INVALID_ARG, "a weight pointer is NULL");
    Plan p = plan(desc, ch, cw, n_rects);
    if (!d_workspace) return fail(MDLSTM_ERR_INVALID_ARG, "workspace is NULL");
    if (misaligned(d_x) || misaligned(d_wx) || misaligned(d_u) || misaligned(d_b) || misaligned(d_workspace))
        return fail(MDLSTM_ERR_INVALID_ARG, "x, weights and workspace must be 16-byte aligned");
    if (ws_bytes < p.total)
        return fail(MDLSTM_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", ws_bytes, p.total);
    out->g = geom(desc, ch, cw);
    out->p = p;
    out->memory = desc->memory_states;
    out->nt = (max_h + 15) / 16;
    if (out->nt < 1) out->nt = 1;
    out->ws = static_cast<char*>(d_workspace);
    return MDLSTM_OK;
}

// Identity of what a workspace holds after layout staging: the layer shape,
// canvas and rectangles (with a hash of the rectangle list).
struct StagedKey {
    int32_t c_in = 0, hidden = 0, dtype = 0, memory = 0, canvas_h = 0, canvas_w = 0, n_rects = -1, device = -1;
    uint64_t hash = 0;
    bool operator==(const StagedKey& o) const {
        return c_in == o.c_in && hidden == o.hidden && dtype == o.dtype && memory == o.memory && canvas_h == o.canvas_h &&
               canvas_w == o.canvas_w && n_rects == o.n_rects && device == o.device && hash == o.hash;
    }
};

StagedKey staged_key(const Common& c, int32_t n_rects, const mdlstm_rect* rects) {
    StagedKey k;
    k.c_in = c.g.c_in;
    k.hidden = c.g.hidden;
    k.dtype = c.g.dtype;
    k.memory = c.memory;
    k.canvas_h = c.g.canvas_h;
    k.canvas_w = c.g.canvas_w;
    k.n_rects = n_rects;
    if (hipGetDevice(&k.device) != hipSuccess) k.device = -2;
    uint64_t h = 1469598103934665603ull;  // FNV-1a over the rectangle bytes
    const unsigned char* b = reinterpret_cast<const unsigned char*>(rects);
    for (size_t i = 0; i < (size_t)(n_rects > 0 ? n_rects : 0) * sizeof(mdlstm_rect); ++i) {
        h ^= b[i];
        h *= 1099511628211ull;
    }
    k.hash = h;
    return k;
}

// Workspaces staged by the last forward call on them. A backward call, whose
// workspace must be untouched since its forward, skips restaging when its
// layout is the one staged there.
std::mutex g_staged_mu;
std::unordered_map<uintptr_t, StagedKey> g_staged;

mdlstm_status stage_layout(const Common& c, int32_t n_rects, const mdlstm_rect* rects, bool reuse, hipStream_t s) {
    const StagedKey key = staged_key(c, n_rects, rects);
    const uintptr_t ws = reinterpret_cast<uintptr_t>(c.ws);
    if (reuse) {
        std::lock_guard<std::mutex> lock(g_staged_mu);
        auto it = g_staged.find(ws);
        if (it != g_staged.end() && it->second == key) return MDLSTM_OK;
    }
    if (n_rects > 0) {
        // rectangles and unit order in one copy (adjacent workspace sections)
        std::vector<int32_t> units = unit_order(n_rects, rects);
        const size_t ubytes = units.size() * 4, span = c.p.units - c.p.rects + ubytes;
        std::vector<unsigned char> host(span, 0);
        std::memcpy(host.data(), rects, (size_t)n_rects * 16);
        std::memcpy(host.data() + (c.p.units - c.p.rects), units.data(), ubytes);
        HIP_OR_FAIL(hipMemcpyAsync(c.ws + c.p.rects, host.data(), span, hipMemcpyHostToDevice, s));
    }
    HIP_OR_FAIL(mdl::launch_rect_ids(n_rects, reinterpret_cast<const int32_t*>(c.ws + c.p.rects), c.g.canvas_h,
                                     c.g.canvas_w, reinterpret_cast<int32_t*>(c.ws + c.p.rid),
                                     reinterpret_cast<unsigned*>(c.ws + c.p.queue), s));
    std::lock_guard<std::mutex> lock(g_staged_mu);
    if (g_staged.size() >= 4096) g_staged.clear();  // bound the table; a miss only restages
    g_staged[ws] = key;
    return MDLSTM_OK;
}

size_t pack_ws_bytes(int32_t n) {
    size_t nn = (size_t)(n > 0 ? n : 1);
    return align_up(nn * 8) + align_up(nn * 16) + align_up((6 * nn + 1) * 4);
}

// Size checks shared by the two placement entry points (no HIP call).
mdlstm_status check_pack_sizes(int32_t n, const int32_t* heights, const int32_t* widths, int32_t canvas_w,
                               mdlstm_rect* rects, int32_t* canvas_h) {
    if (n < 0) return fail(MDLSTM_ERR_INVALID_ARG, "n is negative");
    if (n > kMaxPackN) return fail(MDLSTM_ERR_UNSUPPORTED, "at most %d examples per packing call", kMaxPackN);
    if (!canvas_h) return fail(MDLSTM_ERR_INVALID_ARG, "canvas_h is NULL");
    if (n > 0 && (!heights || !widths || !rects)) return fail(MDLSTM_ERR_INVALID_ARG, "size or rect array is NULL");
    if (canvas_w < 1 || canvas_w > kMaxDim) return fail(MDLSTM_ERR_INVALID_ARG, "canvas width %d out of range", canvas_w);
    for (int32_t k = 0; k < n; ++k) {
        if (heights[k] < 1 || widths[k] < 1 || heights[k] > kMaxDim || widths[k] > kMaxDim)
            return fail(MDLSTM_ERR_INVALID_ARG, "example %d has size %dx%d", k, heights[k], widths[k]);
        if (widths[k] > canvas_w)
            return fail(MDLSTM_ERR_TOO_WIDE, "example %d is %d wide; the canvas is %d", k, widths[k], canvas_w);
    }
    // total canvas height must stay addressable
    int64_t hsum = 0;
    for (int32_t k = 0; k < n; ++k) hsum += (int64_t)heights[k] + 1;
    if (hsum > kMaxDim) return fail(MDLSTM_ERR_UNSUPPORTED, "packed canvas could exceed %d rows", kMaxDim);
    if (n == 0) *canvas_h = 0;
    return MDLSTM_OK;
}

// Placement kernel, then (with d_mask) the mask. d_hw: 2n device int32 (the
// sizes, uploaded here); d_out: 4n + 1 device int32 (the placement, then the
// canvas height), read again by the mask kernel; host: 6n + 1 host int32 of
// staging. Waits for the placement (rects and canvas_h are host outputs); the
// mask kernel stays queued on s.
mdlstm_status place_and_mask(int32_t n, const int32_t* heights, const int32_t* widths, int32_t canvas_w,
                             mdlstm_rect* rects, int32_t* canvas_h, uint8_t* d_mask, size_t mask_bytes,
                             int32_t* d_hw, int32_t* d_out, int32_t* host, hipStream_t s) {
    const size_t nn = (size_t)n;
    std::copy(heights, heights + n, host);
    std::copy(widths, widths + n, host + nn);
    HIP_OR_FAIL(hipMemcpyAsync(d_hw, host, 2 * nn * 4, hipMemcpyHostToDevice, s));
    HIP_OR_FAIL(mdl::launch_pack_place(n, canvas_w, d_hw, d_out, nullptr, s));
    int32_t* res = host + 2 * nn;
    HIP_OR_FAIL(hipMemcpyAsync(res, d_out, (4 * nn + 1) * 4, hipMemcpyDeviceToHost, s));
    HIP_OR_FAIL(hipStreamSynchronize(s));
    for (size_t k = 0; k < nn; ++k) {
        rects[k].y0 = res[4 * k];
        rects[k].x0 = res[4 * k + 1];
        rects[k].h = res[4 * k + 2];
        rects[k].w = res[4 * k + 3];
    }
    *canvas_h = res[4 * nn];
    if (d_mask) {
        const size_t need = (size_t)(*canvas_h) * (size_t)canvas_w;
        if (mask_bytes < need)
            return fail(MDLSTM_ERR_WORKSPACE, "mask of %zu bytes, %zu needed", mask_bytes, need);
        HIP_OR_FAIL(mdl::launch_mask(n, d_out, *canvas_h, canvas_w, d_mask, s));
    }
    return MDLSTM_OK;
}

// ---------------------------------------------------------------------------
// Scratch of the allocation-free placement (mdlstm_pack_layout_noalloc): the
// sizes (2n words) and the placement (4n + 1 words) of at most
// MDLSTM_NOALLOC_MAX_N examples in a file-scope device array, which every GPU
// holds its own copy of. Host code never passes the array's name to a kernel
// or a copy (on the host it is only a stand-in for the symbol): the device
// address comes from hipGetSymbolAddress, taken once per device with that
// device current on the first call there, and kept per device.
// ---------------------------------------------------------------------------
constexpr size_t kScratchWords = 6 * (size_t)MDLSTM_NOALLOC_MAX_N + 1;
static_assert(MDLSTM_NOALLOC_MAX_N <= kMaxPackN, "the allocation-free placement shares the placement kernel");
static __device__ __align__(256) int32_t scratch[kScratchWords];

constexpr int kMaxDevices = 256;
std::mutex g_scratch_mu;
int32_t* g_scratch_ptr[kMaxDevices] = {};

mdlstm_status scratch_for_current_device(int32_t** out) {
    int dev = -1;
    HIP_OR_FAIL(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return fail(MDLSTM_ERR_DEVICE, "device index %d out of range", dev);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        HIP_OR_FAIL(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) return fail(MDLSTM_ERR_DEVICE, "hipGetSymbolAddress returned no address for the scratch array");
        g_scratch_ptr[dev] = static_cast<int32_t*>(p);
    }
    *out = g_scratch_ptr[dev];
    return MDLSTM_OK;
}

}  // namespace

extern "C" {

const char* mdlstm_last_error(void) { return g_last_error.c_str(); }

mdlstm_status mdlstm_set_phase_events(int32_t n, void* const* events) {
    if (n == 0) {
        g_phase_on = false;
        return MDLSTM_OK;
    }
    if (n != 8 || !events) return fail(MDLSTM_ERR_INVALID_ARG, "phase events: n must be 0 or 8");
    for (int i = 0; i < 8; ++i) g_phase_events[i] = reinterpret_cast<hipEvent_t>(events[i]);  // NULL: not recorded
    g_phase_on = true;
    return MDLSTM_OK;
}

size_t mdlstm_pack_workspace_bytes(int32_t n) { return pack_ws_bytes(n); }

mdlstm_status mdlstm_pack_layout(int32_t n, const int32_t* heights, const int32_t* widths, int32_t canvas_w,
                                 mdlstm_rect* rects, int32_t* canvas_h, uint8_t* d_mask, size_t mask_bytes,
                                 void* d_workspace, size_t workspace_bytes, void* stream) {
    mdlstm_status st = check_pack_sizes(n, heights, widths, canvas_w, rects, canvas_h);
    if (st != MDLSTM_OK || n == 0) return st;
    if (!d_workspace || workspace_bytes < pack_ws_bytes(n))
        return fail(MDLSTM_ERR_WORKSPACE, "packing workspace of %zu bytes, %zu needed", workspace_bytes,
                    pack_ws_bytes(n));
    const size_t nn = (size_t)n;
    int32_t* d_hw = reinterpret_cast<int32_t*>(static_cast<char*>(d_workspace) + align_up(nn * 8) + align_up(nn * 16));
    std::vector<int32_t> host(6 * nn + 1);
    return place_and_mask(n, heights, widths, canvas_w, rects, canvas_h, d_mask, mask_bytes, d_hw, d_hw + 2 * nn,
                          host.data(), as_stream(stream));
}

mdlstm_status mdlstm_pack_layout_noalloc(int32_t n, const int32_t* heights, const int32_t* widths,
                                         int32_t canvas_w, mdlstm_rect* rects, int32_t* canvas_h, uint8_t* d_mask,
                                         size_t mask_bytes, void* stream) {
    mdlstm_status st = check_pack_sizes(n, heights, widths, canvas_w, rects, canvas_h);
    if (st != MDLSTM_OK || n == 0) return st;
    if (n > MDLSTM_NOALLOC_MAX_N)
        return fail(MDLSTM_ERR_UNSUPPORTED, "at most %d examples per allocation-free packing call",
                    MDLSTM_NOALLOC_MAX_N);
    int32_t* d_scratch = nullptr;
    st = scratch_for_current_device(&d_scratch);
    if (st != MDLSTM_OK) return st;
    // host staging without heap allocation: one buffer per calling thread
    static thread_local int32_t host[kScratchWords];
    return place_and_mask(n, heights, widths, canvas_w, rects, canvas_h, d_mask, mask_bytes, d_scratch,
                          d_scratch + 2 * (size_t)n, host, as_stream(stream));
}

mdlstm_status mdlstm_pad_layout(int32_t n, const int32_t* heights, const int32_t* widths, mdlstm_rect* tiles,
                                mdlstm_rect* place, int32_t* canvas_h, int32_t* canvas_w, uint8_t* d_mask,
                                size_t mask_bytes, void* d_workspace, size_t workspace_bytes, void* stream) {
    if (n < 0) return fail(MDLSTM_ERR_INVALID_ARG, "n is negative");
    if (!canvas_h || !canvas_w) return fail(MDLSTM_ERR_INVALID_ARG, "canvas_h or canvas_w is NULL");
    if (n > 0 && (!heights || !widths || !tiles || !place))
        return fail(MDLSTM_ERR_INVALID_ARG, "size or rect array is NULL");
    int32_t hm = 0, wm = 0;
    for (int32_t k = 0; k < n; ++k) {
        if (heights[k] < 1 || widths[k] < 1 || heights[k] > kMaxDim || widths[k] > kMaxDim)
            return fail(MDLSTM_ERR_INVALID_ARG, "example %d has size %dx%d", k, heights[k], widths[k]);
        hm = std::max(hm, heights[k]);
        wm = std::max(wm, widths[k]);
    }
    if ((int64_t)hm * n > kMaxDim) return fail(MDLSTM_ERR_UNSUPPORTED, "padded canvas exceeds %d rows", kMaxDim);
    for (int32_t k = 0; k < n; ++k) {
        tiles[k] = mdlstm_rect{k * hm, 0, hm, wm};
        place[k] = mdlstm_rect{k * hm, 0, heights[k], widths[k]};
    }
    *canvas_h = n * hm;
    *canvas_w = wm;
    if (d_mask && n > 0) {
        const size_t need = (size_t)(*canvas_h) * (size_t)wm;
        if (mask_bytes < need) return fail(MDLSTM_ERR_WORKSPACE, "mask of %zu bytes, %zu needed", mask_bytes, need);
        if (!d_workspace || workspace_bytes < pack_ws_bytes(n))
            return fail(MDLSTM_ERR_WORKSPACE, "packing workspace of %zu bytes, %zu needed", workspace_bytes,
                        pack_ws_bytes(n));
        hipStream_t s = as_stream(stream);
        int32_t* d_r = reinterpret_cast<int32_t*>(static_cast<char*>(d_workspace) + align_up((size_t)n * 8));
        HIP_OR_FAIL(hipMemcpyAsync(d_r, place, (size_t)n * 16, hipMemcpyHostToDevice, s));
        HIP_OR_FAIL(mdl::launch_mask(n, d_r, *canvas_h, wm, d_mask, s));
    }
    return MDLSTM_OK;
}

static mdlstm_status pack_io(bool pack, int32_t n, const void* const* ptrs, const mdlstm_rect* rects,
                             int32_t canvas_h, int32_t canvas_w, int32_t c, int32_t dt, const void* d_canvas,
                             void* d_workspace, size_t workspace_bytes, void* stream) {
    if (n < 0 || c < 1) return fail(MDLSTM_ERR_INVALID_ARG, "n must be >= 0 and c >= 1");
    if (dt != MDLSTM_F32 && dt != MDLSTM_BF16) return fail(MDLSTM_ERR_INVALID_ARG, "dtype %d unknown", dt);
    if (canvas_h < 0 || canvas_w < 0 || canvas_h > kMaxDim || canvas_w > kMaxDim)
        return fail(MDLSTM_ERR_INVALID_ARG, "canvas %dx%d out of range", canvas_h, canvas_w);
    if ((int64_t)canvas_h * canvas_w > 0 && !d_canvas) return fail(MDLSTM_ERR_INVALID_ARG, "canvas is NULL");
    if (n > 0 && (!ptrs || !rects)) return fail(MDLSTM_ERR_INVALID_ARG, "example or rect array is NULL");
    int32_t max_h = 0;
    for (int32_t k = 0; k < n; ++k) {
        const mdlstm_rect& a = rects[k];
        if (!ptrs[k]) return fail(MDLSTM_ERR_INVALID_ARG, "example %d pointer is NULL", k);
        if (a.h < 1 || a.w < 1 || a.y0 < 0 || a.x0 < 0 || (int64_t)a.y0 + a.h > canvas_h ||
            (int64_t)a.x0 + a.w > canvas_w)
            return fail(MDLSTM_ERR_BAD_LAYOUT, "rect %d (%d,%d,%d,%d) leaves the %dx%d canvas", k, a.y0, a.x0, a.h,
                        a.w, canvas_h, canvas_w);
        max_h = std::max(max_h, a.h);
    }
    const int esize = dt == MDLSTM_BF16 ? 2 : 4;
    hipStream_t s = as_stream(stream);
    if (n == 0) {
        if (pack) HIP_OR_FAIL(mdl::launch_scatter(0, nullptr, nullptr, canvas_h, canvas_w, c, esize,
                                                  const_cast<void*>(d_canvas), 0, s));
        return MDLSTM_OK;
    }
    if (!d_workspace || workspace_bytes < pack_ws_bytes(n))
        return fail(MDLSTM_ERR_WORKSPACE, "packing workspace of %zu bytes, %zu needed", workspace_bytes,
                    pack_ws_bytes(n));
    char* ws = static_cast<char*>(d_workspace);
    void** d_ptrs = reinterpret_cast<void**>(ws);
    int32_t* d_r = reinterpret_cast<int32_t*>(ws + align_up((size_t)n * 8));
    HIP_OR_FAIL(hipMemcpyAsync(d_ptrs, ptrs, (size_t)n * 8, hipMemcpyHostToDevice, s));
    HIP_OR_FAIL(hipMemcpyAsync(d_r, rects, (size_t)n * 16, hipMemcpyHostToDevice, s));
    if (pack)
        HIP_OR_FAIL(mdl::launch_scatter(n, d_ptrs, d_r, canvas_h, canvas_w, c, esize, const_cast<void*>(d_canvas),
                                        max_h, s));
    else
        HIP_OR_FAIL(mdl::launch_gather(n, d_ptrs, d_r, canvas_w, c, esize, d_canvas, max_h, s));
    return MDLSTM_OK;
}

mdlstm_status mdlstm_pack_data(int32_t n, const void* const* d_examples, const mdlstm_rect* rects, int32_t canvas_h,
                               int32_t canvas_w, int32_t c, int32_t dt, void* d_canvas, void* d_workspace,
                               size_t workspace_bytes, void* stream) {
    return pack_io(true, n, d_examples, rects, canvas_h, canvas_w, c, dt, d_canvas, d_workspace, workspace_bytes,
                   stream);
}

mdlstm_status mdlstm_unpack_data(int32_t n, void* const* d_examples, const mdlstm_rect* rects, int32_t canvas_h,
                                 int32_t canvas_w, int32_t c, int32_t dt, const void* d_canvas, void* d_workspace,
                                 size_t workspace_bytes, void* stream) {
    return pack_io(false, n, reinterpret_cast<const void* const*>(d_examples), rects, canvas_h, canvas_w, c, dt,
                   d_canvas, d_workspace, workspace_bytes, stream);
}

size_t mdlstm_workspace_bytes(const mdlstm_layer_desc* desc, int32_t canvas_h, int32_t canvas_w, int32_t n_rects) {
    mdlstm_layer_desc in;
    if (inner_desc(desc, &in) != MDLSTM_OK) return 0;
    if (canvas_h < 0 || canvas_w < 0 || canvas_h > kMaxDim || canvas_w > kMaxDim || n_rects < 0 ||
        n_rects > kMaxRects) {
        fail(MDLSTM_ERR_INVALID_ARG, "canvas %dx%d or %d rectangles out of range", canvas_h, canvas_w, n_rects);
        return 0;
    }
    return pad_plan(desc, in, canvas_h, canvas_w).total + plan(&in, canvas_h, canvas_w, n_rects).total;
}

int32_t mdlstm_gradients_fused(const mdlstm_layer_desc* desc) {
    mdlstm_layer_desc in;
    if (inner_desc(desc, &in) != MDLSTM_OK) return -1;
    return mdl::strip_supported(geom(&in, 1, 1)) ? 1 : 0;
}

namespace {

// The per-diagonal graph of the last mdlstm_forward_stepwise call on this
// thread and the arguments it was recorded for. Deliberately never freed at
// exit: destroying a graph after the HIP runtime has shut down is unsafe.
struct StepGraph {
    std::vector<uintptr_t> key;
    hipGraphExec_t exec = nullptr;
};

mdlstm_status forward_impl(bool stepwise, const mdlstm_layer_desc* desc, int32_t canvas_h, int32_t canvas_w,
                           const void* d_x, const uint8_t* d_mask, int32_t n_rects, const mdlstm_rect* rects,
                           const void* d_wx, const void* d_u, const void* d_b, void* d_y, void* d_workspace,
                           size_t workspace_bytes, void* stream) {
    Common c;
    mdlstm_status st = prepare(desc, canvas_h, canvas_w, d_x, d_mask, n_rects, rects, d_wx, d_u, d_b, d_workspace,
                               workspace_bytes, &c);
    if (st != MDLSTM_OK) return st;
    if (c.g.n_cells > 0 && !d_y) return fail(MDLSTM_ERR_INVALID_ARG, "y is NULL");
    if (misaligned(d_y)) return fail(MDLSTM_ERR_INVALID_ARG, "y must be 16-byte aligned");
    if (c.g.n_cells == 0) return MDLSTM_OK;
    hipStream_t s = as_stream(stream);
    if (poison_requested()) {
        // gates and cell states, and the gradient scratch the backward writes
        if ((st = poison(c.ws, c.p.z, c.p.rid, s)) != MDLSTM_OK) return st;
        if ((st = poison(c.ws, c.p.part, c.p.flags, s)) != MDLSTM_OK) return st;
        if ((st = poison(c.ws, c.p.wxt, c.p.queue, s)) != MDLSTM_OK) return st;
    }
    st = stage_layout(c, n_rects, rects, false, s);
    if (st != MDLSTM_OK) return st;
    const int32_t* rid = reinterpret_cast<const int32_t*>(c.ws + c.p.rid);
    const int32_t* units = reinterpret_cast<const int32_t*>(c.ws + c.p.units);
    const int32_t* drects = reinterpret_cast<const int32_t*>(c.ws + c.p.rects);
    float* cs = reinterpret_cast<float*>(c.ws + c.p.c);
    if (desc->memory_states && stepwise)
        return fail(MDLSTM_ERR_UNSUPPORTED, "the per-diagonal schedule is not built with memory-state matrices");
    HIP_OR_FAIL(mark(0, s));
    HIP_OR_FAIL(mdl::launch_projection(c.g, d_x, d_wx, d_b, rid, c.ws + c.p.z, s));
    HIP_OR_FAIL(mark(1, s));
    if (stepwise || n_rects == 0 || desc->memory_states)
        HIP_OR_FAIL(mdl::launch_zero_invalid(c.g, 4 * c.g.hidden, d_mask, rid, d_y, s));
    HIP_OR_FAIL(mark(2, s));
    if (desc->memory_states) {
        const int64_t nu = 4 * (int64_t)c.g.hidden * 5 * 2 * c.g.hidden;  // floats of U before V
        mdl::MemArgs m{units, drects, d_mask, static_cast<const float*>(d_u), static_cast<const float*>(d_u) + nu,
                       reinterpret_cast<float*>(c.ws + c.p.z), cs, static_cast<float*>(d_y), nullptr, canvas_w,
                       nullptr};
        HIP_OR_FAIL(mdl::launch_wavefront_mem(true, c.g, 4 * n_rects, m, s));
    } else if (!stepwise) {
        // the persistent launch also zeroes the output rows of the invalid cells
        HIP_OR_FAIL(mdl::launch_wavefront_fwd(c.g, c.nt, 4 * n_rects, units, drects, d_mask, rid, d_u, c.ws + c.p.z,
                                              cs, d_y, reinterpret_cast<unsigned*>(c.ws + c.p.queue), s));
    } else if (n_rects > 0) {
        int32_t max_steps = 0;
        for (int32_t k = 0; k < n_rects; ++k) max_steps = std::max(max_steps, rects[k].h + rects[k].w - 1);
        static thread_local StepGraph* cache = new StepGraph;
        std::vector<uintptr_t> key = {(uintptr_t)desc->c_in, (uintptr_t)desc->hidden, (uintptr_t)desc->dtype,
                                      (uintptr_t)canvas_h, (uintptr_t)canvas_w, (uintptr_t)d_mask, (uintptr_t)d_u,
                                      (uintptr_t)d_y, (uintptr_t)d_workspace, (uintptr_t)n_rects};
        for (int32_t k = 0; k < n_rects; ++k) {
            key.push_back(((uintptr_t)(uint32_t)rects[k].y0 << 32) | (uint32_t)rects[k].x0);
            key.push_back(((uintptr_t)(uint32_t)rects[k].h << 32) | (uint32_t)rects[k].w);
        }
        if (!cache->exec || cache->key != key) {
            if (cache->exec) {
                HIP_OR_FAIL(hipGraphExecDestroy(cache->exec));
                cache->exec = nullptr;
            }
            HIP_OR_FAIL(mdl::build_wavefront_fwd_graph(c.g, c.nt, 4 * n_rects, max_steps, units, drects, d_mask, d_u,
                                                       c.ws + c.p.z, cs, d_y, &cache->exec));
            cache->key = std::move(key);
        }
        HIP_OR_FAIL(hipGraphLaunch(cache->exec, s));
    }
    HIP_OR_FAIL(mark(3, s));
    if (check_finite_requested()) {
        unsigned long long* cnt = reinterpret_cast<unsigned long long*>(c.ws + c.p.check);
        HIP_OR_FAIL(mdl::launch_zero_f32(reinterpret_cast<float*>(cnt), 2, s));
        // the cell state outside the examples' cells is not defined: count
        // over the cells whose mask byte is set
        HIP_OR_FAIL(mdl::launch_count_nonfinite(d_y, c.g.n_cells, 4 * c.g.hidden, d_mask, c.g.dtype, cnt, s));
        HIP_OR_FAIL(mdl::launch_count_nonfinite(cs, c.g.n_cells, 4 * c.g.hidden, d_mask, 0, cnt, s));
        unsigned long long h = 0;
        HIP_OR_FAIL(hipMemcpyAsync(&h, cnt, sizeof(h), hipMemcpyDeviceToHost, s));
        HIP_OR_FAIL(hipStreamSynchronize(s));
        if (h) return fail(MDLSTM_ERR_NUMERIC, "%llu non-finite values in the output and cell state", h);
    }
    return MDLSTM_OK;
}

mdlstm_status backward_impl(const mdlstm_layer_desc* desc, int32_t canvas_h, int32_t canvas_w, const void* d_x,
                            const uint8_t* d_mask, int32_t n_rects, const mdlstm_rect* rects, const void* d_wx,
                            const void* d_u, const void* d_b, const void* d_y, const void* d_dy, void* d_dx,
                            float* d_dwx, float* d_du, float* d_db, void* d_workspace, size_t workspace_bytes,
                            void* stream) {
    Common c;
    mdlstm_status st = prepare(desc, canvas_h, canvas_w, d_x, d_mask, n_rects, rects, d_wx, d_u, d_b, d_workspace,
                               workspace_bytes, &c);
    if (st != MDLSTM_OK) return st;
    if (!d_dwx || !d_du || !d_db) return fail(MDLSTM_ERR_INVALID_ARG, "a weight-gradient pointer is NULL");
    if (c.g.n_cells > 0 && (!d_y || !d_dy || !d_dx)) return fail(MDLSTM_ERR_INVALID_ARG, "y, dy or dx is NULL");
    if (misaligned(d_y) || misaligned(d_dy) || misaligned(d_dx) || misaligned(d_dwx) || misaligned(d_du) ||
        misaligned(d_db))
        return fail(MDLSTM_ERR_INVALID_ARG, "y, dy, dx and the weight gradients must be 16-byte aligned");
    hipStream_t s = as_stream(stream);
    st = stage_layout(c, n_rects, rects, true, s);
    if (st != MDLSTM_OK) return st;
    if (poison_requested() && c.g.n_cells > 0) {
        // the gradient scratch (partials, transposed Wx, dV partials); the
        // gates and cell states are the forward's
        if ((st = poison(c.ws, c.p.part, c.p.flags, s)) != MDLSTM_OK) return st;
        if ((st = poison(c.ws, c.p.wxt, c.p.queue, s)) != MDLSTM_OK) return st;
    }
    const int32_t* rid = reinterpret_cast<const int32_t*>(c.ws + c.p.rid);
    HIP_OR_FAIL(mark(4, s));
    if (c.g.n_cells > 0 && desc->memory_states) {
        const int64_t nu = 4 * (int64_t)c.g.hidden * 5 * 2 * c.g.hidden;  // floats of U (and dU) before V (dV)
        const int32_t* units = reinterpret_cast<const int32_t*>(c.ws + c.p.units);
        float* part = reinterpret_cast<float*>(c.ws + c.p.dvpart);
        mdl::MemArgs m{units, reinterpret_cast<const int32_t*>(c.ws + c.p.rects), d_mask,
                       static_cast<const float*>(d_u), static_cast<const float*>(d_u) + nu,
                       reinterpret_cast<float*>(c.ws + c.p.z), reinterpret_cast<float*>(c.ws + c.p.c), nullptr,
                       static_cast<const float*>(d_dy), canvas_w, part};
        HIP_OR_FAIL(mdl::launch_wavefront_mem(false, c.g, 4 * n_rects, m, s));
        if (n_rects > 0) HIP_OR_FAIL(mdl::launch_dv_reduce(c.g, 4 * n_rects, units, part, d_du + nu, s));
        else HIP_OR_FAIL(mdl::launch_zero_f32(d_du + nu, 4 * (int64_t)c.g.hidden * 3 * 2 * c.g.hidden, s));
    } else if (c.g.n_cells > 0) {
        HIP_OR_FAIL(mdl::launch_wavefront_bwd(c.g, c.nt, 4 * n_rects,
                                              reinterpret_cast<const int32_t*>(c.ws + c.p.units),
                                              reinterpret_cast<const int32_t*>(c.ws + c.p.rects), d_mask, d_u, d_dy,
                                              c.ws + c.p.z, reinterpret_cast<const float*>(c.ws + c.p.c),
                                              reinterpret_cast<unsigned*>(c.ws + c.p.queue), s));
    } else if (desc->memory_states) {
        const int64_t nu = 4 * (int64_t)c.g.hidden * 5 * 2 * c.g.hidden;
        HIP_OR_FAIL(mdl::launch_zero_f32(d_du + nu, 4 * (int64_t)c.g.hidden * 3 * 2 * c.g.hidden, s));
    }
    HIP_OR_FAIL(mark(5, s));
    if (c.g.n_cells > 0 && mdl::strip_supported(c.g)) {
        // input and weight gradients in one pass (phase boundary 6 coincides with 5)
        HIP_OR_FAIL(mark(6, s));
        HIP_OR_FAIL(mdl::launch_bwd_strip(c.g, c.ws + c.p.z, d_x, d_y, d_wx, d_mask, rid,
                                          reinterpret_cast<int32_t*>(c.ws + c.p.flags), d_dx,
                                          reinterpret_cast<float*>(c.ws + c.p.part), d_dwx, d_du, d_db, s));
    } else {
        // tiled products: the input gradient (boundary 6), then the weight gradients
        if (c.g.n_cells > 0) {
            uint8_t* flags = reinterpret_cast<uint8_t*>(c.ws + c.p.flags);
            HIP_OR_FAIL(mdl::launch_bwd_big_dx(c.g, c.ws + c.p.z, d_wx, d_mask, rid, d_dx, flags, c.ws + c.p.wxt, s));
            HIP_OR_FAIL(mark(6, s));
            HIP_OR_FAIL(mdl::launch_bwd_big_dw(c.g, c.ws + c.p.z, d_x, d_y, flags,
                                               reinterpret_cast<float*>(c.ws + c.p.part), d_dwx, d_du, d_db, s));
        } else {
            HIP_OR_FAIL(mark(6, s));
            HIP_OR_FAIL(mdl::launch_zero_f32(d_dwx, (int64_t)4 * 5 * c.g.hidden * c.g.c_in, s));
            HIP_OR_FAIL(mdl::launch_zero_f32(d_du, (int64_t)4 * 5 * c.g.hidden * 2 * c.g.hidden, s));
            HIP_OR_FAIL(mdl::launch_zero_f32(d_db, (int64_t)4 * 5 * c.g.hidden, s));
        }
    }
    HIP_OR_FAIL(mark(7, s));
    return MDLSTM_OK;
}

// Arguments of a layer call at its own sizes, checked before the padded
// copies are written.
mdlstm_status check_padded_call(const PadPlan& q, const mdlstm_layer_desc& in, int32_t ch, int32_t cw,
                                const void* d_x, const uint8_t* d_mask, int32_t n_rects, const mdlstm_rect* rects,
                                const void* d_wx, const void* d_u, const void* d_b, void* d_workspace,
                                size_t ws_bytes) {
    if (ch < 0 || cw < 0 || ch > kMaxDim || cw > kMaxDim)
        return fail(MDLSTM_ERR_INVALID_ARG, "canvas %dx%d out of range", ch, cw);
    int32_t max_h = 0;
    mdlstm_status st = check_rects(n_rects, rects, ch, cw, &max_h);
    if (st != MDLSTM_OK) return st;
    if ((int64_t)ch * cw > 0 && (!d_x || !d_mask)) return fail(MDLSTM_ERR_INVALID_ARG, "x or mask is NULL");
    if (!d_wx || !d_u || !d_b) return fail(MDLSTM_ERR_INVALID_ARG, "a weight pointer is NULL");
    if (!d_workspace) return fail(MDLSTM_ERR_INVALID_ARG, "workspace is NULL");
    if (misaligned(d_x) || misaligned(d_wx) || misaligned(d_u) || misaligned(d_b) || misaligned(d_workspace))
        return fail(MDLSTM_ERR_INVALID_ARG, "x, weights and workspace must be 16-byte aligned");
    const size_t need = q.total + plan(&in, ch, cw, n_rects).total;
    if (ws_bytes < need) return fail(MDLSTM_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", ws_bytes, need);
    return MDLSTM_OK;
}

// Weights at the layer's sizes into the padded sections: Wx [4][5H][C],
// U [4][5H][2H] (+ V [4][3H][2H]) and b [4][5H], each gate block and each
// predecessor block padded on its own.
mdlstm_status pad_weights(const mdlstm_layer_desc* d, const mdlstm_layer_desc& in, const PadPlan& q,
                          const void* d_wx, const void* d_u, const void* d_b, char* ws, hipStream_t s) {
    const int es = d->dtype == MDLSTM_BF16 ? 2 : 4, H = d->hidden, Hp = in.hidden;
    HIP_OR_FAIL(mdl::launch_remap(d_wx, ws + q.wx, es, 4, 5, H, Hp, 1, d->c_in, in.c_in, s));
    HIP_OR_FAIL(mdl::launch_remap(d_u, ws + q.u, es, 4, 5, H, Hp, 2, H, Hp, s));
    if (d->memory_states)
        HIP_OR_FAIL(mdl::launch_remap(static_cast<const char*>(d_u) + (size_t)4 * 5 * H * 2 * H * es,
                                      ws + q.u + (size_t)4 * 5 * Hp * 2 * Hp * es, es, 4, 3, H, Hp, 2, H, Hp, s));
    HIP_OR_FAIL(mdl::launch_remap(d_b, ws + q.b, es, 4, 5, H, Hp, 1, 1, 1, s));
    return MDLSTM_OK;
}

mdlstm_status padded_forward(bool stepwise, const mdlstm_layer_desc* desc, int32_t canvas_h, int32_t canvas_w,
                             const void* d_x, const uint8_t* d_mask, int32_t n_rects, const mdlstm_rect* rects,
                             const void* d_wx, const void* d_u, const void* d_b, void* d_y, void* d_workspace,
                             size_t workspace_bytes, void* stream) {
    mdlstm_layer_desc in;
    mdlstm_status st = inner_desc(desc, &in);
    if (st != MDLSTM_OK) return st;
    if (same_shape(desc, in))
        return forward_impl(stepwise, desc, canvas_h, canvas_w, d_x, d_mask, n_rects, rects, d_wx, d_u, d_b, d_y,
                            d_workspace, workspace_bytes, stream);
    if (in.memory_states && stepwise)
        return fail(MDLSTM_ERR_UNSUPPORTED, "the per-diagonal schedule is not built with memory-state matrices");
    const PadPlan q = pad_plan(desc, in, canvas_h, canvas_w);
    st = check_padded_call(q, in, canvas_h, canvas_w, d_x, d_mask, n_rects, rects, d_wx, d_u, d_b, d_workspace,
                           workspace_bytes);
    if (st != MDLSTM_OK) return st;
    const int64_t cells = (int64_t)canvas_h * canvas_w;
    if (cells > 0 && !d_y) return fail(MDLSTM_ERR_INVALID_ARG, "y is NULL");
    if (misaligned(d_y)) return fail(MDLSTM_ERR_INVALID_ARG, "y must be 16-byte aligned");
    if (cells == 0) return MDLSTM_OK;
    hipStream_t s = as_stream(stream);
    char* ws = static_cast<char*>(d_workspace);
    const int es = desc->dtype == MDLSTM_BF16 ? 2 : 4;
    if ((st = pad_weights(desc, in, q, d_wx, d_u, d_b, ws, s)) != MDLSTM_OK) return st;
    const void* x = d_x;
    if (q.pad_c) {
        HIP_OR_FAIL(mdl::launch_remap(d_x, ws + q.x, es, cells, 1, 1, 1, 1, desc->c_in, in.c_in, s));
        x = ws + q.x;
    }
    void* y = q.pad_h ? static_cast<void*>(ws + q.y) : d_y;
    st = forward_impl(stepwise, &in, canvas_h, canvas_w, x, d_mask, n_rects, rects, ws + q.wx, ws + q.u, ws + q.b, y,
                      ws + q.total, workspace_bytes - q.total, stream);
    if (st != MDLSTM_OK) return st;
    if (q.pad_h) HIP_OR_FAIL(mdl::launch_remap(y, d_y, es, cells, 1, 1, 1, 4, in.hidden, desc->hidden, s));
    return MDLSTM_OK;
}

mdlstm_status padded_backward(const mdlstm_layer_desc* desc, int32_t canvas_h, int32_t canvas_w, const void* d_x,
                              const uint8_t* d_mask, int32_t n_rects, const mdlstm_rect* rects, const void* d_wx,
                              const void* d_u, const void* d_b, const void* d_y, const void* d_dy, void* d_dx,
                              float* d_dwx, float* d_du, float* d_db, void* d_workspace, size_t workspace_bytes,
                              void* stream) {
    mdlstm_layer_desc in;
    mdlstm_status st = inner_desc(desc, &in);
    if (st != MDLSTM_OK) return st;
    if (same_shape(desc, in))
        return backward_impl(desc, canvas_h, canvas_w, d_x, d_mask, n_rects, rects, d_wx, d_u, d_b, d_y, d_dy, d_dx,
                             d_dwx, d_du, d_db, d_workspace, workspace_bytes, stream);
    const PadPlan q = pad_plan(desc, in, canvas_h, canvas_w);
    st = check_padded_call(q, in, canvas_h, canvas_w, d_x, d_mask, n_rects, rects, d_wx, d_u, d_b, d_workspace,
                           workspace_bytes);
    if (st != MDLSTM_OK) return st;
    const int64_t cells = (int64_t)canvas_h * canvas_w;
    if (!d_dwx || !d_du || !d_db) return fail(MDLSTM_ERR_INVALID_ARG, "a weight-gradient pointer is NULL");
    if (cells > 0 && (!d_y || !d_dy || !d_dx)) return fail(MDLSTM_ERR_INVALID_ARG, "y, dy or dx is NULL");
    if (misaligned(d_y) || misaligned(d_dy) || misaligned(d_dx) || misaligned(d_dwx) || misaligned(d_du) ||
        misaligned(d_db))
        return fail(MDLSTM_ERR_INVALID_ARG, "y, dy, dx and the weight gradients must be 16-byte aligned");
    hipStream_t s = as_stream(stream);
    char* ws = static_cast<char*>(d_workspace);
    const int es = desc->dtype == MDLSTM_BF16 ? 2 : 4, H = desc->hidden, Hp = in.hidden;
    if ((st = pad_weights(desc, in, q, d_wx, d_u, d_b, ws, s)) != MDLSTM_OK) return st;
    const void *x = d_x, *y = d_y, *dy = d_dy;
    void* dx = d_dx;
    if (q.pad_c && cells > 0) {
        HIP_OR_FAIL(mdl::launch_remap(d_x, ws + q.x, es, cells, 1, 1, 1, 1, desc->c_in, in.c_in, s));
        x = ws + q.x;
        dx = ws + q.dx;
    }
    if (q.pad_h && cells > 0) {
        HIP_OR_FAIL(mdl::launch_remap(d_y, ws + q.y, es, cells, 1, 1, 1, 4, H, Hp, s));
        HIP_OR_FAIL(mdl::launch_remap(d_dy, ws + q.dy, es, cells, 1, 1, 1, 4, H, Hp, s));
        y = ws + q.y;
        dy = ws + q.dy;
    }
    float* dwx = reinterpret_cast<float*>(ws + q.dwx);
    float* du = reinterpret_cast<float*>(ws + q.du);
    float* db = reinterpret_cast<float*>(ws + q.db);
    st = backward_impl(&in, canvas_h, canvas_w, x, d_mask, n_rects, rects, ws + q.wx, ws + q.u, ws + q.b, y, dy, dx,
                       dwx, du, db, ws + q.total, workspace_bytes - q.total, stream);
    if (st != MDLSTM_OK) return st;
    if (q.pad_c && cells > 0) HIP_OR_FAIL(mdl::launch_remap(dx, d_dx, es, cells, 1, 1, 1, 1, in.c_in, desc->c_in, s));
    HIP_OR_FAIL(mdl::launch_remap(dwx, d_dwx, 4, 4, 5, Hp, H, 1, in.c_in, desc->c_in, s));
    HIP_OR_FAIL(mdl::launch_remap(du, d_du, 4, 4, 5, Hp, H, 2, Hp, H, s));
    if (desc->memory_states)
        HIP_OR_FAIL(mdl::launch_remap(du + (size_t)4 * 5 * Hp * 2 * Hp, d_du + (size_t)4 * 5 * H * 2 * H, 4, 4, 3, Hp,
                                      H, 2, Hp, H, s));
    HIP_OR_FAIL(mdl::launch_remap(db, d_db, 4, 4, 5, Hp, H, 1, 1, 1, s));
    return MDLSTM_OK;
}

}  // namespace

mdlstm_status mdlstm_forward(const mdlstm_layer_desc* desc, int32_t canvas_h, int32_t canvas_w, const void* d_x,
                             const uint8_t* d_mask, int32_t n_rects, const mdlstm_rect* rects, const void* d_wx,
                             const void* d_u, const void* d_b, void* d_y, void* d_workspace, size_t workspace_bytes,
                             void* stream) {
    return padded_forward(false, desc, canvas_h, canvas_w, d_x, d_mask, n_rects, rects, d_wx, d_u, d_b, d_y,
                          d_workspace, workspace_bytes, stream);
}

mdlstm_status mdlstm_forward_stepwise(const mdlstm_layer_desc* desc, int32_t canvas_h, int32_t canvas_w,
                                      const void* d_x, const uint8_t* d_mask, int32_t n_rects,
                                      const mdlstm_rect* rects, const void* d_wx, const void* d_u, const void* d_b,
                                      void* d_y, void* d_workspace, size_t workspace_bytes, void* stream) {
    return padded_forward(true, desc, canvas_h, canvas_w, d_x, d_mask, n_rects, rects, d_wx, d_u, d_b, d_y,
                          d_workspace, workspace_bytes, stream);
}

mdlstm_status mdlstm_backward(const mdlstm_layer_desc* desc, int32_t canvas_h, int32_t canvas_w, const void* d_x,
                              const uint8_t* d_mask, int32_t n_rects, const mdlstm_rect* rects, const void* d_wx,
                              const void* d_u, const void* d_b, const void* d_y, const void* d_dy, void* d_dx,
                              float* d_dwx, float* d_du, float* d_db, void* d_workspace, size_t workspace_bytes,
                              void* stream) {
    return padded_backward(desc, canvas_h, canvas_w, d_x, d_mask, n_rects, rects, d_wx, d_u, d_b, d_y, d_dy, d_dx,
                           d_dwx, d_du, d_db, d_workspace, workspace_bytes, stream);
}

// ---------------------------------------------------------------------------
// Output layer shared by the directions, row collapse, CTC loss.
// ---------------------------------------------------------------------------
namespace {

constexpr int32_t kMaxHeadClasses = 128;
constexpr int32_t kMaxLabel = 960;  // labels per example (LDS of the CTC kernel)

mdlstm_status check_head_desc(const mdlstm_head_desc* d) {
    if (!d) return fail(MDLSTM_ERR_INVALID_ARG, "head desc is NULL");
    if (d->hidden < 4 || d->hidden > 64 || d->hidden % 4)
        return fail(MDLSTM_ERR_UNSUPPORTED, "head hidden size %d: a multiple of 4 in [4, 64] is built", d->hidden);
    if (d->classes < 2 || d->classes > kMaxHeadClasses)
        return fail(MDLSTM_ERR_UNSUPPORTED, "head classes %d: 2 to %d are built", d->classes, kMaxHeadClasses);
    return MDLSTM_OK;
}

// Workspace sections. The first part (tiles .. weight-gradient partials)
// serves the layer's forward and backward; the second (label tables .. the
// backward variables) the CTC loss.
struct HeadPlan {
    int64_t frames = 0;
    int32_t n_tiles = 0, chunks = 0, labels = 0, max_label = 0, nm = 1;
    size_t tiles, rects, frame_off, S, part, part1_end, lab_off, lab, occ, lp, alpha, beta, total;
};

HeadPlan head_plan(const mdlstm_head_desc* d, int32_t n, const mdlstm_rect* rects, const int32_t* label_lens) {
    HeadPlan p;
    const int hc = mdl::head_tile_frames();
    for (int32_t i = 0; i < n; ++i) {
        p.frames += rects[i].w;
        p.n_tiles += (rects[i].w + hc - 1) / hc;
        if (label_lens) {
            p.labels += label_lens[i];
            p.max_label = std::max(p.max_label, label_lens[i]);
        }
    }
    const int dwf = mdl::head_dw_chunk_frames();
    p.chunks = (int32_t)((p.frames + dwf - 1) / dwf);
    const size_t nn = (size_t)(n > 0 ? n : 1);
    size_t off = 0;
    p.tiles = off;
    off += align_up((size_t)std::max(p.n_tiles, 1) * 8);
    p.rects = off;
    off += align_up(nn * 16);
    p.frame_off = off;
    off += align_up((nn + 1) * 4);
    p.S = off;
    off += align_up((size_t)std::max<int64_t>(p.frames, 1) * (d->hidden + 4) * 4);
    p.part = off;
    off += align_up((size_t)std::max(p.chunks, 1) * d->classes * (d->hidden + 1) * 4);
    p.part1_end = off;
    p.lab_off = off;
    off += align_up((nn + 1) * 4);
    p.lab = off;
    off += align_up((size_t)std::max(p.labels, 1) * 4);
    p.occ = off;
    off += align_up((size_t)std::max(p.labels, 1) * 4);
    p.lp = off;
    off += align_up((size_t)std::max<int64_t>(p.frames, 1) * d->classes * 8);
    // rows of 64 nm states per frame for the CTC scans: mantissas (double)
    // and exponents (int32) of the forward, then the backward variables
    p.nm = mdl::ctc_states_per_lane(p.max_label);
    const size_t rows = (size_t)std::max<int64_t>(p.frames, 1) * 64 * p.nm;
    p.alpha = off;
    off += align_up(rows * 8) + align_up(rows * 4);
    p.beta = off;
    off += align_up(rows * 8) + align_up(rows * 4);
    p.total = off;
    return p;
}

// Validation shared by the three calls (rectangles inside the canvas and
// disjoint when a canvas is given; the frames of all examples addressable).
mdlstm_status check_head_rects(int32_t n, const mdlstm_rect* rects, int32_t ch, int32_t cw) {
    if (n < 0) return fail(MDLSTM_ERR_INVALID_ARG, "n is negative");
    if (n > kMaxRects) return fail(MDLSTM_ERR_UNSUPPORTED, "%d examples; at most %d per call", n, kMaxRects);
    if (n > 0 && !rects) return fail(MDLSTM_ERR_INVALID_ARG, "rects is NULL");
    int64_t frames = 0;
    for (int32_t i = 0; i < n; ++i) {
        if (rects[i].h < 1 || rects[i].w < 1)
            return fail(MDLSTM_ERR_BAD_LAYOUT, "rect %d has size %dx%d", i, rects[i].h, rects[i].w);
        frames += rects[i].w;
    }
    if (frames > (int64_t)INT32_MAX / 256) return fail(MDLSTM_ERR_UNSUPPORTED, "%lld frames", (long long)frames);
    if (ch >= 0) {
        if (ch > kMaxDim || cw < 0 || cw > kMaxDim) return fail(MDLSTM_ERR_INVALID_ARG, "canvas %dx%d out of range", ch, cw);
        int32_t mh = 0;
        return check_rects(n, rects, ch, cw, &mh, kMaxDim);
    }
    return MDLSTM_OK;
}

// The small host-computed tables of the first workspace part, staged in one copy.
mdlstm_status stage_head_tables(const HeadPlan& p, int32_t n, const mdlstm_rect* rects, char* ws, hipStream_t s) {
    std::vector<unsigned char> host(p.S - p.tiles, 0);
    int32_t* tiles = reinterpret_cast<int32_t*>(host.data() + (p.tiles - p.tiles));
    int32_t* fo = reinterpret_cast<int32_t*>(host.data() + (p.frame_off - p.tiles));
    const int hc = mdl::head_tile_frames();
    int32_t t = 0, f = 0;
    for (int32_t i = 0; i < n; ++i) {
        fo[i] = f;
        f += rects[i].w;
        for (int32_t c = 0; c < rects[i].w; c += hc) {
            tiles[2 * t] = i;
            tiles[2 * t + 1] = c;
            ++t;
        }
    }
    fo[n] = f;
    if (n > 0) std::memcpy(host.data() + (p.rects - p.tiles), rects, (size_t)n * 16);
    HIP_OR_FAIL(hipMemcpyAsync(ws + p.tiles, host.data(), host.size(), hipMemcpyHostToDevice, s));
    return MDLSTM_OK;
}

}  // namespace

size_t mdlstm_head_workspace_bytes(const mdlstm_head_desc* desc, int32_t n, const mdlstm_rect* rects,
                                   const int32_t* label_lens) {
    if (check_head_desc(desc) != MDLSTM_OK || check_head_rects(n, rects, -1, -1) != MDLSTM_OK) return 0;
    for (int32_t i = 0; label_lens && i < n; ++i)
        if (label_lens[i] < 0 || label_lens[i] > kMaxLabel || label_lens[i] > rects[i].w) {
            fail(MDLSTM_ERR_INVALID_ARG, "example %d: %d labels for %d frames", i, label_lens[i], rects[i].w);
            return 0;
        }
    const HeadPlan p = head_plan(desc, n, rects, label_lens);
    return label_lens ? p.total : p.part1_end;
}

mdlstm_status mdlstm_head_forward(const mdlstm_head_desc* desc, int32_t canvas_h, int32_t canvas_w, const float* d_y,
                                  int32_t n, const mdlstm_rect* rects, const float* d_w, const float* d_b,
                                  float* d_logits, void* d_workspace, size_t workspace_bytes, void* stream) {
    mdlstm_status st = check_head_desc(desc);
    if (st != MDLSTM_OK) return st;
    if (canvas_h < 0) return fail(MDLSTM_ERR_INVALID_ARG, "canvas_h is negative");
    st = check_head_rects(n, rects, canvas_h, canvas_w);
    if (st != MDLSTM_OK) return st;
    if (n > 0 && (!d_y || !d_w || !d_b || !d_logits)) return fail(MDLSTM_ERR_INVALID_ARG, "a device pointer is NULL");
    if (misaligned(d_y) || misaligned(d_w) || misaligned(d_workspace))
        return fail(MDLSTM_ERR_INVALID_ARG, "y, w and workspace must be 16-byte aligned");
    const HeadPlan p = head_plan(desc, n, rects, nullptr);
    if (!d_workspace || workspace_bytes < p.part1_end)
        return fail(MDLSTM_ERR_WORKSPACE, "head workspace of %zu bytes, %zu needed", workspace_bytes, p.part1_end);
    if (n == 0) return MDLSTM_OK;
    hipStream_t s = as_stream(stream);
    char* ws = static_cast<char*>(d_workspace);
    if (poison_requested() && (st = poison(ws, p.S, p.part1_end, s)) != MDLSTM_OK) return st;  // column sums, partials
    st = stage_head_tables(p, n, rects, ws, s);
    if (st != MDLSTM_OK) return st;
    mdl::HeadArgs a{};
    a.H = desc->hidden;
    a.K = desc->classes;
    a.canvas_w = canvas_w;
    a.n_tiles = p.n_tiles;
    a.frames = (int)p.frames;
    a.y = d_y;
    a.rects = reinterpret_cast<const int32_t*>(ws + p.rects);
    a.frame_off = reinterpret_cast<const int32_t*>(ws + p.frame_off);
    a.tiles = reinterpret_cast<const int32_t*>(ws + p.tiles);
    a.w = d_w;
    a.b = d_b;
    a.logits = d_logits;
    a.S = reinterpret_cast<float*>(ws + p.S);
    HIP_OR_FAIL(mdl::launch_head_fwd(a, s));
    return MDLSTM_OK;
}

mdlstm_status mdlstm_ctc_loss(const mdlstm_head_desc* desc, int32_t n, const mdlstm_rect* rects,
                              const int32_t* label_lens, const int32_t* labels, const float* d_logits,
                              float* d_losses, float* d_dlogits, void* d_workspace, size_t workspace_bytes,
                              void* stream) {
    mdlstm_status st = check_head_desc(desc);
    if (st != MDLSTM_OK) return st;
    st = check_head_rects(n, rects, -1, -1);
    if (st != MDLSTM_OK) return st;
    if (n > 0 && !label_lens) return fail(MDLSTM_ERR_INVALID_ARG, "label_lens is NULL");
    int64_t total = 0;
    for (int32_t i = 0; i < n; ++i) {
        if (label_lens[i] < 0 || label_lens[i] > kMaxLabel)
            return fail(MDLSTM_ERR_UNSUPPORTED, "example %d: %d labels; 0 to %d are supported", i, label_lens[i],
                        kMaxLabel);
        total += label_lens[i];
    }
    if (total > 0 && !labels) return fail(MDLSTM_ERR_INVALID_ARG, "labels is NULL");
    int64_t o = 0;
    for (int32_t i = 0; i < n; ++i) {
        int32_t repeats = 0;
        for (int32_t j = 0; j < label_lens[i]; ++j) {
            const int32_t c = labels[o + j];
            if (c < 1 || c >= desc->classes)
                return fail(MDLSTM_ERR_INVALID_ARG, "example %d label %d is class %d; 1 to %d are labels (0 is the blank)",
                            i, j, c, desc->classes - 1);
            if (j > 0 && c == labels[o + j - 1]) ++repeats;
        }
        if ((int64_t)label_lens[i] + repeats > rects[i].w)
            return fail(MDLSTM_ERR_INVALID_ARG, "example %d: %d labels (%d repeats) cannot be aligned to %d frames", i,
                        label_lens[i], repeats, rects[i].w);
        o += label_lens[i];
    }
    if (n > 0 && (!d_logits || !d_losses || !d_dlogits)) return fail(MDLSTM_ERR_INVALID_ARG, "a device pointer is NULL");
    if (misaligned(d_workspace)) return fail(MDLSTM_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
    const HeadPlan p = head_plan(desc, n, rects, label_lens);
    if (!d_workspace || workspace_bytes < p.total)
        return fail(MDLSTM_ERR_WORKSPACE, "CTC workspace of %zu bytes, %zu needed", workspace_bytes, p.total);
    if (n == 0) return MDLSTM_OK;
    hipStream_t s = as_stream(stream);
    char* ws = static_cast<char*>(d_workspace);
    if (poison_requested() && (st = poison(ws, p.lp, p.total, s)) != MDLSTM_OK) return st;  // softmax, scan variables
    // frame offsets (first part) and the label tables (second part)
    std::vector<int32_t> fo((size_t)n + 1);
    int32_t f = 0;
    for (int32_t i = 0; i < n; ++i) {
        fo[i] = f;
        f += rects[i].w;
    }
    fo[n] = f;
    std::vector<unsigned char> host(p.lp - p.lab_off, 0);
    int32_t* lo = reinterpret_cast<int32_t*>(host.data());
    int32_t* occ = reinterpret_cast<int32_t*>(host.data() + (p.occ - p.lab_off));
    int32_t l = 0;
    for (int32_t i = 0; i < n; ++i) {
        lo[i] = l;
        l += label_lens[i];
    }
    lo[n] = l;
    if (total > 0) std::memcpy(host.data() + (p.lab - p.lab_off), labels, (size_t)total * 4);
    // per label: the next occurrence of its class in the example (all ones
    // when none) and, in bit 30, whether it is the class's first occurrence
    {
        std::vector<int32_t> last((size_t)desc->classes, -1);
        for (int32_t i = 0; i < n; ++i) {
            const int32_t* lb = labels + lo[i];
            for (int32_t j = label_lens[i] - 1; j >= 0; --j) {
                occ[lo[i] + j] = last[lb[j]] >= 0 ? last[lb[j]] : 0x3fffffff;
                last[lb[j]] = j;
            }
            for (int32_t j = 0; j < label_lens[i]; ++j) {
                if (last[lb[j]] == j) occ[lo[i] + j] |= 1 << 30;  // after the loop above: the first occurrence
                last[lb[j]] = -1;
            }
        }
    }
    HIP_OR_FAIL(hipMemcpyAsync(ws + p.frame_off, fo.data(), fo.size() * 4, hipMemcpyHostToDevice, s));
    HIP_OR_FAIL(hipMemcpyAsync(ws + p.lab_off, host.data(), host.size(), hipMemcpyHostToDevice, s));
    mdl::CtcArgs c{};
    c.n = n;
    c.K = desc->classes;
    c.nm = p.nm;
    c.frames = p.frames;
    c.frame_off = reinterpret_cast<const int32_t*>(ws + p.frame_off);
    c.lab_off = reinterpret_cast<const int32_t*>(ws + p.lab_off);
    c.labels = reinterpret_cast<const int32_t*>(ws + p.lab);
    c.occ = reinterpret_cast<const int32_t*>(ws + p.occ);
    c.logits = d_logits;
    c.y = reinterpret_cast<double*>(ws + p.lp);
    {
        const size_t rows = (size_t)std::max<int64_t>(p.frames, 1) * 64 * p.nm;
        c.am = reinterpret_cast<double*>(ws + p.alpha);
        c.ae = reinterpret_cast<int32_t*>(ws + p.alpha + align_up(rows * 8));
        c.bm = reinterpret_cast<double*>(ws + p.beta);
        c.be = reinterpret_cast<int32_t*>(ws + p.beta + align_up(rows * 8));
    }
    c.losses = d_losses;
    c.dlogits = d_dlogits;
    HIP_OR_FAIL(mdl::launch_ctc(c, s));
    return MDLSTM_OK;
}

mdlstm_status mdlstm_head_backward(const mdlstm_head_desc* desc, int32_t canvas_h, int32_t canvas_w, int32_t n,
                                   const mdlstm_rect* rects, const float* d_w, const float* d_dlogits, float* d_dy,
                                   float* d_dw, float* d_db, void* d_workspace, size_t workspace_bytes,
                                   void* stream) {
    mdlstm_status st = check_head_desc(desc);
    if (st != MDLSTM_OK) return st;
    if (canvas_h < 0) return fail(MDLSTM_ERR_INVALID_ARG, "canvas_h is negative");
    st = check_head_rects(n, rects, canvas_h, canvas_w);
    if (st != MDLSTM_OK) return st;
    if (!d_dw || !d_db) return fail(MDLSTM_ERR_INVALID_ARG, "a weight-gradient pointer is NULL");
    const int64_t canvas_floats = (int64_t)canvas_h * canvas_w * 4 * desc->hidden;
    if (canvas_floats > 0 && !d_dy) return fail(MDLSTM_ERR_INVALID_ARG, "dy is NULL");
    if (n > 0 && (!d_w || !d_dlogits)) return fail(MDLSTM_ERR_INVALID_ARG, "w or dlogits is NULL");
    if (misaligned(d_dy) || misaligned(d_w) || misaligned(d_workspace))
        return fail(MDLSTM_ERR_INVALID_ARG, "dy, w and workspace must be 16-byte aligned");
    const HeadPlan p = head_plan(desc, n, rects, nullptr);
    if (!d_workspace || workspace_bytes < p.part1_end)
        return fail(MDLSTM_ERR_WORKSPACE, "head workspace of %zu bytes, %zu needed", workspace_bytes, p.part1_end);
    hipStream_t s = as_stream(stream);
    char* ws = static_cast<char*>(d_workspace);
    // the weight-gradient partials (the column sums are the forward's)
    if (poison_requested() && n > 0 && (st = poison(ws, p.part, p.part1_end, s)) != MDLSTM_OK) return st;
    if (n > 0) {
        st = stage_head_tables(p, n, rects, ws, s);
        if (st != MDLSTM_OK) return st;
    }
    mdl::HeadArgs a{};
    a.H = desc->hidden;
    a.K = desc->classes;
    a.canvas_w = canvas_w;
    a.n_tiles = p.n_tiles;
    a.frames = (int)p.frames;
    a.rects = reinterpret_cast<const int32_t*>(ws + p.rects);
    a.frame_off = reinterpret_cast<const int32_t*>(ws + p.frame_off);
    a.tiles = reinterpret_cast<const int32_t*>(ws + p.tiles);
    a.w = d_w;
    a.S = reinterpret_cast<float*>(ws + p.S);
    a.dlogits = d_dlogits;
    a.dy = d_dy;
    a.part = reinterpret_cast<float*>(ws + p.part);
    a.dw = d_dw;
    a.db = d_db;
    HIP_OR_FAIL(mdl::launch_head_bwd(a, canvas_floats, s));
    return MDLSTM_OK;
}

// ---------------------------------------------------------------------------
// Stack glue: block reshape and grouped block convolution between layers.
// ---------------------------------------------------------------------------
namespace {

constexpr int kMaxConvChunks = 512;

constexpr int32_t kMaxConvWidth = 1 << 12;  // hidden and og beyond any built shape

size_t blocks_ws_bytes(int32_t n, int32_t hidden, int32_t og) {
    const size_t nn = n > 0 ? (size_t)n : 1;
    size_t b = align_up(nn * 8) + 2 * align_up(nn * 16) + align_up((nn + 1) * 4);
    if (hidden > 0 && og > 0)
        b += align_up((size_t)kMaxConvChunks * ((size_t)4 * og * 8 * hidden + (size_t)4 * og) * 4);
    return b;
}

struct BlockWs {
    void** ptrs;
    int32_t* in_rects;
    int32_t* out_rects;
    int32_t* blk_off;
    float* partial;
};

BlockWs block_ws(void* d_workspace, int32_t n) {
    const size_t nn = n > 0 ? (size_t)n : 1;
    char* ws = static_cast<char*>(d_workspace);
    BlockWs w;
    w.ptrs = reinterpret_cast<void**>(ws);
    ws += align_up(nn * 8);
    w.in_rects = reinterpret_cast<int32_t*>(ws);
    ws += align_up(nn * 16);
    w.out_rects = reinterpret_cast<int32_t*>(ws);
    ws += align_up(nn * 16);
    w.blk_off = reinterpret_cast<int32_t*>(ws);
    ws += align_up((nn + 1) * 4);
    w.partial = reinterpret_cast<float*>(ws);
    return w;
}

// Block offsets (prefix sums of the block rectangles' areas) into off[n + 1].
mdlstm_status block_offsets(int32_t n, const mdlstm_rect* r, std::vector<int32_t>& off) {
    off.assign((size_t)n + 1, 0);
    int64_t t = 0;
    for (int32_t k = 0; k < n; ++k) {
        off[k] = (int32_t)t;
        t += (int64_t)r[k].h * r[k].w;
        if (t > INT32_MAX / 64) return fail(MDLSTM_ERR_UNSUPPORTED, "too many blocks (%lld)", (long long)t);
    }
    off[n] = (int32_t)t;
    return MDLSTM_OK;
}

// Shared validation of the convolution calls; fills the kernel arguments.
mdlstm_status conv_prepare(int32_t n, int32_t hidden, int32_t og, int32_t bh, int32_t bw, const mdlstm_rect* in_rects,
                           int32_t in_h, int32_t in_w, const float* d_y, const float* d_w,
                           const mdlstm_rect* out_rects, int32_t out_h, int32_t out_w, void* d_workspace,
                           size_t workspace_bytes, std::vector<int32_t>& off, mdl::ConvArgs& a) {
    if (n < 0) return fail(MDLSTM_ERR_INVALID_ARG, "n is negative");
    if (!mdl::conv_supported(hidden, og, bh, bw))
        return fail(MDLSTM_ERR_UNSUPPORTED, "block convolution hidden %d, og %d, block %dx%d not built", hidden, og,
                    bh, bw);
    if (in_h < 0 || in_w < 0 || out_h < 0 || out_w < 0 || in_h > kMaxDim || in_w > kMaxDim || out_h > kMaxDim ||
        out_w > kMaxDim)
        return fail(MDLSTM_ERR_INVALID_ARG, "canvas size out of range");
    int32_t mh = 0;
    mdlstm_status st = check_rects(n, in_rects, in_h, in_w, &mh, kMaxDim);
    if (st != MDLSTM_OK) return st;
    st = check_rects(n, out_rects, out_h, out_w, &mh, kMaxDim);
    if (st != MDLSTM_OK) return st;
    for (int32_t k = 0; k < n; ++k)
        if (in_rects[k].h != bh * out_rects[k].h || in_rects[k].w != bw * out_rects[k].w)
            return fail(MDLSTM_ERR_BAD_LAYOUT, "example %d: input %dx%d is not %dx%d blocks of %dx%d", k,
                        in_rects[k].h, in_rects[k].w, out_rects[k].h, out_rects[k].w, bh, bw);
    if (!d_w) return fail(MDLSTM_ERR_INVALID_ARG, "weights are NULL");
    if ((int64_t)in_h * in_w > 0 && !d_y) return fail(MDLSTM_ERR_INVALID_ARG, "input canvas is NULL");
    if (!d_workspace || workspace_bytes < blocks_ws_bytes(n, hidden, og))
        return fail(MDLSTM_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace_bytes,
                    blocks_ws_bytes(n, hidden, og));
    if (misaligned(d_y) || misaligned(d_w) || misaligned(d_workspace))
        return fail(MDLSTM_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
    st = block_offsets(n, out_rects, off);
    if (st != MDLSTM_OK) return st;
    const BlockWs w = block_ws(d_workspace, n);
    a = mdl::ConvArgs{};
    a.n = n;
    a.total_blocks = off[n];
    a.hidden = hidden;
    a.og = og;
    a.bh = bh;
    a.bw = bw;
    a.blk_off = w.blk_off;
    a.in_rects = w.in_rects;
    a.in_w = in_w;
    a.out_rects = w.out_rects;
    a.out_w = out_w;
    a.y = d_y;
    a.w = d_w;
    a.partial = w.partial;
    return MDLSTM_OK;
}

mdlstm_status conv_stage(int32_t n, const mdlstm_rect* in_rects, const mdlstm_rect* out_rects,
                         const std::vector<int32_t>& off, void* d_workspace, hipStream_t s) {
    if (n == 0) return MDLSTM_OK;
    const BlockWs w = block_ws(d_workspace, n);
    HIP_OR_FAIL(hipMemcpyAsync(w.in_rects, in_rects, (size_t)n * 16, hipMemcpyHostToDevice, s));
    HIP_OR_FAIL(hipMemcpyAsync(w.out_rects, out_rects, (size_t)n * 16, hipMemcpyHostToDevice, s));
    HIP_OR_FAIL(hipMemcpyAsync(w.blk_off, off.data(), ((size_t)n + 1) * 4, hipMemcpyHostToDevice, s));
    return MDLSTM_OK;
}

}  // namespace

size_t mdlstm_blocks_workspace_bytes(int32_t n, int32_t hidden, int32_t og) {
    if (n < 0 || hidden < 0 || og < 0 || n > kMaxRects || hidden > kMaxConvWidth || og > kMaxConvWidth) return 0;
    return blocks_ws_bytes(n, hidden, og);
}

mdlstm_status mdlstm_pack_blocks(int32_t n, const float* const* d_images, int32_t c, int32_t bh, int32_t bw,
                                 const mdlstm_rect* rects, int32_t canvas_h, int32_t canvas_w, float* d_canvas,
                                 void* d_workspace, size_t workspace_bytes, void* stream) {
    if (n < 0 || c < 1 || bh < 1 || bw < 1 || (int64_t)bh * bw * c > 4096)
        return fail(MDLSTM_ERR_INVALID_ARG, "n %d, c %d, block %dx%d out of range", n, c, bh, bw);
    if (canvas_h < 0 || canvas_w < 0 || canvas_h > kMaxDim || canvas_w > kMaxDim)
        return fail(MDLSTM_ERR_INVALID_ARG, "canvas %dx%d out of range", canvas_h, canvas_w);
    if ((int64_t)canvas_h * canvas_w > 0 && !d_canvas) return fail(MDLSTM_ERR_INVALID_ARG, "canvas is NULL");
    int32_t mh = 0;
    mdlstm_status st = check_rects(n, rects, canvas_h, canvas_w, &mh, kMaxDim);
    if (st != MDLSTM_OK) return st;
    if (n > 0 && !d_images) return fail(MDLSTM_ERR_INVALID_ARG, "image array is NULL");
    for (int32_t k = 0; k < n; ++k)
        if (!d_images[k]) return fail(MDLSTM_ERR_INVALID_ARG, "image %d is NULL", k);
    if (!d_workspace || workspace_bytes < blocks_ws_bytes(n, 0, 0))
        return fail(MDLSTM_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace_bytes,
                    blocks_ws_bytes(n, 0, 0));
    std::vector<int32_t> off;
    st = block_offsets(n, rects, off);
    if (st != MDLSTM_OK) return st;
    hipStream_t s = as_stream(stream);
    HIP_OR_FAIL(mdl::launch_zero_f32(d_canvas, (int64_t)canvas_h * canvas_w * bh * bw * c, s));
    if (n == 0) return MDLSTM_OK;
    const BlockWs w = block_ws(d_workspace, n);
    HIP_OR_FAIL(hipMemcpyAsync(w.ptrs, d_images, (size_t)n * 8, hipMemcpyHostToDevice, s));
    HIP_OR_FAIL(hipMemcpyAsync(w.out_rects, rects, (size_t)n * 16, hipMemcpyHostToDevice, s));
    HIP_OR_FAIL(hipMemcpyAsync(w.blk_off, off.data(), ((size_t)n + 1) * 4, hipMemcpyHostToDevice, s));
    HIP_OR_FAIL(mdl::launch_pack_blocks(n, reinterpret_cast<const float* const*>(w.ptrs), w.blk_off, off[n],
                                        w.out_rects, canvas_w, c, bh, bw, d_canvas, s));
    return MDLSTM_OK;
}

mdlstm_status mdlstm_block_conv_forward(int32_t n, int32_t hidden, int32_t og, int32_t bh, int32_t bw,
                                        const mdlstm_rect* in_rects, int32_t in_h, int32_t in_w, const float* d_y,
                                        const float* d_w, const float* d_b, const mdlstm_rect* out_rects,
                                        int32_t out_h, int32_t out_w, float* d_out, void* d_workspace,
                                        size_t workspace_bytes, void* stream) {
    std::vector<int32_t> off;
    mdl::ConvArgs a;
    mdlstm_status st = conv_prepare(n, hidden, og, bh, bw, in_rects, in_h, in_w, d_y, d_w, out_rects, out_h, out_w,
                                    d_workspace, workspace_bytes, off, a);
    if (st != MDLSTM_OK) return st;
    if (!d_b) return fail(MDLSTM_ERR_INVALID_ARG, "bias is NULL");
    if ((int64_t)out_h * out_w > 0 && !d_out) return fail(MDLSTM_ERR_INVALID_ARG, "output canvas is NULL");
    if (misaligned(d_b) || misaligned(d_out)) return fail(MDLSTM_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
    a.b = d_b;
    a.out = d_out;
    hipStream_t s = as_stream(stream);
    HIP_OR_FAIL(mdl::launch_zero_f32(d_out, (int64_t)out_h * out_w * 4 * og, s));
    st = conv_stage(n, in_rects, out_rects, off, d_workspace, s);
    if (st != MDLSTM_OK) return st;
    HIP_OR_FAIL(mdl::launch_block_conv(true, a, s));
    return MDLSTM_OK;
}

mdlstm_status mdlstm_block_conv_backward(int32_t n, int32_t hidden, int32_t og, int32_t bh, int32_t bw,
                                         const mdlstm_rect* in_rects, int32_t in_h, int32_t in_w, const float* d_y,
                                         const float* d_w, const mdlstm_rect* out_rects, int32_t out_h,
                                         int32_t out_w, const float* d_out, const float* d_dout, float* d_dy,
                                         float* d_dw, float* d_db, void* d_workspace, size_t workspace_bytes,
                                         void* stream) {
    std::vector<int32_t> off;
    mdl::ConvArgs a;
    mdlstm_status st = conv_prepare(n, hidden, og, bh, bw, in_rects, in_h, in_w, d_y, d_w, out_rects, out_h, out_w,
                                    d_workspace, workspace_bytes, off, a);
    if (st != MDLSTM_OK) return st;
    if (!d_dw || !d_db) return fail(MDLSTM_ERR_INVALID_ARG, "a weight-gradient pointer is NULL");
    if ((int64_t)out_h * out_w > 0 && (!d_out || !d_dout))
        return fail(MDLSTM_ERR_INVALID_ARG, "output or its gradient is NULL");
    if ((int64_t)in_h * in_w > 0 && !d_dy) return fail(MDLSTM_ERR_INVALID_ARG, "input gradient is NULL");
    if (misaligned(d_out) || misaligned(d_dout) || misaligned(d_dy) || misaligned(d_dw) || misaligned(d_db))
        return fail(MDLSTM_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
    a.out = const_cast<float*>(d_out);
    a.dout = d_dout;
    a.dy = d_dy;
    a.dw = d_dw;
    a.db = d_db;
    hipStream_t s = as_stream(stream);
    HIP_OR_FAIL(mdl::launch_zero_f32(d_dy, (int64_t)in_h * in_w * 4 * hidden, s));
    if (a.total_blocks == 0) {  // empty batch: zero gradients
        HIP_OR_FAIL(mdl::launch_zero_f32(d_dw, (int64_t)4 * og * bh * bw * hidden, s));
        HIP_OR_FAIL(mdl::launch_zero_f32(d_db, (int64_t)4 * og, s));
        return MDLSTM_OK;
    }
    st = conv_stage(n, in_rects, out_rects, off, d_workspace, s);
    if (st != MDLSTM_OK) return st;
    HIP_OR_FAIL(mdl::launch_block_conv(false, a, s));
    return MDLSTM_OK;
}

}  // extern "C"
