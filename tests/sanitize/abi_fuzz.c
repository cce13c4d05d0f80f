/*
 * Host-side validation of the C ABI under AddressSanitizer and
 * UndefinedBehaviorSanitizer (test infrastructure, not part of the library).
 *
 * Linked against a build of the library whose host code is instrumented, this
 * program drives every entry point with seeded random arguments: valid and
 * invalid descriptors, canvases and rectangle lists, extreme sizes, NULL and
 * misaligned pointers. Each call that takes device memory is given at least
 * one defect that the host checks must reject (a workspace one byte short or
 * smaller, a NULL or misaligned pointer, an invalid size), so no call reaches
 * the device: a status of MDLSTM_ERR_DEVICE or MDLSTM_OK there is a failure,
 * as is any sanitizer report. The pure host calls (workspace sizes, the
 * padding layout without a mask, the fused-gradient query) run on valid and
 * invalid arguments and their results are checked for consistency.
 *
 * Usage: abi_fuzz [iterations]. Prints one summary line; exit status 0 when
 * every check held.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "mdlstm.h"

static uint64_t g_rng = 0x9e3779b97f4a7c15ull;
static uint64_t next_u64(void) { /* xorshift64* (Vigna) */
    g_rng ^= g_rng >> 12;
    g_rng ^= g_rng << 25;
    g_rng ^= g_rng >> 27;
    return g_rng * 0x2545f4914f6cdd1dull;
}
static int32_t uniform(int32_t lo, int32_t hi) { /* inclusive */
    return lo + (int32_t)(next_u64() % (uint64_t)((int64_t)hi - lo + 1));
}
static int chance(int percent) { return (int)(next_u64() % 100) < percent; }

/* A size drawn from the ordinary range most of the time and from the edges
 * (zero, negative, the canvas limit, INT32_MAX) otherwise. */
static int32_t any_size(int32_t typical) {
    switch (uniform(0, 9)) {
        case 0: return 0;
        case 1: return -uniform(1, 1000);
        case 2: return INT32_MAX - uniform(0, 3);
        case 3: return (1 << 21) - uniform(0, 1);
        case 4: return INT32_MIN + uniform(0, 3);
        default: return uniform(1, typical);
    }
}

/* v * k + a saturated to the int32 range (the driver's own arithmetic on
 * extreme sizes stays defined). */
static int32_t sat(int32_t v, int32_t k, int32_t a) {
    const int64_t r = (int64_t)v * k + a;
    return r > INT32_MAX ? INT32_MAX : r < INT32_MIN ? INT32_MIN : (int32_t)r;
}

static long g_checks = 0, g_failures = 0;
#define CHECK(cond, ...)                                   \
    do {                                                   \
        ++g_checks;                                        \
        if (!(cond)) {                                     \
            ++g_failures;                                  \
            if (g_failures <= 20) {                        \
                fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
                fprintf(stderr, __VA_ARGS__);              \
                fprintf(stderr, "\n");                     \
            }                                              \
        }                                                  \
    } while (0)

/* Device addresses that are never dereferenced: every call below is rejected
 * on the host before any device access. */
#define FAKE ((void*)(uintptr_t)0x100000)
#define FAKE_MIS ((void*)(uintptr_t)0x100004)

/* Status counts per entry point, so that the run shows the random arguments
 * reach every stage of the host checks (the workspace check comes last). */
enum { N_FN = 16, N_ST = 8 };
static const char* g_fn[N_FN];
static long g_hist[N_FN][N_ST];
static void tally(const char* what, mdlstm_status st) {
    int i = 0;
    while (i < N_FN && g_fn[i] && strcmp(g_fn[i], what) != 0) ++i;
    if (i == N_FN) return;
    g_fn[i] = what;
    if ((int)st >= 0 && (int)st < N_ST) ++g_hist[i][st];
}

/* A rejected call: not OK, not a device error, and a message is set. */
static void expect_rejected(mdlstm_status st, const char* what) {
    tally(what, st);
    CHECK(st != MDLSTM_OK && st != MDLSTM_ERR_DEVICE, "%s returned %d", what, (int)st);
    const char* m = mdlstm_last_error();
    CHECK(m != NULL && m[0] != 0 && strlen(m) < 4096, "%s left no message", what);
}

static mdlstm_layer_desc random_desc(void) {
    static const int32_t hs[] = {4, 8, 16, 32, 64, 128, 12, 0, -4, 1 << 20};
    mdlstm_layer_desc d;
    d.c_in = chance(80) ? 4 * uniform(1, 64) : any_size(300);
    d.hidden = hs[uniform(0, 9)];
    d.dtype = chance(90) ? uniform(0, 1) : uniform(-3, 9);
    d.memory_states = chance(85) ? uniform(0, 1) : uniform(-2, 5);
    return d;
}

/* Rectangles: a valid column of disjoint rectangles, or one with a defect. */
static int32_t random_rects(mdlstm_rect* r, int32_t max_n, int32_t* ch, int32_t* cw) {
    const int32_t n = uniform(0, max_n);
    int32_t y = 0;
    *cw = uniform(1, 300);
    for (int32_t k = 0; k < n; ++k) {
        r[k].h = uniform(1, 70);
        r[k].w = uniform(1, *cw);
        r[k].y0 = y;
        r[k].x0 = uniform(0, *cw - r[k].w);
        y += r[k].h + uniform(0, 2);
    }
    *ch = y + uniform(0, 3);
    if (n > 0 && chance(50)) {
        const int32_t k = uniform(0, n - 1);
        switch (uniform(0, 5)) {
            case 0: r[k].h = any_size(10); break;
            case 1: r[k].w = any_size(10); break;
            case 2: r[k].y0 = any_size(*ch); break;
            case 3: r[k].x0 = any_size(*cw); break;
            case 4: if (n > 1) r[k] = r[(k + 1) % n]; break; /* overlap */
            default: *ch = any_size(*ch); break;
        }
    }
    return n;
}

static void fuzz_layer(void) {
    mdlstm_rect rects[8];
    int32_t ch, cw;
    const int32_t n = random_rects(rects, 8, &ch, &cw);
    mdlstm_layer_desc d = random_desc();
    const int32_t qch = chance(10) ? any_size(100) : ch, qcw = chance(10) ? any_size(100) : cw;
    const size_t need = mdlstm_workspace_bytes(&d, qch, qcw, n);
    const size_t again = mdlstm_workspace_bytes(&d, qch, qcw, n);
    CHECK(need == again, "workspace size not deterministic");
    /* one defect that the host checks always catch: the workspace short, or
     * the workspace or a weight pointer NULL or misaligned */
    void* p[13];
    for (int i = 0; i < 13; ++i) p[i] = chance(2) ? NULL : FAKE;
    p[12] = FAKE;
    p[2] = p[3] = p[4] = FAKE;
    size_t ws = need;
    switch (uniform(0, 2)) {
        case 0: ws = need > 0 ? need - 1 - (size_t)uniform(0, (int32_t)(need - 1 < 1000 ? need - 1 : 1000)) : 0; break;
        case 1: p[12] = chance(50) ? NULL : FAKE_MIS; break;
        default: p[uniform(2, 4)] = chance(50) ? NULL : FAKE_MIS; break;
    }
    const mdlstm_layer_desc* dp = chance(3) ? NULL : &d;
    const mdlstm_rect* rp = (n > 0 && chance(3)) ? NULL : rects;
    switch (uniform(0, 2)) {
        case 0:
            expect_rejected(mdlstm_forward(dp, qch, qcw, p[0], (const uint8_t*)p[1], n, rp, p[2], p[3], p[4], p[5],
                                           p[12], ws, NULL),
                            "mdlstm_forward");
            break;
        case 1:
            expect_rejected(mdlstm_forward_stepwise(dp, qch, qcw, p[0], (const uint8_t*)p[1], n, rp, p[2], p[3], p[4],
                                                    p[5], p[12], ws, NULL),
                            "mdlstm_forward_stepwise");
            break;
        default:
            expect_rejected(mdlstm_backward(dp, qch, qcw, p[0], (const uint8_t*)p[1], n, rp, p[2], p[3], p[4], p[5],
                                            p[6], p[7], (float*)p[8], (float*)p[9], (float*)p[10], p[12], ws, NULL),
                            "mdlstm_backward");
            break;
    }
    const int32_t f = mdlstm_gradients_fused(dp);
    CHECK(f == -1 || f == 0 || f == 1, "gradients_fused returned %d", f);
}

static void fuzz_pack(void) {
    enum { N = 40 };
    int32_t hs[N], ws[N];
    mdlstm_rect rects[N], place[N];
    const int32_t n = chance(5) ? any_size(N) : uniform(0, N);
    const int32_t m = n > 0 && n <= N ? n : 0;
    int32_t cw = chance(80) ? uniform(1, 200) : any_size(200);
    for (int32_t k = 0; k < m; ++k) {
        hs[k] = chance(95) ? uniform(1, 40) : any_size(40);
        ws[k] = chance(95) ? uniform(1, 200) : any_size(200);
    }
    int32_t ch = -7;
    const size_t pws = mdlstm_pack_workspace_bytes(n);
    CHECK(pws > 0, "pack workspace 0");
    /* placement with a workspace one byte short (or a size defect) */
    mdlstm_status st = mdlstm_pack_layout(n, m ? hs : NULL, m ? ws : NULL, cw, rects, &ch, NULL, 0, FAKE,
                                          pws - 1, NULL);
    if (n != 0 || cw < 1 || cw >= (1 << 21)) expect_rejected(st, "mdlstm_pack_layout");
    else CHECK(st == MDLSTM_OK && ch == 0, "empty placement: %d %s", (int)st, mdlstm_last_error());
    if (n > MDLSTM_NOALLOC_MAX_N || n < 0) {
        expect_rejected(mdlstm_pack_layout_noalloc(n, m ? hs : NULL, m ? ws : NULL, cw, rects, &ch, NULL, 0, NULL),
                        "mdlstm_pack_layout_noalloc");
    }
    /* the padding layout without a mask is host-only: valid inputs must succeed */
    int32_t pch = -1, pcw = -1;
    st = mdlstm_pad_layout(n, m ? hs : NULL, m ? ws : NULL, rects, place, &pch, &pcw, NULL, 0, NULL, 0, NULL);
    int valid = n >= 0 && n <= N;
    int32_t hm = 0, wm = 0;
    for (int32_t k = 0; k < m; ++k) {
        if (hs[k] < 1 || ws[k] < 1 || hs[k] >= (1 << 21) || ws[k] >= (1 << 21)) valid = 0;
        if (hs[k] > hm) hm = hs[k];
        if (ws[k] > wm) wm = ws[k];
    }
    if (valid && (int64_t)hm * m < (1 << 21)) {
        CHECK(st == MDLSTM_OK, "pad_layout rejected valid sizes: %s", mdlstm_last_error());
        CHECK(pch == m * hm && pcw == wm, "pad canvas %dx%d", pch, pcw);
        for (int32_t k = 0; k < m; ++k) {
            CHECK(rects[k].y0 == k * hm && rects[k].h == hm && rects[k].w == wm, "pad tile %d", k);
            CHECK(place[k].y0 == rects[k].y0 && place[k].x0 == 0 && place[k].h == hs[k] && place[k].w == ws[k],
                  "pad place %d", k);
        }
    } else {
        expect_rejected(st, "mdlstm_pad_layout");
    }
    /* scatter / gather: a defect each */
    const void* ex[N];
    for (int32_t k = 0; k < N; ++k) ex[k] = FAKE;
    if (m > 0) {
        int32_t gch, gcw;
        const int32_t nr = random_rects(rects, m < 8 ? m : 8, &gch, &gcw);
        if (nr > 0) {
            if (chance(50)) ex[uniform(0, nr - 1)] = NULL;
            expect_rejected(mdlstm_pack_data(nr, ex, rects, gch, gcw, uniform(1, 8), uniform(0, 1), FAKE, FAKE,
                                             mdlstm_pack_workspace_bytes(nr) - 1, NULL),
                            "mdlstm_pack_data");
            expect_rejected(mdlstm_unpack_data(nr, (void* const*)ex, rects, gch, gcw, uniform(-1, 8), uniform(0, 2),
                                               FAKE, FAKE, mdlstm_pack_workspace_bytes(nr) - 1, NULL),
                            "mdlstm_unpack_data");
        }
    }
}

static void fuzz_blocks(void) {
    mdlstm_rect in[6], out[6];
    int32_t ih, iw, oh, ow;
    const int32_t n = random_rects(out, 6, &oh, &ow);
    const int32_t bh = chance(80) ? 2 : uniform(-1, 5), bw = chance(80) ? 4 : uniform(-1, 5);
    for (int32_t k = 0; k < n; ++k) {
        in[k].y0 = sat(out[k].y0, 2, 0);
        in[k].x0 = sat(out[k].x0, 4, 0);
        in[k].h = sat(out[k].h, 2, 0);
        in[k].w = sat(out[k].w, 4, 0);
    }
    ih = sat(oh, 2, uniform(-1, 1));
    iw = sat(ow, 4, uniform(-1, 1));
    const int32_t hidden = chance(80) ? 4 * uniform(1, 16) : any_size(64);
    const int32_t og = chance(80) ? 8 * uniform(1, 4) : any_size(16);
    const size_t need = mdlstm_blocks_workspace_bytes(n, hidden, og);
    const size_t ws = need > 0 ? need - 1 : 0;
    expect_rejected(mdlstm_block_conv_forward(n, hidden, og, bh, bw, in, ih, iw, FAKE, FAKE, FAKE, out, oh, ow, FAKE,
                                              FAKE, ws, NULL),
                    "mdlstm_block_conv_forward");
    expect_rejected(mdlstm_block_conv_backward(n, hidden, og, bh, bw, in, ih, iw, FAKE, FAKE, out, oh, ow, FAKE, FAKE,
                                               FAKE, FAKE, FAKE, FAKE, ws, NULL),
                    "mdlstm_block_conv_backward");
    const float* imgs[6] = {FAKE, FAKE, FAKE, FAKE, FAKE, FAKE};
    expect_rejected(mdlstm_pack_blocks(n, imgs, uniform(-1, 4), bh, bw, out, oh, ow, FAKE, FAKE,
                                       mdlstm_blocks_workspace_bytes(n, 0, 0) - 1, NULL),
                    "mdlstm_pack_blocks");
}

static void fuzz_head(void) {
    mdlstm_rect rects[8];
    int32_t ch, cw;
    const int32_t n = random_rects(rects, 8, &ch, &cw);
    int32_t lens[8], labels[8 * 64];
    int32_t total = 0;
    for (int32_t k = 0; k < n; ++k) {
        lens[k] = chance(95) ? uniform(0, 20) : any_size(2000);
        if (lens[k] > 0 && lens[k] <= 64 && total + lens[k] <= 8 * 64) total += lens[k];
        else if (lens[k] > 64) lens[k] = chance(50) ? 64 : lens[k];
    }
    for (int32_t i = 0; i < 8 * 64; ++i) labels[i] = chance(97) ? uniform(1, 9) : uniform(-2, 12);
    mdlstm_head_desc d;
    d.hidden = chance(80) ? 4 * uniform(1, 16) : any_size(70);
    d.classes = chance(80) ? uniform(2, 10) : any_size(200);
    const size_t a = mdlstm_head_workspace_bytes(&d, n, rects, NULL);
    const size_t b = mdlstm_head_workspace_bytes(&d, n, rects, lens);
    CHECK(b == 0 || b >= a, "head workspace with labels smaller than without");
    const size_t ws = b > 0 ? b - 1 : 0;
    expect_rejected(mdlstm_head_forward(&d, ch, cw, FAKE, n, rects, FAKE, FAKE, FAKE, FAKE, a > 0 ? a - 1 : 0, NULL),
                    "mdlstm_head_forward");
    int ok_lens = 1;
    for (int32_t k = 0; k < n; ++k) ok_lens &= lens[k] >= 0 && lens[k] <= 64;
    int32_t sum = 0;
    for (int32_t k = 0; k < n && ok_lens; ++k) sum += lens[k];
    if (ok_lens && sum <= 8 * 64)
        expect_rejected(mdlstm_ctc_loss(&d, n, rects, lens, labels, FAKE, FAKE, FAKE, FAKE, ws, NULL),
                        "mdlstm_ctc_loss");
    expect_rejected(mdlstm_head_backward(&d, ch, cw, n, rects, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, a > 0 ? a - 1 : 0,
                                         NULL),
                    "mdlstm_head_backward");
}

int main(int argc, char** argv) {
    const long iters = argc > 1 ? atol(argv[1]) : 20000;
    void* none[8] = {0};
    CHECK(mdlstm_set_phase_events(3, none) == MDLSTM_ERR_INVALID_ARG, "phase events n = 3");
    CHECK(mdlstm_set_phase_events(8, NULL) == MDLSTM_ERR_INVALID_ARG, "phase events NULL");
    CHECK(mdlstm_set_phase_events(8, none) == MDLSTM_OK, "phase events set");
    CHECK(mdlstm_set_phase_events(0, NULL) == MDLSTM_OK, "phase events clear");
    CHECK(mdlstm_workspace_bytes(NULL, 1, 1, 1) == 0, "NULL desc workspace");
    for (long it = 0; it < iters; ++it) {
        fuzz_layer();
        fuzz_pack();
        if (it % 4 == 0) fuzz_blocks();
        if (it % 2 == 0) fuzz_head();
    }
    for (int i = 0; i < N_FN && g_fn[i]; ++i) {
        printf("%-28s", g_fn[i]); /* INVALID_ARG TOO_WIDE BAD_LAYOUT WORKSPACE UNSUPPORTED DEVICE NUMERIC */
        for (int st = 1; st < N_ST; ++st) printf(" %6ld", g_hist[i][st]);
        printf("\n");
        /* every entry point that takes a workspace met arguments that passed
         * all the checks before the workspace size, the last one */
        const int no_ws = !strcmp(g_fn[i], "mdlstm_pad_layout") || !strcmp(g_fn[i], "mdlstm_pack_layout_noalloc");
        if (iters >= 1000 && !no_ws)
            CHECK(g_hist[i][MDLSTM_ERR_WORKSPACE] > 0, "%s never reached its workspace check", g_fn[i]);
    }
    printf("abi_fuzz: %ld iterations, %ld checks, %ld failures\n", iters, g_checks, g_failures);
    return g_failures == 0 ? 0 : 1;
}
