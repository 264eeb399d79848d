/*
 * oracle.c -- TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.
 *
 * A plain, slow, double-precision CPU definition of the per-frame
 * video/image preprocessing that EasyVideoR1 (arXiv 2604.16893) moves out of
 * the RL loop with its offline tensor cache (Section 3.1.1, "Efficient RL
 * with Video Caching"; Section 3.1.2, "Independent Resolution Budgets";
 * Section 4.1, "Training Configuration"):
 *
 *   temporal frame-index sampling -> smart_resize of (H, W) to multiples of
 *   2P under a pixel budget -> antialiased bicubic resampling of uint8 RGB
 *   frames -> rescale by 1/255 and per-channel mean/std normalisation ->
 *   patchification into merge-window rows of 3*2*P*P values (P = 16: 1536;
 *   P = 14: 1176), with the per-item grid (t, h/P, w/P) and the row-offset
 *   table.
 *
 * The paper names these stages and their parameters (fps, max_frames,
 * max_pixels, separate image/video budgets, identical video_grid_thw in every
 * stage) but prints no formula for any of them.  Every function below states
 * the definition it writes out; where the paper is silent the reading taken
 * is stated in the comment and listed with the others in the design notes.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this library.  It shares no code, header, table or constant with
 * the GPU library; the two are compared on identical seeded inputs.
 *
 * Everything is computed in IEEE double precision, with no fused or
 * reordered arithmetic beyond what each definition states.  Build with
 * plain `gcc -O2 -fPIC -shared` (no -ffast-math, no -ffp-contract=fast).
 *
 * Parity status: every function is pinned by the CPU tests against closed
 * forms, hand-worked values or brute force (see the test suite).  The one
 * result with no closed form -- the resampled value of real-valued noise --
 * is pinned indirectly: exact weight vectors, brute-force 2D summation
 * against the separable form, a dense matrix product, identity, constants,
 * flips, and exact reproduction of quadratics under upscaling.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_OK 0
#define OR_ERR_NULL 1
#define OR_ERR_ARG 2
#define OR_ERR_ASPECT 3
#define OR_ERR_DIMS 4
#define OR_ERR_INDEX 5
#define OR_ERR_FRAMES 6
#define OR_ERR_CAPACITY 7
#define OR_ERR_NOMEM 9

/* Geometry of a Qwen-VL-style vision input: a patch of P x P pixels
 * (P = 16 for Qwen3-VL, 14 for Qwen2-VL and Qwen2.5-VL), spatial merge 2,
 * temporal patch 2, so a merge-window row holds 3 * 2 * P * P values
 * (1536 or 1176).  P is an argument of every function that needs it. */
#define OR_MERGE 2
#define OR_TPATCH 2
#define OR_ROW(P) (3 * OR_TPATCH * (P) * (P))

/* ------------------------------------------------------------------------ */
/* Rounding helpers                                                         */
/* ------------------------------------------------------------------------ */

/* Round half to even of a double (the rounding Python's round() applies to
 * the exact binary value).  x - floor(x) is exact for |x| < 2^52. */
static double round_half_even(double x)
{
    double f = floor(x);
    double d = x - f;
    if (d > 0.5)
        return f + 1.0;
    if (d < 0.5)
        return f;
    return (fmod(f, 2.0) == 0.0) ? f : f + 1.0;
}

/* ------------------------------------------------------------------------ */
/* smart_resize (Section 3.1.1: resize under max_pixels; Section 3.1.2:     */
/* independent image and video budgets; Section 4.1: per-frame budget)      */
/* ------------------------------------------------------------------------ */

/*
 * Target (h, w), both multiples of `factor`, for a source of height x width
 * under the per-frame budget [min_pixels, max_pixels]:
 *   1. error if any size is non-positive, min > max, or max/min side > 200;
 *   2. h = max(F, rhe(H / F) * F), w = max(F, rhe(W / F) * F);
 *   3. if h * w > max_pixels:  beta = sqrt(H * W / max_pixels),
 *        h = max(F, floor(H / beta / F) * F), w = max(F, floor(W / beta / F) * F);
 *   4. else if h * w < min_pixels:  beta = sqrt(min_pixels / (H * W)),
 *        h = ceil(H * beta / F) * F, w = ceil(W * beta / F) * F.
 * Reading: each expression is evaluated in double precision in exactly the
 * written order (H * W as an exact integer converted to double, then one
 * divide, one sqrt, then divides left to right).
 */
int oracle_smart_resize(int64_t height, int64_t width, int64_t factor,
                        int64_t min_pixels, int64_t max_pixels,
                        int64_t *out_h, int64_t *out_w)
{
    if (out_h == NULL || out_w == NULL)
        return OR_ERR_NULL;
    if (height <= 0 || width <= 0 || factor <= 0 || max_pixels <= 0 ||
        min_pixels < 0 || min_pixels > max_pixels)
        return OR_ERR_ARG;
    double H = (double)height;
    double W = (double)width;
    double F = (double)factor;
    double longer = height > width ? H : W;
    double shorter = height > width ? W : H;
    if (longer / shorter > 200.0)
        return OR_ERR_ASPECT;

    int64_t h = (int64_t)round_half_even(H / F) * factor;
    int64_t w = (int64_t)round_half_even(W / F) * factor;
    if (h < factor)
        h = factor;
    if (w < factor)
        w = factor;

    if (h * w > max_pixels) {
        double beta = sqrt((double)(height * width) / (double)max_pixels);
        h = (int64_t)floor(H / beta / F) * factor;
        w = (int64_t)floor(W / beta / F) * factor;
        if (h < factor)
            h = factor;
        if (w < factor)
            w = factor;
    } else if (h * w < min_pixels) {
        double beta = sqrt((double)min_pixels / (double)(height * width));
        h = (int64_t)ceil(H * beta / F) * factor;
        w = (int64_t)ceil(W * beta / F) * factor;
    }
    *out_h = h;
    *out_w = w;
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Frame-index sampling (Section 3.1.1: cache key (path, fps, max_frames,   */
/* max_pixels); Section 4.1: 2 FPS with at most 128 frames)                 */
/* ------------------------------------------------------------------------ */

/*
 * Uniform mode: n indices spread over [0, N-1]:
 *   idx_i = round_half_even(i * (N - 1) / (n - 1)),  i = 0 .. n-1  (n >= 2),
 *   idx_0 = 0 for n = 1.
 * Reading: the rounding is done on the exact rational, in integers, so the
 * result does not depend on any floating-point linspace.
 */
int oracle_sample_uniform(int64_t total, int64_t n, int32_t *out)
{
    if (out == NULL)
        return OR_ERR_NULL;
    if (total < 1 || n < 1 || n > total)
        return OR_ERR_FRAMES;
    if (n == 1) {
        out[0] = 0;
        return OR_OK;
    }
    for (int64_t i = 0; i < n; i++) {
        int64_t num = i * (total - 1);
        int64_t den = n - 1;
        int64_t q = num / den;
        int64_t r = num % den;
        if (2 * r > den || (2 * r == den && (q % 2) == 1))
            q += 1;
        out[i] = (int32_t)q;
    }
    return OR_OK;
}

/*
 * Fps mode: the count follows the clip's duration at the target rate,
 *   n_raw = N / video_fps * fps                         (double),
 *   n     = min(max(n_raw, ceil_even(min_frames)), floor_even(max_frames), N),
 *   n     = 2 * floor(n / 2),
 * an error if n < 2, then the indices of uniform mode for that n.
 * Reading: the temporal patch of 2 makes the count even.
 */
int oracle_sample_fps(int64_t total, double video_fps, double fps,
                      int64_t min_frames, int64_t max_frames,
                      int32_t *out, int64_t capacity, int64_t *count)
{
    if (count == NULL)
        return OR_ERR_NULL;
    if (total < 1 || !(video_fps > 0.0) || !(fps > 0.0) || min_frames < 1 ||
        max_frames < min_frames)
        return OR_ERR_ARG;
    int64_t lo = ((min_frames + 1) / 2) * 2;
    int64_t hi = (max_frames / 2) * 2;
    double n = (double)total / video_fps * fps;
    if (n < (double)lo)
        n = (double)lo;
    if (n > (double)hi)
        n = (double)hi;
    if (n > (double)total)
        n = (double)total;
    int64_t k = (int64_t)floor(n / 2.0) * 2;
    if (k < 2)
        return OR_ERR_FRAMES;
    *count = k;
    if (out == NULL || capacity < k)
        return OR_ERR_CAPACITY;
    return oracle_sample_uniform(total, k, out);
}

/* ------------------------------------------------------------------------ */
/* Antialiased bicubic filter weights                                       */
/* ------------------------------------------------------------------------ */

/*
 * Keys (1981) cubic convolution kernel with a = -0.5:
 *   K(x) = (a+2)|x|^3 - (a+3)|x|^2 + 1        for |x| < 1,
 *   K(x) = a|x|^3 - 5a|x|^2 + 8a|x| - 4a       for 1 <= |x| < 2,
 *   K(x) = 0                                   otherwise.
 */
double oracle_keys_cubic(double x)
{
    const double a = -0.5;
    double t = fabs(x);
    if (t < 1.0)
        return (a + 2.0) * t * t * t - (a + 3.0) * t * t + 1.0;
    if (t < 2.0)
        return a * t * t * t - 5.0 * a * t * t + 8.0 * a * t - 4.0 * a;
    return 0.0;
}

/*
 * Window and normalised weights of output sample i when n_in samples are
 * resampled to n_out.  With scale s = n_in / n_out, the kernel is stretched
 * by sigma = max(s, 1) (that stretch is the antialiasing), so its support is
 * r = 2 * sigma input samples on each side of the centre c = (i + 0.5) * s.
 *   lo = max(0, floor(c - r + 0.5)),  hi = min(n_in, floor(c + r + 0.5)),
 *   u_j = K((j + 0.5 - c) / sigma) for lo <= j < hi,   w_j = u_j / sum(u).
 * Readings: the window is truncated at the borders and renormalised (no edge
 * replication); a = -0.5; double-precision evaluation in the written order.
 * `w` must hold at least `cap` doubles; returns OR_ERR_CAPACITY if the
 * window is longer.
 */
int oracle_filter(int64_t n_in, int64_t n_out, int64_t i,
                  int64_t *lo, int64_t *count, double *w, int64_t cap)
{
    if (lo == NULL || count == NULL || w == NULL)
        return OR_ERR_NULL;
    if (n_in < 1 || n_out < 1 || i < 0 || i >= n_out)
        return OR_ERR_ARG;
    double scale = (double)n_in / (double)n_out;
    double sigma = scale > 1.0 ? scale : 1.0;
    double support = 2.0 * sigma;
    double center = ((double)i + 0.5) * scale;
    int64_t a = (int64_t)floor(center - support + 0.5);
    int64_t b = (int64_t)floor(center + support + 0.5);
    if (a < 0)
        a = 0;
    if (b > n_in)
        b = n_in;
    int64_t n = b - a;
    *lo = a;
    *count = n;
    if (n > cap)
        return OR_ERR_CAPACITY;
    double total = 0.0;
    for (int64_t j = a; j < b; j++) {
        double u = oracle_keys_cubic(((double)j + 0.5 - center) / sigma);
        w[j - a] = u;
        total += u;
    }
    for (int64_t k = 0; k < n; k++)
        w[k] = w[k] / total;
    return OR_OK;
}

/* Longest window over all outputs of one axis. */
int64_t oracle_filter_max_taps(int64_t n_in, int64_t n_out)
{
    int64_t best = 0;
    double scratch[4096];
    for (int64_t i = 0; i < n_out; i++) {
        int64_t lo, cnt;
        if (oracle_filter(n_in, n_out, i, &lo, &cnt, scratch, 4096) != OR_OK)
            return -1;
        if (cnt > best)
            best = cnt;
    }
    return best;
}

/* Full table of one axis: lo[n_out], count[n_out], w[n_out][cap]
 * (zero beyond each window). */
int oracle_filter_table(int64_t n_in, int64_t n_out, int64_t *lo, int64_t *count,
                        double *w, int64_t cap)
{
    for (int64_t i = 0; i < n_out; i++) {
        for (int64_t k = 0; k < cap; k++)
            w[i * cap + k] = 0.0;
        int st = oracle_filter(n_in, n_out, i, &lo[i], &count[i], &w[i * cap], cap);
        if (st != OR_OK)
            return st;
    }
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Resampling of one frame                                                  */
/* ------------------------------------------------------------------------ */

/*
 * Separable resampling of one packed RGB frame F[H][W][3] (uint8) to
 * R[3][h][w] (double):  R[c][i][j] = sum_y wy[i][y] * sum_x wx[j][x] * F[y][x][c],
 * first along x for every source row, then along y.  No clamping and no
 * rounding between or after the two passes (the value may overshoot
 * [0, 255] through the negative lobes of the kernel).
 */
int oracle_resize_frame(const uint8_t *frame, int64_t H, int64_t W, int64_t h, int64_t w,
                        double *out)
{
    if (frame == NULL || out == NULL)
        return OR_ERR_NULL;
    if (H < 1 || W < 1 || h < 1 || w < 1)
        return OR_ERR_DIMS;
    int64_t kx = oracle_filter_max_taps(W, w);
    int64_t ky = oracle_filter_max_taps(H, h);
    if (kx < 1 || ky < 1)
        return OR_ERR_ARG;
    int64_t *xlo = malloc(sizeof(int64_t) * (size_t)w);
    int64_t *xn = malloc(sizeof(int64_t) * (size_t)w);
    double *wx = malloc(sizeof(double) * (size_t)(w * kx));
    int64_t *ylo = malloc(sizeof(int64_t) * (size_t)h);
    int64_t *yn = malloc(sizeof(int64_t) * (size_t)h);
    double *wy = malloc(sizeof(double) * (size_t)(h * ky));
    double *tmp = malloc(sizeof(double) * (size_t)(H * w * 3));
    int st = OR_ERR_NOMEM;
    if (xlo && xn && wx && ylo && yn && wy && tmp) {
        oracle_filter_table(W, w, xlo, xn, wx, kx);
        oracle_filter_table(H, h, ylo, yn, wy, ky);
        /* pass 1: along x, for every source row y */
        for (int64_t y = 0; y < H; y++)
            for (int64_t j = 0; j < w; j++)
                for (int64_t c = 0; c < 3; c++) {
                    double s = 0.0;
                    for (int64_t k = 0; k < xn[j]; k++) {
                        int64_t x = xlo[j] + k;
                        s += wx[j * kx + k] * (double)frame[(y * W + x) * 3 + c];
                    }
                    tmp[(y * w + j) * 3 + c] = s;
                }
        /* pass 2: along y */
        for (int64_t c = 0; c < 3; c++)
            for (int64_t i = 0; i < h; i++)
                for (int64_t j = 0; j < w; j++) {
                    double s = 0.0;
                    for (int64_t k = 0; k < yn[i]; k++) {
                        int64_t y = ylo[i] + k;
                        s += wy[i * ky + k] * tmp[(y * w + j) * 3 + c];
                    }
                    out[(c * h + i) * w + j] = s;
                }
        st = OR_OK;
    }
    free(xlo);
    free(xn);
    free(wx);
    free(ylo);
    free(yn);
    free(wy);
    free(tmp);
    return st;
}

/*
 * One resampled value by the direct two-dimensional sum
 *   R[c][i][j] = sum_y sum_x wy[i][y] * wx[j][x] * F[y][x][c],
 * with no separation into passes.  Used for brute-force checks and for
 * sampled outputs of large workloads.
 */
double oracle_resize_pixel(const uint8_t *frame, int64_t H, int64_t W, int64_t h, int64_t w,
                           int64_t i, int64_t j, int64_t c)
{
    double wy[4096], wx[4096];
    int64_t ylo, yn, xlo, xn;
    if (oracle_filter(H, h, i, &ylo, &yn, wy, 4096) != OR_OK)
        return NAN;
    if (oracle_filter(W, w, j, &xlo, &xn, wx, 4096) != OR_OK)
        return NAN;
    double s = 0.0;
    for (int64_t a = 0; a < yn; a++)
        for (int64_t b = 0; b < xn; b++)
            s += wy[a] * wx[b] * (double)frame[((ylo + a) * W + (xlo + b)) * 3 + c];
    return s;
}

/* ------------------------------------------------------------------------ */
/* uint8 cache writer: fixed-point resampling                               */
/* ------------------------------------------------------------------------ */

/*
 * The cache of Section 3.1.1 stores frames that are already sampled and
 * resized; kept as uint8 they are a quarter of the float tensors.  This
 * variant resamples in integers so that its bytes are reproducible exactly
 * on any machine:
 *   q_j = w_j * 2^22 rounded half away from zero   (w_j: the weights above),
 *   each pass:  out = clamp(floor((sum_j q_j * in_j + 2^21) / 2^22), 0, 255),
 * i.e. a round half up of the exact fixed-point sum, then a clamp to a byte.
 * The horizontal pass runs first, over every source row, into a uint8
 * frame of H x w; the vertical pass reads that.  An axis whose size does
 * not change is the identity (one weight of exactly 2^22).
 * Reading: these are the conventions of PIL-style integer resizers for
 * 8-bit images (22 fractional bits, horizontal pass first, a byte between
 * the passes); the CPU tests pin the result to Pillow's bicubic resize.
 */
int oracle_fixed_weights(int64_t n_in, int64_t n_out, int64_t i, int64_t *lo, int64_t *count,
                         int32_t *q, int64_t cap)
{
    if (q == NULL)
        return OR_ERR_NULL;
    double w[4096];
    if (cap > 4096)
        cap = 4096;
    int st = oracle_filter(n_in, n_out, i, lo, count, w, cap);
    if (st != OR_OK)
        return st;
    for (int64_t k = 0; k < *count; k++) {
        double x = w[k] * 4194304.0;   /* 2^22 */
        q[k] = (int32_t)(x < 0.0 ? x - 0.5 : x + 0.5);   /* truncation: half away from zero */
    }
    return OR_OK;
}

static int check_item(int64_t n_src, int64_t H, int64_t W, const int32_t *indices,
                      int64_t n_idx, int64_t h, int64_t w, int64_t patch);

static uint8_t fixed_to_byte(int64_t acc)
{
    int64_t v = acc + 2097152;   /* + 2^21: round half up */
    if (v < 0)
        return 0;
    v >>= 22;                    /* floor of a non-negative value */
    return (uint8_t)(v > 255 ? 255 : v);
}

/* One frame F[H][W][3] -> out[h][w][3], both uint8, as defined above. */
int oracle_resize_u8(const uint8_t *frame, int64_t H, int64_t W, int64_t h, int64_t w,
                     uint8_t *out)
{
    if (frame == NULL || out == NULL)
        return OR_ERR_NULL;
    if (H < 1 || W < 1 || h < 1 || w < 1)
        return OR_ERR_DIMS;
    uint8_t *mid = malloc((size_t)(H * w * 3));
    int32_t *q = malloc(sizeof(int32_t) * 4096);
    if (!mid || !q) {
        free(mid);
        free(q);
        return OR_ERR_NOMEM;
    }
    int st = OR_OK;
    /* horizontal pass: every source row */
    for (int64_t j = 0; j < w && st == OR_OK; j++) {
        int64_t lo, n;
        st = oracle_fixed_weights(W, w, j, &lo, &n, q, 4096);
        for (int64_t y = 0; y < H && st == OR_OK; y++)
            for (int64_t c = 0; c < 3; c++) {
                int64_t acc = 0;
                for (int64_t k = 0; k < n; k++)
                    acc += (int64_t)q[k] * frame[(y * W + lo + k) * 3 + c];
                mid[(y * w + j) * 3 + c] = fixed_to_byte(acc);
            }
    }
    /* vertical pass */
    for (int64_t i = 0; i < h && st == OR_OK; i++) {
        int64_t lo, n;
        st = oracle_fixed_weights(H, h, i, &lo, &n, q, 4096);
        for (int64_t j = 0; j < w && st == OR_OK; j++)
            for (int64_t c = 0; c < 3; c++) {
                int64_t acc = 0;
                for (int64_t k = 0; k < n; k++)
                    acc += (int64_t)q[k] * mid[((lo + k) * w + j) * 3 + c];
                out[(i * w + j) * 3 + c] = fixed_to_byte(acc);
            }
    }
    free(mid);
    free(q);
    return st;
}

/*
 * Whole item for the cache: frames[n_src][H][W][3] sampled at `indices` (in
 * that order, no temporal padding) and resized to out[n_idx][h][w][3].
 */
int oracle_resize_u8_item(const uint8_t *frames, int64_t n_src, int64_t H, int64_t W,
                          const int32_t *indices, int64_t n_idx, int64_t h, int64_t w,
                          int64_t patch, uint8_t *out)
{
    if (frames == NULL || out == NULL)
        return OR_ERR_NULL;
    int st = check_item(n_src, H, W, indices, n_idx, h, w, patch);
    for (int64_t k = 0; k < n_idx && st == OR_OK; k++)
        st = oracle_resize_u8(frames + (int64_t)indices[k] * H * W * 3, H, W, h, w,
                              out + k * h * w * 3);
    return st;
}

/* ------------------------------------------------------------------------ */
/* Rescale + normalise, temporal padding, patchify                          */
/* ------------------------------------------------------------------------ */

/* v = (R / 255 - mean_c) / std_c   (Section 1 names normalisation as one of
 * the costly preprocessing steps; the constants are per call). */
double oracle_normalize(double r, double mean, double std)
{
    return (r / 255.0 - mean) / std;
}

/*
 * Temporal padding: an odd index count gets its last index repeated, so an
 * image (one frame) becomes two identical frames.  Writes the padded list
 * (capacity n_idx + 1) and returns its length.
 */
static int64_t pad_indices(const int32_t *indices, int64_t n_idx, int32_t *padded)
{
    for (int64_t k = 0; k < n_idx; k++)
        padded[k] = indices[k];
    if (n_idx % 2 == 1) {
        padded[n_idx] = indices[n_idx - 1];
        return n_idx + 1;
    }
    return n_idx;
}

/*
 * Row rho and column k of the patchified output, for grid (t, hg, wg):
 *   rho = ((tt * (hg/2) + bh) * (wg/2) + bw) * 4 + mh * 2 + mw,
 *   k   = ((c * 2 + dt) * 16 + y) * 16 + x,
 *   out[rho][k] = v[frame 2*tt + dt][c][16*(2*bh + mh) + y][16*(2*bw + mw) + x].
 * Each group of four rows is one 2x2 merge window; each row is channel-major,
 * then temporal, then a 16x16 raster.  These two functions map a (rho, k)
 * pair back to (frame-in-pair, channel, pixel row, pixel column).
 */
static void decode_row(int64_t rho, int64_t hg, int64_t wg, int64_t patch, int64_t *tt,
                       int64_t *i0, int64_t *j0)
{
    int64_t hm = hg / OR_MERGE, wm = wg / OR_MERGE;
    int64_t win = rho / 4, sub = rho % 4;
    int64_t mh = sub / 2, mw = sub % 2;
    int64_t bw = win % wm;
    int64_t bh = (win / wm) % hm;
    *tt = win / (wm * hm);
    *i0 = patch * (2 * bh + mh);
    *j0 = patch * (2 * bw + mw);
}

static void decode_col(int64_t k, int64_t patch, int64_t *c, int64_t *dt, int64_t *y, int64_t *x)
{
    *x = k % patch;
    *y = (k / patch) % patch;
    *dt = (k / (patch * patch)) % OR_TPATCH;
    *c = k / (patch * patch * OR_TPATCH);
}

static int check_item(int64_t n_src, int64_t H, int64_t W, const int32_t *indices,
                      int64_t n_idx, int64_t h, int64_t w, int64_t patch)
{
    if (patch < 1)
        return OR_ERR_ARG;
    if (indices == NULL)
        return OR_ERR_NULL;
    if (n_src < 1 || H < 1 || W < 1 || h < 1 || w < 1)
        return OR_ERR_DIMS;
    if (h % (patch * OR_MERGE) != 0 || w % (patch * OR_MERGE) != 0)
        return OR_ERR_DIMS;
    if (n_idx < 1)
        return OR_ERR_FRAMES;
    for (int64_t k = 0; k < n_idx; k++)
        if (indices[k] < 0 || indices[k] >= n_src)
            return OR_ERR_INDEX;
    return OR_OK;
}

/* Number of output rows of one item: t * (h/P) * (w/P), t = ceil(n_idx/2). */
int64_t oracle_item_rows(int64_t n_idx, int64_t h, int64_t w, int64_t patch)
{
    int64_t t = (n_idx + 1) / 2;
    return t * (h / patch) * (w / patch);
}

/*
 * Whole item: frames[n_src][H][W][3] (uint8), sampled at `indices`, resized
 * to h x w, normalised, padded to an even frame count and patchified into
 * rows[oracle_item_rows][6*P*P] (double).  Frame pairs are processed one at a
 * time; the result does not depend on that order.
 */
int oracle_preprocess_item(const uint8_t *frames, int64_t n_src, int64_t H, int64_t W,
                           const int32_t *indices, int64_t n_idx, int64_t h, int64_t w,
                           int64_t patch, const double *mean, const double *std, double *rows)
{
    if (frames == NULL || mean == NULL || std == NULL || rows == NULL)
        return OR_ERR_NULL;
    int st = check_item(n_src, H, W, indices, n_idx, h, w, patch);
    if (st != OR_OK)
        return st;
    int32_t *padded = malloc(sizeof(int32_t) * (size_t)(n_idx + 1));
    double *v0 = malloc(sizeof(double) * (size_t)(3 * h * w));
    double *v1 = malloc(sizeof(double) * (size_t)(3 * h * w));
    if (!padded || !v0 || !v1) {
        free(padded);
        free(v0);
        free(v1);
        return OR_ERR_NOMEM;
    }
    int64_t n_pad = pad_indices(indices, n_idx, padded);
    int64_t t = n_pad / OR_TPATCH, hg = h / patch, wg = w / patch;
    int64_t rows_per_t = hg * wg;
    int64_t frame_bytes = H * W * 3;
    for (int64_t tt = 0; tt < t && st == OR_OK; tt++) {
        double *v[2] = {v0, v1};
        for (int64_t dt = 0; dt < 2 && st == OR_OK; dt++) {
            const uint8_t *f = frames + (int64_t)padded[2 * tt + dt] * frame_bytes;
            st = oracle_resize_frame(f, H, W, h, w, v[dt]);
            for (int64_t c = 0; c < 3 && st == OR_OK; c++)
                for (int64_t p = 0; p < h * w; p++)
                    v[dt][c * h * w + p] = oracle_normalize(v[dt][c * h * w + p], mean[c], std[c]);
        }
        for (int64_t r = 0; r < rows_per_t && st == OR_OK; r++) {
            int64_t rho = tt * rows_per_t + r;
            int64_t t_chk, i0, j0;
            decode_row(rho, hg, wg, patch, &t_chk, &i0, &j0);
            for (int64_t k = 0; k < OR_ROW(patch); k++) {
                int64_t c, dt, y, x;
                decode_col(k, patch, &c, &dt, &y, &x);
                rows[rho * OR_ROW(patch) + k] = v[dt][(c * h + (i0 + y)) * w + (j0 + x)];
            }
        }
    }
    free(padded);
    free(v0);
    free(v1);
    return st;
}

/*
 * Normalise and patchify only: the frames are already at the target size
 * h x w (the cached path of Section 3.1.1, where sampling and resizing were
 * done once offline and each RL stage still rescales, normalises and
 * patchifies).  With the padded index list and (tt, i0, j0), (c, dt, y, x)
 * decoded from (rho, k) as for the full path:
 *   rows[rho][k] = normalise(frames[padded[2 tt + dt]][i0 + y][j0 + x][c]).
 */
int oracle_patchify_item(const uint8_t *frames, int64_t n_src, int64_t h, int64_t w,
                         const int32_t *indices, int64_t n_idx, int64_t patch, const double *mean,
                         const double *std, double *rows)
{
    if (frames == NULL || mean == NULL || std == NULL || rows == NULL)
        return OR_ERR_NULL;
    int st = check_item(n_src, h, w, indices, n_idx, h, w, patch);
    if (st != OR_OK)
        return st;
    int32_t *padded = malloc(sizeof(int32_t) * (size_t)(n_idx + 1));
    if (!padded)
        return OR_ERR_NOMEM;
    pad_indices(indices, n_idx, padded);
    int64_t hg = h / patch, wg = w / patch;
    int64_t frame_bytes = h * w * 3;
    int64_t n_rows = oracle_item_rows(n_idx, h, w, patch);
    for (int64_t rho = 0; rho < n_rows; rho++) {
        int64_t tt, i0, j0;
        decode_row(rho, hg, wg, patch, &tt, &i0, &j0);
        for (int64_t k = 0; k < OR_ROW(patch); k++) {
            int64_t c, dt, y, x;
            decode_col(k, patch, &c, &dt, &y, &x);
            const uint8_t *f = frames + (int64_t)padded[2 * tt + dt] * frame_bytes;
            double r = (double)f[((i0 + y) * w + (j0 + x)) * 3 + c];
            rows[rho * OR_ROW(patch) + k] = oracle_normalize(r, mean[c], std[c]);
        }
    }
    free(padded);
    return OR_OK;
}

/*
 * One output row rho of an item, computed element by element from the
 * direct two-dimensional sum (no separable pass, no frame buffer).  Used to
 * check sampled rows of workloads too large to recompute whole.
 */
int oracle_item_row(const uint8_t *frames, int64_t n_src, int64_t H, int64_t W,
                    const int32_t *indices, int64_t n_idx, int64_t h, int64_t w, int64_t patch,
                    const double *mean, const double *std, int64_t rho, double *row)
{
    if (frames == NULL || mean == NULL || std == NULL || row == NULL)
        return OR_ERR_NULL;
    int st = check_item(n_src, H, W, indices, n_idx, h, w, patch);
    if (st != OR_OK)
        return st;
    if (rho < 0 || rho >= oracle_item_rows(n_idx, h, w, patch))
        return OR_ERR_ARG;
    int32_t *padded = malloc(sizeof(int32_t) * (size_t)(n_idx + 1));
    if (!padded)
        return OR_ERR_NOMEM;
    pad_indices(indices, n_idx, padded);
    int64_t hg = h / patch, wg = w / patch;
    int64_t tt, i0, j0;
    decode_row(rho, hg, wg, patch, &tt, &i0, &j0);
    int64_t frame_bytes = H * W * 3;
    for (int64_t k = 0; k < OR_ROW(patch); k++) {
        int64_t c, dt, y, x;
        decode_col(k, patch, &c, &dt, &y, &x);
        const uint8_t *f = frames + (int64_t)padded[2 * tt + dt] * frame_bytes;
        double r = oracle_resize_pixel(f, H, W, h, w, i0 + y, j0 + x, c);
        row[k] = oracle_normalize(r, mean[c], std[c]);
    }
    free(padded);
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Position tables (Section 1: metadata-consistent spatial-temporal         */
/* positional encoding; Section 3.1.1: the same video_grid_thw everywhere)  */
/* ------------------------------------------------------------------------ */

/*
 * For every output row rho of the batch (item b owns rows [cu[b], cu[b+1])
 * in merge-window order, decoded as in the patchify step):
 *   vit_pos[rho] = (tt, 2*bh + mh, 2*bw + mw)   frame pair, patch row, patch column
 * and for every merge window g = rho / 4 (one token after the 2x2 merge):
 *   llm_pos[g] = (tt, bh, bw).
 * The ViT attends within one frame pair of one item at a time:
 *   vit_cu[0] = 0, vit_cu[s+1] = vit_cu[s] + (h/P)*(w/P) for every frame
 *   pair s of every item in order; returns the number of pairs in *n_slices.
 * Reading: these are the grid coordinates a 2D RoPE (ViT) and a 3-axis
 * M-RoPE (LLM) take; the model's own temporal scaling and text offset are
 * applied by the model, not here.
 */
int oracle_position_ids(int64_t n_items, const int64_t *n_idx, const int64_t *h, const int64_t *w,
                        int64_t patch, int64_t *vit_pos, int64_t *llm_pos, int64_t *vit_cu,
                        int64_t *n_slices)
{
    if (n_idx == NULL || h == NULL || w == NULL || vit_pos == NULL || llm_pos == NULL ||
        vit_cu == NULL || n_slices == NULL)
        return OR_ERR_NULL;
    if (patch < 1)
        return OR_ERR_ARG;
    int64_t row = 0, slice = 0;
    vit_cu[0] = 0;
    for (int64_t b = 0; b < n_items; b++) {
        if (n_idx[b] < 1)
            return OR_ERR_FRAMES;
        if (h[b] < 2 * patch || w[b] < 2 * patch || h[b] % (2 * patch) != 0 || w[b] % (2 * patch) != 0)
            return OR_ERR_DIMS;
        int64_t hg = h[b] / patch, wg = w[b] / patch;
        int64_t n_rows = oracle_item_rows(n_idx[b], h[b], w[b], patch);
        for (int64_t r = 0; r < n_rows; r++) {
            int64_t tt, i0, j0;
            decode_row(r, hg, wg, patch, &tt, &i0, &j0);
            int64_t *v = vit_pos + 3 * (row + r);
            v[0] = tt;
            v[1] = i0 / patch;
            v[2] = j0 / patch;
            if (r % 4 == 0) {
                int64_t *l = llm_pos + 3 * ((row + r) / 4);
                l[0] = tt;
                l[1] = i0 / (patch * OR_MERGE);
                l[2] = j0 / (patch * OR_MERGE);
            }
        }
        int64_t t = (n_idx[b] + 1) / 2;
        for (int64_t k = 0; k < t; k++) {
            vit_cu[slice + 1] = vit_cu[slice] + hg * wg;
            slice++;
        }
        row += n_rows;
    }
    *n_slices = slice;
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* grid_thw and cu_seqlens (Section 3.1.1: every stage must produce the     */
/* same video_grid_thw)                                                     */
/* ------------------------------------------------------------------------ */

/*
 * grid_thw[b] = (t, h/P, w/P) with t = ceil(n_idx / 2);
 * cu[0] = 0, cu[b+1] = cu[b] + t * (h/P) * (w/P).
 */
int oracle_layout(int64_t n_items, const int64_t *n_idx, const int64_t *h, const int64_t *w,
                  int64_t patch, int64_t *grid_thw, int64_t *cu)
{
    if (n_idx == NULL || h == NULL || w == NULL || grid_thw == NULL || cu == NULL)
        return OR_ERR_NULL;
    if (patch < 1)
        return OR_ERR_ARG;
    cu[0] = 0;
    for (int64_t b = 0; b < n_items; b++) {
        if (n_idx[b] < 1)
            return OR_ERR_FRAMES;
        if (h[b] < 1 || w[b] < 1 || h[b] % (2 * patch) != 0 || w[b] % (2 * patch) != 0)
            return OR_ERR_DIMS;
        int64_t t = (n_idx[b] + 1) / 2;
        grid_thw[3 * b + 0] = t;
        grid_thw[3 * b + 1] = h[b] / patch;
        grid_thw[3 * b + 2] = w[b] / patch;
        cu[b + 1] = cu[b] + t * (h[b] / patch) * (w[b] / patch);
    }
    return OR_OK;
}
