/*
 * VoxZip oracle: a plain, slow, fp64 CPU implementation of the hot path of
 * "VoxZip: Semantic-Anchored Temporal KV Cache Compression for Long-Context
 * Audio Inference" (arXiv 2608.08569).
 *
 * TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's
 * CPU-baseline leg may load this library.  The product path (the HIP library
 * under paper_2608_08569_amd/) never calls it, and the two share no code.
 *
 * Every routine reads the same stored bytes the GPU reads (float32, or
 * bfloat16 bits that are widened exactly) and computes in double precision,
 * in the order the paper's equations state, with no blocking or fusion.
 *
 *   orc_fuse          Sec. 3.2.1, Eq. (4) group average pooling, applied per
 *                     layer and KV head to K and V, plus the optional additive
 *                     anchor of the same subsection; Eq. (5) ordering is the
 *                     span order of the offsets.
 *   orc_decode_step   Sec. 3.1 Eq. (1) append, Eq. (2) attention, and
 *                     Sec. 3.2.2 Eq. (6) decayed accumulated score, per layer.
 *   orc_evict_select  Sec. 3.2.2: sink window T, recent window M (20% of the
 *                     budget), Eq. (9) top-N of the middle, Eq. (7)-(8) concat.
 *   orc_build_offsets Sec. 3.2.1: confidence filter, Eq. (3) time -> index,
 *                     uniform partition into groups, background intervals.
 *
 * Readings where the paper is silent (each is listed in the design notes):
 *   - multi-head: query head h reads KV head floor(h * Hkv / Hq); the score
 *     sums the softmax rows of all query heads of the layer;
 *   - the new token is appended before attending and gets score 0 before the
 *     fold (the zero pad of Eq. (6));
 *   - sinks are positions < T, recent are positions >= next_pos - M, ties in
 *     the top-N go to the smaller position, kept rows are in ascending position;
 *   - groups of a semantic interval of length n split into g = min(L_t, n)
 *     non-overlapping runs with boundaries s + floor(j * n / g).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_F32 = 0, ORC_BF16 = 1 };
enum { ORC_OK = 0, ORC_EINVAL = -1 };

static double ld(const void *base, int dtype, size_t i)
{
    if (dtype == ORC_F32)
        return (double)((const float *)base)[i];
    uint32_t bits = (uint32_t)((const uint16_t *)base)[i] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

int orc_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of the later parallel loops (timing only; the results do not
 * depend on it: every loop iteration is one layer, summed in its own order). */
void orc_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Eq. (4): out[l][h][j][:] = (1/|G_j|) * sum_{k in G_j} x[l][h][k][:], where
 * G_j = [off[j], off[j+1]); then + anchor[l][h][j][:] when an anchor is given. */
int orc_fuse(const void *x, int32_t T_in, const int32_t *off, int32_t n_spans,
             const void *anchor, int32_t L, int32_t H, int32_t d, int32_t dtype,
             double *out)
{
    if (n_spans < 0 || T_in < 0 || L < 1 || H < 1 || d < 1)
        return ORC_EINVAL;
    if (off[0] != 0 || off[n_spans] != T_in)
        return ORC_EINVAL;
    for (int32_t j = 0; j < n_spans; ++j)
        if (off[j + 1] <= off[j])
            return ORC_EINVAL;
#pragma omp parallel for schedule(dynamic)
    for (int32_t l = 0; l < L; ++l) {
        for (int32_t h = 0; h < H; ++h) {
            size_t in_base = ((size_t)l * H + h) * (size_t)T_in * d;
            size_t out_base = ((size_t)l * H + h) * (size_t)n_spans * d;
            for (int32_t j = 0; j < n_spans; ++j) {
                int32_t count = off[j + 1] - off[j];
                for (int32_t c = 0; c < d; ++c) {
                    double sum = 0.0;
                    for (int32_t k = off[j]; k < off[j + 1]; ++k)
                        sum += ld(x, dtype, in_base + (size_t)k * d + c);
                    double mean = sum / (double)count;
                    if (anchor)
                        mean += ld(anchor, dtype, out_base + (size_t)j * d + c);
                    out[out_base + (size_t)j * d + c] = mean;
                }
            }
        }
    }
    return ORC_OK;
}

/* One decode step for every layer, from the pre-step state.
 *
 * Inputs: q [L][Hq][d]; k_new, v_new [L][Hkv][d]; k_cache, v_cache
 * [L][Hkv][cap][d] with slots 0..len-1 resident; score_in [L][cap] (fp64);
 * pos_in [L][cap].  Outputs: out [L][Hq][d]; score_out, pos_out [L][len+1]
 * for slots 0..len (slot len is the appended token); p_out (optional)
 * [L][Hq][len+1] holds the softmax rows.
 */
int orc_decode_step(const void *q, const void *k_new, const void *v_new,
                    const void *k_cache, const void *v_cache,
                    const double *score_in, const int32_t *pos_in,
                    int32_t len, int32_t next_pos, double gamma, double sm_scale,
                    int32_t L, int32_t Hq, int32_t Hkv, int32_t d, int32_t cap,
                    int32_t dtype, double *out, double *score_out,
                    int32_t *pos_out, double *p_out)
{
    if (L < 1 || Hq < 1 || Hkv < 1 || d < 1 || Hq % Hkv != 0 || len < 0 || len + 1 > cap)
        return ORC_EINVAL;
    if (!(sm_scale > 0.0))
        sm_scale = 1.0 / sqrt((double)d);
    const int32_t T = len + 1;
#pragma omp parallel for schedule(dynamic)
    for (int32_t l = 0; l < L; ++l) {
        double *s = (double *)malloc(sizeof(double) * (size_t)T);
        double *psum = (double *)calloc((size_t)T, sizeof(double));
        for (int32_t h = 0; h < Hq; ++h) {
            const int32_t g = (int32_t)(((int64_t)h * Hkv) / Hq);
            const size_t qb = ((size_t)l * Hq + h) * d;
            const size_t cb = ((size_t)l * Hkv + g) * (size_t)cap * d;
            const size_t nb = ((size_t)l * Hkv + g) * d;
            /* Eq. (1): K_t = [K_{t-1}, k_t]; row T-1 is the appended key. */
            for (int32_t j = 0; j < T; ++j) {
                double dot = 0.0;
                for (int32_t c = 0; c < d; ++c) {
                    double kv = (j < len) ? ld(k_cache, dtype, cb + (size_t)j * d + c)
                                          : ld(k_new, dtype, nb + c);
                    dot += ld(q, dtype, qb + c) * kv;
                }
                s[j] = dot * sm_scale;
            }
            /* Eq. (2): softmax over all T keys, then o = p V_t. */
            double m = s[0];
            for (int32_t j = 1; j < T; ++j)
                if (s[j] > m)
                    m = s[j];
            double z = 0.0;
            for (int32_t j = 0; j < T; ++j) {
                s[j] = exp(s[j] - m);
                z += s[j];
            }
            for (int32_t j = 0; j < T; ++j)
                s[j] /= z;
            for (int32_t c = 0; c < d; ++c) {
                double acc = 0.0;
                for (int32_t j = 0; j < T; ++j) {
                    double vv = (j < len) ? ld(v_cache, dtype, cb + (size_t)j * d + c)
                                          : ld(v_new, dtype, nb + c);
                    acc += s[j] * vv;
                }
                out[qb + c] = acc;
            }
            for (int32_t j = 0; j < T; ++j)
                psum[j] += s[j];
            if (p_out)
                for (int32_t j = 0; j < T; ++j)
                    p_out[((size_t)l * Hq + h) * T + j] = s[j];
        }
        /* Eq. (6): A^(t) = gamma * [A^(t-1), 0] + sum_h softmax_h. */
        for (int32_t j = 0; j < T; ++j) {
            double prev = (j < len) ? score_in[(size_t)l * cap + j] : 0.0;
            score_out[(size_t)l * T + j] = gamma * prev + psum[j];
            pos_out[(size_t)l * T + j] = (j < len) ? pos_in[(size_t)l * cap + j] : next_pos;
        }
        free(psum);
        free(s);
    }
    return ORC_OK;
}

/* ---- eviction ------------------------------------------------------------ */
typedef struct {
    double score;
    int32_t pos;
    int32_t slot;
} orc_cand;

/* Eq. (9) order: larger score first; equal scores keep the smaller position. */
static int by_score_desc(const void *a, const void *b)
{
    const orc_cand *x = (const orc_cand *)a, *y = (const orc_cand *)b;
    if (x->score > y->score)
        return -1;
    if (x->score < y->score)
        return 1;
    return (x->pos > y->pos) - (x->pos < y->pos);
}

static int by_pos_asc(const void *a, const void *b)
{
    const orc_cand *x = (const orc_cand *)a, *y = (const orc_cand *)b;
    return (x->pos > y->pos) - (x->pos < y->pos);
}

/* Kept slots per layer, ascending by position: sinks (pos < n_sink), the
 * top-N middle slots by score, and the recent window (pos >= next_pos - M),
 * with N = budget - |sinks| - |recent|.  When len <= budget every slot is kept.
 * keep_slot is [L][budget] (entries past new_len are -1). */
int orc_evict_select(const double *score, const int32_t *pos, int32_t len,
                     int32_t budget, int32_t n_sink, int32_t n_recent,
                     int32_t next_pos, int32_t L, int32_t cap,
                     int32_t *keep_slot, int32_t *new_len)
{
    if (L < 1 || len < 0 || len > cap || budget < 1 || n_sink < 0)
        return ORC_EINVAL;
    const int32_t M = n_recent < 0 ? budget / 5 : n_recent;
    if (n_sink + M > budget)
        return ORC_EINVAL;
    int err = 0;
    int32_t kept_len = len <= budget ? len : budget;
    for (int32_t l = 0; l < L; ++l) {
        orc_cand *all = (orc_cand *)malloc(sizeof(orc_cand) * (size_t)(len > 0 ? len : 1));
        orc_cand *mid = (orc_cand *)malloc(sizeof(orc_cand) * (size_t)(len > 0 ? len : 1));
        int32_t n_keep = 0, n_mid = 0;
        for (int32_t j = 0; j < len; ++j) {
            orc_cand c = {score[(size_t)l * cap + j], pos[(size_t)l * cap + j], j};
            if (len <= budget || c.pos < n_sink || c.pos >= next_pos - M)
                all[n_keep++] = c;
            else
                mid[n_mid++] = c;
        }
        int32_t n_top = budget - n_keep;
        if (len > budget) {
            if (n_top < 0) {
                err = 1;
                n_top = 0;
            }
            if (n_top > n_mid)
                n_top = n_mid;
            qsort(mid, (size_t)n_mid, sizeof(orc_cand), by_score_desc);
            for (int32_t i = 0; i < n_top; ++i)
                all[n_keep++] = mid[i];
        }
        qsort(all, (size_t)n_keep, sizeof(orc_cand), by_pos_asc);
        for (int32_t i = 0; i < budget; ++i)
            keep_slot[(size_t)l * budget + i] = i < n_keep ? all[i].slot : -1;
        if (l == 0)
            kept_len = n_keep;
        else if (n_keep != kept_len)
            err = 1;
        free(mid);
        free(all);
    }
    *new_len = kept_len;
    return err ? ORC_EINVAL : ORC_OK;
}

/* ---- Stage-1 span offsets ------------------------------------------------- */
typedef struct {
    int64_t s, e;
    int32_t lt;
    int32_t idx; /* input order, the last tie-break: the order is total */
} orc_seg;

static int seg_by_start(const void *a, const void *b)
{
    const orc_seg *x = (const orc_seg *)a, *y = (const orc_seg *)b;
    if (x->s != y->s)
        return (x->s > y->s) - (x->s < y->s);
    if (x->e != y->e)
        return (x->e > y->e) - (x->e < y->e);
    return (x->idx > y->idx) - (x->idx < y->idx);
}

/* Span offsets for the compressed sequence of Eq. (5).
 * Segments with confidence above the threshold are kept; Eq. (3) maps each
 * timestamp to floor(L_a * tau / tau_total) (exact in 64-bit integers);
 * segments are taken in start order (then end, then input order), a start
 * inside the previous segment is moved to its end, empty ones are dropped.  A semantic interval [s, e) of
 * length n becomes g = min(L_t, n) groups; every uncovered token is a
 * background span of length 1.  off_out needs room for L_a + 1 entries. */
int orc_build_offsets(const int64_t *t_start_ms, const int64_t *t_end_ms,
                      const float *conf, const int32_t *text_len, int32_t n_seg,
                      int64_t t_total_ms, int32_t L_a, float conf_threshold,
                      int32_t *off_out, int32_t *n_spans_out)
{
    if (n_seg < 0 || t_total_ms <= 0 || L_a < 0)
        return ORC_EINVAL;
    orc_seg *seg = (orc_seg *)malloc(sizeof(orc_seg) * (size_t)(n_seg > 0 ? n_seg : 1));
    int32_t n = 0;
    for (int32_t i = 0; i < n_seg; ++i) {
        if (!(conf[i] > conf_threshold))
            continue;
        int64_t ts = t_start_ms[i], te = t_end_ms[i];
        if (ts < 0)
            ts = 0;
        if (te > t_total_ms)
            te = t_total_ms;
        if (te <= ts)
            continue;
        orc_seg sg = {((int64_t)L_a * ts) / t_total_ms, ((int64_t)L_a * te) / t_total_ms,
                      text_len[i], i};
        seg[n++] = sg;
    }
    qsort(seg, (size_t)n, sizeof(orc_seg), seg_by_start);
    int32_t k = 0;     /* spans written */
    int64_t cur = 0;   /* first token not yet covered */
    off_out[0] = 0;
    for (int32_t i = 0; i < n; ++i) {
        int64_t s = seg[i].s < cur ? cur : seg[i].s;
        int64_t e = seg[i].e;
        if (e <= s || seg[i].lt < 1)
            continue;
        for (int64_t t = cur; t < s; ++t)  /* background tokens before it */
            off_out[++k] = (int32_t)(t + 1);
        int64_t len = e - s;
        int64_t g = seg[i].lt < len ? seg[i].lt : len;
        for (int64_t j = 1; j <= g; ++j)
            off_out[++k] = (int32_t)(s + (j * len) / g);
        cur = e;
    }
    for (int64_t t = cur; t < L_a; ++t)
        off_out[++k] = (int32_t)(t + 1);
    *n_spans_out = k;
    free(seg);
    return ORC_OK;
}
