/*
 * fp64 CPU oracle for the DiT attention hot path of xDiT (arXiv 2411.01738).
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product library calls, links or
 * includes this file; only the tests, the smoke check and the CPU-baseline leg
 * of the benchmark load it. It shares no code, header or constant with the HIP
 * path.
 *
 * It writes out the plain definitions the GPU kernels must reproduce, in
 * double precision, one query row at a time, with no tiling, no online
 * rescaling and no fusion:
 *
 *   attention      full (non-causal) multi-head self-attention softmax(s*Q K^T) V
 *                  with s = 1/sqrt(d)  (Section 2 "Diffusion Transformers";
 *                  Section 4.1.2 says DiT attention is full, not causal)
 *   chunk          the same over one K/V chunk, also returning the natural-log
 *                  log-sum-exp of the scaled scores (Section 4.1.1: SP-Ring is a
 *                  parallel FlashAttention over P2P-exchanged K/V sub-blocks)
 *   merge          recombination of chunk partials (Section 4.1.1: the sharded
 *                  computation gives the same result as the serial one)
 *   patch          PipeFusion patch step: the patch's rows of the layer's
 *                  full-sequence K/V buffer are overwritten with fresh K/V, the
 *                  rest keep stale K/V from the previous diffusion step, and the
 *                  patch's queries attend over the whole buffer
 *                  (Section 4.1.2, PipeFusion; Section 4.1.4 on storing
 *                  communicated K/V into that buffer)
 *   stage          one stage micro-step at one attention layer: QKV
 *                  projections of the patch rows, the patch step, the output
 *                  projection (Section 4.1.2; Section 3 on the projections)
 *
 * Layout (a reading: the paper does not fix one): activations are
 * sequence-major [B, N, H, d] with d contiguous; the K/V buffer is
 * [2, B, N, H, d] (plane 0 = K, plane 1 = V); LSE is [B, H, Nq].
 * Inputs are float arrays holding the values exactly as uploaded to the GPU
 * (bf16 values are exact in float); every product and sum is taken in double.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define IDX4(b, n, h, c, N, H, D) ((((int64_t)(b) * (N) + (n)) * (H) + (h)) * (D) + (c))

int xo_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void xo_set_num_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/*
 * One output row of attention, by definition:
 *   s_j   = scale * sum_c q_c k_jc
 *   m     = max_j s_j
 *   lse   = m + ln sum_j exp(s_j - m)
 *   o_c   = sum_j exp(s_j - lse) v_jc
 * With no keys, o = 0 and lse = -inf.  `s` is caller scratch of nk doubles.
 */
static void attention_row(const float* q, const float* k, const float* v,
                          int64_t nk, int64_t row_stride, int64_t d, double scale,
                          double* s, double* o, double* lse) {
    for (int64_t c = 0; c < d; ++c) o[c] = 0.0;
    if (nk == 0) {
        *lse = -INFINITY;
        return;
    }
    double m = -INFINITY;
    for (int64_t j = 0; j < nk; ++j) {
        const float* kj = k + j * row_stride;
        double dot = 0.0;
        for (int64_t c = 0; c < d; ++c) dot += (double)q[c] * (double)kj[c];
        s[j] = scale * dot;
        if (s[j] > m) m = s[j];
    }
    double l = 0.0;
    for (int64_t j = 0; j < nk; ++j) l += exp(s[j] - m);
    const double L = m + log(l);
    for (int64_t j = 0; j < nk; ++j) {
        const double p = exp(s[j] - L);
        const float* vj = v + j * row_stride;
        for (int64_t c = 0; c < d; ++c) o[c] += p * (double)vj[c];
    }
    *lse = L;
}

/*
 * Attention of the queries q [B, Nq, H, d] over keys k and values v
 * [B, Nk, H, d], scale 1/sqrt(d).
 *
 * rows: indices of the query rows to evaluate (NULL = all Nq rows in order);
 *       nrows: how many.  out is [B, nrows, H, d] and lse is [B, H, nrows],
 *       both double; lse may be NULL.
 * Returns 0, or -1 on a bad argument.
 */
int xo_attention(const float* q, const float* k, const float* v,
                 int64_t B, int64_t Nq, int64_t Nk, int64_t H, int64_t d,
                 const int64_t* rows, int64_t nrows, double* out, double* lse) {
    if (B < 0 || Nq < 0 || Nk < 0 || H < 0 || d <= 0 || nrows < 0) return -1;
    if (rows == NULL && nrows != Nq) return -1;
    for (int64_t r = 0; rows != NULL && r < nrows; ++r)
        if (rows[r] < 0 || rows[r] >= Nq) return -1;
    const double scale = 1.0 / sqrt((double)d);
    const int64_t total = B * H * nrows;
#pragma omp parallel
    {
        double* s = (double*)malloc(sizeof(double) * (size_t)(Nk > 0 ? Nk : 1));
#pragma omp for schedule(dynamic, 16)
        for (int64_t t = 0; t < total; ++t) {
            const int64_t r = t % nrows;
            const int64_t h = (t / nrows) % H;
            const int64_t b = t / (nrows * H);
            const int64_t i = rows ? rows[r] : r;
            double row_lse;
            attention_row(q + IDX4(b, i, h, 0, Nq, H, d), k + IDX4(b, 0, h, 0, Nk, H, d),
                          v + IDX4(b, 0, h, 0, Nk, H, d), Nk, H * d, d, scale, s,
                          out + IDX4(b, r, h, 0, nrows, H, d), &row_lse);
            if (lse) lse[(b * H + h) * nrows + r] = row_lse;
        }
        free(s);
    }
    return 0;
}

/*
 * Merge of n attention partials (o_r [B, Nq, H, d], lse_r [B, H, Nq]), each
 * computed over one K/V chunk, into attention over the union of the chunks:
 *   M = max_r lse_r,  L = M + ln sum_r exp(lse_r - M),
 *   o = sum_r exp(lse_r - L) o_r.
 * A partial with lse_r = -inf (an empty chunk) has weight 0; if every partial
 * is empty, o = 0 and L = -inf.
 * outs/lses: arrays of n pointers (float values as stored by the producer).
 * out [B, Nq, H, d] and lse_out [B, H, Nq] (may be NULL) are double.
 */
int xo_merge(const float* const* outs, const float* const* lses, int32_t n,
             int64_t B, int64_t Nq, int64_t H, int64_t d, double* out, double* lse_out) {
    if (n < 1 || B < 0 || Nq < 0 || H < 0 || d <= 0) return -1;
    const int64_t total = B * H * Nq;
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < total; ++t) {
        const int64_t i = t % Nq;
        const int64_t h = (t / Nq) % H;
        const int64_t b = t / (Nq * H);
        const int64_t lidx = (b * H + h) * Nq + i;
        double M = -INFINITY;
        for (int32_t r = 0; r < n; ++r)
            if ((double)lses[r][lidx] > M) M = (double)lses[r][lidx];
        double* o = out + IDX4(b, i, h, 0, Nq, H, d);
        for (int64_t c = 0; c < d; ++c) o[c] = 0.0;
        if (M == -INFINITY) {
            if (lse_out) lse_out[lidx] = -INFINITY;
            continue;
        }
        double sum = 0.0;
        for (int32_t r = 0; r < n; ++r) sum += exp((double)lses[r][lidx] - M);
        const double L = M + log(sum);
        for (int32_t r = 0; r < n; ++r) {
            const double w = exp((double)lses[r][lidx] - L);
            const float* orow = outs[r] + IDX4(b, i, h, 0, Nq, H, d);
            for (int64_t c = 0; c < d; ++c) o[c] += w * (double)orow[c];
        }
        if (lse_out) lse_out[lidx] = L;
    }
    return 0;
}

/*
 * PipeFusion patch step, update half: rows [off, off+len) of both planes of
 * kv_buf [2, B, N, H, d] are replaced by fresh_k / fresh_v [B, len, H, d];
 * every other row keeps its (stale) value.  Exact copy.
 */
int xo_patch_update(float* kv_buf, int64_t off, int64_t len, const float* fresh_k,
                    const float* fresh_v, int64_t B, int64_t N, int64_t H, int64_t d) {
    if (off < 0 || len < 0 || off + len > N || B < 0 || H < 0 || d <= 0) return -1;
    const int64_t plane = B * N * H * d;
    for (int64_t b = 0; b < B; ++b)
        for (int64_t i = 0; i < len; ++i)
            for (int64_t h = 0; h < H; ++h)
                for (int64_t c = 0; c < d; ++c) {
                    kv_buf[IDX4(b, off + i, h, c, N, H, d)] = fresh_k[IDX4(b, i, h, c, len, H, d)];
                    kv_buf[plane + IDX4(b, off + i, h, c, N, H, d)] =
                        fresh_v[IDX4(b, i, h, c, len, H, d)];
                }
    return 0;
}

/*
 * PipeFusion patch step: update kv_buf in place (above), then the patch's
 * queries q [B, len, H, d] attend over the whole updated buffer, so the fresh
 * slice is visible to this step's own attention.  rows/nrows/out/lse as in
 * xo_attention (rows index the patch's queries).
 */
int xo_patch(const float* q, float* kv_buf, int64_t off, int64_t len, const float* fresh_k,
             const float* fresh_v, int64_t B, int64_t N, int64_t H, int64_t d,
             const int64_t* rows, int64_t nrows, double* out, double* lse) {
    int rc = xo_patch_update(kv_buf, off, len, fresh_k, fresh_v, B, N, H, d);
    if (rc) return rc;
    return xo_attention(q, kv_buf, kv_buf + B * N * H * d, B, len, N, H, d, rows, nrows, out,
                        lse);
}

/*
 * Patch step with up to several fresh row ranges and its own query rows.
 *
 * Section 4.1.2: with in-context conditioning the text tokens travel with
 * patch 0, so that micro-step refreshes two row ranges of the buffer (the
 * patch's image rows and the text rows) and its queries are the rows of both.
 * Section 4.1.4: in hybrid parallelism the K/V a PipeFusion stage stores are
 * the ones gathered over its sequence-parallel group, while its queries are
 * only the local shard.
 *
 * fresh_k / fresh_v [B, F, H, d], F = sum of lens, hold the ranges' rows in
 * range order: range r takes fresh rows base_r .. base_r + len_r - 1 with
 * base_r = len_0 + ... + len_{r-1}.  Ranges must lie in [0, N) and be
 * disjoint.  After the update, q [B, Nq, H, d] attends over the whole buffer;
 * rows/nrows/out/lse as in xo_attention (rows index q).
 */
int xo_patch_ranges(const float* q, int64_t Nq, float* kv_buf, int32_t nr, const int64_t* offs,
                    const int64_t* lens, const float* fresh_k, const float* fresh_v, int64_t B,
                    int64_t N, int64_t H, int64_t d, const int64_t* rows, int64_t nrows, double* out,
                    double* lse) {
    if (nr < 0 || Nq < 0 || B < 0 || H < 0 || d <= 0) return -1;
    int64_t F = 0;
    for (int32_t r = 0; r < nr; ++r) {
        if (offs[r] < 0 || lens[r] < 0 || offs[r] + lens[r] > N) return -1;
        for (int32_t s = 0; s < r; ++s)
            if (offs[r] < offs[s] + lens[s] && offs[s] < offs[r] + lens[r]) return -1;
        F += lens[r];
    }
    const int64_t plane = B * N * H * d;
    int64_t base = 0;
    for (int32_t r = 0; r < nr; ++r) {
        for (int64_t b = 0; b < B; ++b)
            for (int64_t i = 0; i < lens[r]; ++i)
                for (int64_t h = 0; h < H; ++h)
                    for (int64_t c = 0; c < d; ++c) {
                        const int64_t dst = IDX4(b, offs[r] + i, h, c, N, H, d);
                        const int64_t src = IDX4(b, base + i, h, c, F, H, d);
                        kv_buf[dst] = fresh_k[src];
                        kv_buf[plane + dst] = fresh_v[src];
                    }
        base += lens[r];
    }
    return xo_attention(q, kv_buf, kv_buf + plane, B, Nq, N, H, d, rows, nrows, out, lse);
}

/*
 * attention_row over double keys and values (the stage step's fresh rows are
 * projections, not values of the I/O type).  Same definition as above.
 */
static void attention_row_d(const double* q, const double* k, const double* v, int64_t nk,
                            int64_t row_stride, int64_t d, double scale, double* s, double* o) {
    for (int64_t c = 0; c < d; ++c) o[c] = 0.0;
    if (nk == 0) return;
    double m = -INFINITY;
    for (int64_t j = 0; j < nk; ++j) {
        const double* kj = k + j * row_stride;
        double dot = 0.0;
        for (int64_t c = 0; c < d; ++c) dot += q[c] * kj[c];
        s[j] = dot * scale;
        if (s[j] > m) m = s[j];
    }
    double l = 0.0;
    for (int64_t j = 0; j < nk; ++j) l += exp(s[j] - m);
    const double lse_j = m + log(l);
    for (int64_t j = 0; j < nk; ++j) {
        const double p = exp(s[j] - lse_j);
        const double* vj = v + j * row_stride;
        for (int64_t c = 0; c < d; ++c) o[c] += p * vj[c];
    }
}

/*
 * One PipeFusion stage micro-step at one attention layer (Section 4.1.2: a
 * device runs a patch through its layers; Section 3: the QKV projections
 * come before self-attention, and the attention output is projected back):
 *
 *   q = x Wq,  k = x Wk,  v = x Wv      x [B, L, C], W [C, H*d]
 *   patch step: rows [off, off+L) of the buffer take (k, v); the patch's
 *               queries attend over the whole buffer (stale rows elsewhere)
 *   y = o Wo                            o [B, L, H*d], Wo [H*d, C]
 *
 * No biases, norms or gates.  Products and sums in double; the fresh rows
 * are stored into kv_buf rounded to float (kv_buf [2, B, N, H, d] in/out).
 * rows/nrows select the patch rows whose outputs are evaluated (NULL = all
 * L in order); y is [B, nrows, C] and o (may be NULL) [B, nrows, H, d],
 * double; pq/pk/pv (each may be NULL) receive q/k/v [B, L, H, d], double.
 */
int xo_stage(const float* x, const float* wq, const float* wk, const float* wv, const float* wo,
             float* kv_buf, int64_t off, int64_t L, int64_t B, int64_t N, int64_t H, int64_t d,
             int64_t C, const int64_t* rows, int64_t nrows, double* y, double* o, double* pq,
             double* pk, double* pv) {
    if (B < 0 || L < 0 || N < 0 || H <= 0 || d <= 0 || C <= 0 || nrows < 0) return -1;
    if (off < 0 || off + L > N) return -1;
    if (rows == NULL && nrows != L) return -1;
    for (int64_t r = 0; rows != NULL && r < nrows; ++r)
        if (rows[r] < 0 || rows[r] >= L) return -1;
    const int64_t HD = H * d, plane = B * N * HD;
    double* q = (double*)malloc(sizeof(double) * (size_t)(B * L * HD + 1));
    double* kd = (double*)malloc(sizeof(double) * (size_t)(B * N * HD + 1));
    double* vd = (double*)malloc(sizeof(double) * (size_t)(B * N * HD + 1));
    double* ob = (double*)malloc(sizeof(double) * (size_t)(B * nrows * HD + 1));
    if (!q || !kd || !vd || !ob) {
        free(q); free(kd); free(vd); free(ob);
        return -2;
    }
    /* stale rows of the buffer, then the projections of the patch rows */
    for (int64_t t = 0; t < plane; ++t) {
        kd[t] = (double)kv_buf[t];
        vd[t] = (double)kv_buf[plane + t];
    }
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < B * L; ++t) {
        const int64_t b = t / L, i = t % L;
        const float* xr = x + t * C;
        double* qr = q + t * HD;
        double* kr = kd + (b * N + off + i) * HD;
        double* vr = vd + (b * N + off + i) * HD;
        for (int64_t n = 0; n < HD; ++n) {
            double sq = 0.0, sk = 0.0, sv = 0.0;
            for (int64_t c = 0; c < C; ++c) {
                sq += (double)xr[c] * (double)wq[c * HD + n];
                sk += (double)xr[c] * (double)wk[c * HD + n];
                sv += (double)xr[c] * (double)wv[c * HD + n];
            }
            qr[n] = sq;
            kr[n] = sk;
            vr[n] = sv;
        }
    }
    for (int64_t b = 0; b < B; ++b)
        for (int64_t i = 0; i < L; ++i)
            for (int64_t n = 0; n < HD; ++n) {
                const int64_t at = (b * N + off + i) * HD + n;
                kv_buf[at] = (float)kd[at];
                kv_buf[plane + at] = (float)vd[at];
                if (pq) pq[(b * L + i) * HD + n] = q[(b * L + i) * HD + n];
                if (pk) pk[(b * L + i) * HD + n] = kd[at];
                if (pv) pv[(b * L + i) * HD + n] = vd[at];
            }
    const double inv_sqrt_d = 1.0 / sqrt((double)d);
    const int64_t total = B * H * nrows;
#pragma omp parallel
    {
        double* s = (double*)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
#pragma omp for schedule(dynamic, 16)
        for (int64_t t = 0; t < total; ++t) {
            const int64_t r = t % nrows;
            const int64_t h = (t / nrows) % H;
            const int64_t b = t / (nrows * H);
            const int64_t i = rows ? rows[r] : r;
            attention_row_d(q + (b * L + i) * HD + h * d, kd + b * N * HD + h * d,
                            vd + b * N * HD + h * d, N, HD, d, inv_sqrt_d, s,
                            ob + (b * nrows + r) * HD + h * d);
        }
        free(s);
    }
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < B * nrows; ++t) {
        const double* orow = ob + t * HD;
        for (int64_t c = 0; c < C; ++c) {
            double acc = 0.0;
            for (int64_t n = 0; n < HD; ++n) acc += orow[n] * (double)wo[n * C + c];
            y[t * C + c] = acc;
        }
        if (o)
            for (int64_t n = 0; n < HD; ++n) o[t * HD + n] = orow[n];
    }
    free(q); free(kd); free(vd); free(ob);
    return 0;
}
